// Max pooling for the network executor: the pooling layers between the
// convolution blocks of VGG, AlexNet and ResNet, kept on the device between
// the convolutions.  Window R x S, stride (sh, sw), padding (ph, pw) with
// padded taps ignored; output size by the same floor formula as the
// convolution.  A NaN in a window makes that output NaN.  HBM-bound: each
// input element is read about (R/sh)*(S/sw) times, mostly from L2.
#include <hip/hip_runtime.h>

#include <string>

#include "mg3m.h"
#include "mg3m_internal.h"

namespace mg3m {

typedef float f32x4p __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float max_nan(float a, float b) { return (b > a || b != b) ? b : a; }

// HWCN: x[H][W][C][N], y[Ho][Wo][C][N].  The C*N values of one pixel are
// contiguous, so one thread takes four of them for one output pixel (vec4)
// or one (C*N not a multiple of 4 or unaligned buffers).
template <bool VEC4>
__global__ __launch_bounds__(256) void maxpool_hwcn(PArgs p) {
  const long long cn = (long long)p.C * p.N;
  const long long per_pix = VEC4 ? cn / 4 : cn;
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= per_pix * p.Ho * p.Wo) return;
  const long long pix = i / per_pix;
  const long long e = (i - pix * per_pix) * (VEC4 ? 4 : 1);
  const int ho = (int)(pix / p.Wo), wo = (int)(pix - (long long)ho * p.Wo);
  const int ih0 = ho * p.sh - p.ph, iw0 = wo * p.sw - p.pw;
  f32x4p m = {-__builtin_inff(), -__builtin_inff(), -__builtin_inff(), -__builtin_inff()};
  for (int r = 0; r < p.R; ++r) {
    const int ih = ih0 + r;
    if ((unsigned)ih >= (unsigned)p.H) continue;
    for (int s = 0; s < p.S; ++s) {
      const int iw = iw0 + s;
      if ((unsigned)iw >= (unsigned)p.W) continue;
      const float* src = p.x + ((long long)ih * p.W + iw) * cn + e;
      if constexpr (VEC4) {
        const f32x4p v = *reinterpret_cast<const f32x4p*>(src);
#pragma unroll
        for (int q = 0; q < 4; ++q) m[q] = max_nan(m[q], v[q]);
      } else {
        m[0] = max_nan(m[0], *src);
      }
    }
  }
  float* dst = p.y + pix * cn + e;
  if constexpr (VEC4) *reinterpret_cast<f32x4p*>(dst) = m;
  else *dst = m[0];
}

// NCHW: x[N][C][H][W], y[N][C][Ho][Wo]; one output per thread, consecutive
// threads along Wo.
__global__ __launch_bounds__(256) void maxpool_nchw(PArgs p) {
  const long long hw = (long long)p.Ho * p.Wo;
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= hw * p.C * p.N) return;
  const long long plane = i / hw;
  const int pix = (int)(i - plane * hw);
  const int ho = pix / p.Wo, wo = pix - ho * p.Wo;
  const int ih0 = ho * p.sh - p.ph, iw0 = wo * p.sw - p.pw;
  const float* src = p.x + plane * p.H * p.W;
  float m = -__builtin_inff();
  for (int r = 0; r < p.R; ++r) {
    const int ih = ih0 + r;
    if ((unsigned)ih >= (unsigned)p.H) continue;
    for (int s = 0; s < p.S; ++s) {
      const int iw = iw0 + s;
      if ((unsigned)iw < (unsigned)p.W) m = max_nan(m, src[(long long)ih * p.W + iw]);
    }
  }
  p.y[i] = m;
}

int launch_maxpool(const PArgs& p, void* stream, std::string* err) {
  const long long outs = (long long)p.N * p.C * p.Ho * p.Wo;
  const bool vec4 = p.layout == kHWCN && ((long long)p.C * p.N) % 4 == 0 && p.aligned16;
  const long long threads = vec4 ? outs / 4 : outs;
  const long long blocks = (threads + 255) / 256;
  if (blocks < 1 || blocks > 0x7fffffffLL) {
    *err = "max pooling: output too large for one launch";
    return MG3M_ERR_TOO_LARGE;
  }
  if (p.layout == kHWCN) {
    if (vec4)
      hipLaunchKernelGGL(maxpool_hwcn<true>, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, p);
    else
      hipLaunchKernelGGL(maxpool_hwcn<false>, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, p);
  } else {
    hipLaunchKernelGGL(maxpool_nchw, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, p);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    *err = std::string("max pooling launch: ") + hipGetErrorString(e);
    return MG3M_ERR_HIP;
  }
  return MG3M_OK;
}

}  // namespace mg3m
