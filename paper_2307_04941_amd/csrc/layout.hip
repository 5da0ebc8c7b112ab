// Layout change for the network executor: out[b][c][a] = in[a][c][b].  With
// (A, Cm, B) = (N, C, H*W) it takes an NCHW tensor to HWCN; with (H*W, C, N)
// it takes HWCN back to NCHW.  NCHW networks run every layer in HWCN (the
// tuned layout) and change layout only at their input and output, and an
// NCHW call whose plan runs it as HWCN changes x, then y, the same way (with
// the fused output stage applied on the way back).
#include <hip/hip_runtime.h>

#include <string>

#include "mg3m.h"
#include "mg3m_internal.h"

namespace {

// One work-group moves a 64 x 64 block of (a, b) for one c through LDS, so
// the reads run along b and the writes along a, both 256 contiguous bytes
// per row.  The extra column keeps the transposed reads off one bank.
__global__ __launch_bounds__(256) void swap_outer_inner(const float* __restrict__ in, float* out, int A, int Cm,
                                                        int B, const float* add, int relu) {
  __shared__ float t[64][65];
  const int b0 = (int)blockIdx.x * 64, a0 = (int)blockIdx.y * 64, c = (int)blockIdx.z;
  const int tx = (int)(threadIdx.x & 63), ty = (int)(threadIdx.x >> 6);
  for (int i = ty; i < 64; i += 4) {
    const int a = a0 + i, b = b0 + tx;
    if (a < A && b < B) t[i][tx] = in[((size_t)a * Cm + c) * B + b];
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const int b = b0 + i, a = a0 + tx;
    if (a < A && b < B) {
      const size_t o = ((size_t)b * Cm + c) * A + a;
      float v = t[tx][i];
      if (add != nullptr) v += add[o];          // add may be out itself: read before the write
      out[o] = (relu != 0 && v < 0.f) ? 0.f : v;  // ReLU keeps NaN
    }
  }
}

}  // namespace

namespace mg3m {

int launch_swap_outer_inner(const float* in, float* out, int A, int Cm, int B, void* stream, std::string* err,
                            const float* add, int relu) {
  if (A < 1 || Cm < 1 || B < 1) {
    *err = "internal: empty layout change";
    return MG3M_ERR_SHAPE;
  }
  const long long ta = (A + 63) / 64, tb = (B + 63) / 64;
  if (ta > 65535 || Cm > 65535 || tb > 0x7fffffffLL) {
    *err = "layout change: a dimension exceeds the launch grid";
    return MG3M_ERR_TOO_LARGE;
  }
  hipLaunchKernelGGL(swap_outer_inner, dim3((unsigned)tb, (unsigned)ta, (unsigned)Cm), dim3(256), 0,
                     static_cast<hipStream_t>(stream), in, out, A, Cm, B, add, relu);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    *err = std::string("layout change launch: ") + hipGetErrorString(e);
    return MG3M_ERR_HIP;
  }
  return MG3M_OK;
}

}  // namespace mg3m
