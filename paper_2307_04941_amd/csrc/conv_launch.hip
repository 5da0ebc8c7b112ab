// Kernel launch: picks the instantiation for a plan's loader variant and
// tile, and the deterministic split-K reduction.
#include <hip/hip_runtime.h>

#include <string>

#include "mg3m.h"
#include "mg3m_internal.h"

namespace mg3m {

typedef float f32x4r __attribute__((ext_vector_type(4)));

// Split-K reduction: y = sum over splits of the partials, in split order, so
// the result does not depend on scheduling.
__global__ __launch_bounds__(256) void splitk_reduce_f32(const float* __restrict__ ws,
                                                         float* __restrict__ y, long long elems,
                                                         int split, int vec4) {
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (vec4) {
    const long long e = i * 4;
    if (e >= elems) return;
    f32x4r s = *reinterpret_cast<const f32x4r*>(ws + e);
    for (int p = 1; p < split; ++p) s += *reinterpret_cast<const f32x4r*>(ws + (long long)p * elems + e);
    *reinterpret_cast<f32x4r*>(y + e) = s;
  } else {
    if (i >= elems) return;
    float s = ws[i];
    for (int p = 1; p < split; ++p) s += ws[(long long)p * elems + i];
    y[i] = s;
  }
}

static KernelFn kernel_for(int variant, int tile) {
  switch (variant) {
    case kVarHwcnVecN: return conv_kernel_hwcn_vecn(tile);
    case kVarHwcnVecNTap: return conv_kernel_hwcn_vecn_tap(tile);
    case kVarHwcnVecC: return conv_kernel_hwcn_vecc(tile);
    case kVarHwcnVecA: return conv_kernel_hwcn_veca(tile);
    case kVarHwcnScalar: return conv_kernel_hwcn_scalar(tile);
    case kVarNchwVecA:
    case kVarNchwScalar: return conv_kernel_nchw(variant, tile);
    default: return nullptr;
  }
}

int launch_conv(const Plan& p, const KArgs& a, void* stream, std::string* err) {
  KernelFn fn = kernel_for(p.variant, p.tile);
  if (fn == nullptr) {
    *err = "internal: no kernel for this loader variant and tile";
    return MG3M_ERR_PLAN;
  }
  if (p.grid < 1 || p.grid > 0x7fffffffLL) {
    *err = "internal: grid size out of range";
    return MG3M_ERR_PLAN;
  }
  hipLaunchKernelGGL(fn, dim3((unsigned)p.grid), dim3(p.t.wm * p.t.wn * 64), 0,
                     (hipStream_t)stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    *err = std::string("kernel launch: ") + hipGetErrorString(e);
    return MG3M_ERR_HIP;
  }
  return MG3M_OK;
}

int launch_splitk_reduce(const float* ws, float* y, long long elems, int split, bool vec4,
                         void* stream, std::string* err) {
  const long long threads = vec4 ? (elems + 3) / 4 : elems;
  const long long blocks = (threads + 255) / 256;
  if (blocks < 1 || blocks > 0x7fffffffLL) {
    *err = "internal: reduction grid out of range";
    return MG3M_ERR_PLAN;
  }
  hipLaunchKernelGGL(splitk_reduce_f32, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream,
                     ws, y, elems, split, vec4 ? 1 : 0);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    *err = std::string("split-K reduction launch: ") + hipGetErrorString(e);
    return MG3M_ERR_HIP;
  }
  return MG3M_OK;
}

}  // namespace mg3m
