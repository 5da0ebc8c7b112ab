// Instantiations of the implicit-GEMM kernel with the fused output stage
// (y = act(conv + add)) for both NCHW loader pairs,
// one per tile shape.
#include "conv_kernel.h"

namespace mg3m {

KernelFn conv_kernel_nchw_fused(int variant, int tile) {
  if (variant == kVarNchwVecA) return kernel_for_tile<kNCHW, kAVecK, kBVecW, true>(tile);
  if (variant == kVarNchwScalar) return kernel_for_tile<kNCHW, kAScalar, kBVecW, true>(tile);
  return nullptr;
}

}  // namespace mg3m
