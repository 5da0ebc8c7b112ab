// Instantiations of the implicit-GEMM kernel for the NCHW layout (Eq. 1's
// index order): vectorised or element-wise filter loads, and input patches
// loaded as 16-byte runs along W where four output columns allow it (else
// per column), one per tile shape.
#include "conv_kernel.h"

namespace mg3m {

KernelFn conv_kernel_nchw(int variant, int tile) {
  if (variant == kVarNchwVecA) return kernel_for_tile<kNCHW, kAVecK, kBVecW>(tile);
  if (variant == kVarNchwScalar) return kernel_for_tile<kNCHW, kAScalar, kBVecW>(tile);
  return nullptr;
}

}  // namespace mg3m
