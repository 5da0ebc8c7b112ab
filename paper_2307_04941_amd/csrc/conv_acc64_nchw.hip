// Instantiations of the fp64-accumulating kernel for the NCHW layout (vector
// or scalar filter loads; patches as 16-byte runs along W where possible),
// one per tile of the fp64 menu.
#include "conv_kernel.h"

namespace mg3m {

KernelFn conv_kernel64_nchw(int variant, int tile) {
  switch (variant) {
    case kVarNchwVecA: return kernel64_for_tile<kNCHW, kAVecK, kBVecW>(tile);
    case kVarNchwScalar: return kernel64_for_tile<kNCHW, kAScalar, kBVecW>(tile);
    case kVarNchwTap: return kernel64_for_tile<kNCHW, kAVecM, kBVecWTap>(tile);
    default: return nullptr;
  }
}

}  // namespace mg3m
