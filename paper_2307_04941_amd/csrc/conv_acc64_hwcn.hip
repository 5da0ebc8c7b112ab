// Instantiations of the fp64-accumulating kernel for the other HWCN loader
// pairs (batch vectors without the one-tap slab, channel vectors, scalar
// patches, scalar filter), one per tile of the fp64 menu.
#include "conv_kernel.h"

namespace mg3m {

KernelFn conv_kernel64_hwcn(int variant, int tile) {
  switch (variant) {
    case kVarHwcnVecN: return kernel64_for_tile<kHWCN, kAVecM, kBVecN>(tile);
    case kVarHwcnVecC: return kernel64_for_tile<kHWCN, kAVecM, kBVecC>(tile);
    case kVarHwcnVecA: return kernel64_for_tile<kHWCN, kAVecM, kBScalar>(tile);
    case kVarHwcnScalar: return kernel64_for_tile<kHWCN, kAScalar, kBScalar>(tile);
    default: return nullptr;
  }
}

}  // namespace mg3m
