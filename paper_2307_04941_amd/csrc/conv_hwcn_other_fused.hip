// Instantiations of the implicit-GEMM kernel with the fused output stage
// (y = act(conv + add)) for the channel-vector, scalar-patch and scalar-filter loader pairs,
// one per tile shape.
#include "conv_kernel.h"

namespace mg3m {

KernelFn conv_kernel_hwcn_other_fused(int variant, int tile) {
  switch (variant) {
    case kVarHwcnVecC: return kernel_for_tile<kHWCN, kAVecM, kBVecC, true>(tile);
    case kVarHwcnVecA: return kernel_for_tile<kHWCN, kAVecM, kBScalar, true>(tile);
    case kVarHwcnScalar: return kernel_for_tile<kHWCN, kAScalar, kBScalar, true>(tile);
    default: return nullptr;
  }
}

}  // namespace mg3m
