// Instantiations of the implicit-GEMM kernel with the fused output stage
// (y = act(conv + add)) for the one-tap HWCN loaders in their direct-to-LDS
// form (AVecMTapDma, BVecNTapDma), one per tile shape.
#include "conv_kernel.h"

namespace mg3m {

KernelFn conv_kernel_hwcn_vecn_tap_dma_fused(int tile) {
  return kernel_for_tile<kHWCN, kAVecM, kBVecNTapDma, true>(tile);
}

}  // namespace mg3m
