// Instantiations of the implicit-GEMM kernel for the HWCN layout with the
// one-tap filter and input-patch loaders in their direct-to-LDS form
// (AVecMTapDma, BVecNTapDma), one per tile shape.
#include "conv_kernel.h"

namespace mg3m {

KernelFn conv_kernel_hwcn_vecn_tap_dma(int tile) { return kernel_for_tile<kHWCN, kAVecM, kBVecNTapDma>(tile); }

}  // namespace mg3m
