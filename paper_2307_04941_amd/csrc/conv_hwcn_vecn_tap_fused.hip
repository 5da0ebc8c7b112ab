// Instantiations of the implicit-GEMM kernel with the fused output stage
// (y = act(conv + add)) for the kAVecM filter loader and the one-tap-per-slab kBVecNTap patch loader,
// one per tile shape.
#include "conv_kernel.h"

namespace mg3m {

KernelFn conv_kernel_hwcn_vecn_tap_fused(int tile) { return kernel_for_tile<kHWCN, kAVecM, kBVecNTap, true>(tile); }

}  // namespace mg3m
