// Instantiations of the fp64-accumulating kernel for the HWCN layout with the
// kAVecM filter loader and the one-tap-per-slab kBVecNTap patch loader, one
// per tile of the fp64 menu.
#include "conv_kernel.h"

namespace mg3m {

KernelFn conv_kernel64_hwcn_vecn_tap(int tile) { return kernel64_for_tile<kHWCN, kAVecM, kBVecNTap>(tile); }

}  // namespace mg3m
