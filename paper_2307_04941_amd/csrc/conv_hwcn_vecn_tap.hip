// Instantiations of the implicit-GEMM kernel for the HWCN layout with the
// kAVecM filter loader and the kBVecNTap input-patch loader (one filter tap
// per staged slab), one per tile shape: the tuned path.
#include "conv_kernel.h"

namespace mg3m {

KernelFn conv_kernel_hwcn_vecn_tap(int tile) { return kernel_for_tile<kHWCN, kAVecM, kBVecNTap>(tile); }

}  // namespace mg3m
