// Instantiations of the implicit-GEMM kernel for NCHW taken tap-major: the
// kAVecM filter loader on the [R][S][C][K] filter copy and the one-tap-per-slab
// kBVecWTap patch loader, one per tile shape.
#include "conv_kernel.h"

namespace mg3m {

KernelFn conv_kernel_nchw_tap(int tile) { return kernel_for_tile<kNCHW, kAVecM, kBVecWTap>(tile); }

}  // namespace mg3m
