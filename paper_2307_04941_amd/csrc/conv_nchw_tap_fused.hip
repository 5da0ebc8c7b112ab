// Instantiations of the implicit-GEMM kernel with the fused output stage
// (y = act(conv + add)) for NCHW taken tap-major (kAVecM on the [R][S][C][K]
// filter copy, kBVecWTap patches), one per tile shape.
#include "conv_kernel.h"

namespace mg3m {

KernelFn conv_kernel_nchw_tap_fused(int tile) { return kernel_for_tile<kNCHW, kAVecM, kBVecWTap, true>(tile); }

}  // namespace mg3m
