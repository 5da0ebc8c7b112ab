// Instantiations of the implicit-GEMM kernel for the HWCN layout with the
// kAVecM filter loader and the kBScalar input-patch loader, one per tile shape.
#include "conv_kernel.h"

namespace mg3m {

KernelFn conv_kernel_hwcn_veca(int tile) { return kernel_for_tile<kHWCN, kAVecM, kBScalar>(tile); }

}  // namespace mg3m
