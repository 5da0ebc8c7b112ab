// Instantiations of the implicit-GEMM kernel for the HWCN layout with the
// kAScalar filter loader and the kBScalar input-patch loader, one per tile shape.
#include "conv_kernel.h"

namespace mg3m {

KernelFn conv_kernel_hwcn_scalar(int tile) { return kernel_for_tile<kHWCN, kAScalar, kBScalar>(tile); }

}  // namespace mg3m
