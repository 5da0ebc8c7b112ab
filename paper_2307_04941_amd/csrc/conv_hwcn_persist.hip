// Instantiations of the persistent whole-tile kernel (conv_igemm_f32_pt) for
// the HWCN layout with the kAVecM filter loader and the batch-vector patch
// loaders: kBVecN (the three-channel stems), kBVecNTap, and kBVecNTap's
// direct-to-LDS form.
#include "conv_kernel.h"

namespace mg3m {

KernelFn conv_kernel_pt(int variant, int tile) {
  switch (variant) {
    case kVarHwcnVecN: return kernel_pt_for_tile<kHWCN, kAVecM, kBVecN>(tile);
    case kVarHwcnVecNTap: return kernel_pt_for_tile<kHWCN, kAVecM, kBVecNTap>(tile);
    case kVarHwcnVecNTapDma: return kernel_pt_for_tile<kHWCN, kAVecM, kBVecNTapDma>(tile);
    default: return nullptr;
  }
}

}  // namespace mg3m
