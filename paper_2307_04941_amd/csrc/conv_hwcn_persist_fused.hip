// Instantiations of the persistent whole-tile kernel with the fused output
// stage y = act(conv + add) (conv_igemm_f32_pt<..., FUSE = true>), for the
// same loaders as conv_hwcn_persist.hip.
#include "conv_kernel.h"

namespace mg3m {

KernelFn conv_kernel_pt_fused(int variant, int tile) {
  switch (variant) {
    case kVarHwcnVecN: return kernel_pt_for_tile<kHWCN, kAVecM, kBVecN, true>(tile);
    case kVarHwcnVecNTap: return kernel_pt_for_tile<kHWCN, kAVecM, kBVecNTap, true>(tile);
    case kVarHwcnVecNTapDma: return kernel_pt_for_tile<kHWCN, kAVecM, kBVecNTapDma, true>(tile);
    default: return nullptr;
  }
}

}  // namespace mg3m
