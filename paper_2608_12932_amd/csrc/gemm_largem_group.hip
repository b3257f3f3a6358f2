// Group-scale instances of the large-M W4A8 GEMM (largem_kernel.h).
//
// This file is built with -mllvm -amdgpu-mfma-vgpr-form: the MFMAs then
// write their int32 partial sums to VGPRs, where the per-step rescale reads
// them directly (from AGPRs every element would first need a
// v_accvgpr_read, one more VALU instruction per element and step in a loop
// that is bound by its VALU work).  The per-channel instances keep the
// default AGPR form, which is faster for them.
#include "largem_kernel.h"

namespace w4a8 {

LargeMKernelFn largem_group_kernel(int cfg, bool swiglu) {
  if (swiglu) return cfg == 1 ? menu_kernel<1, true, true>() : nullptr;  // the gated tile that fits group mode
  switch (cfg) {
    case 1: return menu_kernel<1, true>();
    case 2: return menu_kernel<2, true>();
    case kMenuKSplit: return menu_kernel<kMenuKSplit, true>();
    default: return nullptr;  // 128 x 192 does not fit the group accumulators
  }
}

}  // namespace w4a8
