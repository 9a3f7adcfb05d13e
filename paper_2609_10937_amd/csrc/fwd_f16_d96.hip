// Fused-kernel instantiations for dtype f16, head dimension 96 (t_kv = 64,
// 5 LDS stages, K/V rows padded to 128 elements in LDS): every (query blocks
// per wave, waves per workgroup) the tile derivation can reach for this head
// dimension on a gfx950 descriptor.
#include "fwd_kernel.hpp"

namespace attn {

const FwdInstance* fwd_instances_f16_d96(int* n) {
  static const FwdInstance table[] = {
      {ATTN_F16, 96, 64, 3, 8, launch_fwd<ATTN_F16, 96, 64, 3, 8, 5>},
      {ATTN_F16, 96, 64, 3, 4, launch_fwd<ATTN_F16, 96, 64, 3, 4, 5>},
      {ATTN_F16, 96, 64, 3, 2, launch_fwd<ATTN_F16, 96, 64, 3, 2, 5>},
      {ATTN_F16, 96, 64, 3, 1, launch_fwd<ATTN_F16, 96, 64, 3, 1, 5>},
      {ATTN_F16, 96, 64, 2, 1, launch_fwd<ATTN_F16, 96, 64, 2, 1, 5>},
      {ATTN_F16, 96, 64, 1, 1, launch_fwd<ATTN_F16, 96, 64, 1, 1, 5>},
  };
  *n = (int)(sizeof(table) / sizeof(table[0]));
  return table;
}

}  // namespace attn
