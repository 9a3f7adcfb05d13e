// Fused-kernel instantiations for dtype f16, head dimension 64 (t_kv = 128,
// 5 LDS stages): every (query blocks per wave, waves per workgroup) the tile
// derivation can reach for this head dimension on a gfx950 descriptor, and
// the 8-wave one also as a persistent launch.
#include "fwd_kernel.hpp"

namespace attn {

const FwdInstance* fwd_instances_f16_d64(int* n) {
  static const FwdInstance table[] = {
      {ATTN_F16, 64, 128, 2, 8, launch_fwd<ATTN_F16, 64, 128, 2, 8, 5>,
       launch_fwd<ATTN_F16, 64, 128, 2, 8, 5, true>},
      {ATTN_F16, 64, 128, 2, 4, launch_fwd<ATTN_F16, 64, 128, 2, 4, 5>},
      {ATTN_F16, 64, 128, 2, 2, launch_fwd<ATTN_F16, 64, 128, 2, 2, 5>},
      {ATTN_F16, 64, 128, 2, 1, launch_fwd<ATTN_F16, 64, 128, 2, 1, 5>},
      {ATTN_F16, 64, 128, 1, 1, launch_fwd<ATTN_F16, 64, 128, 1, 1, 5>},
  };
  *n = (int)(sizeof(table) / sizeof(table[0]));
  return table;
}

}  // namespace attn
