// Fused-kernel instantiations for dtype f16, head dimension 256 (t_kv = 32,
// 5 LDS stages): every (query blocks per wave, waves per workgroup) the tile
// derivation can reach for this head dimension on a gfx950 descriptor.
#include "fwd_kernel.hpp"

namespace attn {

const FwdInstance* fwd_instances_f16_d256(int* n) {
  static const FwdInstance table[] = {
      {ATTN_F16, 256, 32, 1, 8, launch_fwd<ATTN_F16, 256, 32, 1, 8, 5>},
      {ATTN_F16, 256, 32, 1, 4, launch_fwd<ATTN_F16, 256, 32, 1, 4, 5>},
      {ATTN_F16, 256, 32, 1, 2, launch_fwd<ATTN_F16, 256, 32, 1, 2, 5>},
      {ATTN_F16, 256, 32, 1, 1, launch_fwd<ATTN_F16, 256, 32, 1, 1, 5>},
  };
  *n = (int)(sizeof(table) / sizeof(table[0]));
  return table;
}

}  // namespace attn
