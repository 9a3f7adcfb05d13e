// Fused-kernel instantiations for dtype bf16, head dimension 128 (t_kv = 64):
// every (query blocks per wave, waves per workgroup) the tile derivation can
// reach for this head dimension on a gfx950 descriptor.
#include "fwd_kernel.hpp"

namespace attn {

const FwdInstance* fwd_instances_bf16_d128(int* n) {
  static const FwdInstance table[] = {
      {ATTN_BF16, 128, 64, 2, 8, launch_fwd<ATTN_BF16, 128, 64, 2, 8>},
      {ATTN_BF16, 128, 64, 1, 8, launch_fwd<ATTN_BF16, 128, 64, 1, 8>},
      {ATTN_BF16, 128, 64, 1, 4, launch_fwd<ATTN_BF16, 128, 64, 1, 4>},
      {ATTN_BF16, 128, 64, 1, 2, launch_fwd<ATTN_BF16, 128, 64, 1, 2>},
  };
  *n = (int)(sizeof(table) / sizeof(table[0]));
  return table;
}

}  // namespace attn
