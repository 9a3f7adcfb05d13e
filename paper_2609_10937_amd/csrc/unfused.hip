// Unfused attention baseline (Section 6.2, Table 3): the L x L score matrix
// goes to device memory between three kernels.
//   GEMM (Q K^T):  S = scale Q K^T, stored in the input type
//   softmax:       S -> P in place, causal-masked entries 0 (the row-softmax
//                  operator of Section 5.3, attn_softmax, on its own tiles)
//   GEMM (P V):    O = P V, stored in the input type
// Both products run on the GEMM kernel with the tiles its derivation gives
// for their shapes (the worked example of Section 4), one product per head
// side by side in the grid.
#include "gemm_internal.h"
#include "internal.h"

namespace attn {

hipError_t launch_unfused(const UnfusedPlan& u, const void* q, const void* k, const void* v, void* o, void* ws,
                          int BH, int L, int d, float scale, int causal, int dtype, hipStream_t s) {
  GemmParams qk{q, k, ws, L, L, d, (L + u.qk.t_m - 1) / u.qk.t_m, (L + u.qk.t_n - 1) / u.qk.t_n};
  qk.batch = BH;
  qk.sa = (int64_t)L * d;
  qk.sb = (int64_t)L * d;
  qk.sc = (int64_t)L * L;
  qk.alpha = scale;
  hipError_t e = u.qk_inst->launch(qk, s);
  if (e != hipSuccess) return e;
  const SoftmaxParams sp{ws, ws, (int64_t)BH * L, L, u.sm.seg, u.sm.split, causal};
  e = launch_softmax(sp, dtype, true, (unsigned)u.sm.grid, s);
  if (e != hipSuccess) return e;
  GemmParams pv{ws, v, o, L, d, L, (L + u.pv.t_m - 1) / u.pv.t_m, (d + u.pv.t_n - 1) / u.pv.t_n};
  pv.batch = BH;
  pv.sa = (int64_t)L * L;
  pv.sb = (int64_t)L * d;
  pv.sc = (int64_t)L * d;
  return u.pv_inst->launch(pv, s);
}

}  // namespace attn
