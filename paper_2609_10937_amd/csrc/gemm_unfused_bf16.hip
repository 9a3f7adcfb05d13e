// The unfused attention baseline's products for bf16 inputs on the GEMM kernel
// and its derived tiles: S = scale Q K^T (K given as Bt), written in bf16, and
// O = P V, written in bf16.
#include "gemm_kernel.hpp"

namespace attn {

#define QK(TM, TN, TK) {ATTN_BF16, TM, TN, TK, launch_gemm<ATTN_BF16, TM, TN, TK, kGemmStages, true, true>}
#define PV(TM, TN, TK) {ATTN_BF16, TM, TN, TK, launch_gemm<ATTN_BF16, TM, TN, TK, kGemmStages, false, true>}
static const GemmInstance kQk[] = {QK(256, 256, 32), QK(128, 256, 32), QK(128, 128, 64),
                                   QK(64, 128, 64),  QK(64, 64, 128),  QK(32, 64, 128)};
static const GemmInstance kPv[] = {PV(256, 256, 32), PV(128, 256, 32), PV(128, 128, 64),
                                   PV(64, 128, 64),  PV(64, 64, 128),  PV(32, 64, 128)};
#undef QK
#undef PV

const GemmInstance* gemm_instances_qk_bf16(int* n) {
  *n = (int)(sizeof(kQk) / sizeof(kQk[0]));
  return kQk;
}
const GemmInstance* gemm_instances_pv_bf16(int* n) {
  *n = (int)(sizeof(kPv) / sizeof(kPv[0]));
  return kPv;
}

}  // namespace attn
