// GEMM instances for f16 inputs: the tiles the closed-form derivation yields
// on gfx950 (256 x 256 x 32 from LDS and registers; the CU rule's halvings
// for small problems).
#include "gemm_kernel.hpp"

namespace attn {

static const GemmInstance kInstances[] = {
    {ATTN_F16, 256, 256, 32, launch_gemm<ATTN_F16, 256, 256, 32, kGemmStages>},
    {ATTN_F16, 128, 256, 32, launch_gemm<ATTN_F16, 128, 256, 32, kGemmStages>},
    {ATTN_F16, 128, 128, 64, launch_gemm<ATTN_F16, 128, 128, 64, kGemmStages>},
    {ATTN_F16, 64, 128, 64, launch_gemm<ATTN_F16, 64, 128, 64, kGemmStages>},
    {ATTN_F16, 64, 64, 128, launch_gemm<ATTN_F16, 64, 64, 128, kGemmStages>},
    {ATTN_F16, 32, 64, 128, launch_gemm<ATTN_F16, 32, 64, 128, kGemmStages>},
};

const GemmInstance* gemm_instances_f16(int* n) {
  *n = (int)(sizeof(kInstances) / sizeof(kInstances[0]));
  return kInstances;
}

}  // namespace attn
