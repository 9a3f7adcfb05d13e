// fp32 GEMM instances: the tiles the closed-form derivation yields on gfx950
// for the fp32 kernel family (192 x 192 x 32 from LDS and registers; the CU
// rule's halvings for smaller problems).
#include "gemm_f32_kernel.hpp"

namespace attn {

static const GemmInstance kInstancesF32[] = {
    {ATTN_F32, 192, 192, 32, launch_gemm_f32<192, 192, 32, kGemm32.stages>},
    {ATTN_F32, 96, 192, 32, launch_gemm_f32<96, 192, 32, kGemm32.stages>},
    {ATTN_F32, 96, 96, 64, launch_gemm_f32<96, 96, 64, kGemm32.stages>},
    {ATTN_F32, 32, 96, 96, launch_gemm_f32<32, 96, 96, kGemm32.stages>},
    {ATTN_F32, 32, 32, 192, launch_gemm_f32<32, 32, 192, kGemm32.stages>},
};

const GemmInstance* gemm_instances_f32(int* n) {
  *n = (int)(sizeof(kInstancesF32) / sizeof(kInstancesF32[0]));
  return kInstancesF32;
}

}  // namespace attn
