// Internal declarations of the GEMM operator (Section 4's worked example):
// shared by the C-ABI layer, the derivation and the HIP translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "attn.h"

namespace attn {

// C[M][N] = A[M][K] B[K][N], all row-major and contiguous; C is fp32 (or, in
// the 16-bit family's OUT16 instances, the input type times alpha).  B may
// be given transposed, as Bt[N][K] (the BT instances).  `batch` independent
// products run side by side (grid y), matrix z at a + z sa, b + z sb,
// c + z sc elements.
struct GemmParams {
  const void* a;
  const void* b;
  void* c;
  int M, N, K;
  int n_tm, n_tn;  // workgroup tiles along M and N
  int batch = 1;
  int64_t sa = 0, sb = 0, sc = 0;
  float alpha = 1.f;
};

using GemmLaunch = hipError_t (*)(const GemmParams&, hipStream_t);

// One compiled instantiation of the GEMM kernel.
struct GemmInstance {
  int dtype;
  int t_m, t_n, t_k;
  GemmLaunch launch;
};

const GemmInstance* gemm_instances_bf16(int* n);
const GemmInstance* gemm_instances_f16(int* n);
// The unfused attention baseline's products, in the input type: S = scale
// Q K^T (K given as Bt) and O = P V.
const GemmInstance* gemm_instances_qk(int dtype, int* n);
const GemmInstance* gemm_instances_pv(int dtype, int* n);

// Fixed structure of a GEMM kernel family: LDS stages of (A, B) tiles, the
// wave grid over the workgroup tile, waves per SIMD (the register budget),
// registers per lane outside the accumulators, and the bytes one wave moves
// per global->LDS copy (each wave copies the same number of whole blocks of
// every tile).
struct GemmStructure {
  int stages, waves_m, waves_n, waves_per_simd, vgpr_fixed, copy_block;
};
// 16-bit inputs (16x16x32 atom): 8 waves, two per SIMD, 5 stages.
constexpr GemmStructure kGemm16 = {5, 2, 4, 2, 96, 1024};
constexpr int kGemmStages = kGemm16.stages, kGemmWavesM = kGemm16.waves_m, kGemmWavesN = kGemm16.waves_n;
// fp32 inputs (16x16x4 atom, 32 cycles per product): 4 waves, one per SIMD,
// 3 stages; halving copy blocks per tile keeps every tile the CU rule reaches
// feasible at 4-byte elements.
constexpr GemmStructure kGemm32 = {3, 2, 2, 1, 128, 1024};

// The structure of the family that runs `atom` (by its input size).
const GemmStructure& gemm_structure(const attn_mfma_atom_t* atom);

int derive_gemm(const attn_hw_desc_t* hw, const attn_mfma_atom_t* atom, int64_t M, int64_t N, int64_t K,
                attn_gemm_report_t* rep);

const GemmInstance* gemm_instances_f32(int* n);

}  // namespace attn
