// Internal declarations of the GEMM operator (Section 4's worked example):
// shared by the C-ABI layer, the derivation and the HIP translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "attn.h"

namespace attn {

// C[M][N] (fp32) = A[M][K] B[K][N], all row-major and contiguous.
struct GemmParams {
  const void* a;
  const void* b;
  float* c;
  int M, N, K;
  int n_tm, n_tn;  // workgroup tiles along M and N
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

// Fixed structure of the GEMM kernel family: LDS stages of (A, B) tiles, the
// wave grid over the workgroup tile, waves per SIMD (the register budget),
// registers per lane outside the accumulators, and the bytes one wave moves
// per global->LDS copy (each wave copies the same number of whole blocks of
// every tile).
constexpr int kGemmStages = 5, kGemmWavesM = 2, kGemmWavesN = 4, kGemmWavesPerSimd = 2, kGemmVgprFixed = 96,
              kGemmCopyBlock = 1024;

int derive_gemm(const attn_hw_desc_t* hw, const attn_mfma_atom_t* atom, int64_t M, int64_t N, int64_t K,
                attn_gemm_report_t* rep);

}  // namespace attn
