// GEMM C = A B in fp32 for gfx950: Section 4's worked example in the type the
// section measures it in, on v_mfma_f32_16x16x4_f32 (2048 flops in 32 cycles),
// with the workgroup tile t_M x t_N x t_K and the per-wave tile from the
// closed-form derivation for this kernel family's structure (3 LDS stages,
// 2 x 2 waves, one per SIMD).
//
// As in the 16-bit kernel the product is formed as C^T = B^T A^T, so a lane's
// result fragment is four consecutive columns of one row of C.  Fragment
// layouts of the 16x16x4 atom: A-role lane (g = lane/16, c = lane%16) holds
// one value at [c][g], B-role one at [g][c], the result [4g + r][c].  For a
// 16-wide k slab the kernel issues four products e = 0..3 in which lane (g, c)
// supplies k = 16 s + 4 g + e: its A^T values for the four products are one
// 16-byte chunk of a row of the A tile (ds_read_b128), its B^T values four
// single reads of one column of the B tile (ds_read_b32, rows 4g + e).
//
// LDS holds ST stages of an A tile [t_M][t_K] and a B tile [t_K][t_N],
// row-major in 16-byte chunks.  A rows are read 16 rows x one chunk per
// 16-lane group: chunk positions are XOR-swizzled per row as in the 16-bit
// kernel's A tile (rows of 128 + 256 n bytes: (r >> 1) & 7; rows of 256 n
// bytes: r & 15).  A b32 read of B covers four rows (one per lane group g)
// x 64 bytes: the chunk index is XORed with 4 ((r >> 2) & 3) so that the
// four rows land on the four 64-byte quarters of the banks (rows of 256 n
// bytes; rows of 128 + 256 n bytes take 4 ((r >> 2) & 1), two quarters).
//
// Pipeline: one step per k tile.  In step j each wave requests its part of
// tile j + 2 (whole 1 KB blocks of both tiles, global_load_lds_dwordx4),
// reads the fragments of tile j slab by slab one slab ahead of the products,
// then waits for its part of tile j + 1 and joins the workgroup barrier.  A
// step is 32 x (t_M/2)(t_N/2)/256 x t_K/4 cycles of matrix work per wave,
// long enough to hide both the copies and the first slab's reads.
#pragma once

#include "gemm_kernel.hpp"

namespace attn {

template <int KC>
__device__ __forceinline__ int f32_a_swz(int r) {
  static_assert((KC * 16) % 256 == 0 || (KC * 16) % 256 == 128, "A row bytes");
  if constexpr ((KC * 16) % 256 == 0) return r & 15;
  else return (r >> 1) & 7;
}
template <int KC>
__device__ __forceinline__ int f32_b_swz(int r) {
  static_assert((KC * 16) % 256 == 0 || (KC * 16) % 256 == 128, "B row bytes");
  if constexpr ((KC * 16) % 256 == 0) return 4 * ((r >> 2) & 3);
  else return 4 * ((r >> 2) & 1);
}

template <int TM, int TN, int TK, int ST>
__global__ void __launch_bounds__(256) matmul_f32_kernel(const GemmParams p) {
  constexpr int WM = kGemm32.waves_m, WN = kGemm32.waves_n, NW = WM * WN;
  static_assert(NW == 4, "four waves");
  constexpr int WTM = TM / WM, WTN = TN / WN;   // per-wave tile of C
  constexpr int NMB = WTM / 16, NNB = WTN / 16, SL = TK / 16;
  constexpr int KCA = TK / 4, KCB = TN / 4;     // 16-byte chunks per row
  constexpr int RA = TK * 4, RB = TN * 4;       // row bytes
  constexpr int ATB = TM * RA, BTB = TK * RB, SB = ATB + BTB;
  constexpr int LPA = ATB / (1024 * NW), LPB = BTB / (1024 * NW), LPT = LPA + LPB;
  constexpr int LEAD = ST - 1;                  // tile j + LEAD is requested in step j
  static_assert(TM % (16 * WM) == 0 && TN % (16 * WN) == 0 && TK % 16 == 0, "atom alignment");
  static_assert(ATB % (1024 * NW) == 0 && BTB % (1024 * NW) == 0, "whole copy blocks per wave");
  static_assert(ST >= 2 && (LEAD - 1) * LPT < 64, "stages and copy counter");
  static_assert(ATB + ((SL - 1) * 16 + 3) * RB + (NMB - 1) * 16 * RA < 65536, "ds offset range");

  __shared__ __attribute__((aligned(1024))) float smem[ST * SB / 4];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, c = lane & 15;
  const int wm = w >> 1, wn = w & 1;
  const int M = p.M, N = p.N, K = p.K;

  // Workgroup -> tile: the XCD-grouped order of the 16-bit kernel.
  const int T = p.n_tm * p.n_tn;
  int t = blockIdx.x;
  if (T % 8 == 0) t = (int)(blockIdx.x % 8) * (T / 8) + (int)(blockIdx.x / 8);
  constexpr int G = 4;
  const int gid = t / (G * p.n_tn), first = gid * G;
  const int gs = min(p.n_tm - first, G);
  const int r_in = t - gid * G * p.n_tn;
  const int tm = first + r_in % gs, tn = r_in / gs;
  const int m0 = tm * TM, n0 = tn * TN;
  const int n_k = (K + TK - 1) / TK;

  const char* const Ab = static_cast<const char*>(p.a) + (size_t)m0 * K * 4;
  const char* const Bb = static_cast<const char*>(p.b) + (size_t)n0 * 4;
  ATTN_LDS char* const lds = (ATTN_LDS char*)smem;
  const uint32_t lds0 = (uint32_t)(size_t)lds;

  // Copies.  Wave w takes blocks w, w + 4, ... of each tile image; lane l
  // fills 16-byte slot l of a block, i.e. image slot P = 64 b + l at row
  // P / (chunks per row), physical chunk P % (chunks per row), whose logical
  // chunk is that XOR the row's swizzle.  Rows past M (A) or K (B) repeat the
  // last one, columns past N and k chunks past K are clamped; their results
  // are never stored or their operands are zeroed.
  uint32_t aoff[LPA];
  int alc[LPA];
#pragma unroll
  for (int i = 0; i < LPA; ++i) {
    const int P = 64 * (w + i * NW) + lane;
    const int row = P / KCA, ph = P % KCA;
    alc[i] = ph ^ f32_a_swz<KCA>(row);
    aoff[i] = (uint32_t)min(row, M - 1 - m0) * (uint32_t)(K * 4);
  }
  int brow[LPB];
  uint32_t bcol[LPB];
#pragma unroll
  for (int i = 0; i < LPB; ++i) {
    const int P = 64 * (w + i * NW) + lane;
    const int row = P / KCB, ph = P % KCB;
    brow[i] = row;
    bcol[i] = (uint32_t)min(ph ^ f32_b_swz<KCB>(row), (N - n0) / 4 - 1) * 16;
  }
  auto issue = [&](int tt, int ci) ATTN_INLINE {
    const int te = min(tt, n_k - 1);
    const int k0 = te * TK;
    const uint32_t dst = (uint32_t)__builtin_amdgcn_readfirstlane(lds0 + (tt % ST) * SB);
    if (ci < LPA) {
      const uint32_t ch = (uint32_t)min(alc[ci], (K - k0) / 4 - 1) * 16;
      copy_to_lds(Ab + (size_t)k0 * 4, aoff[ci] + ch, dst + (w + ci * NW) * 1024);
    } else {
      const int i = ci - LPA;
      const uint32_t row = (uint32_t)min(brow[i], K - 1 - k0);
      copy_to_lds(Bb + (size_t)k0 * N * 4, row * (uint32_t)(N * 4) + bcol[i], dst + ATB + (w + i * NW) * 1024);
    }
  };

  // Fragment addresses.  A^T(s, mb): row wm WTM + 16 mb + c, logical chunk
  // 4 s + g; the swizzle depends on the row's low four bits, i.e. on c.
  // B^T(s, e, nb): row 16 s + 4 g + e, column wn WTN + 16 nb + c, i.e. logical
  // chunk (wn WTN + 16 nb) / 4 + c / 4, float c % 4; the swizzle depends on
  // bits 2..3 of the row, i.e. on g.
  const int sa = f32_a_swz<KCA>(c);
  uint32_t la[SL];
#pragma unroll
  for (int s = 0; s < SL; ++s) la[s] = (uint32_t)((wm * WTM + c) * RA + 16 * ((4 * s + g) ^ sa));
  const int sbg = f32_b_swz<KCB>(4 * g);
  uint32_t lb[NNB];
#pragma unroll
  for (int nb = 0; nb < NNB; ++nb)
    lb[nb] = (uint32_t)(ATB + 4 * g * RB + 16 * (((wn * WTN + 16 * nb) / 4 + (c >> 2)) ^ sbg) + 4 * (c & 3));

  f32x4_t acc[NNB][NMB];
#pragma unroll
  for (int nb = 0; nb < NNB; ++nb)
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb) acc[nb][mb] = (f32x4_t){0.f, 0.f, 0.f, 0.f};

  if (n_k > 0) {
#pragma unroll
    for (int tt = 0; tt < LEAD; ++tt)
#pragma unroll
      for (int ci = 0; ci < LPT; ++ci) issue(tt, ci);
    wait_vmcnt<(LEAD - 1) * LPT>();
    barrier_only();

    // One step: slab s's fragments are read while slab s - 1's products
    // issue.  MASK (the last tile of a K that t_K does not divide): the k
    // positions past K are zeroed in both operands (K is a multiple of 4, so
    // a lane's four values of a slab are all inside or all outside).
    auto step = [&](auto maskc, int j) ATTN_INLINE {
      constexpr bool MASK = decltype(maskc)::value;
      const uint32_t sj = (uint32_t)__builtin_amdgcn_readfirstlane(lds0 + (j % ST) * SB);
      f32x4_t fa[2][NMB];
      float fb[2][NNB][4];
      auto load = [&](int s, int buf) ATTN_INLINE {
#pragma unroll
        for (int mb = 0; mb < NMB; ++mb)
          fa[buf][mb] = *(ATTN_LDS const f32x4_t*)((ATTN_LDS const char*)(size_t)(sj + la[s]) + 16 * mb * RA);
#pragma unroll
        for (int nb = 0; nb < NNB; ++nb)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            fb[buf][nb][e] = *(ATTN_LDS const float*)((ATTN_LDS const char*)(size_t)(sj + lb[nb]) + (16 * s + e) * RB);
      };
      load(0, 0);
#pragma unroll
      for (int ci = 0; ci < LPT; ++ci) issue(j + LEAD, ci);
      const int kvalid = K - j * TK;
#pragma unroll
      for (int s = 0; s < SL; ++s) {
        const int cur = s & 1;
        if (s + 1 < SL) load(s + 1, cur ^ 1);
        bool zero = false;
        if constexpr (MASK) zero = 16 * s + 4 * g >= kvalid;
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
          for (int mb = 0; mb < NMB; ++mb) {
            const float av = zero ? 0.f : fa[cur][mb][e];
#pragma unroll
            for (int nb = 0; nb < NNB; ++nb) {
              const float bv = zero ? 0.f : fb[cur][nb][e];
              acc[nb][mb] = __builtin_amdgcn_mfma_f32_16x16x4f32(bv, av, acc[nb][mb], 0, 0, 0);
            }
          }
      }
      // This wave's copies of tile j + 1 complete (those of tile j + LEAD may
      // still fly); the barrier publishes tile j + 1 and frees tile j's stage.
      wait_vmcnt<(LEAD - 1) * LPT>();
      barrier_only();
    };
    const std::false_type no{};
    const std::true_type yes{};
    for (int j = 0; j + 1 < n_k; ++j) step(no, j);
    if (K % TK != 0) step(yes, n_k - 1);
    else step(no, n_k - 1);
    // The copies of the tiles past the last land before the LDS is released.
    wait_vmcnt<0>();
  }

  // Epilogue: lane (g, c) of block (nb, mb) holds C[m][n .. n+3] with
  // m = m0 + wm WTM + 16 mb + c, n = n0 + wn WTN + 16 nb + 4 g; N is a
  // multiple of 4, so n < N puts all four columns in range.
#pragma unroll
  for (int mb = 0; mb < NMB; ++mb) {
    const int m = m0 + wm * WTM + 16 * mb + c;
    if (m >= M) continue;
    float* crow = static_cast<float*>(p.c) + (size_t)m * N;
#pragma unroll
    for (int nb = 0; nb < NNB; ++nb) {
      const int n = n0 + wn * WTN + 16 * nb + 4 * g;
      if (n < N) *reinterpret_cast<f32x4_t*>(crow + n) = acc[nb][mb];
    }
  }
}

template <int TM, int TN, int TK, int ST>
hipError_t launch_gemm_f32(const GemmParams& p, hipStream_t s) {
  const unsigned grid = (unsigned)p.n_tm * (unsigned)p.n_tn;
  hipLaunchKernelGGL((matmul_f32_kernel<TM, TN, TK, ST>), dim3(grid), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace attn
