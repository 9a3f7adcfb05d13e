// GEMM C = A B for gfx950 (CDNA4): the worked example of Section 4, with the
// workgroup tile t_M x t_N x t_K and the per-wave tile from the closed-form
// derivation (Figure 1's tree: CU tile, wave tile, matrix-core atom).
//
// The kernel computes C^T = B^T A^T on v_mfma_f32_16x16x32_{bf16,f16}: the
// atom's A operand is a 16 (n) x 32 (k) block of B^T and its B operand a
// 32 (k) x 16 (m) block of A^T, so the C fragment of a lane holds four
// consecutive columns of one row of C and the epilogue writes 16 contiguous
// bytes per lane.  Fragment layouts (a hardware fact, checked on the device
// by the layout probe):
//   A-role (B^T): lane (g = lane/16, c = lane%16) holds B[8g + e][c], e = 0..7
//   B-role (A^T): lane holds A[c][8g + e]
//   result:       lane holds C[c][4g + r], r = 0..3
// so the k index of both operands is 8g + e: a lane's A^T fragment is one
// 16-byte chunk of a row of A (ds_read_b128) and its B^T fragment
// four rows of one column of the B tile, read twice with the transposing
// ds_read_b64_tr_b16 (lane j of a 16-lane group addresses row k0 + j/4,
// columns n0 + 4(j%4) .. +3; lane i receives rows k0 .. k0+3 of column n0+i).
//
// LDS holds ST stages, each an A tile and a B tile (64 banks of 4 bytes:
// 16 chunk positions of 16 bytes per 256-byte bank row).  A b128 read is
// served 16 lanes at a time, and the bank-conflict counter rules out every
// grouping except lanes sharing lane-index bits {0, 5} or {1, 4}; the
// layouts below keep each such group on 16 distinct positions.
//  A tile, t_K = 32 (64-byte rows, four to a bank row, so no row-major
//    swizzle can spread a group): 1 KB blocks of 16 rows x 32 k, one per
//    atom fragment, slot 16 q + p holding row p ^ q, 16-byte k chunk q.
//  A tile, t_K >= 64: row-major [t_M][t_K], chunk positions XOR-swizzled
//    per row (whole rows per copy keep the global reads line-sized).
//  B tile: row-major [t_K][t_N], chunk positions XOR-swizzled per row for
//    the transposing reads.
// Tiles move HBM -> LDS with global_load_lds_dwordx4 (each wave copies
// whole 1 KB blocks of both tiles), so no registers stage them.
//
// Pipeline.  Eight waves (2 along M x 4 along N, two per SIMD) take one
// step per k tile: the step's matrix products, with this wave's copies of the
// tile four steps ahead spread among them, and one workgroup barrier at the
// end.  Before the barrier a wave waits for its copies of the tile two steps
// ahead, so the barrier publishes that tile; the operand reads of a step run
// PF fragments ahead of the products, across the barrier into the next
// step's tile, so the matrix core never waits for the first reads of a step.
#pragma once

#include "fwd_kernel.hpp"
#include "gemm_internal.h"

namespace attn {

// Chunk swizzle of a row-major A tile with KCA >= 8 chunks per row.
template <int KCA>
__device__ __forceinline__ int gemm_a_swz(int r) {
  static_assert(KCA == 8 || KCA == 16, "A row chunks");
  if constexpr (KCA == 16) return r & 15;
  else return (r >> 1) & 7;
}
// Chunk swizzle of the B tile: rows of KCB chunks.  A transposing read is
// served 16 lanes (four rows, one logical pair of chunks each) at a time, and
// a 32-lane half covers rows {0..3, 8..11} (+4, +32 kk); even swizzle values
// keep each pair adjacent and give those rows distinct pair positions.
template <int KCB>
__device__ __forceinline__ int gemm_b_swz(int r) {
  static_assert(KCB == 8 || KCB == 16 || KCB == 32, "B row chunks");
  if constexpr (KCB >= 16) return (2 * (r & 3)) | (8 * ((r >> 3) & 1));
  else return 2 * ((r & 3) ^ ((r >> 3) & 1));
}

__device__ __forceinline__ void barrier_only() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_barrier" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

// BT: B is given as Bt[N][K]; its tile then takes the A tile's layout and
// reads (16-byte chunks of k along a row of Bt).  OUT16: C is written in the
// input type, times alpha (the products of the unfused attention baseline).
template <int DT, int TM, int TN, int TK, int ST, bool BT, bool OUT16>
__global__ void __launch_bounds__(512) matmul_kernel(const GemmParams p) {
  using M_ = Mfma<DT>;
  using V8 = typename M_::V8;
  constexpr int WM = kGemmWavesM, WN = kGemmWavesN, NW = WM * WN;
  static_assert(NW == 8, "eight waves");
  constexpr int WTM = TM / WM, WTN = TN / WN;  // per-wave tile of C
  constexpr int NMB = WTM / 16, NNB = WTN / 16, KS = TK / 32;
  constexpr int KCA = TK / 8, KCB = TN / 8;    // 16-byte chunks per row
  constexpr int RA = TK * 2, RB = TN * 2;      // row bytes
  constexpr int ATB = TM * RA, BTB = TK * TN * 2, SB = ATB + BTB;
  constexpr int LPA = ATB / (1024 * NW), LPB = BTB / (1024 * NW), LPT = LPA + LPB;
  constexpr bool ABLK = KCA == 4;                  // A tile in fragment blocks
  constexpr int KBA = KCA / 4;                     // A blocks per 16 rows (ABLK)
  constexpr int RPA = 1024 / RA, RPB = 1024 / RB;  // rows per 1 KB block (row-major)
  constexpr int LEAD = ST - 1;                     // tile j + LEAD is requested in step j
  constexpr int FPK = NNB + NMB, F = KS * FPK;     // operand fragments per k sub-step / step
  constexpr int PF = F < 6 ? F : 6;
  static_assert(TM % (16 * WM) == 0 && TN % (16 * WN) == 0 && TK % 32 == 0, "atom alignment");
  static_assert(ATB % (1024 * NW) == 0 && BTB % (1024 * NW) == 0, "whole copy blocks per wave");
  static_assert((ABLK || (NW * RPA) % 16 == 0) && (BT || (NW * RPB) % 16 == 0), "swizzle period");
  static_assert(ST >= 3 && 2 * LPT < 64, "stages and copy counter");
  static_assert(ATB + (TK - 4) * RB + 2 * WTN * WN < 65536, "ds offset range");

  __shared__ __attribute__((aligned(1024))) uint16_t smem[ST * SB / 2];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, c = lane & 15;
  const int wm = w >> 2, wn = w & 3;
  const int M = p.M, N = p.N, K = p.K;

  // Workgroup -> tile.  Workgroups are dispatched to the 8 XCDs round-robin
  // (block b on XCD b % 8, each XCD with its own L2); when the tile count
  // divides evenly XCD x takes a contiguous range of the tile order, and the
  // order walks groups of 4 tile rows column by column, so the 32 workgroups
  // an XCD runs at once form a 4 x 8 block of C that shares 4 row panels of A
  // and 8 column panels of B through that L2.
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

  const size_t z = blockIdx.y;  // product of the batch
  const char* const Ab = static_cast<const char*>(p.a) + (z * p.sa + (size_t)m0 * K) * 2;
  const char* const Bb = static_cast<const char*>(p.b) + (z * p.sb + (BT ? (size_t)n0 * K : (size_t)n0)) * 2;
  ATTN_LDS char* const lds = (ATTN_LDS char*)smem;
  const uint32_t lds0 = (uint32_t)(size_t)lds;

  // Copies.  Wave w takes blocks w, w + 8, ... of each tile image, lane l
  // filling 16-byte slot l of a block.  In fragment blocks (t_K = 32) block
  // b holds rows 16 b .. +15, slot l row (l % 16) ^ (l / 16), chunk l / 16.
  // A row-major block holds 1 KB / row bytes rows, slot P at row P / (chunks
  // per row) and physical chunk P % (chunks per row), whose logical chunk is
  // that XOR the row's swizzle.  Rows past M and columns past N repeat the
  // last row / column (finite data whose results are never stored); k chunks
  // past K are clamped too and their operands zeroed before use.
  // A tile rows (and, for BT, Bt tile rows): lane offsets of each block.
  int alc, ar0;
  if constexpr (ABLK) {
    alc = lane >> 4;
    ar0 = 16 * w + ((lane & 15) ^ (lane >> 4));
  } else {
    ar0 = w * RPA + lane / KCA;
    alc = (lane % KCA) ^ gemm_a_swz<KCA>(ar0);
  }
  constexpr int ASTEP = ABLK ? 16 * NW : NW * RPA;  // rows between a wave's blocks
  uint32_t aoff[LPA];
#pragma unroll
  for (int i = 0; i < LPA; ++i) aoff[i] = (uint32_t)min(ar0 + i * ASTEP, M - 1 - m0) * (uint32_t)(K * 2);
  uint32_t btoff[BT ? LPB : 1];
  if constexpr (BT) {
#pragma unroll
    for (int i = 0; i < LPB; ++i) btoff[i] = (uint32_t)min(ar0 + i * ASTEP, N - 1 - n0) * (uint32_t)(K * 2);
  }
  const int br0 = w * RPB + lane / KCB;
  const int blc = (lane % KCB) ^ gemm_b_swz<KCB>(br0);
  const uint32_t bcol = (uint32_t)min(blc, (N - n0) / 8 - 1) * 16;
  // Copy ci (0 .. LPT-1) of tile t into stage t % ST; tiles past the last
  // repeat the last one (into a stage no later step reads), so every step
  // makes the same copies.
  auto issue = [&](int tt, int ci) ATTN_INLINE {
    const int te = min(tt, n_k - 1);
    const int k0 = te * TK;
    const uint32_t dst = (uint32_t)__builtin_amdgcn_readfirstlane(lds0 + (tt % ST) * SB) + w * 1024;
    const uint32_t ch = (uint32_t)min(alc, (K - k0) / 8 - 1) * 16;
    if (ci < LPA) {
      copy_to_lds(Ab + (size_t)k0 * 2, aoff[ci] + ch, dst + ci * NW * 1024);
    } else if constexpr (BT) {
      const int i = ci - LPA;
      copy_to_lds(Bb + (size_t)k0 * 2, btoff[i] + ch, dst + ATB + i * NW * 1024);
    } else {
      const int i = ci - LPA;
      const uint32_t row = (uint32_t)min(br0 + i * NW * RPB, K - 1 - k0);
      copy_to_lds(Bb + (size_t)k0 * N * 2, row * (uint32_t)(N * 2) + bcol, dst + ATB + i * NW * 1024);
    }
  };

  // Operand fragments.  A^T(kk, mb): rows wm WTM + 16 mb + c, k chunk
  // 4 kk + g: in fragment blocks block wm WTM / 16 + mb, slot 16 g + (c ^ g);
  // row-major, that row at logical chunk 4 kk + g.  B^T(kk, nb): rows
  // 32 kk + 8 g + c/4 (+4 for the upper half) of the B tile, logical chunk
  // (wn WTN + 16 nb)/8 + (c/2)%2, byte 8 (c%2) within it.  The swizzles
  // depend only on the lane, and kk, mb, nb enter the address through
  // disjoint bit fields, so each address is a lane base XOR a fragment
  // constant plus an immediate offset.
  uint32_t la, lbt;
  if constexpr (ABLK) {
    la = (uint32_t)((wm * WTM / 16) * 1024 + 256 * g + 16 * (c ^ g));
    lbt = (uint32_t)(ATB + (wn * WTN / 16) * 1024 + 256 * g + 16 * (c ^ g));
  } else {
    la = (uint32_t)((wm * WTM + c) * RA + 16 * (g ^ gemm_a_swz<KCA>(c)));
    lbt = (uint32_t)(ATB + (wn * WTN + c) * RA + 16 * (g ^ gemm_a_swz<KCA>(c)));
  }
  const int rb = 8 * g + (c >> 2);
  const int sb = gemm_b_swz<KCB>(rb);
  const uint32_t lb = (uint32_t)(rb * RB + 16 * ((wn * WTN / 8) ^ ((c >> 1) & 1) ^ sb) + 8 * (c & 1));
  auto load = [&](uint32_t sbase, int f) ATTN_INLINE -> V8 {
    const int kk = f / FPK, q = f % FPK;
    if (BT && q < NNB) {
      // B^T(kk, nb) from a Bt tile: rows wn WTN + 16 nb + c, k chunk 4 kk + g.
      if constexpr (ABLK) {
        ATTN_LDS const char* base = (ATTN_LDS const char*)(size_t)(sbase + lbt);
        return __builtin_bit_cast(V8, *(ATTN_LDS const u32x4_t*)(base + q * 1024));
      }
      ATTN_LDS const char* base = (ATTN_LDS const char*)(size_t)(sbase + ((lbt - ATB) ^ (uint32_t)(64 * kk)) + ATB);
      return __builtin_bit_cast(V8, *(ATTN_LDS const u32x4_t*)(base + 16 * q * RA));
    }
    if (q < NNB) {
      ATTN_LDS const char* base = (ATTN_LDS const char*)(size_t)(sbase + (lb ^ (uint32_t)(32 * q)));
      const i16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((ATTN_LDS i16x4_t*)(base + ATB + 32 * kk * RB));
      const i16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((ATTN_LDS i16x4_t*)(base + ATB + (32 * kk + 4) * RB));
      const i16x8_t cat = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      return __builtin_bit_cast(V8, cat);
    }
    if constexpr (ABLK) {
      ATTN_LDS const char* base = (ATTN_LDS const char*)(size_t)(sbase + la);
      return __builtin_bit_cast(V8, *(ATTN_LDS const u32x4_t*)(base + (q - NNB) * 1024));
    }
    ATTN_LDS const char* base = (ATTN_LDS const char*)(size_t)(sbase + (la ^ (uint32_t)(64 * kk)));
    return __builtin_bit_cast(V8, *(ATTN_LDS const u32x4_t*)(base + 16 * (q - NNB) * RA));
  };
  auto stage_base = [&](int j) ATTN_INLINE -> uint32_t {
    return (uint32_t)__builtin_amdgcn_readfirstlane(lds0 + (j % ST) * SB);
  };

  f32x4_t acc[NNB][NMB];
#pragma unroll
  for (int nb = 0; nb < NNB; ++nb)
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb) acc[nb][mb] = (f32x4_t){0.f, 0.f, 0.f, 0.f};

  if (n_k > 0) {
    // Prologue: tiles 0 .. LEAD-1 requested; tiles 0 and 1 complete and
    // published before the first step.
#pragma unroll
    for (int tt = 0; tt < LEAD; ++tt)
#pragma unroll
      for (int ci = 0; ci < LPT; ++ci) issue(tt, ci);
    wait_vmcnt<(LEAD - 2) * LPT>();
    barrier_only();
    // Fragments read ahead across a step boundary live in pa / pb, the two
    // alternating with the step parity (the loop is unrolled by two, so the
    // carried values need no register copies).
    V8 pa[PF], pb[PF];
    {
      const uint32_t s0 = stage_base(0);
#pragma unroll
      for (int f = 0; f < PF; ++f) pa[f] = load(s0, f);
    }

    // One step: the products of tile j from the fragments in cur (the first
    // PF) and read here (the rest, PF ahead of their use), the reads of the
    // first PF fragments of tile j + 1 into nxt, this wave's copies of tile
    // j + LEAD, then the wait for its copies of tile j + 2 and the barrier.
    // MASK (the last tile): k positions past K are zeroed in both operands.
    auto step = [&](auto maskc, int j, V8(&cur)[PF], V8(&nxt)[PF]) ATTN_INLINE {
      constexpr bool MASK = decltype(maskc)::value;
      const uint32_t sj = stage_base(j), sn = stage_base(j + 1);
      V8 buf[F];
#pragma unroll
      for (int f = 0; f < PF; ++f) buf[f] = cur[f];
      const int kvalid = K - j * TK;  // k positions of this tile below K
#pragma unroll
      for (int f = 0; f < F; ++f) {
        const int kk = f / FPK, q = f % FPK;
        if (q >= NNB) {
          const int mb = q - NNB;
          if constexpr (MASK) {
            // Each fragment is zeroed once, at its first use.
            const bool zero = 32 * kk + 8 * g >= kvalid;
            const V8 z = __builtin_bit_cast(V8, (u32x4_t){0u, 0u, 0u, 0u});
            if (mb == 0) {
#pragma unroll
              for (int nb = 0; nb < NNB; ++nb) buf[kk * FPK + nb] = zero ? z : buf[kk * FPK + nb];
            }
            buf[f] = zero ? z : buf[f];
          }
#pragma unroll
          for (int nb = 0; nb < NNB; ++nb) acc[nb][mb] = M_::run(buf[kk * FPK + nb], buf[f], acc[nb][mb]);
        }
        if (f + PF < F) buf[f + PF] = load(sj, f + PF);
        else nxt[f + PF - F] = load(sn, f + PF - F);
#pragma unroll
        for (int ci = 0; ci < LPT; ++ci)
          if (f == (2 * ci + 1) * F / (2 * LPT)) issue(j + LEAD, ci);
      }
      // Keep that order through instruction scheduling: per fragment its
      // products, then the read of the fragment PF places later.
#pragma unroll
      for (int f = 0; f < F; ++f) {
        if (f % FPK >= NNB) __builtin_amdgcn_sched_group_barrier(0x008, NNB, 0);  // matrix products
        if (!BT && ((f + PF) % F) % FPK < NNB) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // DS reads
        else __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      // This wave's copies of tile j + 2 complete (those of j + 3 .. j + LEAD
      // may still fly), then the barrier publishes the tile to every wave and
      // frees the stage of tile j for the copies of the next step.
      wait_vmcnt<(LEAD - 2) * LPT>();
      barrier_only();
    };
    const std::false_type no{};
    const std::true_type yes{};
    int j = 0;
    for (; j + 2 < n_k; j += 2) {
      step(no, j, pa, pb);
      step(no, j + 1, pb, pa);
    }
    if (j + 2 == n_k) {
      step(no, j, pa, pb);
#pragma unroll
      for (int f = 0; f < PF; ++f) pa[f] = pb[f];
      ++j;
    }
    step(yes, j, pa, pb);
    // The copies of the tiles past the last land before the LDS is released.
    wait_vmcnt<0>();
  }

  // Epilogue: lane (g, c) of block (nb, mb) holds C[m][n .. n+3] with
  // m = m0 + wm WTM + 16 mb + c, n = n0 + wn WTN + 16 nb + 4 g; N is a
  // multiple of 8, so n < N puts all four columns in range.
  if constexpr (OUT16) {
    // 16-bit C goes through LDS (free once every copy has landed and every
    // wave is past its last read): the fragments are written as rows of the
    // tile, padded by 32 bytes so the 16 rows of one fragment store take
    // disjoint 8-bank spans, then read back 16 bytes per lane along rows, so
    // each global store writes whole row segments of C instead of 16 rows x
    // 32 bytes.
    using S = typename M_::S;
    constexpr int CRB = TN * 2 + 32;  // LDS bytes per C row
    static_assert(TM * CRB <= ST * SB, "C tile fits the LDS ring");
    __syncthreads();
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb) {
      const int r = wm * WTM + 16 * mb + c;
#pragma unroll
      for (int nb = 0; nb < NNB; ++nb) {
        const int col = wn * WTN + 16 * nb + 4 * g;
        const f32x4_t v = acc[nb][mb] * p.alpha;
        S h4[4] = {(S)v[0], (S)v[1], (S)v[2], (S)v[3]};
        const uint32_t lo = (uint32_t)__builtin_bit_cast(uint16_t, h4[0]) |
                            ((uint32_t)__builtin_bit_cast(uint16_t, h4[1]) << 16);
        const uint32_t hi = (uint32_t)__builtin_bit_cast(uint16_t, h4[2]) |
                            ((uint32_t)__builtin_bit_cast(uint16_t, h4[3]) << 16);
        *(ATTN_LDS u32x2_t*)(lds + r * CRB + col * 2) = (u32x2_t){lo, hi};
      }
    }
    __syncthreads();
    constexpr int CPR = TN / 8;  // 16-byte chunks per C row
    constexpr int CHUNKS = TM * CPR;
#pragma unroll
    for (int ch = tid; ch < CHUNKS; ch += NW * 64) {
      const int r = ch / CPR, q = ch - r * CPR;
      const int m = m0 + r, n = n0 + 8 * q;
      const u32x4_t v = *(ATTN_LDS const u32x4_t*)(lds + r * CRB + 16 * q);
      if (m < M && n < N)
        *reinterpret_cast<u32x4_t*>(static_cast<uint16_t*>(p.c) + z * p.sc + (size_t)m * N + n) = v;
    }
    return;
  }
#pragma unroll
  for (int mb = 0; mb < NMB; ++mb) {
    const int m = m0 + wm * WTM + 16 * mb + c;
    if (m >= M) continue;
    const size_t crow = z * p.sc + (size_t)m * N;
#pragma unroll
    for (int nb = 0; nb < NNB; ++nb) {
      const int n = n0 + wn * WTN + 16 * nb + 4 * g;
      if (n >= N) continue;
      *reinterpret_cast<f32x4_t*>(static_cast<float*>(p.c) + crow + n) = acc[nb][mb];
    }
  }
}

template <int DT, int TM, int TN, int TK, int ST, bool BT = false, bool OUT16 = false>
hipError_t launch_gemm(const GemmParams& p, hipStream_t s) {
  const unsigned grid = (unsigned)p.n_tm * (unsigned)p.n_tn;
  hipLaunchKernelGGL((matmul_kernel<DT, TM, TN, TK, ST, BT, OUT16>), dim3(grid, (unsigned)p.batch), dim3(512), 0, s, p);
  return hipGetLastError();
}

}  // namespace attn
