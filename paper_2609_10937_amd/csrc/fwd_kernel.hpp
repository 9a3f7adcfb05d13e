// Fused attention forward for gfx950 (CDNA4), one workgroup per
// (query tile, head, key-range split); Figure 2 of the paper.
//
// Each wave owns 16*QB query rows and runs Algorithm 1 over the key/value
// tiles of its workgroup's range:
//   GEMM1  S^T = K_t Q^T          (v_mfma_f32_16x16x32_{bf16,f16}, fp32 acc)
//   mask   causal / past-the-end keys -> -inf (Section 4.3 padding rule)
//   stats  running reference max m and sum delta per query row
//   GEMM2  O^T = V_t^T P^T        (same atom, fp32 acc)
// Computing S transposed puts query q on lane%16 in both products: the C
// fragment of S^T (lane holds S^T[4*(lane/16)+r][lane%16]) is, after packing
// to 16 bits, exactly the B operand of the second product once its k index is
// permuted (k = 8*(lane/16)+e  <->  key 4*(lane/16)+e or 16+4*(lane/16)+e-4).
// V^T is read with the same permutation by the transposing LDS read.  So P
// never leaves registers -- the paper's E_t^T LDS round trip (Section 5.3)
// is gone.
//
// Fragment layouts (Section 3.1: a hardware fact, checked on the device by
// attn_mfma_probe):
//   A[16 x 32]: lane holds A[lane%16][8*(lane/16) + 0..7]
//   B[32 x 16]: lane holds B[8*(lane/16) + 0..7][lane%16]
//   C[16 x 16]: lane holds C[4*(lane/16) + 0..3][lane%16]
// ds_read_b64_tr_b16, within each 16-lane group: lane i receives element i%4
// of the 4-element rows addressed by lanes 4e+i/4, e = 0..3.  Pointing lane j
// at V[row0 + j/4][col0 + 4*(j%4)] therefore hands lane i the column
// V[row0 .. row0+3][col0 + i]: four keys of one output column, the A operand.
//
// LDS holds a ring of ST stages, each a K tile and a V tile stored row-major
// ([t_kv][d]) in 16-byte chunks, XOR-swizzled per row so that the operand
// reads of a 16-lane group touch distinct banks.  Tiles move HBM -> LDS with
// global_load_lds_dwordx4 (lane l of a wave writes bytes 16l..16l+15 of a
// 1 KB block; each lane picks the source chunk that belongs at its slot), so
// no registers stage them and nothing is transposed on the way.  Up to
// ST-2 tiles beyond the one being computed are in flight; one barrier per
// tile.
//
// Softmax bookkeeping keeps a per-row reference max m that is only raised
// when a new row maximum exceeds it by more than 2^TAU in the exponent (the
// merge of Section 4.3 holds for any common reference point, so the result is
// the same; exponentiated weights stay below 2^TAU).  Most tiles then need no
// rescaling of O.  The row sum adds the 16-bit weights that enter the second
// product (v_dot2 with ones), so the weights the output is normalised by are
// exactly the ones applied to V.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace attn {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef short i16x8_t __attribute__((ext_vector_type(8)));

#define ATTN_LDS __attribute__((address_space(3)))
#define ATTN_GLOBAL __attribute__((address_space(1)))

template <int DT>
struct Mfma;

template <>
struct Mfma<ATTN_BF16> {
  using V8 = bf16x8_t;
  using V2 = bf16x2_t;
  using S = __bf16;
  static __device__ __forceinline__ f32x4_t run(V8 a, V8 b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  // a.x + a.y (+ acc), exact products with one, fp32 accumulation
  static __device__ __forceinline__ float sum2(V2 a, float acc) {
    const V2 one = {(__bf16)1.0f, (__bf16)1.0f};
    return __builtin_amdgcn_fdot2_f32_bf16(a, one, acc, false);
  }
};

template <>
struct Mfma<ATTN_F16> {
  using V8 = f16x8_t;
  using V2 = f16x2_t;
  using S = _Float16;
  static __device__ __forceinline__ f32x4_t run(V8 a, V8 b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ float sum2(V2 a, float acc) {
    const V2 one = {(_Float16)1.0f, (_Float16)1.0f};
    return __builtin_amdgcn_fdot2(a, one, acc, false);
  }
};

__device__ __forceinline__ u32x4_t ldg16(const uint16_t* p) {
  return *reinterpret_cast<const u32x4_t*>(p);
}

__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

// Maximum over the four 16-lane rows of a wave (lanes l, l^16, l^32, l^48),
// with the row-swapping permutes of CDNA4 (VALU, no LDS round trip).
__device__ __forceinline__ float max_across_rows(float x) {
  const uint32_t u = __builtin_bit_cast(uint32_t, x);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  const float y = fmaxf(__builtin_bit_cast(float, (uint32_t)a[0]), __builtin_bit_cast(float, (uint32_t)a[1]));
  const uint32_t v = __builtin_bit_cast(uint32_t, y);
  const auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return fmaxf(__builtin_bit_cast(float, (uint32_t)b[0]), __builtin_bit_cast(float, (uint32_t)b[1]));
}

__device__ __forceinline__ float sum_across_rows(float x) {
  const uint32_t u = __builtin_bit_cast(uint32_t, x);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  const float y = __builtin_bit_cast(float, (uint32_t)a[0]) + __builtin_bit_cast(float, (uint32_t)a[1]);
  const uint32_t v = __builtin_bit_cast(uint32_t, y);
  const auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return __builtin_bit_cast(float, (uint32_t)b[0]) + __builtin_bit_cast(float, (uint32_t)b[1]);
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding:
// vmcnt[3:0] in bits 3:0, vmcnt[5:4] in bits 15:14; expcnt and lgkmcnt at max).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Workgroup barrier that orders LDS accesses but leaves in-flight
// global->LDS copies alone (the compiler's __syncthreads would drain them).
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// 16-byte chunk swizzles of a row-major [rows][KCH chunks] tile (KCH = 16
// for d = 128, 8 for d = 64), chosen so that every operand read of the
// kernel hits distinct LDS banks:
//  K (GEMM1 A operand, ds_read_b128): 16 lanes read 16 consecutive rows at
//    one logical chunk -> distinct physical chunks across rows.
//  V (GEMM2 A operand, ds_read_b64_tr_b16): a 32-lane pair of groups reads
//    rows base + 0..3 and base + 4..7, two adjacent chunks each -> the row's
//    low three bits select distinct chunk positions.
template <int KCH>
__device__ __forceinline__ int k_swz(int r) {
  if constexpr (KCH == 16) return r & 15;
  else return (r >> 1) & 7;
}
template <int KCH>
__device__ __forceinline__ int v_swz(int r) {
  if constexpr (KCH == 16) return (2 * (r & 3)) | (8 * ((r >> 2) & 1));
  else return 2 * ((r >> 1) & 3);
}

// Online-softmax step of Algorithm 1 for one tile of scores s (S^T
// fragments, raw logits): row maxima, the lazily raised reference max, the
// 16-bit weights packed as the B operand of the second product, and the row
// sums of those weights.  MASK = true for tiles crossing the causal diagonal
// or the end of the sequence.
template <bool MASK, typename M, int NKB, int NP, int QB, int NDB>
__device__ __forceinline__ void softmax_tile(f32x4_t (&s)[NKB][QB], typename M::V8 (&pk)[NP][QB], float (&m)[QB],
                                             float (&l)[QB], f32x4_t (&o)[QB][NDB], int kv0, int q0, int g, int c,
                                             int L, int causal, float cs, float thr) {
  using V2 = typename M::V2;
  using S = typename M::S;
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int q = q0 + 16 * qb + c;
    bool keep[NKB][4];
    if constexpr (MASK) {
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int kv = kv0 + 16 * kb + 4 * g + r;
          keep[kb][r] = kv < L && !(causal && kv > q);
          if (!keep[kb][r]) s[kb][qb][r] = -INFINITY;
        }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
      mx = fmaxf(fmaxf(mx, s[kb][qb][0]), fmaxf(fmaxf(s[kb][qb][1], s[kb][qb][2]), s[kb][qb][3]));
    mx = max_across_rows(mx);
    // Raise the reference only when an exponent would exceed TAU (and on a
    // row's first visible key, whatever the scale).
    const float lim = (m[qb] == -INFINITY) ? -INFINITY : m[qb] + thr;
    if (__any(mx > lim)) {
      const float m_new = fmaxf(m[qb], mx);
      const float corr = (m[qb] == -INFINITY) ? 0.f : exp2_hw((m[qb] - m_new) * cs);
      l[qb] *= corr;
#pragma unroll
      for (int db = 0; db < NDB; ++db) o[qb][db] *= corr;
      m[qb] = m_new;
    }
    const float mc = (m[qb] == -INFINITY) ? 0.f : m[qb] * cs;
    float rs = l[qb];
#pragma unroll
    for (int pp = 0; pp < NP; ++pp) {
      V2 h2[4];
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int r = 0; r < 4; r += 2) {
          float e0 = exp2_hw(__builtin_fmaf(s[2 * pp + h][qb][r], cs, -mc));
          float e1 = exp2_hw(__builtin_fmaf(s[2 * pp + h][qb][r + 1], cs, -mc));
          if constexpr (MASK) {
            e0 = keep[2 * pp + h][r] ? e0 : 0.f;
            e1 = keep[2 * pp + h][r + 1] ? e1 : 0.f;
          }
          h2[2 * h + r / 2] = (V2){(S)e0, (S)e1};
        }
#pragma unroll
      for (int j = 0; j < 4; ++j) rs = M::sum2(h2[j], rs);
      pk[pp][qb] = __builtin_shufflevector(__builtin_shufflevector(h2[0], h2[1], 0, 1, 2, 3),
                                           __builtin_shufflevector(h2[2], h2[3], 0, 1, 2, 3),
                                           0, 1, 2, 3, 4, 5, 6, 7);
    }
    l[qb] = rs;
  }
}

template <int DT, int D, int TKV, int QB, int NW, int ST>
__global__ void __launch_bounds__(NW * 64) fwd_kernel(const FwdParams p) {
  using M = Mfma<DT>;
  using V8 = typename M::V8;
  using V2 = typename M::V2;
  using S = typename M::S;
  constexpr int TQW = 16 * QB;              // query rows per wave
  constexpr int TILE_Q = NW * TQW;          // query rows per workgroup
  constexpr int KC = D / 32;                // k steps of GEMM1
  constexpr int NKB = TKV / 16;             // 16-key blocks of S^T
  constexpr int NP = TKV / 32;              // k steps of GEMM2
  constexpr int NDB = D / 16;               // 16-row blocks of O^T
  constexpr int KCH = D / 8;                // 16-byte chunks per row
  constexpr int TILE = TKV * D;             // elements of one K or V tile
  constexpr int CHUNKS = TKV * KCH;
  constexpr int LPW = CHUNKS / (NW * 64);   // 1 KB copies per wave per tile and tensor
  constexpr float TAU = 8.0f;
  static_assert(TKV % 32 == 0 && D % 32 == 0 && KCH >= 8 && (KCH & (KCH - 1)) == 0, "tile alignment");
  static_assert(CHUNKS % (NW * 64) == 0, "tile copies must split evenly across waves");
  // Tiles kept in flight beyond the one being computed: bounded by the ring
  // (ST - 2) and by the 6-bit vector-memory counter (2*LPW copies per tile).
  constexpr int DEPTH = (ST - 2) < 63 / (2 * LPW) ? (ST - 2) : 63 / (2 * LPW);
  static_assert(ST >= 2 && DEPTH >= 0, "stages");

  __shared__ __attribute__((aligned(1024))) uint16_t smem[ST * 2 * TILE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int g = lane >> 4;
  const int c = lane & 15;
  const int L = p.L;

  // Workgroup -> (query tile, head, split).  Heads vary fastest among
  // workgroups of one query-tile rank; causal launches heavy tiles first.
  const int per_rank = p.BH * p.n_split;
  const int rank = blockIdx.x / per_rank;
  const int rem = blockIdx.x - rank * per_rank;
  const int head = rem / p.n_split;
  const int split = rem - head * p.n_split;
  const int qt = p.causal ? (p.n_qt - 1 - rank) : rank;

  const size_t hoff = (size_t)head * (size_t)L * D;
  const uint16_t* __restrict__ Qh = static_cast<const uint16_t*>(p.q) + hoff;
  const uint16_t* __restrict__ Kh = static_cast<const uint16_t*>(p.k) + hoff;
  const uint16_t* __restrict__ Vh = static_cast<const uint16_t*>(p.v) + hoff;

  const int q_wg = qt * TILE_Q;
  const int q0 = q_wg + w * TQW;

  int n_kv = (L + TKV - 1) / TKV;
  if (p.causal) {
    const int last = min(L, q_wg + TILE_Q);
    n_kv = min(n_kv, (last + TKV - 1) / TKV);
  }
  const int t_begin = split * p.tiles_per_split;
  const int t_end = min(n_kv, t_begin + p.tiles_per_split);

  // Copy tile t of K and V into stage `stage`: the wave's LPW 1 KB blocks of
  // each tile image.  Image slot P holds row P/KCH, logical chunk
  // (P%KCH) ^ swizzle(row).  Rows past the end are clamped to row L-1
  // (finite data that the mask removes).
  auto issue = [&](int t, int stage) {
    const int kv0 = t * TKV;
    uint16_t* ks = smem + stage * 2 * TILE;
    uint16_t* vs = ks + TILE;
#pragma unroll
    for (int i = 0; i < LPW; ++i) {
      const int blk = w * LPW + i;
      const int P = blk * 64 + lane;
      const int r = P / KCH, pc = P % KCH;
      const size_t row = (size_t)min(kv0 + r, L - 1) * D;
      __builtin_amdgcn_global_load_lds((ATTN_GLOBAL void*)(Kh + row + ((pc ^ k_swz<KCH>(r)) * 8)),
                                       (ATTN_LDS void*)(ks + blk * 512), 16, 0, 0);
      __builtin_amdgcn_global_load_lds((ATTN_GLOBAL void*)(Vh + row + ((pc ^ v_swz<KCH>(r)) * 8)),
                                       (ATTN_LDS void*)(vs + blk * 512), 16, 0, 0);
    }
  };

  // Q fragments: B operand of S^T = K Q^T, one 16-byte load per (block, k step).
  V8 qf[QB][KC];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int r = q0 + 16 * qb + c;
#pragma unroll
    for (int kc = 0; kc < KC; ++kc) {
      u32x4_t x = {0u, 0u, 0u, 0u};
      if (r < L) x = ldg16(Qh + (size_t)r * D + 32 * kc + 8 * g);
      qf[qb][kc] = __builtin_bit_cast(V8, x);
    }
  }
  // Drain the Q loads here: the loop's waits count only tile copies.
  wait_vmcnt<0>();
#pragma unroll
  for (int j = 0; j <= DEPTH; ++j)
    if (t_begin + j < t_end) issue(t_begin + j, j);

  f32x4_t o[QB][NDB];
  float m[QB], l[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    m[qb] = -INFINITY;
    l[qb] = 0.f;
#pragma unroll
    for (int db = 0; db < NDB; ++db) o[qb][db] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
  }

  const float cs = p.c;
  const float thr = TAU / cs;  // +inf when cs == 0: the reference never moves
  int stage = 0;
  for (int t = t_begin; t < t_end; ++t) {
    // This wave's copies of tile t are complete once no more than the copies
    // of the tiles issued after it (up to DEPTH tiles) are outstanding;
    // vector-memory operations retire in issue order.
    const int after = min(DEPTH, t_end - 1 - t);
    if (after >= DEPTH) wait_vmcnt<2 * LPW * DEPTH>();
    else if (after == 2) wait_vmcnt<(DEPTH > 2 ? 4 * LPW : 0)>();
    else if (after == 1) wait_vmcnt<(DEPTH > 1 ? 2 * LPW : 0)>();
    else wait_vmcnt<0>();
    lds_barrier();  // tile t visible to all waves; every wave is done with tile t-1
    if (t + DEPTH + 1 < t_end) {
      const int st_next = stage + DEPTH + 1 >= ST ? stage + DEPTH + 1 - ST : stage + DEPTH + 1;
      issue(t + DEPTH + 1, st_next);
    }

    const int kv0 = t * TKV;
    // Wave-uniform: skip waves with no valid row or whose rows all precede the tile.
    const bool live = (q0 < L) && !(p.causal && kv0 > q0 + TQW - 1);
    if (live) {
      const uint16_t* Ks = smem + stage * 2 * TILE;
      const uint16_t* Vs = Ks + TILE;
      const bool need_mask = (kv0 + TKV > L) || (p.causal && kv0 + TKV - 1 > q0);

      // GEMM1: s[kb][qb][r] = <K[kv0 + 16kb + 4g + r], Q[q0 + 16qb + c]>
      f32x4_t s[NKB][QB];
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) s[kb][qb] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
        const int row = 16 * kb + c;
#pragma unroll
        for (int kc = 0; kc < KC; ++kc) {
          const int phys = (4 * kc + g) ^ k_swz<KCH>(row);
          const V8 kf = __builtin_bit_cast(V8, *reinterpret_cast<const u32x4_t*>(Ks + row * D + phys * 8));
#pragma unroll
          for (int qb = 0; qb < QB; ++qb) s[kb][qb] = M::run(kf, qf[qb][kc], s[kb][qb]);
        }
      }

      V8 pk[NP][QB];
      if (need_mask)
        softmax_tile<true, M>(s, pk, m, l, o, kv0, q0, g, c, L, p.causal, cs, thr);
      else
        softmax_tile<false, M>(s, pk, m, l, o, kv0, q0, g, c, L, p.causal, cs, thr);

      // GEMM2: o[qb][db][r] += sum_k V^T[16db + 4g + r][k] P^T[k][q]
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        // lane c addresses row 4g + c/4 (+16 for the upper half), column 16db + 4(c%4)
        const int col = 16 * db + 4 * (c & 3);
        const int cpart = 4 * (c & 1);
#pragma unroll
        for (int pp = 0; pp < NP; ++pp) {
          i16x4_t half[2];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int R = 32 * pp + 16 * h + 4 * g + (c >> 2);
            const int phys = (col >> 3) ^ v_swz<KCH>(R);
            half[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (ATTN_LDS i16x4_t*)(Vs + R * D + phys * 8 + cpart));
          }
          const i16x8_t cat = {half[0][0], half[0][1], half[0][2], half[0][3],
                               half[1][0], half[1][1], half[1][2], half[1][3]};
          const V8 va = __builtin_bit_cast(V8, cat);
#pragma unroll
          for (int qb = 0; qb < QB; ++qb) o[qb][db] = M::run(va, pk[pp][qb], o[qb][db]);
        }
      }
    }
    stage = (stage + 1 == ST) ? 0 : stage + 1;
  }

  // Epilogue.  Each of the four lane groups holds a partial row sum over its
  // key subset (same reference max), so the total is their sum.
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const float lt = sum_across_rows(l[qb]);
    const int q = q0 + 16 * qb + c;
    if (p.n_split == 1) {
      const float inv = lt > 0.f ? 1.f / lt : 0.f;
      if (q < L) {
        uint16_t* orow = static_cast<uint16_t*>(p.o) + hoff + (size_t)q * D;
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          const f32x4_t v = o[qb][db] * inv;
          S h4[4] = {(S)v[0], (S)v[1], (S)v[2], (S)v[3]};
          const uint32_t lo = (uint32_t)__builtin_bit_cast(uint16_t, h4[0]) |
                              ((uint32_t)__builtin_bit_cast(uint16_t, h4[1]) << 16);
          const uint32_t hi = (uint32_t)__builtin_bit_cast(uint16_t, h4[2]) |
                              ((uint32_t)__builtin_bit_cast(uint16_t, h4[3]) << 16);
          *reinterpret_cast<u32x2_t*>(orow + 16 * db + 4 * g) = (u32x2_t){lo, hi};
        }
      }
    } else if (q < L) {
      const size_t prow = ((size_t)split * p.BH + head) * (size_t)L + q;
      float* po = p.part_o + prow * D;
#pragma unroll
      for (int db = 0; db < NDB; ++db) *reinterpret_cast<f32x4_t*>(po + 16 * db + 4 * g) = o[qb][db];
      if (g == 0) *reinterpret_cast<float2*>(p.part_ml + prow * 2) = make_float2(m[qb], lt);
    }
  }
}

template <int DT, int D, int TKV, int QB, int NW, int ST>
hipError_t launch_fwd(const FwdParams& p, unsigned grid, hipStream_t s) {
  hipLaunchKernelGGL((fwd_kernel<DT, D, TKV, QB, NW, ST>), dim3(grid), dim3(NW * 64), 0, s, p);
  return hipGetLastError();
}

}  // namespace attn
