// Fused attention forward for gfx950 (CDNA4), one workgroup per
// (query tile, head, key-range split) -- with causal masking and split key
// ranges, per non-empty piece of a query tile's own key range; Figure 2 of
// the paper.
//
// Each wave owns 16*QB query rows and runs Algorithm 1 over the key/value
// tiles of its workgroup's range:
//   GEMM1  S^T = K_t Q^T          (v_mfma_f32_16x16x32_{bf16,f16}, fp32 acc)
//   mask   causal / past-the-end keys -> -inf (Section 5.3 padding rule)
//   stats  running reference max m and sum delta per query row
//   GEMM2  O^T = V_t^T P^T        (same atom, fp32 acc)
// Computing S transposed puts query q on lane%16 in both products: the C
// fragment of S^T (lane holds S^T[4*(lane/16)+r][lane%16]) is, after packing
// to 16 bits, exactly the B operand of the second product once its k index is
// permuted (k = 8*(lane/16)+e  <->  key 4*(lane/16)+e or 16+4*(lane/16)+e-4).
// V^T is read with the same permutation by the transposing LDS read.  So P
// never leaves registers -- the paper's E_t^T LDS round trip (Section 6.1)
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
// buffer_load_dwordx4 ... lds through a buffer descriptor per tile (lane l of
// a wave writes bytes 16l..16l+15 of a 1 KB block; each lane picks the source
// chunk that belongs at its slot), so no registers stage them and nothing is
// transposed on the way.
//
// Schedule.  A step of a wave is a matrix phase (GEMM2 of the previous tile
// and GEMM1 of the current one: 64 products plus 4 for the row sums) and a
// vector phase (the softmax of the current tile).  With two waves per SIMD
// the two run one phase apart (ping-pong): while one issues matrix products
// the other issues the exponentials, which is the overlap a single wave
// cannot get because its own vector work waits for its products.  Every
// step ends with a workgroup barrier; the operand reads of a matrix phase
// are software-pipelined PF fragments ahead of the products that use them.
//
// PERSIST = true is the same kernel as a persistent launch, one workgroup per
// CU, for launches of many short query tiles: each workgroup runs a fixed list
// of query tiles back to back through one ring of K/V tiles, so the next
// tile's first key tiles and Q rows load while the current one finishes
// instead of after its workgroup has left the CU.
//
// Softmax bookkeeping keeps a per-row reference max m that is only raised
// when a score would give a weight above 2^8 (the merge of Section 5.3 holds
// for any common reference point, so the result is the same).  Most tiles
// then need neither row maxima nor rescaling of O.  The row sums come from
// the second product itself (a block of ones times the packed weights), so
// the weights the output is normalised by are exactly the 16-bit weights
// applied to V.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

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
typedef int32_t i32x4_t __attribute__((ext_vector_type(4)));

#define ATTN_LDS __attribute__((address_space(3)))
#define ATTN_GLOBAL __attribute__((address_space(1)))
// Lambdas of the kernel body: always inlined (a call would spill live state).
#define ATTN_INLINE __attribute__((always_inline))

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
};

template <>
struct Mfma<ATTN_F16> {
  using V8 = f16x8_t;
  using V2 = f16x2_t;
  using S = _Float16;
  static __device__ __forceinline__ f32x4_t run(V8 a, V8 b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
  }
};

// Two 16-bit ones packed in a 32-bit word.
template <int DT>
constexpr uint32_t kOne2 = DT == ATTN_BF16 ? 0x3F803F80u : 0x3C003C00u;

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

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding:
// vmcnt[3:0] in bits 3:0, vmcnt[5:4] in bits 15:14; expcnt and lgkmcnt at max).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// One 16-byte-per-lane copy from global memory straight into LDS
// (global_load_lds_dwordx4): lane l's 16 bytes at base + off land at LDS byte
// address lds_dst + 16 l.  The LDS address goes through M0, which needs one
// wait state before the copy reads it.  Written as inline assembly so that the compiler
// does not treat every later LDS read as depending on the copy: completion
// is tracked here with explicit vector-memory counter waits and barriers.
// base and lds_dst are wave-uniform; they pass through readfirstlane so that
// they are scalar operands whatever the compiler can prove.
__device__ __forceinline__ uint64_t uniform_ptr(const void* p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  return ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(v >> 32)) << 32) |
         (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)v);
}
__device__ __forceinline__ void copy_to_lds(const void* base, uint32_t off, uint32_t lds_dst) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(uniform_ptr(base)),
               "s"(__builtin_amdgcn_readfirstlane(lds_dst))
               : "memory", "m0");
}
// Buffer resource (a gfx9 V#) over `bytes` bytes from `base`: raw (stride 0,
// no swizzle), so a lane whose offset is at or past `bytes` reads zeros and
// touches no memory.  Built from wave-uniform values; the fields pass
// through readfirstlane so that the descriptor lives in scalar registers.
__device__ __forceinline__ i32x4_t buffer_rsrc(uint64_t base, uint32_t bytes) {
  i32x4_t r;
  r[0] = __builtin_amdgcn_readfirstlane((int32_t)(uint32_t)base);
  r[1] = __builtin_amdgcn_readfirstlane((int32_t)((uint32_t)(base >> 32) & 0xffffu));
  r[2] = __builtin_amdgcn_readfirstlane((int32_t)bytes);
  r[3] = 0x00020000;  // 32-bit data format, no swizzle, no index stride
  return r;
}
// One 16-byte-per-lane copy from a buffer straight into LDS
// (buffer_load_dwordx4 ... lds): lane l's 16 bytes at byte offset `off` of
// the buffer land at LDS byte address lds_dst + 16 l, zeros for a lane past
// the buffer's end.  Inline assembly for the same reason as copy_to_lds.
__device__ __forceinline__ void copy_to_lds_buf(i32x4_t rsrc, uint32_t off, uint32_t lds_dst) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds" ::"v"(off), "s"(rsrc),
               "s"(__builtin_amdgcn_readfirstlane(lds_dst))
               : "memory", "m0");
}
// Workgroup barrier that orders LDS accesses but leaves in-flight
// global->LDS copies alone (the compiler's __syncthreads would drain them).
__device__ __forceinline__ void lds_barrier() {
  // Scheduling fences on both sides: no instruction may be moved across a
  // phase boundary (the asm statement alone only orders memory operations).
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

// 16-byte chunk swizzles of a row-major [rows][KCH chunks] tile (KCH = 32
// for d = 256, 16 for d = 128, 8 for d = 64), chosen so that every operand
// read of the kernel hits distinct LDS banks (64 banks of 4 bytes: a chunk's
// bank group is its position modulo 16, and a 256-byte row of banks holds
// 16 chunks):
//  K (GEMM1 A operand, ds_read_b128): 16 lanes read 16 consecutive rows at
//    one logical chunk -> distinct physical chunks modulo 16 across rows.
//  V (GEMM2 A operand, ds_read_b64_tr_b16): a 32-lane pair of groups reads
//    rows base + 0..3 and base + 4..7, two adjacent chunks each -> the row's
//    low three bits select distinct chunk positions.
// Rows of 32 chunks (two rows of banks) take the 16-chunk swizzles: only
// the low four bits of the chunk index decide the bank group.
template <int KCH>
__device__ __forceinline__ int k_swz(int r) {
  static_assert(KCH == 8 || KCH == 16 || KCH == 32, "chunks per row");
  if constexpr (KCH >= 16) return r & 15;
  else return (r >> 1) & 7;
}
template <int KCH>
__device__ __forceinline__ int v_swz(int r) {
  if constexpr (KCH >= 16) return (2 * (r & 3)) | (8 * ((r >> 2) & 1));
  else return 2 * ((r >> 1) & 3);
}

// Online-softmax step of Algorithm 1 for one tile.  On entry s holds the raw
// scores of the tile (S^T fragments); one fma each brings them to the base-2
// domain relative to the row's reference point mref (cs = scale log2 e; the
// product is not pre-scaled through Q, whose rounding to 16 bits would
// double the error of the scores).  The reference of
// a row can be any common point for all of its keys (the merge of Section 5.3
// holds for every choice), so it only moves when a weight would exceed 2^8:
// each lane checks its own scores against lim (8, or -inf while the row has
// no reference yet) and only if one passes are the row maxima taken and the
// reference raised to them; the tile's scores are shifted by the same amount
// and the accumulated output and row sums are rescaled by corr in the next
// matrix phase.  Out: the 16-bit weights 2^s packed as the B operand of the
// second product.  The row sums are formed by the second product itself (a
// block of ones times the packed weights), so they add exactly the 16-bit
// weights that multiply V.  MASK = true for tiles crossing the causal
// diagonal or the end of the sequence.
// Maximum of N values as a tree of 3-way maxima (v_max3_f32): depth
// log3 N instead of a chain of N/2 dependent operations.
template <int N>
__device__ __forceinline__ float tree_max(const float* t) {
  if constexpr (N == 1) {
    return t[0];
  } else if constexpr (N == 2) {
    return fmaxf(t[0], t[1]);
  } else {
    constexpr int K = (N + 2) / 3;
    float u[K];
#pragma unroll
    for (int i = 0; i < N / 3; ++i) u[i] = fmaxf(fmaxf(t[3 * i], t[3 * i + 1]), t[3 * i + 2]);
    if constexpr (N % 3 == 2) u[N / 3] = fmaxf(t[N - 2], t[N - 1]);
    if constexpr (N % 3 == 1) u[N / 3] = t[N - 1];
    return tree_max<K>(u);
  }
}

template <bool MASK, typename M, int NKB, int NP, int QB>
__device__ __forceinline__ void softmax_tile(f32x4_t (&s)[NKB][QB], typename M::V8 (&pk)[NP][QB], float (&mref)[QB],
                                             float (&lim)[QB], float (&corr)[QB], bool& rescale, int kv0, int q0,
                                             int g, int c, int L, int causal, float cs) {
  using V2 = typename M::V2;
  using S = typename M::S;
  // Scores of all row blocks first (independent work for the scheduler),
  // then one check for the whole tile.
  float mx[QB];
  bool hit = false;
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) s[kb][qb][r] = __builtin_fmaf(s[kb][qb][r], cs, -mref[qb]);
    if constexpr (MASK) {
      const int q = q0 + 16 * qb + c;
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int kv = kv0 + 16 * kb + 4 * g + r;
          if (!(kv < L && !(causal && kv > q))) s[kb][qb][r] = -INFINITY;
        }
    }
    float t[4 * NKB];
#pragma unroll
    for (int i = 0; i < 4 * NKB; ++i) t[i] = s[i >> 2][qb][i & 3];
    mx[qb] = tree_max<4 * NKB>(t);
    hit |= mx[qb] > lim[qb];
  }
  if (__any(hit)) {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      if (!__any(mx[qb] > lim[qb])) continue;
      const float rmx = max_across_rows(mx[qb]);
      const bool has = lim[qb] != -INFINITY;
      // New reference: the row maximum if above the old one; a row without
      // a reference takes its maximum as is (nothing has been accumulated).
      const float delta = has ? fmaxf(rmx, 0.f) : (rmx == -INFINITY ? 0.f : rmx);
      if (__any(delta != 0.f)) {
        corr[qb] = has ? exp2_hw(-delta) : 0.f;
        mref[qb] += delta;
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) s[kb][qb] -= delta;
        rescale = true;
      }
      if (rmx != -INFINITY) lim[qb] = 8.f;
    }
  }
#pragma unroll
  for (int qb = 0; qb < QB; ++qb)
#pragma unroll
    for (int pp = 0; pp < NP; ++pp) {
      uint32_t wd[4];
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int r = 0; r < 4; r += 2) {
          const float e0 = exp2_hw(s[2 * pp + h][qb][r]);
          const float e1 = exp2_hw(s[2 * pp + h][qb][r + 1]);
          wd[2 * h + r / 2] = __builtin_bit_cast(uint32_t, (V2){(S)e0, (S)e1});
        }
      pk[pp][qb] = __builtin_bit_cast(typename M::V8, (u32x4_t){wd[0], wd[1], wd[2], wd[3]});
    }
  // The weights are complete here: without this the compiler may sink the
  // exponentials past the end-of-step barrier, next to their first use.
#pragma unroll
  for (int qb = 0; qb < QB; ++qb)
#pragma unroll
    for (int pp = 0; pp < NP; ++pp) asm volatile("" : "+v"(pk[pp][qb]));
}

template <int DT, int D, int TKV, int QB, int NW, int ST, bool PERSIST>
__global__ void __launch_bounds__(NW * 64) fwd_kernel(const FwdParams p) {
  using M = Mfma<DT>;
  using V8 = typename M::V8;
  using S = typename M::S;
  constexpr int TQW = 16 * QB;              // query rows per wave
  constexpr int TILE_Q = NW * TQW;          // query rows per workgroup
  constexpr int KC = D / 32;                // k steps of GEMM1
  constexpr int NKB = TKV / 16;             // 16-key blocks of S^T
  constexpr int NP = TKV / 32;              // k steps of GEMM2
  constexpr int NDB = D / 16;               // 16-row blocks of O^T
  // K/V rows in LDS hold DL elements: d itself when a power of two, else the
  // next power of two (d = 96 -> 128), the chunks past d copies of the last
  // one that no product reads, so every swizzle and copy pattern is the
  // power-of-two one.
  constexpr int DL = (D & (D - 1)) == 0 ? D : (D <= 128 ? 128 : 256);
  constexpr int KCH = DL / 8;               // 16-byte chunks per LDS row
  constexpr int TILE = TKV * DL;            // elements of one K or V tile in LDS
  constexpr int CHUNKS = TKV * KCH;
  constexpr int NCW = NW;                   // waves that copy tiles (all)
  constexpr int LPW = CHUNKS / (NCW * 64);  // 1 KB copies per copying wave per tile and tensor
  static_assert(TKV % 32 == 0 && D % 32 == 0 && D <= DL && KCH >= 8 && (KCH & (KCH - 1)) == 0, "tile alignment");
  static_assert(CHUNKS % (NCW * 64) == 0, "tile copies must split evenly across waves");
  // Tiles requested ahead.  In M(j) a wave requests its part of tile
  // j + 1 + AHEAD, whose stage held tile j + 1 + AHEAD - ST; that V tile is
  // read in M(j + 2 + AHEAD - ST), which every wave must have finished: all
  // have finished M(j - 1) at the barrier before M(j), and the other group
  // may be in M(j) itself, reading tiles j and j - 1; both allow ST - 3.  A
  // wave has at most AHEAD + 1 tiles of 2 LPW copies outstanding, and the
  // 6-bit vector-memory counter holds 63.
  constexpr int AHEAD = (ST - 3) < 63 / (2 * LPW) - 1 ? (ST - 3) : 63 / (2 * LPW) - 1;
  static_assert(ST >= 3 && AHEAD >= 0, "stages");
  constexpr int NVF = NP * NDB;             // V^T fragments per tile (GEMM2 A operands)
  constexpr int NKF = KC * NKB;             // K fragments per tile (GEMM1 A operands)
  constexpr int PF = 4;                     // operand fragments loaded ahead of their use

  __shared__ __attribute__((aligned(1024))) uint16_t smem[ST * 2 * TILE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4;
  const int c = lane & 15;
  const int L = p.L;
  // Waves w and w + 4 of a workgroup share a SIMD.  With two waves per SIMD
  // the second runs half a step behind the first, so that one issues
  // matrix products while the other runs the softmax.
  const int grp = NW == 8 ? (w >> 2) : 0;

  // Workgroup -> (query tile, head, split).  A unit is one (head, split)
  // pair: its n_qt query tiles all read the same key range.  Workgroups are
  // dispatched to the 8 XCDs round-robin (block b on XCD b % 8), each XCD with
  // its own L2, so when the units divide evenly XCD x takes units x, x + 8, ...
  // and runs them xg at a time, ranks outermost within such a group: the
  // workgroups an XCD runs together then stream the same K/V tiles through
  // its L2.  A group holds at least 64 query tiles (two per CU of an XCD) so
  // that heavy and light causal tiles still balance.  Otherwise, with a split
  // key range, all splits of a query tile go to one XCD (tile t, counted
  // head-major, on XCD t % 8), so its L2 fetches the tile's Q rows once
  // instead of once per split: every workgroup loads Q at the start, where
  // its key tiles follow over the whole loop.  Causal launches heavy tiles
  // (high ranks of the query order) first; causal with split key ranges
  // launches only the non-empty pieces of each query tile's own key range
  // (below).  Otherwise the plain order: units fastest within a rank.
  const int units = p.BH * p.n_split;
  int xg;
  const FwdOrder order = fwd_order(p, &xg);
  int head = 0, split = 0, qt = 0;
  bool placed = false;
  if constexpr (TILE_Q % TKV == 0) {
    if (order == kOrderPieces) {
      // Causal with split key ranges: query tile qt sees its first n_kv(qt)
      // key tiles, cut into pieces of P = tiles_per_split tiles.  A whole
      // query tile qt < n_qt - 1 sees C (qt + 1) tiles (C = TILE_Q / TKV), so
      // its piece k exists when C (qt + 1) > k P, that is for the
      // nf - floor(k P / C) whole tiles qt >= floor(k P / C) (nf = n_qt - 1).
      // Heads run fastest; then the last query tile's pieces (whole tile or
      // not); then, piece-major, the first piece of every whole tile
      // (heaviest first), then every second piece, ...  Consecutive
      // workgroups go to consecutive XCDs, and this order gives each XCD a
      // like mix of long and short pieces.
      constexpr int C = TILE_Q / TKV;
      const int P = p.tiles_per_split;
      head = blockIdx.x % p.BH;
      const int j = blockIdx.x / p.BH;
      const int n_last = (min(L, p.n_qt * TILE_Q) + TKV - 1) / TKV;  // key tiles the last query tile sees
      const int a_last = (n_last + P - 1) / P;
      if (j < a_last) {
        qt = p.n_qt - 1;
        split = j;
      } else {
        // The host launches exactly the pieces (at most n_split per tile), so
        // jp falls within piece k before k reaches n_split - 1.
        const int nf = p.n_qt - 1;
        int jp = j - a_last, k = 0;
        for (; k + 1 < p.n_split; ++k) {
          const int cnt = nf - (k * P) / C;
          if (jp < cnt) break;
          jp -= cnt;
        }
        qt = max(0, nf - 1 - jp);
        split = k;
      }
      placed = true;
    }
  }
  // Workgroup b of the order above -> (head, split, query tile).
  auto decode = [&](int b, int& hd_out, int& sp_out, int& qt_out) ATTN_INLINE {
    int unit, rank;
    if (order == kOrderUnits) {
      const int x = b % 8, i = b / 8;
      const int per_group = xg * p.n_qt;
      const int gi = i / per_group, r = i - gi * per_group;
      rank = r / xg;
      unit = x + 8 * (gi * xg + (r - rank * xg));
    } else if (order == kOrderTiles) {
      const int x = b % 8, i = b / 8;
      const int sp = i % p.n_split;
      const int t = (i / p.n_split) * 8 + x;
      const int hd = t / p.n_qt;
      rank = t - hd * p.n_qt;
      unit = hd * p.n_split + sp;
    } else {
      rank = b / units;
      unit = b - rank * units;
    }
    hd_out = unit / p.n_split;
    sp_out = unit - hd_out * p.n_split;
    qt_out = p.causal ? (p.n_qt - 1 - rank) : rank;
  };

  // Persistent launch (PERSIST: one workgroup per CU, without split key
  // ranges, so the order above has one workgroup per query tile, BH n_qt in
  // all).  The workgroups b = 8 i + x that the order above puts on XCD x
  // become units of work shared by the launch's S = gridDim.x / 8 workgroups
  // on that XCD, in rounds taken snake-wise: in round r slot s takes item
  // r S + s when r is even and r S + S - 1 - s when r is odd, so that a
  // heavy causal query tile of one round pairs with a light one of the next.
  // A workgroup runs its units back to back through one ring of K/V tiles.
  [[maybe_unused]] const int px = blockIdx.x % 8, ps = blockIdx.x / 8, pS = gridDim.x / 8;
  [[maybe_unused]] const int p_items = PERSIST ? (p.BH * p.n_qt - px + 7) / 8 : 0;
  [[maybe_unused]] auto p_item = [&](int r) ATTN_INLINE { return r * pS + ((r & 1) ? pS - 1 - ps : ps); };
  if constexpr (PERSIST) {
    if (p_item(0) >= p_items) return;  // no unit here (the whole workgroup leaves before any barrier)
    decode(8 * p_item(0) + px, head, split, qt);
  } else if (!placed) {
    decode(blockIdx.x, head, split, qt);
  }

  size_t hoff = (size_t)head * (size_t)L * D;
  const uint16_t* __restrict__ Qh = static_cast<const uint16_t*>(p.q) + hoff;
  const uint16_t* __restrict__ Kh = static_cast<const uint16_t*>(p.k) + hoff;
  const uint16_t* __restrict__ Vh = static_cast<const uint16_t*>(p.v) + hoff;

  // Key tiles query tile qt_ sees (causal: up to its last row).
  auto tiles_of = [&](int qt_) ATTN_INLINE {
    int nk = (L + TKV - 1) / TKV;
    if (p.causal) nk = min(nk, (min(L, qt_ * TILE_Q + TILE_Q) + TKV - 1) / TKV);
    return nk;
  };
  int q0 = qt * TILE_Q + w * TQW;
  const int n_kv = tiles_of(qt);
  const int t_begin = split * p.tiles_per_split;
  const int n = min(n_kv, t_begin + p.tiles_per_split) - t_begin;  // tiles of this workgroup

  // LDS image: stage st holds the K tile at byte st*STAGEB and the V tile
  // TILEB after it, each row-major [TKV][DL] in 16-byte chunks, chunk
  // positions XOR-swizzled per row (k_swz / v_swz).
  constexpr int ROWB = DL * 2;              // bytes per K/V row in LDS
  constexpr int GROWB = D * 2;              // bytes per K/V row in HBM
  constexpr int TILEB = TKV * ROWB;         // bytes per K or V tile
  constexpr int STAGEB = 2 * TILEB;
  ATTN_LDS char* const lds = (ATTN_LDS char*)smem;
  const uint32_t lds0 = (uint32_t)(size_t)lds;

  // Copy tile j (relative to t_begin) of K and V into stage j % ST: the
  // copying wave's LPW 1 KB blocks of each tile image.  Image slot P holds
  // row P/KCH, logical chunk (P%KCH) ^ swizzle(row).  Block b of a tile image
  // (1 KB) holds rows b*RPB .. b*RPB + RPB - 1; copying wave cw takes blocks
  // cw, cw + NCW, cw + 2 NCW, ..., so block i of a lane sits at row
  // r0 + i NCW RPB.  Each copy reads through a buffer descriptor whose base is
  // the tile's first row and whose size covers the rows of this workgroup's
  // key range that the tile holds (none for tiles past the range), so a
  // lane's byte offset within the tile is the same for every tile and rows
  // past the range or the sequence arrive as zeros (finite; the mask removes
  // their keys) without touching memory.  When NCW * RPB is a multiple of
  // 16 rows (the period of both swizzles) the chunk offsets of all of a
  // lane's blocks coincide.
  constexpr int RPB = 1024 / ROWB;
  constexpr bool SHIFT = (NCW * RPB) % 16 == 0;
  const int cw = w;  // index among the copying waves
  const uint32_t r0 = (uint32_t)((cw * 64 + lane) / KCH);
  // A lane's byte offset within a tile for its block i of K (V = false) or
  // V: loop-invariant registers when the blocks share their chunk offsets
  // (the 4- and 8-wave kernels), else formed at each copy.
  auto block_off = [&](int i, bool is_v) ATTN_INLINE -> uint32_t {
    const int r = (int)r0 + i * NCW * RPB, pc = lane % KCH;
    int ch = pc ^ (is_v ? v_swz<KCH>(r) : k_swz<KCH>(r));
    if constexpr (D != DL) ch = min(ch, D / 8 - 1);
    return (uint32_t)(r * GROWB + ch * 16);
  };
  constexpr int NOFF = SHIFT ? LPW : 1;
  uint32_t koff[NOFF], voff[NOFF];
#pragma unroll
  for (int i = 0; i < NOFF; ++i) {
    koff[i] = block_off(i, false);
    voff[i] = block_off(i, true);
  }
  uint64_t kh_base = uniform_ptr(Kh), vh_base = uniform_ptr(Vh);
  // Key rows this workgroup reads: its split's range, clipped to the sequence.
  int kv_end = __builtin_amdgcn_readfirstlane(min(L, (t_begin + max(n, 0)) * TKV));
  // PERSIST: tile indices j count over all of the workgroup's units; the
  // current unit holds j in [cur_start, cur_end), the next one (if any)
  // starts at nx_start = cur_end and has its own bases and key range
  // (nx_kv_end = 0 when there is none, so tiles past the last unit are empty).
  [[maybe_unused]] int cur_start = 0, cur_end = n, nx_start = n, nx_kv_end = 0;
  [[maybe_unused]] uint64_t nkh = kh_base, nvh = vh_base;
  // This wave's part of tile j: its LPW blocks of the K image and of the V
  // image, as copies 0 .. NC-1 (copy 2i is block i of K, 2i+1 block i of V);
  // issue(j, lo, hi) makes copies lo .. hi-1.
  constexpr int NC = 2 * LPW;
  // The K and V buffer descriptors of tile j.
  struct TileRsrc {
    i32x4_t k, v;
  };
  auto tile_rsrc = [&](int j) ATTN_INLINE -> TileRsrc {
    uint64_t kb = kh_base, vb = vh_base;
    int kv0 = (t_begin + j) * TKV, end = kv_end;
    if constexpr (PERSIST) {
      kv0 = (j - cur_start) * TKV;
      if (j >= cur_end) {
        kb = nkh;
        vb = nvh;
        kv0 = (j - nx_start) * TKV;
        end = nx_kv_end;
      }
    }
    const uint32_t bytes = (uint32_t)max(0, min(end - kv0, TKV)) * GROWB;
    return TileRsrc{buffer_rsrc(kb + (uint64_t)kv0 * GROWB, bytes), buffer_rsrc(vb + (uint64_t)kv0 * GROWB, bytes)};
  };
  auto issue_r = [&](const TileRsrc& rs, int j, int lo, int hi) ATTN_INLINE {
    const i32x4_t kr = rs.k, vr = rs.v;
    const uint32_t kdst = (uint32_t)__builtin_amdgcn_readfirstlane(lds0 + (j % ST) * STAGEB) + cw * 1024;
#pragma unroll
    for (int ci = lo; ci < hi; ++ci) {
      const int i = ci >> 1;
      if (ci & 1) copy_to_lds_buf(vr, SHIFT ? voff[i % NOFF] : block_off(i, true), kdst + TILEB + i * NCW * 1024);
      else copy_to_lds_buf(kr, SHIFT ? koff[i % NOFF] : block_off(i, false), kdst + i * NCW * 1024);
    }
  };
  auto issue = [&](int j, int lo, int hi) ATTN_INLINE { issue_r(tile_rsrc(j), j, lo, hi); };
  // This wave's copies of tile j are complete once no more than the copies
  // of the tiles requested after it are outstanding (vector-memory
  // operations retire in issue order).
  auto wait_tile = [&](int j, int last_issued) ATTN_INLINE {
    const int after = last_issued - j;
    if (after >= 3) wait_vmcnt<(AHEAD >= 3 ? 6 * LPW : 0)>();
    else if (after == 2) wait_vmcnt<(AHEAD >= 2 ? 4 * LPW : 0)>();
    else if (after == 1) wait_vmcnt<2 * LPW>();
    else wait_vmcnt<0>();
  };

  const float cs = p.c;  // scale * log2(e): scores in the base-2 domain

  // Prologue copies: tile 0, then the Q loads, then tiles 1 .. AHEAD, so
  // that the Q loads and the first tile travel together; both are complete
  // once only the later tiles' copies are outstanding.
  if (n > 0) issue(0, 0, NC);
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
  if (n > 0) {
#pragma unroll
    for (int j = 1; j <= AHEAD; ++j) issue(j, 0, NC);
    wait_tile(0, AHEAD);
  } else {
    wait_vmcnt<0>();
  }

  f32x4_t o[QB][NDB];
  f32x4_t lacc[QB];  // row sums of the weights (all four entries of a lane equal)
  // Per row: the reference point in the base-2 domain (cs times a logit) and
  // the check limit (-inf until the row has seen a key, then 8).
  float mref[QB], lim[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    mref[qb] = 0.f;
    lim[qb] = -INFINITY;
    lacc[qb] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int db = 0; db < NDB; ++db) o[qb][db] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
  }
  // A raised reference rescales the accumulated output by corr; the softmax
  // only records it, and the next matrix phase applies it before adding the
  // tile's products (so the vector phase never rewrites o) and resets corr.
  float corr[QB];
  bool rescale = false;
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) corr[qb] = 1.f;
  f32x4_t s[NKB][QB];  // scores of the tile between its GEMM1 and its softmax
  V8 pk[NP][QB];       // 16-bit weights of the tile between its softmax and its GEMM2

  // Operand fragments.  V^T (GEMM2 A operand, 16 d x 32 keys): lane c
  // addresses row 4g + c/4 (+16 for the upper half) and column
  // 16db + 4(c%4) of the row-major V tile; the transposing read hands it
  // four keys of one column.  K (GEMM1 A operand, 16 keys x 32 d): one
  // 16-byte read of row 16kb + c.  Neither swizzle depends on the row bits
  // that pp, h or kb set, and db (kc) enters a lane's byte address only
  // through the bits 32*db (64*kc), XORed with the lane's swizzle: so the
  // address is a lane base XOR a per-fragment constant, plus a row offset
  // that the read instruction carries.
  static_assert(ROWB >= 256 || KC * 64 <= ROWB, "operand address bits");
  uint32_t kbase, vbase;
  {
    kbase = (uint32_t)(c * ROWB + ((g ^ k_swz<KCH>(c)) & 3) * 16 + ((k_swz<KCH>(c) >> 2) * 64));
    const int R0 = 4 * g + (c >> 2);
    const int sw = v_swz<KCH>(R0);
    vbase = (uint32_t)(R0 * ROWB + (((c & 3) >> 1) ^ (sw & 1)) * 16 + (sw >> 1) * 32 + 8 * (c & 1));
  }
  auto load_v = [&](uint32_t vb, int pp, int db) ATTN_INLINE -> V8 {
    ATTN_LDS const char* base = (ATTN_LDS const char*)(size_t)(vb ^ (uint32_t)(32 * db));
    const i16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((ATTN_LDS i16x4_t*)(base + (32 * pp) * ROWB));
    const i16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((ATTN_LDS i16x4_t*)(base + (32 * pp + 16) * ROWB));
    const i16x8_t cat = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(V8, cat);
  };
  auto load_k = [&](uint32_t kb0, int kc, int kb) ATTN_INLINE -> V8 {
    ATTN_LDS const char* base = (ATTN_LDS const char*)(size_t)(kb0 ^ (uint32_t)(64 * kc));
    return __builtin_bit_cast(V8, *(ATTN_LDS const u32x4_t*)(base + kb * 16 * ROWB));
  };

  // The stage offsets pass through readfirstlane: as opaque wave-uniform
  // values they stay one scalar add per phase instead of becoming one
  // induction variable per fragment address.
  // The phase also carries this wave's copies of tile jc, spread over the
  // products: the products keep the matrix core busy while a copy waits for
  // the address unit, and the copies of the workgroup's waves do not all
  // queue at once.  Tiles past the range are copied too (in-bounds rows, into
  // stages no later phase reads), which keeps the phase one basic block and
  // the copy count per step constant.
  auto mphase = [&](auto g2c, auto g1c, int j, int jc, const V8 (&qa)[QB][KC]) ATTN_INLINE {
    constexpr bool G2 = decltype(g2c)::value, G1 = decltype(g1c)::value;
    constexpr int F = (G2 ? NVF : 0) + (G1 ? NKF : 0);
    const uint32_t Vs = vbase + (uint32_t)__builtin_amdgcn_readfirstlane(lds0 + ((j + ST - 1) % ST) * STAGEB + TILEB);
    const uint32_t Ks = kbase + (uint32_t)__builtin_amdgcn_readfirstlane(lds0 + (j % ST) * STAGEB);
    TileRsrc crs{};
    if constexpr (G1) crs = tile_rsrc(jc);
    auto load = [&](int f) ATTN_INLINE -> V8 {
      if (G2 && f < NVF) return load_v(Vs, f / NDB, f % NDB);
      const int fk = f - (G2 ? NVF : 0);
      return load_k(Ks, fk / NKB, fk % NKB);
    };
    if (G2 && rescale) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
        for (int db = 0; db < NDB; ++db) o[qb][db] *= corr[qb];
        lacc[qb] *= corr[qb];
        corr[qb] = 1.f;
      }
      rescale = false;
    }
    V8 buf[F];
#pragma unroll
    for (int f = 0; f < PF && f < F; ++f) buf[f] = load(f);
    // Row sums of the previous tile's weights: a 16 x 32 block of ones times
    // P^T, while the first operand reads are in flight.
    if constexpr (G2) {
      const V8 ones = __builtin_bit_cast(V8, (u32x4_t){kOne2<DT>, kOne2<DT>, kOne2<DT>, kOne2<DT>});
#pragma unroll
      for (int pp = 0; pp < NP; ++pp)
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) lacc[qb] = M::run(ones, pk[pp][qb], lacc[qb]);
    }
#pragma unroll
    for (int f = 0; f < F; ++f) {
      if (G2 && f < NVF) {
        const int pp = f / NDB, db = f % NDB;
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) o[qb][db] = M::run(buf[f], pk[pp][qb], o[qb][db]);
      } else {
        const int fk = f - (G2 ? NVF : 0);
        const int kc = fk / NKB, kb = fk % NKB;
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
          s[kb][qb] = M::run(buf[f], qa[qb][kc], kc == 0 ? (f32x4_t){0.f, 0.f, 0.f, 0.f} : s[kb][qb]);
      }
      if (f + PF < F) buf[f + PF] = load(f + PF);
      if constexpr (G1) {
#pragma unroll
        for (int ci = 0; ci < NC; ++ci)
          if (f == (2 * ci + 1) * F / (2 * NC)) issue_r(crs, jc, ci, ci + 1);
      }
    }
    // Keep that order through instruction scheduling: the first PF
    // fragments' reads, then per fragment its QB products and the reads of
    // the fragment PF places later (a V^T fragment is two reads).
    auto reads_of = [](int f) ATTN_INLINE {
      if (G2 && f < NVF) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // DS reads
      else __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    };
#pragma unroll
    for (int f = 0; f < PF && f < F; ++f) reads_of(f);
    if constexpr (G2) __builtin_amdgcn_sched_group_barrier(0x008, NP * QB, 0);  // row-sum products
#pragma unroll
    for (int f = 0; f < F; ++f) {
      __builtin_amdgcn_sched_group_barrier(0x008, QB, 0);  // matrix products
      if (f + PF < F) reads_of(f + PF);
    }
  };

  // Vector phase S(j): the softmax of tile j.  Only tiles that cross the
  // causal diagonal or the end of the sequence take the masked body.
  auto sphase = [&](int j) ATTN_INLINE {
    int kv0 = (t_begin + j) * TKV;
    if constexpr (PERSIST) kv0 = (j - cur_start) * TKV;
    if ((kv0 + TKV > L) || (p.causal && kv0 + TKV - 1 > q0))
      softmax_tile<true, M>(s, pk, mref, lim, corr, rescale, kv0, q0, g, c, L, p.causal, cs);
    else
      softmax_tile<false, M>(s, pk, mref, lim, corr, rescale, kv0, q0, g, c, L, p.causal, cs);
  };

  // Epilogue.  Each of the four lane groups holds a partial row sum over its
  // key subset (same reference), so the total is their sum.  Without a split
  // O / sum is rounded to the input type and stored.  A split stores the same
  // normalised output of its key range (a convex combination of V rows, so in
  // the range of the input type), and beside it, in fp32, its reference (base
  // 2, -inf for a row that saw no key) and its sum, which the merge needs to
  // weigh the splits.
  auto pack4 = [&](const f32x4_t& v) ATTN_INLINE -> u32x2_t {
    S h4[4] = {(S)v[0], (S)v[1], (S)v[2], (S)v[3]};
    const uint32_t lo = (uint32_t)__builtin_bit_cast(uint16_t, h4[0]) |
                        ((uint32_t)__builtin_bit_cast(uint16_t, h4[1]) << 16);
    const uint32_t hi = (uint32_t)__builtin_bit_cast(uint16_t, h4[2]) |
                        ((uint32_t)__builtin_bit_cast(uint16_t, h4[3]) << 16);
    return (u32x2_t){lo, hi};
  };
  auto store_row = [&](uint16_t* row, const f32x4_t (&acc)[NDB], float inv) ATTN_INLINE {
#pragma unroll
    for (int db = 0; db < NDB; ++db) *reinterpret_cast<u32x2_t*>(row + 16 * db + 4 * g) = pack4(acc[db] * inv);
  };
  // PERSIST: the current unit's rows (no split), through a buffer descriptor
  // over its head's O, so rows past the sequence are dropped by the
  // descriptor's range and every wave issues exactly QB * NDB stores (the
  // waits of the unit switch count them).
  [[maybe_unused]] auto store_unit_rows = [&]() ATTN_INLINE {
    const __amdgpu_buffer_rsrc_t ors = __builtin_amdgcn_make_buffer_rsrc(
        reinterpret_cast<void*>(uniform_ptr(static_cast<uint16_t*>(p.o) + hoff)), (short)0,
        __builtin_amdgcn_readfirstlane((int)((uint32_t)L * (uint32_t)(D * 2))), 0x00020000);
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const float lt = lacc[qb][0];
      const float inv = lt > 0.f ? 1.f / lt : 0.f;
      const uint32_t rowb = (uint32_t)(q0 + 16 * qb + c) * (uint32_t)(D * 2) + 8u * (uint32_t)g;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
        __builtin_amdgcn_raw_buffer_store_b64(pack4(o[qb][db] * inv), ors, (int)(rowb + 32u * (uint32_t)db), 0, 0);
    }
  };

  // Phase schedule.  M(j) is the matrix phase of tile j (GEMM2 of tile j-1
  // and GEMM1 of tile j), S(j) its vector phase.  One workgroup barrier per
  // step: between barriers B(j) and B(j+1) group 0 runs M(j) then S(j) and
  // group 1 runs S(j-1) then M(j), so the two waves of a SIMD start each
  // step in different kinds of phase (the matrix phase at raised priority)
  // and drift back into step at every barrier.  Every wave computes every
  // tile of the range: a wave whose rows all precede a tile (causal) sees
  // only masked keys there and adds nothing, which keeps one straight path
  // through the loop.
  //
  // Copies.  A wave requests its part of tile j + 1 + AHEAD during M(j) and
  // has its part of tile j + 1 complete before B(j + 1); the barrier then
  // publishes the whole tile to M(j + 1) of both groups.
  if (n > 0) {
    auto matrix = [&](auto g2c, auto g1c, int j, const V8 (&qa)[QB][KC]) ATTN_INLINE {
      __builtin_amdgcn_s_setprio(1);
      mphase(g2c, g1c, j, j + 1 + AHEAD, qa);
      __builtin_amdgcn_s_setprio(0);
    };
    const std::false_type no{};
    const std::true_type yes{};
    lds_barrier();  // B(0)
    if constexpr (!PERSIST) {
      // End of a wave's step j: its part of tile j + 1 complete, then the
      // barrier.  Group 1's steps end after its matrix phases, group 0's after
      // its vector phases; the phases themselves are one straight sequence.
      auto end_step = [&](int j, int last_issued) ATTN_INLINE {
        if (j + 1 < n) wait_tile(j + 1, last_issued);
        lds_barrier();
      };
      matrix(no, yes, 0, qf);
      if (grp == 1) end_step(0, 1 + AHEAD);
      sphase(0);
      if (grp == 0) end_step(0, 1 + AHEAD);
      for (int j = 1; j < n; ++j) {
        matrix(yes, yes, j, qf);
        if (grp == 1) end_step(j, j + 1 + AHEAD);
        sphase(j);
        if (grp == 0) end_step(j, j + 1 + AHEAD);
      }
      matrix(yes, no, n, qf);
    } else {
      // Units back to back.  The tiles of the next unit are requested like
      // any tile, AHEAD + 1 matrix phases before their own; its Q rows at
      // the start of M(J - 2), J = nx_start its first tile, into qn.  M(J)
      // runs the second product of the finished unit's last tile beside the
      // first product of the new unit (on qn, which becomes qf), and right
      // after it each wave stores the finished unit's rows and starts the
      // statistics over: group 1's S(J - 1) still belongs to the old unit,
      // group 0's S(J) to the new one.  Every unit has at least AHEAD + 2
      // tiles (the host checks), so the copies and the Q rows in flight
      // belong to the current or the next unit only.
      static_assert(AHEAD == 2, "the switch's waits assume two tiles requested ahead");
      constexpr int NST = QB * NDB;  // store instructions of a unit's rows, per wave
      constexpr int QL = QB * KC;    // load instructions of a unit's Q rows, per wave
      static_assert(4 * LPW + NST + QL < 64, "vmcnt range");
      int r = 0;  // round of the current unit
      bool nx_valid = false;
      int nx_head = 0, nx_qt = 0, nx_n = 0;
      auto set_next = [&]() ATTN_INLINE {
        nx_start = cur_end;
        const int it = p_item(r + 1);
        nx_valid = it < p_items;
        nx_kv_end = 0;
        nkh = kh_base;
        nvh = vh_base;
        if (nx_valid) {
          int sp;
          decode(8 * it + px, nx_head, sp, nx_qt);
          nx_n = tiles_of(nx_qt);
          const size_t ho = (size_t)nx_head * (size_t)L * D;
          nkh = uniform_ptr(static_cast<const uint16_t*>(p.k) + ho);
          nvh = uniform_ptr(static_cast<const uint16_t*>(p.v) + ho);
          nx_kv_end = __builtin_amdgcn_readfirstlane(min(L, nx_n * TKV));
        }
      };
      set_next();
      V8 qn[QB][KC];
      // The next unit's Q fragments: one 16-byte buffer load each (rows past
      // the sequence read as zeros).
      auto load_next_q = [&]() ATTN_INLINE {
        const __amdgpu_buffer_rsrc_t qrs = __builtin_amdgcn_make_buffer_rsrc(
            reinterpret_cast<void*>(uniform_ptr(static_cast<const uint16_t*>(p.q) + (size_t)nx_head * (size_t)L * D)),
            (short)0, __builtin_amdgcn_readfirstlane((int)((uint32_t)L * (uint32_t)(D * 2))), 0x00020000);
        const uint32_t rowb = (uint32_t)(nx_qt * TILE_Q + w * TQW + c) * (uint32_t)(D * 2) + 16u * (uint32_t)g;
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
          for (int kc = 0; kc < KC; ++kc)
            qn[qb][kc] = __builtin_bit_cast(
                V8, __builtin_amdgcn_raw_buffer_load_b128(
                        qrs, (int)(rowb + (uint32_t)(16 * qb) * (uint32_t)(D * 2) + 64u * (uint32_t)kc), 0, 0));
        __builtin_amdgcn_sched_barrier(0);
      };
      int last_switch = -8;  // step of the last switch (the finished unit's rows stored after its M)
      // End of step j: this wave's part of tile j + 1 complete, then the
      // barrier.  The copies of tile j + 1 were requested in M(j - 2); the
      // wait counts the operations issued after them (they complete in issue
      // order): two tiles of copies, plus the next unit's Q loads (issued at
      // the start of M(s - 2) for a switch at step s: steps s - 2 and s - 1)
      // and the last unit's stores (after M(s): steps s to s + 2).  The last
      // step waits for a tile past the range, whose copies are empty.
      auto end_step_p = [&](int j) ATTN_INLINE {
        const int e = j - (nx_valid && nx_start - j <= 2 ? nx_start : last_switch);
        if (e >= -2 && e <= 2) {
          if (e < 0) wait_vmcnt<4 * LPW + QL>();
          else wait_vmcnt<4 * LPW + NST>();
        } else {
          wait_vmcnt<4 * LPW>();
        }
        lds_barrier();
      };
      matrix(no, yes, 0, qf);
      if (grp == 1) end_step_p(0);
      sphase(0);
      if (grp == 0) end_step_p(0);
      for (int j = 1;; ++j) {
        const bool sw_now = j == nx_start;
        if (sw_now && !nx_valid) break;  // the last unit's tiles are done
        if (nx_valid && j + 2 == nx_start) load_next_q();
        if (sw_now) {
          // The compiler waits for the Q loads here (and with them for every
          // copy requested before this point: they complete in issue order).
#pragma unroll
          for (int qb = 0; qb < QB; ++qb)
#pragma unroll
            for (int kc = 0; kc < KC; ++kc) qf[qb][kc] = qn[qb][kc];
        }
        matrix(yes, yes, j, qf);
        if (sw_now) {
          store_unit_rows();
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int qb = 0; qb < QB; ++qb) {
            mref[qb] = 0.f;
            lim[qb] = -INFINITY;
            corr[qb] = 1.f;
            lacc[qb] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int db = 0; db < NDB; ++db) o[qb][db] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
          }
          rescale = false;
          head = nx_head;
          qt = nx_qt;
          hoff = (size_t)head * (size_t)L * D;
          q0 = qt * TILE_Q + w * TQW;
          kh_base = nkh;
          vh_base = nvh;
          kv_end = nx_kv_end;
          cur_start = j;
          cur_end = j + nx_n;
          ++r;
          set_next();
          last_switch = j;
        }
        if (grp == 1) end_step_p(j);
        sphase(j);
        if (grp == 0) end_step_p(j);
      }
      matrix(yes, no, cur_end, qf);
    }
    // The copies of the tiles past the range land before the workgroup's
    // LDS is released.
    wait_vmcnt<0>();
  }

  if constexpr (PERSIST) {
    store_unit_rows();
  } else {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const float lt = lacc[qb][0];
      const float inv = lt > 0.f ? 1.f / lt : 0.f;
      int q = q0 + 16 * qb + c;
      // Row offsets at a d that is not a power of two are multiplications: keep
      // the compiler from carrying the Q loads' ones through the loop.
      if constexpr (D != DL) asm volatile("" : "+v"(q));
      if (q >= L) continue;
      if (p.n_split == 1) {
        store_row(static_cast<uint16_t*>(p.o) + hoff + (size_t)q * D, o[qb], inv);
      } else {
        const size_t prow = ((size_t)split * p.BH + head) * (size_t)L + q;
        store_row(static_cast<uint16_t*>(p.part_o) + prow * D, o[qb], inv);
        if (g == 0)
          *reinterpret_cast<float2*>(p.part_ml + prow * 2) =
              make_float2(lim[qb] == -INFINITY ? -INFINITY : mref[qb], lt);
      }
    }
  }
}

template <int DT, int D, int TKV, int QB, int NW, int ST, bool PERSIST = false>
hipError_t launch_fwd(const FwdParams& p, unsigned grid, hipStream_t s) {
  hipLaunchKernelGGL((fwd_kernel<DT, D, TKV, QB, NW, ST, PERSIST>), dim3(grid), dim3(NW * 64), 0, s, p);
  return hipGetLastError();
}

}  // namespace attn
