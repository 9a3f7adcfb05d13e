// Merge of key-range partial results (Section 5.3: the associative operator
// on (max, sum), carried over to the output, applied across the splits).
// Split s left, per row, its output normalised by its own sum (O_s / l_s, in
// the input type), its reference point m_s in the base-2 domain (scale log2 e
// times a logit; -inf for a row that saw none of the split's keys) and its
// sum l_s in fp32.  Against the largest reference M the split weighs
// w_s = l_s 2^(m_s - M), and the output is sum_s w_s (O_s / l_s) / sum_s w_s.
// One thread per (row, 8 consecutive output columns): one 16-byte load per
// split, one 16-byte store.
#include "fwd_kernel.hpp"

namespace attn {

template <int DT>
__device__ __forceinline__ float widen(uint16_t h) {
  if constexpr (DT == ATTN_BF16) return __builtin_bit_cast(float, (uint32_t)h << 16);
  else return (float)__builtin_bit_cast(_Float16, h);
}

// When the fused kernel ran every split of query tile t on XCD t % 8
// (kOrderTiles), BY_TILE orders the merge's workgroups the same way: the
// chunks of 256 (row, octet) items of tile t run on XCD t % 8, whose L2 still
// holds the partials that XCD wrote.  Otherwise one flat order.
//
// With causal pieces (FwdParams::pieces) a row has as many slots as its
// query tile has pieces, computed from the tile sizes.
//
// NS is a compile-time bound on the split count (2, 4, 8 or 16).  Every
// thread first issues all of its loads (NS reference/sum pairs as one 8-byte
// load each and NS 16-byte partials) and only then does arithmetic, so the
// loads overlap instead of waiting for each other one split at a time.  Slots
// past the actual count n re-read split n - 1 (cache hits) and take weight 0,
// which leaves the maximum, the sum and the accumulator unchanged.
template <int DT, int D, int NS, bool BY_TILE>
__global__ void __launch_bounds__(256) combine_kernel(const FwdParams p) {
  using S = typename Mfma<DT>::S;
  constexpr int OCTS = D / 8;
  int n_split = p.n_split;
  const int64_t rows = (int64_t)p.BH * p.L;
  int64_t row;
  int d8;
  if constexpr (BY_TILE) {
    const int wpt = p.tile_q * OCTS / 256;  // workgroups per query tile
    const int x = blockIdx.x % 8, i = blockIdx.x / 8;
    const int t = (i / wpt) * 8 + x;
    const int hd = t / p.n_qt, rank = t - hd * p.n_qt;
    const int item = (i - (i / wpt) * wpt) * 256 + threadIdx.x;
    const int q = rank * p.tile_q + item / OCTS;
    if (q >= p.L) return;
    row = (int64_t)hd * p.L + q;
    d8 = item % OCTS;
  } else {
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= rows * OCTS) return;
    row = idx / OCTS;
    d8 = (int)(idx - row * OCTS);
  }
  if (p.pieces > 0) {
    // Causal pieces: the row's query tile has one piece per tiles_per_split
    // of the key tiles it sees; its later slots hold nothing.
    const int q = (int)(row % p.L), qt = q / p.tile_q;
    const int seen = (min(p.L, (qt + 1) * p.tile_q) + p.t_kv - 1) / p.t_kv;
    n_split = (seen + p.tiles_per_split - 1) / p.tiles_per_split;
  }
  const int64_t stride = rows;  // rows per split
  const float2* __restrict__ ml = reinterpret_cast<const float2*>(p.part_ml);
  const uint16_t* __restrict__ part = static_cast<const uint16_t*>(p.part_o);

  float2 st[NS];
  u32x4_t po[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    const int64_t sr = min(s, n_split - 1) * stride + row;
    st[s] = ml[sr];
    po[s] = *reinterpret_cast<const u32x4_t*>(part + sr * D + 8 * d8);
  }
  // Keep the scheduler from sinking loads below this point.
  __builtin_amdgcn_sched_barrier(0);

  float m = -INFINITY;
#pragma unroll
  for (int s = 0; s < NS; ++s) m = fmaxf(m, st[s].x);
  float lt = 0.f;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    const float wgt = (s >= n_split || st[s].x == -INFINITY) ? 0.f : st[s].y * exp2_hw(st[s].x - m);
    lt += wgt;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[2 * e] += wgt * widen<DT>((uint16_t)(po[s][e] & 0xffffu));
      acc[2 * e + 1] += wgt * widen<DT>((uint16_t)(po[s][e] >> 16));
    }
  }
  const float inv = lt > 0.f ? 1.f / lt : 0.f;
  uint32_t out[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const S a = (S)(acc[2 * e] * inv), b = (S)(acc[2 * e + 1] * inv);
    out[e] = (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
  }
  *reinterpret_cast<u32x4_t*>(static_cast<uint16_t*>(p.o) + row * D + 8 * d8) = (u32x4_t){out[0], out[1], out[2], out[3]};
}

template <int DT, int D, bool BY_TILE>
static void launch_combine_o(const FwdParams& p, unsigned grid, hipStream_t s) {
  if (p.n_split <= 2) hipLaunchKernelGGL((combine_kernel<DT, D, 2, BY_TILE>), dim3(grid), dim3(256), 0, s, p);
  else if (p.n_split <= 4) hipLaunchKernelGGL((combine_kernel<DT, D, 4, BY_TILE>), dim3(grid), dim3(256), 0, s, p);
  else if (p.n_split <= 8) hipLaunchKernelGGL((combine_kernel<DT, D, 8, BY_TILE>), dim3(grid), dim3(256), 0, s, p);
  else hipLaunchKernelGGL((combine_kernel<DT, D, 16, BY_TILE>), dim3(grid), dim3(256), 0, s, p);
}

template <int DT, int D>
static void launch_combine_d(const FwdParams& p, bool by_tile, unsigned grid, hipStream_t s) {
  if (by_tile) launch_combine_o<DT, D, true>(p, grid, s);
  else launch_combine_o<DT, D, false>(p, grid, s);
}

template <int DT>
static void launch_combine_t(const FwdParams& p, int d, bool by_tile, unsigned grid, hipStream_t s) {
  if (d == 256) launch_combine_d<DT, 256>(p, by_tile, grid, s);
  else if (d == 128) launch_combine_d<DT, 128>(p, by_tile, grid, s);
  else if (d == 96) launch_combine_d<DT, 96>(p, by_tile, grid, s);
  else launch_combine_d<DT, 64>(p, by_tile, grid, s);
}

hipError_t launch_combine(const FwdParams& p, int d, int dtype, hipStream_t s) {
  if (p.n_split < 1 || p.n_split > 16) return hipErrorInvalidValue;  // the largest compiled bound
  int xg;
  // Tile order needs whole 256-item chunks per query tile and tiles that
  // cover the sequence.
  const bool by_tile = fwd_order(p, &xg) == kOrderTiles && p.tile_q > 0 &&
                       (p.tile_q * (d / 8)) % 256 == 0 && (int64_t)p.n_qt * p.tile_q >= p.L;
  const int64_t grid = by_tile ? (int64_t)p.BH * p.n_qt * (p.tile_q * (d / 8) / 256)
                               : ((int64_t)p.BH * p.L * (d / 8) + 255) / 256;
  if (grid > 0x7fffffffLL) return hipErrorInvalidValue;
  if (dtype == ATTN_BF16) launch_combine_t<ATTN_BF16>(p, d, by_tile, (unsigned)grid, s);
  else launch_combine_t<ATTN_F16>(p, d, by_tile, (unsigned)grid, s);
  return hipGetLastError();
}

}  // namespace attn
