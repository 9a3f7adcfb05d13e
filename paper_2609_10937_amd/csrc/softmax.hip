// Row softmax with the online algorithm of Section 5.3, as a standalone
// operator: Y = softmax(X) along each row of a rows x n matrix.
//
// A wave owns one segment of a row (the CU rule splits a row over up to the
// workgroup's waves; their partial statistics are merged with the operator
// of Section 5.3 through LDS).  The segment is read in tiles of one 16-byte
// load per lane (64 lanes x 8 elements): for every tile the lane's running
// maximum m and denominator d take the correction exp(m - m_new) and the
// tile's exponentials; the first MAXT tiles stay in registers (packed 16-bit),
// so a segment of up to MAXT tiles is read from HBM once, and longer ones are
// read again for the output.  Elements past the segment, or above the
// diagonal when causal, enter as -inf (the padding rule of Section 5.3).
// The 64 lanes' (m, d) pairs and then the segments' are merged with the same
// operator, and the output pass writes exp(x - m) / d in the input type.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace attn {

namespace {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

template <int DT>
struct Elem;
template <>
struct Elem<ATTN_BF16> {
  using S = __bf16;
};
template <>
struct Elem<ATTN_F16> {
  using S = _Float16;
};

constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

// (m_a, d_a) (+) (m_b, d_b) with maxima in input units; a side with m = -inf
// (no entries yet) contributes nothing.
__device__ __forceinline__ void merge(float& m, float& d, float mb, float db) {
  const float mn = fmaxf(m, mb);
  const float ref = (mn == -INFINITY ? 0.f : mn) * kLog2e;
  d = d * exp2_hw(__builtin_fmaf(m, kLog2e, -ref)) + db * exp2_hw(__builtin_fmaf(mb, kLog2e, -ref));
  m = mn;
}

template <int DT>
__device__ __forceinline__ float to_f32(uint32_t w, int half) {
  const uint16_t h = (uint16_t)(half ? (w >> 16) : (w & 0xFFFFu));
  return (float)__builtin_bit_cast(typename Elem<DT>::S, h);
}

template <int DT>
__device__ __forceinline__ uint32_t pack2(float a, float b) {
  using S = typename Elem<DT>::S;
  return (uint32_t)__builtin_bit_cast(uint16_t, (S)a) | ((uint32_t)__builtin_bit_cast(uint16_t, (S)b) << 16);
}

}  // namespace

// One workgroup of W waves; waves w and the S - 1 after it (S = p.split)
// share row blockIdx.x * (W / S) + w / S.  ALIGNED: n % 8 == 0 and 16-byte
// aligned bases, so every lane's 8 elements are one 16-byte access; otherwise
// elements are loaded and stored one by one.
template <int DT, int W, int MAXT, bool ALIGNED>
__global__ void __launch_bounds__(W * 64) softmax_kernel(const SoftmaxParams p) {
  __shared__ float2 part[W];
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int S = p.split;
  const int64_t row = (int64_t)blockIdx.x * (W / S) + w / S;
  const int s = w % S;
  const bool live = row < p.rows;
  const int64_t n = p.n;
  const int64_t c0 = (int64_t)s * p.seg;
  const int64_t c1 = live ? (c0 + p.seg < n ? c0 + p.seg : n) : c0;
  // causal: columns above the diagonal of the row's square block are masked
  const int64_t lim = p.causal ? (row % n) + 1 : n;
  const int64_t cend = c1 < lim ? c1 : (lim > c0 ? lim : c0);   // end of the visible columns
  const int64_t ntiles = c1 > c0 ? (c1 - c0 + 511) / 512 : 0;
  const uint16_t* __restrict__ x = static_cast<const uint16_t*>(p.x) + (live ? row : 0) * n;
  uint16_t* __restrict__ y = static_cast<uint16_t*>(p.y) + (live ? row : 0) * n;

  // 8 elements of tile t for this lane as packed words
  auto load = [&](int64_t t, u32x4_t& v) {
    const int64_t col = c0 + t * 512 + 8 * lane;
    if constexpr (ALIGNED) {
      v = (u32x4_t){0u, 0u, 0u, 0u};
      if (col < c1) v = *reinterpret_cast<const u32x4_t*>(x + col);
    } else {
      uint32_t wv[4] = {0u, 0u, 0u, 0u};
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (col + e < c1) wv[e >> 1] |= (uint32_t)x[col + e] << (16 * (e & 1));
      v = (u32x4_t){wv[0], wv[1], wv[2], wv[3]};
    }
  };
  // values of tile t; columns past the segment or above the diagonal -inf
  auto values = [&](int64_t t, const u32x4_t& v, float (&f)[8]) {
    const int64_t col = c0 + t * 512 + 8 * lane;
#pragma unroll
    for (int e = 0; e < 8; ++e) f[e] = col + e < cend ? to_f32<DT>(v[e >> 1], e & 1) : -INFINITY;
  };

  // Pass 1: online statistics over the segment's tiles: m in input units,
  // d in base 2 (each exponential is exp2(x log2 e - m log2 e), one fma).
  float m = -INFINITY, d = 0.f;
  u32x4_t keep[MAXT];
  auto update = [&](int64_t t, const u32x4_t& v) {
    float f[8];
    values(t, v, f);
    float tm = f[0];
#pragma unroll
    for (int e = 1; e < 8; ++e) tm = fmaxf(tm, f[e]);
    const float mn = fmaxf(m, tm);
    const float ref = (mn == -INFINITY ? 0.f : mn) * kLog2e;
    float acc = d * exp2_hw(__builtin_fmaf(m, kLog2e, -ref));     // correction of the old sum
#pragma unroll
    for (int e = 0; e < 8; ++e) acc += exp2_hw(__builtin_fmaf(f[e], kLog2e, -ref));
    d = acc;
    m = mn;
  };
#pragma unroll
  for (int t = 0; t < MAXT; ++t)
    if (t < ntiles) load(t, keep[t]);
#pragma unroll
  for (int t = 0; t < MAXT; ++t)
    if (t < ntiles) update(t, keep[t]);
  for (int64_t t = MAXT; t < ntiles; ++t) {
    u32x4_t v;
    load(t, v);
    update(t, v);
  }
  // Merge the 64 lanes, then the S segments of the row.
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float mo = __shfl_xor(m, off);
    const float dd = __shfl_xor(d, off);
    merge(m, d, mo, dd);
  }
  if (S > 1) {
    if (lane == 0) part[w] = make_float2(m, d);
    __syncthreads();
    const int base = w - s;
    m = -INFINITY;
    d = 0.f;
    for (int i = 0; i < S; ++i) merge(m, d, part[base + i].x, part[base + i].y);
  }
  if (!live || ntiles == 0) return;
  const float ref = (m == -INFINITY ? 0.f : m) * kLog2e;
  const float inv = d > 0.f ? 1.f / d : 0.f;

  // Pass 2: outputs.
  auto store = [&](int64_t t, const u32x4_t& v) {
    const int64_t col = c0 + t * 512 + 8 * lane;
    if (col >= c1) return;
    float f[8];
    values(t, v, f);
    uint32_t o[4];
#pragma unroll
    for (int e = 0; e < 8; e += 2)
      o[e >> 1] = pack2<DT>(exp2_hw(__builtin_fmaf(f[e], kLog2e, -ref)) * inv,
                            exp2_hw(__builtin_fmaf(f[e + 1], kLog2e, -ref)) * inv);
    if constexpr (ALIGNED) {
      // The output is not read again here: a streaming (non-temporal) store.
      __builtin_nontemporal_store((u32x4_t){o[0], o[1], o[2], o[3]}, reinterpret_cast<u32x4_t*>(y + col));
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (col + e < c1) y[col + e] = (uint16_t)(o[e >> 1] >> (16 * (e & 1)));
    }
  };
#pragma unroll
  for (int t = 0; t < MAXT; ++t)
    if (t < ntiles) store(t, keep[t]);
  for (int64_t t = MAXT; t < ntiles; ++t) {
    u32x4_t v;
    load(t, v);
    store(t, v);
  }
}

hipError_t launch_softmax(const SoftmaxParams& p, int dtype, bool aligned, unsigned grid, hipStream_t s) {
  constexpr int W = kSoftmaxWaves, T = kSoftmaxTiles;
  if (dtype == ATTN_BF16) {
    if (aligned) hipLaunchKernelGGL((softmax_kernel<ATTN_BF16, W, T, true>), dim3(grid), dim3(W * 64), 0, s, p);
    else hipLaunchKernelGGL((softmax_kernel<ATTN_BF16, W, T, false>), dim3(grid), dim3(W * 64), 0, s, p);
  } else {
    if (aligned) hipLaunchKernelGGL((softmax_kernel<ATTN_F16, W, T, true>), dim3(grid), dim3(W * 64), 0, s, p);
    else hipLaunchKernelGGL((softmax_kernel<ATTN_F16, W, T, false>), dim3(grid), dim3(W * 64), 0, s, p);
  }
  return hipGetLastError();
}

}  // namespace attn
