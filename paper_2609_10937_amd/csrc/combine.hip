// Merge of key-range partial results (Section 5.3, the associative operator
// on (max, sum) extended to the output accumulator, applied across splits).
// Each split's reference point is stored in the base-2 domain (scale log2 e
// times a logit), so the weights are plain powers of two.
// One thread per (row, 4 consecutive output columns).
#include "fwd_kernel.hpp"

namespace attn {

// NS is a compile-time bound on the split count (2, 4, 8 or 16), so each
// thread's loads (NS reference/sum pairs and NS 16-byte partials) issue
// together.  Slots past the actual count n re-read split n - 1 (cache hits)
// and take weight 0, which leaves the maximum, the sum and the accumulator
// unchanged.
template <int DT, int D, int NS>
__global__ void __launch_bounds__(256) combine_kernel(const FwdParams p) {
  using S = typename Mfma<DT>::S;
  constexpr int QUADS = D / 4;
  const int n_split = p.n_split;
  const int64_t rows = (int64_t)p.BH * p.L;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= rows * QUADS) return;
  const int64_t row = idx / QUADS;
  const int d4 = (int)(idx - row * QUADS);
  const int64_t stride = rows;  // rows per split

  float m = -INFINITY;
#pragma unroll
  for (int s = 0; s < NS; ++s) m = fmaxf(m, p.part_ml[(min(s, n_split - 1) * stride + row) * 2]);
  float lt = 0.f;
  f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    const int64_t sr = min(s, n_split - 1) * stride + row;
    const float ms = p.part_ml[sr * 2];
    const float ls = p.part_ml[sr * 2 + 1];
    const float wgt = (s >= n_split || ms == -INFINITY) ? 0.f : exp2_hw(ms - m);
    lt += wgt * ls;
    const f32x4_t po = *reinterpret_cast<const f32x4_t*>(p.part_o + sr * D + 4 * d4);
    acc += wgt * po;
  }
  const float inv = lt > 0.f ? 1.f / lt : 0.f;
  acc *= inv;
  S h4[4] = {(S)acc[0], (S)acc[1], (S)acc[2], (S)acc[3]};
  const uint32_t lo = (uint32_t)__builtin_bit_cast(uint16_t, h4[0]) |
                      ((uint32_t)__builtin_bit_cast(uint16_t, h4[1]) << 16);
  const uint32_t hi = (uint32_t)__builtin_bit_cast(uint16_t, h4[2]) |
                      ((uint32_t)__builtin_bit_cast(uint16_t, h4[3]) << 16);
  *reinterpret_cast<u32x2_t*>(static_cast<uint16_t*>(p.o) + row * D + 4 * d4) = (u32x2_t){lo, hi};
}

template <int DT, int D>
static void launch_combine_d(const FwdParams& p, unsigned grid, hipStream_t s) {
  if (p.n_split <= 2) hipLaunchKernelGGL((combine_kernel<DT, D, 2>), dim3(grid), dim3(256), 0, s, p);
  else if (p.n_split <= 4) hipLaunchKernelGGL((combine_kernel<DT, D, 4>), dim3(grid), dim3(256), 0, s, p);
  else if (p.n_split <= 8) hipLaunchKernelGGL((combine_kernel<DT, D, 8>), dim3(grid), dim3(256), 0, s, p);
  else hipLaunchKernelGGL((combine_kernel<DT, D, 16>), dim3(grid), dim3(256), 0, s, p);
}

template <int DT>
static void launch_combine_t(const FwdParams& p, int d, unsigned grid, hipStream_t s) {
  if (d == 256) launch_combine_d<DT, 256>(p, grid, s);
  else if (d == 128) launch_combine_d<DT, 128>(p, grid, s);
  else if (d == 96) launch_combine_d<DT, 96>(p, grid, s);
  else launch_combine_d<DT, 64>(p, grid, s);
}

hipError_t launch_combine(const FwdParams& p, int d, int dtype, hipStream_t s) {
  if (p.n_split < 1 || p.n_split > 16) return hipErrorInvalidValue;  // the largest compiled bound
  const int64_t threads = (int64_t)p.BH * p.L * (d / 4);
  const unsigned grid = (unsigned)((threads + 255) / 256);
  if (dtype == ATTN_BF16) launch_combine_t<ATTN_BF16>(p, d, grid, s);
  else launch_combine_t<ATTN_F16>(p, d, grid, s);
  return hipGetLastError();
}

}  // namespace attn
