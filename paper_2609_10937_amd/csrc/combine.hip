// Merge of key-range partial results (Section 4.3, the associative operator
// on (max, sum) extended to the output accumulator, applied across splits).
// Each split's reference point is stored in the base-2 domain (scale log2 e
// times a logit), so the weights are plain powers of two.
// One thread per (row, 4 consecutive output columns).
#include "fwd_kernel.hpp"

namespace attn {

template <int DT, int D>
__global__ void __launch_bounds__(256) combine_kernel(const FwdParams p) {
  using S = typename Mfma<DT>::S;
  constexpr int QUADS = D / 4;
  const int64_t rows = (int64_t)p.BH * p.L;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= rows * QUADS) return;
  const int64_t row = idx / QUADS;
  const int d4 = (int)(idx - row * QUADS);
  const int64_t stride = rows;  // rows per split

  float m = -INFINITY;
  for (int s = 0; s < p.n_split; ++s) m = fmaxf(m, p.part_ml[(s * stride + row) * 2]);
  float lt = 0.f;
  f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < p.n_split; ++s) {
    const float ms = p.part_ml[(s * stride + row) * 2];
    const float ls = p.part_ml[(s * stride + row) * 2 + 1];
    const float wgt = (ms == -INFINITY) ? 0.f : exp2_hw(ms - m);
    lt += wgt * ls;
    const f32x4_t po = *reinterpret_cast<const f32x4_t*>(p.part_o + (s * stride + row) * D + 4 * d4);
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

hipError_t launch_combine(const FwdParams& p, int d, int dtype, hipStream_t s) {
  const int64_t threads = (int64_t)p.BH * p.L * (d / 4);
  const unsigned grid = (unsigned)((threads + 255) / 256);
  if (dtype == ATTN_BF16) {
    if (d == 256) hipLaunchKernelGGL((combine_kernel<ATTN_BF16, 256>), dim3(grid), dim3(256), 0, s, p);
    else if (d == 128) hipLaunchKernelGGL((combine_kernel<ATTN_BF16, 128>), dim3(grid), dim3(256), 0, s, p);
    else if (d == 96) hipLaunchKernelGGL((combine_kernel<ATTN_BF16, 96>), dim3(grid), dim3(256), 0, s, p);
    else hipLaunchKernelGGL((combine_kernel<ATTN_BF16, 64>), dim3(grid), dim3(256), 0, s, p);
  } else {
    if (d == 256) hipLaunchKernelGGL((combine_kernel<ATTN_F16, 256>), dim3(grid), dim3(256), 0, s, p);
    else if (d == 128) hipLaunchKernelGGL((combine_kernel<ATTN_F16, 128>), dim3(grid), dim3(256), 0, s, p);
    else if (d == 96) hipLaunchKernelGGL((combine_kernel<ATTN_F16, 96>), dim3(grid), dim3(256), 0, s, p);
    else hipLaunchKernelGGL((combine_kernel<ATTN_F16, 64>), dim3(grid), dim3(256), 0, s, p);
  }
  return hipGetLastError();
}

}  // namespace attn
