// Matrix-core fragment-layout probe (Section 3.1: which lane owns which
// element is a property of the hardware and must be checked there).
// One wave loads A (row-major 16 x 32) and B (row-major 32 x 16) into the
// operand fragments the attention kernel assumes, runs one 16x16x32 product
// and scatters the accumulator through the assumed C layout.
#include "fwd_kernel.hpp"

namespace attn {

template <int DT>
__global__ void __launch_bounds__(64) mfma_probe_kernel(const uint16_t* a, const uint16_t* b, float* c) {
  using M = Mfma<DT>;
  using V8 = typename M::V8;
  const int lane = threadIdx.x;
  const int g = lane >> 4, col = lane & 15;
  // A fragment: row lane%16, k = 8*(lane/16) + e.
  const V8 af = __builtin_bit_cast(V8, ldg16(a + col * 32 + 8 * g));
  // B fragment: k = 8*(lane/16) + e, column lane%16.
  uint16_t bb[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) bb[e] = b[(8 * g + e) * 16 + col];
  const u32x4_t bw = {(uint32_t)bb[0] | ((uint32_t)bb[1] << 16), (uint32_t)bb[2] | ((uint32_t)bb[3] << 16),
                      (uint32_t)bb[4] | ((uint32_t)bb[5] << 16), (uint32_t)bb[6] | ((uint32_t)bb[7] << 16)};
  const V8 bf = __builtin_bit_cast(V8, bw);
  const f32x4_t acc = M::run(af, bf, (f32x4_t){0.f, 0.f, 0.f, 0.f});
  // C fragment: row 4*(lane/16) + r, column lane%16.
#pragma unroll
  for (int r = 0; r < 4; ++r) c[(4 * g + r) * 16 + col] = acc[r];
}

hipError_t launch_mfma_probe(int atom, const void* a, const void* b, float* c, hipStream_t s) {
  if (atom == ATTN_BF16)
    hipLaunchKernelGGL((mfma_probe_kernel<ATTN_BF16>), dim3(1), dim3(64), 0, s,
                       static_cast<const uint16_t*>(a), static_cast<const uint16_t*>(b), c);
  else
    hipLaunchKernelGGL((mfma_probe_kernel<ATTN_F16>), dim3(1), dim3(64), 0, s,
                       static_cast<const uint16_t*>(a), static_cast<const uint16_t*>(b), c);
  return hipGetLastError();
}

}  // namespace attn
