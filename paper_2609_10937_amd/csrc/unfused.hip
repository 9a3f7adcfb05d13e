// Unfused attention baseline (Section 5.4, Table 3): the L x L score matrix
// goes to device memory between three kernels.
//   gemm (A B^T):  S = scale Q K^T, stored in the input type
//   softmax:       S -> P in place, causal-masked entries 0 (the row-softmax
//                  operator of Section 4.3, attn_softmax, on its own tiles)
//   gemm (A B):    O = P V
// The products use the same 16x16x32 matrix-core atom and fragment layouts as
// the fused kernel; operands are staged through LDS in 16-byte chunks.
#include "fwd_kernel.hpp"

namespace attn {

// C[z] (M x N, row-major, type DT) = alpha * A[z] (M x K, row-major) * op(B[z]),
// op(B) = B^T for B stored N x K (B_KN = false) or B for B stored K x N (B_KN = true).
// 256 threads: 2 x 2 waves, each owning a (BM/2) x 64 block of C.  K % 8 == 0.
template <int DT, bool B_KN, int BM>
__global__ void __launch_bounds__(256) gemm_kernel(const uint16_t* __restrict__ A, const uint16_t* __restrict__ B,
                                                   uint16_t* __restrict__ C, int M, int N, int K, float alpha) {
  using Mf = Mfma<DT>;
  using V8 = typename Mf::V8;
  using S = typename Mf::S;
  constexpr int BN = 128, BK = 32;
  constexpr int MT = BM / 32;                       // 16-row blocks per wave
  constexpr int A_CH = BM * BK / 8;                 // 16-byte chunks of the A tile
  constexpr int A_PT = (A_CH + 255) / 256;
  constexpr int B_CH = BN * BK / 8;
  constexpr int B_PT = (B_CH + 255) / 256;
  constexpr int B_UNITS = (BK / 4) * (BN / 8);      // K x N layout: 4 k-rows x 8 columns
  __shared__ __attribute__((aligned(16))) uint16_t As[BM * BK];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[BN * BK];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, c = lane & 15;
  const int wm = w >> 1, wn = w & 1;
  const int m_blk = blockIdx.x * BM, n_blk = blockIdx.y * BN;
  const size_t z = blockIdx.z;
  A += z * (size_t)M * K;
  B += z * (size_t)N * K;
  C += z * (size_t)M * N;

  // 16-byte chunk ch of a 64-byte LDS row r lives at chunk ch ^ ((r >> 1) & 3).
  auto swz = [](int r, int ch) { return ch ^ ((r >> 1) & 3); };

  u32x4_t ar[A_PT];
  u32x4_t br[B_KN ? 1 : B_PT];
  u32x4_t bu[B_KN ? 4 : 1];

  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < A_PT; ++i) {
      const int ci = tid + 256 * i;
      const int r = ci >> 2, ch = ci & 3;
      u32x4_t x = {0u, 0u, 0u, 0u};
      if ((A_CH % 256 == 0 || ci < A_CH) && m_blk + r < M && k0 + 8 * ch < K)
        x = ldg16(A + (size_t)(m_blk + r) * K + k0 + 8 * ch);
      ar[i] = x;
    }
    if constexpr (!B_KN) {
#pragma unroll
      for (int i = 0; i < B_PT; ++i) {
        const int ci = tid + 256 * i;
        const int r = ci >> 2, ch = ci & 3;
        u32x4_t x = {0u, 0u, 0u, 0u};
        if (n_blk + r < N && k0 + 8 * ch < K) x = ldg16(B + (size_t)(n_blk + r) * K + k0 + 8 * ch);
        br[i] = x;
      }
    } else {
      // unit = 4 consecutive k rows x 8 consecutive columns
      const int kq = tid % (BK / 4), nc = tid / (BK / 4);
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        u32x4_t x = {0u, 0u, 0u, 0u};
        const int kk = k0 + 4 * kq + rr, nn = n_blk + 8 * nc;
        if (tid < B_UNITS && kk < K && nn < N) x = ldg16(B + (size_t)kk * N + nn);
        bu[rr] = x;
      }
    }
  };

  auto lstore = [&]() {
#pragma unroll
    for (int i = 0; i < A_PT; ++i) {
      const int ci = tid + 256 * i;
      if (A_CH % 256 == 0 || ci < A_CH) {
        const int r = ci >> 2, ch = ci & 3;
        *reinterpret_cast<u32x4_t*>(As + r * BK + swz(r, ch) * 8) = ar[i];
      }
    }
    if constexpr (!B_KN) {
#pragma unroll
      for (int i = 0; i < B_PT; ++i) {
        const int ci = tid + 256 * i;
        const int r = ci >> 2, ch = ci & 3;
        *reinterpret_cast<u32x4_t*>(Bs + r * BK + swz(r, ch) * 8) = br[i];
      }
    } else if (tid < B_UNITS) {
      const int kq = tid % (BK / 4), nc = tid / (BK / 4);
      // granule kq (4 k values) of LDS rows n = 8nc + e
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int j = e >> 1;
        uint32_t lo, hi;
        if (e & 1) {
          lo = (bu[0][j] >> 16) | (bu[1][j] & 0xffff0000u);
          hi = (bu[2][j] >> 16) | (bu[3][j] & 0xffff0000u);
        } else {
          lo = (bu[0][j] & 0xffffu) | (bu[1][j] << 16);
          hi = (bu[2][j] & 0xffffu) | (bu[3][j] << 16);
        }
        const int n = 8 * nc + e;
        *reinterpret_cast<u32x2_t*>(Bs + n * BK + swz(n, kq >> 1) * 8 + (kq & 1) * 4) = (u32x2_t){lo, hi};
      }
    }
  };

  f32x4_t acc[MT][4];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = (f32x4_t){0.f, 0.f, 0.f, 0.f};

  gload(0);
  for (int k0 = 0; k0 < K; k0 += BK) {
    __syncthreads();
    lstore();
    __syncthreads();
    if (k0 + BK < K) gload(k0 + BK);
    V8 af[MT], bf[4];
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      const int r = wm * (BM / 2) + 16 * i + c;
      af[i] = __builtin_bit_cast(V8, *reinterpret_cast<const u32x4_t*>(As + r * BK + swz(r, g) * 8));
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = wn * 64 + 16 * j + c;
      bf[j] = __builtin_bit_cast(V8, *reinterpret_cast<const u32x4_t*>(Bs + r * BK + swz(r, g) * 8));
    }
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = Mf::run(af[i], bf[j], acc[i][j]);
  }

#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m_blk + wm * (BM / 2) + 16 * i + 4 * g + r;
        const int n = n_blk + wn * 64 + 16 * j + c;
        if (m < M && n < N) {
          const S v = (S)(alpha * acc[i][j][r]);
          C[(size_t)m * N + n] = __builtin_bit_cast(uint16_t, v);
        }
      }
}

template <int DT>
static hipError_t run_unfused(const void* q, const void* k, const void* v, void* o, void* ws, int BH, int L,
                              int d, float scale, int causal, const attn_softmax_report_t& sm, hipStream_t s) {
  const uint16_t* Q = static_cast<const uint16_t*>(q);
  const uint16_t* K = static_cast<const uint16_t*>(k);
  const uint16_t* V = static_cast<const uint16_t*>(v);
  uint16_t* Sm = static_cast<uint16_t*>(ws);
  uint16_t* O = static_cast<uint16_t*>(o);
  hipLaunchKernelGGL((gemm_kernel<DT, false, 128>), dim3((L + 127) / 128, (L + 127) / 128, BH), dim3(256), 0, s,
                     Q, K, Sm, L, L, d, scale);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const SoftmaxParams sp{Sm, Sm, (int64_t)BH * L, L, sm.seg, sm.split, causal};
  e = launch_softmax(sp, DT, true, (unsigned)sm.grid, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((gemm_kernel<DT, true, 64>), dim3((L + 63) / 64, (d + 127) / 128, BH), dim3(256), 0, s,
                     static_cast<const uint16_t*>(Sm), V, O, L, d, L, 1.0f);
  return hipGetLastError();
}

hipError_t launch_unfused(const void* q, const void* k, const void* v, void* o, void* ws, int BH, int L, int d,
                          float scale, int causal, int dtype, const attn_softmax_report_t& sm, hipStream_t s) {
  if (dtype == ATTN_BF16) return run_unfused<ATTN_BF16>(q, k, v, o, ws, BH, L, d, scale, causal, sm, s);
  return run_unfused<ATTN_F16>(q, k, v, o, ws, BH, L, d, scale, causal, sm, s);
}

}  // namespace attn
