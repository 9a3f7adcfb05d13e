// Fused attention forward for gfx950 (CDNA4), one workgroup per
// (query tile, head, key-range split); Figure 2 of the paper.
//
// Each wave owns 16*QB query rows and runs Algorithm 1 over the key/value
// tiles of its workgroup's range:
//   GEMM1  S^T = K_t Q^T          (v_mfma_f32_16x16x32_{bf16,f16}, fp32 acc)
//   mask   causal / past-the-end keys -> -inf (Section 4.3 padding rule)
//   stats  running max m and sum delta per query row (online softmax)
//   GEMM2  O^T = V_t^T P^T        (same atom, fp32 acc)
// Computing S transposed puts query q on lane%16 in both products: the C
// fragment of S^T (lane holds S^T[4*(lane/16)+r][lane%16]) is, after packing
// to 16 bits, exactly the B operand of the second product once its k index is
// permuted (k = 8*(lane/16)+e  <->  key 4*(lane/16)+e or 16+4*(lane/16)+e-4);
// V^T is read from LDS with the same permutation.  So P never leaves
// registers -- the paper's E_t^T LDS round trip (Section 5.3) is gone.
//
// Fragment layouts (Section 3.1 warns they are a hardware fact, not a
// consequence of the shape; attn_mfma_probe checks them on the device):
//   A[16 x 32]: lane holds A[lane%16][8*(lane/16) + 0..7]
//   B[32 x 16]: lane holds B[8*(lane/16) + 0..7][lane%16]
//   C[16 x 16]: lane holds C[4*(lane/16) + 0..3][lane%16]
//
// LDS holds two buffers of {K tile row-major [t_kv][d], V tile transposed
// [d][t_kv]}.  16-byte K chunks are XOR-swizzled by row and 8-byte V^T
// granules by d so that the operand reads of one wave hit distinct banks.
// The next tile is loaded from HBM into registers while the current one is
// computed (one barrier per tile).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace attn {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

template <int DT>
struct Mfma;

template <>
struct Mfma<ATTN_BF16> {
  using V8 = bf16x8_t;
  using S = __bf16;
  static __device__ __forceinline__ f32x4_t run(V8 a, V8 b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};

template <>
struct Mfma<ATTN_F16> {
  using V8 = f16x8_t;
  using S = _Float16;
  static __device__ __forceinline__ f32x4_t run(V8 a, V8 b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
  }
};

__device__ __forceinline__ u32x4_t ldg16(const uint16_t* p) {
  return *reinterpret_cast<const u32x4_t*>(p);
}

__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

// XOR swizzle of the 8-byte granule index of a V^T row (granules per row = G).
template <int G>
__device__ __forceinline__ int vt_swizzle(int d) {
  if constexpr (G % 16 == 0)
    return d & 15;
  else
    return (d >> 1) & 7;
}

template <int DT, int D, int TKV, int QB, int NW>
__global__ void __launch_bounds__(NW * 64) fwd_kernel(const FwdParams p) {
  using M = Mfma<DT>;
  using V8 = typename M::V8;
  using S = typename M::S;
  constexpr int NT = NW * 64;
  constexpr int TQW = 16 * QB;          // query rows per wave
  constexpr int TILE_Q = NW * TQW;      // query rows per workgroup
  constexpr int KC = D / 32;            // k steps of GEMM1
  constexpr int NKB = TKV / 16;         // 16-key blocks of S^T
  constexpr int NP = TKV / 32;          // k steps of GEMM2
  constexpr int NDB = D / 16;           // 16-row blocks of O^T
  constexpr int KCH = D / 8;            // 16-byte chunks per K row
  constexpr int K_CHUNKS = TKV * KCH;
  constexpr int K_PT = (K_CHUNKS + NT - 1) / NT;
  constexpr int VG = TKV / 4;           // 8-byte granules per V^T row
  constexpr int V_UNITS = VG * (D / 8); // 4 keys x 8 columns per unit
  constexpr int V_PT = (V_UNITS + NT - 1) / NT;
  constexpr int TILE = TKV * D;
  static_assert(TKV % 32 == 0 && D % 32 == 0 && (KCH & (KCH - 1)) == 0, "tile alignment");

  __shared__ __attribute__((aligned(16))) uint16_t smem[4 * TILE];

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

  f32x4_t o[QB][NDB];
  float m[QB], l[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    m[qb] = -INFINITY;
    l[qb] = 0.f;
#pragma unroll
    for (int db = 0; db < NDB; ++db) o[qb][db] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
  }

  u32x4_t kst[K_PT];
  u32x4_t vst[V_PT][4];

  auto gload = [&](int t) {
    const int kv0 = t * TKV;
#pragma unroll
    for (int i = 0; i < K_PT; ++i) {
      const int ci = tid + i * NT;
      u32x4_t x = {0u, 0u, 0u, 0u};
      if (K_CHUNKS % NT == 0 || ci < K_CHUNKS) {
        const int r = ci / KCH, cc = ci % KCH;
        if (kv0 + r < L) x = ldg16(Kh + (size_t)(kv0 + r) * D + cc * 8);
      }
      kst[i] = x;
    }
#pragma unroll
    for (int i = 0; i < V_PT; ++i) {
      const int ui = tid + i * NT;
      const int kq = ui % VG, dc = ui / VG;
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        u32x4_t x = {0u, 0u, 0u, 0u};
        const int kv = kv0 + 4 * kq + rr;
        if ((V_UNITS % NT == 0 || ui < V_UNITS) && kv < L) x = ldg16(Vh + (size_t)kv * D + dc * 8);
        vst[i][rr] = x;
      }
    }
  };

  auto lstore = [&](int buf) {
    uint16_t* Ks = smem + buf * 2 * TILE;
    uint16_t* Vt = Ks + TILE;
#pragma unroll
    for (int i = 0; i < K_PT; ++i) {
      const int ci = tid + i * NT;
      if (K_CHUNKS % NT == 0 || ci < K_CHUNKS) {
        const int r = ci / KCH, cc = ci % KCH;
        const int phys = cc ^ (r & (KCH - 1));
        *reinterpret_cast<u32x4_t*>(Ks + r * D + phys * 8) = kst[i];
      }
    }
#pragma unroll
    for (int i = 0; i < V_PT; ++i) {
      const int ui = tid + i * NT;
      if (V_UNITS % NT == 0 || ui < V_UNITS) {
        const int kq = ui % VG, dc = ui / VG;
        // vst[i][rr] = V[kv0 + 4kq + rr][8dc .. 8dc+7]; write column e of these
        // four rows as one 8-byte granule of V^T row 8dc+e.
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int j = e >> 1;
          uint32_t lo, hi;
          if (e & 1) {
            lo = (vst[i][0][j] >> 16) | (vst[i][1][j] & 0xffff0000u);
            hi = (vst[i][2][j] >> 16) | (vst[i][3][j] & 0xffff0000u);
          } else {
            lo = (vst[i][0][j] & 0xffffu) | (vst[i][1][j] << 16);
            hi = (vst[i][2][j] & 0xffffu) | (vst[i][3][j] << 16);
          }
          const int d = 8 * dc + e;
          const int phys = kq ^ vt_swizzle<VG>(d);
          *reinterpret_cast<u32x2_t*>(Vt + d * TKV + phys * 4) = (u32x2_t){lo, hi};
        }
      }
    }
  };

  const float cs = p.c;
  if (t_begin < t_end) gload(t_begin);
  int buf = 0;
  for (int t = t_begin; t < t_end; ++t) {
    lstore(buf);
    __syncthreads();
    if (t + 1 < t_end) gload(t + 1);

    const int kv0 = t * TKV;
    // Wave-uniform: skip waves with no valid row or whose rows all precede the tile.
    const bool live = (q0 < L) && !(p.causal && kv0 > q0 + TQW - 1);
    if (live) {
      const uint16_t* Ks = smem + buf * 2 * TILE;
      const uint16_t* Vt = Ks + TILE;
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
          const int phys = (4 * kc + g) ^ (row & (KCH - 1));
          const V8 kf = __builtin_bit_cast(V8, *reinterpret_cast<const u32x4_t*>(Ks + row * D + phys * 8));
#pragma unroll
          for (int qb = 0; qb < QB; ++qb) s[kb][qb] = M::run(kf, qf[qb][kc], s[kb][qb]);
        }
      }

      V8 pk[NP][QB];
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        if (need_mask) {
          const int q = q0 + 16 * qb + c;
#pragma unroll
          for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int kv = kv0 + 16 * kb + 4 * g + r;
              if (kv >= L || (p.causal && kv > q)) s[kb][qb][r] = -INFINITY;
            }
        }
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
          for (int r = 0; r < 4; ++r) mx = fmaxf(mx, s[kb][qb][r]);
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float m_new = fmaxf(m[qb], mx);
        // A row that has seen only masked keys keeps reference 0 (no exp(-inf+inf)).
        const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
        const float corr = (m[qb] == -INFINITY) ? 0.f : exp2_hw((m[qb] - m_use) * cs);
        const float mc = m_use * cs;
        float rs = 0.f;
#pragma unroll
        for (int pp = 0; pp < NP; ++pp) {
          S e8[8];
#pragma unroll
          for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const float x = s[2 * pp + h][qb][r];
              float e = exp2_hw(__builtin_fmaf(x, cs, -mc));
              if (need_mask && x == -INFINITY) e = 0.f;
              e8[4 * h + r] = (S)e;
              rs += (float)e8[4 * h + r];  // the sum uses the rounded weights
            }
          pk[pp][qb] = (V8){e8[0], e8[1], e8[2], e8[3], e8[4], e8[5], e8[6], e8[7]};
        }
        l[qb] = l[qb] * corr + rs;
        m[qb] = m_new;
#pragma unroll
        for (int db = 0; db < NDB; ++db) o[qb][db] *= corr;
      }

      // GEMM2: o[qb][db][r] += sum_k V^T[16db + 4g + r][k] P^T[k][q]
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const int d = 16 * db + c;
        const int sw = vt_swizzle<VG>(d);
        const uint16_t* vrow = Vt + d * TKV;
#pragma unroll
        for (int pp = 0; pp < NP; ++pp) {
          const u32x2_t a0 = *reinterpret_cast<const u32x2_t*>(vrow + (((8 * pp + g) ^ sw) * 4));
          const u32x2_t a1 = *reinterpret_cast<const u32x2_t*>(vrow + (((8 * pp + 4 + g) ^ sw) * 4));
          const V8 vf = __builtin_bit_cast(V8, (u32x4_t){a0.x, a0.y, a1.x, a1.y});
#pragma unroll
          for (int qb = 0; qb < QB; ++qb) o[qb][db] = M::run(vf, pk[pp][qb], o[qb][db]);
        }
      }
    }
    buf ^= 1;
  }

  // Epilogue.  Each of the four lane groups holds a partial row sum over its
  // key subset (same reference max), so the total is their sum.
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    float lt = l[qb] + __shfl_xor(l[qb], 16);
    lt += __shfl_xor(lt, 32);
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

template <int DT, int D, int TKV, int QB, int NW>
hipError_t launch_fwd(const FwdParams& p, unsigned grid, hipStream_t s) {
  hipLaunchKernelGGL((fwd_kernel<DT, D, TKV, QB, NW>), dim3(grid), dim3(NW * 64), 0, s, p);
  return hipGetLastError();
}

}  // namespace attn
