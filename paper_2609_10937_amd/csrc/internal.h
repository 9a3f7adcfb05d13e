// Internal declarations shared by the C-ABI layer and the HIP translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "attn.h"

namespace attn {

// Arguments of the fused kernel.  Tensor pointers are [B*H, L, d] contiguous.
struct FwdParams {
  const void* q;
  const void* k;
  const void* v;
  void* o;
  void* part_o;     // [n_split, BH, L, d] per-split outputs normalised by their sums, input type (n_split > 1)
  float* part_ml;   // [n_split, BH, L, 2] per-split reference point (base 2) and sum
  int BH;
  int L;
  int n_qt;             // query tiles per head
  int n_split;          // key-range splits
  int tiles_per_split;  // key tiles per split
  int causal;
  float c;              // scale * log2(e): exp(scale*(x - m)) = exp2(c*(x - m))
  int tile_q;           // query rows per workgroup of the fused kernel
  int t_kv;             // key rows per key tile
  // Causal with split key ranges: workgroups per head, one per non-empty
  // piece of tiles_per_split key tiles of a query tile's own key range
  // (the piece order of fwd_kernel); 0 otherwise.
  int pieces;
};

// The fused kernel's workgroup order (the XCD a workgroup runs on is its
// index mod 8), decided alike on the host and the device:
//   kOrderPieces  causal with split key ranges: the pieces of each query
//                 tile's own key range, heaviest query tiles first;
//   kOrderUnits   units (head, split) spread over the XCDs, xg at a time;
//   kOrderTiles   with a split key range, all splits of query tile t
//                 (counted head-major) on XCD t % 8;
//   kOrderPlain   units fastest within a query rank.
// xg is the smallest power of two with xg * n_qt >= 64.
enum FwdOrder { kOrderPieces, kOrderUnits, kOrderTiles, kOrderPlain };
__host__ __device__ inline FwdOrder fwd_order(const FwdParams& p, int* xg_out) {
  int xg = 1;
  while (xg * p.n_qt < 64) xg *= 2;
  *xg_out = xg;
  if (p.pieces > 0) return kOrderPieces;
  if ((p.BH * p.n_split) % (8 * xg) == 0) return kOrderUnits;
  if (p.n_split > 1 && (p.BH * p.n_qt) % 8 == 0) return kOrderTiles;
  return kOrderPlain;
}

using FwdLaunch = hipError_t (*)(const FwdParams&, unsigned grid, hipStream_t);

// One compiled instantiation of the fused kernel.
struct FwdInstance {
  int dtype;
  int d;
  int t_kv;
  int q_blocks;   // query rows per wave / 16
  int n_waves;
  FwdLaunch launch;
  // The same kernel as a persistent launch (one workgroup per CU running
  // several query tiles back to back), or null when not compiled.
  FwdLaunch launch_persist;
};

const FwdInstance* fwd_instances(int* count);

// Argument checks, tile derivation on the current device's descriptor,
// instance lookup and kernel parameters shared by the forward entry points
// (no device memory is touched; the workspace pointers stay unset).
struct Prepared {
  attn_tile_report_t rep;
  const FwdInstance* inst;
  FwdParams p;
  size_t ws_bytes;  // split workspace the plan needs (0 without a split)
};
int prepare(const void* Q, const void* K, const void* V, void* O, int B, int H, int L, int d, float scale, int causal,
            int dtype, Prepared* out);
// Enqueue the fused kernel of a prepared call (persistent when the plan's
// launch grid differs from its grid).
hipError_t launch_fused(const Prepared& pr, hipStream_t s);
// Point the split partials of `p` into a workspace of at least Prepared::ws_bytes.
void bind_workspace(FwdParams& p, void* ws, int d);

hipError_t launch_combine(const FwdParams& p, int d, int dtype, hipStream_t s);

// The unfused baseline's three steps: the row-softmax derivation for the
// (B*H*L) x L score matrix and the GEMM derivations (and compiled instances)
// of its two products.
struct GemmInstance;
struct UnfusedPlan {
  attn_softmax_report_t sm;
  attn_gemm_report_t qk, pv;
  const GemmInstance* qk_inst;
  const GemmInstance* pv_inst;
};
hipError_t launch_unfused(const UnfusedPlan& u, const void* q, const void* k, const void* v, void* o, void* ws,
                          int BH, int L, int d, float scale, int causal, int dtype, hipStream_t s);

hipError_t launch_mfma_probe(int atom, const void* a, const void* b, float* c, hipStream_t s);

// Row softmax (Section 5.3).  x, y: [rows, n] contiguous; a wave owns `seg`
// elements of a row and `split` waves share a row.
struct SoftmaxParams {
  const void* x;
  void* y;
  int64_t rows;
  int64_t n;
  int64_t seg;
  int split;
  int causal;   // mask column j > (row mod n)
};
// Fixed structure of the softmax kernel: waves per workgroup, waves per SIMD
// (the register budget), registers outside the resident tiles, and the
// resident tiles of the compiled kernel.
constexpr int kSoftmaxWaves = 4, kSoftmaxWavesPerSimd = 2, kSoftmaxVgprFixed = 48, kSoftmaxTiles = 32;
hipError_t launch_softmax(const SoftmaxParams& p, int dtype, bool aligned, unsigned grid, hipStream_t s);
int derive_softmax(const attn_hw_desc_t* hw, int64_t rows, int64_t n, int elem_bytes, attn_softmax_report_t* rep);

int derive_tiles(const attn_hw_desc_t* hw, const attn_mfma_atom_t* atom, const attn_op_t* op,
                 attn_tile_report_t* rep);
int64_t vgpr_estimate(const attn_hw_desc_t* hw, const attn_mfma_atom_t* atom, const attn_op_t* op,
                      int64_t t_q, int64_t t_kv, int64_t n_w);

}  // namespace attn
