// C ABI of the fused-attention library: argument checks, hardware
// descriptors, tile derivation and dispatch to compiled kernel instances.
#include <math.h>
#include <string.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <tuple>
#include <vector>

#include "gemm_internal.h"
#include "internal.h"

namespace attn {
const GemmInstance* gemm_instances_qk_bf16(int* n);
const GemmInstance* gemm_instances_qk_f16(int* n);
const GemmInstance* gemm_instances_pv_bf16(int* n);
const GemmInstance* gemm_instances_pv_f16(int* n);
const GemmInstance* gemm_instances_qk(int dtype, int* n) {
  return dtype == ATTN_BF16 ? gemm_instances_qk_bf16(n) : gemm_instances_qk_f16(n);
}
const GemmInstance* gemm_instances_pv(int dtype, int* n) {
  return dtype == ATTN_BF16 ? gemm_instances_pv_bf16(n) : gemm_instances_pv_f16(n);
}
const FwdInstance* fwd_instances_bf16_d64(int* n);
const FwdInstance* fwd_instances_bf16_d128(int* n);
const FwdInstance* fwd_instances_f16_d64(int* n);
const FwdInstance* fwd_instances_f16_d128(int* n);
const FwdInstance* fwd_instances_bf16_d256(int* n);
const FwdInstance* fwd_instances_f16_d256(int* n);
const FwdInstance* fwd_instances_bf16_d96(int* n);
const FwdInstance* fwd_instances_f16_d96(int* n);
}  // namespace attn

using namespace attn;

namespace {

// Fixed structure of the fused kernel family in fwd_kernel.hpp: all of LDS
// holds a ring of 5 stages of (K tile, V tile) filled by direct HBM->LDS
// copies (no registers stage them), 8 waves per workgroup at 2 waves per
// SIMD.  What a wave holds at the point where the second product of tile
// j - 1 runs beside the first product of tile j, besides Q, S and O:
//  - the 16-bit weights of tile j - 1 (kPTiles = 1: P stays in registers);
//  - per 16-row block, a 4-register row-sum accumulator (the sums come from
//    a matrix product), the reference point, the check limit and the
//    pending correction factor (kStatRegs = 7);
//  - the operand fragment being consumed and the 4 read ahead of it
//    (kOperandFrags = 5, 4 registers each at the 16x16x32 atom);
//  - kVgprFixed = 14 counted registers: the lane bases of the K and V
//    fragment reads (2), the two stage bases of the phase (2), the lane's
//    byte offsets within a tile for its two K and two V copies (4; the
//    copies read through per-tile buffer descriptors, so the offsets do not
//    change from tile to tile), the all-ones A operand of the row-sum
//    product (4), and the lane's query row and key group for masking (2).
constexpr int kKvLdsNum = 1, kKvLdsDen = 1, kKvTiles = 10, kStageTiles = 0, kScoreTiles = 1;
constexpr int kPTiles = 1, kStatRegs = 7, kOperandFrags = 5;
constexpr int kWavesPerWg = 8, kWavesPerSimd = 2, kVgprFixed = 14, kMaxSplit = 16;
// A workgroup's fixed cost (loading Q and filling the ring, the epilogue) in
// steps of one key tile: one launch measures about 12 us plus 1.594 us per
// step (d = 128), so about 8 steps.
constexpr int kWgFixedSteps = 8;

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

int check_shape(int B, int H, int L, int d, int dtype) {
  if (B <= 0 || H <= 0 || L <= 0 || L > ATTN_MAX_L) return ATTN_E_SHAPE;
  if (d != 64 && d != 96 && d != 128 && d != 256) return ATTN_E_UNSUPPORTED_D;
  if ((int64_t)L * d * 2 > (int64_t(1) << 32)) return ATTN_E_SHAPE;  // byte offsets within a head are 32-bit
  if (dtype != ATTN_BF16 && dtype != ATTN_F16) return ATTN_E_DTYPE;
  const long double elems = (long double)B * H * L * d;
  if (elems >= 4.6e18L) return ATTN_E_SHAPE;
  if ((int64_t)B * H > (int64_t)1 << 30) return ATTN_E_SHAPE;
  return ATTN_OK;
}

int check_tensors(const void* Q, const void* K, const void* V, const void* O) {
  if (!Q || !K || !V || !O) return ATTN_E_NULLPTR;
  if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(O)) return ATTN_E_ALIGN;
  return ATTN_OK;
}

int check_scale(float scale) {
  if (!isfinite(scale) || scale < 0.f) return ATTN_E_SCALE;
  return ATTN_OK;
}

void fill_name(attn_hw_desc_t* d, const char* n) {
  memset(d->name, 0, sizeof(d->name));
  strncpy(d->name, n, sizeof(d->name) - 1);
}

void gfx950_desc(attn_hw_desc_t* d) {
  memset(d, 0, sizeof(*d));
  d->lds_bytes = 160 * 1024;
  d->vgpr_per_thread = 512;       // 256 arch + 256 accumulation registers at one wave per SIMD
  d->wavefront_size = 64;
  d->num_cus = 256;
  d->simds_per_cu = 4;
  d->lds_bytes_per_clk = 128;
  d->mfma_flops_per_clk_cu = 4096;  // dense bf16/fp16
  d->hbm_tbps = 8.0;
  d->peak_tflops = 2516.6;
  d->clock_ghz = 2.4;
  fill_name(d, "gfx950");
}

attn_mfma_atom_t atom_for(int dtype) {
  (void)dtype;  // bf16 and f16 share the 16x16x32 shape and fp32 accumulation
  attn_mfma_atom_t a = {16, 16, 32, 2, 4};
  return a;
}

// attn_fwd's split workspace: one buffer per (device, stream), so calls
// on different streams never share one, and calls on one stream use it in
// stream order.  A buffer that is outgrown is retired, never freed: work
// enqueued earlier (or a graph captured earlier) may still reference it, and
// freeing would also synchronise the device.
struct StreamWorkspace {
  void* ptr = nullptr;
  size_t bytes = 0;
};

// A forward plan: the derived tiles of one shape and the compiled instance
// that runs them.  The derivation is a pure function of the device's
// descriptor and the shape, so each device keeps the plans of the shapes it
// has run (at most kMaxPlans, then the table starts over).
struct FwdPlan {
  attn_tile_report_t rep;
  const FwdInstance* inst;
};
using PlanKey = std::tuple<int, int, int, int, int, int>;  // B, H, L, d, causal, dtype
constexpr size_t kMaxPlans = 1024;

struct DeviceState {
  bool have_desc = false;
  attn_hw_desc_t desc{};
  std::map<PlanKey, FwdPlan> plans;
  std::map<hipStream_t, StreamWorkspace> ws;
  std::vector<void*> retired;
};

std::mutex g_mu;
std::map<int, DeviceState> g_dev;

// The unfused baseline's product instance (qk: S = scale Q K^T, else O = P V)
// for derived tiles, or null.
const GemmInstance* find_gemm(int dtype, bool qk, const attn_gemm_report_t& r) {
  int n = 0;
  const GemmInstance* t = qk ? gemm_instances_qk(dtype, &n) : gemm_instances_pv(dtype, &n);
  for (int i = 0; i < n; ++i)
    if (t[i].t_m == r.t_m && t[i].t_n == r.t_n && t[i].t_k == r.t_k) return &t[i];
  return nullptr;
}

const FwdInstance* find_instance(int dtype, int d, int t_kv, int q_blocks, int n_waves) {
  using Fn = const FwdInstance* (*)(int*);
  Fn fns[] = {fwd_instances_bf16_d64, fwd_instances_bf16_d96, fwd_instances_bf16_d128, fwd_instances_bf16_d256,
              fwd_instances_f16_d64,  fwd_instances_f16_d96,  fwd_instances_f16_d128,  fwd_instances_f16_d256};
  for (Fn f : fns) {
    int n = 0;
    const FwdInstance* t = f(&n);
    for (int i = 0; i < n; ++i)
      if (t[i].dtype == dtype && t[i].d == d && t[i].t_kv == t_kv && t[i].q_blocks == q_blocks &&
          t[i].n_waves == n_waves)
        return &t[i];
  }
  return nullptr;
}

int query_desc(int device, attn_hw_desc_t* out) {
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, device) != hipSuccess) return ATTN_E_HIP;
  if (strncmp(prop.gcnArchName, "gfx950", 6) != 0) return ATTN_E_DEVICE;
  gfx950_desc(out);
  out->num_cus = prop.multiProcessorCount;
  out->lds_bytes = (int64_t)prop.sharedMemPerBlock;
  out->wavefront_size = prop.warpSize;
  if (prop.clockRate > 0) out->clock_ghz = prop.clockRate / 1e6;
  out->peak_tflops = (double)out->mfma_flops_per_clk_cu * out->num_cus * out->clock_ghz / 1e3;
  return ATTN_OK;
}

int device_desc(int device, attn_hw_desc_t* out) {
  std::lock_guard<std::mutex> lk(g_mu);
  DeviceState& st = g_dev[device];
  if (!st.have_desc) {
    const int rc = query_desc(device, &st.desc);
    if (rc != ATTN_OK) return rc;
    st.have_desc = true;
  }
  *out = st.desc;
  return ATTN_OK;
}

int make_op(int B, int H, int L, int d, int causal, int dtype, attn_op_t* op) {
  memset(op, 0, sizeof(*op));
  op->B = B;
  op->H = H;
  op->L = L;
  op->d = d;
  op->elem_bytes = 2;
  op->causal = causal != 0;
  op->kv_lds_num = kKvLdsNum;
  op->kv_lds_den = kKvLdsDen;
  op->kv_tiles = kKvTiles;
  op->stage_tiles = kStageTiles;
  op->score_tiles = kScoreTiles;
  op->p_tiles = kPTiles;
  op->stat_regs = kStatRegs;
  op->operand_frags = kOperandFrags;
  op->waves_per_wg = kWavesPerWg;
  op->waves_per_simd = kWavesPerSimd;
  op->vgpr_fixed = kVgprFixed;
  op->max_split = kMaxSplit;
  op->wg_fixed_steps = kWgFixedSteps;
  (void)dtype;
  return ATTN_OK;
}

// Persistent launches (the fused kernel's PERSIST variant: one workgroup per
// CU running a fixed list of query tiles back to back) for plans without
// split key ranges that have more query tiles than CUs (num_cus a multiple
// of 8, the XCD count), every query tile at least kPersistMinTiles key tiles
// long (the unit switch keeps the copies in flight within the current and
// the next tile), at most kPersistMaxMeanTiles on average, and the byte
// offsets of a head's rows, up to the end of its last query tile, below
// 4 GiB (its buffer descriptors).  The mean bound is measured: a query tile
// of a workgroup's own costs about as much as 6 to 9 key tiles, which the
// persistent schedule hides, while its loop runs a few percent slower per
// key tile; at 16 key tiles per query tile (L = 1024, d = 128) it gains 8%,
// at 32 nothing, and at the configurations with 34 and 130 it loses 3 to 7%.
constexpr int kPersistMinTiles = 4, kPersistMaxMeanTiles = 24;

bool persistent(const attn_tile_report_t& rep, const FwdInstance* inst, int L, int d, int causal, int num_cus) {
  if (!inst->launch_persist || rep.n_split != 1 || num_cus <= 0 || num_cus % 8 != 0) return false;
  if (rep.grid <= num_cus) return false;
  if ((int64_t)(L + rep.tile_q) * d * 2 >= ((int64_t)1 << 32)) return false;
  const int64_t n_kv = (L + rep.t_kv - 1) / rep.t_kv, n_qt = (L + rep.tile_q - 1) / rep.tile_q;
  int64_t shortest = n_kv, total = n_kv * n_qt;
  if (causal) {
    total = 0;
    for (int64_t qt = 0; qt < n_qt; ++qt)
      total += std::min(n_kv, (std::min<int64_t>(L, (qt + 1) * rep.tile_q) + rep.t_kv - 1) / rep.t_kv);
    shortest = std::min(n_kv, (std::min<int64_t>(L, rep.tile_q) + rep.t_kv - 1) / rep.t_kv);
  }
  return shortest >= kPersistMinTiles && total <= (int64_t)kPersistMaxMeanTiles * n_qt;
}

int plan(const attn_hw_desc_t* hw, int B, int H, int L, int d, int causal, int dtype, attn_tile_report_t* rep,
         const FwdInstance** inst) {
  attn_op_t op;
  make_op(B, H, L, d, causal, dtype, &op);
  const attn_mfma_atom_t atom = atom_for(dtype);
  const int rc = derive_tiles(hw, &atom, &op, rep);
  if (rc != ATTN_OK) return rc;
  if (rep->t_q_wave % 16) return ATTN_E_NO_INSTANCE;
  const FwdInstance* f = find_instance(dtype, d, rep->t_kv, rep->t_q_wave / 16, rep->n_waves);
  if (!f) return ATTN_E_NO_INSTANCE;
  if (inst) *inst = f;
  if (rep->grid > 0x7fffffffLL) return ATTN_E_SHAPE;
  if (persistent(*rep, f, L, d, causal, hw->num_cus)) rep->launch_grid = hw->num_cus;
  return ATTN_OK;
}

// The plan of a shape on the given device: derived on the device's first
// call with that shape, then read from its table.
int device_plan(int device, int B, int H, int L, int d, int causal, int dtype, attn_tile_report_t* rep,
                const FwdInstance** inst) {
  std::lock_guard<std::mutex> lk(g_mu);
  DeviceState& st = g_dev[device];
  if (!st.have_desc) {
    const int rc = query_desc(device, &st.desc);
    if (rc != ATTN_OK) return rc;
    st.have_desc = true;
  }
  const PlanKey key{B, H, L, d, causal != 0, dtype};
  const auto it = st.plans.find(key);
  if (it != st.plans.end()) {
    *rep = it->second.rep;
    *inst = it->second.inst;
    return ATTN_OK;
  }
  const int rc = plan(&st.desc, B, H, L, d, causal, dtype, rep, inst);
  if (rc != ATTN_OK) return rc;
  if (st.plans.size() >= kMaxPlans) st.plans.clear();
  st.plans.emplace(key, FwdPlan{*rep, *inst});
  return ATTN_OK;
}

}  // namespace

namespace attn {

int prepare(const void* Q, const void* K, const void* V, void* O, int B, int H, int L, int d, float scale, int causal,
            int dtype, Prepared* out) {
  int rc = check_tensors(Q, K, V, O);
  if (rc != ATTN_OK) return rc;
  rc = check_shape(B, H, L, d, dtype);
  if (rc != ATTN_OK) return rc;
  rc = check_scale(scale);
  if (rc != ATTN_OK) return rc;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return ATTN_E_HIP;
  rc = device_plan(dev, B, H, L, d, causal, dtype, &out->rep, &out->inst);
  if (rc != ATTN_OK) return rc;
  FwdParams& p = out->p;
  p = FwdParams{};
  p.q = Q;
  p.k = K;
  p.v = V;
  p.o = O;
  p.BH = B * H;
  p.L = L;
  p.n_qt = (L + out->rep.tile_q - 1) / out->rep.tile_q;
  p.n_split = out->rep.n_split;
  p.tiles_per_split = out->rep.tiles_per_split;
  p.t_kv = out->rep.t_kv;
  // Causal pieces: the derivation then reports fewer workgroups than query
  // tiles times splits (only non-empty pieces).
  const int64_t n_qt_splits = (int64_t)p.BH * p.n_qt * p.n_split;
  p.pieces = causal && p.n_split > 1 && out->rep.grid < n_qt_splits ? (int)(out->rep.grid / p.BH) : 0;
  p.causal = causal != 0;
  p.c = scale * 1.4426950408889634f;
  p.tile_q = out->rep.tile_q;
  const size_t rows = (size_t)p.n_split * p.BH * L;
  out->ws_bytes = p.n_split > 1 ? rows * (size_t)d * 2 + rows * 8 : 0;
  return ATTN_OK;
}

hipError_t launch_fused(const Prepared& pr, hipStream_t s) {
  const bool persist = pr.rep.launch_grid != pr.rep.grid;
  return (persist ? pr.inst->launch_persist : pr.inst->launch)(pr.p, (unsigned)pr.rep.launch_grid, s);
}

void bind_workspace(FwdParams& p, void* ws, int d) {
  const size_t rows = (size_t)p.n_split * p.BH * p.L;
  p.part_o = ws;
  p.part_ml = reinterpret_cast<float*>(static_cast<char*>(ws) + rows * (size_t)d * 2);
}

}  // namespace attn

extern "C" {

const char* attn_strerror(int status) {
  switch (status) {
    case ATTN_OK: return "ok";
    case ATTN_E_NULLPTR: return "null pointer argument";
    case ATTN_E_SHAPE: return "B, H or L out of range";
    case ATTN_E_UNSUPPORTED_D: return "head dimension must be 64, 96, 128 or 256";
    case ATTN_E_DTYPE: return "dtype must be ATTN_BF16 or ATTN_F16";
    case ATTN_E_ALIGN: return "tensor base address not 16-byte aligned";
    case ATTN_E_INFEASIBLE: return "tile derivation infeasible";
    case ATTN_E_NO_INSTANCE: return "no compiled kernel for the derived tiles";
    case ATTN_E_HIP: return "HIP runtime error";
    case ATTN_E_WORKSPACE: return "workspace missing or too small";
    case ATTN_E_SCALE: return "scale must be finite and >= 0";
    case ATTN_E_ARG: return "invalid argument";
    case ATTN_E_DEVICE: return "current device is not gfx950";
    case ATTN_E_SCRATCH: return "split workspace larger than the static scratch of attn_fwd_noalloc";
    default: return "unknown status";
  }
}

int attn_hw_desc_preset(const char* name, attn_hw_desc_t* out) {
  if (!name || !out) return ATTN_E_NULLPTR;
  if (strcmp(name, "gfx950") == 0) {
    gfx950_desc(out);
    return ATTN_OK;
  }
  if (strcmp(name, "gfx942") == 0) {
    // MI300X public figures: 304 CUs, 64 KiB LDS, 512 registers per lane at one
    // wave per SIMD, dense bf16 1307.4 TFLOP/s at 2.1 GHz (2048 per clock per
    // CU, on the 16x16x16 atom), 5.3 TB/s.
    memset(out, 0, sizeof(*out));
    out->lds_bytes = 64 * 1024;
    out->vgpr_per_thread = 512;
    out->wavefront_size = 64;
    out->num_cus = 304;
    out->simds_per_cu = 4;
    out->lds_bytes_per_clk = 128;
    out->mfma_flops_per_clk_cu = 2048;
    out->hbm_tbps = 5.3;
    out->peak_tflops = 1307.4;
    out->clock_ghz = 2.1;
    fill_name(out, "gfx942");
    return ATTN_OK;
  }
  const bool a = strcmp(name, "paper_gpu_a") == 0, b = strcmp(name, "paper_gpu_b") == 0;
  if (!a && !b) return ATTN_E_ARG;
  // Section 3, the two CDNA descriptors of the listing.
  memset(out, 0, sizeof(*out));
  out->lds_bytes = 64 * 1024;
  out->vgpr_per_thread = 256;
  out->wavefront_size = 64;
  out->num_cus = a ? 120 : 304;
  out->simds_per_cu = 4;
  out->hbm_tbps = a ? 1.2 : 5.3;
  out->peak_tflops = a ? 11.5 : 383.0;
  fill_name(out, name);
  return ATTN_OK;
}

int attn_hw_desc_query(int device, attn_hw_desc_t* out) {
  if (!out) return ATTN_E_NULLPTR;
  if (device < 0) return ATTN_E_ARG;
  return device_desc(device, out);
}

int attn_atom_preset(const char* name, attn_mfma_atom_t* out) {
  if (!name || !out) return ATTN_E_NULLPTR;
  if (strcmp(name, "f32_16x16x4") == 0) {
    *out = {16, 16, 4, 4, 4};
    return ATTN_OK;
  }
  if (strcmp(name, "bf16_16x16x32") == 0 || strcmp(name, "f16_16x16x32") == 0) {
    *out = {16, 16, 32, 2, 4};
    return ATTN_OK;
  }
  if (strcmp(name, "bf16_16x16x16") == 0 || strcmp(name, "f16_16x16x16") == 0) {  // gfx942's 16-bit atom
    *out = {16, 16, 16, 2, 4};
    return ATTN_OK;
  }
  return ATTN_E_ARG;
}

int attn_fwd_op(int B, int H, int L, int d, int causal, int dtype, attn_op_t* out) {
  if (!out) return ATTN_E_NULLPTR;
  const int rc = check_shape(B, H, L, d, dtype);
  if (rc != ATTN_OK) return rc;
  return make_op(B, H, L, d, causal, dtype, out);
}

int attn_vgpr_estimate(const attn_hw_desc_t* hw, const attn_mfma_atom_t* atom, const attn_op_t* op, int t_q_wave,
                       int t_kv, int n_waves, int32_t* out) {
  if (!hw || !atom || !op || !out) return ATTN_E_NULLPTR;
  if (t_q_wave <= 0 || t_kv <= 0 || n_waves <= 0 || hw->wavefront_size <= 0 || atom->n <= 0) return ATTN_E_ARG;
  *out = (int32_t)vgpr_estimate(hw, atom, op, t_q_wave, t_kv, n_waves);
  return ATTN_OK;
}

int attn_tile_derive(const attn_hw_desc_t* hw, const attn_mfma_atom_t* atom, const attn_op_t* op,
                     attn_tile_report_t* report) {
  return derive_tiles(hw, atom, op, report);
}

int attn_fwd_plan(const attn_hw_desc_t* hw, int B, int H, int L, int d, int causal, int dtype,
                  attn_tile_report_t* report) {
  if (!report) return ATTN_E_NULLPTR;
  int rc = check_shape(B, H, L, d, dtype);
  if (rc != ATTN_OK) return rc;
  attn_hw_desc_t desc;
  if (!hw) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return ATTN_E_HIP;
    rc = device_desc(dev, &desc);
    if (rc != ATTN_OK) return rc;
    hw = &desc;
  }
  return plan(hw, B, H, L, d, causal, dtype, report, nullptr);
}

int attn_fwd(const void* Q, const void* K, const void* V, void* O, int B, int H, int L, int d, float scale,
             int causal, int dtype, void* stream) {
  Prepared pr;
  int rc = prepare(Q, K, V, O, B, H, L, d, scale, causal, dtype, &pr);
  if (rc != ATTN_OK) return rc;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (pr.ws_bytes == 0) return launch_fused(pr, s) == hipSuccess ? ATTN_OK : ATTN_E_HIP;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return ATTN_E_HIP;
  // The lock covers binding the stream's buffer and enqueueing both kernels,
  // so two host threads on one stream cannot interleave their launches.
  std::lock_guard<std::mutex> lk(g_mu);
  DeviceState& st = g_dev[dev];
  StreamWorkspace& w = st.ws[s];
  if (w.bytes < pr.ws_bytes) {
    // Allocating is not stream-ordered: never under capture.
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(s, &cap) != hipSuccess) return ATTN_E_HIP;
    if (cap != hipStreamCaptureStatusNone) return ATTN_E_WORKSPACE;
    const size_t grow = w.bytes > pr.ws_bytes / 2 ? 2 * w.bytes : pr.ws_bytes;
    void* nb = nullptr;
    if (hipMalloc(&nb, grow) != hipSuccess) return ATTN_E_HIP;
    if (w.ptr) st.retired.push_back(w.ptr);
    w.ptr = nb;
    w.bytes = grow;
  }
  bind_workspace(pr.p, w.ptr, d);
  if (launch_fused(pr, s) != hipSuccess) return ATTN_E_HIP;
  return launch_combine(pr.p, d, dtype, s) == hipSuccess ? ATTN_OK : ATTN_E_HIP;
}

int attn_fwd_workspace_bytes(int B, int H, int L, int d, int causal, int dtype, size_t* out) {
  if (!out) return ATTN_E_NULLPTR;
  *out = 0;
  const void* fake = reinterpret_cast<const void*>((uintptr_t)1 << 20);  // passes the pointer checks
  Prepared pr;
  const int rc = prepare(fake, fake, fake, const_cast<void*>(fake), B, H, L, d, 1.0f, causal, dtype, &pr);
  if (rc != ATTN_OK) return rc;
  *out = pr.ws_bytes;
  return ATTN_OK;
}

int attn_fwd_partial(const void* Q, const void* K, const void* V, void* O, int B, int H, int L, int d, float scale,
                     int causal, int dtype, void* workspace, size_t workspace_bytes, void* stream) {
  Prepared pr;
  int rc = prepare(Q, K, V, O, B, H, L, d, scale, causal, dtype, &pr);
  if (rc != ATTN_OK) return rc;
  if (pr.ws_bytes > 0) {
    if (!workspace || workspace_bytes < pr.ws_bytes) return ATTN_E_WORKSPACE;
    if (!aligned16(workspace)) return ATTN_E_ALIGN;
    bind_workspace(pr.p, workspace, d);
  }
  return launch_fused(pr, static_cast<hipStream_t>(stream)) == hipSuccess ? ATTN_OK
                                                                                                   : ATTN_E_HIP;
}

int attn_fwd_merge(const void* workspace, size_t workspace_bytes, void* O, int B, int H, int L, int d, float scale,
                   int causal, int dtype, void* stream) {
  const void* fake = reinterpret_cast<const void*>((uintptr_t)1 << 20);
  Prepared pr;
  int rc = prepare(fake, fake, fake, O, B, H, L, d, scale, causal, dtype, &pr);
  if (rc != ATTN_OK) return rc;
  if (pr.ws_bytes == 0) return ATTN_OK;  // the partial call already wrote O
  if (!workspace || workspace_bytes < pr.ws_bytes) return ATTN_E_WORKSPACE;
  if (!aligned16(workspace)) return ATTN_E_ALIGN;
  bind_workspace(pr.p, const_cast<void*>(workspace), d);
  return launch_combine(pr.p, d, dtype, static_cast<hipStream_t>(stream)) == hipSuccess ? ATTN_OK : ATTN_E_HIP;
}

size_t attn_unfused_workspace_bytes(int B, int H, int L, int dtype) {
  if (B <= 0 || H <= 0 || L <= 0 || (dtype != ATTN_BF16 && dtype != ATTN_F16)) return 0;
  return (size_t)B * H * (size_t)L * (size_t)L * 2;
}

int attn_fwd_unfused(const void* Q, const void* K, const void* V, void* O, int B, int H, int L, int d, float scale,
                     int causal, int dtype, void* workspace, size_t workspace_bytes, void* stream) {
  int rc = check_tensors(Q, K, V, O);
  if (rc != ATTN_OK) return rc;
  rc = check_shape(B, H, L, d, dtype);
  if (rc != ATTN_OK) return rc;
  if (L % 8 || L > (1 << 22)) return ATTN_E_SHAPE;  // 16-byte rows of the L x L matrix; K of the P V product
  rc = check_scale(scale);
  if (rc != ATTN_OK) return rc;
  if (!workspace) return ATTN_E_WORKSPACE;
  if (!aligned16(workspace)) return ATTN_E_ALIGN;
  if (workspace_bytes < attn_unfused_workspace_bytes(B, H, L, dtype)) return ATTN_E_WORKSPACE;
  if ((int64_t)B * H > 65535 || (int64_t)B * H * L > 0x7fffffffLL) return ATTN_E_SHAPE;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return ATTN_E_HIP;
  attn_hw_desc_t desc;
  rc = device_desc(dev, &desc);
  if (rc != ATTN_OK) return rc;
  UnfusedPlan u;
  rc = derive_softmax(&desc, (int64_t)B * H * L, L, 2, &u.sm);
  if (rc != ATTN_OK) return rc;
  if (u.sm.resident_tiles != kSoftmaxTiles || u.sm.waves_per_wg != kSoftmaxWaves) return ATTN_E_NO_INSTANCE;
  const attn_mfma_atom_t atom = {16, 16, 32, 2, 4};
  rc = derive_gemm(&desc, &atom, L, L, d, &u.qk);
  if (rc != ATTN_OK) return rc;
  rc = derive_gemm(&desc, &atom, L, d, L, &u.pv);
  if (rc != ATTN_OK) return rc;
  u.qk_inst = find_gemm(dtype, true, u.qk);
  u.pv_inst = find_gemm(dtype, false, u.pv);
  if (!u.qk_inst || !u.pv_inst) return ATTN_E_NO_INSTANCE;
  const hipError_t e =
      launch_unfused(u, Q, K, V, O, workspace, B * H, L, d, scale, causal != 0, dtype, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? ATTN_OK : ATTN_E_HIP;
}

int attn_softmax_derive(const attn_hw_desc_t* hw, int64_t rows, int64_t n, int elem_bytes,
                        attn_softmax_report_t* out) {
  return derive_softmax(hw, rows, n, elem_bytes, out);
}

int attn_softmax(const void* X, void* Y, int64_t rows, int64_t n, int causal, int dtype, void* stream) {
  if (!X || !Y) return ATTN_E_NULLPTR;
  if (dtype != ATTN_BF16 && dtype != ATTN_F16) return ATTN_E_DTYPE;
  if (rows < 1 || n < 1 || n > (int64_t(1) << 31)) return ATTN_E_SHAPE;
  if (((uintptr_t)X & 1u) || ((uintptr_t)Y & 1u)) return ATTN_E_ALIGN;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return ATTN_E_HIP;
  attn_hw_desc_t desc;
  int rc = device_desc(dev, &desc);
  if (rc != ATTN_OK) return rc;
  attn_softmax_report_t rep;
  rc = derive_softmax(&desc, rows, n, 2, &rep);
  if (rc != ATTN_OK) return rc;
  if (rep.resident_tiles != kSoftmaxTiles || rep.waves_per_wg != kSoftmaxWaves) return ATTN_E_NO_INSTANCE;
  if (rep.grid > 0x7fffffffLL) return ATTN_E_SHAPE;
  SoftmaxParams p{X, Y, rows, n, rep.seg, rep.split, causal != 0};
  const bool aligned = n % 8 == 0 && aligned16(X) && aligned16(Y);
  return launch_softmax(p, dtype, aligned, (unsigned)rep.grid, static_cast<hipStream_t>(stream)) == hipSuccess
             ? ATTN_OK
             : ATTN_E_HIP;
}

int attn_gemm_derive(const attn_hw_desc_t* hw, const attn_mfma_atom_t* atom, int64_t M, int64_t N, int64_t K,
                     attn_gemm_report_t* out) {
  return derive_gemm(hw, atom, M, N, K, out);
}

int attn_gemm(const void* A, const void* B, float* C, int64_t M, int64_t N, int64_t K, int dtype, void* stream) {
  if (!A || !B || !C) return ATTN_E_NULLPTR;
  if (dtype != ATTN_BF16 && dtype != ATTN_F16 && dtype != ATTN_F32) return ATTN_E_DTYPE;
  // Whole 16-byte chunks along N and K; 32-bit lane offsets within a
  // workgroup's panels (t_M K e and t_K N e bytes below 2^32).
  const int64_t per_chunk = dtype == ATTN_F32 ? 4 : 8;
  const int64_t max_n = dtype == ATTN_F32 ? (int64_t(1) << 22) : (int64_t(1) << 24);
  if (M < 1 || M > 0x7fffffffLL || N < per_chunk || N > max_n || N % per_chunk != 0 || K < per_chunk ||
      K > (int64_t(1) << 22) || K % per_chunk != 0)
    return ATTN_E_SHAPE;
  if (!aligned16(A) || !aligned16(B) || !aligned16(C)) return ATTN_E_ALIGN;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return ATTN_E_HIP;
  attn_hw_desc_t desc;
  int rc = device_desc(dev, &desc);
  if (rc != ATTN_OK) return rc;
  const attn_mfma_atom_t atom = dtype == ATTN_F32 ? attn_mfma_atom_t{16, 16, 4, 4, 4} : attn_mfma_atom_t{16, 16, 32, 2, 4};
  attn_gemm_report_t rep;
  rc = derive_gemm(&desc, &atom, M, N, K, &rep);
  if (rc != ATTN_OK) return rc;
  const int64_t n_tm = (M + rep.t_m - 1) / rep.t_m, n_tn = (N + rep.t_n - 1) / rep.t_n;
  if (n_tm * n_tn > 0x7fffffffLL) return ATTN_E_SHAPE;
  const GemmInstance* inst = nullptr;
  int n = 0;
  const GemmInstance* table = dtype == ATTN_BF16 ? gemm_instances_bf16(&n)
                              : dtype == ATTN_F16 ? gemm_instances_f16(&n)
                                                  : gemm_instances_f32(&n);
  for (int i = 0; i < n; ++i)
    if (table[i].t_m == rep.t_m && table[i].t_n == rep.t_n && table[i].t_k == rep.t_k) inst = &table[i];
  if (!inst) return ATTN_E_NO_INSTANCE;
  const GemmParams p{A, B, C, (int)M, (int)N, (int)K, (int)n_tm, (int)n_tn};
  return inst->launch(p, static_cast<hipStream_t>(stream)) == hipSuccess ? ATTN_OK : ATTN_E_HIP;
}

int attn_mfma_probe(int atom, const void* A, const void* Bm, float* C, void* stream) {
  if (!A || !Bm || !C) return ATTN_E_NULLPTR;
  if (atom != ATTN_BF16 && atom != ATTN_F16) return ATTN_E_ARG;
  if (!aligned16(A)) return ATTN_E_ALIGN;
  return launch_mfma_probe(atom, A, Bm, C, static_cast<hipStream_t>(stream)) == hipSuccess ? ATTN_OK : ATTN_E_HIP;
}

}  // extern "C"
