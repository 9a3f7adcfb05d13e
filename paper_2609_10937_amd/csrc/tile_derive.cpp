// Closed-formula tile derivation for the fused attention kernel.
//
// Sections 3, 4 and 6 of the paper: tiles follow from three hardware constraints in
// a CU-centric order, checked against the atom shape.
//   1. LDS fixes the key/value tile: the staged tiles fill the LDS share the
//      kernel structure gives them (Section 4, LDS constraint).
//   2. The register budget fixes the query rows per wave, counting every array
//      live at the synchronisation point between the two products: the Q
//      operand, the fp32 score tile(s), the fp32 output accumulator, the 16-bit
//      weights kept for the second product (when they stay in registers), the
//      running statistics per row block, the operand fragments read ahead of
//      their products, staging registers, and the kernel family's counted
//      addresses and constants (Section 6.2, Table 2 caption; Section 4, VGPR
//      constraint).
//   3. The CU count bounds the grid from below: split the key range (the
//      merge of Section 5.3 is associative), then shrink the query tile
//      (Section 4, occupancy constraint).
//   4. Atom alignment (Section 4).
// The count in step 2 is affine in t_q up to per-array register rounding, so
// t_q is solved in closed form and then moved by at most a few atom steps to
// absorb that rounding.
#include <string.h>

#include <algorithm>
#include <cmath>
#include <numeric>

#include "gemm_internal.h"
#include "internal.h"

namespace attn {

static int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

static int64_t causal_pieces(int64_t L, int64_t tile_q, int64_t t_kv, int64_t n_qt, int64_t n_kv, int64_t per) {
  int64_t pieces = 0;
  for (int64_t qt = 0; qt < n_qt; ++qt) pieces += cdiv(std::min(n_kv, cdiv(std::min(L, (qt + 1) * tile_q), t_kv)), per);
  return pieces;
}

int64_t vgpr_estimate(const attn_hw_desc_t* hw, const attn_mfma_atom_t* atom, const attn_op_t* op,
                      int64_t t_q, int64_t t_kv, int64_t n_w) {
  const int64_t lane_words = 4 * (int64_t)hw->wavefront_size;  // bytes in one register across a wave
  const int64_t q_operand = cdiv(t_q * op->d * op->elem_bytes, lane_words);
  const int64_t scores = op->score_tiles * cdiv(t_q * t_kv * atom->acc_bytes, lane_words);
  const int64_t out_acc = cdiv(t_q * op->d * atom->acc_bytes, lane_words);
  const int64_t weights = op->p_tiles * cdiv(t_q * t_kv * atom->in_bytes, lane_words);
  const int64_t stats = op->stat_regs * cdiv(t_q, atom->n);
  const int64_t frags = op->operand_frags * cdiv((int64_t)atom->m * atom->k * atom->in_bytes, lane_words);
  const int64_t staging = cdiv((int64_t)op->stage_tiles * t_kv * op->d * op->elem_bytes, lane_words * n_w);
  return q_operand + scores + out_acc + weights + stats + frags + staging + op->vgpr_fixed;
}

template <typename Report>
static void set_binding(Report* r, const char* s) {
  memset(r->binding, 0, sizeof(r->binding));
  strncpy(r->binding, s, sizeof(r->binding) - 1);
}

int derive_tiles(const attn_hw_desc_t* hw, const attn_mfma_atom_t* atom, const attn_op_t* op,
                 attn_tile_report_t* rep) {
  if (!hw || !atom || !op || !rep) return ATTN_E_NULLPTR;
  if (hw->lds_bytes <= 0 || hw->vgpr_per_thread <= 0 || hw->wavefront_size <= 0 ||
      hw->num_cus <= 0 || hw->simds_per_cu <= 0)
    return ATTN_E_ARG;
  if (atom->m <= 0 || atom->n <= 0 || atom->k <= 0 || atom->in_bytes <= 0 || atom->acc_bytes <= 0)
    return ATTN_E_ARG;
  if (op->B <= 0 || op->H <= 0 || op->L <= 0 || op->d <= 0 || op->elem_bytes <= 0) return ATTN_E_ARG;
  if (op->kv_lds_num <= 0 || op->kv_lds_den <= 0 || op->kv_tiles <= 0 || op->stage_tiles < 0 || op->score_tiles < 1 ||
      op->p_tiles < 0 || op->stat_regs < 0 || op->operand_frags < 0 || op->waves_per_wg <= 0 ||
      op->waves_per_simd <= 0 || op->vgpr_fixed < 0 || op->max_split < 1 || op->wg_fixed_steps < 0)
    return ATTN_E_ARG;

  memset(rep, 0, sizeof(*rep));
  rep->n_split = 1;
  rep->low_occupancy = 1;
  rep->lds_bw_ok = 1;
  const int64_t align_kv = std::lcm((int64_t)atom->n, (int64_t)atom->k);
  const int64_t align_q = atom->n;
  const int64_t lds_share = hw->lds_bytes * op->kv_lds_num / op->kv_lds_den;
  const int64_t budget = hw->vgpr_per_thread / op->waves_per_simd;
  rep->lds_budget = lds_share;
  rep->vgpr_budget = (int32_t)budget;

  // 4. The contraction over d (first product) and the d rows of the second
  //    product must both be whole atoms.
  if (op->d % atom->k || op->d % atom->m) {
    set_binding(rep, "atom");
    return ATTN_E_INFEASIBLE;
  }

  // 1. LDS -> t_kv.
  int64_t t_kv = lds_share / ((int64_t)op->kv_tiles * op->d * op->elem_bytes);
  t_kv -= t_kv % align_kv;
  if (t_kv <= 0) {
    set_binding(rep, "LDS");
    return ATTN_E_INFEASIBLE;
  }
  rep->t_kv = (int32_t)t_kv;
  rep->lds_used = (int64_t)op->kv_tiles * t_kv * op->d * op->elem_bytes;

  // 2. Registers -> t_q per wave.  Without rounding the count is
  //    t_q * slope + intercept with
  //    slope = (d*elem + t_kv*acc + d*acc) / (4*wf) + 2/n.
  int64_t n_w = op->waves_per_wg;
  const double lw = 4.0 * hw->wavefront_size;
  const double slope = ((double)op->d * op->elem_bytes + (double)op->score_tiles * t_kv * atom->acc_bytes +
                        (double)op->d * atom->acc_bytes + (double)op->p_tiles * t_kv * atom->in_bytes) / lw +
                       (double)op->stat_regs / atom->n;
  const double intercept = (double)op->stage_tiles * t_kv * op->d * op->elem_bytes / (lw * n_w) +
                           (double)op->operand_frags * atom->m * atom->k * atom->in_bytes / lw + op->vgpr_fixed;
  int64_t t_q = 0;
  if (budget > intercept) {
    t_q = (int64_t)((budget - intercept) / slope);
    t_q -= t_q % align_q;
  }
  // Rounding of each array up to whole registers can only raise the count,
  // by less than one register per term; step to the exact boundary.
  while (t_q > 0 && vgpr_estimate(hw, atom, op, t_q, t_kv, n_w) > budget) t_q -= align_q;
  while (vgpr_estimate(hw, atom, op, t_q + align_q, t_kv, n_w) <= budget) t_q += align_q;
  if (t_q <= 0) {
    set_binding(rep, "VGPR");
    rep->vgpr_est = (int32_t)vgpr_estimate(hw, atom, op, align_q, t_kv, n_w);
    return ATTN_E_INFEASIBLE;
  }

  // 3. CU count -> grid.
  const char* binding = "VGPR";
  const int64_t heads = (int64_t)op->B * op->H;
  const int64_t n_kv = cdiv(op->L, t_kv);
  int64_t n_qt = cdiv(op->L, n_w * t_q);
  int64_t n_split = 1;
  bool fills = false;
  if (heads * n_qt < hw->num_cus && op->max_split > 1) {
    // The grid runs in rounds of num_cus workgroups and a workgroup's time
    // is its fixed cost plus its key tiles: take the split count with the
    // fewest rounds x (wg_fixed_steps + tiles per split), the smallest on
    // ties; a count that would leave a split empty collapses onto the smaller
    // count with the same tiles per split.
    const int64_t s_max = cdiv(n_kv, cdiv(n_kv, std::min((int64_t)op->max_split, n_kv)));
    int64_t best_cost = -1, best = 1;
    for (int64_t s = 1; s <= s_max; ++s) {
      const int64_t per = cdiv(n_kv, s), eff = cdiv(n_kv, per);
      const int64_t cost = cdiv(heads * n_qt * eff, hw->num_cus) * (op->wg_fixed_steps + per);
      if (best_cost < 0 || cost < best_cost) best_cost = cost, best = eff;
    }
    fills = heads * n_qt * s_max >= hw->num_cus;
    n_split = fills ? best : s_max;
    if (n_split > 1) binding = "CU";
  }
  // Fewer workgroups than CUs that splitting cannot make up: shrink the Q tile.
  while (!fills && heads * n_qt * n_split < hw->num_cus) {
    if (n_w > 1 && vgpr_estimate(hw, atom, op, t_q, t_kv, n_w / 2) <= budget)
      n_w /= 2;
    else if (t_q > align_q)
      t_q -= align_q;
    else
      break;
    n_qt = cdiv(op->L, n_w * t_q);
    binding = "CU";
  }

  const int64_t tile_q = n_w * t_q;
  int64_t per = cdiv(n_kv, n_split);
  int64_t grid = heads * n_qt * n_split;
  if (op->causal && n_split > 1 && tile_q % t_kv == 0) {
    // Causal: query tile qt sees only its first min(n_kv, ceil(min(L,
    // (qt+1) tile_q) / t_kv)) key tiles, so fixed key ranges would leave the
    // early tiles' later splits empty and give the last tiles all the work.
    // Each query tile's own key tiles are cut into pieces of p_per tiles,
    // only non-empty pieces are workgroups, and p_per is the smallest size
    // (at most max_split pieces per tile) whose workgroups fit one round of
    // CUs.  The search starts at the bound that the pieces of all query
    // tiles, at least their key tiles over p_per, fit the CUs.
    const int64_t seen = causal_pieces(op->L, tile_q, t_kv, n_qt, n_kv, 1);  // key tiles over all query tiles
    int64_t p_per = std::max(cdiv(n_kv, op->max_split), cdiv(heads * seen, hw->num_cus));
    int64_t pieces = 0;
    for (;; ++p_per) {
      pieces = causal_pieces(op->L, tile_q, t_kv, n_qt, n_kv, p_per);
      if (heads * pieces <= hw->num_cus || p_per >= n_kv) break;
    }
    // Kept when that one round is shorter than the fixed ranges' rounds, each
    // workgroup costing wg_fixed_steps plus its key tiles.
    const int64_t c0 = op->wg_fixed_steps;
    if (c0 + p_per < cdiv(grid, hw->num_cus) * (c0 + per)) {
      per = p_per;
      n_split = cdiv(n_kv, per);
      grid = heads * pieces;
    }
  } else if (op->causal && n_split == 1 && tile_q % t_kv == 0 && op->max_split >= 2 &&
             heads * n_qt >= hw->num_cus && heads * n_qt < 2 * (int64_t)hw->num_cus) {
    // Causal launches that fill between one and two rounds unsplit are bound
    // by their longest query tile (n_kv key tiles against an average of about
    // half that per CU).  Halves of a query tile's own key range (whole
    // multiples of c key tiles), when the halves fit two rounds of CUs and a
    // half is at least four times a workgroup's fixed cost.
    const int64_t c = tile_q / t_kv;
    const int64_t half = c * cdiv(cdiv(n_kv, 2), c);
    const int64_t halves = heads * causal_pieces(op->L, tile_q, t_kv, n_qt, n_kv, half);
    if (half >= 4 * (int64_t)op->wg_fixed_steps && half < n_kv && halves <= 2 * (int64_t)hw->num_cus) {
      per = half;
      n_split = cdiv(n_kv, per);
      grid = halves;
      binding = "CU";
    }
  }
  rep->feasible = 1;
  rep->t_q_wave = (int32_t)t_q;
  rep->n_waves = (int32_t)n_w;
  rep->tile_q = (int32_t)tile_q;
  rep->n_split = (int32_t)n_split;
  rep->tiles_per_split = (int32_t)per;
  rep->grid = grid;
  rep->launch_grid = grid;
  rep->vgpr_est = (int32_t)vgpr_estimate(hw, atom, op, t_q, t_kv, n_w);
  rep->wg_per_cu = (double)grid / hw->num_cus;
  rep->low_occupancy = grid < hw->num_cus;
  if (hw->lds_bytes_per_clk > 0 && hw->mfma_flops_per_clk_cu > 0)
    rep->lds_bw_ok = t_q * hw->lds_bytes_per_clk >= hw->mfma_flops_per_clk_cu;
  set_binding(rep, binding);
  return ATTN_OK;
}

// The row softmax (Section 5.3) on the same CU-centric rules:
//   tile      one 16-byte load per lane: wavefront_size * 16 / elem_bytes elements;
//   registers the budget at the kernel's waves per SIMD, less its fixed
//             registers, holds R = (budget - fixed) / (16 / 4) packed tiles per
//             lane, rounded down to a power of two (the compiled instances);
//   CU count  split a row over 2, 4, ... waves of the workgroup (at most all of
//             them, at most one per tile) while the grid is below the CU count.
int derive_softmax(const attn_hw_desc_t* hw, int64_t rows, int64_t n, int elem_bytes, attn_softmax_report_t* rep) {
  if (!hw || !rep) return ATTN_E_NULLPTR;
  if (hw->vgpr_per_thread <= 0 || hw->wavefront_size <= 0 || hw->num_cus <= 0 || elem_bytes <= 0 ||
      16 % elem_bytes != 0)
    return ATTN_E_ARG;
  if (rows < 1 || n < 1) return ATTN_E_SHAPE;
  memset(rep, 0, sizeof(*rep));
  const int64_t W = kSoftmaxWaves;
  const int64_t per_lane = 16 / elem_bytes;
  const int64_t tile = (int64_t)hw->wavefront_size * per_lane;
  const int64_t budget = hw->vgpr_per_thread / kSoftmaxWavesPerSimd;
  const int64_t regs_per_tile = 16 / 4;
  rep->vgpr_budget = (int32_t)budget;
  if (budget < kSoftmaxVgprFixed + regs_per_tile) {
    rep->feasible = 0;
    set_binding(rep, "VGPR");
    return ATTN_E_INFEASIBLE;
  }
  int64_t resident = 1;
  while (2 * resident <= (budget - kSoftmaxVgprFixed) / regs_per_tile) resident *= 2;
  int64_t split = 1;
  const char* binding = "none";
  while (cdiv(rows * split, W) < hw->num_cus && split < W && split * tile < n) split *= 2;
  const int64_t grid = cdiv(rows * split, W);
  if (grid < hw->num_cus) binding = "CU";
  const int64_t seg = cdiv(cdiv(n, split), 8) * 8;
  const int passes = seg <= resident * tile ? 1 : 2;
  if (passes == 2) binding = "VGPR";
  const int64_t reread = passes == 2 ? std::min<int64_t>(n, split * (seg - resident * tile)) : 0;
  rep->feasible = 1;
  rep->tile_elems = (int32_t)tile;
  rep->resident_tiles = (int32_t)resident;
  rep->split = (int32_t)split;
  rep->waves_per_wg = (int32_t)W;
  rep->rows_per_wg = (int32_t)(W / split);
  rep->seg = seg;
  rep->grid = grid;
  rep->passes = passes;
  rep->vgpr_est = (int32_t)(resident * regs_per_tile + kSoftmaxVgprFixed);
  rep->wg_per_cu = (double)grid / hw->num_cus;
  rep->hbm_bytes = rows * (2 * n + reread) * elem_bytes;
  set_binding(rep, binding);
  return ATTN_OK;
}

// The GEMM of Section 4 (its worked example) on the same rules, for the
// structure of the kernel family that runs the atom (gemm_internal.h):
//   LDS       square tile t = floor(sqrt(LDS / elem)) (the reading of the
//             printed formula that reproduces the section's own numbers),
//             each side aligned down to the atom times the waves along it;
//             t_K = floor(LDS / (stages (t_M + t_N) elem)), aligned down to
//             the atom's k and to whole copy blocks of both tiles per wave;
//   VGPR      per wave (t_M / W_M)(t_N / W_N) fp32 accumulators plus the
//             fixed registers within the budget at the kernel's waves per
//             SIMD: the larger side halves until they fit;
//   CU count  while the grid is below the CU count the larger side halves,
//             down to one atom per wave.
const GemmStructure& gemm_structure(const attn_mfma_atom_t* atom) {
  return atom->in_bytes >= 4 ? kGemm32 : kGemm16;
}

static int64_t gemm_vgpr(const GemmStructure& st, const attn_mfma_atom_t* atom, int64_t wave_words, int64_t tm,
                         int64_t tn) {
  const int64_t wm = tm / st.waves_m, wn = tn / st.waves_n;
  const int64_t per_atom = cdiv((int64_t)atom->m * atom->n * atom->acc_bytes, wave_words);
  return (wm / atom->m) * (wn / atom->n) * per_atom + st.vgpr_fixed;
}

static int64_t gemm_t_k(const GemmStructure& st, const attn_hw_desc_t* hw, const attn_mfma_atom_t* atom,
                        int64_t tm, int64_t tn) {
  const int64_t elem = atom->in_bytes;
  const int64_t unit = (int64_t)st.copy_block * st.waves_m * st.waves_n;
  int64_t step = atom->k;
  for (const int64_t side : {tm, tn}) {
    const int64_t need = unit / std::gcd(unit, side * elem);
    step = std::lcm(step, need);
  }
  return hw->lds_bytes / (st.stages * (tm + tn) * elem) / step * step;
}

int derive_gemm(const attn_hw_desc_t* hw, const attn_mfma_atom_t* atom, int64_t M, int64_t N, int64_t K,
                attn_gemm_report_t* rep) {
  if (!hw || !atom || !rep) return ATTN_E_NULLPTR;
  if (hw->lds_bytes <= 0 || hw->vgpr_per_thread <= 0 || hw->wavefront_size <= 0 || hw->num_cus <= 0)
    return ATTN_E_ARG;
  if (atom->m <= 0 || atom->n <= 0 || atom->k <= 0 || atom->in_bytes <= 0 || atom->acc_bytes <= 0)
    return ATTN_E_ARG;
  if (M < 1 || N < 1 || K < 1) return ATTN_E_SHAPE;
  const GemmStructure& st = gemm_structure(atom);
  memset(rep, 0, sizeof(*rep));
  rep->stages = st.stages;
  rep->waves_per_wg = st.waves_m * st.waves_n;
  rep->lds_budget = hw->lds_bytes;
  const int64_t budget = hw->vgpr_per_thread / st.waves_per_simd;
  rep->vgpr_budget = (int32_t)budget;
  const int64_t am = (int64_t)atom->m * st.waves_m, an = (int64_t)atom->n * st.waves_n;
  const int64_t wave_words = 4 * (int64_t)hw->wavefront_size;
  const int64_t q = hw->lds_bytes / atom->in_bytes;
  int64_t t = (int64_t)std::sqrt((double)q);  // floor(sqrt(q)), corrected to be exact
  while (t * t > q) --t;
  while ((t + 1) * (t + 1) <= q) ++t;
  int64_t tm = t / am * am, tn = t / an * an;
  const char* binding = "LDS";
  if (tm < am || tn < an) {
    set_binding(rep, "LDS");
    return ATTN_E_INFEASIBLE;
  }
  while (gemm_vgpr(st, atom, wave_words, tm, tn) > budget) {
    if (tm >= tn && tm > am) {
      tm = std::max(am, tm / 2 / am * am);
    } else if (tn > an) {
      tn = std::max(an, tn / 2 / an * an);
    } else {
      set_binding(rep, "VGPR");
      return ATTN_E_INFEASIBLE;
    }
    binding = "VGPR";
  }
  while (cdiv(M, tm) * cdiv(N, tn) < hw->num_cus && (tm > am || tn > an)) {
    if ((tm >= tn && tm > am) || tn <= an) tm = std::max(am, tm / 2 / am * am);
    else tn = std::max(an, tn / 2 / an * an);
    binding = "CU";
  }
  const int64_t tk = gemm_t_k(st, hw, atom, tm, tn);
  if (tk < atom->k) {
    set_binding(rep, "LDS");
    return ATTN_E_INFEASIBLE;
  }
  const int64_t grid = cdiv(M, tm) * cdiv(N, tn);
  rep->feasible = 1;
  rep->t_m = (int32_t)tm;
  rep->t_n = (int32_t)tn;
  rep->t_k = (int32_t)tk;
  rep->warp_m = (int32_t)(tm / st.waves_m);
  rep->warp_n = (int32_t)(tn / st.waves_n);
  rep->grid = grid;
  rep->vgpr_est = (int32_t)gemm_vgpr(st, atom, wave_words, tm, tn);
  rep->lds_used = (int64_t)st.stages * (tm + tn) * tk * atom->in_bytes;
  rep->wg_per_cu = (double)grid / hw->num_cus;
  set_binding(rep, binding);
  return ATTN_OK;
}

}  // namespace attn
