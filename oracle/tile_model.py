"""Closed-formula tile derivation for fused attention (model of the C++ routine).

Test infrastructure only.  Written from Sections 3, 4 and 6 of the paper, applied in
the paper's CU-centric order (Section 4):

1. LDS -> KV tile.  The staged K/V tiles must fit the LDS share the kernel
   structure gives them: t_KV = floor(share / (kv_tiles * d * elem)), aligned
   down to the atom (Section 4, "LDS constraint" and "Atom alignment").  The
   paper's attention instance gives half of LDS to one streamed t_KV x d tile
   (Table 2: t_KV = 64 at d=128, 128 at d=64 with fp32 elements).
2. VGPR -> Q tile per wave.  Every array live at the synchronisation point
   between the two GEMMs is counted (Section 6.2, Table 2 caption): the Q
   operand, the fp32 score tile(s), the fp32 output accumulator and the
   running (m, delta) pair, plus, for kernel structures that have them, the
   16-bit weights kept in registers for the second GEMM, more statistics per
   row block, operand fragments read ahead, the registers used to stage the
   next K/V tile, and a fixed overhead of addresses and constants.  t_Q is the largest multiple of the atom width whose count
   fits the per-wave budget (Section 4, "VGPR constraint").  The count
   reproduces all four rows of Table 2 with the paper's fp32 instance.
3. CU count -> grid.  If fewer workgroups than CUs result, the derivation
   splits the key range (the merge of Section 5.3 is associative), then
   reduces the Q tile -- waves per workgroup first, then rows per wave --
   until every CU has a workgroup or the tile is one atom (Section 4,
   "Occupancy constraint").
4. Atom alignment of every tile dimension (Section 4).

All quantities are integers; the result is unique for its inputs.
"""
from __future__ import annotations

import dataclasses
import math


@dataclasses.dataclass(frozen=True)
class Hardware:
    lds_bytes: int
    vgpr_per_thread: int
    wavefront_size: int
    num_cus: int
    simds_per_cu: int = 4
    lds_bytes_per_clk: int = 0
    mfma_flops_per_clk_cu: int = 0


@dataclasses.dataclass(frozen=True)
class Atom:
    m: int
    n: int
    k: int
    in_bytes: int
    acc_bytes: int


@dataclasses.dataclass(frozen=True)
class Op:
    B: int
    H: int
    L: int
    d: int
    elem_bytes: int
    causal: bool = False


@dataclasses.dataclass(frozen=True)
class Structure:
    """Fixed properties of one kernel family (chosen once, never searched)."""
    kv_lds_num: int = 1      # share of LDS that holds staged K/V tiles ...
    kv_lds_den: int = 1      # ... as the fraction num/den
    kv_tiles: int = 1        # t_KV x d tiles resident in that share
    stage_tiles: int = 0     # t_KV x d tiles passed through VGPRs per step
    score_tiles: int = 1     # fp32 score tiles live at once (2 when the loop is pipelined)
    p_tiles: int = 0         # 16-bit weight tiles kept in registers for the second GEMM (0: through LDS)
    stat_regs: int = 2       # registers of running statistics per atom-row block (m and delta)
    operand_frags: int = 0   # A-operand fragments of the atom read ahead of their products
    waves_per_wg: int = 1
    waves_per_simd: int = 1  # resident waves per SIMD (divides the register file)
    vgpr_fixed: int = 16     # addresses, loop state, constants
    max_split: int = 1       # key-range splits allowed by the CU rule
    wg_fixed_steps: int = 0  # a workgroup's fixed cost in steps of one key tile (CU rule)


def _cdiv(a, b):
    return -(-a // b)


def vgpr_count(hw, atom, op, st, t_q, t_kv, n_w):
    """Registers per lane live at the GEMM1/GEMM2 synchronisation point."""
    wf = hw.wavefront_size
    q_reg = _cdiv(t_q * op.d * op.elem_bytes, 4 * wf)        # Q operand
    s_reg = st.score_tiles * _cdiv(t_q * t_kv * atom.acc_bytes, 4 * wf)  # score tiles, fp32
    o_reg = _cdiv(t_q * op.d * atom.acc_bytes, 4 * wf)       # output accumulator, fp32
    p_reg = st.p_tiles * _cdiv(t_q * t_kv * atom.in_bytes, 4 * wf)  # 16-bit weights for the second GEMM
    stats = st.stat_regs * _cdiv(t_q, atom.n)                # running statistics per row block
    frags = st.operand_frags * _cdiv(atom.m * atom.k * atom.in_bytes, 4 * wf)  # operands in flight
    stage = _cdiv(st.stage_tiles * t_kv * op.d * op.elem_bytes, 4 * wf * n_w)
    return q_reg + s_reg + o_reg + p_reg + stats + frags + stage + st.vgpr_fixed


def derive(hw, atom, op, st):
    """Return a dict with the tiles, the grid and the feasibility report."""
    rep = dict(feasible=False, binding="", t_kv=0, t_q_wave=0, n_waves=0, tile_q=0,
               n_split=1, tiles_per_split=0, grid=0, vgpr_est=0, vgpr_budget=0, lds_used=0, lds_budget=0,
               wg_per_cu=0.0, low_occupancy=True, lds_bw_ok=True)
    align_kv = math.lcm(atom.n, atom.k)
    align_q = atom.n
    lds_share = hw.lds_bytes * st.kv_lds_num // st.kv_lds_den
    rep["lds_budget"] = lds_share
    budget = hw.vgpr_per_thread // st.waves_per_simd
    rep["vgpr_budget"] = budget

    # 4 (checked first because the others assume it): the contraction over d
    # and the d-rows of the second product must be whole atoms.
    if op.d % atom.k or op.d % atom.m:
        rep["binding"] = "atom"
        return rep

    # 1. LDS -> t_KV
    t_kv = lds_share // (st.kv_tiles * op.d * op.elem_bytes)
    t_kv -= t_kv % align_kv
    if t_kv <= 0:
        rep["binding"] = "LDS"
        return rep
    rep["t_kv"] = t_kv
    rep["lds_used"] = st.kv_tiles * t_kv * op.d * op.elem_bytes

    # 2. VGPR -> t_Q per wave: the largest aligned size whose live set fits.
    n_w = st.waves_per_wg
    t_q = 0
    cand = align_q
    while vgpr_count(hw, atom, op, st, cand, t_kv, n_w) <= budget:
        t_q = cand
        cand += align_q
    if t_q == 0:
        rep["binding"] = "VGPR"
        rep["vgpr_est"] = vgpr_count(hw, atom, op, st, align_q, t_kv, n_w)
        return rep

    # 3. CU count -> grid.
    binding = "VGPR"
    n_kv = _cdiv(op.L, t_kv)
    n_qt = _cdiv(op.L, n_w * t_q)
    heads = op.B * op.H
    n_split = 1
    fills = False
    if heads * n_qt < hw.num_cus and st.max_split > 1:
        # Split count (our addition to the CU rule): the grid runs in rounds of
        # num_cus workgroups and a workgroup's time is its fixed cost plus its
        # key tiles, so take the count with the fewest rounds x (fixed cost +
        # tiles per split), the smallest on ties.  Counts that leave a split
        # empty collapse onto a smaller one.
        s_max = _cdiv(n_kv, _cdiv(n_kv, min(st.max_split, n_kv)))
        best = None
        for s in range(1, s_max + 1):
            per = _cdiv(n_kv, s)
            eff = _cdiv(n_kv, per)
            # rounds x (a workgroup's fixed cost + its key tiles)
            cost = _cdiv(heads * n_qt * eff, hw.num_cus) * (st.wg_fixed_steps + per)
            if best is None or cost < best[0]:
                best = (cost, eff)
        fills = heads * n_qt * s_max >= hw.num_cus
        n_split = best[1] if fills else s_max
        if n_split > 1:
            binding = "CU"
    # Fewer workgroups than CUs that splitting cannot make up: shrink the Q
    # tile, first by halving the waves per workgroup (if the registers that
    # staging needs per lane still fit), else by one atom step of the per-wave
    # tile.
    while not fills and heads * n_qt * n_split < hw.num_cus:
        if n_w > 1 and vgpr_count(hw, atom, op, st, t_q, t_kv, n_w // 2) <= budget:
            n_w //= 2
        elif t_q > align_q:
            t_q -= align_q
        else:
            break
        n_qt = _cdiv(op.L, n_w * t_q)
        binding = "CU"

    tile_q = n_w * t_q
    per = _cdiv(n_kv, n_split)
    grid = heads * n_qt * n_split
    if op.causal and n_split > 1 and tile_q % t_kv == 0:
        # Causal (our addition): query tile qt sees only its first
        # min(n_kv, ceil(min(L, (qt+1) tile_q) / t_kv)) key tiles, so fixed
        # key ranges leave the early tiles' later splits empty and give the
        # last tiles all the work.  Instead each query tile's own key tiles
        # are cut into pieces of per tiles, only non-empty pieces are
        # workgroups, and per is the smallest size -- with at most max_split
        # pieces per tile -- whose workgroups fit one round of CUs; kept when
        # that one round is shorter than the fixed ranges' rounds, each
        # workgroup costing its fixed cost plus its key tiles.
        p_per = _cdiv(n_kv, st.max_split)
        while True:
            pieces = 0
            for qt in range(n_qt):
                seen = min(n_kv, _cdiv(min(op.L, (qt + 1) * tile_q), t_kv))
                pieces += _cdiv(seen, p_per)
            if heads * pieces <= hw.num_cus or p_per >= n_kv:
                break
            p_per += 1
        c0 = st.wg_fixed_steps
        if c0 + p_per < _cdiv(grid, hw.num_cus) * (c0 + per):
            per = p_per
            n_split = _cdiv(n_kv, per)
            grid = heads * pieces
    elif (op.causal and n_split == 1 and tile_q % t_kv == 0 and st.max_split >= 2
          and hw.num_cus <= heads * n_qt < 2 * hw.num_cus):
        # Causal launches that fill between one and two rounds unsplit are
        # bound by their longest query tile (n_kv key tiles against an average
        # of about half that per CU).  Halves of a query tile's own key range
        # (whole multiples of c key tiles), when the halves fit two rounds of
        # CUs and a half is at least four times a workgroup's fixed cost.
        c = tile_q // t_kv
        half = c * _cdiv(_cdiv(n_kv, 2), c)
        halves = heads * sum(_cdiv(min(n_kv, _cdiv(min(op.L, (qt + 1) * tile_q), t_kv)), half)
                             for qt in range(n_qt))
        if 4 * st.wg_fixed_steps <= half < n_kv and halves <= 2 * hw.num_cus:
            per = half
            n_split = _cdiv(n_kv, per)
            grid = halves
            binding = "CU"
    rep.update(feasible=True, binding=binding, t_q_wave=t_q, n_waves=n_w, tile_q=tile_q,
               n_split=n_split, tiles_per_split=per, grid=grid,
               vgpr_est=vgpr_count(hw, atom, op, st, t_q, t_kv, n_w),
               wg_per_cu=grid / hw.num_cus, low_occupancy=grid < hw.num_cus)
    if hw.lds_bytes_per_clk > 0 and hw.mfma_flops_per_clk_cu > 0:
        rep["lds_bw_ok"] = t_q * hw.lds_bytes_per_clk >= hw.mfma_flops_per_clk_cu
    return rep


# ---------------------------------------------------------------- row softmax

@dataclasses.dataclass(frozen=True)
class SoftmaxStructure:
    """Fixed properties of the row-softmax kernel family (Section 5.3 operator)."""
    waves_per_wg: int = 4
    waves_per_simd: int = 2
    vgpr_fixed: int = 48
    load_bytes: int = 16      # bytes one lane moves per tile


def derive_softmax(hw: Hardware, rows: int, n: int, elem_bytes: int, st: SoftmaxStructure = SoftmaxStructure()):
    """The CU-centric rules applied to a bandwidth-bound row softmax.

    Tile: one load of st.load_bytes per lane of a wave.  Registers: the budget
    at st.waves_per_simd holds (budget - fixed) / (load_bytes / 4) tiles per
    lane, kept as a power of two.  CU count: a row is split over 2, 4, ...
    waves of a workgroup (never more waves than the workgroup has, never more
    than one per tile) while the grid has fewer workgroups than CUs; the
    per-wave running statistics are merged with the Section 5.3 operator.
    Returns a dict, or None when not even one tile fits the registers.
    """
    if rows < 1 or n < 1:
        raise ValueError("empty softmax")
    per_lane = st.load_bytes // elem_bytes
    tile = hw.wavefront_size * per_lane
    budget = hw.vgpr_per_thread // st.waves_per_simd
    regs = st.load_bytes // 4
    fit = (budget - st.vgpr_fixed) // regs
    if fit < 1:
        return None
    resident = 1 << int(math.floor(math.log2(fit)))
    W = st.waves_per_wg
    split = 1
    while -(-rows * split // W) < hw.num_cus and split < W and split * tile < n:
        split *= 2
    grid = -(-rows * split // W)
    seg = -(-(-(-n // split)) // 8) * 8
    passes = 1 if seg <= resident * tile else 2
    reread = min(n, split * (seg - resident * tile)) if passes == 2 else 0
    binding = "VGPR" if passes == 2 else ("CU" if grid < hw.num_cus else "none")
    return dict(tile_elems=tile, resident_tiles=resident, split=split, waves_per_wg=W, rows_per_wg=W // split,
                seg=seg, grid=grid, passes=passes, vgpr_est=resident * regs + st.vgpr_fixed, vgpr_budget=budget,
                hbm_bytes=rows * (2 * n + reread) * elem_bytes, binding=binding)
