"""Pins of the tile-derivation and traffic models against the paper's printed values.

Table 2 (all four rows), the gpu_a / gpu_b portability example of Section 3
and the HBM traffic figures of Section 6.2 are stored in tests/golden with
their citations.  The remaining checks are properties any correct derivation
has: budgets never exceeded, tiles aligned to the atom, maximality (one more
atom step would break the budget) and monotonicity in the budgets.
"""
import json
import math
import os

import pytest
from hypothesis import given, settings, strategies as stg

from oracle import tile_model as T
from oracle import traffic

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _paper():
    with open(os.path.join(GOLD, "paper_tiles.json")) as f:
        return json.load(f)


def paper_instance(g, which="gpu_a"):
    hw = T.Hardware(**g[which])
    atom = T.Atom(**g["atom"])
    # the paper's attention kernel: half of LDS holds one streamed K/V tile,
    # one wave per workgroup, one wave per SIMD, fixed overhead 16 VGPRs
    st = T.Structure(kv_lds_num=1, kv_lds_den=2, kv_tiles=1, stage_tiles=0,
                     waves_per_wg=1, waves_per_simd=1, vgpr_fixed=16, max_split=1)
    return hw, atom, st


@pytest.mark.parametrize("row", range(4))
def test_table2_rows(row):
    g = _paper()
    r = g["table2"][row]
    hw, atom, st = paper_instance(g)
    op = T.Op(1, 1, 16384, r["d"], g["elem_bytes"])
    rep = T.derive(hw, atom, op, st)
    assert rep["feasible"]
    assert rep["t_kv"] == r["t_kv"]
    v = T.vgpr_count(hw, atom, op, st, r["t_q"], r["t_kv"], 1)
    assert v == r["vgprs"]
    assert (v <= hw.vgpr_per_thread) == r["feasible"]
    if r["feasible"]:
        assert rep["t_q_wave"] == r["t_q"] and rep["vgpr_est"] == r["vgprs"]


@pytest.mark.parametrize("which", ["gpu_a", "gpu_b"])
def test_portability_same_tiles(which):
    g = _paper()
    hw, atom, st = paper_instance(g, which)
    p = g["portability"]
    rep = T.derive(hw, atom, T.Op(1, 1, p["L"], p["d"], g["elem_bytes"]), st)
    assert (rep["tile_q"], rep["t_kv"]) == (p["tile_q"], p["tile_kv"])
    assert rep["grid"] == p["L"] // p["tile_q"]


def test_fragment_counts():
    g = _paper()
    a = T.Atom(**g["atom"])
    wf = g["gpu_a"]["wavefront_size"]
    assert (a.m * a.k // wf, a.k * a.n // wf, a.m * a.n // wf) == (
        g["fragments"]["a"], g["fragments"]["b"], g["fragments"]["c"])


def test_infeasible_reports_binding():
    g = _paper()
    hw, atom, st = paper_instance(g)
    tiny_lds = T.Hardware(lds_bytes=1024, vgpr_per_thread=256, wavefront_size=64, num_cus=120)
    assert T.derive(tiny_lds, atom, T.Op(1, 1, 1024, 128, 4), st)["binding"] == "LDS"
    tiny_vgpr = T.Hardware(lds_bytes=65536, vgpr_per_thread=40, wavefront_size=64, num_cus=120)
    rep = T.derive(tiny_vgpr, atom, T.Op(1, 1, 1024, 128, 4), st)
    assert not rep["feasible"] and rep["binding"] == "VGPR"
    rep = T.derive(hw, T.Atom(16, 16, 32, 2, 4), T.Op(1, 1, 1024, 48, 2), st)
    assert not rep["feasible"] and rep["binding"] == "atom"


def test_cu_rule_splits_then_shrinks():
    hw = T.Hardware(lds_bytes=160 * 1024, vgpr_per_thread=512, wavefront_size=64, num_cus=256)
    atom = T.Atom(16, 16, 32, 2, 4)
    st = T.Structure(kv_lds_num=1, kv_lds_den=1, kv_tiles=8, stage_tiles=2, waves_per_wg=8,
                     waves_per_simd=2, vgpr_fixed=32, max_split=8)
    rep = T.derive(hw, atom, T.Op(1, 1, 16384, 128, 2), st)
    # 43 query tiles of 384 rows, 256 key tiles, at most 8 splits: 5 splits make
    # one round of 215 workgroups x 52 tiles, 8 splits two rounds x 32 tiles
    assert rep["feasible"] and (rep["tile_q"], rep["n_split"], rep["grid"]) == (384, 5, 215)
    assert rep["binding"] == "CU"
    st1 = T.Structure(**{**st.__dict__, "max_split": 1})
    rep1 = T.derive(hw, atom, T.Op(1, 1, 16384, 128, 2), st1)
    assert rep1["n_split"] == 1 and rep1["grid"] >= 256 and rep1["binding"] == "CU"
    assert rep1["tile_q"] <= rep["tile_q"]
    big = T.derive(hw, atom, T.Op(4, 32, 16384, 128, 2, True), st)
    assert big["n_split"] == 1 and big["n_waves"] == 8 and big["binding"] == "VGPR"


hw_s = stg.builds(T.Hardware,
                  lds_bytes=stg.integers(1, 320).map(lambda x: x * 1024),
                  vgpr_per_thread=stg.sampled_from([128, 256, 512]),
                  wavefront_size=stg.sampled_from([32, 64]),
                  num_cus=stg.integers(1, 512),
                  simds_per_cu=stg.sampled_from([2, 4]))
atom_s = stg.sampled_from([T.Atom(16, 16, 4, 4, 4), T.Atom(16, 16, 32, 2, 4),
                           T.Atom(32, 32, 16, 2, 4), T.Atom(16, 16, 16, 2, 4)])
op_s = stg.builds(T.Op, B=stg.integers(1, 8), H=stg.integers(1, 64),
                  L=stg.integers(1, 70000), d=stg.sampled_from([32, 64, 96, 128, 256]),
                  elem_bytes=stg.sampled_from([2, 4]), causal=stg.booleans())
st_s = stg.builds(T.Structure, kv_lds_num=stg.just(1), kv_lds_den=stg.sampled_from([1, 2]),
                  kv_tiles=stg.sampled_from([1, 2, 4, 8]), stage_tiles=stg.sampled_from([0, 2]),
                  score_tiles=stg.sampled_from([1, 2]), p_tiles=stg.sampled_from([0, 1]),
                  stat_regs=stg.integers(0, 8), operand_frags=stg.integers(0, 6),
                  waves_per_wg=stg.sampled_from([1, 2, 4, 8]), waves_per_simd=stg.sampled_from([1, 2]),
                  vgpr_fixed=stg.integers(0, 64), max_split=stg.sampled_from([1, 4, 8, 16]),
                  wg_fixed_steps=stg.sampled_from([0, 8]))


@settings(max_examples=400, deadline=None)
@given(hw_s, atom_s, op_s, st_s)
def test_budgets_alignment_maximality(hw, atom, op, st):
    rep = T.derive(hw, atom, op, st)
    if not rep["feasible"]:
        assert rep["binding"] in ("LDS", "VGPR", "atom")
        return
    align_kv = math.lcm(atom.n, atom.k)
    assert rep["t_kv"] % align_kv == 0 and rep["t_q_wave"] % atom.n == 0
    assert op.d % atom.k == 0 and op.d % atom.m == 0
    assert rep["lds_used"] <= rep["lds_budget"] <= hw.lds_bytes
    assert (rep["t_kv"] + align_kv) * st.kv_tiles * op.d * op.elem_bytes > rep["lds_budget"]
    assert rep["vgpr_est"] <= rep["vgpr_budget"]
    if rep["binding"] != "CU":
        assert T.vgpr_count(hw, atom, op, st, rep["t_q_wave"] + atom.n, rep["t_kv"],
                            st.waves_per_wg) > rep["vgpr_budget"]
    assert rep["tile_q"] == rep["n_waves"] * rep["t_q_wave"]
    n_qt = -(-op.L // rep["tile_q"])
    n_kv = -(-op.L // rep["t_kv"])
    per = rep["tiles_per_split"]
    assert 1 <= rep["n_split"] <= max(1, st.max_split)
    assert rep["n_split"] == -(-n_kv // per)
    assert rep["low_occupancy"] == (rep["grid"] < hw.num_cus)
    if op.causal and rep["grid"] < op.B * op.H * n_qt * rep["n_split"]:
        # causal pieces: the grid counts the non-empty pieces of every query
        # tile's own key range, fits one round, and one key tile less per
        # piece would not
        c = rep["tile_q"] // rep["t_kv"]
        def pieces(pp):
            return sum(-(-min(n_kv, -(-min(op.L, (qt + 1) * rep["tile_q"]) // rep["t_kv"])) // pp)
                       for qt in range(n_qt))
        heads = op.B * op.H
        assert rep["grid"] == heads * pieces(per)
        if heads * n_qt < hw.num_cus:
            # one round, and one key tile less per piece would not fit it
            assert rep["grid"] <= hw.num_cus
            if per > 1 and -(-n_kv // (per - 1)) <= st.max_split:
                assert heads * pieces(per - 1) > hw.num_cus
        else:
            # filled between one and two rounds unsplit: halves of at least 32
            # key tiles that fit two rounds
            assert heads * n_qt < 2 * hw.num_cus and rep["n_split"] == 2
            assert per == c * -(-(-(-n_kv // 2)) // c) and 4 * st.wg_fixed_steps <= per < n_kv
            assert rep["grid"] <= 2 * hw.num_cus
    else:
        assert rep["grid"] == op.B * op.H * n_qt * rep["n_split"]
        assert per == -(-n_kv // rep["n_split"])


@settings(max_examples=200, deadline=None)
@given(hw_s, atom_s, op_s, st_s, stg.integers(1, 4))
def test_monotone_in_budgets(hw, atom, op, st, f):
    base = T.derive(hw, atom, op, st)
    more_lds = T.derive(T.Hardware(**{**hw.__dict__, "lds_bytes": hw.lds_bytes * f}), atom, op, st)
    if base["feasible"]:
        assert more_lds["t_kv"] >= base["t_kv"]
    more_v = T.derive(T.Hardware(**{**hw.__dict__, "vgpr_per_thread": hw.vgpr_per_thread * f}),
                      atom, op, st)
    if base["feasible"]:
        assert more_v["feasible"] and more_v["t_q_wave"] >= base["t_q_wave"]
        assert more_v["t_kv"] == base["t_kv"]


# ---------------------------------------------------------------- traffic

def test_traffic_figures():
    with open(os.path.join(GOLD, "paper_traffic.json")) as f:
        g = json.load(f)
    e, d = g["elem_bytes"], g["d"]
    r = g["L16384"]
    assert round(traffic.fused_bytes(1, 1, 16384, d, e) / 1e6) == r["fused_MB"]
    assert round(traffic.unfused_bytes(1, 1, 16384, d, e) / 1e6) == r["unfused_MB"]
    assert round(traffic.score_matrix_bytes(1, 1, 16384, e) / 1e6) == r["S_MB"]
    assert traffic.traffic_ratio(16384, d) == r["ratio"]
    assert round(traffic.unfused_bytes(1, 1, 16384, d, e) / traffic.fused_bytes(1, 1, 16384, d, e)) \
        == r["ratio"]
    r2 = g["L32768"]
    assert round(traffic.unfused_bytes(1, 1, 32768, d, e) / 1e9) == r2["unfused_GB"]
    assert round(traffic.score_matrix_bytes(1, 1, 32768, e) / 1e9) == r2["S_GB"]
    assert traffic.savings_equation(16384, d) == g["savings_equation"]["value"]


def test_flop_counts():
    assert traffic.attention_flops(1, 1, 16384, 128, False) == 4 * 16384 ** 2 * 128
    assert traffic.attention_flops(1, 1, 3, 2, True) == 4 * 6 * 2
