"""Host-side tests of libattn.so: exports, argument checks, tile derivation.

No GPU is touched: every argument check runs before the first HIP call, and
the derivation is host integer arithmetic.  The C++ derivation is compared
bit for bit with the oracle's model of the paper's rules (oracle/tile_model),
which is itself pinned to Table 2.
"""
import ctypes
import itertools
import json
import os
import re

import pytest
from hypothesis import given, settings, strategies as stg

from oracle import tile_model as T
from paper_2609_10937_amd import capi, inputs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_every_declared_function_is_exported(lib):
    with open(os.path.join(ROOT, "include", "attn.h")) as f:
        header = f.read()
    declared = set(re.findall(r"^(?:int|size_t|const char\*)\s+(attn_\w+)\(", header, re.M))
    assert declared == set(capi.EXPORTS)
    for name in declared:
        assert hasattr(lib, name)


def test_strerror_names_every_status(lib):
    for code in capi.STATUS:
        assert capi.attn_strerror(code) and capi.attn_strerror(code) != "unknown status"


def test_presets():
    g = capi.attn_hw_desc_preset("gfx950")
    assert (g.lds_bytes, g.vgpr_per_thread, g.wavefront_size, g.num_cus) == (163840, 512, 64, 256)
    a = capi.attn_hw_desc_preset("paper_gpu_a")
    b = capi.attn_hw_desc_preset("paper_gpu_b")
    assert (a.num_cus, b.num_cus, a.lds_bytes, a.vgpr_per_thread) == (120, 304, 65536, 256)
    with pytest.raises(capi.AttnError) as e:
        capi.attn_hw_desc_preset("gfx908")
    assert e.value.status == capi.CODE["ATTN_E_ARG"]
    at = capi.attn_atom_preset("f32_16x16x4")
    assert (at.m, at.n, at.k, at.in_bytes, at.acc_bytes) == (16, 16, 4, 4, 4)


def _to_c(hw, atom, op, st):
    h = capi.HwDesc(lds_bytes=hw.lds_bytes, vgpr_per_thread=hw.vgpr_per_thread,
                    wavefront_size=hw.wavefront_size, num_cus=hw.num_cus,
                    simds_per_cu=hw.simds_per_cu, lds_bytes_per_clk=hw.lds_bytes_per_clk,
                    mfma_flops_per_clk_cu=hw.mfma_flops_per_clk_cu)
    a = capi.Atom(m=atom.m, n=atom.n, k=atom.k, in_bytes=atom.in_bytes, acc_bytes=atom.acc_bytes)
    o = capi.Op(B=op.B, H=op.H, L=op.L, d=op.d, elem_bytes=op.elem_bytes, causal=int(op.causal),
                kv_lds_num=st.kv_lds_num, kv_lds_den=st.kv_lds_den, kv_tiles=st.kv_tiles,
                stage_tiles=st.stage_tiles, score_tiles=st.score_tiles, p_tiles=st.p_tiles,
                stat_regs=st.stat_regs, operand_frags=st.operand_frags, waves_per_wg=st.waves_per_wg,
                waves_per_simd=st.waves_per_simd, vgpr_fixed=st.vgpr_fixed, max_split=st.max_split,
                wg_fixed_steps=st.wg_fixed_steps)
    return h, a, o


def _same(rc, rep, ref):
    assert (rc == 0) == ref["feasible"]
    assert rep.binding.decode() == ref["binding"]
    if not ref["feasible"]:
        return
    for k in ("t_kv", "n_waves", "tile_q", "n_split", "tiles_per_split", "grid", "vgpr_est", "vgpr_budget",
              "lds_used", "lds_budget"):
        assert getattr(rep, k) == ref[k], k
    assert rep.t_q_wave == ref["t_q_wave"]
    assert bool(rep.low_occupancy) == ref["low_occupancy"]
    assert bool(rep.lds_bw_ok) == ref["lds_bw_ok"]
    assert rep.wg_per_cu == pytest.approx(ref["wg_per_cu"], rel=1e-12)


def test_table2_through_the_library():
    with open(os.path.join(ROOT, "tests", "golden", "paper_tiles.json")) as f:
        g = json.load(f)
    hw = capi.attn_hw_desc_preset("paper_gpu_a")
    atom = capi.attn_atom_preset("f32_16x16x4")
    for r in g["table2"]:
        op = capi.Op(B=1, H=1, L=16384, d=r["d"], elem_bytes=4, causal=0, kv_lds_num=1, kv_lds_den=2,
                     kv_tiles=1, stage_tiles=0, score_tiles=1, p_tiles=0, stat_regs=2, operand_frags=0,
                     waves_per_wg=1, waves_per_simd=1, vgpr_fixed=16, max_split=1)
        rc, rep = capi.attn_tile_derive(hw, atom, op)
        assert rc == 0 and rep.t_kv == r["t_kv"]
        assert capi.attn_vgpr_estimate(hw, atom, op, r["t_q"], r["t_kv"], 1) == r["vgprs"]
        if r["feasible"]:
            assert rep.t_q_wave == r["t_q"] and rep.vgpr_est == r["vgprs"]
    for name in ("paper_gpu_a", "paper_gpu_b"):
        hw = capi.attn_hw_desc_preset(name)
        rc, rep = capi.attn_tile_derive(hw, atom, op)
        assert (rep.tile_q, rep.t_kv) == (g["portability"]["tile_q"], g["portability"]["tile_kv"])


hw_s = stg.builds(T.Hardware,
                  lds_bytes=stg.integers(1, 320).map(lambda x: x * 1024),
                  vgpr_per_thread=stg.sampled_from([128, 256, 512]),
                  wavefront_size=stg.sampled_from([32, 64]),
                  num_cus=stg.integers(1, 512),
                  simds_per_cu=stg.sampled_from([2, 4]),
                  lds_bytes_per_clk=stg.sampled_from([0, 128, 256]),
                  mfma_flops_per_clk_cu=stg.sampled_from([0, 2048, 4096]))
atom_s = stg.sampled_from([T.Atom(16, 16, 4, 4, 4), T.Atom(16, 16, 32, 2, 4),
                           T.Atom(32, 32, 16, 2, 4), T.Atom(16, 16, 16, 2, 4)])
op_s = stg.builds(T.Op, B=stg.integers(1, 8), H=stg.integers(1, 64),
                  L=stg.integers(1, 1 << 20), d=stg.sampled_from([16, 32, 48, 64, 96, 128, 256]),
                  elem_bytes=stg.sampled_from([2, 4]), causal=stg.booleans())
st_s = stg.builds(T.Structure, kv_lds_num=stg.just(1), kv_lds_den=stg.sampled_from([1, 2, 4]),
                  kv_tiles=stg.sampled_from([1, 2, 4, 8]), stage_tiles=stg.sampled_from([0, 1, 2]),
                  score_tiles=stg.sampled_from([1, 2]), p_tiles=stg.sampled_from([0, 1, 2]),
                  stat_regs=stg.integers(0, 8), operand_frags=stg.integers(0, 8),
                  waves_per_wg=stg.sampled_from([1, 2, 4, 8, 16]),
                  waves_per_simd=stg.sampled_from([1, 2, 4]),
                  vgpr_fixed=stg.integers(0, 128), max_split=stg.sampled_from([1, 2, 8, 16]),
                  wg_fixed_steps=stg.sampled_from([0, 1, 8, 20]))


@settings(max_examples=1500, deadline=None)
@given(hw_s, atom_s, op_s, st_s)
def test_library_derivation_matches_oracle_model(hw, atom, op, st):
    ref = T.derive(hw, atom, op, st)
    rc, rep = capi.attn_tile_derive(*_to_c(hw, atom, op, st))
    _same(rc, rep, ref)


def test_fused_structure_plans_every_shape():
    """Every shape the API accepts maps to a compiled instance on the gfx950 descriptor."""
    hw = capi.attn_hw_desc_preset("gfx950")
    shapes = [(w.B, w.H, w.L, w.d, w.causal) for w in inputs.WORKLOADS.values()]
    for d in (64, 96, 128, 256):
        for L in (1, 2, 15, 16, 17, 31, 33, 63, 64, 65, 100, 127, 129, 159, 161, 1000, 1023, 4097,
                  16384, 65536, 1 << 20, capi.ATTN_MAX_L):
            for B, H in ((1, 1), (1, 3), (2, 8), (4, 32), (64, 64)):
                for causal in (0, 1):
                    shapes.append((B, H, L, d, causal))
    seen = set()
    for B, H, L, d, causal in shapes:
        for dt in (capi.ATTN_BF16, capi.ATTN_F16):
            if B * H * L > (1 << 31) // 2 or L * d * 2 > (1 << 32):
                continue
            r = capi.attn_fwd_plan(B, H, L, d, causal, dt, hw=hw)
            assert r.feasible and r.grid >= 1
            assert r.vgpr_est <= r.vgpr_budget and r.lds_used <= r.lds_budget
            seen.add((d, r.t_kv, r.t_q_wave, r.n_waves))
    assert (128, 64, 32, 8) in seen and (256, 32, 16, 8) in seen and (96, 64, 48, 8) in seen


def test_head_bytes_fit_32_bit_offsets():
    """A head's Q, K or V must stay within 4 GiB (L d 2 <= 2^32): L = 2^23 is the
    largest sequence at d = 256, while d = 128 reaches ATTN_MAX_L = 2^24."""
    hw = capi.attn_hw_desc_preset("gfx950")
    assert capi.attn_fwd_plan(1, 1, 1 << 23, 256, 0, capi.ATTN_BF16, hw=hw).feasible
    assert capi.attn_fwd_plan(1, 1, capi.ATTN_MAX_L, 128, 0, capi.ATTN_BF16, hw=hw).feasible
    with pytest.raises(capi.AttnError) as e:
        capi.attn_fwd_plan(1, 1, (1 << 23) + 1, 256, 0, capi.ATTN_BF16, hw=hw)
    assert e.value.status == capi.CODE["ATTN_E_SHAPE"]


def test_headline_plans():
    hw = capi.attn_hw_desc_preset("gfx950")
    r = capi.attn_fwd_plan(1, 1, 16384, 128, 0, capi.ATTN_BF16, hw=hw)
    assert (r.t_kv, r.t_q_wave, r.n_waves, r.tile_q, r.lds_used) == (64, 32, 8, 256, 160 * 1024)
    assert r.n_split == 4 and r.grid == 256 and r.binding == b"CU"
    r = capi.attn_fwd_plan(4, 32, 16384, 128, 1, capi.ATTN_BF16, hw=hw)
    assert (r.n_split, r.grid, r.binding) == (1, 8192, b"VGPR")


@pytest.mark.parametrize("shape,split,grid", [
    # Cost: rounds x (8 steps of fixed cost + key tiles per split).
    # 64 query tiles, 256 key tiles: 4 splits fill one round exactly,
    # 8 + 64 = 72 (8 splits: two rounds of 8 + 32 = 80)
    ((1, 1, 16384, 128), 4, 256),
    # d = 96: 43 query tiles of 384 rows, 256 key tiles.  5 splits: one round
    # of 215 workgroups, 8 + 52 = 60; 11 splits: two rounds of 8 + 24 = 64;
    # 8 splits: two rounds of 8 + 32 = 80
    ((1, 1, 16384, 96), 5, 215),
    # L = 10000: 40 query tiles, 157 key tiles; 6 splits of 27 tiles make one
    # round of 240, 8 + 27 = 35 (8 splits: 320 workgroups, two rounds of
    # 8 + 20 = 56)
    ((1, 1, 10000, 128), 6, 240),
    # splitting cannot fill the CUs: the most splits (16), then halve the waves
    ((1, 4, 1000, 96), 16, 384),
])
def test_split_count_by_rounds(shape, split, grid):
    """The split count minimises rounds of CU-count workgroups times (a
    workgroup's fixed cost of 8 steps + key tiles per split), worked by hand."""
    hw = capi.attn_hw_desc_preset("gfx950")
    r = capi.attn_fwd_plan(*shape, 0, capi.ATTN_BF16, hw=hw)
    assert (r.n_split, r.grid, r.binding) == (split, grid, b"CU")


@pytest.mark.parametrize("L,per,n_split,grid", [
    # 64 query tiles of 256 rows, 256 key tiles; query tile x = qt + 1 sees
    # 4x key tiles (8320 in all), so a piece holds at least
    # max(256 / 16, 8320 / 256) -> 33 tiles.  Pieces of 36: ceil(4x / 36) is
    # 1..7 for nine x each and 8 for x = 64: 9 (1 + ... + 7) + 8 = 260 > 256;
    # of 37: 1, 2, 3 for nine x each, 4 for ten, 5, 6, 7 for nine each:
    # 9 + 18 + 27 + 40 + 45 + 54 + 63 = 256
    (16384, 37, 7, 256),
    # 32 query tiles, 128 key tiles, 2112 in all: at least 9 per piece; of
    # 9: ceil(4x / 9) for x = 1..32 adds up to 249
    (8192, 9, 15, 249),
])
def test_causal_pieces_by_hand(L, per, n_split, grid):
    """Causal single heads: each query tile's own key tiles are cut into the
    smallest pieces whose count fits one round of 256 CUs (worked by hand)."""
    hw = capi.attn_hw_desc_preset("gfx950")
    r = capi.attn_fwd_plan(1, 1, L, 128, 1, capi.ATTN_BF16, hw=hw)
    assert (r.tile_q, r.t_kv) == (256, 64)
    assert (r.tiles_per_split, r.n_split, r.grid, r.binding) == (per, n_split, grid, b"CU")


def _piece_of(b, BH, n_qt, L, tile_q, t_kv, P, n_split):
    """The fused kernel's placement of workgroup b of a causal-pieces launch,
    restated: heads fastest, the last query tile's pieces first, then
    piece-major over the whole query tiles, heaviest first."""
    C = tile_q // t_kv
    head, j = b % BH, b // BH
    n_last = -(-min(L, n_qt * tile_q) // t_kv)
    a_last = -(-n_last // P)
    if j < a_last:
        return head, n_qt - 1, j
    nf, jp, k = n_qt - 1, j - a_last, 0
    while k + 1 < n_split:
        cnt = nf - (k * P) // C
        if jp < cnt:
            break
        jp -= cnt
        k += 1
    return head, max(0, nf - 1 - jp), k


def test_causal_piece_placement_covers_every_piece_once():
    """For every plan that cuts causal query tiles into pieces, the kernel's
    placement maps the launched workgroups one to one onto the non-empty
    pieces (query tile qt has ceil(n_kv(qt) / P) of them)."""
    hw = capi.attn_hw_desc_preset("gfx950")
    n = 0
    for H, L, d in itertools.product((1, 2, 3), (1000, 3000, 5000, 8192, 12345, 16384, 20000, 32768),
                                     (64, 96, 128, 256)):
        r = capi.attn_fwd_plan(1, H, L, d, 1, capi.ATTN_BF16, hw=hw)
        n_qt = -(-L // r.tile_q)
        if r.n_split == 1 or r.grid == H * n_qt * r.n_split:
            continue  # no pieces
        n_kv = -(-L // r.t_kv)
        P = r.tiles_per_split
        want = {(h, qt, k) for h in range(H) for qt in range(n_qt)
                for k in range(-(-min(n_kv, -(-min(L, (qt + 1) * r.tile_q) // r.t_kv)) // P))}
        got = [_piece_of(b, H, n_qt, L, r.tile_q, r.t_kv, P, r.n_split) for b in range(r.grid)]
        assert len(got) == len(set(got)) == len(want) and set(got) == want, (H, L, d)
        n += 1
    assert n >= 20


def _persistent_launch(r, L, d, causal, num_cus=256):
    """The persistent-launch rule restated: no split, more query tiles than
    CUs, d = 64 or 128 (the compiled variants), every query tile at least 4
    key tiles long and on average at most 24, head offsets below 4 GiB."""
    if d not in (64, 128) or r.n_split != 1 or r.grid <= num_cus or r.n_waves != 8:
        return r.grid
    if (L + r.tile_q) * d * 2 >= 1 << 32:
        return r.grid
    n_kv, n_qt = -(-L // r.t_kv), -(-L // r.tile_q)
    tiles = [min(n_kv, -(-min(L, (qt + 1) * r.tile_q) // r.t_kv)) if causal else n_kv for qt in range(n_qt)]
    return num_cus if min(tiles) >= 4 and sum(tiles) <= 24 * n_qt else r.grid


def test_persistent_launch_by_hand():
    hw = capi.attn_hw_desc_preset("gfx950")
    bf = capi.ATTN_BF16
    cases = [
        # (B, H, L, d, causal) -> (grid, launch_grid)
        ((1, 1024, 512, 128, 0), (2048, 256)),   # 8 key tiles per query tile
        ((1, 128, 4096, 128, 0), (2048, 2048)),  # 64 key tiles: longer than 24
        ((2, 16, 4096, 128, 1), (512, 512)),     # config 3: 4, 8, ..., 64 key tiles, mean 34
        ((1, 512, 1024, 128, 1), (2048, 256)),   # causal: 4, 8, 12, 16, mean 10
        ((8, 40, 200, 128, 0), (320, 256)),      # 4 key tiles, rows 200..255 past the sequence
        ((1, 1000, 100, 128, 0), (1000, 1000)),  # 2 key tiles: too short for the switch
        ((1, 64, 1024, 128, 0), (256, 256)),     # one round already
        ((1, 512, 1024, 64, 0), (2048, 256)),    # d = 64: 8 key tiles of 128
        ((1, 512, 1024, 64, 1), (2048, 2048)),   # d = 64 causal: the first query tile sees 2
        ((1, 1024, 512, 256, 0), (4096, 4096)),  # d = 256: no persistent variant
        ((1, 1024, 512, 96, 0), (2048, 2048)),   # d = 96: no persistent variant
        ((1, 8, 1024, 128, 0), (256, 256)),      # split key ranges
    ]
    for (B, H, L, d, causal), (grid, launch) in cases:
        r = capi.attn_fwd_plan(B, H, L, d, causal, bf, hw=hw)
        assert (r.grid, r.launch_grid) == (grid, launch), (B, H, L, d, causal)
    # The derivation alone always launches its own grid.
    atom = capi.attn_atom_preset("bf16_16x16x32")
    op = capi.attn_fwd_op(1, 1024, 512, 128, 0, bf)
    rep = capi.attn_tile_derive(hw, atom, op)[1]
    assert rep.launch_grid == rep.grid == 2048


def test_persistent_launch_rule_over_shapes():
    hw = capi.attn_hw_desc_preset("gfx950")
    n = 0
    for B, H, L, d, causal, dt in itertools.product((1, 2, 8), (1, 16, 40, 128, 512), (100, 200, 256, 300, 512, 700,
                                                    1024, 1536, 2048, 4096), (64, 96, 128, 256), (0, 1),
                                                   (capi.ATTN_BF16, capi.ATTN_F16)):
        r = capi.attn_fwd_plan(B, H, L, d, causal, dt, hw=hw)
        assert r.launch_grid == _persistent_launch(r, L, d, causal), (B, H, L, d, causal)
        n += r.launch_grid != r.grid
    assert n > 100


def test_causal_halves_over_two_rounds_by_hand():
    """Four causal heads at L = 16384 fill one round of 256 CUs unsplit (64
    query tiles each), bound by the last tiles' 256 key tiles.  Halves of 128
    key tiles: query tiles 32 .. 63 (more than 128 key tiles) have two pieces,
    0 .. 31 one, so 4 (2 * 32 + 32) = 384 workgroups over two rounds."""
    hw = capi.attn_hw_desc_preset("gfx950")
    r = capi.attn_fwd_plan(1, 4, 16384, 128, 1, capi.ATTN_BF16, hw=hw)
    assert (r.tile_q, r.t_kv, r.tiles_per_split, r.n_split, r.grid, r.binding) == (256, 64, 128, 2, 384, b"CU")
    # 32 heads at L = 2048: halves would be 16 key tiles, too short to pay; unsplit
    r = capi.attn_fwd_plan(1, 32, 2048, 128, 1, capi.ATTN_BF16, hw=hw)
    assert (r.n_split, r.grid) == (1, 256)
    # 6 heads at L = 16384: 384 query tiles unsplit; halves would be 6 * 96 =
    # 576 workgroups, more than two rounds; unsplit
    r = capi.attn_fwd_plan(1, 6, 16384, 128, 1, capi.ATTN_BF16, hw=hw)
    assert (r.n_split, r.grid) == (1, 384)


# ------------------------------------------------------------ argument checks

P = 1 << 20  # a 16-byte aligned fake device address; never dereferenced


def _fwd(lib, q=P, k=P, v=P, o=P, B=1, H=1, L=16, d=64, scale=0.125, causal=0, dtype=0):
    return lib.attn_fwd(q, k, v, o, B, H, L, d, scale, causal, dtype, None)


@pytest.mark.parametrize("kw,code", [
    (dict(q=None), "ATTN_E_NULLPTR"), (dict(o=None), "ATTN_E_NULLPTR"),
    (dict(k=P + 8), "ATTN_E_ALIGN"), (dict(v=P + 2), "ATTN_E_ALIGN"),
    (dict(B=0), "ATTN_E_SHAPE"), (dict(H=-1), "ATTN_E_SHAPE"), (dict(L=0), "ATTN_E_SHAPE"),
    (dict(L=(1 << 24) + 1), "ATTN_E_SHAPE"), (dict(d=80), "ATTN_E_UNSUPPORTED_D"),
    (dict(d=0), "ATTN_E_UNSUPPORTED_D"), (dict(dtype=2), "ATTN_E_DTYPE"),
    (dict(scale=-1.0), "ATTN_E_SCALE"), (dict(scale=float("nan")), "ATTN_E_SCALE"),
    (dict(scale=float("inf")), "ATTN_E_SCALE"),
])
def test_fwd_rejects_bad_arguments(lib, kw, code):
    assert _fwd(lib, **kw) == capi.CODE[code]


def test_unfused_rejects_bad_arguments(lib):
    f = lib.attn_fwd_unfused
    ws = capi.attn_unfused_workspace_bytes(1, 1, 16, 0)
    assert ws == 16 * 16 * 2
    assert f(P, P, P, P, 1, 1, 16, 64, 0.1, 0, 0, None, ws, None) == capi.CODE["ATTN_E_WORKSPACE"]
    assert f(P, P, P, P, 1, 1, 16, 64, 0.1, 0, 0, P, ws - 1, None) == capi.CODE["ATTN_E_WORKSPACE"]
    assert f(P, P, P, P, 1, 1, 16, 64, 0.1, 0, 0, P + 4, ws, None) == capi.CODE["ATTN_E_ALIGN"]
    assert f(P, P, P, P, 1, 1, 12, 64, 0.1, 0, 0, P, ws, None) == capi.CODE["ATTN_E_SHAPE"]
    assert f(None, P, P, P, 1, 1, 16, 64, 0.1, 0, 0, P, ws, None) == capi.CODE["ATTN_E_NULLPTR"]
    assert capi.attn_unfused_workspace_bytes(0, 1, 16, 0) == 0


def test_partial_and_merge_reject_bad_arguments(lib):
    f = lib.attn_fwd_partial
    assert f(None, P, P, P, 1, 1, 16, 64, 0.1, 0, 0, None, 0, None) == capi.CODE["ATTN_E_NULLPTR"]
    assert f(P, P, P, P, 1, 1, 16, 80, 0.1, 0, 0, None, 0, None) == capi.CODE["ATTN_E_UNSUPPORTED_D"]
    assert f(P, P, P, P, 1, 1, 16, 64, -0.1, 0, 0, None, 0, None) == capi.CODE["ATTN_E_SCALE"]
    g = lib.attn_fwd_merge
    assert g(None, 0, None, 1, 1, 16, 64, 0.1, 0, 0, None) == capi.CODE["ATTN_E_NULLPTR"]
    assert g(None, 0, P, 0, 1, 16, 64, 0.1, 0, 0, None) == capi.CODE["ATTN_E_SHAPE"]
    out = ctypes.c_size_t(7)
    assert lib.attn_fwd_workspace_bytes(1, 1, 16, 80, 0, 0, ctypes.byref(out)) == capi.CODE["ATTN_E_UNSUPPORTED_D"]
    assert out.value == 0
    assert lib.attn_fwd_workspace_bytes(1, 1, 16, 64, 0, 0, None) == capi.CODE["ATTN_E_NULLPTR"]


def test_noalloc_rejects_bad_arguments(lib):
    f = lib.attn_fwd_noalloc
    assert f(None, P, P, P, 1, 1, 16, 64, 0.1, 0, 0, None) == capi.CODE["ATTN_E_NULLPTR"]
    assert f(P, P + 4, P, P, 1, 1, 16, 64, 0.1, 0, 0, None) == capi.CODE["ATTN_E_ALIGN"]
    assert f(P, P, P, P, 1, 1, 16, 80, 0.1, 0, 0, None) == capi.CODE["ATTN_E_UNSUPPORTED_D"]
    assert f(P, P, P, P, 1, 1, 16, 64, -0.1, 0, 0, None) == capi.CODE["ATTN_E_SCALE"]
    assert f(P, P, P, P, 0, 1, 16, 64, 0.1, 0, 0, None) == capi.CODE["ATTN_E_SHAPE"]
    with open(os.path.join(ROOT, "include", "attn.h")) as fh:
        m = re.search(r"#define ATTN_NOALLOC_SCRATCH_BYTES \((\d+)u << (\d+)\)", fh.read())
    assert int(m.group(1)) << int(m.group(2)) == capi.NOALLOC_SCRATCH_BYTES
    assert capi.attn_strerror(capi.CODE["ATTN_E_SCRATCH"]) != "unknown status"


def test_probe_rejects_bad_arguments(lib):
    assert lib.attn_mfma_probe(0, None, P, P, None) == capi.CODE["ATTN_E_NULLPTR"]
    assert lib.attn_mfma_probe(5, P, P, P, None) == capi.CODE["ATTN_E_ARG"]
    assert lib.attn_mfma_probe(0, P + 8, P, P, None) == capi.CODE["ATTN_E_ALIGN"]


def test_derive_rejects_bad_descriptors():
    hw = capi.attn_hw_desc_preset("gfx950")
    atom = capi.attn_atom_preset("bf16_16x16x32")
    op = capi.attn_fwd_op(1, 1, 128, 64, 0, capi.ATTN_BF16)
    bad = capi.HwDesc.from_buffer_copy(hw)
    bad.num_cus = 0
    with pytest.raises(capi.AttnError) as e:
        capi.attn_tile_derive(bad, atom, op)
    assert e.value.status == capi.CODE["ATTN_E_ARG"]
    with pytest.raises(capi.AttnError):
        capi.attn_fwd_op(1, 1, 128, 80, 0, capi.ATTN_BF16)


# ------------------------------------------------------------ compiled resources

def test_compiled_kernels_fit_without_scratch():
    path = os.path.join(ROOT, "_build", "kernel_resources.json")
    if not os.path.exists(path):
        pytest.skip("resource report is written by the build")
    with open(path) as f:
        res = json.load(f)
    fwd = {k: v for k, v in res.items() if "fwd_kernel" in k}
    # 40 instances, and the persistent variant of the 8-wave one at d = 64 and
    # 128 for both types.
    assert len(fwd) == 44
    persist = sorted(re.search(r"ILi(\d+)ELi(\d+)ELi\d+ELi\d+ELi8ELi5ELb1EE", k).groups() for k in fwd if "ELb1EE" in k)
    assert persist == [("0", "128"), ("0", "64"), ("1", "128"), ("1", "64")]
    for name, r in res.items():
        assert r["scratch"] == 0, name
    for name, r in fwd.items():
        nw = int(re.search(r"ILi\d+ELi\d+ELi\d+ELi\d+ELi(\d+)ELi\d+ELb[01]EE", name).group(1))
        waves_per_simd = max(1, nw // 4)
        assert r["vgpr"] + r["agpr"] <= 512 // waves_per_simd, name
        assert r["lds"] <= 160 * 1024
    # The named count of this kernel family: every tile the derivation accepts
    # at two waves per SIMD is one of the compiled 8-wave instances above (no
    # scratch, within 256 registers), and one more query block per wave is
    # refused by counting, at every head dimension.
    hw = capi.attn_hw_desc_preset("gfx950")
    atom = capi.attn_atom_preset("bf16_16x16x32")
    est = {}
    for d, t_kv, t_q in ((64, 128, 32), (96, 64, 48), (128, 64, 32), (256, 32, 16)):
        op = capi.attn_fwd_op(1, 1, 16384, d, 0, capi.ATTN_BF16)
        assert (op.p_tiles, op.stat_regs, op.operand_frags, op.vgpr_fixed) == (1, 7, 5, 14)
        est[d] = capi.attn_vgpr_estimate(hw, atom, op, t_q, t_kv, 8)
        assert est[d] <= 256 < capi.attn_vgpr_estimate(hw, atom, op, t_q + 16, t_kv, 8), d
        r = capi.attn_fwd_plan(1, 1, 16384, d, 0, capi.ATTN_BF16, hw=hw)
        assert (r.t_kv, r.t_q_wave, r.vgpr_est) == (t_kv, t_q, est[d])
        tag = f"ILi0ELi{d}ELi{t_kv}ELi{t_q // 16}ELi8ELi5ELb0EE"
        comp = [v for k, v in fwd.items() if tag in k][0]
        assert comp["scratch"] == 0 and comp["vgpr"] + comp["agpr"] <= 256
    # d = 128, 32 rows: 32 (Q) + 32 (S) + 64 (O) + 16 (P) + 2 x 7 (statistics)
    # + 5 x 4 (fragments) + 14 (addresses, copy offsets and constants) = 192
    assert est[128] == 192
    # the d = 64, 48-row tile: 24 + 96 + 48 + 48 + 21 + 20 + 14 = 271 > 256
    op64 = capi.attn_fwd_op(1, 1, 16384, 64, 0, capi.ATTN_BF16)
    assert capi.attn_vgpr_estimate(hw, atom, op64, 48, 128, 8) == 271


def test_one_hip_runtime_after_load():
    """Loading the library in a fresh process, before anything imports torch,
    leaves one HIP runtime mapped: the binding loads torch's copy first, so
    torch's streams and pointers are valid in the library's calls."""
    import subprocess
    import sys
    code = ("import sys; sys.path.insert(0, %r)\n"
            "from paper_2609_10937_amd import capi\n"
            "capi.load()\n"
            "paths = {l.split()[-1] for l in open('/proc/self/maps') if 'libamdhip64' in l}\n"
            "print(len(paths)); print(sorted(paths))\n") % ROOT
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    assert out.returncode == 0, out.stderr
    lines = out.stdout.split("\n")
    assert lines[0] == "1", out.stdout


def test_gfx942_class_descriptor():
    """The derivation on MI300X's published figures (64 KiB LDS, 512 registers,
    304 CUs, the 16x16x16 atom) for this library's kernel structures: the ten
    staged K/V tiles leave t_kv = floor(65536 / (10 * 128 * 2)) = 25 -> 16 at
    d = 128 and nothing at d = 256; the GEMM's five stages of 1 KB copy blocks
    leave no t_K.  A port needs fewer stages; the kernels are built for gfx950."""
    hw = capi.attn_hw_desc_preset("gfx942")
    assert (hw.lds_bytes, hw.vgpr_per_thread, hw.num_cus, hw.name) == (65536, 512, 304, b"gfx942")
    atom = capi.attn_atom_preset("bf16_16x16x16")
    assert (atom.m, atom.n, atom.k) == (16, 16, 16)
    op = capi.attn_fwd_op(1, 1, 16384, 128, 0, capi.ATTN_BF16)
    rc, r = capi.attn_tile_derive(hw, atom, op)
    assert rc == 0 and r.t_kv == 16 and r.lds_used == 10 * 16 * 128 * 2
    # 43 query tiles of 384 rows, 1024 key tiles: 7 splits of 147 tiles fill
    # one round of 301 workgroups on 304 CUs (8 splits would take two rounds).
    assert (r.tile_q, r.n_split, r.grid) == (384, 7, 301)
    assert r.vgpr_est <= r.vgpr_budget == 256
    op = capi.attn_fwd_op(1, 1, 16384, 256, 0, capi.ATTN_BF16)
    rc, r = capi.attn_tile_derive(hw, atom, op)
    assert rc == capi.CODE["ATTN_E_INFEASIBLE"] and r.binding == b"LDS"
    with pytest.raises(capi.AttnError) as e:
        capi.attn_gemm_derive(hw, atom, 4096, 4096, 4096)
    assert e.value.status == capi.CODE["ATTN_E_INFEASIBLE"]
    with pytest.raises(capi.AttnError):
        capi.attn_hw_desc_preset("gfx90x")
