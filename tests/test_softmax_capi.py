"""Host side of the row-softmax operator: the library's derivation against
the oracle's model and closed forms, and the C ABI's argument checks (no
GPU needed)."""
import ctypes

import pytest
from hypothesis import given, settings, strategies as stg

from oracle import tile_model as T
from paper_2609_10937_amd import capi


def _hw(**kw):
    base = capi.attn_hw_desc_preset("gfx950")
    for k, v in kw.items():
        setattr(base, k, v)
    return base


def _model_hw(h):
    return T.Hardware(lds_bytes=h.lds_bytes, vgpr_per_thread=h.vgpr_per_thread, wavefront_size=h.wavefront_size,
                      num_cus=h.num_cus, simds_per_cu=h.simds_per_cu)


def _same(r, m):
    for k, v in m.items():
        got = getattr(r, k)
        got = got.decode() if isinstance(got, bytes) else got
        assert got == v, (k, got, v)


def test_gfx950_closed_forms():
    hw = _hw()
    r = capi.attn_softmax_derive(hw, 512, 512)       # the paper's validation shape
    assert (r.tile_elems, r.resident_tiles, r.vgpr_budget) == (512, 32, 256)
    assert (r.split, r.rows_per_wg, r.grid, r.passes, r.binding) == (1, 4, 128, 1, b"CU")
    r = capi.attn_softmax_derive(hw, 16384, 16384)   # the scores of one L=16384 head
    assert (r.split, r.grid, r.passes, r.binding, r.hbm_bytes) == (1, 4096, 1, b"none", 2 * 16384 * 16384 * 2)
    r = capi.attn_softmax_derive(hw, 1, 100000)      # one long row: split over the workgroup, read twice
    assert (r.split, r.seg, r.passes, r.binding) == (4, 25000, 2, b"VGPR")
    assert r.vgpr_est == 32 * 4 + 48 <= r.vgpr_budget


@settings(max_examples=400, deadline=None)
@given(vgpr=stg.sampled_from([128, 256, 512]), wf=stg.sampled_from([32, 64]), cus=stg.integers(1, 512),
       rows=stg.integers(1, 1 << 22), n=stg.integers(1, 1 << 24), elem=stg.sampled_from([1, 2, 4]))
def test_library_matches_oracle_model(vgpr, wf, cus, rows, n, elem):
    hw = _hw(vgpr_per_thread=vgpr, wavefront_size=wf, num_cus=cus)
    m = T.derive_softmax(_model_hw(hw), rows, n, elem)
    if m is None:
        with pytest.raises(capi.AttnError):
            capi.attn_softmax_derive(hw, rows, n, elem)
        return
    r = capi.attn_softmax_derive(hw, rows, n, elem)
    _same(r, m)
    # the tiles cover the row, fit the registers, and the grid covers the rows
    assert r.split * r.seg >= n and r.seg % 8 == 0
    assert r.vgpr_est <= r.vgpr_budget
    assert r.grid * r.rows_per_wg >= rows
    assert r.split == 1 or r.split * r.tile_elems <= 2 * n


def test_argument_checks():
    lib = capi.load()
    P = 1 << 20
    f = lib.attn_softmax
    assert f(None, P, 4, 8, 0, 0, None) == capi.CODE["ATTN_E_NULLPTR"]
    assert f(P, P, 4, 8, 0, 7, None) == capi.CODE["ATTN_E_DTYPE"]
    assert f(P, P, 0, 8, 0, 0, None) == capi.CODE["ATTN_E_SHAPE"]
    assert f(P, P, 4, 0, 0, 0, None) == capi.CODE["ATTN_E_SHAPE"]
    assert f(P, P, 4, (1 << 31) + 1, 0, 0, None) == capi.CODE["ATTN_E_SHAPE"]
    assert f(P + 1, P, 4, 8, 0, 0, None) == capi.CODE["ATTN_E_ALIGN"]
    r = capi.SoftmaxReport()
    assert lib.attn_softmax_derive(ctypes.byref(_hw()), 0, 5, 2, ctypes.byref(r)) == capi.CODE["ATTN_E_SHAPE"]
    assert lib.attn_softmax_derive(ctypes.byref(_hw()), 5, 5, 3, ctypes.byref(r)) == capi.CODE["ATTN_E_ARG"]
