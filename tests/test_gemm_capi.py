"""Host side of the GEMM operator (Section 4's worked example): the library's
derivation against the oracle's model and closed forms, and the C ABI's
argument checks (no GPU needed)."""
import ctypes

import pytest
from hypothesis import given, settings, strategies as stg

from oracle import gemm as G
from paper_2609_10937_amd import capi

# The kernel families' fixed structures.  16-bit atoms: 5 LDS stages, 2 x 4
# waves, 2 waves per SIMD, 96 registers outside the accumulators; fp32 atoms:
# 3 stages, 2 x 2 waves, 1 wave per SIMD, 128; both with 1 KB copy blocks.
STRUCT = G.GemmStructure(stages=5, waves_m=2, waves_n=4, waves_per_simd=2, vgpr_fixed=96, copy_block=1024)
STRUCT32 = G.GemmStructure(stages=3, waves_m=2, waves_n=2, waves_per_simd=1, vgpr_fixed=128, copy_block=1024)
ATOM16 = capi.attn_atom_preset("bf16_16x16x32")
ATOM32 = capi.attn_atom_preset("f32_16x16x4")


def _hw(**kw):
    base = capi.attn_hw_desc_preset("gfx950")
    for k, v in kw.items():
        setattr(base, k, v)
    return base


def _model(hw, atom, M, N, K):
    return G.derive(hw.lds_bytes, hw.vgpr_per_thread, hw.wavefront_size, hw.num_cus, atom.m, atom.n, atom.k,
                    atom.in_bytes, atom.acc_bytes, M, N, K, STRUCT32 if atom.in_bytes == 4 else STRUCT)


# (M, N, K) -> tile the derivation gives on gfx950 (256 CUs, 160 KB LDS)
TILES = [
    ((4096, 4096, 4096), (256, 256, 32, "LDS", 256)),   # the paper's shape: one tile per CU
    ((8192, 8192, 8192), (256, 256, 32, "LDS", 1024)),
    ((4096, 2048, 512), (128, 256, 32, "CU", 256)),
    ((2048, 2048, 256), (128, 128, 64, "CU", 256)),
    ((1536, 1536, 200), (64, 128, 64, "CU", 288)),
    ((1000, 1000, 136), (64, 64, 128, "CU", 256)),
    ((512, 512, 512), (32, 64, 128, "CU", 128)),        # floor: one atom per wave
]


@pytest.mark.parametrize("shape,want", TILES)
def test_gfx950_tiles(shape, want):
    r = capi.attn_gemm_derive(_hw(), ATOM16, *shape)
    assert (r.t_m, r.t_n, r.t_k, r.binding.decode(), r.grid) == want
    assert r.lds_used <= r.lds_budget == 163840 and r.vgpr_est <= r.vgpr_budget == 256
    assert (r.stages, r.waves_per_wg, r.warp_m, r.warp_n) == (5, 8, r.t_m // 2, r.t_n // 4)


# fp32 (the section's own type) on its family's structure
TILES32 = [
    ((4096, 4096, 4096), (192, 192, 32, "LDS", 484)),   # sqrt(40960) = 202 -> 192 (aligned to 32 x 2)
    ((256, 16384, 1000), (96, 192, 32, "CU", 258)),
    ((256, 8192, 512), (96, 96, 64, "CU", 258)),
    ((64, 16384, 512), (32, 96, 96, "CU", 342)),
    ((100, 64, 40), (32, 32, 192, "CU", 8)),
]


@pytest.mark.parametrize("shape,want", TILES32)
def test_gfx950_tiles_fp32(shape, want):
    r = capi.attn_gemm_derive(_hw(), ATOM32, *shape)
    assert (r.t_m, r.t_n, r.t_k, r.binding.decode(), r.grid) == want
    assert r.lds_used <= r.lds_budget and r.vgpr_est <= r.vgpr_budget == 512
    assert (r.stages, r.waves_per_wg, r.warp_m, r.warp_n) == (3, 4, r.t_m // 2, r.t_n // 2)


def test_fp32_tile_closed_form():
    """192 x 192 x 32 at 4-byte elements: t_K = 160 KB / (3 * 384 * 4 B) = 35,
    aligned down to 32 (the A and B tiles, 192 x 32 x 4 B = 24 KB each, are
    6 whole 1 KB blocks per wave); 96 x 96 accumulators per wave = 36 atoms x 4
    registers + 128 fixed = 272 of the 512 at one wave per SIMD."""
    r = capi.attn_gemm_derive(_hw(), ATOM32, 4096, 4096, 4096)
    assert (r.lds_used, r.vgpr_est) == (3 * 384 * 32 * 4, 272)


def test_square_tile_fills_lds():
    """sqrt(160 KB / 2 B) = 286 -> 256 x 256; t_K = 160 KB / (5 * 512 * 2 B) = 32:
    the five stages take all of LDS and the 128 accumulators per lane plus the
    fixed registers (224) fit the 256 of two waves per SIMD."""
    r = capi.attn_gemm_derive(_hw(), ATOM16, 4096, 4096, 4096)
    assert r.lds_used == 163840 and r.vgpr_est == 224 and r.wg_per_cu == 1.0


def test_vgpr_rule_binds():
    """At a budget of 128 registers per lane the 256 x 256 tile's 128
    accumulators no longer fit: 128 x 256 still needs 64 + 96, 128 x 128
    needs 32 + 96 = 128."""
    r = capi.attn_gemm_derive(_hw(vgpr_per_thread=256), ATOM16, 8192, 8192, 8192)
    assert (r.t_m, r.t_n, r.vgpr_est, r.binding.decode()) == (128, 128, 128, "VGPR")


def test_infeasible():
    with pytest.raises(capi.AttnError) as e:
        capi.attn_gemm_derive(_hw(lds_bytes=4096), ATOM16, 64, 64, 64)
    assert e.value.status == capi.CODE["ATTN_E_INFEASIBLE"]
    with pytest.raises(capi.AttnError) as e:
        capi.attn_gemm_derive(_hw(), ATOM16, 0, 64, 64)
    assert e.value.status == capi.CODE["ATTN_E_SHAPE"]


@settings(max_examples=400, deadline=None)
@given(lds=stg.sampled_from([32768, 65536, 98304, 131072, 163840, 262144]),
       vgpr=stg.sampled_from([256, 384, 512]),
       cus=stg.integers(1, 400),
       atom=stg.sampled_from(["bf16_16x16x32", "f32_16x16x4"]),
       M=stg.integers(1, 1 << 15), N=stg.integers(1, 1 << 15), K=stg.integers(1, 1 << 14))
def test_matches_oracle_model(lds, vgpr, cus, atom, M, N, K):
    hw = _hw(lds_bytes=lds, vgpr_per_thread=vgpr, num_cus=cus)
    a = capi.attn_atom_preset(atom)
    ref = _model(hw, a, M, N, K)
    if ref is None:
        with pytest.raises(capi.AttnError):
            capi.attn_gemm_derive(hw, a, M, N, K)
        return
    r = capi.attn_gemm_derive(hw, a, M, N, K)
    for k in ("t_m", "t_n", "t_k", "warp_m", "warp_n", "grid", "vgpr_est", "vgpr_budget", "lds_used"):
        assert getattr(r, k) == ref[k], k
    assert r.binding.decode() == ref["binding"]
    assert r.wg_per_cu == pytest.approx(ref["wg_per_cu"])


def _p(v):
    return ctypes.c_void_p(v)


@pytest.mark.parametrize("M,N,K,code", [
    (0, 64, 64, "ATTN_E_SHAPE"), (64, 4, 64, "ATTN_E_SHAPE"), (64, 68, 64, "ATTN_E_SHAPE"),
    (64, 64, 4, "ATTN_E_SHAPE"), (64, 64, 68, "ATTN_E_SHAPE"), (64, 64, (1 << 22) + 8, "ATTN_E_SHAPE"),
    (64, (1 << 24) + 8, 64, "ATTN_E_SHAPE"), (1 << 31, 64, 64, "ATTN_E_SHAPE"),
])
def test_rejects_shapes(lib, M, N, K, code):
    assert lib.attn_gemm(_p(256), _p(512), _p(1024), M, N, K, 0, None) == capi.CODE[code]


@pytest.mark.parametrize("M,N,K", [(64, 2, 64), (64, 66, 64), (64, 64, 66), (64, (1 << 22) + 4, 64),
                                   (64, 64, (1 << 22) + 4)])
def test_rejects_shapes_fp32(lib, M, N, K):
    assert lib.attn_gemm(_p(256), _p(512), _p(1024), M, N, K, capi.ATTN_F32, None) == capi.CODE["ATTN_E_SHAPE"]


def test_rejects_pointers_and_dtype(lib):
    assert lib.attn_gemm(None, _p(512), _p(1024), 64, 64, 64, 0, None) == capi.CODE["ATTN_E_NULLPTR"]
    assert lib.attn_gemm(_p(256), _p(512), None, 64, 64, 64, 0, None) == capi.CODE["ATTN_E_NULLPTR"]
    assert lib.attn_gemm(_p(256), _p(512), _p(1024), 64, 64, 64, 7, None) == capi.CODE["ATTN_E_DTYPE"]
    assert lib.attn_fwd(_p(256), _p(256), _p(256), _p(256), 1, 1, 16, 64, 0.1, 0, capi.ATTN_F32,
                        None) == capi.CODE["ATTN_E_DTYPE"]
    assert lib.attn_gemm(_p(264), _p(512), _p(1024), 64, 64, 64, 0, None) == capi.CODE["ATTN_E_ALIGN"]
    assert lib.attn_gemm(_p(256), _p(512), _p(1028), 64, 64, 64, 1, None) == capi.CODE["ATTN_E_ALIGN"]
