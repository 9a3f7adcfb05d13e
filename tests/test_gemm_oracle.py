"""Pins of the GEMM oracle and of its tile derivation (Section 4)."""
import math

import numpy as np
import pytest

from oracle import gemm as G


def _brute(a, b):
    return [[math.fsum(a[i][k] * b[k][j] for k in range(len(b))) for j in range(len(b[0]))] for i in range(len(a))]


@pytest.mark.parametrize("shape", [(1, 1, 1), (3, 5, 7), (8, 16, 4)])
def test_gemm_matches_brute_force(shape):
    M, N, K = shape
    rng = np.random.default_rng(M * 100 + N)
    a, b = rng.standard_normal((M, K)), rng.standard_normal((K, N))
    assert np.allclose(G.gemm(a, b), _brute(a.tolist(), b.tolist()), rtol=1e-13, atol=1e-14)


def test_gemm_closed_forms():
    rng = np.random.default_rng(3)
    a, b, c = rng.standard_normal((6, 5)), rng.standard_normal((5, 4)), rng.standard_normal((4, 3))
    assert np.array_equal(G.gemm(np.eye(6), a), a) and np.array_equal(G.gemm(a, np.eye(5)), a)
    assert np.allclose(G.gemm(G.gemm(a, b), c), G.gemm(a, G.gemm(b, c)), rtol=1e-12)
    assert np.allclose(G.gemm(a, b).T, G.gemm(b.T, a.T), rtol=1e-13)
    # small integers: exact
    ai, bi = rng.integers(-8, 9, (7, 9)), rng.integers(-8, 9, (9, 3))
    assert np.array_equal(G.gemm(ai, bi), (ai @ bi).astype(np.float64))


def test_copy_blocks_align_t_k():
    """The smallest tile (32 x 64, the CU rule's floor) takes t_K = 128, not the
    160 that LDS alone allows: with 160 the A tile (32 x 160 x 2 B = 10 KB) is
    not a whole number of 1 KB blocks for each of the 8 waves."""
    r = G.derive(163840, 512, 64, 256, 16, 16, 32, 2, 4, 64, 64, 4096, GFX950)
    assert (r["t_m"], r["t_n"], r["t_k"]) == (32, 64, 128)


def test_paper_gemm_tree():
    """Figure 1 / Section 4: 64 KB LDS, 4-byte elements, 16x16x4 atom, 120 CUs:
    CU tile 128 x 128 x 32, 32 KB of LDS per stage, 32 x 32 = 1024 tiles
    (8.5 per CU), warp tile 32 x 32 with 16 accumulators per lane."""
    st = G.GemmStructure(stages=2, waves_m=4, waves_n=4, waves_per_simd=1, vgpr_fixed=32)
    r = G.derive(65536, 256, 64, 120, 16, 16, 4, 4, 4, 4096, 4096, 4096, st)
    assert (r["t_m"], r["t_n"], r["t_k"]) == (128, 128, 32)
    assert r["lds_used"] // st.stages == 32 * 1024
    assert r["grid"] == 1024 and round(r["wg_per_cu"], 1) == 8.5
    assert (r["warp_m"], r["warp_n"]) == (32, 32) and r["vgpr_est"] - st.vgpr_fixed == 16


GFX950 = G.GemmStructure(stages=5, waves_m=2, waves_n=4, waves_per_simd=2, vgpr_fixed=96, copy_block=1024)


def test_gfx950_tiles():
    st = GFX950
    r = G.derive(163840, 512, 64, 256, 16, 16, 32, 2, 4, 4096, 4096, 4096, st)
    assert (r["t_m"], r["t_n"], r["t_k"], r["grid"]) == (256, 256, 32, 256)
    assert r["vgpr_est"] == 128 + 96 <= r["vgpr_budget"] == 256
    assert r["lds_used"] == 5 * 512 * 32 * 2 <= 163840
    # a small problem: the CU rule shrinks the tile until the grid covers the CUs
    r = G.derive(163840, 512, 64, 256, 16, 16, 32, 2, 4, 1024, 1024, 4096, st)
    assert r["binding"] == "CU" and r["grid"] >= 256 and r["t_m"] * r["t_n"] < 256 * 256


@pytest.mark.parametrize("M,N", [(1, 1), (100, 3000), (4096, 4096), (50000, 64), (1024, 1024)])
def test_derivation_invariants(M, N):
    st = GFX950
    r = G.derive(163840, 512, 64, 256, 16, 16, 32, 2, 4, M, N, 256, st)
    assert r["t_m"] % 32 == 0 and r["t_n"] % 64 == 0 and r["t_k"] % 32 == 0
    assert (r["t_m"] * r["t_k"] * 2) % 8192 == 0 and (r["t_n"] * r["t_k"] * 2) % 8192 == 0
    assert r["lds_used"] <= 163840 and r["vgpr_est"] <= r["vgpr_budget"]
    assert r["grid"] == -(-M // r["t_m"]) * -(-N // r["t_n"])
