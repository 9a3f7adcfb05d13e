"""GPU parity of the GEMM operator (Section 4's worked example, Figure 1) with
the float64 oracle, through the C ABI.

The inputs are exact in the storage type and every product of two 16-bit
values is exact in fp32, so the only error is the fp32 summation of K terms:
|C - A B| <= K u (|A| |B|) element-wise with u = 2^-24 (the standard bound
for any summation order).  The section validates its GEMM at machine
precision against a double-precision reference; here that bound is checked
for every element, and the relative Frobenius error is held to a few fp32
roundings."""
import numpy as np
import pytest

from oracle import gemm as G
from paper_2609_10937_amd import capi, inputs

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import _gpu  # noqa: E402

U32 = 2.0 ** -24


def _run(M, N, K, dtype, seed, spread=1.0):
    print(f"case gemm {M}x{N}x{K} {dtype} seed {seed}", flush=True)
    a = inputs.make_matrix(M, K, dtype, seed=seed, spread=spread)
    b = inputs.make_matrix(K, N, dtype, seed=seed + 1, spread=spread)
    ta, tb = _gpu.upload(a, dtype), _gpu.upload(b, dtype)
    tc = torch.empty((M, N), dtype=torch.float32, device="cuda")
    capi.attn_gemm(ta, tb, tc)
    torch.cuda.synchronize()
    return inputs.bits_to_f64(a, dtype), inputs.bits_to_f64(b, dtype), tc.cpu().numpy().astype(np.float64)


def _check(af, bf, got, what):
    ref = G.gemm(af, bf)
    bound = af.shape[1] * U32 * G.gemm(np.abs(af), np.abs(bf)) + 1e-30
    err = np.abs(got - ref)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    bad = err > bound
    assert not bad.any(), f"{what}: {int(bad.sum())} elements beyond K u |A||B| (max ratio {float((err / bound).max()):.2f})"
    rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300)
    assert rel < 4 * U32 * np.sqrt(af.shape[1]), f"{what}: relative Frobenius error {rel:.3e}"
    return rel


# Each shape reaches a different tile of the derivation on gfx950 (the
# instance table); K not a multiple of t_K takes the last-tile masking, M and
# N not multiples of the tile take the clamped edge tiles.
SHAPES = [
    (4096, 4096, 4096, "bf16"),   # the section's 4096^3: 256 x 256 x 32, one tile per CU
    (4100, 4104, 1000, "bf16"),   # 256 x 256 x 32 with ragged M, N and K
    (4096, 2048, 520, "f16"),     # 128 x 256 x 32
    (2048, 2048, 256, "bf16"),    # 128 x 128 x 64
    (1536, 1536, 200, "f16"),     # 64 x 128 x 64, ragged K
    (1000, 1000, 136, "bf16"),    # 64 x 64 x 128, ragged M, N, K
    (300, 104, 40, "f16"),        # 32 x 64 x 128: one partial k tile
    (1, 8, 8, "bf16"),            # smallest admitted problem
    (4096, 4096, 8, "bf16"),      # one k tile of 8 columns
    (33, 4104, 4104, "f16"),      # many k tiles, ragged tail of 8
]


@pytest.mark.parametrize("M,N,K,dtype", SHAPES)
def test_gemm_matches_oracle(M, N, K, dtype):
    af, bf, got = _run(M, N, K, dtype, seed=M * 7 + N * 3 + K)
    _check(af, bf, got, f"{M}x{N}x{K} {dtype}")


def test_identity_is_exact():
    """A I = A exactly (every sum has one nonzero term), at the 4096^3 tile."""
    M = K = N = 1024
    a = inputs.make_matrix(M, K, "bf16", seed=5)
    eye = inputs.round_bits(np.eye(K, dtype=np.float32), "bf16")
    ta, tb = _gpu.upload(a, "bf16"), _gpu.upload(eye, "bf16")
    tc = torch.empty((M, N), dtype=torch.float32, device="cuda")
    capi.attn_gemm(ta, tb, tc)
    torch.cuda.synchronize()
    assert np.array_equal(tc.cpu().numpy().astype(np.float64), inputs.bits_to_f64(a, "bf16"))


def test_large_values_and_repeat_calls():
    """Wide dynamic range, two calls in a row into the same output (no state
    carried between calls)."""
    af, bf, got = _run(2048, 1024, 512, "bf16", seed=77, spread=1000.0)
    _check(af, bf, got, "spread 1000")
    af2, bf2, got2 = _run(2048, 1024, 512, "bf16", seed=78)
    _check(af2, bf2, got2, "second call")


def test_rejects_mismatched_tensors():
    a = torch.zeros((64, 64), dtype=torch.bfloat16, device="cuda")
    b = torch.zeros((64, 64), dtype=torch.float16, device="cuda")
    c = torch.zeros((64, 64), dtype=torch.float32, device="cuda")
    with pytest.raises(capi.AttnError):
        capi.attn_gemm(a, b, c)
    with pytest.raises(capi.AttnError):
        capi.attn_gemm(a, a, c.to(torch.bfloat16))


# ------------------------------------------------------------ fp32 (the section's own type)

def _run32(M, N, K, seed, spread=1.0):
    print(f"case gemm fp32 {M}x{N}x{K} seed {seed}", flush=True)
    a = inputs.make_matrix_f32(M, K, seed=seed, spread=spread)
    b = inputs.make_matrix_f32(K, N, seed=seed + 1, spread=spread)
    tc = torch.empty((M, N), dtype=torch.float32, device="cuda")
    capi.attn_gemm(torch.from_numpy(a).cuda(), torch.from_numpy(b).cuda(), tc)
    torch.cuda.synchronize()
    return a.astype(np.float64), b.astype(np.float64), tc.cpu().numpy().astype(np.float64)


def _check32(af, bf, got, what):
    """fp32 products are rounded too: each element is within (K + 4) u |A||B|
    of the fp64 product (the inner-product bound gamma_K with slack), and the
    relative Frobenius error stays at a few fp32 roundings."""
    ref = G.gemm(af, bf)
    bound = (af.shape[1] + 4) * U32 * G.gemm(np.abs(af), np.abs(bf)) + 1e-30
    err = np.abs(got - ref)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    bad = err > bound
    assert not bad.any(), f"{what}: {int(bad.sum())} elements beyond (K+4) u |A||B| (max ratio {float((err / bound).max()):.2f})"
    rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300)
    assert rel < 4 * U32 * np.sqrt(af.shape[1]), f"{what}: relative Frobenius error {rel:.3e}"
    return rel


SHAPES32 = [
    (4096, 4096, 4096),    # the section's 4096^3: 192 x 192 x 32, 484 tiles
    (4100, 4100, 1000),    # 192 x 192 x 32 with ragged M, N and K
    (256, 16384, 1000),    # 96 x 192 x 32
    (256, 8192, 516),      # 96 x 96 x 64, ragged K
    (64, 16384, 500),      # 32 x 96 x 96, ragged K
    (100, 64, 40),         # 32 x 32 x 192: one partial k tile
    (1, 4, 4),             # smallest admitted problem
]


@pytest.mark.parametrize("M,N,K", SHAPES32)
def test_gemm_fp32_matches_oracle(M, N, K):
    af, bf, got = _run32(M, N, K, seed=M * 5 + N * 3 + K)
    rel = _check32(af, bf, got, f"fp32 {M}x{N}x{K}")
    print(f"  fp32 {M}x{N}x{K}: relative error {rel:.3e}", flush=True)


def test_gemm_fp32_identity_is_exact():
    """A I = A exactly in fp32 (one nonzero term per sum)."""
    a = inputs.make_matrix_f32(1000, 1000, seed=9)
    tc = torch.empty((1000, 1000), dtype=torch.float32, device="cuda")
    capi.attn_gemm(torch.from_numpy(a).cuda(), torch.eye(1000, dtype=torch.float32, device="cuda"), tc)
    torch.cuda.synchronize()
    assert np.array_equal(tc.cpu().numpy(), a)


def _random_gemm_cases(n=16, seed=4096):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        dtype = str(rng.choice(["bf16", "f16", "f32"]))
        step = 4 if dtype == "f32" else 8
        out.append((int(rng.integers(1, 3001)), step * int(rng.integers(1, 3001 // step + 1)),
                    step * int(rng.integers(1, 2049 // step + 1)), dtype))
    return out


@pytest.mark.parametrize("M,N,K,dtype", _random_gemm_cases())
def test_gemm_random_shapes(M, N, K, dtype):
    """Seeded random shapes (any M; N and K multiples of the 16-byte chunk),
    every type, through whatever tile the derivation picks: the element-wise
    summation bound against the oracle."""
    if dtype == "f32":
        af, bf, got = _run32(M, N, K, seed=M + N + K)
        _check32(af, bf, got, f"random fp32 {M}x{N}x{K}")
    else:
        af, bf, got = _run(M, N, K, dtype, seed=M + N + K)
        _check(af, bf, got, f"random {dtype} {M}x{N}x{K}")
