"""GPU parity of the row-softmax operator (Section 5.3) with the float64 oracle."""
import numpy as np
import pytest

from oracle import softmax as SM
from paper_2609_10937_amd import capi, inputs

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import _gpu  # noqa: E402


def _check(got, ref, dtype, what):
    # every output is a probability: the parity bar of the fused kernel, and
    # element-wise one rounding of the output type on top of fp32 arithmetic
    _gpu.assert_close(got, ref, dtype, what)
    ulp = 2.0 ** -8 if dtype == "bf16" else 2.0 ** -11
    bad = np.abs(got - ref) > ulp * ref + 1e-6
    assert not bad.any(), f"{what}: {int(bad.sum())} elements beyond one rounding"


CASES = [
    (512, 512, "bf16", 1.0),       # the paper's validation shape
    (512, 512, "f16", 3.0),
    (7, 1001, "f16", 1.0),         # odd row length: element-wise accesses
    (1, 1, "bf16", 1.0),
    (3, 20000, "bf16", 3.0),       # rows split over the workgroup's waves
    (1, 100000, "bf16", 1.0),      # split and longer than the resident tiles: read twice
    (16, 300001, "f16", 0.1),      # flat rows, read twice, odd length
    (300, 40000, "bf16", 3.0),
]


@pytest.mark.parametrize("rows,n,dtype,spread", CASES)
def test_softmax_rows(rows, n, dtype, spread):
    print(f"case softmax {rows}x{n} {dtype} spread {spread}", flush=True)
    x = inputs.make_matrix(rows, n, dtype, seed=rows * 31 + n, spread=spread)
    tx = _gpu.upload(x, dtype)
    ty = torch.empty_like(tx)
    capi.attn_softmax(tx, ty)
    torch.cuda.synchronize()
    ref = SM.softmax_rows(inputs.bits_to_f64(x, dtype))
    _check(_gpu.download(ty, dtype), ref, dtype, f"{rows}x{n}")


@pytest.mark.parametrize("n,blocks,dtype", [(1000, 2, "bf16"), (4096, 1, "f16"), (64, 5, "bf16")])
def test_softmax_causal_in_place(n, blocks, dtype):
    """Square n x n blocks stacked along the rows, masked above each block's
    diagonal, written over the input (the attention score layout)."""
    print(f"case softmax causal {blocks}x{n}x{n} {dtype}", flush=True)
    x = inputs.make_matrix(blocks * n, n, dtype, seed=n + blocks, spread=2.0)
    tx = _gpu.upload(x, dtype)
    capi.attn_softmax(tx, tx, causal=True)
    torch.cuda.synchronize()
    xf = inputs.bits_to_f64(x, dtype).reshape(blocks, n, n)
    ref = np.concatenate([SM.softmax_rows(b, causal=True) for b in xf])
    got = _gpu.download(tx, dtype)
    _check(got, ref, dtype, f"causal {n}")
    assert np.all(got[np.triu(np.ones((n, n), bool), 1)[None].repeat(blocks, 0).reshape(-1, n)] == 0)


def test_softmax_rows_sum_to_one_large():
    """rows x n = 16384 x 16384 (the scores of one L=16384 head): sampled rows
    against the oracle and every row's sum within rounding of 1."""
    rows = n = 16384
    print(f"case softmax {rows}x{n} (sampled)", flush=True)
    x = inputs.make_matrix(rows, n, "bf16", seed=77, spread=2.0)
    tx = _gpu.upload(x, "bf16")
    ty = torch.empty_like(tx)
    capi.attn_softmax(tx, ty)
    torch.cuda.synchronize()
    sums = ty.float().sum(dim=1)
    assert torch.all((sums - 1).abs() < 2e-2)
    idx = np.unique(np.concatenate([np.arange(8), np.arange(rows - 8, rows),
                                    np.random.default_rng(4).integers(0, rows, 48)]))
    ref = SM.softmax_rows(inputs.bits_to_f64(x[idx], "bf16"))
    _check(_gpu.download(ty[torch.from_numpy(idx).cuda()], "bf16"), ref, "bf16", "16384 sampled")


def _random_softmax_cases(n=16, seed=512):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        rows = int(rng.integers(1, 400))
        cols = int(rng.choice([int(rng.integers(1, 70000)), 8 * int(rng.integers(1, 8000))]))
        out.append((rows, cols, str(rng.choice(["bf16", "f16"])), float(rng.choice([0.1, 1.0, 3.0]))))
    return out


@pytest.mark.parametrize("rows,n,dtype,spread", _random_softmax_cases())
def test_softmax_random_shapes(rows, n, dtype, spread):
    """Seeded random shapes (row lengths with and without the 16-byte path,
    resident or read twice, split or not): every element against the oracle."""
    print(f"case softmax random {rows}x{n} {dtype} spread {spread}", flush=True)
    x = inputs.make_matrix(rows, n, dtype, seed=rows * 7 + n, spread=spread)
    tx = _gpu.upload(x, dtype)
    ty = torch.empty_like(tx)
    capi.attn_softmax(tx, ty)
    torch.cuda.synchronize()
    ref = SM.softmax_rows(inputs.bits_to_f64(x, dtype))
    _check(_gpu.download(ty, dtype), ref, dtype, f"random {rows}x{n}")
