"""GPU parity at the size limits of the forward entry point.

* Tensors past 4 GiB (more than 2^31 elements): heads whose byte offsets no
  32-bit integer holds, through the plain launch and through the persistent
  one, at every head dimension (bf16, and f16 at d = 64).  Every head copies
  one of seven seeded base heads (head f takes base f mod 7; no power of two
  is a multiple of 7, so the heads 2^k apart that a wrapped 32-bit offset
  would confuse hold different data).  The kernel's arithmetic for a
  head does not depend on where the head sits, so every head's output must
  equal its base's bit for bit, and the seven bases are compared row by row
  with the float64 oracle: all rows of all heads are checked.
* A million-token sequence (L = 2^20 + 77): sampled rows against the oracle
  and every row inside the range of the values it averages.

Inputs come from the seeded generator; expected values from oracle/ only.
"""
import numpy as np
import pytest

from oracle import attention as A
from paper_2609_10937_amd import capi, inputs

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import _gpu  # noqa: E402

N_BASE = 7


def _f64(bits, dtype):
    return inputs.bits_to_f64(bits, dtype)


BEYOND_4GIB = [
    # B, H, L, d, causal, type, persistent launch expected
    (2, 2050, 4096, 128, False, "bf16", False),
    (2, 2050, 4096, 128, True, "bf16", False),
    (1, 32800, 512, 128, False, "bf16", True),
    (4, 8200, 512, 128, True, "bf16", True),
    (2, 4100, 4096, 64, True, "f16", False),
    (1, 65600, 512, 64, False, "f16", True),
    (2, 1030, 4096, 256, False, "bf16", False),
    (2, 2740, 4096, 96, True, "bf16", False),
]


@pytest.mark.parametrize("B,H,L,d,causal,dtype,persistent", BEYOND_4GIB)
def test_tensors_beyond_4gib_all_heads(B, H, L, d, causal, dtype, persistent):
    BH = B * H
    assert BH * L * d > 1 << 31
    plan = capi.attn_fwd_plan(B, H, L, d, causal, capi.ATTN_BF16 if dtype == "bf16" else capi.ATTN_F16)
    assert plan.n_split == 1
    assert (plan.launch_grid < plan.grid) == persistent
    print(f"case beyond_4gib B{B} H{H} L{L} d{d} causal{int(causal)} {dtype} grid {plan.grid} "
          f"launch {plan.launch_grid}", flush=True)
    q, k, v = inputs.make_qkv(1, N_BASE, L, d, dtype, seed=1301 + L + d + int(causal))
    idx = torch.arange(BH, device="cuda") % N_BASE
    tq, tk, tv = (_gpu.upload(x, dtype)[0][idx].view(B, H, L, d) for x in (q, k, v))
    o = torch.full_like(tq, float("nan"))
    s = inputs.softmax_scale(d)
    capi.attn_fwd(tq, tk, tv, o, s, causal)
    torch.cuda.synchronize()
    del tq, tk, tv
    of = o.view(BH, L, d).view(torch.int16)
    for r in range(N_BASE):
        assert torch.equal(of[r::N_BASE], of[r].expand(of[r::N_BASE].shape)), f"heads of base {r} differ"
    # the heads on either side of the first one past 2^31 elements (2^32
    # bytes) and the last head, compared with the oracle directly: their
    # inputs are those of base f mod 7
    hb = (1 << 31) // (L * d)
    far = [hb - 1, hb, hb + 1, BH - 1]
    got = _gpu.download(o.view(BH, L, d)[:N_BASE], dtype)
    got_far = _gpu.download(o.view(BH, L, d)[torch.tensor(far, device="cuda")], dtype)
    del o, of
    torch.cuda.empty_cache()
    ref = A.attention(_f64(q, dtype), _f64(k, dtype), _f64(v, dtype), s, causal)[0]
    mx, mn = _gpu.assert_close(got, ref, dtype, "beyond 4 GiB")
    _gpu.assert_close(got_far, ref[[f % N_BASE for f in far]], dtype, f"heads {far}")
    print(f"  max_abs {mx:.3e} mean_abs {mn:.3e} over {N_BASE} base heads; heads {far} checked too", flush=True)


@pytest.mark.parametrize("causal", [False, True])
def test_million_token_sequence_sampled_rows(causal):
    d, dtype = 128, "bf16"
    L = (1 << 20) + 77
    plan = capi.attn_fwd_plan(1, 1, L, d, causal, capi.ATTN_BF16)
    print(f"case long_sequence L{L} d{d} causal{int(causal)} grid {plan.grid} splits {plan.n_split}",
          flush=True)
    q, k, v = inputs.make_qkv(1, 1, L, d, dtype, seed=1311 + int(causal))
    tq, tk, tv = (_gpu.upload(x, dtype) for x in (q, k, v))
    o = torch.full_like(tq, float("nan"))
    s = inputs.softmax_scale(d)
    capi.attn_fwd(tq, tk, tv, o, s, causal)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([np.arange(0, 24), np.arange(L - 24, L),
                                     np.random.default_rng(1313).integers(0, L, 48),
                                     [255, 256, 257, (1 << 19) - 1, 1 << 19, (1 << 20) - 1, 1 << 20]]))
    got = _gpu.download(o[0, 0, torch.from_numpy(rows).to("cuda")], dtype)
    ref = A.attention_head(_f64(q[0, 0], dtype), _f64(k[0, 0], dtype), _f64(v[0, 0], dtype), s, causal,
                           rows=rows)
    mx, mn = _gpu.assert_close(got, ref, dtype, "long sequence")
    print(f"  max_abs {mx:.3e} mean_abs {mn:.3e} over {rows.size} rows", flush=True)
    of = o.float()[0, 0]
    vf = tv.float()[0, 0]
    assert torch.isfinite(of).all()
    if causal:
        vmax = torch.cummax(vf, dim=0).values
        vmin = -torch.cummax(-vf, dim=0).values
    else:
        vmax = vf.max(dim=0, keepdim=True).values
        vmin = vf.min(dim=0, keepdim=True).values
    slack = 2e-2
    assert (of <= vmax + slack).all() and (of >= vmin - slack).all()
