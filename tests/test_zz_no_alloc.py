"""attn_fwd_noalloc (split workspace in the library's static per-GPU array,
no allocation) against attn_fwd through the C ABI: two calls in a row, the
second with a smaller input, each bit for bit equal to attn_fwd and within
the parity bar of the float64 oracle; a shape whose split workspace exceeds
the array is refused before any device work."""
import numpy as np
import pytest

from oracle import attention as A
from paper_2609_10937_amd import capi, inputs

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import _gpu  # noqa: E402


def _run_both(w):
    q, k, v = inputs.workload_inputs(w)
    t = [_gpu.upload(x, w.dtype) for x in (q, k, v)]
    ref_o = _gpu.fused(t[0], t[1], t[2], w.scale, w.causal)
    o = torch.full_like(t[0], float("nan"))
    capi.attn_fwd_noalloc(t[0], t[1], t[2], o, w.scale, w.causal)
    torch.cuda.synchronize()
    return (q, k, v), ref_o, o


def test_noalloc_matches_attn_fwd_two_calls():
    first = inputs.WORKLOADS["single_head_l16384_d128"]   # 4 key splits
    second = inputs.WORKLOADS["sweep_l8192_d128"]         # smaller input, 8 key splits
    for w in (first, second):
        dt = capi.ATTN_BF16 if w.dtype == "bf16" else capi.ATTN_F16
        nb = capi.attn_fwd_workspace_bytes(w.B, w.H, w.L, w.d, w.causal, dt)
        assert 0 < nb <= capi.NOALLOC_SCRATCH_BYTES
        print(f"case noalloc {w.name} workspace {nb} bytes", flush=True)
        (q, k, v), a, b = _run_both(w)
        assert torch.equal(a.view(torch.int16), b.view(torch.int16)), w.name
        rows = np.unique(np.concatenate([np.arange(48), np.arange(w.L - 48, w.L),
                                         np.random.default_rng(11).integers(0, w.L, 160)]))
        got = _gpu.download(b[0, 0, torch.from_numpy(rows).to("cuda")], w.dtype)
        ref = A.attention_head(inputs.bits_to_f64(q[0, 0], w.dtype), inputs.bits_to_f64(k[0, 0], w.dtype),
                               inputs.bits_to_f64(v[0, 0], w.dtype), w.scale, w.causal, rows=rows)
        _gpu.assert_close(got, ref, w.dtype, f"noalloc {w.name}")


def test_noalloc_without_split_and_refusal():
    w = inputs.WORKLOADS["tiny_f16_l128_d64"]
    print(f"case noalloc {w.name} (no split)", flush=True)
    _, a, b = _run_both(w)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    # no split, a persistent launch
    w = inputs.WORKLOADS["heads1024_l512_d128"]
    plan = capi.attn_fwd_plan(w.B, w.H, w.L, w.d, w.causal, capi.ATTN_BF16)
    assert plan.launch_grid < plan.grid
    print(f"case noalloc {w.name} (persistent)", flush=True)
    _, a, b = _run_both(w)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    # one head, L = 20000, d = 96: 9 key splits, 36.0 MB of partials
    B, H, L, d = 1, 1, 20000, 96
    nb = capi.attn_fwd_workspace_bytes(B, H, L, d, False, capi.ATTN_BF16)
    assert nb > capi.NOALLOC_SCRATCH_BYTES
    print(f"case noalloc refusal B{B} H{H} L{L} d{d} workspace {nb} bytes", flush=True)
    t = torch.zeros((B, H, L, d), dtype=torch.bfloat16, device="cuda")
    o = torch.zeros_like(t)
    with pytest.raises(capi.AttnError) as e:
        capi.attn_fwd_noalloc(t, t, t, o, inputs.softmax_scale(d), False)
    assert e.value.status == capi.CODE["ATTN_E_SCRATCH"]
    torch.cuda.synchronize()
    assert not torch.any(o.view(torch.int16))  # refused before any device work
