"""Helpers for the GPU tests: upload seeded inputs, run through the C ABI, compare."""
import numpy as np

from paper_2609_10937_amd import capi, inputs

# Parity bar: element-wise against the float64 oracle (max-abs, mean-abs).
TOL = {"bf16": (2e-2, 2e-3), "f16": (1e-2, 1e-3)}


def torch_dtype(dtype):
    import torch
    return torch.bfloat16 if dtype == "bf16" else torch.float16


def upload(bits, dtype):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to("cuda").view(torch_dtype(dtype))


def download(t, dtype):
    import torch
    return inputs.bits_to_f64(t.view(torch.int16).cpu().numpy().view(np.uint16), dtype)


def fused(q, k, v, scale, causal):
    import torch
    o = torch.empty_like(q)
    capi.attn_fwd(q, k, v, o, scale, causal)
    torch.cuda.synchronize()
    return o


def errors(got, ref):
    e = np.abs(got - ref)
    return float(e.max()), float(e.mean())


def assert_close(got, ref, dtype, what=""):
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    mx, mn = errors(got, ref)
    tmax, tmean = TOL[dtype]
    assert mx <= tmax and mn <= tmean, f"{what}: max_abs {mx:.3e} (<= {tmax}), mean_abs {mn:.3e} (<= {tmean})"
    return mx, mn
