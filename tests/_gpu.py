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


def oracle_heads_parallel(q64_of, k64_of, v64_of, heads, scale, causal, consume, workers=16):
    """Evaluate the float64 oracle for each (b, h) in `heads` on a pool of
    threads (numpy and BLAS release the GIL; BLAS itself is held to one thread
    per worker) and hand each head's result to consume(b, h, ref) as it
    completes.  q64_of(b, h) etc. return one head's inputs as float64."""
    import concurrent.futures as cf

    from threadpoolctl import threadpool_limits

    from oracle import attention as A

    def one(bh):
        b, h = bh
        return b, h, A.attention_head(q64_of(b, h), k64_of(b, h), v64_of(b, h), scale, causal, block_rows=256)

    with threadpool_limits(1), cf.ThreadPoolExecutor(workers) as ex:
        for b, h, ref in ex.map(one, heads):
            consume(b, h, ref)
