"""The forward entry points captured into a HIP graph and replayed.

A serving loop captures the call once and replays it with new contents in
the same buffers.  Each case runs one call on a side stream first (for
attn_fwd that sizes the stream's split workspace, which may not grow under
capture), captures the call on that stream, then replays the graph four
times with alternating inputs copied into the captured buffers and the
output refilled with NaN, with the program's own eager calls and a device
synchronisation between replays.  Every replay must equal, bit for bit, the
eager call on the same inputs (same plan, same kernels), and the eager
result is checked against the oracle.

Inputs come from the seeded generator; expected values from oracle/ only.
"""
import pytest

from oracle import attention as A
from paper_2609_10937_amd import capi, inputs

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import _gpu  # noqa: E402

CASES = [
    # name, B, H, L, d, causal, type
    ("split", 1, 1, 4096, 128, False, "bf16"),
    ("causal_pieces", 1, 1, 8192, 128, True, "bf16"),
    ("persistent", 1, 300, 700, 128, False, "bf16"),
    ("causal_split_f16_d64", 2, 8, 1000, 64, True, "f16"),
]


@pytest.mark.parametrize("entry", ["attn_fwd", "attn_fwd_noalloc"])
@pytest.mark.parametrize("name,B,H,L,d,causal,dtype", CASES)
def test_graph_replays_match_eager(name, B, H, L, d, causal, dtype, entry):
    fn = getattr(capi, entry)
    plan = capi.attn_fwd_plan(B, H, L, d, causal, capi.ATTN_BF16 if dtype == "bf16" else capi.ATTN_F16)
    print(f"case graph {name} {entry} B{B} H{H} L{L} d{d} causal{int(causal)} {dtype} grid {plan.grid} "
          f"launch {plan.launch_grid} splits {plan.n_split}", flush=True)
    s = inputs.softmax_scale(d)
    host = [inputs.make_qkv(B, H, L, d, dtype, seed=1401 + 17 * i + L) for i in range(2)]
    sets = [tuple(_gpu.upload(x, dtype) for x in qkv) for qkv in host]

    eager = []
    for tq, tk, tv in sets:
        o = torch.empty_like(tq)
        fn(tq, tk, tv, o, s, causal)
        eager.append(o)
    torch.cuda.synchronize()
    ref = A.attention(_gpu.download(sets[0][0], dtype), _gpu.download(sets[0][1], dtype),
                      _gpu.download(sets[0][2], dtype), s, causal)
    _gpu.assert_close(_gpu.download(eager[0], dtype), ref, dtype, f"{name} eager")

    q, k, v = (torch.empty_like(t) for t in sets[0])
    o = torch.empty_like(q)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for dst, src in zip((q, k, v), sets[0]):
            dst.copy_(src)
        fn(q, k, v, o, s, causal)
    side.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        fn(q, k, v, o, s, causal)
    torch.cuda.synchronize()

    other = torch.empty_like(q)
    for rep in range(4):
        src = sets[rep % 2]
        for dst, x in zip((q, k, v), src):
            dst.copy_(x)
        o.fill_(float("nan"))
        g.replay()
        # eager work of the program between replays
        fn(*sets[(rep + 1) % 2], other, s, causal)
        torch.cuda.synchronize()
        assert torch.equal(o.view(torch.int16), eager[rep % 2].view(torch.int16)), f"replay {rep} differs"
        assert torch.equal(other.view(torch.int16), eager[(rep + 1) % 2].view(torch.int16))
    del g
    torch.cuda.synchronize()


def test_capture_refuses_to_grow_the_workspace():
    """A split call captured on a stream that has no workspace yet must not
    allocate under capture: attn_fwd returns ATTN_E_WORKSPACE and records
    nothing; after the capture ends the same call runs eagerly and matches
    the call on the default stream."""
    import ctypes
    hip = ctypes.CDLL("libamdhip64.so")
    hip.hipStreamBeginCapture.argtypes = [ctypes.c_void_p, ctypes.c_int]
    hip.hipStreamEndCapture.argtypes = [ctypes.c_void_p, ctypes.POINTER(ctypes.c_void_p)]
    hip.hipGraphDestroy.argtypes = [ctypes.c_void_p]
    hip.hipStreamCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
    hip.hipStreamSynchronize.argtypes = [ctypes.c_void_p]
    hip.hipStreamDestroy.argtypes = [ctypes.c_void_p]
    B, H, L, d, dtype = 1, 1, 4096, 128, "bf16"
    assert capi.attn_fwd_plan(B, H, L, d, False, capi.ATTN_BF16).n_split > 1
    print(f"case graph capture refusal B{B} H{H} L{L} d{d}", flush=True)
    s = inputs.softmax_scale(d)
    tq, tk, tv = (_gpu.upload(x, dtype) for x in inputs.make_qkv(B, H, L, d, dtype, seed=1451))
    o_ref = torch.empty_like(tq)
    capi.attn_fwd(tq, tk, tv, o_ref, s, False)
    torch.cuda.synchronize()
    # a stream of its own (torch's streams come from a pool that earlier
    # calls may have used, and their workspaces would already fit)
    handle = ctypes.c_void_p()
    assert hip.hipStreamCreate(ctypes.byref(handle)) == 0
    fresh = handle.value
    try:
        o = torch.full_like(tq, float("nan"))
        torch.cuda.synchronize()
        assert hip.hipStreamBeginCapture(fresh, 0) == 0  # global capture mode
        try:
            with pytest.raises(capi.AttnError) as e:
                capi.attn_fwd(tq, tk, tv, o, s, False, stream=fresh)
        finally:
            graph = ctypes.c_void_p()
            end = hip.hipStreamEndCapture(fresh, ctypes.byref(graph))
        assert end == 0
        if graph.value:
            hip.hipGraphDestroy(graph)
        assert e.value.status == capi.CODE["ATTN_E_WORKSPACE"]
        capi.attn_fwd(tq, tk, tv, o, s, False, stream=fresh)
        assert hip.hipStreamSynchronize(fresh) == 0
        assert torch.equal(o.view(torch.int16), o_ref.view(torch.int16))
    finally:
        torch.cuda.synchronize()
        hip.hipStreamDestroy(fresh)
