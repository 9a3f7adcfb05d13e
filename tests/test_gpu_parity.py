"""GPU parity of the fused kernel (and the unfused baseline) with the CPU oracle.

Every case prints its name before touching the GPU so a failure is
attributable.  Inputs come from the seeded generator; expected values from
oracle/ only.
"""
import numpy as np
import pytest

from oracle import attention as A
from paper_2609_10937_amd import capi, inputs

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import _gpu  # noqa: E402


def _f64(bits, dtype):
    return inputs.bits_to_f64(bits, dtype)


# ------------------------------------------------------------ matrix-core layout

@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_mfma_fragment_layouts(dtype):
    """Random small-integer operands: A B is exact in fp32, so C must match bit for bit."""
    print(f"case mfma_probe {dtype}", flush=True)
    rng = np.random.default_rng(5)
    a = rng.integers(-8, 9, size=(16, 32)).astype(np.float32)
    b = rng.integers(-8, 9, size=(32, 16)).astype(np.float32)
    ta = _gpu.upload(inputs.round_bits(a, dtype), dtype)
    tb = _gpu.upload(inputs.round_bits(b, dtype), dtype)
    tc = torch.zeros((16, 16), dtype=torch.float32, device="cuda")
    capi.attn_mfma_probe(0 if dtype == "bf16" else 1, ta, tb, tc)
    torch.cuda.synchronize()
    assert np.array_equal(tc.cpu().numpy(), a @ b)


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_paper_structured_layout_case(dtype):
    """Section 3.1: Q[i,:] = i and K = I give C[i,:] = i; in the transposed
    product the kernel uses (K Q^T) the same data gives C[:, j] = j."""
    print(f"case mfma_structured {dtype}", flush=True)
    q = np.repeat(np.arange(16, dtype=np.float32)[:, None], 32, axis=1)   # Q[i, :] = i
    eye = np.zeros((16, 32), np.float32)
    eye[:, :16] = np.eye(16)                                              # K = I (first 16 of d)
    tc = torch.zeros((16, 16), dtype=torch.float32, device="cuda")
    atom = 0 if dtype == "bf16" else 1
    capi.attn_mfma_probe(atom, _gpu.upload(inputs.round_bits(q, dtype), dtype),
                         _gpu.upload(inputs.round_bits(np.ascontiguousarray(eye.T), dtype), dtype), tc)
    torch.cuda.synchronize()
    assert np.array_equal(tc.cpu().numpy(), np.repeat(np.arange(16, dtype=np.float32)[:, None], 16, axis=1))
    capi.attn_mfma_probe(atom, _gpu.upload(inputs.round_bits(eye, dtype), dtype),
                         _gpu.upload(inputs.round_bits(np.ascontiguousarray(q.T), dtype), dtype), tc)
    torch.cuda.synchronize()
    assert np.array_equal(tc.cpu().numpy(), np.repeat(np.arange(16, dtype=np.float32)[None, :], 16, axis=0))


# ------------------------------------------------------------ named workloads

SMALL = ["tiny_f16_l128_d64", "h8_l1024_d128", "causal_b2h16_l4096_d128_kx3", "single_head_l16384_d128",
         "sweep_l4096_d128", "sweep_l8192_d128"]


@pytest.mark.parametrize("name", SMALL)
def test_workload_all_rows(name):
    w = inputs.WORKLOADS[name]
    print(f"case workload {name}", flush=True)
    q, k, v = inputs.workload_inputs(w)
    o = _gpu.fused(_gpu.upload(q, w.dtype), _gpu.upload(k, w.dtype), _gpu.upload(v, w.dtype), w.scale, w.causal)
    got = _gpu.download(o, w.dtype)
    ref = A.attention(_f64(q, w.dtype), _f64(k, w.dtype), _f64(v, w.dtype), w.scale, w.causal)
    mx, mn = _gpu.assert_close(got, ref, w.dtype, name)
    floor = np.abs(_f64(inputs.round_bits(ref.astype(np.float32), w.dtype), w.dtype) - ref).max()
    print(f"  {name}: max_abs {mx:.3e} mean_abs {mn:.3e} (rounding floor {floor:.3e})", flush=True)


@pytest.mark.timeout(900)
def test_full_occupancy_causal_all_rows():
    """B=4, H=32, L=16384 causal (the full-occupancy workload, in the launch
    configuration bench.py times): every one of its 2,097,152 rows against the
    float64 oracle, evaluated head by head on a thread pool."""
    w = inputs.WORKLOADS["causal_b4h32_l16384_d128"]
    print(f"case workload {w.name} (all rows)", flush=True)
    q, k, v = inputs.workload_inputs(w)
    tq, tk, tv = (_gpu.upload(x, w.dtype) for x in (q, k, v))
    o = _gpu.fused(tq, tk, tv, w.scale, w.causal)
    got_bits = o.view(torch.int16).cpu().numpy().view(np.uint16)
    del tq, tk, tv, o
    torch.cuda.empty_cache()
    stats = {"max": 0.0, "sum": 0.0, "n": 0, "finite": True}

    def consume(b, h, ref):
        got = _f64(got_bits[b, h], w.dtype)
        e = np.abs(got - ref)
        stats["finite"] &= bool(np.all(np.isfinite(got)))
        stats["max"] = max(stats["max"], float(e.max()))
        stats["sum"] += float(e.sum())
        stats["n"] += e.size

    heads = [(b, h) for b in range(w.B) for h in range(w.H)]
    _gpu.oracle_heads_parallel(lambda b, h: _f64(q[b, h], w.dtype), lambda b, h: _f64(k[b, h], w.dtype),
                               lambda b, h: _f64(v[b, h], w.dtype), heads, w.scale, True, consume)
    mean = stats["sum"] / stats["n"]
    print(f"  {w.name}: {stats['n'] // w.d} rows, max_abs {stats['max']:.3e} mean_abs {mean:.3e}", flush=True)
    assert stats["n"] == w.B * w.H * w.L * w.d and stats["finite"]
    tmax, tmean = _gpu.TOL[w.dtype]
    assert stats["max"] <= tmax and mean <= tmean


def test_sweep_l32768_sampled_rows():
    """The longest point of the sequence-length sweep (B=H=1, L=32768, d=128):
    sampled rows against the oracle, and every row inside the range of V."""
    w = inputs.WORKLOADS["sweep_l32768_d128"]
    print(f"case workload {w.name} (sampled)", flush=True)
    q, k, v = inputs.workload_inputs(w)
    tq, tk, tv = (_gpu.upload(x, w.dtype) for x in (q, k, v))
    o = _gpu.fused(tq, tk, tv, w.scale, w.causal)
    L = w.L
    rows = np.unique(np.concatenate([np.arange(0, 40), np.arange(L - 40, L),
                                     np.random.default_rng(78).integers(0, L, 160),
                                     [255, 256, 257, 8191, 8192, 16383, 16384]]))
    got = _gpu.download(o[0, 0, torch.from_numpy(rows).to("cuda")], w.dtype)
    ref = A.attention_head(_f64(q[0, 0], w.dtype), _f64(k[0, 0], w.dtype), _f64(v[0, 0], w.dtype),
                           w.scale, False, rows=rows)
    mx, mn = _gpu.assert_close(got, ref, w.dtype, w.name)
    print(f"  {w.name}: max_abs {mx:.3e} mean_abs {mn:.3e} over {rows.size} rows", flush=True)
    of = o.float()[0, 0]
    vf = tv.float()[0, 0]
    assert torch.isfinite(of).all()
    slack = 2e-2
    assert (of <= vf.max(dim=0).values + slack).all() and (of >= vf.min(dim=0).values - slack).all()


@pytest.mark.parametrize("name", [w.name for w in inputs.HEAD_DIM_64 + inputs.HEAD_DIM_96 + inputs.HEAD_DIM_256])
def test_head_dim_workloads_sampled_rows(name):
    """The head-dimension workloads the benchmark times, at their full sizes:
    sampled heads and rows against the oracle, and every row inside the range
    of V (the running range for causal rows)."""
    w = inputs.WORKLOADS[name]
    print(f"case workload {w.name} (sampled)", flush=True)
    q, k, v = inputs.workload_inputs(w)
    tq, tk, tv = (_gpu.upload(x, w.dtype) for x in (q, k, v))
    o = _gpu.fused(tq, tk, tv, w.scale, w.causal)
    L = w.L
    rng = np.random.default_rng(w.seed)
    heads = [(0, 0)] if w.B * w.H == 1 else [(0, 0), (w.B - 1, w.H - 1), (1, w.H // 2)]
    for b, h in heads:
        rows = np.unique(np.concatenate([np.arange(0, 24), np.arange(L - 24, L),
                                         rng.integers(0, L, 64), [255, 256, 257, 8191, 8192]]))
        got = _gpu.download(o[b, h, torch.from_numpy(rows).to("cuda")], w.dtype)
        ref = A.attention_head(_f64(q[b, h], w.dtype), _f64(k[b, h], w.dtype), _f64(v[b, h], w.dtype),
                               w.scale, w.causal, rows=rows)
        mx, mn = _gpu.assert_close(got, ref, w.dtype, f"{w.name} b{b} h{h}")
        print(f"  {w.name} b{b} h{h}: max_abs {mx:.3e} mean_abs {mn:.3e} over {rows.size} rows", flush=True)
    of = o.float()
    vf = tv.float()
    assert torch.isfinite(of).all()
    slack = 2e-2
    if w.causal:
        vmax = torch.cummax(vf, dim=2).values
        vmin = -torch.cummax(-vf, dim=2).values
    else:
        vmax = vf.max(dim=2, keepdim=True).values
        vmin = vf.min(dim=2, keepdim=True).values
    assert (of <= vmax + slack).all() and (of >= vmin - slack).all()


# ------------------------------------------------------------ edge shapes

EDGE = [(L, d, causal, dt) for L in (1, 17, 100, 1000, 4097) for d in (64, 96, 128, 256)
        for causal in (False, True) for dt in ("bf16", "f16")]


@pytest.mark.parametrize("L,d,dtype", [(16384, 128, "bf16"), (8192, 128, "f16"), (6000, 128, "bf16"),
                                       (16384, 64, "bf16"), (16384, 96, "bf16"), (16384, 256, "f16"),
                                       (9000, 96, "bf16"), (20000, 128, "bf16"), (3000, 256, "bf16")])
def test_causal_pieces_all_rows(L, d, dtype):
    """Causal single heads, split as pieces of each query tile's own key range
    (only non-empty pieces launched, heaviest query tiles first; the merge
    reads as many slots per row as the row's query tile has pieces): all rows
    against the oracle."""
    dt = capi.ATTN_BF16 if dtype == "bf16" else capi.ATTN_F16
    plan = capi.attn_fwd_plan(1, 1, L, d, True, dt)
    n_qt = -(-L // plan.tile_q)
    assert plan.n_split > 1 and plan.tile_q % plan.t_kv == 0 and plan.grid < n_qt * plan.n_split
    print(f"case causal pieces L{L} d{d} {dtype}: {plan.tiles_per_split} key tiles per piece, "
          f"{plan.n_split} slots, {plan.grid} workgroups", flush=True)
    q, k, v = inputs.make_qkv(1, 1, L, d, dtype, seed=3 * L + d)
    scale = inputs.softmax_scale(d)
    o = _gpu.fused(_gpu.upload(q, dtype), _gpu.upload(k, dtype), _gpu.upload(v, dtype), scale, True)
    ref = A.attention(_f64(q, dtype), _f64(k, dtype), _f64(v, dtype), scale, True)
    mx, mn = _gpu.assert_close(_gpu.download(o, dtype), ref, dtype, f"causal pieces L{L} d{d}")
    print(f"  max_abs {mx:.3e} mean_abs {mn:.3e}", flush=True)


@pytest.mark.parametrize("H,L,d,dtype", [(16, 4096, 128, "bf16"), (8, 8192, 128, "f16"), (4, 16384, 64, "bf16")])
def test_causal_halves_all_rows(H, L, d, dtype):
    """Causal launches that fill one round of CUs unsplit, run as halves of each
    query tile's own key range over two rounds (piece-major order): all rows
    of every head against the oracle."""
    dt = capi.ATTN_BF16 if dtype == "bf16" else capi.ATTN_F16
    plan = capi.attn_fwd_plan(1, H, L, d, True, dt)
    n_qt = -(-L // plan.tile_q)
    assert plan.n_split == 2 and 256 < plan.grid < H * n_qt * 2
    print(f"case causal halves H{H} L{L} d{d} {dtype}: {plan.grid} workgroups", flush=True)
    q, k, v = inputs.make_qkv(1, H, L, d, dtype, seed=5 * L + H)
    scale = inputs.softmax_scale(d)
    o = _gpu.fused(_gpu.upload(q, dtype), _gpu.upload(k, dtype), _gpu.upload(v, dtype), scale, True)
    ref = A.attention(_f64(q, dtype), _f64(k, dtype), _f64(v, dtype), scale, True)
    mx, mn = _gpu.assert_close(_gpu.download(o, dtype), ref, dtype, f"causal halves H{H} L{L} d{d}")
    print(f"  max_abs {mx:.3e} mean_abs {mn:.3e}", flush=True)


@pytest.mark.parametrize("L,d,causal,dtype", [(10000, 128, False, "bf16"), (10000, 128, True, "f16"),
                                               (9000, 96, False, "bf16")])
def test_split_counts_not_powers_of_two(L, d, causal, dtype):
    """Single heads whose derived key split is not a power of two (the merge
    then reads its split count at run time): all rows against the oracle."""
    dt = capi.ATTN_BF16 if dtype == "bf16" else capi.ATTN_F16
    plan = capi.attn_fwd_plan(1, 1, L, d, causal, dt)
    assert plan.n_split > 1 and plan.n_split & (plan.n_split - 1)
    print(f"case split L{L} d{d} causal{int(causal)} {dtype} n_split {plan.n_split}", flush=True)
    q, k, v = inputs.make_qkv(1, 1, L, d, dtype, seed=L + d)
    scale = inputs.softmax_scale(d)
    o = _gpu.fused(_gpu.upload(q, dtype), _gpu.upload(k, dtype), _gpu.upload(v, dtype), scale, causal)
    ref = A.attention(_f64(q, dtype), _f64(k, dtype), _f64(v, dtype), scale, causal)
    _gpu.assert_close(_gpu.download(o, dtype), ref, dtype, f"split L{L} d{d}")


@pytest.mark.parametrize("L,d,causal,dtype", EDGE)
def test_edge_shapes(L, d, causal, dtype):
    B, H = (2, 3) if L <= 1000 else (1, 2)
    print(f"case edge L{L} d{d} causal{int(causal)} {dtype}", flush=True)
    q, k, v = inputs.make_qkv(B, H, L, d, dtype, seed=L * 7 + d, k_scale=2.0)
    scale = inputs.softmax_scale(d)
    o = _gpu.fused(_gpu.upload(q, dtype), _gpu.upload(k, dtype), _gpu.upload(v, dtype), scale, causal)
    ref = A.attention(_f64(q, dtype), _f64(k, dtype), _f64(v, dtype), scale, causal)
    _gpu.assert_close(_gpu.download(o, dtype), ref, dtype, f"L{L} d{d} c{causal} {dtype}")


@pytest.mark.parametrize("B,H,L,causal,dtype", [(1, 4, 2048, False, "bf16"), (2, 2, 3000, True, "f16"),
                                                 (1, 1, 8192, False, "bf16")])
def test_head_dim_256_all_rows(B, H, L, causal, dtype):
    """d = 256 (t_kv = 32, 16 rows per wave): all rows against the oracle; the
    single-head case runs with split key ranges, the L = 3000 case has a ragged
    tail tile."""
    print(f"case d256 B{B} H{H} L{L} causal{int(causal)} {dtype}", flush=True)
    q, k, v = inputs.make_qkv(B, H, L, 256, dtype, seed=L + 256)
    s = inputs.softmax_scale(256)
    o = _gpu.fused(_gpu.upload(q, dtype), _gpu.upload(k, dtype), _gpu.upload(v, dtype), s, causal)
    ref = A.attention(_f64(q, dtype), _f64(k, dtype), _f64(v, dtype), s, causal)
    mx, mn = _gpu.assert_close(_gpu.download(o, dtype), ref, dtype, f"d256 L{L}")
    print(f"  d256 L{L}: max_abs {mx:.3e} mean_abs {mn:.3e}", flush=True)


# (B, H, L, causal, dtype) -> the (rows per wave, waves) instance the derivation picks
D96 = [((2, 8, 2048, True, "bf16"), (48, 8)), ((1, 4, 1000, False, "f16"), (48, 4)),
       ((1, 2, 1000, True, "bf16"), (48, 2)), ((4, 32, 63, False, "bf16"), (48, 1)),
       ((2, 8, 161, True, "f16"), (32, 1)), ((1, 1, 100, False, "bf16"), (16, 1)),
       ((1, 1, 8192, False, "bf16"), (48, 8))]


@pytest.mark.parametrize("case,instance", D96)
def test_head_dim_96_all_rows(case, instance):
    """d = 96 (t_kv = 64, K/V rows padded to 128 elements in LDS): all rows
    against the oracle, one case per compiled instance; the single-head case
    runs with 16 key-range splits."""
    B, H, L, causal, dtype = case
    r = capi.attn_fwd_plan(B, H, L, 96, causal, capi.ATTN_BF16 if dtype == "bf16" else capi.ATTN_F16)
    assert (r.t_q_wave, r.n_waves) == instance
    print(f"case d96 B{B} H{H} L{L} causal{int(causal)} {dtype} instance {instance}", flush=True)
    q, k, v = inputs.make_qkv(B, H, L, 96, dtype, seed=L + 96)
    s = inputs.softmax_scale(96)
    o = _gpu.fused(_gpu.upload(q, dtype), _gpu.upload(k, dtype), _gpu.upload(v, dtype), s, causal)
    ref = A.attention(_f64(q, dtype), _f64(k, dtype), _f64(v, dtype), s, causal)
    mx, mn = _gpu.assert_close(_gpu.download(o, dtype), ref, dtype, f"d96 L{L}")
    print(f"  d96 L{L}: max_abs {mx:.3e} mean_abs {mn:.3e}", flush=True)


@pytest.mark.parametrize("causal", [False, True])
def test_many_heads_small_l(causal):
    """B*H large enough that the grid covers the CUs without splitting."""
    print(f"case many_heads causal{int(causal)}", flush=True)
    q, k, v = inputs.make_qkv(8, 40, 200, 128, "bf16", seed=91)
    s = inputs.softmax_scale(128)
    o = _gpu.fused(_gpu.upload(q, "bf16"), _gpu.upload(k, "bf16"), _gpu.upload(v, "bf16"), s, causal)
    ref = A.attention(_f64(q, "bf16"), _f64(k, "bf16"), _f64(v, "bf16"), s, causal)
    _gpu.assert_close(_gpu.download(o, "bf16"), ref, "bf16", "many heads")


PERSISTENT = [
    (1, 300, 700, 128, False, "bf16"),  # plain order, a ragged last query tile (rows 700..767 dropped)
    (2, 160, 512, 64, False, "f16"),    # d = 64
    (1, 520, 256, 128, True, "bf16"),   # causal query tiles of exactly 4 key tiles: switches 4 steps apart
    (1, 288, 1024, 128, True, "f16"),   # causal, 4 to 16 key tiles per query tile
    (4, 64, 512, 128, False, "bf16"),   # the XCD-grouped order
]


@pytest.mark.parametrize("B,H,L,d,causal,dtype", PERSISTENT)
def test_persistent_launch_all_rows(B, H, L, d, causal, dtype):
    """Plans that run as a persistent launch (one workgroup per CU taking a
    fixed list of query tiles back to back): every row against the oracle,
    into an output first filled with NaN, so that a row no workgroup wrote
    fails."""
    import torch
    dt = capi.ATTN_BF16 if dtype == "bf16" else capi.ATTN_F16
    plan = capi.attn_fwd_plan(B, H, L, d, causal, dt)
    assert plan.launch_grid < plan.grid, "shape expected to run persistent"
    print(f"case persistent B{B} H{H} L{L} d{d} causal{int(causal)} {dtype} grid {plan.grid} "
          f"launch {plan.launch_grid}", flush=True)
    q, k, v = inputs.make_qkv(B, H, L, d, dtype, seed=L * 7 + H)
    s = inputs.softmax_scale(d)
    tq, tk, tv = (_gpu.upload(x, dtype) for x in (q, k, v))
    o = torch.full_like(tq, float("nan"))
    capi.attn_fwd(tq, tk, tv, o, s, causal)
    torch.cuda.synchronize()
    ref = A.attention(_f64(q, dtype), _f64(k, dtype), _f64(v, dtype), s, causal)
    _gpu.assert_close(_gpu.download(o, dtype), ref, dtype, "persistent")


def _persistent_random_cases(n=12, seed=4242):
    """Seeded shapes whose plans run persistent: d = 64 or 128, causal or not,
    either type, L from 200 to 1600 (ragged last query tiles included), and
    enough heads for 260 to 700 query tiles (planned on the gfx950 preset)."""
    rng = np.random.default_rng(seed)
    hw = capi.attn_hw_desc_preset("gfx950")
    out = []
    while len(out) < n:
        d = int(rng.choice([64, 128]))
        causal = bool(rng.integers(0, 2))
        dtype = str(rng.choice(["bf16", "f16"]))
        L = int(rng.integers(200, 1601))
        n_qt = -(-L // 256)
        bh = int(rng.integers(-(-260 // n_qt), 700 // n_qt + 1))
        B = int(rng.choice([1, 2])) if bh % 2 == 0 else 1
        H = bh // B
        r = capi.attn_fwd_plan(B, H, L, d, causal, capi.ATTN_BF16 if dtype == "bf16" else capi.ATTN_F16, hw=hw)
        if r.launch_grid < r.grid:
            out.append((B, H, L, d, causal, dtype))
    return out


@pytest.mark.parametrize("B,H,L,d,causal,dtype", _persistent_random_cases())
def test_persistent_random_shapes(B, H, L, d, causal, dtype):
    """Seeded persistent plans: every row against the oracle, into an output
    first filled with NaN."""
    import torch
    dt = capi.ATTN_BF16 if dtype == "bf16" else capi.ATTN_F16
    plan = capi.attn_fwd_plan(B, H, L, d, causal, dt)
    assert plan.launch_grid < plan.grid
    print(f"case persistent-random B{B} H{H} L{L} d{d} causal{int(causal)} {dtype} grid {plan.grid}", flush=True)
    q, k, v = inputs.make_qkv(B, H, L, d, dtype, seed=L * 13 + H * 3 + d)
    s = inputs.softmax_scale(d)
    tq, tk, tv = (_gpu.upload(x, dtype) for x in (q, k, v))
    o = torch.full_like(tq, float("nan"))
    capi.attn_fwd(tq, tk, tv, o, s, causal)
    torch.cuda.synchronize()
    ref = A.attention(_f64(q, dtype), _f64(k, dtype), _f64(v, dtype), s, causal)
    _gpu.assert_close(_gpu.download(o, dtype), ref, dtype, "persistent random")


def _pieces_random_cases(n=8, seed=5150):
    """Seeded causal shapes of one or two heads whose plans cut query tiles
    into pieces: every head dimension, either type, L from 2000 to 20000
    (12000 at d = 256), planned on the gfx950 preset."""
    rng = np.random.default_rng(seed)
    hw = capi.attn_hw_desc_preset("gfx950")
    out = []
    while len(out) < n:
        d = int(rng.choice([64, 96, 128, 256]))
        H = int(rng.integers(1, 3))
        L = int(rng.integers(2000, 12001 if d == 256 else 20001))
        dtype = str(rng.choice(["bf16", "f16"]))
        r = capi.attn_fwd_plan(1, H, L, d, 1, capi.ATTN_BF16 if dtype == "bf16" else capi.ATTN_F16, hw=hw)
        if r.n_split > 1 and r.grid < H * (-(-L // r.tile_q)) * r.n_split:
            out.append((H, L, d, dtype))
    return out


@pytest.mark.parametrize("H,L,d,dtype", _pieces_random_cases())
def test_causal_pieces_random_shapes(H, L, d, dtype):
    """Seeded causal-pieces plans: every row against the oracle, into an
    output first filled with NaN (a piece no workgroup ran leaves NaN)."""
    import torch
    dt = capi.ATTN_BF16 if dtype == "bf16" else capi.ATTN_F16
    plan = capi.attn_fwd_plan(1, H, L, d, True, dt)
    print(f"case pieces-random H{H} L{L} d{d} {dtype} P {plan.tiles_per_split} slots {plan.n_split} "
          f"grid {plan.grid}", flush=True)
    q, k, v = inputs.make_qkv(1, H, L, d, dtype, seed=L + 31 * d + H)
    s = inputs.softmax_scale(d)
    tq, tk, tv = (_gpu.upload(x, dtype) for x in (q, k, v))
    o = torch.full_like(tq, float("nan"))
    capi.attn_fwd(tq, tk, tv, o, s, True)
    torch.cuda.synchronize()
    ref = A.attention(_f64(q, dtype), _f64(k, dtype), _f64(v, dtype), s, True)
    _gpu.assert_close(_gpu.download(o, dtype), ref, dtype, "pieces random")


# ------------------------------------------------------------ invariants on the GPU

def test_gpu_invariants():
    print("case invariants", flush=True)
    B, H, L, d = 1, 2, 700, 128
    q, k, v = inputs.make_qkv(B, H, L, d, "bf16", seed=123)
    s = inputs.softmax_scale(d)
    tq, tk, tv = (_gpu.upload(x, "bf16") for x in (q, k, v))
    # constant V -> O equals that constant exactly (weights sum to one in fp32)
    vc = tv.clone()
    vc[:] = tv[:, :, :1, :]
    for causal in (False, True):
        o = _gpu.fused(tq, tk, vc, s, causal)
        assert torch.equal(o, vc), "constant V"
    # causal row 0 is V[0] exactly
    o = _gpu.fused(tq, tk, tv, s, True)
    assert torch.equal(o[:, :, 0], tv[:, :, 0])
    # Q = 0 (or scale 0) -> column means of V (prefix means when causal)
    vf = _f64(v, "bf16")
    mean = vf.mean(axis=2, keepdims=True)
    prefix = np.cumsum(vf, axis=2) / np.arange(1, L + 1)[None, None, :, None]
    for zq, sc in ((True, s), (False, 0.0)):
        qq = torch.zeros_like(tq) if zq else tq
        o = _gpu.download(_gpu.fused(qq, tk, tv, sc, False), "bf16")
        _gpu.assert_close(o, np.broadcast_to(mean, o.shape), "bf16", "uniform weights")
        oc = _gpu.download(_gpu.fused(qq, tk, tv, sc, True), "bf16")
        _gpu.assert_close(oc, prefix, "bf16", "uniform causal weights")


# ------------------------------------------------------------ the method's edge cases

@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("scale", [50.0, 1e4])
def test_one_hot_rows_at_huge_scale(causal, scale):
    """A huge scale makes each row's softmax one-hot on its largest logit: the
    output is that key's value row.  Rows whose runner-up logit trails by more
    than 60 in the base-2 exponent must equal V[argmax] bit for bit (their
    other weights are below 2^-60); every row matches the oracle where the
    fp32 logits are accurate enough (scale 50), and is finite and inside the
    range of the visible V rows at any scale.  One head of L = 1000 runs with
    split key ranges, so the merge sees one-hot partials too."""
    B, H, L, d = 1, 2, 1000, 128
    print(f"case one_hot scale {scale} causal{int(causal)}", flush=True)
    q, k, v = inputs.make_qkv(B, H, L, d, "bf16", seed=4242)
    assert capi.attn_fwd_plan(B, H, L, d, causal, capi.ATTN_BF16).n_split > 1
    o = _gpu.fused(_gpu.upload(q, "bf16"), _gpu.upload(k, "bf16"), _gpu.upload(v, "bf16"), scale, causal)
    got = _gpu.download(o, "bf16")
    qf, kf, vf = _f64(q, "bf16"), _f64(k, "bf16"), _f64(v, "bf16")
    assert np.all(np.isfinite(got))
    c = scale * np.log2(np.e)
    clear_rows = 0
    for b in range(B):
        for h in range(H):
            s = qf[b, h] @ kf[b, h].T
            if causal:
                s[np.triu(np.ones((L, L), bool), 1)] = -np.inf
            arg = np.argmax(s, axis=1)
            top2 = np.sort(s, axis=1)[:, -2:]
            gap = (top2[:, 1] - top2[:, 0]) * c
            clear = (gap > 60.0) | (np.arange(L) == 0) & causal
            clear_rows += int(clear.sum())
            assert np.array_equal(got[b, h][clear], vf[b, h][arg[clear]])
            if causal:
                hi = np.maximum.accumulate(vf[b, h], axis=0)
                lo = np.minimum.accumulate(vf[b, h], axis=0)
            else:
                hi, lo = vf[b, h].max(axis=0), vf[b, h].min(axis=0)
            assert np.all(got[b, h] <= hi + 1e-2) and np.all(got[b, h] >= lo - 1e-2)
    assert clear_rows >= B * H * L // 2
    if scale <= 50.0:
        ref = A.attention(qf, kf, vf, scale, causal)
        _gpu.assert_close(got, ref, "bf16", f"one-hot scale {scale}")
    print(f"  {clear_rows} of {B * H * L} rows one-hot and exact", flush=True)


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_logits_rising_on_every_tile(causal, dtype):
    """Keys whose logits grow by about 10.5 (base 2) per 64 keys, so every key
    tile carries a maximum more than 2^8 above the running reference: the
    reference is raised and the accumulated output and sums are rescaled on
    every tile (Algorithm 1's correction factor, every step), and the splits
    of the single head are merged across very different references.  All
    rows against the oracle."""
    B, H, L, d = 1, 1, 2048, 128
    scale = inputs.softmax_scale(d)
    c = scale * np.log2(np.e)
    rng = np.random.default_rng(97)
    q = rng.standard_normal((B, H, L, d)).astype(np.float32) * np.float32(0.05)
    k = rng.standard_normal((B, H, L, d)).astype(np.float32) * np.float32(0.05)
    q[..., 0] += 1.0
    k[..., 0] += (10.5 / c) * (np.arange(L, dtype=np.float32) / 64.0)
    v = rng.standard_normal((B, H, L, d)).astype(np.float32)
    qb, kb, vb = (inputs.round_bits(x, dtype) for x in (q, k, v))
    dt = capi.ATTN_BF16 if dtype == "bf16" else capi.ATTN_F16
    assert capi.attn_fwd_plan(B, H, L, d, causal, dt).n_split > 1
    print(f"case rising logits causal{int(causal)} {dtype}", flush=True)
    qf, kf = _f64(qb, dtype), _f64(kb, dtype)
    steps = np.diff(c * (qf[0, 0, :1] @ kf[0, 0].T)[0].reshape(-1, 64).max(axis=1))
    assert steps.min() > 8.0  # every tile's maximum exceeds the previous one by more than 2^8
    o = _gpu.fused(_gpu.upload(qb, dtype), _gpu.upload(kb, dtype), _gpu.upload(vb, dtype), scale, causal)
    ref = A.attention(qf, kf, _f64(vb, dtype), scale, causal)
    mx, mn = _gpu.assert_close(_gpu.download(o, dtype), ref, dtype, "rising logits")
    print(f"  rising logits: max_abs {mx:.3e} mean_abs {mn:.3e}", flush=True)


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_k_times_10_causal_with_splits(dtype):
    """K ten times wider than N(0,1), causal, one head split across key
    ranges: large, frequent jumps of the row maxima inside and across splits.
    All rows against the oracle."""
    B, H, L, d = 1, 1, 4096, 128
    dt = capi.ATTN_BF16 if dtype == "bf16" else capi.ATTN_F16
    plan = capi.attn_fwd_plan(B, H, L, d, True, dt)
    assert plan.n_split > 1
    print(f"case K x10 causal {dtype} n_split {plan.n_split}", flush=True)
    q, k, v = inputs.make_qkv(B, H, L, d, dtype, seed=1010, k_scale=10.0)
    scale = inputs.softmax_scale(d)
    o = _gpu.fused(_gpu.upload(q, dtype), _gpu.upload(k, dtype), _gpu.upload(v, dtype), scale, True)
    ref = A.attention(_f64(q, dtype), _f64(k, dtype), _f64(v, dtype), scale, True)
    mx, mn = _gpu.assert_close(_gpu.download(o, dtype), ref, dtype, "K x10")
    print(f"  K x10: max_abs {mx:.3e} mean_abs {mn:.3e}", flush=True)


# ------------------------------------------------------------ streams

def test_two_streams_without_synchronisation():
    """Two shapes that both split their key ranges, enqueued alternately on two
    streams with no synchronisation between them: each stream has its own
    workspace, so both results match the oracle and a single-stream run bit
    for bit."""
    print("case two streams", flush=True)
    shapes = [((1, 1, 8192, 128), False, "bf16", 7001), ((1, 2, 4096, 64), True, "f16", 7002)]
    data = []
    for (B, H, L, d), causal, dtype, seed in shapes:
        dt = capi.ATTN_BF16 if dtype == "bf16" else capi.ATTN_F16
        assert capi.attn_fwd_plan(B, H, L, d, causal, dt).n_split > 1
        q, k, v = inputs.make_qkv(B, H, L, d, dtype, seed=seed)
        t = [_gpu.upload(x, dtype) for x in (q, k, v)]
        data.append((t, torch.empty_like(t[0]), inputs.softmax_scale(d), causal, dtype, (q, k, v)))
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for _ in range(4):
        for (t, o, sc, causal, _, _), st in zip(data, streams):
            with torch.cuda.stream(st):
                capi.attn_fwd(t[0], t[1], t[2], o, sc, causal)
    torch.cuda.synchronize()
    for t, o, sc, causal, dtype, (q, k, v) in data:
        single = _gpu.fused(t[0], t[1], t[2], sc, causal)
        assert torch.equal(o.view(torch.int16), single.view(torch.int16))
        ref = A.attention(_f64(q, dtype), _f64(k, dtype), _f64(v, dtype), sc, causal)
        _gpu.assert_close(_gpu.download(o, dtype), ref, dtype, "two streams")


@pytest.mark.parametrize("B,H,L,d,dtype", [(1, 1, 16384, 128, "bf16"), (1, 2, 3000, 256, "f16")])
def test_partial_then_merge_equals_fused_causal_pieces(B, H, L, d, dtype):
    """Causal plans that launch pieces of each query tile's own key range: the
    caller-workspace path (attn_fwd_partial + attn_fwd_merge) equals attn_fwd
    bit for bit, the merge reading only the slots a row's query tile has."""
    dt = capi.ATTN_BF16 if dtype == "bf16" else capi.ATTN_F16
    plan = capi.attn_fwd_plan(B, H, L, d, True, dt)
    assert plan.grid < B * H * -(-L // plan.tile_q) * plan.n_split
    print(f"case partial+merge causal pieces B{B} H{H} L{L} d{d} {dtype}", flush=True)
    q, k, v = (_gpu.upload(x, dtype) for x in inputs.make_qkv(B, H, L, d, dtype, seed=L + 7))
    scale = inputs.softmax_scale(d)
    a = _gpu.fused(q, k, v, scale, True)
    nb = capi.attn_fwd_workspace_bytes(B, H, L, d, True, dt)
    ws = torch.full((nb,), 0xFF, dtype=torch.uint8, device="cuda")  # unwritten slots hold NaN bits
    b = torch.empty_like(q)
    capi.attn_fwd_partial(q, k, v, b, scale, True, ws)
    capi.attn_fwd_merge(ws, b, scale, True)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


@pytest.mark.parametrize("name", ["single_head_l16384_d128", "h8_l1024_d128", "tiny_f16_l128_d64",
                                  "heads1024_l512_d128"])
def test_partial_then_merge_equals_fused(name):
    """attn_fwd_partial + attn_fwd_merge with a caller workspace == attn_fwd, bit
    for bit (the last workload runs as a persistent launch)."""
    w = inputs.WORKLOADS[name]
    print(f"case partial+merge {name}", flush=True)
    q, k, v = (_gpu.upload(x, w.dtype) for x in inputs.workload_inputs(w))
    a = _gpu.fused(q, k, v, w.scale, w.causal)
    dt = capi.ATTN_BF16 if w.dtype == "bf16" else capi.ATTN_F16
    nb = capi.attn_fwd_workspace_bytes(w.B, w.H, w.L, w.d, w.causal, dt)
    plan = capi.attn_fwd_plan(w.B, w.H, w.L, w.d, w.causal, dt)
    assert (nb > 0) == (plan.n_split > 1)
    ws = torch.empty(max(nb, 16), dtype=torch.uint8, device="cuda") if nb else None
    b = torch.empty_like(q)
    capi.attn_fwd_partial(q, k, v, b, w.scale, w.causal, ws)
    capi.attn_fwd_merge(ws, b, w.scale, w.causal)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    if nb:
        small = torch.empty(nb - 16, dtype=torch.uint8, device="cuda")
        with pytest.raises(capi.AttnError) as e:
            capi.attn_fwd_partial(q, k, v, b, w.scale, w.causal, small)
        assert e.value.status == capi.CODE["ATTN_E_WORKSPACE"]


def test_bitwise_deterministic():
    print("case determinism", flush=True)
    w = inputs.WORKLOADS["single_head_l16384_d128"]
    q, k, v = (_gpu.upload(x, w.dtype) for x in inputs.workload_inputs(w))
    a = _gpu.fused(q, k, v, w.scale, w.causal)
    b = _gpu.fused(q, k, v, w.scale, w.causal)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


# ------------------------------------------------------------ unfused baseline

@pytest.mark.parametrize("L,causal", [(1024, False), (256, True), (1000, False), (520, True)])
def test_unfused_baseline(L, causal):
    """Scores and probabilities are stored in bf16 between the kernels, so the
    baseline is held to a looser bound than the fused kernel (it is a
    reference for time and traffic, not for accuracy)."""
    print(f"case unfused L{L} causal{int(causal)}", flush=True)
    B, H, d = 1, 8, 128
    q, k, v = inputs.make_qkv(B, H, L, d, "bf16", seed=1002)
    s = inputs.softmax_scale(d)
    tq, tk, tv = (_gpu.upload(x, "bf16") for x in (q, k, v))
    o = torch.empty_like(tq)
    ws = torch.empty(capi.attn_unfused_workspace_bytes(B, H, L, capi.ATTN_BF16), dtype=torch.uint8, device="cuda")
    capi.attn_fwd_unfused(tq, tk, tv, o, s, causal, ws)
    torch.cuda.synchronize()
    got = _gpu.download(o, "bf16")
    ref = A.attention(_f64(q, "bf16"), _f64(k, "bf16"), _f64(v, "bf16"), s, causal)
    mx, mn = _gpu.errors(got, ref)
    print(f"  unfused max_abs {mx:.3e} mean_abs {mn:.3e}", flush=True)
    assert np.all(np.isfinite(got)) and mx <= 6e-2 and mn <= 6e-3


def test_unfused_baseline_at_the_timed_size():
    """The baseline as bench.py times it (B = H = 1, L = 16384, d = 128, bf16):
    sampled rows against the oracle within the baseline's bound, every row finite."""
    w = inputs.WORKLOADS["single_head_l16384_d128"]
    print(f"case unfused {w.name} (sampled)", flush=True)
    q, k, v = inputs.workload_inputs(w)
    tq, tk, tv = (_gpu.upload(x, w.dtype) for x in (q, k, v))
    o = torch.empty_like(tq)
    ws = torch.empty(capi.attn_unfused_workspace_bytes(w.B, w.H, w.L, capi.ATTN_BF16), dtype=torch.uint8,
                     device="cuda")
    capi.attn_fwd_unfused(tq, tk, tv, o, w.scale, w.causal, ws)
    torch.cuda.synchronize()
    del ws
    L = w.L
    rows = np.unique(np.concatenate([np.arange(0, 16), np.arange(L - 16, L),
                                     np.random.default_rng(79).integers(0, L, 96)]))
    got = _gpu.download(o[0, 0, torch.from_numpy(rows).to("cuda")], w.dtype)
    ref = A.attention_head(_f64(q[0, 0], w.dtype), _f64(k[0, 0], w.dtype), _f64(v[0, 0], w.dtype),
                           w.scale, False, rows=rows)
    mx, mn = _gpu.errors(got, ref)
    print(f"  unfused {w.name}: max_abs {mx:.3e} mean_abs {mn:.3e} over {rows.size} rows", flush=True)
    assert torch.isfinite(o.float()).all() and mx <= 6e-2 and mn <= 6e-3


def _random_cases(n=24, seed=2609):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        d = int(rng.choice([64, 96, 128, 256]))
        L = int(rng.integers(1, 3001))
        B, H = int(rng.integers(1, 3)), int(rng.integers(1, 4))
        out.append((B, H, L, d, bool(rng.integers(0, 2)), str(rng.choice(["bf16", "f16"])), float(rng.choice([0.5, 1, 3]))))
    return out


@pytest.mark.parametrize("B,H,L,d,causal,dtype,kx", _random_cases())
def test_random_shapes(B, H, L, d, causal, dtype, kx):
    """Seeded random shapes (any L up to 3000, every head dimension, both types,
    causal or not, K spread 0.5-3): all rows against the oracle, through
    whatever tile, split count and instance the derivation picks."""
    dt = capi.ATTN_BF16 if dtype == "bf16" else capi.ATTN_F16
    plan = capi.attn_fwd_plan(B, H, L, d, causal, dt)
    print(f"case random B{B} H{H} L{L} d{d} causal{int(causal)} {dtype} kx{kx} "
          f"tile {plan.t_q_wave}x{plan.n_waves} split {plan.n_split}", flush=True)
    q, k, v = inputs.make_qkv(B, H, L, d, dtype, seed=L * 31 + d, k_scale=kx)
    scale = inputs.softmax_scale(d)
    o = _gpu.fused(_gpu.upload(q, dtype), _gpu.upload(k, dtype), _gpu.upload(v, dtype), scale, causal)
    ref = A.attention(_f64(q, dtype), _f64(k, dtype), _f64(v, dtype), scale, causal)
    _gpu.assert_close(_gpu.download(o, dtype), ref, dtype, f"random L{L} d{d}")
