"""Fused attention forward benchmark on one MI355X.

python bench.py [--gpus 1] [--steps K] [--warmup W] [--prewarm-ms T]

A step is one fused attention forward (all of Algorithm 1 for every query
tile, plus the split merge when the tile derivation splits the key range)
over the single-head L=16384, d=128 bf16 workload, with Q, K, V already
resident in device memory.  W untimed steps, then untimed steps until T ms of
sustained work have passed (the GPU clock ramps up under load), then K timed
steps.  Prints one JSON line: throughput in TFLOP/s (4 L^2 d algorithmic
flops per step), the roofline entry of the fused kernel, the other four
workload configurations (each with its own roofline entry; the 8-head one
also with the unfused baseline), the unfused three-kernel baseline, the
sequence-length sweep, HBM byte counts, and the CPU oracle's throughput on
the host cores (float32, float64 beside it).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2609_10937_amd import capi, inputs  # noqa: E402

WORKLOAD = "single_head_l16384_d128"
# The five workload configurations in order, with the timed calls of each.
CONFIGS = (("tiny_f16_l128_d64", 200), ("h8_l1024_d128", 100), ("causal_b2h16_l4096_d128_kx3", 40),
           ("single_head_l16384_d128", 0), ("causal_b4h32_l16384_d128", 8))
METRIC = "fused attention fwd TFLOPS (% bf16 MFMA peak) + HBM bytes vs unfused, L=16384 d=128"
PEAK_BF16_TFLOPS = 2516.6   # MI355X dense bf16 matrix-core peak
CLOCK_GHZ = 2.4             # the clock the published peak assumes
PEAK_F32_MFMA_TFLOPS = 157.3  # MI355X dense fp32 matrix-core peak
HBM_TBPS = 8.0


def flops(w):
    pairs = w.L * (w.L + 1) // 2 if w.causal else w.L * w.L
    return 4.0 * w.B * w.H * pairs * w.d


def fused_bytes(w):
    return 4 * w.B * w.H * w.L * w.d * 2


def unfused_bytes(w):
    return fused_bytes(w) + 4 * w.B * w.H * w.L * w.L * 2


def upload(bits, dtype):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to("cuda")
    return t.view(torch.bfloat16 if dtype == "bf16" else torch.float16)


def prewarm(fn, min_ms):
    """Untimed sustained calls until at least min_ms of wall time has passed:
    the GPU raises its clock over the first milliseconds of sustained work
    (the first launches after an idle period run 10-30% slower), so the timed
    region starts at the steady clock.  Returns (calls, ms)."""
    import torch
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    calls = 0
    while True:
        for _ in range(10):
            fn()
        calls += 10
        torch.cuda.synchronize()
        el = (time.perf_counter() - t0) * 1e3
        if el >= min_ms:
            return calls, el


def time_steps(fn, steps, warmup, warm_ms=0.0):
    """Warm up (`warmup` calls, then sustained calls until warm_ms of wall time
    has passed), then time exactly `steps` calls back to back, synchronised
    before and after, with one HIP event pair on the launch stream around the
    whole batch and nothing between the calls; then the same number of calls
    again with an event pair around each (their sorted times go to
    LAST_EVENT_MS for the median and minimum).  Returns (wall ms per call,
    batch event ms per call): the first is the throughput, the second the
    average time a call takes on the stream."""
    import torch
    for _ in range(warmup):
        fn()
    if warm_ms > 0:
        LAST_PREWARM[:] = prewarm(fn, warm_ms)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record()
    for _ in range(steps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3 / steps
    batch = e0.elapsed_time(e1) / steps
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    for i in range(steps):
        starts[i].record()
        fn()
        ends[i].record()
    torch.cuda.synchronize()
    LAST_EVENT_MS[:] = sorted(st.elapsed_time(en) for st, en in zip(starts, ends))
    return wall, batch


LAST_EVENT_MS = []  # the per-call event times of the latest time_steps, sorted
LAST_PREWARM = [0, 0.0]  # (calls, ms) of the latest time-based pre-warm


def event_stats():
    t = LAST_EVENT_MS
    return {"median_ms": round(t[len(t) // 2], 5), "min_ms": round(t[0], 5)}


def at_clock(tflops, counters):
    """Fraction of the dense bf16 peak scaled to the clock the counters measured."""
    if not counters:
        return None
    return round(tflops / (PEAK_BF16_TFLOPS * counters["clock_ghz"] / CLOCK_GHZ), 5)


def _time_oracle(A, qh, kh, vh, w, dtype, min_s):
    """The oracle over all rows of one head in `dtype`, repeated until at least
    min_s seconds of work (one untimed warm-up on a row block first).
    Returns (passes, seconds)."""
    A.attention_head(qh, kh, vh, w.scale, w.causal, rows=np.arange(256), dtype=dtype)
    passes, t0 = 0, time.perf_counter()
    while True:
        A.attention_head(qh, kh, vh, w.scale, w.causal, dtype=dtype)
        passes += 1
        dt = time.perf_counter() - t0
        if dt >= min_s:
            return passes, dt


def cpu_baseline(w, q, k, v):
    """The oracle as it stands, timed on the host's cores over a bounded sample
    of the same workload (whole passes over its one head, every query row
    against every key): float32 (the reported value) and float64 (the parity
    precision), BLAS held to the cores this process may run on."""
    from threadpoolctl import threadpool_limits

    from oracle import attention as A
    cores = len(os.sched_getaffinity(0))
    qh = inputs.bits_to_f64(q[0, 0], w.dtype)
    kh = inputs.bits_to_f64(k[0, 0], w.dtype)
    vh = inputs.bits_to_f64(v[0, 0], w.dtype)
    with threadpool_limits(cores):
        n32, dt32 = _time_oracle(A, qh, kh, vh, w, np.float32, 10.0)
        n64, dt64 = _time_oracle(A, qh, kh, vh, w, np.float64, 5.0)
    fl = flops(w)
    return {"value": n32 * fl / dt32 / 1e12, "unit": "TFLOP/s", "cores": int(cores), "kind": "oracle",
            "sample": f"float32 oracle, {n32} passes over all {w.L} query rows x {w.L} keys of the "
                      f"B=1, H=1, d={w.d} head, {dt32:.2f} s",
            "fp64": {"value": n64 * fl / dt64 / 1e12, "unit": "TFLOP/s",
                     "sample": f"the same oracle in float64, {n64} passes, {dt64:.2f} s"}}


def _code_only(text):
    """C/C++ source without comments and with whitespace runs collapsed: a
    change to comments alone leaves the code, and its measured traffic, the same."""
    import re
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def _sources_hash(pick):
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2609_10937_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        if pick(name):
            with open(os.path.join(csrc, name), encoding="utf-8") as f:
                h.update(name.encode() + _code_only(f.read()).encode())
    return h.hexdigest()[:16]


def kernel_source_hash():
    """Hash of the fused kernel's code (comments aside): a traffic figure measured
    on other code is stale."""
    return _sources_hash(lambda name: name.startswith("fwd_") or name == "internal.h")


def measured_traffic(workload):
    """HBM bytes per fused-kernel launch from the committed counter summary, if it
    was taken on the current kernel sources (else None)."""
    path = os.path.join(ROOT, "profiles", "fwd_kernel_traffic.json")
    try:
        with open(path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_hash") != kernel_source_hash():
        return None
    entry = rec.get("workloads", {}).get(workload)
    return None if entry is None else entry.get("hbm_bytes_per_launch")


def unfused_source_hash():
    """Hash of the unfused baseline's code (its products, row softmax and driver)."""
    return _sources_hash(lambda name: name.startswith("gemm_") or name in ("softmax.hip", "unfused.hip"))


def measured_unfused_bytes(workload):
    """HBM bytes of one unfused-baseline call (its three kernels) from the
    committed counter summary, if taken on the current sources (else None)."""
    try:
        with open(os.path.join(ROOT, "profiles", "unfused_traffic.json")) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("source_hash") != unfused_source_hash():
        return None
    e = rec.get("workloads", {}).get(workload)
    return None if e is None else e.get("hbm_bytes_per_call")


def measured_mfma(workload):
    """Matrix-core busy fraction and clock of the fused kernel from the committed
    counter summary, if it was taken on the current kernel sources (else None)."""
    path = os.path.join(ROOT, "profiles", "fwd_kernel_mfma_busy.json")
    try:
        with open(path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_hash") != kernel_source_hash():
        return None
    e = rec.get("workloads", {}).get(workload)
    if e is None:
        return None
    return {"busy_frac": e["mfma_busy_frac"], "clock_ghz": e["clock_ghz"],
            "source": "profiles/fwd_kernel_mfma_busy.md"}


def gemm_source_hash():
    """Hash of the GEMM kernel's sources (counter figures taken on other sources are stale)."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2609_10937_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        if name.startswith("gemm_"):
            with open(os.path.join(csrc, name), "rb") as f:
                h.update(name.encode() + f.read())
    return h.hexdigest()[:16]


def measured_gemm_counters():
    """HBM bytes and matrix-core busy fraction of the 4096^3 GEMM from the committed
    counter summary, if it was taken on the current GEMM sources (else None)."""
    try:
        with open(os.path.join(ROOT, "profiles", "gemm_4096_bf16_counters.json")) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("gemm_source_hash") != gemm_source_hash():
        return None
    return rec["kernels"]["attn_gemm"]


def sampled_parity(w, q, k, v, out):
    from oracle import attention as A
    import torch
    rows = np.unique(np.concatenate([np.arange(64), np.arange(w.L - 64, w.L),
                                     np.random.default_rng(3).integers(0, w.L, 128)]))
    got = inputs.bits_to_f64(out[0, 0, torch.from_numpy(rows).cuda()].view(torch.int16).cpu().numpy()
                             .view(np.uint16), w.dtype)
    ref = A.attention_head(inputs.bits_to_f64(q[0, 0], w.dtype), inputs.bits_to_f64(k[0, 0], w.dtype),
                           inputs.bits_to_f64(v[0, 0], w.dtype), w.scale, w.causal, rows=rows)
    e = np.abs(got - ref)
    return {"rows": int(rows.size), "max_abs": float(e.max()), "mean_abs": float(e.mean())}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=50)
    # Sustained work raises the GPU clock over the first milliseconds; after
    # the --warmup steps, untimed steps continue for this long before timing.
    ap.add_argument("--prewarm-ms", type=float, default=300.0)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle timing")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the other four workload configurations (tiny f16, 8 heads, batched causal x2)")
    ap.add_argument("--configs", default="1,2,3,5", help="which of the other configurations to run (1-5)")
    ap.add_argument("--config-steps", type=int, default=0,
                    help="timed calls per configuration (0: each configuration's own count)")
    ap.add_argument("--no-unfused", action="store_true", help="skip the unfused baseline")
    ap.add_argument("--no-sweep", action="store_true", help="skip the sequence-length sweep (Table 3)")
    ap.add_argument("--no-d256", action="store_true", help="skip the head-dimension-256 workloads")
    ap.add_argument("--no-d96", action="store_true", help="skip the head-dimension-96 workloads")
    ap.add_argument("--no-d64", action="store_true", help="skip the head-dimension-64 workloads")
    ap.add_argument("--no-causal-few", action="store_true", help="skip the few-head causal workloads")
    ap.add_argument("--no-short", action="store_true", help="skip the many-head short-sequence workloads")
    ap.add_argument("--no-softmax", action="store_true", help="skip the row-softmax operator")
    ap.add_argument("--no-gemm", action="store_true", help="skip the GEMM operator")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="finish with two plain 256 MiB device copies (reference for byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(heads shard across GPUs with no exchange; see the design notes)", file=sys.stderr)
        sys.exit(2)

    import torch
    capi.load()
    w = inputs.WORKLOADS[WORKLOAD]
    print(f"bench: generating {w.name}", file=sys.stderr, flush=True)
    q, k, v = inputs.workload_inputs(w)
    tq, tk, tv = upload(q, w.dtype), upload(k, w.dtype), upload(v, w.dtype)
    to = torch.empty_like(tq)
    plan = capi.attn_fwd_plan(w.B, w.H, w.L, w.d, w.causal, capi.ATTN_BF16)
    desc = capi.attn_hw_desc_query(torch.cuda.current_device())

    def step():
        capi.attn_fwd(tq, tk, tv, to, w.scale, w.causal)

    print("bench: fused", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    wall_ms, ev_ms = time_steps(step, args.steps, args.warmup, args.prewarm_ms)
    prewarm_info = {"calls": LAST_PREWARM[0], "ms": round(LAST_PREWARM[1], 1),
                    "note": "untimed steps after the --warmup steps, until the GPU clock is steady"}
    fl = flops(w)
    value = fl / (wall_ms * 1e-3) / 1e12
    parity = sampled_parity(w, q, k, v, to)

    # The dominant kernel on its own: attn_fwd_partial launches exactly the
    # fused kernel (the split merge, when there is one, is attn_fwd_merge).
    ws_bytes = capi.attn_fwd_workspace_bytes(w.B, w.H, w.L, w.d, w.causal, capi.ATTN_BF16)
    ws = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device="cuda") if ws_bytes else None

    def kstep():
        capi.attn_fwd_partial(tq, tk, tv, to, w.scale, w.causal, ws)

    _, k_ms = time_steps(kstep, args.steps, args.warmup, min(100.0, args.prewarm_ms))
    k_stats = event_stats()
    achieved = fl / (k_ms * 1e-3) / 1e12
    del ws

    u_ev = None
    if not args.no_unfused:
        print("bench: unfused", file=sys.stderr, flush=True)
        ws = torch.empty(capi.attn_unfused_workspace_bytes(w.B, w.H, w.L, capi.ATTN_BF16), dtype=torch.uint8,
                         device="cuda")
        tu = torch.empty_like(tq)

        def ustep():
            capi.attn_fwd_unfused(tq, tk, tv, tu, w.scale, w.causal, ws)

        _, u_ev = time_steps(ustep, max(3, args.steps // 2), 2)
        # Context for the baseline's two products: the same shapes through
        # torch.mm (hipBLASLt), S and P in bf16 like the baseline's.
        sq, sk, sv = tq.view(w.L, w.d), tk.view(w.L, w.d), tv.view(w.L, w.d)
        s_lib = ws[:w.L * w.L * 2].view(torch.bfloat16).view(w.L, w.L)
        o_lib = torch.empty(w.L, w.d, dtype=torch.bfloat16, device="cuda")
        _, lib_qk = time_steps(lambda: torch.mm(sq, sk.t(), out=s_lib), max(3, args.steps // 2), 2)
        _, lib_pv = time_steps(lambda: torch.mm(s_lib, sv, out=o_lib), max(3, args.steps // 2), 2)
        del ws, s_lib, o_lib
        torch.cuda.empty_cache()

    def config_leg(w2, n_steps, with_unfused=False):
        """One workload configuration: the whole forward (attn_fwd) and the fused
        kernel alone (attn_fwd_partial), HIP events per call, after a pre-warm."""
        dt2 = capi.ATTN_BF16 if w2.dtype == "bf16" else capi.ATTN_F16
        t2 = [upload(x, w2.dtype) for x in inputs.workload_inputs(w2)]
        o2 = torch.empty_like(t2[0])
        warm = min(100.0, args.prewarm_ms)
        _, ev2 = time_steps(lambda: capi.attn_fwd(t2[0], t2[1], t2[2], o2, w2.scale, w2.causal), n_steps, 2, warm)
        st2 = event_stats()
        nb2 = capi.attn_fwd_workspace_bytes(w2.B, w2.H, w2.L, w2.d, w2.causal, dt2)
        ws2 = torch.empty(max(nb2, 16), dtype=torch.uint8, device="cuda") if nb2 else None
        _, kev2 = time_steps(lambda: capi.attn_fwd_partial(t2[0], t2[1], t2[2], o2, w2.scale, w2.causal, ws2),
                             n_steps, 2, warm / 2)
        kst2 = event_stats()
        p2 = capi.attn_fwd_plan(w2.B, w2.H, w2.L, w2.d, w2.causal, dt2)
        fl2 = flops(w2)
        mc2 = measured_mfma(w2.name)
        ach = fl2 / (kev2 * 1e-3) / 1e12
        entry = {"workload": w2.name, "B": w2.B, "H": w2.H, "L": w2.L, "d": w2.d, "dtype": w2.dtype,
                 "causal": w2.causal, "k_scale": w2.k_scale,
                 "ms": round(ev2, 5), "ms_median_per_call": st2["median_ms"], "min_ms": st2["min_ms"],
                 "tflops": round(fl2 / (ev2 * 1e-3) / 1e12, 2),
                 "pct_peak": round(100 * fl2 / (ev2 * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 2),
                 "roofline": {"bound": "mfma", "achieved": round(ach, 2), "peak": PEAK_BF16_TFLOPS,
                              "unit": "TFLOP/s", "frac": round(ach / PEAK_BF16_TFLOPS, 5),
                              "traffic": measured_traffic(w2.name),
                              "kernel": "fwd_kernel (attn_fwd_partial): one HIP event pair around the "
                                        "back-to-back timed launches, per launch",
                              "kernel_ms": round(kev2, 5), "kernel_ms_median_per_call": kst2["median_ms"],
                              "kernel_ms_min": kst2["min_ms"],
                              "frac_at_counter_clock": at_clock(ach, mc2), "mfma_counters": mc2},
                 "algorithmic_flops": fl2, "algorithmic_bytes": fused_bytes(w2),
                 "tiles": {"t_kv": p2.t_kv, "t_q_wave": p2.t_q_wave, "n_waves": p2.n_waves,
                           "n_split": p2.n_split, "grid": p2.grid, "launch_grid": p2.launch_grid,
                           "binding": p2.binding.decode()}}
        del ws2
        if with_unfused:
            wsu = torch.empty(capi.attn_unfused_workspace_bytes(w2.B, w2.H, w2.L, dt2), dtype=torch.uint8,
                              device="cuda")
            ou = torch.empty_like(o2)
            _, uev = time_steps(lambda: capi.attn_fwd_unfused(t2[0], t2[1], t2[2], ou, w2.scale, w2.causal, wsu),
                                n_steps, 2, warm / 2)
            entry["unfused"] = {"ms": round(uev, 5),
                                "tflops": round(fl2 / (uev * 1e-3) / 1e12, 2),
                                "speedup_fused_over_unfused": round(uev / ev2, 3),
                                "algorithmic_bytes": unfused_bytes(w2),
                                "bytes_ratio": round(unfused_bytes(w2) / fused_bytes(w2), 3),
                                "measured_bytes": measured_unfused_bytes(w2.name)}
            del wsu, ou
        del t2, o2
        torch.cuda.empty_cache()
        return entry

    configs = None
    if not args.no_configs:
        # The five workload configurations; the headline (config 4) is the one
        # timed above, the others here.
        configs = []
        chosen = {int(x) for x in args.configs.split(",") if x.strip()}
        for i, (name, n_steps) in enumerate(CONFIGS, start=1):
            if i not in chosen:
                continue
            if name == WORKLOAD:
                configs.append({"config": i, "workload": name, "headline": True})
                continue
            print(f"bench: config {i} {name}", file=sys.stderr, flush=True)
            configs.append({"config": i, **config_leg(inputs.WORKLOADS[name], args.config_steps or n_steps,
                                                      with_unfused=name == "h8_l1024_d128")})

    sweep = None
    if not args.no_sweep:
        # Table 3: fused vs unfused over L at d=128, one head.  The paper's
        # speedups (its fp32 GPU) ride along as context.
        paper_speedup = {4096: 0.95, 8192: 1.25, 16384: 1.50, 32768: 1.68}
        sweep = []
        for ws_w in inputs.SWEEP:
            print(f"bench: sweep L={ws_w.L}", file=sys.stderr, flush=True)
            ts = [upload(x, ws_w.dtype) for x in inputs.workload_inputs(ws_w)]
            tos = torch.empty_like(ts[0])
            _, f_ms = time_steps(lambda: capi.attn_fwd(ts[0], ts[1], ts[2], tos, ws_w.scale, ws_w.causal), 20, 20,
                                 min(50.0, args.prewarm_ms))
            wsu = torch.empty(capi.attn_unfused_workspace_bytes(1, 1, ws_w.L, capi.ATTN_BF16), dtype=torch.uint8,
                              device="cuda")
            _, u_ms = time_steps(lambda: capi.attn_fwd_unfused(ts[0], ts[1], ts[2], tos, ws_w.scale, ws_w.causal,
                                                               wsu), 5, 2)
            fl_s = flops(ws_w)
            sweep.append({"L": ws_w.L, "fused_ms": round(f_ms, 4), "unfused_ms": round(u_ms, 4),
                          "speedup": round(u_ms / f_ms, 2), "paper_speedup": paper_speedup.get(ws_w.L),
                          "fused_tflops": round(fl_s / (f_ms * 1e-3) / 1e12, 1),
                          "fused_pct_peak": round(100 * fl_s / (f_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 1),
                          "fused_bytes": fused_bytes(ws_w), "unfused_bytes": unfused_bytes(ws_w)})
            del ts, tos, wsu
            torch.cuda.empty_cache()

    def head_dim_leg(workloads):
        out = []
        for w3 in workloads:
            print(f"bench: {w3.name}", file=sys.stderr, flush=True)
            t3 = [upload(x, w3.dtype) for x in inputs.workload_inputs(w3)]
            o3 = torch.empty_like(t3[0])
            n3 = 20 if w3.B * w3.H == 1 else 5
            _, ev3 = time_steps(lambda: capi.attn_fwd(t3[0], t3[1], t3[2], o3, w3.scale, w3.causal), n3, n3,
                                min(50.0, args.prewarm_ms))
            p3 = capi.attn_fwd_plan(w3.B, w3.H, w3.L, w3.d, w3.causal, capi.ATTN_BF16)
            out.append({"workload": w3.name, "ms": round(ev3, 4),
                        "tflops": round(flops(w3) / (ev3 * 1e-3) / 1e12, 1),
                        "pct_peak": round(100 * flops(w3) / (ev3 * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 1),
                        "tiles": {"t_kv": p3.t_kv, "t_q_wave": p3.t_q_wave, "n_waves": p3.n_waves,
                                  "n_split": p3.n_split, "tiles_per_split": p3.tiles_per_split,
                                  "grid": p3.grid, "launch_grid": p3.launch_grid}})
            del t3, o3
            torch.cuda.empty_cache()
        return out

    d256 = None if args.no_d256 else head_dim_leg(inputs.HEAD_DIM_256)
    d96 = None if args.no_d96 else head_dim_leg(inputs.HEAD_DIM_96)
    d64 = None if args.no_d64 else head_dim_leg(inputs.HEAD_DIM_64)
    causal_few = None if args.no_causal_few else head_dim_leg(inputs.CAUSAL_FEW_HEADS)
    short = None if args.no_short else head_dim_leg(inputs.SHORT_SEQUENCES)

    smx = None
    if not args.no_softmax:
        # The row-softmax operator of Section 5.3: the paper's 512 x 512 and the
        # score matrix of one L=16384 head; HBM-bound, so reported against 8 TB/s.
        smx = []
        hwq = capi.attn_hw_desc_query(torch.cuda.current_device())
        for rows, n_cols in ((512, 512), (16384, 16384)):
            print(f"bench: softmax {rows}x{n_cols}", file=sys.stderr, flush=True)
            xs = upload(inputs.make_matrix(rows, n_cols, "bf16", seed=1301, spread=2.0), "bf16")
            ys = torch.empty_like(xs)
            rep = capi.attn_softmax_derive(hwq, rows, n_cols)
            _, s_ms = time_steps(lambda: capi.attn_softmax(xs, ys), 50, 50)
            smx.append({"rows": rows, "n": n_cols, "us": round(1e3 * s_ms, 2), "hbm_bytes": rep.hbm_bytes,
                        "tbps": round(rep.hbm_bytes / (s_ms * 1e-3) / 1e12, 3),
                        "frac_hbm": round(rep.hbm_bytes / (s_ms * 1e-3) / 1e12 / HBM_TBPS, 3),
                        "tiles": {"split": rep.split, "resident_tiles": rep.resident_tiles, "passes": rep.passes,
                                  "grid": rep.grid, "binding": rep.binding.decode()}})
            del xs, ys
        torch.cuda.empty_cache()

    gemm = None
    if not args.no_gemm:
        # The GEMM of Section 4 (Figure 1's 4096^3, bf16 inputs, fp32 accumulate and
        # output) on the derived tiles; torch.mm (the vendor library, bf16 output)
        # on the same inputs for reference.
        M = N = K = 4096
        print(f"bench: gemm {M}x{N}x{K}", file=sys.stderr, flush=True)
        hwq = capi.attn_hw_desc_query(torch.cuda.current_device())
        rep = capi.attn_gemm_derive(hwq, capi.attn_atom_preset("bf16_16x16x32"), M, N, K)
        ga = upload(inputs.make_matrix(M, K, "bf16", seed=1401), "bf16")
        gb = upload(inputs.make_matrix(K, N, "bf16", seed=1402), "bf16")
        gc = torch.empty((M, N), dtype=torch.float32, device="cuda")
        _, g_ms = time_steps(lambda: capi.attn_gemm(ga, gb, gc), 50, 50)
        _, t_ms = time_steps(lambda: torch.mm(ga, gb), 50, 50)
        # The same product with fp32 output (this operator's output type), where
        # the installed torch offers it.
        try:
            _, t32_ms = time_steps(lambda: torch.mm(ga, gb, out_dtype=torch.float32), 50, 50)
        except (RuntimeError, TypeError, NotImplementedError):
            t32_ms = None
        gfl = 2.0 * M * N * K
        gc_ = measured_gemm_counters()
        gemm = {"M": M, "N": N, "K": K, "dtype": "bf16", "out": "f32", "us": round(1e3 * g_ms, 2),
                "tflops": round(gfl / (g_ms * 1e-3) / 1e12, 1),
                "frac_peak": round(gfl / (g_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
                "roofline": {"bound": "mfma", "achieved": round(gfl / (g_ms * 1e-3) / 1e12, 1),
                             "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                             "frac": round(gfl / (g_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
                             "traffic": None if gc_ is None else gc_["hbm_bytes_per_launch"],
                             "algorithmic_bytes": 2 * M * K * 2 + M * N * 4,
                             "mfma_busy_frac": None if gc_ is None else gc_["mfma_busy_frac"],
                             "clock_ghz": None if gc_ is None else gc_["clock_ghz"]},
                "torch_mm_bf16_us": round(1e3 * t_ms, 2),
                "torch_mm_tflops": round(gfl / (t_ms * 1e-3) / 1e12, 1),
                "torch_mm_f32_out_us": None if t32_ms is None else round(1e3 * t32_ms, 2),
                "torch_mm_f32_out_tflops": None if t32_ms is None else round(gfl / (t32_ms * 1e-3) / 1e12, 1),
                "tiles": {"t_m": rep.t_m, "t_n": rep.t_n, "t_k": rep.t_k, "warp_m": rep.warp_m,
                          "warp_n": rep.warp_n, "grid": rep.grid, "vgpr_est": rep.vgpr_est,
                          "binding": rep.binding.decode()}}
        del ga, gb, gc
        # The same shape in fp32 (the section's type: 12.3 TFLOP/s = 53% of its GPU's
        # fp32 matrix peak) on the fp32 family's tiles, against MI355X's fp32 matrix peak.
        rep32 = capi.attn_gemm_derive(hwq, capi.attn_atom_preset("f32_16x16x4"), M, N, K)
        fa = torch.from_numpy(inputs.make_matrix_f32(M, K, seed=1403)).cuda()
        fb = torch.from_numpy(inputs.make_matrix_f32(K, N, seed=1404)).cuda()
        fc = torch.empty((M, N), dtype=torch.float32, device="cuda")
        _, f_ms = time_steps(lambda: capi.attn_gemm(fa, fb, fc), 20, 20)
        _, tf_ms = time_steps(lambda: torch.mm(fa, fb), 20, 20)
        gemm["fp32"] = {"us": round(1e3 * f_ms, 2), "tflops": round(gfl / (f_ms * 1e-3) / 1e12, 1),
                        "peak": PEAK_F32_MFMA_TFLOPS,
                        "frac_peak": round(gfl / (f_ms * 1e-3) / 1e12 / PEAK_F32_MFMA_TFLOPS, 4),
                        "paper": {"tflops": 12.3, "frac_peak": 0.53, "peak": 23.1},
                        "torch_mm_fp32_us": round(1e3 * tf_ms, 2),
                        "torch_mm_tflops": round(gfl / (tf_ms * 1e-3) / 1e12, 1),
                        "tiles": {"t_m": rep32.t_m, "t_n": rep32.t_n, "t_k": rep32.t_k, "warp_m": rep32.warp_m,
                                  "warp_n": rep32.warp_n, "grid": rep32.grid, "vgpr_est": rep32.vgpr_est,
                                  "binding": rep32.binding.decode()}}
        del fa, fb, fc
        torch.cuda.empty_cache()

    cpu = None
    if not args.no_cpu:
        print("bench: cpu oracle", file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, q, k, v)

    out = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall_ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "H": w.H, "L": w.L, "d": w.d, "causal": w.causal,
                   "inputs": "N(0,1) float32 rounded to bf16, seed 1004",
                   "tiles": {"t_kv": plan.t_kv, "t_q_wave": plan.t_q_wave, "n_waves": plan.n_waves,
                             "tile_q": plan.tile_q, "n_split": plan.n_split, "grid": plan.grid,
                             "launch_grid": plan.launch_grid, "vgpr_est": plan.vgpr_est,
                             "binding": plan.binding.decode()},
                   "device": {"num_cus": desc.num_cus, "lds_bytes": desc.lds_bytes,
                              "clock_ghz": desc.clock_ghz}},
        "pct_peak": round(100 * value / PEAK_BF16_TFLOPS, 2),
        "roofline": {"bound": "mfma", "achieved": round(achieved, 3), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 5),
                     "traffic": measured_traffic(w.name),
                     "kernel": "fwd_kernel (attn_fwd_partial): one HIP event pair around the back-to-back timed "
                               "launches on their stream, per launch",
                     "kernel_ms": round(k_ms, 5), "kernel_ms_median": k_stats["median_ms"],
                     "kernel_ms_min": k_stats["min_ms"], "step_event_ms": round(ev_ms, 5),
                     "frac_at_counter_clock": at_clock(achieved, measured_mfma(w.name)),
                     "mfma_counters": measured_mfma(w.name),
                     "algorithmic_flops_per_launch": fl, "algorithmic_bytes_per_launch": fused_bytes(w)},
        "hbm_bytes": {"fused_algorithmic": fused_bytes(w), "unfused_algorithmic": unfused_bytes(w),
                      "ratio": unfused_bytes(w) / fused_bytes(w)},
        "unfused": None if u_ev is None else {
            "ms": round(u_ev, 4), "tflops": round(fl / (u_ev * 1e-3) / 1e12, 2),
            "speedup_fused_over_unfused": round(u_ev / ev_ms, 3),
            "algorithmic_bytes": unfused_bytes(w),
            "hbm_rate_tbps": round(unfused_bytes(w) / (u_ev * 1e-3) / 1e12, 3),
            "torch_mm_products_ms": {"qk": round(lib_qk, 4), "pv": round(lib_pv, 4)}},
        "parity": parity,
        "prewarm": prewarm_info,
        "configs": configs,
        "l_sweep": sweep,
        "head_dim_256": d256,
        "head_dim_96": d96,
        "head_dim_64": d64,
        "causal_few_heads": causal_few,
        "short_sequences": short,
        "softmax": smx,
        "gemm": gemm,
        "cpu_baseline": cpu,
    }
    if args.copy_calibration:
        src = torch.ones(64 << 20, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(2):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
