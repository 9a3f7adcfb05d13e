"""Host logic of bench.py: the flop and byte counts its figures rest on, the
timing statistics, the clock scaling, and the one-GPU contract (CPU only)."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
from paper_2609_10937_amd import inputs  # noqa: E402


def test_flops_of_the_workloads():
    """4 d flops per (query, visible key) pair; causal keeps L(L+1)/2 pairs per head."""
    W = inputs.WORKLOADS
    assert bench.flops(W["single_head_l16384_d128"]) == 4 * 16384 ** 2 * 128 == 137438953472
    assert round(bench.flops(W["causal_b4h32_l16384_d128"]) / 1e9, 1) == 8796.6
    assert round(bench.flops(W["causal_b2h16_l4096_d128_kx3"]) / 1e9, 2) == 137.47
    assert bench.flops(W["tiny_f16_l128_d64"]) == 4 * 128 * 128 * 64


def test_byte_counts_and_the_129x_ratio():
    """Fused: Q, K, V read and O written once; unfused adds S written and read and
    P written and read (4 L^2 e per head), a ratio of 1 + L/d."""
    w = inputs.WORKLOADS["single_head_l16384_d128"]
    assert bench.fused_bytes(w) == 16777216
    assert bench.unfused_bytes(w) == 2164260864
    assert bench.unfused_bytes(w) / bench.fused_bytes(w) == 1 + w.L / w.d == 129


def test_event_stats_and_clock_scaling():
    bench.LAST_EVENT_MS[:] = [0.10, 0.11, 0.12, 0.13, 0.20]
    assert bench.event_stats() == {"median_ms": 0.12, "min_ms": 0.1}
    assert bench.at_clock(1258.3, {"clock_ghz": 1.2}) == 1.0
    assert bench.at_clock(1000.0, None) is None


def test_configs_cover_the_five_workloads_in_order():
    names = [n for n, _ in bench.CONFIGS]
    assert names == ["tiny_f16_l128_d64", "h8_l1024_d128", "causal_b2h16_l4096_d128_kx3",
                     "single_head_l16384_d128", "causal_b4h32_l16384_d128"]
    assert bench.WORKLOAD == names[3]
    assert all(n > 0 for name, n in bench.CONFIGS if name != bench.WORKLOAD)


def test_prewarm_runs_until_the_time_has_passed(monkeypatch):
    import time
    torch = pytest.importorskip("torch")
    monkeypatch.setattr(torch.cuda, "synchronize", lambda: None)
    calls = []
    calls_n, ms = bench.prewarm(lambda: (calls.append(1), time.sleep(0.0005)), 20.0)
    assert ms >= 20.0 and calls_n == len(calls) and calls_n % 10 == 0


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)
