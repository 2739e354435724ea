"""CPU checks of bench.py's contract that need no GPU: the one-GPU refusal,
the peaks it reports against, and that the committed rocprofv3 summaries of
the attention workloads were taken from the attention kernel source as it
stands (bench.py attaches their HBM traffic and SQ counters to its line only
then; a kernel change without new profiles would drop them silently)."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402

PROFILED = ["dense_d128_s2k", "causal_d64_s1k", "causal_peaky_d128_s8k", "gqa4_causal_d128_s4k",
            "tiny_d64_s128"]


def test_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert "one GPU" in (r.stdout + r.stderr)
    assert '"value"' not in r.stdout


def test_peaks():
    # MI355X: 256 CUs x 2.4 GHz x 4096 dense bf16 flop/clk/CU; 8 TB/s HBM3E
    assert abs(bench.PEAK_BF16_TFLOPS - 256 * 2.4e9 * 4096 / 1e12) < 0.1
    assert bench.HBM_PEAK_GBS == 8000.0


@pytest.mark.parametrize("workload", PROFILED)
def test_profiles_match_kernel_source(workload):
    traffic = bench.read_traffic(workload)
    assert traffic is not None, f"profiles/attn_fwd_{workload}_traffic.md is stale or missing"
    counters = bench.read_counters(workload, 1.0)
    assert counters is not None, f"profiles/attn_fwd_{workload}_counters.md is stale or missing"
    assert 0.0 <= counters["mfma_busy_pct"] <= 100.0


def test_dense_traffic_is_algorithmic():
    """The dense workload's measured HBM bytes per launch equal its
    algorithmic bytes (Q, K, V read once; O, LSE written once) within 1 %."""
    w = bench.gen.WORKLOADS["dense_d128_s2k"]
    assert abs(bench.read_traffic(w.name) / w.bytes() - 1.0) < 0.01
