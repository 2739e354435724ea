"""Benchmark of the fused attention forward (libtileattn) on one MI355X.

A step is one attn_fwd launch over one batch of the workload, inputs already
resident in HBM.  Prints ONE JSON line with the throughput in TFLOP/s (matmul
flops over visible query-key pairs), the roofline position of the kernel
against the dense bf16 MFMA peak, and the fp64 CPU oracle's throughput on a
bounded sample of the same workload as a reported baseline.  The oracle is
touched only in that CPU leg, after the timed region: it spot-checks a few
outputs, times itself, and (attention and MLA) compares every row it
computed with the last timed launch's output (a failed check ends the run
without a number); --no-cpu-baseline skips the leg and never loads the
oracle.

  python bench.py [--steps K] [--warmup W] [--workload NAME] [--out f32|bf16]
                  [--splits 1|N|auto] [--no-cpu-baseline]
  python bench.py --oracle-all-configs
                                    # the fp64 oracle on every element of the five
                                    # target configurations, timed per configuration
                                    # (and compared with the GPU output if present)
  python bench.py --copy-probe      # plain device copy of known size, for
                                    # scaling rocprofv3 FETCH_SIZE/WRITE_SIZE
  python bench.py --workload gemm_m5 [--out f32|bf16]
                                    # C = A B (gemm_bf16) at one of the paper's
                                    # M0-M7 shapes, with hipBLASLt timed beside it
  python bench.py --workload gemv_v0 [--out f32|bf16] [--splits 1|N|auto]
                                    # the same call at M = 1 (the paper's V0-V7
                                    # matrix-vector shapes), HBM-bound; with more
                                    # than one split, gemv_bf16_split
  python bench.py --workload mla_b64_s8k [--splits auto|N]
                                    # one multi-head latent attention decode step
                                    # (mla_decode) instead of attn_fwd
  python bench.py --workload ssd_b64_s8k [--op chunk_scan|chunk_state]
                                    # one Mamba-2 SSD chunk function at one of the
                                    # paper's linear-attention shapes
  python bench.py --sustain 8 [--gemm-reference]
                                    # run the step back to back for 8 s while
                                    # sampling board power and XCD clocks
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2504_17577_amd import gen  # noqa: E402

METRIC = "attention fwd TFLOP/s and % of MI355X bf16 MFMA peak, 1 GPU"
DEFAULT_WORKLOAD = "dense_d128_s2k"
# MI355X dense bf16 MFMA peak: 256 CUs x 2.4 GHz x 4096 flop/clk/CU
PEAK_BF16_TFLOPS = 2516.6
HBM_PEAK_GBS = 8000.0
KERNEL_SRC = os.path.join(ROOT, "paper_2504_17577_amd", "csrc", "attn_fwd.hip")
PROFILES = os.path.join(ROOT, "profiles")


def kernel_digest() -> str:
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.blake2b(f.read(), digest_size=8).hexdigest()


def _profile_fields(workload: str, kind: str):
    """The machine-readable ``key: value`` lines of a committed rocprofv3
    summary (profiles/attn_fwd_<workload>_<kind>.md), or None when there is
    none or the kernel source changed since it was taken."""
    path = os.path.join(PROFILES, f"attn_fwd_{workload}_{kind}.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_src = re.search(r"^kernel_source_blake2b:\s*([0-9a-f]+)", text, re.M)
    if not m_src or m_src.group(1) != kernel_digest():
        return None
    return {k: float(v) for k, v in
            re.findall(r"^([a-z][a-z0-9_]*):\s*([-0-9.eE+]+)\s*$", text, re.M)}


def read_traffic(workload: str):
    """HBM bytes per launch from the committed rocprofv3 --pmc FETCH_SIZE /
    WRITE_SIZE summary (scaled by the copy probe), or None."""
    f = _profile_fields(workload, "traffic")
    return None if f is None or "hbm_bytes_per_launch" not in f else f["hbm_bytes_per_launch"]


def read_counters(workload: str, ms: float):
    """MFMA busy fraction, LDS bank-conflict cycles and measured HBM GB/s of
    the kernel, from the committed SQ-counter and traffic summaries of the
    same kernel source (rocprofv3 --pmc runs of this command), or None."""
    f = _profile_fields(workload, "counters")
    if f is None:
        return None
    out = {"source": f"profiles/attn_fwd_{workload}_counters.md"}
    for key in ("mfma_busy_pct", "lds_bank_conflict_cycles_per_launch", "shader_clock_ghz",
                "valu_insts_per_mfma"):
        if key in f:
            out[key] = f[key]
    traffic = read_traffic(workload)
    if traffic is not None:
        out["hbm_gbs_measured"] = round(traffic / (ms * 1e-3) / 1e9, 1)
    return out


def host_cores() -> int:
    """Cores this process may run on (its affinity mask)."""
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:
        return os.cpu_count() or 1


def blas_threads() -> int:
    """Threads of numpy's BLAS pool (the numpy oracles' matmuls run there)."""
    try:
        from threadpoolctl import threadpool_info
        n = [p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"]
        return max(n) if n else 1
    except Exception:
        return 1


def to_device(a, torch):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()


def cpu_baseline(w, q, k, v, budget_s: float = 15.0):
    """fp64 oracle throughput on whole heads of the workload, as many as fit
    in about ``budget_s`` seconds of wall time (at least one)."""
    import oracle

    threads = oracle.default_threads()
    lib = oracle.load()

    def head_rows(hidx):
        b, h = divmod(hidx, w.Hq)
        i = np.arange(w.Sq, dtype=np.int64)
        return np.stack([np.full_like(i, b), np.full_like(i, h), i], axis=1)

    t0 = time.perf_counter()
    oracle.attn_rows(q, k, v, w.causal, w.scale, head_rows(0), nthreads=threads, lib=lib)
    t1 = time.perf_counter() - t0
    n_heads = int(max(1, min(w.B * w.Hq - 1, budget_s / max(t1, 1e-6) - 1)))
    rows = np.concatenate([head_rows(1 + i) for i in range(n_heads)]) if n_heads else None
    t0 = time.perf_counter()
    ro, rl = oracle.attn_rows(q, k, v, w.causal, w.scale, rows, nthreads=threads, lib=lib)
    dt = time.perf_counter() - t0
    flops = w.flops() / (w.B * w.Hq) * n_heads
    info = {
        "value": flops / dt / 1e12,
        "unit": "TFLOP/s",
        "cores": threads,
        "host_cores": host_cores(),
        "kind": "oracle",
        "sample": f"{n_heads} of {w.B * w.Hq} heads of {w.name} (all {w.Sq} query rows each), "
                  f"fp64 C oracle, {dt:.1f} s wall",
    }
    return info, rows, ro, rl


class PowerSampler:
    """Samples socket power and the eight XCD shader clocks with ``amd-smi
    metric -p -c`` in a background thread (a child process per sample)."""

    def __init__(self):
        import threading
        self.samples = []
        self._stop = threading.Event()
        self._thread = threading.Thread(target=self._run, daemon=True)

    def _run(self):
        import subprocess
        while not self._stop.is_set():
            try:
                out = subprocess.run(["amd-smi", "metric", "-p", "-c"], capture_output=True,
                                     text=True, timeout=10).stdout
            except (OSError, subprocess.SubprocessError):
                return
            p = re.search(r"SOCKET_POWER:\s*(\d+)", out)
            clk = [int(c) for c in re.findall(r"GFX_\d+:\s*\n\s*CLK:\s*(\d+)", out)]
            if p and clk:
                self.samples.append((time.perf_counter(), int(p.group(1)), clk))
            self._stop.wait(0.2)

    def __enter__(self):
        self._thread.start()
        return self

    def __exit__(self, *exc):
        self._stop.set()
        self._thread.join()

    def summary(self, t0: float, t1: float):
        ss = [s for s in self.samples if t0 <= s[0] <= t1]
        if not ss:
            return None
        n_x = min(len(s[2]) for s in ss)
        clk = [sum(s[2][x] for s in ss) / len(ss) for x in range(n_x)]
        return {"socket_power_w": round(sum(s[1] for s in ss) / len(ss), 1),
                "xcd_clock_mhz_mean": round(sum(clk) / n_x, 1),
                "xcd_clock_mhz_min": round(min(clk), 1), "xcd_clock_mhz_max": round(max(clk), 1),
                "samples": len(ss)}


def sustained(torch, fn, flops: float, seconds: float, sampler: PowerSampler):
    """Run ``fn`` back to back for about ``seconds`` s; report the rate and the
    power/clock samples taken after the first second (clocks settle)."""
    fn()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record()
    n = 0
    while time.perf_counter() - t0 < seconds:
        for _ in range(20):
            fn()
        torch.cuda.synchronize()
        n += 20
    end.record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms = start.elapsed_time(end) / n
    return {"tflops": round(flops / (ms * 1e-3) / 1e12, 2), "ms_per_call": round(ms, 5),
            "calls": n, **(sampler.summary(t0 + 1.0, t1) or {})}


def copy_probe(torch, mib: int = 1024, reps: int = 5):
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes_read": n * 4, "copy_probe_bytes_written": n * 4,
                      "reps": reps}), flush=True)


MLA_METRIC = "MLA decode TFLOP/s and % of MI355X bf16 MFMA peak, 1 GPU"


def mla_cpu_baseline(w, q, q_pe, kv, k_pe, budget_s: float = 15.0):
    """fp64 oracle throughput on whole batch elements of an MLA workload (all
    heads each), as many as fit in about ``budget_s`` seconds."""
    import oracle

    threads = oracle.default_threads()
    lib = oracle.load()

    def heads(b):
        return [(b, h) for h in range(w.H)]

    t0 = time.perf_counter()
    oracle.mla_rows(q, q_pe, kv, k_pe, w.scale, heads(0), nthreads=threads, lib=lib)
    t1 = time.perf_counter() - t0
    n_b = int(max(1, min(w.B - 1, budget_s / max(t1, 1e-6) - 1)))
    rows = [r for b in range(1, 1 + n_b) for r in heads(b)]
    t0 = time.perf_counter()
    ro, rl = oracle.mla_rows(q, q_pe, kv, k_pe, w.scale, rows, nthreads=threads, lib=lib)
    dt = time.perf_counter() - t0
    flops = w.flops() / w.B * n_b
    info = {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": threads,
            "host_cores": host_cores(), "kind": "oracle",
            "sample": f"{n_b} of {w.B} batch elements of {w.name} (all {w.H} heads each), "
                      f"fp64 C oracle, {dt:.1f} s wall"}
    return info, rows, ro, rl


def bench_mla(args, torch, tileattn):
    """One MLA decode step per launch (plus the split merge when split)."""
    w = gen.MLA_WORKLOADS[args.workload]
    q, q_pe, kv, k_pe = gen.make_mla_inputs(w, seed=args.seed)
    dq, dqp, dkv, dkp = (to_device(x, torch) for x in (q, q_pe, kv, k_pe))
    o = torch.empty((w.B, w.H, w.Dl), dtype=torch.float32, device="cuda")
    lse = torch.empty((w.B, w.H), dtype=torch.float32, device="cuda")
    n_split = (tileattn.mla_split_heuristic(w.B, w.H, w.Hkv, w.Skv) if args.splits == "auto"
               else int(args.splits))
    ws = torch.empty(max(16, tileattn.mla_workspace_bytes(w.B, w.H, n_split)), dtype=torch.uint8,
                     device="cuda")
    stream = torch.cuda.current_stream()

    def step():
        tileattn.mla_decode(dq, dqp, dkv, dkp, scale=w.scale, num_splits=n_split, out=o, lse=lse,
                            workspace=ws, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record(stream)
    for _ in range(args.steps):
        step()
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = start.elapsed_time(end) / args.steps
    tflops = w.flops() / (ms * 1e-3) / 1e12
    gbs = w.bytes() / (ms * 1e-3) / 1e9
    result = {
        "metric": MLA_METRIC, "value": round(tflops, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "splits": n_split, "data": "synthetic",
        "config": {"workload": w.name, "shape": w.describe(), "B": w.B, "H": w.H, "Hkv": w.Hkv,
                   "Skv": w.Skv, "Dl": w.Dl, "Dr": w.Dr, "seed": args.seed,
                   "flops_per_step": w.flops(), "bytes_per_step": w.bytes()},
        "pct_of_peak": round(100 * tflops / PEAK_BF16_TFLOPS, 2),
        "roofline": {"bound": "mfma", "achieved": round(tflops, 2), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(tflops / PEAK_BF16_TFLOPS, 4),
                     "traffic": None, "hbm_gbs_algorithmic": round(gbs, 1),
                     "hbm_frac": round(gbs / HBM_PEAK_GBS, 4)},
        "wall_s_timed": round(wall, 4),
    }
    if not args.no_cpu_baseline:
        # the CPU-oracle leg: spot check, then the oracle's throughput
        import oracle
        rows = [(0, 0), (w.B - 1, w.H - 1), (w.B // 2, w.H // 2)]
        ro, rl = oracle.mla_rows(q, q_pe, kv, k_pe, w.scale, rows)
        idx = tuple(torch.tensor(c) for c in zip(*rows))
        err_o = float(np.abs(o[idx].cpu().numpy() - ro).max())
        err_l = float(np.abs(lse[idx].cpu().numpy() - rl).max())
        if not (err_o <= 2e-2 and err_l <= 1e-3):
            raise SystemExit(f"bench: result check failed (max|dO|={err_o}, max|dLSE|={err_l})")
        info, rows2, ro, rl = mla_cpu_baseline(w, q, q_pe, kv, k_pe)
        # every head the oracle leg computed, against the last timed launch
        idx = tuple(torch.tensor(c) for c in zip(*rows2))
        err_o = max(err_o, float(np.abs(o[idx].cpu().numpy() - ro).max()))
        err_l = max(err_l, float(np.abs(lse[idx].cpu().numpy() - rl).max()))
        if not (err_o <= 2e-2 and err_l <= 1e-3):
            raise SystemExit(f"bench: result check failed (max|dO|={err_o}, max|dLSE|={err_l})")
        result["check"] = {"max_abs_dO": err_o, "max_abs_dLSE": err_l,
                           "rows": len(rows) + len(rows2)}
        result["cpu_baseline"] = info
    print(json.dumps(result), flush=True)


GEMM_METRIC = "GEMM TFLOP/s and % of MI355X bf16 MFMA peak, 1 GPU"
GEMV_METRIC = "matrix-vector product throughput (algorithmic HBM GB/s), 1 GPU"


def bench_gemm(args, torch, tileattn):
    """C = A B at a GEMM workload; torch.matmul (hipBLASLt) on the same
    operands is timed the same way as a reference."""
    w = gen.GEMM_WORKLOADS[args.workload]
    a, b = gen.make_gemm_inputs(w, seed=args.seed)
    da, db = to_device(a, torch), to_device(b, torch)
    c_bf16 = args.out != "f32"
    dt = torch.bfloat16 if c_bf16 else torch.float32
    c = torch.empty((w.M, w.N), dtype=dt, device="cuda")
    stream = torch.cuda.current_stream()

    gemv = w.M == 1
    n_split = 1
    if gemv:
        # gemv_bf16_split (K split over workgroups, fp32 partials merged by a
        # second kernel); 1 is gemm_bf16's matrix-vector kernel
        n_split = (tileattn.gemv_split_heuristic(w.N, w.K) if args.splits == "auto"
                   else int(args.splits))
    elif args.splits != "1":
        raise SystemExit("bench: --splits applies to attention, MLA and matrix-vector workloads")
    ws = torch.empty(max(16, tileattn.gemv_split_workspace_bytes(w.N, n_split) if gemv else 16),
                     dtype=torch.uint8, device="cuda")

    def step():
        if n_split > 1:
            tileattn.gemv_bf16_split(da, db, num_splits=n_split, out=c, out_dtype=dt, workspace=ws,
                                     stream=stream)
        else:
            tileattn.gemm_bf16(da, db, out=c, out_dtype=dt, stream=stream)

    def timed(fn):
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        start = torch.cuda.Event(enable_timing=True)
        end = torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        start.record(stream)
        for _ in range(args.steps):
            fn()
        end.record(stream)
        torch.cuda.synchronize()
        return start.elapsed_time(end) / args.steps, time.perf_counter() - t0

    ms, wall = timed(step)
    ref_out = torch.empty((w.M, w.N), dtype=torch.bfloat16, device="cuda")
    ms_ref, _ = timed(lambda: torch.matmul(da, db, out=ref_out))
    tflops = w.flops() / (ms * 1e-3) / 1e12
    gbs = w.bytes(2 if c_bf16 else 4) / (ms * 1e-3) / 1e9
    common = {
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "out_dtype": "bf16" if c_bf16 else "f32", "data": "synthetic",
        "config": {"workload": w.name, "shape": w.describe(), "M": w.M, "N": w.N, "K": w.K,
                   "splits": n_split, "seed": args.seed, "flops_per_step": w.flops(),
                   "bytes_per_step": w.bytes(2 if c_bf16 else 4)},
    }
    if gemv:
        result = {"metric": GEMV_METRIC, "value": round(gbs, 1), "unit": "GB/s", **common,
                  "pct_of_peak": round(100 * gbs / HBM_PEAK_GBS, 2),
                  "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS,
                               "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
                               "traffic": None, "tflops": round(tflops, 3)}}
    else:
        result = {"metric": GEMM_METRIC, "value": round(tflops, 2), "unit": "TFLOP/s", **common,
                  "pct_of_peak": round(100 * tflops / PEAK_BF16_TFLOPS, 2),
                  "roofline": {"bound": "mfma", "achieved": round(tflops, 2),
                               "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                               "frac": round(tflops / PEAK_BF16_TFLOPS, 4), "traffic": None,
                               "hbm_gbs_algorithmic": round(gbs, 1)}}
    result.update({
        "vendor_reference": {"op": "torch.matmul bf16 -> bf16 (hipBLASLt)",
                             "tflops": round(w.flops() / (ms_ref * 1e-3) / 1e12, 3),
                             "ms_per_call": round(ms_ref, 5),
                             "ratio": round(ms_ref / ms, 4)},
        "wall_s_timed": round(wall, 4),
    })
    if not args.no_cpu_baseline:
        # the CPU-oracle leg: spot check of the output, then the oracle's
        # throughput
        import oracle
        if gemv:
            # M = 1: sampled columns (the oracle would widen all of B otherwise)
            rng = np.random.default_rng(args.seed + 1)
            cols = np.unique(np.concatenate([[0, 63, 64, w.N - 1], rng.integers(0, w.N, size=60)]))
            bs = np.ascontiguousarray(b[:, cols])
            ref, scale = oracle.gemm(a, bs)[0], oracle.gemm_abs(a, bs)[0]
            got = c.float()[0, torch.from_numpy(cols).cuda()].cpu().numpy()
            checked = {"columns": int(len(cols))}
        else:
            rows = [0, w.M // 2, w.M - 1]
            ref = oracle.gemm(a, b, rows=rows)
            scale = oracle.gemm_abs(a, b, rows=rows)
            got = c.float()[torch.tensor(rows)].cpu().numpy()
            checked = {"rows": len(rows)}
        tol = 1e-5 * scale + (2.0 ** -8 * np.abs(ref) if c_bf16 else 0.0)
        worst = float((np.abs(got - ref) / tol).max())
        if not worst <= 1.0:
            raise SystemExit(f"bench: result check failed (worst err/tol {worst})")
        result["check"] = {"worst_err_over_tol": worst, **checked}
        # fp64 oracle on a bounded share of the output (about 10 s), calibrated
        # on a small share after one untimed call (the first pays numpy's set-up)
        if gemv:
            def part(n):
                return oracle.gemm(a, np.ascontiguousarray(b[:, :n]))
            total, unit_name, cal = w.N, "columns", 64
        else:
            def part(n):
                return oracle.gemm(a, b, rows=list(range(n)))
            total, unit_name, cal = w.M, "rows", 16
        part(1)
        t0 = time.perf_counter()
        part(cal)
        t1 = max(time.perf_counter() - t0, 1e-6) / cal
        n = int(max(1, min(total, 10.0 / t1)))
        t0 = time.perf_counter()
        part(n)
        dt_s = time.perf_counter() - t0
        share = n / total
        if gemv:
            value, unit = w.bytes(2) * share / dt_s / 1e9, "GB/s"
        else:
            value, unit = w.flops() * share / dt_s / 1e12, "TFLOP/s"
        result["cpu_baseline"] = {
            "value": value, "unit": unit,
            "cores": blas_threads(), "host_cores": host_cores(), "kind": "oracle",
            "sample": f"{n} of {total} {unit_name} of {w.name}, float64 numpy matmul "
                      f"(BLAS threads), {dt_s:.1f} s wall"}
    print(json.dumps(result), flush=True)


SSD_METRIC = {"chunk_scan": "SSD chunk-scan throughput (algorithmic HBM GB/s), 1 GPU",
              "chunk_state": "SSD chunk-state throughput (algorithmic HBM GB/s), 1 GPU"}


def bench_ssd(args, torch, tileattn):
    """One Mamba-2 SSD chunk function per step (chunk_scan by default, or
    chunk_state) at an SSD workload.  Its other inputs (states, the chunk
    matrix) are made beforehand on the GPU by the library's own chunk-state,
    state-passing and chunk-matrix kernels."""
    op = args.op or "chunk_scan"
    w = gen.SSD_WORKLOADS[args.workload]
    inp = gen.make_ssd_inputs(w, seed=args.seed)
    f32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
    dx, dB, dC = (to_device(inp[k], torch) for k in ("x", "Bm", "Cm"))
    ddt, dA, dD = f32(inp["dt"]), f32(inp["A"]), f32(inp["D"])
    stream = torch.cuda.current_stream()
    states = tileattn.ssd_chunk_state(dx, dB, ddt, dA, stream=stream)
    prev, _ = tileattn.ssd_state_passing(states, ddt, dA, stream=stream)
    cb = tileattn.ssd_bmm_chunk(dC, dB, stream=stream)
    y = torch.empty((w.B, w.L, w.H, w.P), dtype=torch.float32, device="cuda")
    if op == "chunk_scan":
        def step():
            tileattn.ssd_chunk_scan(dx, dC, cb, ddt, dA, prev, dD, out=y, stream=stream)
        flops, nbytes = w.flops_scan(), w.bytes_scan()
    else:
        def step():
            tileattn.ssd_chunk_state(dx, dB, ddt, dA, out=states, stream=stream)
        flops, nbytes = w.flops_state(), w.bytes_state()
    step()
    torch.cuda.synchronize()


    for _ in range(args.warmup):
        step()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record(stream)
    for _ in range(args.steps):
        step()
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = start.elapsed_time(end) / args.steps
    gbs = nbytes / (ms * 1e-3) / 1e9
    result = {
        "metric": SSD_METRIC[op], "value": round(gbs, 1), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "op": op, "shape": w.describe(), "B": w.B, "L": w.L,
                   "H": w.H, "G": w.G, "P": w.P, "N": w.N, "chunk": w.Q, "seed": args.seed,
                   "flops_per_step": flops, "bytes_per_step": nbytes},
        "tflops": round(flops / (ms * 1e-3) / 1e12, 2),
        "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None},
        "wall_s_timed": round(wall, 4),
    }
    if not args.no_cpu_baseline:
        # the CPU-oracle leg: spot check, then the oracle's throughput
        import oracle.ssd as ossd
        # spot check two (batch, head) slices against the oracle's own chain
        Q = w.Q
        worst = 0.0
        for b, h in ((0, 0), (w.B - 1, w.H - 1)):
            g = h // (w.H // w.G)
            sub = dict(x=inp["x"][b:b + 1, :, [h]], Bm=inp["Bm"][b:b + 1, :, [g]],
                       Cm=inp["Cm"][b:b + 1, :, [g]], dt=inp["dt"][b:b + 1, :, [h]],
                       A=inp["A"][[h]], D=inp["D"][[h]])
            if op == "chunk_scan":
                ref, _ = ossd.ssd_forward(sub["x"], sub["dt"], sub["A"], sub["Bm"], sub["Cm"], sub["D"], Q)
                ab = lambda u: np.ascontiguousarray(u) & np.uint16(0x7FFF)
                s_abs = ossd.chunk_state_abs(sub["x"], sub["Bm"], sub["dt"], sub["A"], Q)
                p_abs, _ = ossd.state_passing(s_abs, sub["dt"], sub["A"], Q)
                cb_abs = ossd.bmm_chunk(ab(sub["Cm"]), ab(sub["Bm"]), Q)
                scale = ossd.chunk_scan_abs(sub["x"], sub["Cm"], cb_abs, sub["dt"], sub["A"], p_abs,
                                            sub["D"], Q)
                got, bound = y[b:b + 1, :, [h]].cpu().numpy(), 2.0 ** -6
            else:
                ref = ossd.chunk_state(sub["x"], sub["Bm"], sub["dt"], sub["A"], Q)
                scale = ossd.chunk_state_abs(sub["x"], sub["Bm"], sub["dt"], sub["A"], Q)
                got, bound = states[b:b + 1, :, [h]].cpu().numpy(), 2.0 ** -7
            worst = max(worst, float((np.abs(got - ref) / np.maximum(scale, 1e-30)).max() / bound))
        if not worst <= 1.0:
            raise SystemExit(f"bench: result check failed (worst err/bound {worst})")
        result["check"] = {"worst_err_over_bound": worst, "slices": 2}
        # the oracle's chain on whole (batch, head) slices, about 10 s
        def one(b, h):
            g = h // (w.H // w.G)
            xs, dts = inp["x"][b:b + 1, :, [h]], inp["dt"][b:b + 1, :, [h]]
            if op == "chunk_scan":
                ossd.chunk_scan(xs, inp["Cm"][b:b + 1, :, [g]], np.zeros((1, w.nc, 1, Q, Q)), dts,
                                inp["A"][[h]], np.zeros((1, w.nc, 1, w.P, w.N)), inp["D"][[h]], Q)
            else:
                ossd.chunk_state(xs, inp["Bm"][b:b + 1, :, [g]], dts, inp["A"][[h]], Q)
        t0 = time.perf_counter()
        one(0, 0)
        t1 = max(time.perf_counter() - t0, 1e-6)
        n = int(max(1, min(w.B * w.H, 10.0 / t1)))
        t0 = time.perf_counter()
        for i in range(n):
            one(i // w.H % w.B, i % w.H)
        dt_s = time.perf_counter() - t0
        frac = n / (w.B * w.H)
        result["cpu_baseline"] = {
            "value": round(nbytes * frac / dt_s / 1e9, 3), "unit": "GB/s",
            "cores": blas_threads(), "host_cores": host_cores(), "kind": "oracle",
            "sample": f"{n} of {w.B * w.H} (batch, head) slices of {w.name}, {op}, numpy float64 "
                      f"(einsum; BLAS threads where it calls BLAS), {dt_s:.1f} s wall"}
    print(json.dumps(result), flush=True)


TARGET_WORKLOADS = ("tiny_d64_s128", "causal_d64_s1k", "dense_d128_s2k",
                    "causal_peaky_d128_s8k", "gqa4_causal_d128_s4k")


def oracle_all_configs(args):
    """The fp64 oracle timed on every output element of the five target
    configurations (no sampling), each on this host's cores; with a GPU the
    attention kernel's output is compared with it element by element.  One
    JSON line per configuration."""
    import oracle

    torch = None
    try:
        import torch as _t
        if _t.cuda.is_available():
            torch = _t
            from paper_2504_17577_amd import tileattn
    except ImportError:
        pass
    threads = oracle.default_threads()
    lib = oracle.load()
    for name in TARGET_WORKLOADS:
        w = gen.WORKLOADS[name]
        q, k, v = gen.make_inputs(w, seed=args.seed)
        t0 = time.perf_counter()
        ro, rl = oracle.attn_fwd(q, k, v, w.causal, w.scale, nthreads=threads, lib=lib)
        dt = time.perf_counter() - t0
        line = {"workload": name, "shape": w.describe(), "flops": w.flops(),
                "oracle_s": round(dt, 3), "oracle_gflops_fp64": round(w.flops() / dt / 1e9, 2),
                "cores": threads, "host_cores": host_cores(), "elements_compared": None}
        if torch is not None:
            o, lse = tileattn.attn_fwd(to_device(q, torch), to_device(k, torch),
                                       to_device(v, torch), causal=w.causal, scale=w.scale)
            torch.cuda.synchronize()
            eo = float(np.abs(o.cpu().numpy() - ro).max())
            el = float(np.abs(lse.cpu().numpy() - rl).max())
            line.update({"max_abs_dO": eo, "max_abs_dLSE": el, "elements_compared": int(ro.size),
                         "within_tolerance": bool(eo <= 2e-2 and el <= 1e-3)})
        print(json.dumps(line), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD,
                    choices=sorted(gen.WORKLOADS) + sorted(gen.MLA_WORKLOADS)
                    + sorted(gen.GEMM_WORKLOADS) + sorted(gen.SSD_WORKLOADS))
    ap.add_argument("--op", choices=("chunk_scan", "chunk_state"), default=None,
                    help="SSD workloads: the function timed (default chunk_scan)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--out", choices=("f32", "bf16"), default=None,
                    help="output dtype: attention O f32 (default, attn_fwd) or bf16 "
                         "(attn_fwd_bf16out); GEMM C bf16 (default) or f32")
    ap.add_argument("--splits", default="1",
                    help="key splits per query tile: 1 (attn_fwd), N or auto "
                         "(attn_fwd_split with ta_split_heuristic; workspace allocated "
                         "before the timed region); MLA: cache splits; matrix-vector "
                         "workloads: K splits (gemv_bf16_split, gemv_split_heuristic)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--oracle-all-configs", action="store_true",
                    help="time the fp64 oracle on every element of the five target "
                         "configurations (and compare the GPU output where there is one)")
    ap.add_argument("--copy-probe", action="store_true")
    ap.add_argument("--sustain", type=float, default=0.0,
                    help="also run the step back to back for this many seconds while "
                         "sampling board power and XCD clocks (amd-smi)")
    ap.add_argument("--gemm-reference", action="store_true",
                    help="with --sustain: the same for a bf16 8192^3 torch.matmul, as a "
                         "reference for what the matrix cores sustain at the power limit")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the attention forward here has no multi-GPU "
              f"path (asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)

    if args.oracle_all_configs:
        oracle_all_configs(args)
        return

    import torch

    from paper_2504_17577_amd import tileattn

    if args.copy_probe:
        copy_probe(torch)
        return
    if args.workload in gen.MLA_WORKLOADS:
        bench_mla(args, torch, tileattn)
        return
    if args.workload in gen.GEMM_WORKLOADS:
        bench_gemm(args, torch, tileattn)
        return
    if args.workload in gen.SSD_WORKLOADS:
        bench_ssd(args, torch, tileattn)
        return
    if args.out is None:
        args.out = "f32"

    w = gen.WORKLOADS[args.workload]
    q, k, v = gen.make_inputs(w, seed=args.seed)
    dq, dk, dv = to_device(q, torch), to_device(k, torch), to_device(v, torch)
    o_bf16 = args.out == "bf16"
    o = torch.empty((w.B, w.Hq, w.Sq, w.D), dtype=torch.bfloat16 if o_bf16 else torch.float32,
                    device="cuda")
    lse = torch.empty((w.B, w.Hq, w.Sq), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()

    n_split = (tileattn.ta_split_heuristic(w.B, w.Hq, w.Hkv, w.Sq, w.Sk, w.D, w.causal)
               if args.splits == "auto" else int(args.splits))
    if n_split > 1:
        ws = torch.empty(max(16, tileattn.ta_split_workspace_bytes(w.B, w.Hq, w.Sq, w.D, n_split)),
                         dtype=torch.uint8, device="cuda")
        o_dt = torch.bfloat16 if o_bf16 else torch.float32

        def step():
            tileattn.attn_fwd_split(dq, dk, dv, causal=w.causal, scale=w.scale,
                                    num_splits=n_split, out=o, lse=lse, workspace=ws,
                                    out_dtype=o_dt, stream=stream)
    else:
        fwd = tileattn.attn_fwd_bf16out if o_bf16 else tileattn.attn_fwd

        def step():
            fwd(dq, dk, dv, causal=w.causal, scale=w.scale, out=o, lse=lse, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # timed region: K launches on this stream between two HIP events, with
    # events between five equal sub-batches as well (recorded on the stream,
    # no synchronisation inside the region): the board's power management
    # lowers the clock for the first tens of launches after idle, and the
    # sub-batch times show where the timed region sat on that curve
    n_b = 5 if args.steps >= 5 else 1
    cuts = [round(i * args.steps / n_b) for i in range(n_b + 1)]
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(n_b + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    evs[0].record(stream)
    for i in range(n_b):
        for _ in range(cuts[i + 1] - cuts[i]):
            step()
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = evs[0].elapsed_time(evs[-1]) / args.steps
    batch_ms = [evs[i].elapsed_time(evs[i + 1]) / (cuts[i + 1] - cuts[i]) for i in range(n_b)]
    tflops = w.flops() / (ms * 1e-3) / 1e12

    traffic = None if (o_bf16 or n_split > 1) else read_traffic(w.name)
    result = {
        "metric": METRIC,
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "out_dtype": args.out,
        "splits": n_split,
        "data": "synthetic",
        "config": {"workload": w.name, "shape": w.describe(), "B": w.B, "Hq": w.Hq, "Hkv": w.Hkv,
                   "Sq": w.Sq, "Sk": w.Sk, "D": w.D, "causal": w.causal, "seed": args.seed,
                   "flops_per_step": w.flops(), "inputs_blake2b": gen.digest(q)[:8] +
                   gen.digest(k)[:8] + gen.digest(v)[:8]},
        "pct_of_peak": round(100 * tflops / PEAK_BF16_TFLOPS, 2),
        "roofline": {
            "bound": "mfma",
            "achieved": round(tflops, 2),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(tflops / PEAK_BF16_TFLOPS, 4),
            "traffic": traffic,
            "hbm_gbs_algorithmic": round(w.bytes(2 if o_bf16 else 4) / (ms * 1e-3) / 1e9, 1),
        },
        "wall_s_timed": round(wall, 4),
        "timed_sub_batches": {"launches": [cuts[i + 1] - cuts[i] for i in range(n_b)],
                              "ms_per_launch": [round(x, 5) for x in batch_ms],
                              "median_ms": round(float(np.median(batch_ms)), 5)},
    }
    counters = None if (o_bf16 or n_split > 1) else read_counters(w.name, ms)
    result["counters"] = counters
    if args.sustain > 0:
        with PowerSampler() as sampler:
            result["sustained"] = sustained(torch, step, w.flops(), args.sustain, sampler)
            if args.gemm_reference:
                time.sleep(2.0)
                n = 8192
                ga = torch.randn(n, n, device="cuda", dtype=torch.bfloat16)
                gb = torch.randn(n, n, device="cuda", dtype=torch.bfloat16)
                gc = torch.empty_like(ga)
                result["sustained_gemm_reference"] = {
                    "op": f"torch.matmul bf16 {n}x{n}x{n}",
                    **sustained(torch, lambda: torch.matmul(ga, gb, out=gc), 2.0 * n ** 3,
                                args.sustain, sampler)}
    if not args.no_cpu_baseline:
        # the CPU-oracle leg: a spot check of a few rows (so that a broken
        # build cannot post a number), then the oracle's own throughput on
        # whole heads, whose rows are compared as well
        import oracle
        rows = [(0, 0, 0), (w.B - 1, w.Hq - 1, w.Sq - 1), (w.B // 2, w.Hq // 2, w.Sq // 2)]
        ro, rl = oracle.attn_rows(q, k, v, w.causal, w.scale, rows)
        idx = tuple(torch.tensor(c) for c in zip(*rows))
        err_o = float(np.abs(o[idx].float().cpu().numpy() - ro).max())
        err_l = float(np.abs(lse[idx].cpu().numpy() - rl).max())
        if not (err_o <= 2e-2 and err_l <= 1e-3):
            raise SystemExit(f"bench: result check failed (max|dO|={err_o}, max|dLSE|={err_l})")
        info, rows, ro, rl = cpu_baseline(w, q, k, v)
        # the rows the oracle leg computed, every element of them, against
        # the output of the last timed launch
        idx = tuple(torch.from_numpy(np.ascontiguousarray(rows[:, c])) for c in range(3))
        err_o = max(err_o, float(np.abs(o[idx].float().cpu().numpy() - ro).max()))
        err_l = max(err_l, float(np.abs(lse[idx].cpu().numpy() - rl).max()))
        if not (err_o <= 2e-2 and err_l <= 1e-3):
            raise SystemExit(f"bench: result check failed (max|dO|={err_o}, max|dLSE|={err_l})")
        result["check"] = {"max_abs_dO": err_o, "max_abs_dLSE": err_l, "rows": 3 + len(rows)}
        result["cpu_baseline"] = info
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
