"""Benchmark of the dilated-attention forward pass on one MI355X.

One step = one dilated_attn_fwd call over the N=32768, H=12, D=64 bf16
workload with the five patterns (2048,1) (4096,2) (8192,4) (16384,6)
(32768,12), inputs resident in HBM.  The call is two launches: the attention
kernel over every pattern, then the kernel that mixes the patterns.

Prints one JSON line: effective TFLOP/s over the exact sparse flops (4*D per
unmasked query-key pair) and tokens/s of the timed back-to-back steps, the
times of the call's two launches from a second pass in which the library
records HIP events around them on the call's stream, the attention kernel's
MFMA roofline fraction and the combine kernel's HBM bandwidth, and the CPU
oracle timed on a bounded sample on this host.  Every timed region follows at
least --warmup-seconds of untimed calls.  After the timed region, a further
pass times each step on its own (median, minimum, mean), once as is and once
with a 512 MiB buffer written before each step so that the inputs are no
longer held in the Infinity Cache.  Then the same call is timed on the
N=262144 (H=16, D=64, 8 patterns) and N=1048576 (H=16, D=128, 6 patterns)
workloads, whose per-pattern workspaces (1.1 and 8.7 GB) are far larger than
the 256 MB Infinity Cache: their combine launch gives the combine's HBM rate.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "dilated-attn fwd effective TFLOP/s + tokens/s at N=32K, MFMA util %"
DEFAULT_WORKLOAD = "n32k_h12_d64_5pat"
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3       # MI355X fp32 vector
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E
PROFILED_TRAFFIC = os.path.join(ROOT, "profiles", "traffic.json")
# Sources of the two forward kernels whose hashes key the profiled figures.
PROFILED_SOURCES = ("attn_fwd.hip", "combine.hip", "device_common.h", "kernels.h")


def parse():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--warmup-seconds", type=float, default=1.0,
                    help="untimed calls continue until at least this long has passed (the GPU raises "
                         "its clocks only after some time under load)")
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="minimum CPU time spent on the oracle sample (0 skips the CPU baseline)")
    ap.add_argument("--dist-steps", type=int, default=20,
                    help="steps of the per-step pass (unflushed and flushed each); 0 skips it")
    ap.add_argument("--large", default="n256k_h16_d64_8pat_geo,n1m_h16_d128_6pat",
                    help="comma-separated workloads also timed (call, attention and combine launches) after "
                         "the benchmark workload; empty skips them")
    ap.add_argument("--sweep", action="store_true",
                    help="instead of the benchmark: the dense-versus-dilated sweep over N = 8K..1M "
                         "(fixed tokens per batch), one JSON line per (N, variant)")
    ap.add_argument("--backward", action="store_true",
                    help="instead of the benchmark: time the backward pass on the workload, one JSON line")
    ap.add_argument("--layer", action="store_true",
                    help="time the LongNet attention layer (LayerNorm, projections, xPos, dilated attention, "
                         "sub-LayerNorm, output projection) forward and forward+backward on the workload's "
                         "shape instead")
    ap.add_argument("--per-pattern", action="store_true",
                    help="instead of the benchmark: each pattern of the workload run alone (a one-pattern "
                         "forward call), its attention launch timed against the MFMA peak; one JSON line "
                         "per pattern (under a profiler each pattern's launches are separate dispatches)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="only run a plain device-to-device copy of this many MiB (5 times), to "
                         "calibrate the HBM byte counters of a profiler against a known size")
    return ap.parse_args()


def copy_calibration(mib):
    """A plain copy of a known number of bytes (read mib MiB, write mib MiB),
    five launches for the counters, then the same copy timed back to back
    after a warm-up (bytes read plus bytes written per second): the HBM rate
    a streaming kernel of that size reaches in practice."""
    import torch
    x = torch.ones(mib * (1 << 20) // 4, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    for _ in range(5):
        y.copy_(x)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < 1.0:
        y.copy_(x)
        torch.cuda.synchronize()
    reps = max(5, int(2e10 // (mib << 20)))
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        y.copy_(x)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    print(json.dumps({"copy_calibration_bytes_each_way": mib * (1 << 20), "launches": 5, "timed_copies": reps,
                      "ms_per_copy": round(ms, 5), "gbps_read_plus_write": round(2 * (mib << 20) / (ms * 1e-3) / 1e9, 1)}),
          flush=True)


def profiled_counters(workload):
    """Per-launch figures measured with rocprofv3 counters for the current
    kernel sources: HBM bytes of the attention and combine kernels
    (FETCH_SIZE / WRITE_SIZE scaled by a plain copy of known size) and the
    attention kernel's MFMA busy percentage.  Empty when a source of the
    attention or the combine kernel changed since the measurement."""
    import hashlib
    if not os.path.exists(PROFILED_TRAFFIC):
        return {}
    with open(PROFILED_TRAFFIC) as f:
        rec = json.load(f).get(workload)
    if not rec:
        return {}
    for name in PROFILED_SOURCES:
        with open(os.path.join(ROOT, "paper_2307_02486_amd", "csrc", name), "rb") as f:
            sha = hashlib.sha256(f.read()).hexdigest()[:16]
        if sha != rec.get(name.replace(".", "_") + "_sha256_16"):
            return {}
    return rec


def step_distribution(step, stream, steps, flush_bytes):
    """Times `steps` single steps with events around each one; with
    flush_bytes > 0 a buffer of that size is written before every step."""
    import statistics

    import torch
    scratch = torch.empty(flush_bytes // 4, dtype=torch.float32, device=stream.device) if flush_bytes else None
    times = []
    for i in range(steps):
        if scratch is not None:
            scratch.fill_(float(i))
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        step()
        e1.record(stream)
        e1.synchronize()
        times.append(e0.elapsed_time(e1))
    return {"median_ms": round(statistics.median(times), 5), "min_ms": round(min(times), 5),
            "mean_ms": round(statistics.fmean(times), 5), "steps": steps}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(wl, q, k, v, min_seconds):
    """Time the CPU oracle, as it stands, on whole heads of the same workload
    until at least `min_seconds` have passed; report flops/s over those heads."""
    import numpy as np

    import oracle
    try:
        from threadpoolctl import threadpool_info
        pools = threadpool_info()
        threads = max((p.get("num_threads", 1) for p in pools), default=1)
        blas = ",".join(sorted({p.get("internal_api", "?") for p in pools}))
    except Exception:  # threadpoolctl missing or failing: report the affinity count
        threads, blas = len(os.sched_getaffinity(0)), "unknown"
    q64 = q.to("cpu").double().numpy()
    k64 = k.to("cpu").double().numpy()
    v64 = v.to("cpu").double().numpy()
    pats = list(wl.patterns)
    done, flops = [], 0
    t0 = time.perf_counter()
    for h in range(wl.H):
        oracle.dilated_attention_ref(q64, k64, v64, pats, wl.causal, heads=[h])
        done.append(h)
        flops += 4 * wl.D * wl.B * sum(
            (L * (L + 1) // 2 if wl.causal else L * L)
            for (w, r) in pats for g in range(oracle.num_segments(wl.N, w))
            for L in [oracle.index_set(wl.N, w, r, h, g).size])
        if time.perf_counter() - t0 >= min_seconds:
            break
    dt = time.perf_counter() - t0
    return {
        "value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
        "sample": f"{len(done)} of {wl.H} heads of {wl.name} (all patterns, all rows), fp64 NumPy "
                  f"({blas}), {dt:.1f} s",
        "tokens_per_s": wl.B * wl.N * len(done) / wl.H / dt,
        "host_cpus": len(os.sched_getaffinity(0)),
        "cpu_model": cpu_model(),
    }


def sweep(args):
    """Dense (w = N, r = 1) and dilated ({(2048, 1), (N, N/2048)}) forward
    passes at a fixed 2^20 tokens per batch for N = 8K .. 1M; per (N, variant)
    the median of `steps` timed calls (events on the call's stream) after
    `warmup` calls."""
    import statistics

    import torch

    import workloads
    from paper_2307_02486_amd import dilated_attn, plan, workspace_for
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)
    steps, warm = max(1, min(args.steps, 5)), max(1, min(args.warmup, 2))
    for N in workloads.SWEEP_N:
        for variant in ("dense", "dilated"):
            wl = workloads.sweep_workload(N, variant)
            q, k, v = workloads.make_qkv(wl, device=dev)
            pats = list(wl.patterns)
            info = plan(wl.B, wl.N, wl.H, wl.D, pats, wl.causal, wl.torch_dtype)
            out = torch.empty_like(q)
            lse = torch.empty((wl.B, wl.H, wl.N), dtype=torch.float32, device=dev)
            ws = workspace_for(q, pats, wl.causal)
            t0, n = time.perf_counter(), 0
            while n < warm or time.perf_counter() - t0 < min(args.warmup_seconds, 0.5):
                dilated_attn(q, k, v, pats, wl.causal, out=out, lse=lse, workspace=ws, stream=stream)
                torch.cuda.synchronize()
                n += 1
            times = []
            for _ in range(steps):
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                dilated_attn(q, k, v, pats, wl.causal, out=out, lse=lse, workspace=ws, stream=stream)
                e1.record(stream)
                e1.synchronize()
                times.append(e0.elapsed_time(e1))
            ms = statistics.median(times)
            print(json.dumps({"sweep": "dense-vs-dilated", "variant": variant, "N": N, "B": wl.B,
                              "H": wl.H, "D": wl.D, "dtype": "bf16", "patterns": [list(p) for p in pats],
                              "median_ms": round(ms, 4), "min_ms": round(min(times), 4), "steps": steps,
                              "sparse_flops": info["sparse_flops"],
                              "tflops": round(info["sparse_flops"] / (ms * 1e-3) / 1e12, 2),
                              "tokens_per_s": round(wl.B * wl.N / (ms * 1e-3), 1)}), flush=True)
            del q, k, v, out, lse, ws
            torch.cuda.empty_cache()


def backward(args):
    """Backward pass on the workload: `warmup` untimed calls, then `steps`
    back-to-back calls timed with events on the stream; effective TFLOP/s over
    10*D per unmasked pair (the five products of the derivative)."""
    import statistics

    import torch

    import workloads
    from paper_2307_02486_amd import bwd_workspace_for, dilated_attn, dilated_attn_bwd, plan_bwd
    wl = workloads.BY_NAME[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)
    q, k, v = workloads.make_qkv(wl, device=dev)
    dout = workloads.make_random(q.shape, wl.torch_dtype, 1.0, wl.seed, dev, 3)
    pats = list(wl.patterns)
    out, lse = dilated_attn(q, k, v, pats, wl.causal, stream=stream)
    info = plan_bwd(wl.B, wl.N, wl.H, wl.D, pats, wl.causal, wl.torch_dtype)
    ws = bwd_workspace_for(q, pats, wl.causal)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(q), torch.empty_like(q)

    def step():
        dilated_attn_bwd(q, k, v, out, lse, dout, pats, wl.causal, dq=dq, dk=dk, dv=dv, workspace=ws, stream=stream)

    t0, n = time.perf_counter(), 0
    while n < args.warmup or time.perf_counter() - t0 < args.warmup_seconds:
        step()
        n += 1
        torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    single = []
    for _ in range(min(args.steps, 20)):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        step()
        b.record(stream)
        b.synchronize()
        single.append(a.elapsed_time(b))
    flops = info["sparse_flops"]
    print(json.dumps({"metric": "dilated-attn bwd effective TFLOP/s (10*D per unmasked pair)",
                      "value": round(flops / (ms * 1e-3) / 1e12, 3), "unit": "TFLOP/s", "ms_per_step": round(ms, 5),
                      "steps": args.steps, "warmup": args.warmup, "dtype": wl.dtype, "config": wl.describe(),
                      "flops": flops, "tokens_per_s": round(wl.B * wl.N / (ms * 1e-3), 1),
                      "isolated_step_ms": {"median": round(statistics.median(single), 5),
                                           "min": round(min(single), 5)},
                      "algorithmic_bytes": {"gradient_kernels": info["bytes_attn"],
                                            "delta_and_sum_kernels": info["bytes_combine"]}}), flush=True)


def layer(args):
    """The LongNet attention layer on the workload's shape (E = H * D, bf16,
    random-init parameters): forward, and forward + backward, per step; the
    dilated attention's own forward and backward on the same q, k, v; and
    the xPos kernel's bandwidth (read + write of one [B, N, H, D] tensor)."""
    import torch

    import workloads
    from paper_2307_02486_amd import dilated_attn, dilated_attn_bwd, wgrad, xpos
    from paper_2307_02486_amd.layer import LongNetAttention

    wl = workloads.BY_NAME[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    E = wl.H * wl.D
    torch.manual_seed(0)
    mod = LongNetAttention(E, wl.H, list(wl.patterns), wl.causal, device=dev, dtype=wl.torch_dtype)
    x = workloads.make_random((wl.B, wl.N, E), wl.torch_dtype, 1.0, wl.seed, dev, 0).requires_grad_(True)
    dy = workloads.make_random((wl.B, wl.N, E), wl.torch_dtype, 1.0, wl.seed, dev, 1)
    q, k, v = workloads.make_qkv(wl, device=dev)
    pats = list(wl.patterns)

    def fwd():
        with torch.no_grad():
            mod(x)

    def fwd_bwd():
        mod(x).backward(dy)

    def attn_fwd():
        dilated_attn(q, k, v, pats, wl.causal)

    out, lse = dilated_attn(q, k, v, pats, wl.causal)

    def attn_bwd():
        dilated_attn_bwd(q, k, v, out, lse, q, pats, wl.causal)

    xo = torch.empty_like(q)

    def xp():
        xpos(q, 1, out=xo)

    dy2, x2 = dy.view(-1, E), x.detach().view(-1, E)
    wo = torch.empty((E, E), dtype=dy.dtype, device=dev)

    def wg():
        wgrad(dy2, x2, out=wo)

    def wg_torch():
        torch.mm(dy2.t(), x2)

    def timed(fn, steps):
        t0, n = time.perf_counter(), 0
        while n < args.warmup or time.perf_counter() - t0 < args.warmup_seconds:
            fn()
            n += 1
            torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    steps = max(1, args.steps)
    ms_f, ms_fb = timed(fwd, steps), timed(fwd_bwd, steps)
    ms_af, ms_ab = timed(attn_fwd, steps), timed(attn_bwd, steps)
    ms_x = timed(xp, steps)
    ms_w, ms_wt = timed(wg, steps), timed(wg_torch, steps)
    tok = wl.B * wl.N
    w_flop = 2.0 * tok * E * E
    x_bytes = 2 * q.numel() * q.element_size()
    print(json.dumps({
        "metric": "LongNet attention layer fwd / fwd+bwd tokens/s", "workload": wl.describe(), "embed_dim": E,
        "dtype": wl.dtype, "steps": steps, "layer_fwd_ms": round(ms_f, 4), "layer_fwd_bwd_ms": round(ms_fb, 4),
        "fwd_tokens_per_s": round(tok / (ms_f * 1e-3), 1), "fwd_bwd_tokens_per_s": round(tok / (ms_fb * 1e-3), 1),
        "dilated_attn_fwd_ms": round(ms_af, 4), "dilated_attn_bwd_ms": round(ms_ab, 4),
        "attention_share_of_fwd_bwd": round((ms_af + ms_ab) / ms_fb, 3),
        "xpos_ms": round(ms_x, 5), "xpos_gbps": round(x_bytes / (ms_x * 1e-3) / 1e9, 1),
        "wgrad_ms": round(ms_w, 5), "wgrad_tflops": round(w_flop / (ms_w * 1e-3) / 1e12, 1),
        "torch_mm_wgrad_ms": round(ms_wt, 5)}), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: this benchmark runs on one GPU only (asked for --gpus {args.gpus}); "
              "the sequence-parallel multi-GPU path is not built", file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration_mib > 0:
        copy_calibration(args.copy_calibration_mib)
        return
    if args.sweep:
        sweep(args)
        return
    if args.backward:
        backward(args)
        return
    if args.layer:
        layer(args)
        return
    if args.per_pattern:
        per_pattern(args)
        return
    import torch

    import workloads
    from paper_2307_02486_amd import StageTimer, dilated_attn, plan, workspace_for

    if not torch.cuda.is_available():
        print("bench.py: no HIP device visible", file=sys.stderr)
        sys.exit(1)
    wl = workloads.BY_NAME[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    q, k, v = workloads.make_qkv(wl, device=dev)
    pats = list(wl.patterns)
    info = plan(wl.B, wl.N, wl.H, wl.D, pats, wl.causal, wl.torch_dtype)
    out = torch.empty_like(q)
    lse = torch.empty((wl.B, wl.H, wl.N), dtype=torch.float32, device=dev)
    ws = workspace_for(q, pats, wl.causal)
    stream = torch.cuda.current_stream(dev)

    def step():
        dilated_attn(q, k, v, pats, wl.causal, out=out, lse=lse, workspace=ws, stream=stream)

    def warm():
        """At least `warmup` untimed calls, and calls for at least
        `warmup_seconds`: a short warm-up leaves the GPU at a lower clock and
        the first timed region up to 10 % slower than later ones."""
        t0 = time.perf_counter()
        n = 0
        while n < args.warmup or time.perf_counter() - t0 < args.warmup_seconds:
            for _ in range(5):
                step()
            n += 5
            torch.cuda.synchronize()

    def timed(steps):
        """Mean ms per call over `steps` back-to-back calls, then the mean ms
        of the call's two launches over as many calls again."""
        warm()
        t_start = torch.cuda.Event(enable_timing=True)
        t_end = torch.cuda.Event(enable_timing=True)
        # Timed region: exactly `steps` back-to-back calls, nothing else on the stream.
        t_start.record(stream)
        for _ in range(steps):
            step()
        t_end.record(stream)
        torch.cuda.synchronize()
        ms = t_start.elapsed_time(t_end) / steps
        # The library records HIP events around its two launches on the call's stream.
        with StageTimer(capacity=max(1, steps)) as st:
            for _ in range(steps):
                step()
            torch.cuda.synchronize()
        return ms, st.ms_attention / max(1, st.calls), st.ms_combine / max(1, st.calls)

    flops = info["sparse_flops"]
    peak = PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_F32_TFLOPS
    ms, ms_attn, ms_comb = timed(args.steps)
    prof = profiled_counters(wl.name)
    tflops = flops / (ms * 1e-3) / 1e12
    attn_tflops = flops / (ms_attn * 1e-3) / 1e12
    comb_gbs = info["bytes_combine"] / (ms_comb * 1e-3) / 1e9
    res = {
        "metric": METRIC,
        "value": round(tflops, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic (seeded N(0, sigma^2), rounded to dtype)",
        "config": wl.describe(),
        "tokens_per_s": round(wl.B * wl.N / (ms * 1e-3), 1),
        "sparse_flops": flops,
        "launches": {"attention_ms": round(ms_attn, 5), "combine_ms": round(ms_comb, 5)},
        "attention_stage": {"ms": round(ms_attn, 5), "tflops": round(attn_tflops, 3),
                            "frac_of_mfma_peak": round(attn_tflops / peak, 4),
                            "algorithmic_bytes": info["bytes_attn"],
                            "mfma_busy_pct_profiled": prof.get("attention_mfma_busy_pct")},
        "combine_stage": {"ms": round(ms_comb, 5), "algorithmic_bytes": info["bytes_combine"],
                          "gbps": round(comb_gbs, 1), "frac_of_hbm_peak": round(comb_gbs / PEAK_HBM_GBS, 4),
                          "traffic": prof.get("combine_bytes_per_launch"),
                          "note": "workspace of this size can be held in the 256 MB Infinity Cache; "
                                  "see large_workloads for the combine's HBM rate"},
        "roofline": {"bound": "mfma", "achieved": round(attn_tflops, 3), "peak": peak,
                     "unit": "TFLOP/s", "frac": round(attn_tflops / peak, 4),
                     "traffic": prof.get("attention_bytes_per_launch")},
        "cpu_baseline": None,
    }
    # Host side of one call (Python binding, ctypes, plan, two launches): the
    # GPU is kept busy by a queue of calls, so enqueueing never waits on it.
    warm()
    for _ in range(20):
        step()
    n_host = 100
    t0 = time.perf_counter()
    for _ in range(n_host):
        step()
    host_us = (time.perf_counter() - t0) / n_host * 1e6
    torch.cuda.synchronize()
    res["host_us_per_call"] = round(host_us, 2)
    if args.dist_steps > 0:
        warm()
        res["step_distribution"] = {
            "unflushed": step_distribution(step, stream, args.dist_steps, 0),
            "flushed_512MiB": step_distribution(step, stream, args.dist_steps, 512 << 20),
        }
    if args.cpu_seconds > 0:
        res["cpu_baseline"] = cpu_baseline(wl, q, k, v, args.cpu_seconds)
    names = [n for n in args.large.split(",") if n and n != wl.name]
    if names:
        del q, k, v, out, lse, ws
        torch.cuda.empty_cache()
        res["large_workloads"] = [large_workload(workloads.BY_NAME[n], args) for n in names]
    print(json.dumps(res), flush=True)


def per_pattern(args):
    """Each (w, r) of the workload as a one-pattern problem: the attention
    launch's mean duration over back-to-back calls after the warm-up, its
    sparse FLOPs and the fraction of the MFMA peak.  The patterns run in the
    workload's order, `steps` timed calls each."""
    import torch

    import workloads
    from paper_2307_02486_amd import StageTimer, dilated_attn, plan, workspace_for
    wl = workloads.BY_NAME[args.workload]
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    q, k, v = workloads.make_qkv(wl, device=dev)
    out = torch.empty_like(q)
    lse = torch.empty((wl.B, wl.H, wl.N), dtype=torch.float32, device=dev)
    peak = PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_F32_TFLOPS
    for (w, r) in wl.patterns:
        pats = [(w, r)]
        info = plan(wl.B, wl.N, wl.H, wl.D, pats, wl.causal, wl.torch_dtype)
        ws = workspace_for(q, pats, wl.causal)

        def step():
            dilated_attn(q, k, v, pats, wl.causal, out=out, lse=lse, workspace=ws, stream=stream)

        t0, n = time.perf_counter(), 0
        while n < args.warmup or time.perf_counter() - t0 < args.warmup_seconds:
            step()
            n += 1
            torch.cuda.synchronize()
        with StageTimer(capacity=args.steps) as st:
            for _ in range(args.steps):
                step()
            torch.cuda.synchronize()
        ms_attn = st.ms_attention / st.calls
        tf = info["sparse_flops"] / (ms_attn * 1e-3) / 1e12
        print(json.dumps({"workload": wl.name, "pattern": [w, r], "work_items": info["num_work_items"],
                          "sparse_flops": info["sparse_flops"], "attention_ms": round(ms_attn, 5),
                          "tflops": round(tf, 3), "frac_of_mfma_peak": round(tf / peak, 4),
                          "calls": st.calls}), flush=True)
        del ws
        torch.cuda.empty_cache()


def large_workload(wl, args):
    """One more workload: mean ms per call over back-to-back calls after the
    warm-up, then the mean of each launch over as many calls (events recorded
    by the library around its two launches), the attention launch against
    the MFMA peak and the combine launch's algorithmic bytes against the HBM
    peak.  Its workspace is far larger than the Infinity Cache."""
    import torch

    import workloads
    from paper_2307_02486_amd import StageTimer, dilated_attn, plan, workspace_for
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    q, k, v = workloads.make_qkv(wl, device=dev)
    pats = list(wl.patterns)
    info = plan(wl.B, wl.N, wl.H, wl.D, pats, wl.causal, wl.torch_dtype)
    out = torch.empty_like(q)
    lse = torch.empty((wl.B, wl.H, wl.N), dtype=torch.float32, device=dev)
    ws = workspace_for(q, pats, wl.causal)

    def step():
        dilated_attn(q, k, v, pats, wl.causal, out=out, lse=lse, workspace=ws, stream=stream)

    t0, n = time.perf_counter(), 0
    while n < 3 or time.perf_counter() - t0 < args.warmup_seconds:
        step()
        n += 1
        torch.cuda.synchronize()
    calls = max(3, min(args.steps, int(2000.0 / max(1.0, 1e3 * (time.perf_counter() - t0) / n))))
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(calls):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / calls
    with StageTimer(capacity=calls) as st:
        for _ in range(calls):
            step()
        torch.cuda.synchronize()
    ms_attn, ms_comb = st.ms_attention / st.calls, st.ms_combine / st.calls
    flops = info["sparse_flops"]
    attn_tflops = flops / (ms_attn * 1e-3) / 1e12
    comb_gbs = info["bytes_combine"] / (ms_comb * 1e-3) / 1e9
    prof = profiled_counters(wl.name)
    rec = {"config": wl.describe(), "calls": calls, "ms_per_call": round(ms, 4),
           "tflops": round(flops / (ms * 1e-3) / 1e12, 3), "tokens_per_s": round(wl.B * wl.N / (ms * 1e-3), 1),
           "sparse_flops": flops, "workspace_bytes": info["workspace_bytes"],
           "attention_stage": {"ms": round(ms_attn, 4), "tflops": round(attn_tflops, 3),
                               "frac_of_mfma_peak": round(attn_tflops / PEAK_BF16_TFLOPS, 4),
                               "algorithmic_bytes": info["bytes_attn"],
                               "traffic": prof.get("attention_bytes_per_launch"),
                               "mfma_busy_pct_profiled": prof.get("attention_mfma_busy_pct")},
           "combine_stage": {"ms": round(ms_comb, 4), "algorithmic_bytes": info["bytes_combine"],
                             "gbps": round(comb_gbs, 1), "frac_of_hbm_peak": round(comb_gbs / PEAK_HBM_GBS, 4),
                             "traffic": prof.get("combine_bytes_per_launch")}}
    del q, k, v, out, lse, ws
    torch.cuda.empty_cache()
    return rec


if __name__ == "__main__":
    main()
