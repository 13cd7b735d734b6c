#!/usr/bin/env python3
"""Throughput of one aggregation step of the unbiased max-norm quantisers
(arXiv 2109.12497, Algorithms 1-2) on one MI355X.

A step is the whole hot path over M workers' gradients resident in HBM:
shared max-norm scale (+ shared scale index) -> quantise every worker ->
integer sum of the codes -> reconstruct the averaged gradient.  The metric is
gradient elements (M * d worker-coordinates) per second, and the fraction of
the 8 TB/s HBM peak the step's algorithmic bytes reach.

Prints one JSON line.  Extra modes:
  --workload NAME       another workload of synth.WORKLOADS (default resnet18)
  --graph               time replays of the step captured in a HIP graph
  --no-cpu-baseline     skip the oracle leg (for profiling runs)
  --copy-probe BYTES    time and run only a plain device copy (counter calibration)
  --stream-probe        achievable bandwidth of the hot path's access patterns
                        with no work, on the workload's gradients
"""
import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "G gradient elements/s quantize+sum+dequantize; % of HBM peak GB/s"
HBM_PEAK_GBS = 8000.0
# workers up to which the shared scale takes the fused norm + row-maximum pass
FUSED_MAX_ROWS = 16
KERNEL_SOURCES = ["paper_2109_12497_amd/csrc/uq_kernels.hip", "paper_2109_12497_amd/csrc/uq_device.hpp"]


def code_bytes(d: int, bits: int) -> int:
    return (d * bits + 7) // 8


def quantize_bytes_per_launch(d: int, rows: int, K: int, bits: int = 8) -> int:
    """One quantiser launch over `rows` workers: their gradients in, their
    codes out, and (several scales) the shared index, needed once."""
    return rows * (4 * d + code_bytes(d, bits)) + (d if K > 1 else 0)


def algorithmic_bytes(d: int, M: int, K: int, streamed: bool, bits: int = 8) -> dict:
    """Bytes each stage must move at minimum (reads + writes), per step.  With
    several scales and 2 to 16 workers the norm pass also writes the
    largest |g| over the workers (4 bytes per coordinate), which the index
    pass reads instead of the gradients; with more workers the index pass
    reads every gradient again.  The sum stores the int32 sums and, in the
    same pass, the reconstruction (the sums are not read back)."""
    multi = K > 1
    cb = code_bytes(d, bits)
    if not multi:
        scale_bytes = 4 * M * d
    elif 2 <= M <= FUSED_MAX_ROWS:
        scale_bytes = 4 * M * d + 4 * d + 4 * d + d
    else:
        scale_bytes = 4 * M * d + 4 * M * d + d
    b = {
        "shared_scale": scale_bytes,
        "quantize": ((M * quantize_bytes_per_launch(d, 1, K, bits)) if streamed
                     else quantize_bytes_per_launch(d, M, K, bits)),
        "sum_dequantize": (((M * cb + 4 * d) if not streamed else (cb + 4 * d) + (M - 1) * (cb + 8 * d)) +
                           d * (4 + (1 if multi else 0))),
    }
    b["total"] = sum(b.values())
    return b


def _code_of(text: str) -> str:
    """The kernel source without its comments and with whitespace runs
    collapsed: counters stay tied to the code, not to its comments."""
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def source_digest() -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), encoding="utf-8") as f:
            h.update(_code_of(f.read()).encode())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch from the committed counter summary, or None when
    there is none or the kernel sources changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_counters.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"^traffic_bytes_per_launch:\s*([0-9.eE+]+)", text, re.M)
    s = re.search(r"^source_digest:\s*([0-9a-f]+)", text, re.M)
    if not m or not s or s.group(1) != source_digest():
        return None
    return float(m.group(1))


def stream_probe(workload: str, reps: int) -> None:
    """Achievable bandwidth of the hot path's two access patterns with no work,
    on the workload's gradient buffer: the norm pass (read M*d floats) and the
    quantiser (read M*d floats, write M*d bytes).  Kernels from libuq_probe.so,
    timed back to back between events."""
    import ctypes

    import torch

    import synth

    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2109_12497_amd", "libuq_probe.so"))
    P, i64 = ctypes.c_void_p, ctypes.c_int64
    lib.uqp_read.argtypes = [P, i64, P, P]
    lib.uqp_read_write8.argtypes = [P, i64, P, P]
    lib.uqp_read_out_floats.argtypes = [i64]
    lib.uqp_read_out_floats.restype = i64
    g, cfg = synth.make_gradients(workload, device="cuda")
    n = g.numel() // 512 * 512
    codes = torch.empty(n, dtype=torch.uint8, device="cuda")
    out = torch.empty(int(lib.uqp_read_out_floats(n)), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    h = stream.cuda_stream

    def timed(fn):
        for _ in range(max(20, reps // 4)):
            assert fn() == 0
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(reps):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps * 1e-3

    t_r = timed(lambda: lib.uqp_read(g.data_ptr(), n, out.data_ptr(), h))
    t_rw = timed(lambda: lib.uqp_read_write8(g.data_ptr(), n, codes.data_ptr(), h))
    print(json.dumps({"stream_probe": workload, "elements": n,
                      "read_GBps": round(4 * n / t_r / 1e9, 1), "read_us": round(t_r * 1e6, 2),
                      "read4_write1_GBps": round(5 * n / t_rw / 1e9, 1), "read4_write1_us": round(t_rw * 1e6, 2)}))


def copy_probe(nbytes: int) -> None:
    import torch

    n = nbytes // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    reps = 10
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / reps
    print(json.dumps({"copy_probe_bytes": nbytes, "read_plus_write_GBps": 2 * nbytes / dt / 1e9}))


def stage_ms_per_call(torch, stream, fn, reps: int, rounds: int = 3) -> float:
    """GPU time per call (ms) of fn repeated back to back between two events
    on `stream`, its inputs already in place.  Best of `rounds` rounds: a
    round in which the host fell behind the GPU (a stall in the runtime's
    launch path) reads high, so the lowest round is the stage's own time."""
    best = float("inf")
    for _ in range(rounds):
        fn()
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(reps):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        best = min(best, a.elapsed_time(b) / reps)
    return best


def stage_reps(steps: int, step_s: float) -> int:
    """Calls per timing round of one stage: the bench's step count, fewer for
    long steps (a round of about 0.1 s), at least 10."""
    return max(10, min(steps, int(0.1 / max(step_s, 1e-9))))


def cpu_baseline(g, cfg, budget_s: float):
    """The oracle on the host cores over a bounded sample of the workload."""
    import numpy as np

    from oracle import oracle

    d, M, scales, seed = cfg["d"], cfg["M"], cfg["scales"], cfg["seed"]
    # ~41 ns per worker-coordinate for the oracle's whole step on one core
    dn = min(d, max(4096, int(budget_s / (45e-9 * M))))
    host = g[:, :dn].cpu().numpy()
    t0 = time.perf_counter()
    ref = oracle.pipeline(host, scales, seed, d=dn)
    dt = time.perf_counter() - t0
    # a sample that finishes well inside the budget is run again (same input,
    # same result) until about the budget is spent, so the rate is not one
    # short run's
    runs = 1
    while dt < 0.75 * budget_s and runs < 64 and dt / runs * (runs + 1) <= budget_s:
        t1 = time.perf_counter()
        oracle.pipeline(host, scales, seed, d=dn)
        dt += time.perf_counter() - t1
        runs += 1
    sample = "full workload" if dn == d else f"all {M} workers, coordinates [0, {dn}) of {d}"
    if runs > 1:
        sample += f", {runs} runs"
    return {"value": round(M * dn * runs / dt / 1e9, 6), "unit": "G elements/s", "cores": 1, "kind": "oracle",
            "sample": sample, "seconds": round(dt, 2)}, ref, dn


def bench_randk(args, g, cfg) -> int:
    """GlobalRandK step (Sec. 3.3-3.4): select -> gather -> Algorithm 1/2 on
    the k sampled coordinates -> scatter into the d-vector."""
    import torch

    from paper_2109_12497_amd.step import RandKStep

    d, M, scales, seed, k = cfg["d"], cfg["M"], cfg["scales"], cfg["seed"], cfg["randk"]
    st = RandKStep(d, M, k, scales, device="cuda")
    stream = torch.cuda.current_stream()
    from paper_2109_12497_amd.step import capture

    replay = capture(st, g, seed).replay if args.graph else (lambda: st.run(g, seed))
    for _ in range(args.warmup):
        replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        replay()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    # per-stage times: each stage repeated back to back between two events
    def stage_time(fn, reps):
        return stage_ms_per_call(torch, stream, fn, reps)

    reps = stage_reps(args.steps, elapsed / args.steps)
    stage_ms = {"select": stage_time(lambda: st.select(seed), reps),
                "gather": stage_time(lambda: st.gather(g), reps),
                "aggregate": stage_time(lambda: st.inner.run(st.sub, seed), reps),
                "scatter": stage_time(lambda: st.scatter(), reps)}
    stage_ms = {k: round(v, 4) for k, v in stage_ms.items()}
    base, parity = None, None
    if not args.no_cpu_baseline:
        base, parity = randk_cpu_baseline(g, cfg, args.cpu_budget, st, seed)
    result = {
        "metric": METRIC, "value": round(M * d * args.steps / elapsed / 1e9, 3), "unit": "G elements/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": args.workload, "d": d, "M": M, "scales": scales, "seed": seed, "randk": k,
                   "quantizer": "multi" if len(scales) > 1 else "single",
                   "launch": "hip graph replay per step" if args.graph else "host launches",
                   "parallelism": "one GPU, M workers simulated"},
        "stage_ms": stage_ms, "roofline": None, "cpu_baseline": base}
    if parity is not None:
        result["parity_vs_oracle"] = parity
    print(json.dumps(result))
    return 0


def randk_cpu_baseline(g, cfg, budget_s: float, st, seed: int):
    """The oracle's GlobalRandK step (its selection over all d keys, then
    Algorithm 1/2 on the k gathered coordinates) on the host cores over the
    whole workload, repeated up to about the budget; then one device step
    compared with it bit for bit."""
    import numpy as np
    import torch

    from oracle import oracle

    d, M, scales, k = cfg["d"], cfg["M"], cfg["scales"], cfg["randk"]
    host = g[:, :d].cpu().numpy()
    t0 = time.perf_counter()
    ref = oracle.randk_pipeline(host, k, scales, seed, d=d)
    dt, runs = time.perf_counter() - t0, 1
    while dt < 0.75 * budget_s and runs < 64 and dt / runs * (runs + 1) <= budget_s:
        t1 = time.perf_counter()
        oracle.randk_pipeline(host, k, scales, seed, d=d)
        dt += time.perf_counter() - t1
        runs += 1
    base = {"value": round(M * d * runs / dt / 1e9, 6), "unit": "G elements/s", "cores": 1, "kind": "oracle",
            "sample": "full workload" + (f", {runs} runs" if runs > 1 else ""), "seconds": round(dt, 2)}
    st.run(g, seed)
    torch.cuda.synchronize()
    W = np.float32(st.inner.w[0].item())
    if W != ref["W_oracle"]:
        ref = oracle.randk_pipeline(host, k, scales, seed, d=d, W=W)
    ok = (np.array_equal(st.sel[:k].cpu().numpy().view(np.uint32), ref["sel"]) and
          np.array_equal(st.out[:d].cpu().numpy().view(np.int32), ref["full"].view(np.int32)))
    return base, "bit-exact" if ok else "MISMATCH"


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    # the first few tens of steps of a process run slower than the rest
    # (clocks ramping up); the defaults time 200 steps after 50 untimed ones
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default="resnet18")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of oracle work to aim for")
    ap.add_argument("--copy-probe", type=int, default=0)
    ap.add_argument("--stream-probe", action="store_true")
    ap.add_argument("--graph", action="store_true",
                    help="time replays of the step captured in a HIP graph instead of host launches")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the simulated workers' codes are summed on-device; "
              "multi-GPU runs are not part of this build (use --gpus 1).", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return 0
    if args.stream_probe:
        stream_probe(args.workload, max(10, args.steps))
        return 0

    import synth
    from paper_2109_12497_amd.step import Step  # fails loudly if libuq.so is not built

    g, cfg = synth.make_gradients(args.workload, device="cuda")
    d, M, scales, seed = cfg["d"], cfg["M"], cfg["scales"], cfg["seed"]
    streamed = bool(cfg.get("streamed", False))
    K = len(scales)
    stream = torch.cuda.current_stream()
    if cfg.get("randk"):
        return bench_randk(args, g, cfg)
    bits = int(cfg.get("bits", 8))
    step = Step(d, M, scales, device="cuda", streamed=streamed, bits=bits)
    torch.cuda.synchronize()

    for _ in range(args.warmup):
        step.run(g, seed)
    torch.cuda.synchronize()

    # -- timed region: K whole steps (host launches, or with --graph replays
    # of the step's kernels captured once in a HIP graph)
    from paper_2109_12497_amd.step import capture

    if args.graph:
        replay = capture(step, g, seed).replay
    else:
        replay = lambda: step.run(g, seed)  # noqa: E731
    for _ in range(args.warmup):
        replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        replay()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_per_step = elapsed / args.steps * 1e3
    value = M * d * args.steps / elapsed / 1e9

    # -- per-stage times: each stage repeated back to back between two events
    # on the stream (its inputs are the previous stage's outputs, already in
    # place), so host launch overhead does not enter the figures
    def stage_time(fn, reps):
        return stage_ms_per_call(torch, stream, fn, reps)

    reps = stage_reps(args.steps, elapsed / args.steps)
    stage_ms = {"shared_scale": stage_time(lambda: step.shared_scale(g), reps)}
    if streamed:
        # one worker row per call, M calls per step, the last of them fused
        # with the reconstruction
        stage_ms["quantize"] = M * stage_time(lambda: step.quantize(g[:1], seed, rows=1), reps)
        stage_ms["sum_dequantize"] = ((M - 1) * stage_time(lambda: step.sum_codes(rows=1, accumulate=1), reps) +
                                      stage_time(lambda: step.sum_dequantize(rows=1, accumulate=1), reps))
    else:
        stage_ms["quantize"] = stage_time(lambda: step.quantize(g, seed), reps)
        stage_ms["sum_dequantize"] = stage_time(lambda: step.sum_dequantize(), reps)
    nbytes = algorithmic_bytes(d, M, K, streamed, bits)

    # -- dominant kernel (the quantiser): launches back to back between two
    # events on the stream it runs on, so the average is the kernel's own
    # duration (the figure rocprofv3 reports for k_quantise); best of three
    # rounds, as for the stages, so that a round in which the host stalled
    # does not count idle time as kernel time
    reps = max(10, args.steps)
    rows_per_launch = 1 if streamed else M
    step.shared_scale(g)
    q_launch_ms = stage_ms_per_call(
        torch, stream, lambda: step.quantize(g[:rows_per_launch], seed, rows=rows_per_launch), reps)
    q_bytes_launch = quantize_bytes_per_launch(d, rows_per_launch, K, bits)
    achieved = q_bytes_launch / (q_launch_ms * 1e-3) / 1e9
    kernel_name = ("k_quantise_multi" if K > 1 else "k_quantise_single") + ("" if bits == 8 else f"_{bits}bit")
    traffic = measured_traffic(kernel_name, args.workload)

    result = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "G elements/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": args.workload, "d": d, "M": M, "scales": scales, "seed": seed,
                   "quantizer": "multi" if K > 1 else "single", "streamed": streamed, "code_bits": bits,
                   "launch": "hip graph replay per step" if args.graph else "host launches",
                   "parallelism": "one GPU, M workers simulated"},
        "pct_hbm_peak": round(100 * nbytes["total"] / (elapsed / args.steps) / 1e9 / HBM_PEAK_GBS, 2),
        "stage_ms": {k: round(v, 4) for k, v in stage_ms.items()},
        "roofline": {"bound": "hbm", "kernel": kernel_name, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic, "algorithmic_bytes_per_launch": q_bytes_launch,
                     "avg_launch_us": round(q_launch_ms * 1e3, 2)},
        "cpu_baseline": None,
    }

    if not args.no_cpu_baseline:
        base, ref, dn = cpu_baseline(g, cfg, args.cpu_budget)
        result["cpu_baseline"] = base
        step.run(g, seed)  # one whole step, after the stage timings
        torch.cuda.synchronize()
        # the oracle ran on the same inputs: compare what it covers (free parity check)
        W = np.float32(step.w[0].item())
        if dn == d and not streamed:
            same_w = W == ref["W_oracle"]
            if not same_w:
                from oracle import oracle

                ref = oracle.pipeline(g[:, :d].cpu().numpy(), scales, seed, d=d, W=W)
            ok = (np.array_equal(step.codes[:, :d].cpu().numpy(), ref["codes"]) and
                  np.array_equal(step.sum[:d].cpu().numpy(), ref["sum"]) and
                  np.array_equal(step.out[:d].cpu().numpy().view(np.int32), ref["out"].view(np.int32)))
            result["parity_vs_oracle"] = "bit-exact" if ok else "MISMATCH"
    print(json.dumps(result))
    return 0


if __name__ == "__main__":
    sys.exit(main())
