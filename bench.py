#!/usr/bin/env python3
"""Throughput of one aggregation step of the unbiased max-norm quantisers
(arXiv 2109.12497, Algorithms 1-2) on one MI355X.

A step is the whole hot path over M workers' gradients resident in HBM:
shared max-norm scale (+ shared scale index) -> quantise every worker ->
integer sum of the codes -> reconstruct the averaged gradient.  The metric is
gradient elements (M * d worker-coordinates) per second, and the fraction of
the 8 TB/s HBM peak the step's algorithmic bytes reach.

The default workload is the largest that fits one GPU: d = 2^30 heavy-tailed
(Student-t) coordinates, 16 workers streamed one at a time through a resident
int32 sum, eight scales (Algorithm 2), each worker quantised and added into
the sum in one fused call (with resident workers, one call quantises and sums
all rows, and with several scales and at most 16 workers it also forms the
shared scale index from the rows it holds, so the shared-scale call forms W
only; workloads with packed codes store them, then sum them).

Prints one JSON line: the step's rate, its stages' times and shares, the
roofline of the stage with the largest share, the oracle's rate on one core
and on all cores over a bounded sample, and the device's results on that
sample checked against the oracle's.  Extra modes:
  --workload NAME       another workload of synth.WORKLOADS
  --composed            codes stored, then summed (separate calls)
  --index-pass          resident workers, several scales: the shared index
                        from the shared-scale call's own pass, not formed
                        inside the quantise-and-sum (or, with packed codes,
                        inside the quantiser)
  --byte-index          the shared index as bytes, not 4-bit fields, where the
                        quantise-and-sum reads a separately formed one
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
# the sources whose code the counter summaries are tied to (kernels, device
# helpers, launch planning and workspace layout)
KERNEL_SOURCES = ["paper_2109_12497_amd/csrc/uq_kernels.hip", "paper_2109_12497_amd/csrc/uq_device.hpp",
                  "paper_2109_12497_amd/csrc/uq_launch.hpp", "paper_2109_12497_amd/csrc/uq_randk.hip"]


# GlobalRandK's selection is bound by Philox arithmetic, not bytes: its
# roofline counts Philox4x32-10 blocks.  A block is at least 40 VALU
# instructions per lane (10 rounds of two 32x32->64 multiplies and two
# three-input XORs); the chip issues 256 CUs x 4 SIMDs x 16 lanes per cycle at
# 2.4 GHz, so at most 983 G blocks/s even with every instruction at full rate.
PHILOX_BLOCK_MIN_INSTRUCTIONS = 40
VALU_LANE_OPS_PER_S = 256 * 4 * 16 * 2.4e9
PHILOX_PEAK_GBLOCKS = VALU_LANE_OPS_PER_S / PHILOX_BLOCK_MIN_INSTRUCTIONS / 1e9


def selection_roofline(d: int, select_ms: float) -> dict:
    """The selection's one key pass evaluates one Philox block (the keys' high
    words) per four coordinates; the rare keys inside the bracket cost one
    more block each, not counted.  Rate over the whole select call."""
    blocks = (d + 3) // 4
    achieved = blocks / (select_ms * 1e-3) / 1e9
    return {"bound": "alu", "kernel": "k_rk_init+k_rk_collect+k_rk_sort", "stage": "select",
            "achieved": round(achieved, 1), "peak": round(PHILOX_PEAK_GBLOCKS, 1), "unit": "G Philox blocks/s",
            "frac": round(achieved / PHILOX_PEAK_GBLOCKS, 4), "traffic": None,
            "algorithmic_blocks_per_launch": blocks, "avg_launch_us": round(select_ms * 1e3, 2),
            "launches_per_step": 1}


def code_bytes(d: int, bits: int) -> int:
    return (d * bits + 7) // 8


def quantize_bytes_per_launch(d: int, rows: int, K: int, bits: int = 8) -> int:
    """One quantiser launch over `rows` workers: their gradients in, their
    codes out, and (several scales) the shared index, needed once."""
    return rows * (4 * d + code_bytes(d, bits)) + (d if K > 1 else 0)


def index_bytes(d: int, index_bits: int = 8) -> int:
    """The shared index: one byte per coordinate, or 4-bit fields."""
    return d if index_bits == 8 else (d + 1) // 2


def quant_sum_bytes_per_call(d: int, rows: int, K: int, accumulate: bool, reconstruct: bool,
                             index_bits: int = 8) -> int:
    """One fused quantise-and-sum call: the rows' gradients and (several
    scales) the shared index in, the int32 sums out (the old sums in too when
    accumulating) and, when it reconstructs, the output."""
    return (4 * rows * d + (index_bytes(d, index_bits) if K > 1 else 0) + (4 * d if accumulate else 0) + 4 * d
            + (4 * d if reconstruct else 0))


def scale_kernels(M: int, K: int) -> list:
    """The kernels of one uq_shared_scale call, the longest first."""
    if K == 1:
        return ["k_sumsq", "k_finish"]
    if 2 <= M <= FUSED_MAX_ROWS:
        return ["k_norm_max", "k_rowsum", "k_index_prep", "k_index_max"]
    return ["k_sumsq", "k_finish", "k_index"]


def shared_scale_bytes(d: int, M: int, K: int, index_bits: int = 8) -> int:
    """The gradients read once for the norm; with several scales and 2 to 16
    workers that pass also writes a 16-bit key of the largest |g| over the
    workers (2 bytes per coordinate), which the index pass reads instead of
    the gradients; with more workers (or one) the index pass reads every
    gradient again.  The index is written once."""
    if K == 1:
        return 4 * M * d
    ib = index_bytes(d, index_bits)
    if 2 <= M <= FUSED_MAX_ROWS:
        return 4 * M * d + 2 * d + 2 * d + ib
    return 4 * M * d + 4 * M * d + ib


def plan_stages(d: int, M: int, K: int, bits: int = 8, streamed: bool = False, quant_sum: bool = False,
                index_in_pass: bool = False, index_bits: int = 8) -> list:
    """The library calls of one step as stages: name, the kernel it launches
    (several for the shared scale, the longest first), calls per step and the
    algorithmic bytes per call.  index_bits = 4: the shared index held as
    4-bit fields (the quantise-and-sum with a separate index pass)."""
    multi = K > 1
    ib = d if multi else 0
    cb = code_bytes(d, bits)
    qk = ("k_quantise_multi" if multi else "k_quantise_single") + ("" if bits == 8 else f"_{bits}bit")
    if index_in_pass and quant_sum:
        # W alone (the one-scale norm pass), then one call that reads every
        # row, writes the index it forms, the sums and the output
        return [dict(name="shared_scale", kernels=scale_kernels(M, 1), calls=1, bytes=shared_scale_bytes(d, M, 1)),
                dict(name="index_quant_sum", kernels=["k_index_quant_sum"], calls=1,
                     bytes=4 * M * d + d + 4 * d + 4 * d)]
    if index_in_pass:
        # W alone, then one call that reads every row and writes the index it
        # forms and every row's codes, then the sum with the reconstruction
        iq = "k_index_quantise" + ("" if bits == 8 else f"_{bits}bit")
        return [dict(name="shared_scale", kernels=scale_kernels(M, 1), calls=1, bytes=shared_scale_bytes(d, M, 1)),
                dict(name="index_quantize", kernels=[iq], calls=1, bytes=4 * M * d + d + M * cb),
                dict(name="sum_dequantize", kernels=["k_sum_dequant"], calls=1, bytes=M * cb + 4 * d + 4 * d + ib)]
    xb = index_bits if quant_sum else 8
    st = [dict(name="shared_scale", kernels=scale_kernels(M, K), calls=1, bytes=shared_scale_bytes(d, M, K, xb))]
    if quant_sum and streamed:
        # one worker per call into the running sum; the last call reconstructs
        if M == 1:
            st.append(dict(name="quant_sum_last", kernels=["k_quant_sum_set_deq"], calls=1,
                           bytes=quant_sum_bytes_per_call(d, 1, K, False, True, xb)))
        else:
            st.append(dict(name="quant_sum_first", kernels=["k_quant_sum_set"], calls=1,
                           bytes=quant_sum_bytes_per_call(d, 1, K, False, False, xb)))
            if M > 2:
                st.append(dict(name="quant_sum", kernels=["k_quant_sum_acc"], calls=M - 2,
                               bytes=quant_sum_bytes_per_call(d, 1, K, True, False, xb)))
            st.append(dict(name="quant_sum_last", kernels=["k_quant_sum_acc_deq"], calls=1,
                           bytes=quant_sum_bytes_per_call(d, 1, K, True, True, xb)))
    elif quant_sum:
        # one scale and 5 to 16 rows: a tile's rows split over a block's waves
        kern = "k_quant_sum_split" if K == 1 and 4 < M <= FUSED_MAX_ROWS else "k_quant_sum_set_deq"
        st.append(dict(name="quant_sum", kernels=[kern], calls=1,
                       bytes=quant_sum_bytes_per_call(d, M, K, False, True, xb)))
    elif streamed:
        # the codes of one worker per call, then summed into the running sum
        st.append(dict(name="quantize", kernels=[qk], calls=M, bytes=quantize_bytes_per_launch(d, 1, K, bits)))
        if M > 1:
            st.append(dict(name="sum_first", kernels=["k_sum"], calls=1, bytes=cb + 4 * d))
            if M > 2:
                st.append(dict(name="sum", kernels=["k_sum"], calls=M - 2, bytes=cb + 8 * d))
        st.append(dict(name="sum_dequantize", kernels=["k_sum_dequant"], calls=1,
                       bytes=cb + (8 * d if M > 1 else 4 * d) + 4 * d + ib))
    else:
        st.append(dict(name="quantize", kernels=[qk], calls=1, bytes=quantize_bytes_per_launch(d, M, K, bits)))
        st.append(dict(name="sum_dequantize", kernels=["k_sum_dequant"], calls=1, bytes=M * cb + 4 * d + 4 * d + ib))
    return st


def algorithmic_bytes(d: int, M: int, K: int, streamed: bool, bits: int = 8, quant_sum: bool = False,
                      index_in_pass: bool = False, index_bits: int = 8) -> dict:
    """Bytes each stage must move at minimum (reads + writes) per step, and
    their total."""
    b = {}
    for s in plan_stages(d, M, K, bits, streamed, quant_sum, index_in_pass, index_bits):
        b[s["name"]] = b.get(s["name"], 0) + s["calls"] * s["bytes"]
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
    """Achievable bandwidth of the hot path's access patterns with no work, on
    the workload's gradients (kernels of libuq_probe.so, timed back to back
    between events, mean of three rounds):
      read            every element of the [M, ldg] buffer, grid-stride;
      read4_write1    4 bytes read and 1 written per element (the quantiser);
      rows_read       the first d floats of each of the M rows, by blocks of
                      one chunk of one row (the norm pass's bytes);
      accumulate      4 + 1 + 4 bytes read and 4 written per coordinate of one
                      row (the fused quantise-and-sum of a streamed worker);
      copy            one row copied (4 bytes read, 4 written);
      keys_index<o>   d 16-bit keys read, d bytes written (the index pass's
                      bytes), o octets of keys per thread."""
    import ctypes

    import torch

    import synth

    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2109_12497_amd", "libuq_probe.so"))
    P, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.uqp_read.argtypes = [P, i64, P, P]
    lib.uqp_read_write8.argtypes = [P, i64, P, P]
    lib.uqp_read_out_floats.argtypes = [i64]
    lib.uqp_read_out_floats.restype = i64
    lib.uqp_rows_read.argtypes = [P, i64, i32, i64, P, P]
    lib.uqp_rows_out_floats.argtypes = [i64, i32]
    lib.uqp_rows_out_floats.restype = i64
    lib.uqp_accumulate.argtypes = [P, P, P, i64, P]
    lib.uqp_copy.argtypes = [P, P, i64, P]
    lib.uqp_keys_index.argtypes = [P, i64, P, i32, P]
    g, cfg = synth.make_gradients(workload, device="cuda")
    M, d = cfg["M"], cfg["d"]
    n = g.numel() // 512 * 512
    dn = d // 512 * 512
    codes = torch.empty(n, dtype=torch.uint8, device="cuda")
    out = torch.empty(int(lib.uqp_read_out_floats(n)), dtype=torch.float32, device="cuda")
    rows_out = torch.empty(int(lib.uqp_rows_out_floats(dn, M)), dtype=torch.float32, device="cuda")
    idx = torch.ones(dn, dtype=torch.uint8, device="cuda")
    acc = torch.zeros(dn, dtype=torch.int32, device="cuda")
    dst = torch.empty(dn, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    h = stream.cuda_stream

    def timed(fn):
        for _ in range(3):
            assert fn() == 0
        return stage_ms_per_call(torch, stream, fn, max(5, reps // 4)) * 1e-3

    t_r = timed(lambda: lib.uqp_read(g.data_ptr(), n, out.data_ptr(), h))
    t_rw = timed(lambda: lib.uqp_read_write8(g.data_ptr(), n, codes.data_ptr(), h))
    t_rows = timed(lambda: lib.uqp_rows_read(g.data_ptr(), dn, M, g.stride(0), rows_out.data_ptr(), h))
    t_acc = timed(lambda: lib.uqp_accumulate(g.data_ptr(), idx.data_ptr(), acc.data_ptr(), dn, h))
    t_copy = timed(lambda: lib.uqp_copy(g.data_ptr(), dst.data_ptr(), dn, h))
    # the keys are the first 2 dn bytes of the gradient buffer, the index the
    # first dn bytes of the byte buffer
    t_ki = {o: timed(lambda o=o: lib.uqp_keys_index(g.data_ptr(), dn, codes.data_ptr(), o, h)) for o in (2, 4, 8)}
    res = {"stream_probe": workload, "elements": n, "d": dn, "M": M}
    for name, nbytes, t in (("read", 4 * n, t_r), ("read4_write1", 5 * n, t_rw), ("rows_read", 4 * M * dn, t_rows),
                            ("accumulate", 13 * dn, t_acc), ("copy", 8 * dn, t_copy),
                            *((f"keys_index{o}", 3 * dn, t) for o, t in t_ki.items())):
        res[f"{name}_us"] = round(t * 1e6, 2)
        res[f"{name}_GBps"] = round(nbytes / t / 1e9, 1)
    print(json.dumps(res))


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
    on `stream`, its inputs already in place: the mean over `rounds` rounds of
    `reps` calls (rounds in which the host fell behind the GPU count too)."""
    total = 0.0
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
        total += a.elapsed_time(b) / reps
    return total / rounds


def stage_reps(steps: int, step_s: float) -> int:
    """Calls per timing round of one stage: the bench's step count, fewer for
    long steps (a round of about 0.1 s), at least 10."""
    return max(10, min(steps, int(0.1 / max(step_s, 1e-9))))


# One core's oracle time per worker-coordinate for the whole step, about:
# two Philox blocks per code dominate; several scales add the index rule.
ORACLE_NS_PER_ELEMENT = {False: 48e-9, True: 58e-9}


def sample_size(d: int, M: int, multi: bool, budget_s: float) -> int:
    """Coordinates of the CPU baseline's sample: about budget_s of one core's
    oracle work over all M workers, at least 4096, at most d."""
    return min(d, max(4096, int(budget_s / (ORACLE_NS_PER_ELEMENT[multi] * M))))


def _timed_runs(fn, budget_s: float):
    """fn() once, then again on the same input until about budget_s is spent
    (a sample that finishes well inside the budget is not one short run).
    Returns (first result, runs, seconds)."""
    t0 = time.perf_counter()
    first = fn()
    dt, runs = time.perf_counter() - t0, 1
    while dt < 0.75 * budget_s and runs < 64 and dt / runs * (runs + 1) <= budget_s:
        t1 = time.perf_counter()
        fn()
        dt += time.perf_counter() - t1
        runs += 1
    return first, runs, dt


def cpu_baseline(g, cfg, budget_s: float, W=None, threads=None):
    """The oracle over a bounded sample of the workload (all M workers,
    coordinates [0, dn)), on one host core and on `threads` cores (default:
    the cores this process may use, at most 16).  W: the scale the later
    steps use (the device's, so that its results are comparable); the oracle
    still forms its own norm over the sample, so the work is the whole step's.
    Returns the baseline record, the one-core run's result and dn."""
    from oracle import oracle

    d, M, scales, seed = cfg["d"], cfg["M"], cfg["scales"], cfg["seed"]
    threads = oracle.default_threads() if threads is None else threads
    dn = sample_size(d, M, len(scales) > 1, budget_s)
    host = g[:, :dn].cpu().numpy()
    ref, runs1, dt1 = _timed_runs(lambda: oracle.pipeline(host, scales, seed, d=dn, W=W), budget_s)
    _, runsn, dtn = _timed_runs(lambda: oracle.pipeline_threaded(host, scales, seed, d=dn, W=W, threads=threads),
                                budget_s)
    sample = "full workload" if dn == d else f"all {M} workers, coordinates [0, {dn}) of {d}"
    rec = {"value": round(M * dn * runsn / dtn / 1e9, 6), "unit": "G elements/s", "cores": threads,
           "kind": "oracle", "sample": f"{sample}, {runsn} runs", "seconds": round(dtn, 2),
           "one_core": {"value": round(M * dn * runs1 / dt1 / 1e9, 6), "cores": 1, "runs": runs1,
                        "seconds": round(dt1, 2)}}
    return rec, ref, dn


def parity_on_sample(step, ref, dn: int, d: int, bits: int) -> str:
    """The device's step against the oracle's run on coordinates [0, dn) with
    the same W: scale index, codes (when the step keeps them; packed codes
    unpacked), sums and outputs bit for bit; W within one binary32 ulp of the
    oracle's own when the sample is the whole vector."""
    import numpy as np

    from oracle import oracle

    ok = True
    if dn == d:
        a = int(np.float32(step.w[0].item()).view(np.int32))
        ok = abs(a - int(np.float32(ref["W_oracle"]).view(np.int32))) <= 1
    if ref["idx"] is not None:
        ok = ok and np.array_equal(step.index_host(0, dn), ref["idx"])
    if step.codes is not None and not step.streamed:
        if bits == 8:
            ok = ok and np.array_equal(step.codes[:, :dn].cpu().numpy(), ref["codes"])
        else:
            packed = step.codes[:, :(dn * bits + 7) // 8].cpu().numpy()
            ok = ok and all(np.array_equal(oracle.unpack_codes(packed[m], dn, bits), ref["codes"][m])
                            for m in range(packed.shape[0]))
    ok = ok and np.array_equal(step.sum[:dn].cpu().numpy(), ref["sum"])
    ok = ok and np.array_equal(step.out[:dn].cpu().numpy().view(np.int32), ref["out"].view(np.int32))
    return "bit-exact" if ok else "MISMATCH"


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
        "stage_ms": stage_ms, "roofline": selection_roofline(d, stage_ms["select"]), "cpu_baseline": base}
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


def progress(msg: str) -> None:
    """One line on stderr per finished phase of the run."""
    print(f"bench: {msg}", file=sys.stderr, flush=True)


def stage_fns(step, g, seed: int, M: int) -> dict:
    """The library call behind each stage of plan_stages, on the step's own
    buffers (its inputs are the previous stage's outputs, already in place)."""
    last = M - 1
    return {
        "shared_scale": lambda: step.shared_scale(g, w_only=step.index_in_pass),
        "index_quant_sum": lambda: step.index_quantize_sum(g, seed),
        "index_quantize": lambda: step.index_quantize(g, seed),
        "quant_sum_first": lambda: step.quantize_sum(g[0:1], seed, rows=1, worker0=0, accumulate=0,
                                                     reconstruct=False),
        "quant_sum": ((lambda: step.quantize_sum(g[1:2], seed, rows=1, worker0=1, accumulate=1, reconstruct=False))
                      if step.streamed else (lambda: step.quantize_sum(g, seed))),
        "quant_sum_last": lambda: step.quantize_sum(g[last:last + 1], seed, rows=1, worker0=last,
                                                    accumulate=1 if M > 1 else 0, reconstruct=True),
        "quantize": ((lambda: step.quantize(g[:1], seed, rows=1)) if step.streamed
                     else (lambda: step.quantize(g, seed))),
        "sum_first": lambda: step.sum_codes(rows=1, accumulate=0),
        "sum": lambda: step.sum_codes(rows=1, accumulate=1),
        "sum_dequantize": ((lambda: step.sum_dequantize(rows=1, accumulate=1 if M > 1 else 0)) if step.streamed
                           else (lambda: step.sum_dequantize())),
    }


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    # the first few tens of steps of a process run slower than the rest
    # (clocks ramping up); the defaults time 100 steps after 20 untimed ones
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="student-t")
    ap.add_argument("--composed", action="store_true",
                    help="quantise and sum in separate calls (the codes through HBM) instead of the fused "
                         "quantise-and-sum (packed-code workloads always store their codes)")
    ap.add_argument("--index-pass", action="store_true",
                    help="resident workers with several scales: the shared index from the shared-scale call's own "
                         "pass instead of formed inside the quantise-and-sum or, with packed codes, the quantiser")
    ap.add_argument("--byte-index", action="store_true",
                    help="the quantise-and-sum reads a separately formed shared index as one byte per coordinate "
                         "instead of 4-bit fields")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=12.0,
                    help="seconds of oracle work to aim for, for each of the two CPU figures")
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
    from paper_2109_12497_amd.step import Step, capture  # fails loudly if libuq.so is not built

    g, cfg = synth.make_gradients(args.workload, device="cuda")
    d, M, scales, seed = cfg["d"], cfg["M"], cfg["scales"], cfg["seed"]
    streamed = bool(cfg.get("streamed", False))
    K = len(scales)
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()
    progress(f"{args.workload}: {M} x {d} gradients generated")
    if cfg.get("randk"):
        return bench_randk(args, g, cfg)
    bits = int(cfg.get("bits", 8))
    # int8 codes: quantised and summed in one fused call unless asked for;
    # packed codes are stored (their packing is what those workloads show)
    quant_sum = bits == 8 and not args.composed
    # the quantise-and-sum calls that read a separately formed index read it
    # as 4-bit fields unless asked for bytes
    index_bits = 4 if quant_sum and K > 1 and (streamed or args.index_pass) and not args.byte_index else 8
    step = Step(d, M, scales, device="cuda", streamed=streamed, bits=bits, quant_sum=quant_sum,
                index_in_pass=False if args.index_pass else None, index_bits=index_bits)
    torch.cuda.synchronize()

    # -- timed region: K whole steps (host launches, or with --graph replays
    # of the step's kernels captured once in a HIP graph)
    replay = capture(step, g, seed).replay if args.graph else (lambda: step.run(g, seed))
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
    progress(f"{args.steps} steps timed: {ms_per_step:.4f} ms per step")

    # -- per-stage times: each stage's call repeated back to back between two
    # events on the stream (mean over rounds), so host launch overhead does
    # not enter them; a stage's share of the step is calls x time per call
    stages = plan_stages(d, M, K, bits, streamed, quant_sum, step.index_in_pass, step.index_bits)
    fns = stage_fns(step, g, seed, M)
    reps = stage_reps(args.steps, elapsed / args.steps)
    for st in stages:
        st["ms"] = stage_ms_per_call(torch, stream, fns[st["name"]], reps)
    step_bytes = sum(st["calls"] * st["bytes"] for st in stages)
    progress("stages timed: " + ", ".join(f"{st['name']} {st['ms']:.4f} ms x {st['calls']}" for st in stages))

    # -- the roofline of the stage with the largest share of the step: its
    # algorithmic bytes per call over its mean time per call (for the shared
    # scale, one call runs its two or three kernels: the figure then covers
    # them together)
    dom = max(stages, key=lambda st: st["calls"] * st["ms"])
    achieved = dom["bytes"] / (dom["ms"] * 1e-3) / 1e9
    traffic = None
    per_kernel = [measured_traffic(k, args.workload) for k in dom["kernels"]]
    if all(t is not None for t in per_kernel):
        traffic = sum(per_kernel)

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
                   "path": ("quantise-and-sum fused, index formed in it" if step.index_in_pass and quant_sum
                            else "quantise-and-sum fused" if quant_sum
                            else "codes stored with the index formed in the quantiser, then summed"
                            if step.index_in_pass else "codes stored, then summed"),
                   "index_bits": step.index_bits if K > 1 else None,
                   "launch": "hip graph replay per step" if args.graph else "host launches",
                   "parallelism": "one GPU, M workers simulated"},
        "pct_hbm_peak": round(100 * step_bytes / (elapsed / args.steps) / 1e9 / HBM_PEAK_GBS, 2),
        "step_bytes": step_bytes,
        "stage_ms": {st["name"]: round(st["ms"], 4) for st in stages},
        "stage_share": {st["name"]: round(st["calls"] * st["ms"] / ms_per_step, 3) for st in stages},
        "roofline": {"bound": "hbm", "kernel": "+".join(dom["kernels"]), "stage": dom["name"],
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                     "algorithmic_bytes_per_launch": dom["bytes"], "avg_launch_us": round(dom["ms"] * 1e3, 2),
                     "launches_per_step": dom["calls"]},
        "cpu_baseline": None,
    }

    if not args.no_cpu_baseline:
        import numpy as np

        # one whole step after the stage timings, then the oracle on the same
        # inputs and the same W over a bounded sample: the CPU figures, and the
        # device's results on that sample checked against them
        step.run(g, seed)
        torch.cuda.synchronize()
        W = np.float32(step.w[0].item())
        base, ref, dn = cpu_baseline(g, cfg, args.cpu_budget, W=W)
        progress(f"oracle: {base['one_core']['value']} G el/s on one core, {base['value']} on {base['cores']}")
        result["cpu_baseline"] = base
        result["parity_vs_oracle"] = parity_on_sample(step, ref, dn, d, bits)
        progress(f"parity on coordinates [0, {dn}): {result['parity_vs_oracle']}")
        result["parity_sample"] = f"coordinates [0, {dn}) of {d}, every worker"
    print(json.dumps(result))
    return 0


if __name__ == "__main__":
    sys.exit(main())
