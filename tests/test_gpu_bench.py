"""bench.py end to end on the GPU at the small workload (d = 2^20, 4 workers,
one scale s = 127): one JSON line carrying the throughput, the roofline of
the stage with the largest share of the step and the oracle's rate on one and
on several cores over the same input, with the device's step bit-exact
against that oracle run; host launches and HIP-graph replays.  Also the
default line (2^30 coordinates, 16 streamed workers, eight scales) in a
short run, and the GlobalRandK line at the ResNet-18 shape."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
D, M = 1 << 20, 4


def run_bench(*extra, workload="small-gaussian", steps=20, warmup=5):
    cmd = [sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--steps", str(steps), "--warmup", str(warmup),
           "--cpu-budget", "1", *extra]
    if workload:
        cmd += ["--workload", workload]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1, r.stdout
    return json.loads(lines[0])


@pytest.mark.parametrize("extra", [(), ("--graph",)], ids=["host-launches", "graph"])
def test_bench_line(extra):
    j = run_bench(*extra)
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better", "scaling",
                "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert key in j, key
    assert (j["n_gpus"], j["steps"], j["warmup"]) == (1, 20, 5)
    assert j["higher_is_better"] is True and j["data"] == "synthetic" and j["dtype"] == "f32"
    cfg = j["config"]
    assert (cfg["workload"], cfg["d"], cfg["M"]) == ("small-gaussian", D, M)
    assert cfg["launch"] == ("hip graph replay per step" if extra else "host launches")
    # M·d worker-coordinates per step, in G elements/s
    assert j["value"] == pytest.approx(M * D / (j["ms_per_step"] * 1e-3) / 1e9, rel=0.02)

    check_roofline(j)
    base = j["cpu_baseline"]
    assert base["kind"] == "oracle" and base["cores"] >= 1 and base["value"] > 0 and base["sample"]
    assert base["one_core"]["cores"] == 1 and base["one_core"]["value"] > 0
    assert j["parity_vs_oracle"] == "bit-exact"


def check_roofline(j, share_lo=0.4, share_hi=1.3):
    roof = j["roofline"]
    assert (roof["bound"], roof["peak"], roof["unit"]) == ("hbm", 8000.0, "GB/s")
    share = j["stage_share"]
    # the roofline is the stage with the largest share of the step
    assert roof["stage"] == max(share, key=share.get)
    assert roof["achieved"] == pytest.approx(roof["algorithmic_bytes_per_launch"] / (roof["avg_launch_us"] * 1e3),
                                             rel=0.01)
    assert roof["frac"] == pytest.approx(roof["achieved"] / roof["peak"], rel=1e-3)
    # stage_ms carries four decimals of a millisecond
    assert roof["avg_launch_us"] == pytest.approx(j["stage_ms"][roof["stage"]] * 1e3, abs=0.06)
    # the stages run back to back take about the step's time (less where the
    # step is bound by host launches)
    assert share_lo < sum(share.values()) < share_hi


def test_default_bench_line():
    """`python bench.py` with no workload: 2^30 coordinates, 16 workers
    streamed through the fused quantise-and-sum, eight scales, the shared
    index as 4-bit fields."""
    j = run_bench(workload=None, steps=3, warmup=1)
    cfg = j["config"]
    assert (cfg["workload"], cfg["d"], cfg["M"], len(cfg["scales"]), cfg["streamed"]) == \
        ("student-t", 1 << 30, 16, 8, True)
    assert cfg["path"] == "quantise-and-sum fused" and cfg["index_bits"] == 4
    # 17 M + 5 bytes per coordinate with a byte index; its 4-bit fields save
    # half a byte in the index pass and in each of the M workers' calls
    assert j["step_bytes"] == (2 * (17 * 16 + 5) - 17) * (1 << 29)
    check_roofline(j, 0.85, 1.15)
    assert j["roofline"]["stage"] == "quant_sum" and j["roofline"]["launches_per_step"] == 14
    assert j["cpu_baseline"]["one_core"]["value"] > 0
    assert j["parity_vs_oracle"] == "bit-exact"


def test_randk_bench_line():
    # GlobalRandK (k = 10000) on the ResNet-18-shaped workload: the oracle's
    # whole selection and step as the CPU baseline, the device step bit-exact
    j = run_bench(workload="resnet18-grandk")
    d, m = 11_173_962, 8
    assert (j["config"]["workload"], j["config"]["d"], j["config"]["M"], j["config"]["randk"]) == \
        ("resnet18-grandk", d, m, 10_000)
    assert j["value"] == pytest.approx(m * d / (j["ms_per_step"] * 1e-3) / 1e9, rel=0.02)
    assert set(j["stage_ms"]) == {"select", "gather", "aggregate", "scatter"}
    # the selection, bound by Philox arithmetic, carries an ALU roofline
    roof = j["roofline"]
    assert roof["bound"] == "alu" and roof["stage"] == "select" and roof["traffic"] is None
    assert roof["achieved"] == pytest.approx((d + 3) // 4 / (j["stage_ms"]["select"] * 1e-3) / 1e9, rel=0.01)
    assert 0 < roof["frac"] < 1
    base = j["cpu_baseline"]
    assert base["kind"] == "oracle" and base["cores"] >= 1 and base["value"] > 0
    assert base["sample"].startswith("full workload")
    assert j["parity_vs_oracle"] == "bit-exact"
