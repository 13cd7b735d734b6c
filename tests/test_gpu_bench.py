"""bench.py end to end on the GPU at the small workload (d = 2^20, 4 workers,
one scale s = 127): one JSON line carrying the throughput, the dominant
kernel's roofline and the oracle's rate on the same input, with the device's
step bit-exact against that oracle run; host launches and HIP-graph replays.
Also the GlobalRandK line at the ResNet-18 shape."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
D, M = 1 << 20, 4


def run_bench(*extra, workload="small-gaussian"):
    cmd = [sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--workload", workload, "--steps", "20",
           "--warmup", "5", "--cpu-budget", "1", *extra]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=240, cwd=ROOT)
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

    roof = j["roofline"]
    assert (roof["bound"], roof["peak"], roof["unit"]) == ("hbm", 8000.0, "GB/s")
    # one quantiser launch over all rows: 4 bytes read and 1 written per coordinate
    assert roof["algorithmic_bytes_per_launch"] == M * D * 5
    assert roof["achieved"] == pytest.approx(roof["algorithmic_bytes_per_launch"] / (roof["avg_launch_us"] * 1e3),
                                             rel=0.01)
    assert roof["frac"] == pytest.approx(roof["achieved"] / roof["peak"], rel=1e-3)

    base = j["cpu_baseline"]
    assert base["kind"] == "oracle" and base["cores"] >= 1 and base["value"] > 0 and base["sample"]
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
    base = j["cpu_baseline"]
    assert base["kind"] == "oracle" and base["cores"] >= 1 and base["value"] > 0
    assert base["sample"].startswith("full workload")
    assert j["parity_vs_oracle"] == "bit-exact"
