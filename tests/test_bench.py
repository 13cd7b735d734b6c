"""bench.py's host-side pieces (no GPU): the per-coordinate byte accounting of
the step, the refusal of multi-GPU runs, the stage timing's round sizing, the
counter-traffic lookup tied to the kernel sources, and the CPU baseline."""
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def per_coord(M, K, streamed=False, bits=8, d=1 << 20):
    b = bench.algorithmic_bytes(d, M, K, streamed, bits)
    assert b["total"] % d == 0
    return b["total"] // d


@pytest.mark.parametrize("M", [1, 2, 8, 16, 17, 300])
def test_step_bytes_per_coordinate(M):
    # one scale: norm 4M, quantise 5M, sum M + 4 with the reconstruction's
    # 4-byte output in the same pass
    assert per_coord(M, 1) == 10 * M + 8
    # several scales: the index read once by the quantiser and once by the
    # sum's reconstruction; with 2 to 16 workers the norm pass also writes the
    # row maxima the index pass reads
    want = 10 * M + 19 if 2 <= M <= bench.FUSED_MAX_ROWS else 14 * M + 11
    assert per_coord(M, 4) == want


def test_streamed_and_packed_bytes():
    d, M, K = 1 << 20, 16, 8
    b = bench.algorithmic_bytes(d, M, K, True)
    # quantise row by row (the index read by every launch), accumulate into
    # the int32 sum (set for the first row, += after)
    assert b["quantize"] == M * (5 * d + d)
    # (and in the last call the output and the index for the reconstruction)
    assert b["sum_dequantize"] == (d + 4 * d) + (M - 1) * (d + 8 * d) + 4 * d + d
    # 4-bit codes: half a byte per code written and read back
    assert bench.code_bytes(1001, 4) == 501 and bench.code_bytes(1001, 2) == 251
    assert bench.quantize_bytes_per_launch(1000, 3, 1, 4) == 3 * (4000 + 500)
    assert bench.quantize_bytes_per_launch(1000, 3, 2, 8) == 3 * 5000 + 1000


def test_stage_reps():
    assert bench.stage_reps(200, 0.163e-3) == 200
    assert bench.stage_reps(200, 66e-3) == 10
    assert 10 <= bench.stage_reps(200, 4.5e-3) <= 200


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr and r.stdout == ""


def test_counter_traffic_follows_the_sources(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    for rel in bench.KERNEL_SOURCES:
        p = tmp_path / rel
        p.parent.mkdir(parents=True, exist_ok=True)
        p.write_text("// kernel source " + rel)
    prof = tmp_path / "profiles"
    prof.mkdir()
    digest = bench.source_digest()
    (prof / "k_quantise_single_w_counters.md").write_text(
        f"traffic_bytes_per_launch: 12345\nsource_digest: {digest}\n")
    assert bench.measured_traffic("k_quantise_single", "w") == 12345.0
    assert bench.measured_traffic("k_quantise_single", "other") is None
    # a changed comment or layout keeps them; changed code makes them stale
    (tmp_path / bench.KERNEL_SOURCES[0]).write_text("/* a note */ //   another\n\n")
    assert bench.measured_traffic("k_quantise_single", "w") == 12345.0
    (tmp_path / bench.KERNEL_SOURCES[0]).write_text("int x;")
    assert bench.measured_traffic("k_quantise_single", "w") is None


def test_cpu_baseline_on_a_small_sample():
    torch = pytest.importorskip("torch")
    g = torch.from_numpy(np.random.default_rng(0).standard_normal((2, 5000)).astype(np.float32) * 1e-3)
    base, ref, dn = bench.cpu_baseline(g, dict(d=5000, M=2, scales=[127.0], seed=3), 0.2)
    assert dn == 5000 and base["kind"] == "oracle" and base["cores"] == 1 and base["value"] > 0
    assert base["sample"].startswith("full workload")
    assert ref["codes"].shape == (2, 5000)
