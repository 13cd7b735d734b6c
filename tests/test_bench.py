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


def per_coord(M, K, streamed=False, bits=8, d=1 << 20, quant_sum=False):
    b = bench.algorithmic_bytes(d, M, K, streamed, bits, quant_sum)
    assert b["total"] % d == 0
    return b["total"] // d


@pytest.mark.parametrize("M", [1, 2, 8, 16, 17, 300])
def test_step_bytes_per_coordinate(M):
    # one scale: norm 4M, quantise 5M, sum M + 4 with the reconstruction's
    # 4-byte output in the same pass
    assert per_coord(M, 1) == 10 * M + 8
    # several scales: the index read once by the quantiser and once by the
    # sum's reconstruction; with 2 to 16 workers the norm pass also writes the
    # row maxima's 16-bit keys, which the index pass reads
    want = 10 * M + 15 if 2 <= M <= bench.FUSED_MAX_ROWS else 14 * M + 11
    assert per_coord(M, 4) == want
    # all rows quantised and summed in one fused call: the gradients and the
    # index in, the sums and the output out
    assert per_coord(M, 1, quant_sum=True) - 4 * M == 4 * M + 8
    assert per_coord(M, 4, quant_sum=True) == want - (10 * M + 15 - (8 * M + 14) if 2 <= M <= 16 else
                                                      14 * M + 11 - (12 * M + 10))


@pytest.mark.parametrize("M", [1, 2, 8, 16])
def test_index_in_pass_bytes(M):
    """Several scales, all rows in one call that also forms the index: the
    one-scale norm pass (4M), then the rows in (4M), the index, the sums and
    the output out (1 + 4 + 4); no row maxima and no index pass."""
    d = 1 << 20
    b = bench.algorithmic_bytes(d, M, 4, False, 8, True, True)
    assert b["shared_scale"] == 4 * M * d and b["index_quant_sum"] == (4 * M + 9) * d
    assert b["total"] == (8 * M + 9) * d
    st = bench.plan_stages(d, M, 4, 8, False, True, True)
    assert [s["kernels"] for s in st] == [["k_sumsq", "k_finish"], ["k_index_quant_sum"]]


@pytest.mark.parametrize("M,bits", [(2, 4), (16, 4), (8, 2), (16, 8)])
def test_index_quantize_bytes(M, bits):
    """Several scales, codes stored, the index formed in the quantiser: the
    one-scale norm pass (4M), the rows in and the index and every row's codes
    out (4M + 1 + M b/8), then the codes, the index and the sums / output of
    the sum with the reconstruction (M b/8 + 1 + 8)."""
    d = 1 << 20
    cb = d * bits // 8
    b = bench.algorithmic_bytes(d, M, 4, False, bits, False, True)
    assert b["shared_scale"] == 4 * M * d and b["index_quantize"] == 4 * M * d + d + M * cb
    assert b["sum_dequantize"] == M * cb + 9 * d
    assert b["total"] == 8 * M * d + 10 * d + 2 * M * cb
    st = bench.plan_stages(d, M, 4, bits, False, False, True)
    kq = "k_index_quantise" + ("" if bits == 8 else f"_{bits}bit")
    assert [s["kernels"] for s in st] == [["k_sumsq", "k_finish"], [kq], ["k_sum_dequant"]]


def test_streamed_bytes():
    d, M, K = 1 << 20, 16, 8
    # codes stored, then summed: the quantiser row by row (the index read by
    # every launch), the sum set for the first row and += after, the last
    # call with the output and the index for the reconstruction
    b = bench.algorithmic_bytes(d, M, K, True)
    assert b["quantize"] == M * (5 * d + d)
    assert b["sum_first"] + b["sum"] + b["sum_dequantize"] == (d + 4 * d) + (M - 1) * (d + 8 * d) + 4 * d + d
    # fused: the first worker 4 + 1 in, 4 out; the others also read the old
    # sums; the last also writes the output
    f = bench.algorithmic_bytes(d, M, K, True, quant_sum=True)
    assert f["quant_sum_first"] == 9 * d and f["quant_sum"] == (M - 2) * 13 * d and f["quant_sum_last"] == 17 * d
    # the whole step: norm + maxima keys 4M + 2, index 2 + 1, then 9 + 13 (M - 2) + 17
    assert per_coord(M, K, True, quant_sum=True) == 17 * M + 5
    assert per_coord(1, K, True, quant_sum=True) == per_coord(1, K, False, quant_sum=True)


def test_four_bit_index_bytes():
    """The index as 4-bit fields: the index pass writes (d + 1) / 2 bytes and
    every quantise-and-sum call reads as many."""
    d, M, K = 1 << 20, 16, 8
    assert bench.index_bytes(1001, 4) == 501 and bench.index_bytes(1001, 8) == 1001
    f = bench.algorithmic_bytes(d, M, K, True, quant_sum=True, index_bits=4)
    assert f["shared_scale"] == (4 * M + 2 + 2) * d + d // 2
    assert f["quant_sum_first"] == 8 * d + d // 2 and f["quant_sum"] == (M - 2) * (12 * d + d // 2)
    assert f["quant_sum_last"] == 16 * d + d // 2
    assert 2 * f["total"] == (2 * (17 * M + 5) - (M + 1)) * d
    # the composed path reads the byte index whatever is asked
    assert bench.algorithmic_bytes(d, M, K, True, index_bits=4) == bench.algorithmic_bytes(d, M, K, True)


def test_packed_bytes():
    assert bench.code_bytes(1001, 4) == 501 and bench.code_bytes(1001, 2) == 251
    assert bench.quantize_bytes_per_launch(1000, 3, 1, 4) == 3 * (4000 + 500)
    assert bench.quantize_bytes_per_launch(1000, 3, 2, 8) == 3 * 5000 + 1000


def test_stage_plan_names_the_kernels():
    st = bench.plan_stages(1 << 20, 16, 8, 8, True, True)
    assert [s["name"] for s in st] == ["shared_scale", "quant_sum_first", "quant_sum", "quant_sum_last"]
    assert st[0]["kernels"] == ["k_norm_max", "k_rowsum", "k_index_prep", "k_index_max"]
    assert [s["calls"] for s in st] == [1, 1, 14, 1]
    assert bench.plan_stages(100, 8, 1)[1]["kernels"] == ["k_quantise_single"]
    assert bench.plan_stages(100, 16, 4, 4)[1]["kernels"] == ["k_quantise_multi_4bit"]
    assert bench.plan_stages(100, 17, 4)[0]["kernels"] == ["k_sumsq", "k_finish", "k_index"]
    # all rows through one quantise-and-sum call: one scale and 5 to 16 rows
    # split a tile's rows over a block's waves
    assert bench.plan_stages(100, 16, 1, 8, False, True)[1]["kernels"] == ["k_quant_sum_split"]
    assert bench.plan_stages(100, 5, 1, 8, False, True)[1]["kernels"] == ["k_quant_sum_split"]
    assert bench.plan_stages(100, 4, 1, 8, False, True)[1]["kernels"] == ["k_quant_sum_set_deq"]
    assert bench.plan_stages(100, 16, 4, 8, False, True)[1]["kernels"] == ["k_quant_sum_set_deq"]
    assert bench.plan_stages(100, 16, 4, 8, False, True, True)[1]["kernels"] == ["k_index_quant_sum"]
    for M in (1, 2, 3):
        st = bench.plan_stages(100, M, 2, 8, True, True)
        assert sum(s["calls"] for s in st[1:]) == M


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
    base, ref, dn = bench.cpu_baseline(g, dict(d=5000, M=2, scales=[127.0], seed=3), 0.2, threads=3)
    assert dn == 5000 and base["kind"] == "oracle" and base["cores"] == 3 and base["value"] > 0
    assert base["one_core"]["cores"] == 1 and base["one_core"]["value"] > 0
    assert base["sample"].startswith("full workload")
    assert ref["codes"].shape == (2, 5000)


class FakeStep:
    """The buffers bench.py reads back from a step, as host tensors."""

    def __init__(self, torch, ref, M, d, bits, streamed=False, index_bits=8):
        from oracle import oracle

        self.d, self.index_bits = d, index_bits
        self.w = torch.tensor([float(ref["W"])], dtype=torch.float32)
        if ref["idx"] is None:
            self.idx = None
        elif index_bits == 8:
            self.idx = torch.from_numpy(ref["idx"].copy())
        else:
            # 4-bit fields, the low nibble first (written out here by hand)
            nib = np.zeros((d + 1) // 2 + 7, dtype=np.uint8)
            for i, v in enumerate(ref["idx"]):
                nib[i // 2] |= np.uint8(int(v) << (4 * (i % 2)))
            self.idx = torch.from_numpy(nib)
        self.sum = torch.from_numpy(ref["sum"].copy())
        self.out = torch.from_numpy(ref["out"].copy())
        self.streamed = streamed
        if streamed:
            self.codes = None
        elif bits == 8:
            self.codes = torch.from_numpy(ref["codes"].copy())
        else:
            ld = ((d * bits + 7) // 8 + 255) // 256 * 256
            packed = np.zeros((M, ld), dtype=np.uint8)
            for m in range(M):
                p = oracle.pack_codes(ref["codes"][m], bits)
                packed[m, :p.size] = p
            self.codes = torch.from_numpy(packed)

    def index_host(self, i0=0, i1=None):
        from paper_2109_12497_amd.step import Step

        return Step.index_host(self, i0, i1)


@pytest.mark.parametrize("bits,scales", [(8, [127.0]), (8, [127.0, 2032.0]), (4, [7.0]), (4, [7.0, 112.0]),
                                         (2, [1.0])])
@pytest.mark.parametrize("streamed", [False, True])
def test_parity_on_sample_reads_every_code_width(bits, scales, streamed):
    """The bench's parity check unpacks packed codes before comparing them
    with the oracle's int8 codes; a changed code, sum or output is caught."""
    torch = pytest.importorskip("torch")
    from oracle import oracle

    M, d = 3, 1001
    g = np.random.default_rng(bits).standard_normal((M, d)).astype(np.float32) * 1e-3
    ref = oracle.pipeline(g, scales, 9, d=d)
    st = FakeStep(torch, ref, M, d, bits, streamed)
    assert bench.parity_on_sample(st, ref, d, d, bits) == "bit-exact"
    if len(scales) > 1:
        # the index held as 4-bit fields reads out the same; a changed field
        # is caught
        st = FakeStep(torch, ref, M, d, bits, streamed, index_bits=4)
        assert ref["idx"].any() and bench.parity_on_sample(st, ref, d, d, bits) == "bit-exact"
        st.idx[250] ^= 0x10
        assert bench.parity_on_sample(st, ref, d, d, bits) == "MISMATCH"
    st.sum[5] += 1
    assert bench.parity_on_sample(st, ref, d, d, bits) == "MISMATCH"
    st = FakeStep(torch, ref, M, d, bits, streamed)
    st.out[7] = -st.out[7] + 1.0
    assert bench.parity_on_sample(st, ref, d, d, bits) == "MISMATCH"
    if not streamed:
        st = FakeStep(torch, ref, M, d, bits, streamed)
        if bits == 8:
            st.codes[1, 3] += 1
        else:
            st.codes[1, 0] ^= 1
        assert bench.parity_on_sample(st, ref, d, d, bits) == "MISMATCH"


def test_selection_roofline():
    """GlobalRandK's selection is priced in Philox blocks (one per four
    coordinates) against the issue-rate bound of 40 instructions per block."""
    assert abs(bench.PHILOX_PEAK_GBLOCKS - 983.04) < 1e-6
    r = bench.selection_roofline(11_173_962, 0.0285)
    assert r["bound"] == "alu" and r["algorithmic_blocks_per_launch"] == 2_793_491
    assert abs(r["achieved"] - 2_793_491 / 28.5e-6 / 1e9) < 0.1
    assert abs(r["frac"] - r["achieved"] / 983.04) < 1e-3 and r["traffic"] is None
