"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Bar (include/uq.h arithmetic contract): scale index, codes, sums and the
reconstructed output bit-exact; W within one binary32 ulp of the oracle's
sequential fp64 norm, and every later stage is checked with the oracle fed
the device's W.  Small cases span several tiles and ragged tails; the full
workloads are checked in full where the oracle finishes in seconds and on
sampled coordinate windows otherwise.
"""
import math

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU-only hosts, run only with a GPU
    pytest.skip("needs a GPU", allow_module_level=True)

import synth  # noqa: E402
from oracle import oracle as O  # noqa: E402
import paper_2109_12497_amd as uq  # noqa: E402
from paper_2109_12497_amd.step import Step  # noqa: E402

DEV = torch.device("cuda:0")
S_SINGLE = [127.0]
S_MULTI4 = synth.scales_for(8, 4)


def ulps(a, b) -> int:
    return abs(int(np.float32(a).view(np.int32)) - int(np.float32(b).view(np.int32)))


def gpu_step(host_g, d, scales, seed, streamed=False, quant_sum=None):
    g = torch.from_numpy(np.ascontiguousarray(host_g)).to(DEV)
    M = host_g.shape[0]
    step = Step(d, M, scales, device=DEV, streamed=streamed, quant_sum=quant_sum)
    step.run(g, seed)
    torch.cuda.synchronize()
    res = dict(W=np.float32(step.w[0].item()), sum=step.sum[:d].cpu().numpy(),
               out=step.out[:d].cpu().numpy(),
               idx=None if step.idx is None else step.idx[:d].cpu().numpy())
    if step.codes is not None and not streamed:
        res["codes"] = step.codes[:, :d].cpu().numpy()
    return res, step, g


def assert_matches_oracle(res, host_g, d, scales, seed, worker0=0):
    ref = O.pipeline(host_g, scales, seed, d=d, W=res["W"], worker0=worker0)
    assert ulps(res["W"], ref["W_oracle"]) <= 1, (res["W"], ref["W_oracle"])
    if len(scales) > 1:
        assert np.array_equal(res["idx"], ref["idx"]), "scale index differs"
    if "codes" in res:
        bad = np.argwhere(res["codes"] != ref["codes"])
        assert bad.size == 0, f"codes differ at {bad[:5].tolist()}"
    assert np.array_equal(res["sum"], ref["sum"]), "sums differ"
    assert np.array_equal(res["out"].view(np.int32), ref["out"].view(np.int32)), "outputs differ"
    return ref


# ---------------------------------------------------------------------------
# Small shapes: several tiles, ragged tails, edge values
# ---------------------------------------------------------------------------

SHAPES = [1, 2, 3, 4, 5, 7, 8, 9, 15, 16, 17, 31, 33, 255, 1000, 2049, 4097, 10007, 65539]


@pytest.mark.parametrize("d", SHAPES)
@pytest.mark.parametrize("scales", [S_SINGLE, [7.0], [1.0], S_MULTI4, [7.0, 112.0], synth.scales_for(8, 8)],
                         ids=["s127", "s7", "s1", "K4", "K2", "K8"])
def test_small_shapes(d, scales):
    M = 3
    host = synth.mixed_rows(M, d, seed=d, ldg=synth.round_up(d, 64))
    res, _, _ = gpu_step(host, d, scales, seed=1000 + d)
    assert_matches_oracle(res, host, d, scales, seed=1000 + d)


@pytest.mark.parametrize("M", [1, 2, 3, 4, 5, 8, 9, 16, 17, 300])
def test_worker_counts(M):
    """From 2 to 16 rows the shared scale with several scales takes the fused
    norm + row-maximum pass (4, 8 or 16 accumulators, exact or with rows to
    spare); one row, and 17 and more, take the separate norm and index
    passes."""
    d = 12_345
    host = synth.gaussian_rows(M, d, seed=M, ldg=synth.round_up(d, 64))
    for scales in (S_SINGLE, S_MULTI4):
        res, _, _ = gpu_step(host, d, scales, seed=77)
        assert_matches_oracle(res, host, d, scales, seed=77)


@pytest.mark.parametrize("d", [7, 600])
def test_max_rows(d):
    """The largest row count the ABI accepts (the grid's y extent): every
    worker id up to 65534 enters the random stream."""
    M = 65535
    host = synth.gaussian_rows(M, d, seed=d, ldg=64 * ((d + 63) // 64))
    for scales in (S_SINGLE, S_MULTI4):
        res, _, _ = gpu_step(host, d, scales, seed=99)
        assert_matches_oracle(res, host, d, scales, seed=99)


@pytest.mark.parametrize("scales,bits", [(S_SINGLE, 8), (S_MULTI4, 8), ([7.0], 4), ([7.0, 112.0, 1792.0], 4),
                                         ([1.0], 2), ([1.0, 16.0], 2)],
                         ids=["s127", "K4", "s7-4bit", "K3-4bit", "s1-2bit", "K2-2bit"])
@pytest.mark.parametrize("d", [1, 5, 4095, 4097, 65_539])
def test_fused_sum_reconstruction_equals_separate_calls(scales, bits, d):
    """uq_sum_dequantize against the sum call followed by uq_dequantize: the
    same sums and outputs bit for bit, when the sum is set and when three of
    the five workers' rows are added to a running sum."""
    M = 5
    host = synth.mixed_rows(M, d, seed=d + bits, ldg=synth.round_up(d, 64))
    g = torch.from_numpy(np.ascontiguousarray(host)).to(DEV)
    sep = Step(d, M, scales, device=DEV, bits=bits, fused=False)
    fus = Step(d, M, scales, device=DEV, bits=bits, fused=True)
    sep.run(g, 5)
    fus.run(g, 5)
    torch.cuda.synchronize()
    assert torch.equal(sep.codes, fus.codes)

    def same():
        assert torch.equal(sep.sum[:d], fus.sum[:d])
        assert torch.equal(sep.out[:d].view(torch.int32), fus.out[:d].view(torch.int32))

    same()
    sep.sum_codes(rows=3, accumulate=1)
    sep.dequantize()
    fus.sum_dequantize(rows=3, accumulate=1)
    torch.cuda.synchronize()
    same()


@pytest.mark.parametrize("streamed", [False, True], ids=["rows", "streamed"])
@pytest.mark.parametrize("scales", [S_SINGLE, S_MULTI4], ids=["s127", "K4"])
def test_separate_sum_and_reconstruction_match_oracle(scales, streamed):
    """The step with the separate sum and reconstruction calls, against the oracle."""
    M, d = 6, 20_011
    host = synth.mixed_rows(M, d, seed=M + d, ldg=synth.round_up(d, 64))
    g = torch.from_numpy(np.ascontiguousarray(host)).to(DEV)
    step = Step(d, M, scales, device=DEV, streamed=streamed, fused=False)
    step.run(g, 41)
    torch.cuda.synchronize()
    res = dict(W=np.float32(step.w[0].item()), sum=step.sum[:d].cpu().numpy(), out=step.out[:d].cpu().numpy(),
               idx=None if step.idx is None else step.idx[:d].cpu().numpy())
    if not streamed:
        res["codes"] = step.codes[:, :d].cpu().numpy()
    assert_matches_oracle(res, host, d, scales, seed=41)


@pytest.mark.parametrize("cap", [8, 24, 1000])
@pytest.mark.parametrize("M", [1, 3, 17])
def test_capped_grids(cap, M):
    """Every streaming pass on a grid capped far below its one-shot size, so
    that its threads, waves and blocks stride over several units (the default
    cap of 2^22 blocks binds only past about 2^33 coordinates); one row, the
    fused pass's row counts and more than 16 rows.  The results must not
    depend on the grid."""
    d = 100_003
    host = synth.mixed_rows(M, d, seed=M + cap, ldg=synth.round_up(d, 64))
    uq.uq_set_grid_cap(cap)
    try:
        for scales in (S_SINGLE, S_MULTI4):
            res, _, _ = gpu_step(host, d, scales, seed=cap + M)
            assert_matches_oracle(res, host, d, scales, seed=cap + M)
            # one row at a time into the running sum, the last call with the
            # reconstruction: fused quantise-and-sum, and codes stored then summed
            for qs in (True, False):
                res, _, _ = gpu_step(host, d, scales, seed=cap + M, streamed=True, quant_sum=qs)
                assert_matches_oracle(res, host, d, scales, seed=cap + M)
    finally:
        uq.uq_set_grid_cap(0)


@pytest.mark.parametrize("scales", [S_SINGLE, S_MULTI4], ids=["s127", "K4"])
def test_capped_grids_separate_sum_and_reconstruction(scales):
    """The separate sum and reconstruction kernels on a grid capped at 8 blocks."""
    M, d = 3, 70_001
    host = synth.mixed_rows(M, d, seed=17, ldg=synth.round_up(d, 64))
    g = torch.from_numpy(np.ascontiguousarray(host)).to(DEV)
    uq.uq_set_grid_cap(8)
    try:
        step = Step(d, M, scales, device=DEV, fused=False)
        step.run(g, 19)
        torch.cuda.synchronize()
    finally:
        uq.uq_set_grid_cap(0)
    res = dict(W=np.float32(step.w[0].item()), sum=step.sum[:d].cpu().numpy(), out=step.out[:d].cpu().numpy(),
               idx=None if step.idx is None else step.idx[:d].cpu().numpy(), codes=step.codes[:, :d].cpu().numpy())
    assert_matches_oracle(res, host, d, scales, seed=19)


@pytest.mark.parametrize("scales", [S_SINGLE, S_MULTI4], ids=["s127", "K4"])
@pytest.mark.parametrize("M", [5, 17])
def test_tightest_leading_dimensions(scales, M):
    """Gradient rows padded only to a multiple of 4 floats and code rows only
    to a multiple of 16 bytes, so that rows start at irregular addresses."""
    d = 10_003
    ldg, ldc = 10_004, 10_016
    host = synth.mixed_rows(M, d, seed=M + 40, ldg=ldg)
    g = torch.from_numpy(np.ascontiguousarray(host)).to(DEV)
    assert g.stride(0) == ldg
    step = Step(d, M, scales, device=DEV, ldc=ldc)
    assert step.codes.stride(0) == ldc
    step.run(g, 314)
    torch.cuda.synchronize()
    res = dict(W=np.float32(step.w[0].item()), sum=step.sum[:d].cpu().numpy(), out=step.out[:d].cpu().numpy(),
               idx=None if step.idx is None else step.idx[:d].cpu().numpy(), codes=step.codes[:, :d].cpu().numpy())
    assert_matches_oracle(res, host, d, scales, seed=314)


def test_seed_high_word_and_worker_offset():
    d, M = 3001, 2
    host = synth.gaussian_rows(M, d, seed=5, ldg=3008)
    seed = (0xDEADBEEF << 32) | 0x12345678
    g = torch.from_numpy(host).to(DEV)
    step = Step(d, M, S_MULTI4, device=DEV)
    step.shared_scale(g)
    step.quantize(g, seed, rows=M, worker0=1000)
    torch.cuda.synchronize()
    W = np.float32(step.w[0].item())
    ref = O.pipeline(host, S_MULTI4, seed, d=d, W=W, worker0=1000)
    assert np.array_equal(step.codes[:, :d].cpu().numpy(), ref["codes"])


def test_one_call_equals_per_worker_calls():
    """rows = M in one call (one grid) equals M calls with rows = 1 (another grid)."""
    d, M = 50_003, 6
    host = synth.mixed_rows(M, d, seed=3, ldg=synth.round_up(d, 64))
    g = torch.from_numpy(host).to(DEV)
    for scales in (S_SINGLE, S_MULTI4):
        step = Step(d, M, scales, device=DEV)
        step.shared_scale(g)
        step.quantize(g, seed=9)
        whole = step.codes.clone()
        for m in range(M):
            step.quantize(g[m:m + 1], seed=9, rows=1, worker0=m, codes=step.codes[m:m + 1])
        torch.cuda.synchronize()
        assert torch.equal(whole, step.codes)


def test_accumulate_equals_set():
    d, M = 40_000, 5
    host = synth.gaussian_rows(M, d, seed=8, ldg=40_000)
    res, step, g = gpu_step(host, d, S_MULTI4, seed=4)
    for qs in (True, False):
        res_s, _, _ = gpu_step(host, d, S_MULTI4, seed=4, streamed=True, quant_sum=qs)
        assert np.array_equal(res["sum"], res_s["sum"])
        assert np.array_equal(res["out"].view(np.int32), res_s["out"].view(np.int32))


def test_repeatable():
    d, M = 100_000, 4
    host = synth.mixed_rows(M, d, seed=12, ldg=synth.round_up(d, 64))
    a, _, _ = gpu_step(host, d, S_MULTI4, seed=5)
    b, _, _ = gpu_step(host, d, S_MULTI4, seed=5)
    for k in ("W", "sum", "out", "idx", "codes"):
        assert np.array_equal(np.asarray(a[k]), np.asarray(b[k]))


# ---------------------------------------------------------------------------
# Degenerate cases
# ---------------------------------------------------------------------------

def test_zero_gradients():
    d, M = 1025, 3
    host = np.zeros((M, 1088), dtype=np.float32)
    for scales in (S_SINGLE, S_MULTI4):
        res, _, _ = gpu_step(host, d, scales, seed=1)
        assert res["W"] == 0 and not res["codes"].any() and not res["sum"].any() and not res["out"].any()
        if len(scales) > 1:
            assert np.all(res["idx"] == len(scales) - 1)


def _largest_passing(inv: np.float32, s0: np.float32) -> np.float32:
    """Largest binary32 a with RN32(a * inv) <= s0, by stepping ulps from s0 / inv."""
    a = np.float32(np.float64(s0) / np.float64(inv))
    while np.float32(a * inv) > s0:
        a = np.nextafter(a, np.float32(0))
    while np.float32(np.nextafter(a, np.float32(np.inf)) * inv) <= s0:
        a = np.nextafter(a, np.float32(np.inf))
    return a


@pytest.mark.parametrize("M", [4, 17])
def test_index_at_scale_boundaries(M):
    """Coordinates exactly at, and one ulp either side of, the largest |g|
    each scale k >= 1 admits (RN32(|g| inv_k) <= s_0), with W fixed by a
    one-hot row at a value that is not a power of two: the shared index
    (M = 4: from the row maxima of the fused pass; M = 17: from the rows)
    and everything after it match the oracle."""
    scales = S_MULTI4
    Wv = np.float32(0.7)
    d = 4096 + 37
    host = np.zeros((M, synth.round_up(d, 64)), dtype=np.float32)
    host[0, 0] = Wv
    rng = np.random.default_rng(M)
    host[1:, :d] = (rng.standard_normal((M - 1, d)) * 1e-6).astype(np.float32)
    col = 100
    for k in range(1, len(scales)):
        inv = np.float32(np.float64(np.float32(scales[k])) / np.float64(Wv))
        T = _largest_passing(inv, np.float32(scales[0]))
        for v in (T, np.nextafter(T, np.float32(0)), np.nextafter(T, np.float32(np.inf))):
            for sign in (1, -1):
                host[1 + (col % (M - 1)), col] = sign * v
                col += 7
    assert np.sqrt((host.astype(np.float64) ** 2).sum(axis=1)).max() == np.float64(Wv)
    res, _, _ = gpu_step(host, d, scales, seed=5)
    assert res["W"] == Wv
    ref = assert_matches_oracle(res, host, d, scales, seed=5)
    # the boundary coordinates really do split between neighbouring indices
    assert len(set(ref["idx"][100:col:7].tolist())) >= 3


@pytest.mark.parametrize("cap", [0, 8], ids=["one-shot", "capped"])
@pytest.mark.parametrize("M", [2, 8, 16])
def test_many_maxima_in_a_thresholds_key_bucket(M, cap):
    """With several scales and 2 to 16 rows the index pass reads the row
    maxima and compares each with the scales' limits: thousands of
    coordinates placed within 2^-9 (relative) of the limits (at most 150 per
    row near W/16, so that a one-hot row still sets W), in the binades where
    the pass's exponent table holds them, plus tiny denormal maxima (the
    table's lowest binade); on one-shot grids and on grids of 8 blocks; all
    against the oracle."""
    scales = synth.scales_for(8, 4)
    Wv = np.float32(0.9)
    d = 40_000 + 13
    rng = np.random.default_rng(M)
    host = np.zeros((M, synth.round_up(d, 64)), dtype=np.float32)
    host[1:, 1:d] = (rng.standard_normal((M - 1, d - 1)) * 1e-7).astype(np.float32)
    cols = rng.permutation(np.arange(1, d))
    counts = {1: 150 * (M - 1), 2: 6000, 3: 12000}
    at = 0
    for k in range(1, len(scales)):
        inv = np.float32(np.float64(np.float32(scales[k])) / np.float64(Wv))
        T = _largest_passing(inv, np.float32(scales[0]))
        c = cols[at:at + counts[k]]
        at += counts[k]
        vals = (T * (1.0 + rng.uniform(-2.0 ** -9, 2.0 ** -9, size=c.size))).astype(np.float32)
        rows = 1 + np.arange(c.size) % (M - 1)  # spread evenly over the rows after the first
        host[rows, c] = vals * rng.choice(np.array([1, -1], dtype=np.float32), size=c.size)
    tiny = cols[at:at + 5000]
    host[1 + np.arange(tiny.size) % (M - 1), tiny] = (rng.integers(1, 1 << 14, size=tiny.size) *
                                                      (2.0 ** -149)).astype(np.float32)
    host[0, :] = 0.0
    host[0, 0] = Wv  # a one-hot row: its norm is W
    assert np.sqrt((host.astype(np.float64) ** 2).sum(axis=1)).max() == np.float64(Wv)
    uq.uq_set_grid_cap(cap)  # 8 blocks: the passes' grid-stride loops
    try:
        res, _, _ = gpu_step(host, d, scales, seed=9)
    finally:
        uq.uq_set_grid_cap(0)
    assert res["W"] == Wv
    ref = assert_matches_oracle(res, host, d, scales, seed=9)
    assert len(set(ref["idx"].tolist())) == len(scales)


@pytest.mark.parametrize("bad", [np.inf, -np.inf, np.nan])
def test_non_finite_inputs_take_zero_path(bad):
    d, M = 999, 2
    host = synth.gaussian_rows(M, d, seed=2, ldg=1024)
    host[1, 500] = bad
    for scales in (S_SINGLE, S_MULTI4):
        res, _, _ = gpu_step(host, d, scales, seed=1)
        assert not np.isfinite(res["W"])
        assert not res["codes"].any() and not res["out"].any()
        assert_matches_oracle(res, host, d, scales, seed=1)


@pytest.mark.parametrize("W", [0.0, -1.0, np.inf, np.nan, 1e-45, 3e-38, 1e-33, 5e-30])
def test_forced_scale_values(W):
    """Stages after the norm with a caller-chosen W, including the zero path
    and W small enough that the larger scales' reciprocals overflow."""
    d, M = 4099, 3
    host = synth.mixed_rows(M, d, seed=6, ldg=4160) * np.float32(1e-30)
    g = torch.from_numpy(host).to(DEV)
    for scales in (S_SINGLE, synth.scales_for(8, 8)):
        step = Step(d, M, scales, device=DEV)
        step.w.fill_(float(W))
        if len(scales) > 1:
            idx_host = O.scale_index_shared(host, np.float32(W), scales, d=d)
            step.idx[:d].copy_(torch.from_numpy(idx_host))
        step.quantize(g, seed=3)
        step.sum_codes()
        step.dequantize()
        torch.cuda.synchronize()
        ref = O.pipeline(host, scales, 3, d=d, W=np.float32(W))
        assert np.array_equal(step.codes[:, :d].cpu().numpy(), ref["codes"])
        assert np.array_equal(step.out[:d].cpu().numpy().view(np.int32), ref["out"].view(np.int32))


@pytest.mark.parametrize("tiny", [1e-32, 1e-36])
def test_tiny_norms(tiny):
    """Rows so small that s_k / W exceeds 2^100: the quantiser then applies
    its 2^16 scaling after the clamp instead of folding it into the tables."""
    d, M = 5000, 3
    host = synth.mixed_rows(M, d, seed=9, ldg=5056) * np.float32(tiny)
    for scales in (S_SINGLE, [7.0], S_MULTI4):
        res, _, _ = gpu_step(host, d, scales, seed=4)
        assert np.isfinite(res["W"]) and scales[-1] / float(res["W"]) > 2.0 ** 100
        assert_matches_oracle(res, host, d, scales, seed=4)


@pytest.mark.parametrize("W", [1.0, 1e-33])
def test_non_finite_values_with_given_scale(W):
    """With a caller-given finite W, NaN and infinite coordinates get code 0
    and the others their usual codes (a tile with and one without them)."""
    d, M = 3000, 2
    host = synth.gaussian_rows(M, d, seed=11, ldg=3008)
    host[0, [5, 700, 2999]] = [np.inf, np.nan, -np.inf]
    host[1, [0, 511, 1500]] = [-np.nan, np.inf, np.nan]
    g = torch.from_numpy(host).to(DEV)
    for scales in (S_SINGLE, S_MULTI4):
        step = Step(d, M, scales, device=DEV)
        step.w.fill_(float(W))
        idx_host = None
        if len(scales) > 1:
            idx_host = O.scale_index_shared(np.nan_to_num(host, nan=0.0, posinf=0.0, neginf=0.0), np.float32(W),
                                            scales, d=d)
            step.idx[:d].copy_(torch.from_numpy(idx_host))
        step.quantize(g, seed=5)
        step.sum_codes()
        step.dequantize()
        torch.cuda.synchronize()
        codes = np.stack([O.quantize(host[m, :d], np.float32(W), scales, 5, worker=m, idx=idx_host)
                          for m in range(M)])
        assert codes[0, 700] == 0 and codes[1, 511] == 0
        assert np.array_equal(step.codes[:, :d].cpu().numpy(), codes)
        out = O.dequantize(O.sum_codes(codes), M, np.float32(W), scales, idx_host)
        assert np.array_equal(step.out[:d].cpu().numpy().view(np.int32), out.view(np.int32))


def test_index_entries_beyond_K_read_as_last():
    d, M = 777, 2
    host = synth.gaussian_rows(M, d, seed=4, ldg=832)
    g = torch.from_numpy(host).to(DEV)
    step = Step(d, M, S_MULTI4, device=DEV)
    step.shared_scale(g)
    torch.cuda.synchronize()
    idx_host = np.random.default_rng(0).integers(0, 256, size=d).astype(np.uint8)
    step.idx[:d].copy_(torch.from_numpy(idx_host))
    step.quantize(g, seed=8)
    step.sum_codes()
    step.dequantize()
    torch.cuda.synchronize()
    W = np.float32(step.w[0].item())
    codes = np.stack([O.quantize(host[m, :d], W, S_MULTI4, 8, worker=m, idx=idx_host) for m in range(M)])
    assert np.array_equal(step.codes[:, :d].cpu().numpy(), codes)
    out = O.dequantize(O.sum_codes(codes), M, W, S_MULTI4, idx_host)
    assert np.array_equal(step.out[:d].cpu().numpy().view(np.int32), out.view(np.int32))


def test_empty_vector():
    step = Step(0, 2, S_MULTI4, device=DEV)
    g = torch.ones((2, 64), device=DEV)
    step.w.fill_(7.0)
    step.run(g, seed=1)
    torch.cuda.synchronize()
    assert step.w[0].item() == 0.0


# ---------------------------------------------------------------------------
# The paper-shaped workloads at full size, in the launch configuration the
# benchmark times (the same Step calls)
# ---------------------------------------------------------------------------

def device_norm_check(g, d, W):
    """W within one ulp of RN32(sqrt(max_m sum g^2)) computed by torch in fp64."""
    best = 0.0
    for m in range(g.shape[0]):
        s = 0.0
        for c in range(0, d, 1 << 26):
            x = g[m, c:min(d, c + (1 << 26))].double()
            s += float(torch.dot(x, x))
        best = max(best, s)
    assert ulps(W, np.float32(math.sqrt(best))) <= 1


def check_windows(step, g, d, scales, seed, windows, streamed):
    W = np.float32(step.w[0].item())
    M = g.shape[0]
    for i0, n in windows:
        i1 = min(d, i0 + n)
        host = g[:, i0:i1].cpu().numpy()
        idx = O.scale_index_shared(host, W, scales) if len(scales) > 1 else None
        if idx is not None:
            assert np.array_equal(step.idx[i0:i1].cpu().numpy(), idx), f"idx window {i0}"
        codes = np.stack([O.quantize(host[m], W, scales, seed, worker=m, i0=i0, idx=idx) for m in range(M)])
        if not streamed:
            assert np.array_equal(step.codes[:, i0:i1].cpu().numpy(), codes), f"codes window {i0}"
        sums = O.sum_codes(codes)
        assert np.array_equal(step.sum[i0:i1].cpu().numpy(), sums), f"sum window {i0}"
        out = O.dequantize(sums, M, W, scales, idx)
        assert np.array_equal(step.out[i0:i1].cpu().numpy().view(np.int32), out.view(np.int32)), f"out {i0}"


def sample_windows(d, n_windows=12, width=1 << 14, seed=0):
    rng = np.random.default_rng(seed)
    starts = [0, max(0, d - width - 5)] + [int(x) for x in rng.integers(0, d - width, size=n_windows)]
    return [(s, width + 5) for s in starts]


@pytest.mark.parametrize("name", ["small-gaussian", "resnet18", "resnet50"])
def test_workload_full_parity(name):
    g, cfg = synth.make_gradients(name, device=DEV)
    d, M, scales, seed = cfg["d"], cfg["M"], cfg["scales"], cfg["seed"]
    step = Step(d, M, scales, device=DEV)
    step.run(g, seed)
    torch.cuda.synchronize()
    host = g[:, :d].cpu().numpy()
    res = dict(W=np.float32(step.w[0].item()), codes=step.codes[:, :d].cpu().numpy(),
               sum=step.sum[:d].cpu().numpy(), out=step.out[:d].cpu().numpy(),
               idx=None if step.idx is None else step.idx[:d].cpu().numpy())
    assert_matches_oracle(res, host, d, scales, seed)


def test_student_t_streamed_composed_sampled_parity():
    """The 2^30-coordinate workload with each streamed worker's codes stored
    and then summed (two calls per worker; the fused quantise-and-sum the
    benchmark times is compared at every coordinate elsewhere): windows
    against the oracle."""
    g, cfg = synth.make_gradients("student-t", device=DEV)
    d, M, scales, seed = cfg["d"], cfg["M"], cfg["scales"], cfg["seed"]
    step = Step(d, M, scales, device=DEV, streamed=True, quant_sum=False)
    step.run(g, seed)
    torch.cuda.synchronize()
    device_norm_check(g, d, np.float32(step.w[0].item()))
    check_windows(step, g, d, scales, seed, sample_windows(d, n_windows=8, seed=5), streamed=True)
    assert int(step.sum[:d].abs().max()) <= M * scales[0]


def test_rows_longer_than_2_pow_31():
    """d = 2^31 + 777 coordinates per row (64-bit indexing, grid caps, Philox
    counters above 2^28): oracle windows around 2^31 and at the ragged end,
    W against a float64 norm, and the integer sum over every coordinate."""
    d, M = (1 << 31) + 777, 2
    scales = S_MULTI4
    ldg = synth.round_up(d, 64)
    gen = torch.Generator(device=DEV)
    gen.manual_seed(31)
    g = torch.zeros((M, ldg), dtype=torch.float32, device=DEV)
    for m in range(M):
        for c in range(0, d, 1 << 28):
            n = min(1 << 28, d - c)
            g[m, c:c + n].normal_(0.0, 1e-3, generator=gen)
    g[1, (1 << 31) + 5] = 0.25  # a large coordinate past 2^31 sets the shared index there
    step = Step(d, M, scales, device=DEV)
    step.run(g, 4321)
    torch.cuda.synchronize()
    device_norm_check(g, d, np.float32(step.w[0].item()))
    w = 1 << 14
    windows = [(0, w), ((1 << 31) - w // 2, w), ((1 << 31) + 1, w), (d - w, w), ((1 << 30) + 12345, w)]
    check_windows(step, g, d, scales, 4321, windows, streamed=False)
    for c in range(0, d, 1 << 28):
        e = min(d, c + (1 << 28))
        assert torch.equal(step.codes[:, c:e].to(torch.int32).sum(dim=0), step.sum[c:e]), c
    del g, step
    torch.cuda.empty_cache()


def test_shared_scale_rows_longer_than_2_pow_32():
    """d = 2^32 + 2^22 + 333 coordinates, two rows, four scales: the norm
    pass's partial sums then take more than 256 second-level sums per row,
    the one size range where the index pass's set-up sums each row in the
    fixed order of the first level instead of one partial per thread.  W
    against a float64 norm; the shared index against the oracle on windows
    around 2^32 and at the ragged end."""
    d, M = (1 << 32) + (1 << 22) + 333, 2
    scales = S_MULTI4
    g = _long_rows(d, M, seed=32)
    g[0, (1 << 32) + 77] = 0.5  # a large coordinate past 2^32 sets the index there
    w = torch.zeros(4, dtype=torch.float32, device=DEV)
    idx = torch.zeros(synth.round_up(d, 256), dtype=torch.uint8, device=DEV)
    wsb = uq.uq_workspace_bytes(d, M)
    ws = torch.zeros(wsb // 8 + 1, dtype=torch.float64, device=DEV)
    uq.uq_shared_scale(g, d, M, g.stride(0), scales, len(scales), w, idx, ws, wsb)
    torch.cuda.synchronize()
    W = np.float32(w[0].item())
    device_norm_check(g, d, W)
    n = 1 << 14
    for i0 in (0, (1 << 32) - n // 2, (1 << 32) + 1, d - n):
        host = g[:, i0:i0 + n].cpu().numpy()
        ref = O.scale_index_shared(host, W, scales)
        assert np.array_equal(idx[i0:i0 + n].cpu().numpy(), ref), f"idx window {i0}"
    del g, idx, ws
    torch.cuda.empty_cache()


def _long_rows(d, M, seed):
    ldg = synth.round_up(d, 64)
    gen = torch.Generator(device=DEV)
    gen.manual_seed(seed)
    g = torch.zeros((M, ldg), dtype=torch.float32, device=DEV)
    for m in range(M):
        for c in range(0, d, 1 << 28):
            n = min(1 << 28, d - c)
            g[m, c:c + n].normal_(0.0, 1e-3, generator=gen)
    return g


def test_packed_rows_longer_than_2_pow_31():
    """4-bit packed codes over 2^31 + 777 coordinates: oracle windows (the
    packed row unpacked) around 2^31 and at the ragged end."""
    d, M, scales, seed = (1 << 31) + 777, 2, [7.0, 112.0], 77
    g = _long_rows(d, M, 32)
    step = Step(d, M, scales, device=DEV, bits=4)
    step.run(g, seed)
    torch.cuda.synchronize()
    W = np.float32(step.w[0].item())
    w = 1 << 14
    # even window starts: a window begins on a byte of the packed row
    for i0 in ((1 << 31) - w // 2, (1 << 31) + 2, (d - w) & ~1):
        i1 = min(d, i0 + w)
        host = g[:, i0:i1].cpu().numpy()
        idx = O.scale_index_shared(host, W, scales)
        assert np.array_equal(step.idx[i0:i1].cpu().numpy(), idx), i0
        codes = np.stack([O.quantize(host[m], W, scales, seed, worker=m, i0=i0, idx=idx) for m in range(M)])
        packed = step.codes[:, i0 // 2:(i1 + 1) // 2].cpu().numpy()
        for m in range(M):
            assert np.array_equal(O.unpack_codes(packed[m], i1 - i0, 4), codes[m]), (i0, m)
        assert np.array_equal(step.sum[i0:i1].cpu().numpy(), O.sum_codes(codes)), i0
    del g, step
    torch.cuda.empty_cache()


def test_streamed_rows_longer_than_2_pow_31():
    """The streamed accumulator (one code row reused, sum += per worker) over
    2^31 + 777 coordinates: windows against the oracle, and the sum bounded."""
    d, M, scales, seed = (1 << 31) + 777, 2, synth.scales_for(8, 3), 78
    g = _long_rows(d, M, 33)
    step = Step(d, M, scales, device=DEV, streamed=True)
    step.run(g, seed)
    torch.cuda.synchronize()
    device_norm_check(g, d, np.float32(step.w[0].item()))
    w = 1 << 14
    check_windows(step, g, d, scales, seed, [((1 << 31) - w // 2, w), (d - w, w)], streamed=True)
    assert int(step.sum[:d].abs().max()) <= M * scales[0]
    del g, step
    torch.cuda.empty_cache()


# (scales, whether two limits share a binade when W = 0.9)
CLOSE_SCALES = [([3.0, 100.0, 110.0, 120.0], True), ([7.0, 112.0, 120.0, 1792.0], True),
                ([3.0, 20.0, 50.0, 120.0, 300.0], False), ([1.0, 3.0, 7.0, 15.0, 31.0, 63.0, 127.0], False)]


@pytest.mark.parametrize("scales,crowded", CLOSE_SCALES, ids=["crowded3", "crowded2", "adjacent4", "adjacent6"])
@pytest.mark.parametrize("M", [3, 16])
def test_index_with_close_scales(scales, crowded, M):
    """Scale sets whose limits share a binade (the index pass then counts
    with K compares per coordinate) or sit one per binade in neighbouring
    binades (its exponent table): coordinates at, and one ulp either side of,
    every limit, and magnitudes spread over many binades, against the oracle
    (Eq. (11) and the min over workers)."""
    Wv = np.float32(0.9)
    limits = []
    for k in range(1, len(scales)):
        inv = np.float32(np.float64(np.float32(scales[k])) / np.float64(Wv))
        limits.append(_largest_passing(inv, np.float32(scales[0])))
    binades = [int(np.float32(t).view(np.uint32)) >> 23 for t in limits]
    assert (len(set(binades)) < len(binades)) == crowded
    d = 8192 + 37
    rng = np.random.default_rng(M + len(scales))
    host = np.zeros((M, synth.round_up(d, 64)), dtype=np.float32)
    host[0, 0] = Wv  # a one-hot row: its norm is W
    for m in range(1, M):
        cols = rng.choice(np.arange(1, d), size=100, replace=False)
        host[m, cols] = (10.0 ** rng.uniform(-6.0, np.log10(0.05), size=100) *
                         rng.choice([-1.0, 1.0], size=100)).astype(np.float32)
    col = 9
    for T in limits:
        for v in (T, np.nextafter(T, np.float32(0)), np.nextafter(T, np.float32(np.inf))):
            for sign in (1, -1):
                host[1 + (col % (M - 1)), col] = sign * v
                col += 11
    assert np.sqrt((host.astype(np.float64) ** 2).sum(axis=1)).max() == np.float64(Wv)
    res, _, _ = gpu_step(host, d, scales, seed=23)
    assert res["W"] == Wv
    ref = assert_matches_oracle(res, host, d, scales, seed=23)
    assert len(set(ref["idx"][9:col:11].tolist())) >= 3


def _random_configs(n=24, seed=2109):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        bits = int(rng.choice([8, 8, 4, 2]))
        K = int(rng.integers(1, 6))
        d = int(rng.choice([int(rng.integers(1, 600)), int(rng.integers(600, 40_000)),
                            int(rng.integers(40_000, 300_000))]))
        M = int(rng.choice([1, 2, 3, 5, 8, 16, 17, 23]))
        out.append(dict(d=d, M=M, scales=synth.scales_for(bits, K), bits=bits,
                        streamed=bool(rng.integers(0, 2)), fused=bool(rng.integers(0, 3) > 0),
                        cap=int(rng.choice([0, 0, 8, 64])), seed=int(rng.integers(0, 2 ** 63)), case=i))
    return out


@pytest.mark.parametrize("cfg", _random_configs(), ids=lambda c: f"case{c['case']}")
def test_random_configurations(cfg):
    """Seeded random mixes of d (ragged, one tile to several hundred), worker
    count (across the fused pass's 2..16 and beyond), scale count, code width,
    streamed or materialised codes, fused or separate sum and reconstruction,
    and grid cap, against the oracle."""
    d, M, scales, bits, seed = cfg["d"], cfg["M"], cfg["scales"], cfg["bits"], cfg["seed"]
    host = synth.mixed_rows(M, d, seed=cfg["case"] + 100, ldg=synth.round_up(d, 64))
    g = torch.from_numpy(np.ascontiguousarray(host)).to(DEV)
    uq.uq_set_grid_cap(cfg["cap"])
    try:
        step = Step(d, M, scales, device=DEV, streamed=cfg["streamed"], bits=bits, fused=cfg["fused"])
        step.run(g, seed)
        torch.cuda.synchronize()
    finally:
        uq.uq_set_grid_cap(0)
    W = np.float32(step.w[0].item())
    ref = O.pipeline(host, scales, seed, d=d, W=W)
    assert ulps(W, ref["W_oracle"]) <= 1, (W, ref["W_oracle"])
    if len(scales) > 1:
        assert np.array_equal(step.idx[:d].cpu().numpy(), ref["idx"]), "scale index differs"
    if not cfg["streamed"]:
        if bits == 8:
            assert np.array_equal(step.codes[:, :d].cpu().numpy(), ref["codes"]), "codes differ"
        else:
            packed = step.codes[:, :(d * bits + 7) // 8].cpu().numpy()
            for m in range(M):
                assert np.array_equal(O.unpack_codes(packed[m], d, bits), ref["codes"][m]), f"codes row {m}"
    assert np.array_equal(step.sum[:d].cpu().numpy(), ref["sum"]), "sums differ"
    assert np.array_equal(step.out[:d].cpu().numpy().view(np.int32), ref["out"].view(np.int32)), "outputs differ"


def test_concurrent_steps_on_two_streams():
    """The library keeps no state between calls: two steps with their own
    buffers, issued interleaved on two streams (default priority), give the
    results each gives alone."""
    d1, d2, M = 200_003, 150_001, 5
    h1 = synth.mixed_rows(M, d1, seed=61, ldg=synth.round_up(d1, 64))
    h2 = synth.mixed_rows(M, d2, seed=62, ldg=synth.round_up(d2, 64))
    g1 = torch.from_numpy(np.ascontiguousarray(h1)).to(DEV)
    g2 = torch.from_numpy(np.ascontiguousarray(h2)).to(DEV)
    a = Step(d1, M, S_SINGLE, device=DEV)
    b = Step(d2, M, S_MULTI4, device=DEV)
    a.run(g1, 7)
    b.run(g2, 8)
    torch.cuda.synchronize()
    ref_a, ref_b = a.out[:d1].clone(), b.out[:d2].clone()
    ref_ca, ref_cb = a.codes.clone(), b.codes.clone()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    s1.wait_stream(torch.cuda.current_stream())
    s2.wait_stream(torch.cuda.current_stream())
    for _ in range(5):
        a.run(g1, 7, stream=s1)
        b.run(g2, 8, stream=s2)
    torch.cuda.synchronize()
    assert torch.equal(a.codes, ref_ca) and torch.equal(b.codes, ref_cb)
    assert torch.equal(a.out[:d1].view(torch.int32), ref_a.view(torch.int32))
    assert torch.equal(b.out[:d2].view(torch.int32), ref_b.view(torch.int32))
