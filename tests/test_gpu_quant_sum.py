"""GPU parity of the fused quantise-and-sum (uq_quantize_sum) through the C ABI.

Its sums and reconstruction must equal, bit for bit, the oracle's integer sum
of the workers' codes (Eq. (8)/(12) and the all-reduce of Algorithm 1/2) and
its reconstruction (Eq. (9)/(13)), and the composed calls uq_quantize_* ->
uq_sum_codes -> uq_dequantize: one row per call into a running sum (a worker
streamed through a resident accumulator), all rows in one call, accumulating
onto sums already stored, on capped grids and past the 16-bit lane sums'
flush at 256 rows.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import synth  # noqa: E402
from oracle import oracle as O  # noqa: E402
import paper_2109_12497_amd as uq  # noqa: E402
from paper_2109_12497_amd.step import Step  # noqa: E402

DEV = torch.device("cuda:0")
SCALE_SETS = {"s127": [127.0], "s7": [7.0], "s1": [1.0], "K4": synth.scales_for(8, 4), "K2": [7.0, 112.0],
              "K8": synth.scales_for(8, 8)}


def ulps(a, b) -> int:
    return abs(int(np.float32(a).view(np.int32)) - int(np.float32(b).view(np.int32)))


def run_step(host, d, scales, seed, **kw):
    g = torch.from_numpy(np.ascontiguousarray(host)).to(DEV)
    st = Step(d, host.shape[0], scales, device=DEV, **kw)
    st.run(g, seed)
    torch.cuda.synchronize()
    return st, g


def check_oracle(st, host, d, scales, seed):
    W = np.float32(st.w[0].item())
    ref = O.pipeline(host, scales, seed, d=d, W=W)
    assert ulps(W, ref["W_oracle"]) <= 1
    if len(scales) > 1:
        assert np.array_equal(st.idx[:d].cpu().numpy(), ref["idx"]), "scale index differs"
    got = st.sum[:d].cpu().numpy()
    bad = np.flatnonzero(got != ref["sum"])
    assert bad.size == 0, f"sums differ at {bad[:8].tolist()}"
    assert np.array_equal(st.out[:d].cpu().numpy().view(np.int32), ref["out"].view(np.int32)), "outputs differ"


# forming the shared index inside the call needs several scales
FORMS = [(form, name) for form in ("per-worker", "all-rows", "all-rows-index-in-pass") for name in SCALE_SETS
         if form != "all-rows-index-in-pass" or len(SCALE_SETS[name]) > 1]


@pytest.mark.parametrize("d", [1, 5, 8, 9, 511, 512, 513, 1000, 4097, 10_007, 65_539, 200_003])
@pytest.mark.parametrize("form,name", FORMS)
def test_quant_sum_matches_oracle(d, name, form):
    """Per-worker calls, and all rows in one call with the shared index from
    uq_shared_scale or (several scales) formed inside the call."""
    scales = SCALE_SETS[name]
    M = 5
    host = synth.mixed_rows(M, d, seed=d + 3, ldg=synth.round_up(d, 64))
    kw = dict(streamed=form == "per-worker", quant_sum=True)
    if form != "per-worker":
        kw["index_in_pass"] = form == "all-rows-index-in-pass"
    st, _ = run_step(host, d, scales, seed=900 + d, **kw)
    assert st.codes is None  # no code row is kept
    check_oracle(st, host, d, scales, seed=900 + d)


@pytest.mark.parametrize("M", [1, 2, 3, 16, 17])
@pytest.mark.parametrize("name", ["s127", "K4"])
def test_quant_sum_equals_composed_calls(M, name):
    """Per-worker calls, one call for all rows, and the composed quantise /
    sum / reconstruction calls give the same sums and outputs."""
    scales = SCALE_SETS[name]
    d = 123_457
    host = synth.mixed_rows(M, d, seed=M, ldg=synth.round_up(d, 64))
    a, _ = run_step(host, d, scales, seed=11, streamed=True, quant_sum=True)
    b, _ = run_step(host, d, scales, seed=11, streamed=False, quant_sum=True, index_in_pass=False)
    c, _ = run_step(host, d, scales, seed=11, streamed=True, quant_sum=False)
    e, _ = run_step(host, d, scales, seed=11, streamed=False, fused=False)
    for st in (b, c, e):
        assert torch.equal(a.sum[:d], st.sum[:d])
        assert torch.equal(a.out[:d].view(torch.int32), st.out[:d].view(torch.int32))


def test_accumulates_onto_stored_sums():
    """accumulate = 1 adds to whatever the sums hold; without an output the
    reconstruction is not written."""
    d, M = 70_001, 3
    scales = SCALE_SETS["K4"]
    host = synth.gaussian_rows(M, d, seed=5, ldg=synth.round_up(d, 64))
    st, g = run_step(host, d, scales, seed=6, streamed=False, fused=False)
    W = np.float32(st.w[0].item())
    ref = O.pipeline(host, scales, 6, d=d, W=W)
    base = np.random.default_rng(1).integers(-10 ** 6, 10 ** 6, size=d).astype(np.int32)
    st.sum[:d].copy_(torch.from_numpy(base))
    st.out.fill_(-7.0)
    uq.uq_quantize_sum(g, d, M, g.stride(0), 0, st.w, scales, len(scales), st.idx, 6, 1, st.sum, M, None)
    torch.cuda.synchronize()
    assert np.array_equal(st.sum[:d].cpu().numpy(), base + ref["sum"])
    assert bool((st.out[:d] == -7.0).all())
    # the last worker alone, onto the first M - 1 workers' sum, with the reconstruction
    first = O.sum_codes(ref["codes"][:M - 1])
    st.sum[:d].copy_(torch.from_numpy(first))
    uq.uq_quantize_sum(g[M - 1:], d, 1, g.stride(0), M - 1, st.w, scales, len(scales), st.idx, 6, 1, st.sum, M,
                       st.out)
    torch.cuda.synchronize()
    assert np.array_equal(st.sum[:d].cpu().numpy(), ref["sum"])
    assert np.array_equal(st.out[:d].cpu().numpy().view(np.int32), ref["out"].view(np.int32))


@pytest.mark.parametrize("cap", [8, 24])
@pytest.mark.parametrize("streamed", [True, False], ids=["per-worker", "all-rows"])
def test_quant_sum_capped_grids(cap, streamed):
    """Waves striding over several tiles (the grid capped far below one tile
    per wave); the results must not depend on the grid."""
    d, M = 100_003, 4
    host = synth.mixed_rows(M, d, seed=cap, ldg=synth.round_up(d, 64))
    uq.uq_set_grid_cap(cap)
    try:
        for scales in (SCALE_SETS["s127"], SCALE_SETS["K4"]):
            for iip in ((None,) if streamed or len(scales) == 1 else (False, True)):
                st, _ = run_step(host, d, scales, seed=cap, streamed=streamed, quant_sum=True, index_in_pass=iip)
                check_oracle(st, host, d, scales, seed=cap)
    finally:
        uq.uq_set_grid_cap(0)


@pytest.mark.parametrize("M", [256, 257, 300])
@pytest.mark.parametrize("sign", [1.0, -1.0])
def test_more_rows_than_the_16_bit_lane_sums_hold(M, sign):
    """All rows in one call: the codes are summed in 16-bit lanes for up to
    256 rows, then widened.  Every row is one-hot at coordinate 0 (plus
    values too small to move its norm off 1), so that coordinate takes code
    +-127 in every row and its sum passes +-2^15 from 258 rows on."""
    d = 3_001
    scales = [127.0]
    host = np.zeros((M, synth.round_up(d, 64)), dtype=np.float32)
    host[:, 0] = sign
    host[:, 100:200] = synth.gaussian_rows(M, 100, seed=M, sigma=1e-6)
    st, _ = run_step(host, d, scales, seed=3, streamed=False, quant_sum=True)
    assert st.w[0].item() == 1.0
    assert int(st.sum[0].item()) == int(sign) * 127 * M
    check_oracle(st, host, d, scales, seed=3)


@pytest.mark.parametrize("W", [0.0, -1.0, float("inf"), float("nan"), 1e-45])
def test_forced_scale_values(W):
    """A W that is zero, negative, non-finite or so small that s_0 / W
    overflows selects the zero path: every sum and output 0."""
    d, M = 5_000, 3
    scales = SCALE_SETS["K4"]
    host = synth.gaussian_rows(M, d, seed=2, ldg=synth.round_up(d, 64))
    g = torch.from_numpy(host).to(DEV)
    st = Step(d, M, scales, device=DEV, streamed=True)
    st.shared_scale(g)
    st.w.fill_(W)
    st.sum.fill_(5)
    for m in range(M):
        st.quantize_sum(g[m:m + 1], 1, rows=1, worker0=m, accumulate=1 if m else 0, reconstruct=m == M - 1)
    torch.cuda.synchronize()
    assert int(st.sum[:d].abs().max()) == 0
    assert int(st.out[:d].view(torch.int32).abs().max()) == 0


@pytest.mark.parametrize("M", [5, 6, 8, 9, 12, 16])
@pytest.mark.parametrize("d", [1, 511, 513, 4097, 100_003])
@pytest.mark.parametrize("name", ["s127", "s7"])
def test_one_scale_rows_split_over_waves(M, d, name):
    """One scale with 5 to 16 rows set and reconstructed in one call runs the
    form that splits a tile's rows over a block's waves (two rows per wave up
    to 8 rows, four beyond); against the oracle."""
    scales = SCALE_SETS[name]
    host = synth.mixed_rows(M, d, seed=M * 7 + d, ldg=synth.round_up(d, 64))
    st, _ = run_step(host, d, scales, seed=d + M, streamed=False, quant_sum=True)
    check_oracle(st, host, d, scales, seed=d + M)


def test_rows_split_over_waves_from_a_worker_offset():
    """Rows 3..13 of 14 workers (11 rows, worker ids 3..13) in one call: the
    sums of those workers' codes and their reconstruction with M = 14."""
    d, M, seed = 50_001, 14, 21
    scales = [127.0]
    host = synth.mixed_rows(M, d, seed=4, ldg=synth.round_up(d, 64))
    st, g = run_step(host, d, scales, seed=seed, streamed=False, fused=False)
    W = np.float32(st.w[0].item())
    ref = O.pipeline(host, scales, seed, d=d, W=W)
    uq.uq_quantize_sum(g[3:], d, 11, g.stride(0), 3, st.w, scales, 1, None, seed, 0, st.sum, M, st.out)
    torch.cuda.synchronize()
    want = O.sum_codes(ref["codes"][3:14])
    assert np.array_equal(st.sum[:d].cpu().numpy(), want)
    out = O.dequantize(want, M, W, scales)
    assert np.array_equal(st.out[:d].cpu().numpy().view(np.int32), out.view(np.int32))


@pytest.mark.parametrize("cap", [8, 24])
@pytest.mark.parametrize("M", [7, 16])
def test_rows_split_over_waves_capped_grids(cap, M):
    """Blocks striding over several tiles (their LDS sums alternate between
    two buffers by tile); the results must not depend on the grid."""
    d = 100_003
    host = synth.mixed_rows(M, d, seed=cap + M, ldg=synth.round_up(d, 64))
    uq.uq_set_grid_cap(cap)
    try:
        st, _ = run_step(host, d, SCALE_SETS["s7"], seed=cap, streamed=False, quant_sum=True)
        check_oracle(st, host, d, SCALE_SETS["s7"], seed=cap)
    finally:
        uq.uq_set_grid_cap(0)


@pytest.mark.parametrize("W", [0.0, float("inf"), float("nan"), 1e-45])
@pytest.mark.parametrize("M", [6, 12])
def test_rows_split_over_waves_forced_scale_values(W, M):
    d = 5_003
    host = synth.gaussian_rows(M, d, seed=2, ldg=synth.round_up(d, 64))
    g = torch.from_numpy(host).to(DEV)
    st = Step(d, M, [127.0], device=DEV, streamed=False, quant_sum=True)
    st.shared_scale(g)
    st.w.fill_(W)
    st.sum.fill_(5)
    st.quantize_sum(g, 1)
    torch.cuda.synchronize()
    assert int(st.sum[:d].abs().max()) == 0
    assert int(st.out[:d].view(torch.int32).abs().max()) == 0
