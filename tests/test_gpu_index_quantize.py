"""GPU parity of the shared index formed inside the multi-scale quantiser with
the codes stored (uq_index_quantize) through the C ABI.

With several scales and at most 16 workers held at once, the shared scale
index of Sec. 3.2 (the rule of Eq. (11) and the min over the workers) is
formed from each coordinate's exact largest |g| over the rows, in the pass
that quantises them (Eq. (12)) and stores every worker's codes, as int8 or as
4- or 2-bit fields.  The index and the codes (unpacked) must equal the
oracle's, bit for bit, given the device's W, and the bytes of uq_shared_scale
followed by uq_quantize_multi / uq_quantize_packed given the same W: at
ragged sizes, for every row count and code width, with limits sharing a
binade, on capped grids, on the zero path and with non-finite inputs.  The
sum with the reconstruction that follows reads those codes and that index.
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
# scale sets whose smallest scale fits each code width
SCALE_SETS = {8: {"K4": synth.scales_for(8, 4), "K8": synth.scales_for(8, 8), "crowded": [3.0, 100.0, 110.0, 120.0]},
              4: {"K4": synth.scales_for(4, 4), "K2": [7.0, 112.0], "crowded": [3.0, 100.0, 110.0, 120.0]},
              2: {"K4": synth.scales_for(2, 4), "K3": [1.0, 16.0, 256.0]}}
CASES = [(bits, name) for bits in (8, 4, 2) for name in SCALE_SETS[bits]]


def ulps(a, b) -> int:
    return abs(int(np.float32(a).view(np.int32)) - int(np.float32(b).view(np.int32)))


def run_step(host, d, scales, seed, bits, index_in_pass=True, fused=True):
    g = torch.from_numpy(np.ascontiguousarray(host)).to(DEV)
    st = Step(d, host.shape[0], scales, device=DEV, streamed=False, bits=bits, quant_sum=False, fused=fused,
              index_in_pass=index_in_pass)
    st.run(g, seed)
    torch.cuda.synchronize()
    return st, g


def codes_of(st, d):
    """The step's code rows as int8 [rows, d] (packed fields unpacked by the oracle's routine)."""
    c = st.codes.cpu().numpy().view(np.uint8)
    if st.bits == 8:
        return c[:, :d].view(np.int8)
    nb = (d * st.bits + 7) // 8
    return np.stack([O.unpack_codes(c[m, :nb], d, st.bits) for m in range(c.shape[0])])


def check_oracle(st, host, d, scales, seed):
    W = np.float32(st.w[0].item())
    ref = O.pipeline(host, scales, seed, d=d, W=W)
    if not np.isnan(W):
        assert ulps(W, ref["W_oracle"]) <= 1
    bad = np.flatnonzero(st.idx[:d].cpu().numpy() != ref["idx"])
    assert bad.size == 0, f"scale index differs at {bad[:8].tolist()}"
    bad = np.argwhere(codes_of(st, d) != ref["codes"])
    assert bad.size == 0, f"codes differ at (worker, coordinate) {bad[:5].tolist()}"
    assert np.array_equal(st.sum[:d].cpu().numpy(), ref["sum"]), "sums differ"
    assert np.array_equal(st.out[:d].cpu().numpy().view(np.int32), ref["out"].view(np.int32)), "outputs differ"
    return ref


@pytest.mark.parametrize("d", [1, 5, 8, 9, 511, 512, 513, 1000, 4097, 10_007, 65_539])
@pytest.mark.parametrize("bits,name", CASES)
def test_matches_oracle(d, bits, name):
    scales = SCALE_SETS[bits][name]
    M = 5
    host = synth.mixed_rows(M, d, seed=d + bits, ldg=synth.round_up(d, 64))
    st, _ = run_step(host, d, scales, seed=300 + d, bits=bits)
    assert st.index_in_pass
    check_oracle(st, host, d, scales, seed=300 + d)


@pytest.mark.parametrize("M", [1, 2, 3, 4, 7, 8, 9, 15, 16])
@pytest.mark.parametrize("bits", [8, 4])
def test_every_row_count(M, bits):
    """Each register-tile instance (2, 4, 8 and 16 rows), with rows past M
    re-reading row M - 1 and not quantised."""
    d = 20_011
    scales = SCALE_SETS[bits]["K4"]
    host = synth.mixed_rows(M, d, seed=M, ldg=synth.round_up(d, 64))
    st, _ = run_step(host, d, scales, seed=M + 100, bits=bits)
    check_oracle(st, host, d, scales, seed=M + 100)


@pytest.mark.parametrize("M", [2, 6, 16])
@pytest.mark.parametrize("bits,name", CASES)
def test_equals_separate_index_pass(M, bits, name):
    """Bit for bit the separate calls given the same W: uq_shared_scale's
    index and the quantiser's code bytes (every byte of each row's codes)."""
    d = 70_001
    scales = SCALE_SETS[bits][name]
    host = synth.mixed_rows(M, d, seed=M + 7, ldg=synth.round_up(d, 64))
    a, g = run_step(host, d, scales, seed=77, bits=bits, index_in_pass=False)
    b = Step(d, M, scales, device=DEV, streamed=False, bits=bits, quant_sum=False, index_in_pass=True)
    b.w.copy_(a.w)
    b.index_quantize(g, 77)
    torch.cuda.synchronize()
    assert torch.equal(a.idx[:d], b.idx[:d])
    nb = (d * bits + 7) // 8
    assert torch.equal(a.codes[:, :nb], b.codes[:, :nb])


@pytest.mark.parametrize("cap", [8, 24])
@pytest.mark.parametrize("M", [3, 16])
def test_capped_grids(cap, M):
    """Waves striding over several tiles (the grid capped far below one tile
    per wave): the results must not depend on the grid."""
    d = 100_003
    host = synth.mixed_rows(M, d, seed=cap + M, ldg=synth.round_up(d, 64))
    uq.uq_set_grid_cap(cap)
    try:
        for bits, name in ((4, "K4"), (8, "crowded"), (2, "K3")):
            scales = SCALE_SETS[bits][name]
            st, _ = run_step(host, d, scales, seed=cap, bits=bits)
            check_oracle(st, host, d, scales, seed=cap)
    finally:
        uq.uq_set_grid_cap(0)


@pytest.mark.parametrize("W", [0.0, -1.0, float("inf"), float("nan"), 1e-45])
@pytest.mark.parametrize("bits", [8, 4])
def test_forced_scale_values(W, bits):
    """A W that is zero, negative, non-finite or so small that s_0 / W
    overflows selects the zero path: every index K - 1, every code 0."""
    d, M = 5_000 + 3, 3
    scales = SCALE_SETS[bits]["K4"]
    host = synth.gaussian_rows(M, d, seed=2, ldg=synth.round_up(d, 64))
    g = torch.from_numpy(host).to(DEV)
    st = Step(d, M, scales, device=DEV, streamed=False, bits=bits, quant_sum=False, index_in_pass=True)
    st.shared_scale(g, w_only=True)
    st.w.fill_(W)
    st.codes.fill_(0x55)
    st.idx.fill_(0)
    st.index_quantize(g, 1)
    torch.cuda.synchronize()
    assert bool((st.idx[:d] == len(scales) - 1).all())
    assert not codes_of(st, d).any()


@pytest.mark.parametrize("bad", [np.inf, -np.inf, np.nan])
def test_non_finite_inputs(bad):
    """A non-finite gradient makes W non-finite: the zero path, as the
    oracle takes it."""
    d, M = 999, 4
    scales = SCALE_SETS[4]["K4"]
    host = synth.gaussian_rows(M, d, seed=3, ldg=synth.round_up(d, 64))
    host[2, 500] = bad
    st, _ = run_step(host, d, scales, seed=4, bits=4)
    check_oracle(st, host, d, scales, seed=4)


def test_separate_sum_and_reconstruction():
    """fused = False: the codes summed, then reconstructed by their own calls."""
    d, M = 33_333, 9
    scales = SCALE_SETS[4]["K4"]
    host = synth.mixed_rows(M, d, seed=9, ldg=synth.round_up(d, 64))
    st, _ = run_step(host, d, scales, seed=5, bits=4, fused=False)
    check_oracle(st, host, d, scales, seed=5)


def test_rejects_more_than_16_rows():
    d, M = 1000, 17
    g = torch.zeros((M, 1024), dtype=torch.float32, device=DEV)
    st = Step(d, 16, SCALE_SETS[4]["K4"], device=DEV, streamed=False, bits=4, quant_sum=False)
    codes = torch.zeros((M, 512), dtype=torch.uint8, device=DEV)
    with pytest.raises(uq.UQError) as e:
        uq.uq_index_quantize(g, d, M, g.stride(0), st.w, SCALE_SETS[4]["K4"], 4, 1, 4, st.idx, codes, 512)
    assert e.value.status == uq.UQ_ERANGE
