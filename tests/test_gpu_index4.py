"""GPU parity of the shared index held as 4-bit fields (uq_shared_scale_idx4,
uq_quantize_sum_idx4) through the C ABI.

Sec. 3.2 (the rule of Eq. (11) with scale sharing) forms one index per
coordinate; with at most 16 scales it fits a nibble, two coordinates a byte
(the low nibble first).  The index values must equal uq_shared_scale's at
every coordinate, on every kernel path that forms them (the norm + maxima
pass for 2 to 16 rows, the row re-reading pass for one row or more than 16),
with the unused high nibble of an odd d left 0; and the quantise-and-sum
reading them (one streamed worker per call or all rows in one call,
accumulating, with and without the reconstruction) must give the sums and
outputs of uq_quantize_sum with the byte index and of the oracle, bit for
bit: at ragged sizes, on capped grids and with limits sharing a binade.
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
from paper_2109_12497_amd.step import Step, round_up  # noqa: E402

DEV = torch.device("cuda:0")
SCALE_SETS = {"K2": [7.0, 112.0], "K4": synth.scales_for(8, 4), "K8": synth.scales_for(8, 8),
              "crowded": [3.0, 100.0, 110.0, 120.0],
              "K16": [float(2 ** k) for k in range(16)]}


def nibbles(idx4, d):
    """Host values of the 4-bit layout, written out from its definition."""
    b = idx4[:(d + 1) // 2].cpu().numpy()
    out = np.empty(2 * b.size, dtype=np.uint8)
    out[0::2] = b & 0xF
    out[1::2] = b >> 4
    return out[:d], b


def both_indices(host, d, scales):
    g = torch.from_numpy(np.ascontiguousarray(host)).to(DEV)
    M = host.shape[0]
    ws_bytes = uq.uq_workspace_bytes(d, M)
    ws = torch.zeros(ws_bytes // 8 + 1, dtype=torch.float64, device=DEV)
    w8 = torch.zeros(4, dtype=torch.float32, device=DEV)
    w4 = torch.zeros(4, dtype=torch.float32, device=DEV)
    idx8 = torch.zeros(round_up(max(d, 1), 256), dtype=torch.uint8, device=DEV)
    idx4 = torch.full((round_up((max(d, 1) + 1) // 2, 256),), 0xEE, dtype=torch.uint8, device=DEV)
    uq.uq_shared_scale(g, d, M, g.stride(0), scales, len(scales), w8, idx8, ws, ws_bytes)
    uq.uq_shared_scale_idx4(g, d, M, g.stride(0), scales, len(scales), w4, idx4, ws, ws_bytes)
    torch.cuda.synchronize()
    return g, w8, w4, idx8, idx4


@pytest.mark.parametrize("d", [1, 2, 3, 7, 8, 9, 15, 17, 1000, 1001, 4097, 65_539, 200_003])
@pytest.mark.parametrize("M", [1, 2, 5, 16, 17])
def test_index_values_equal_the_byte_layout(d, M):
    scales = SCALE_SETS["K8"] if M != 5 else SCALE_SETS["crowded"]
    host = synth.mixed_rows(M, d, seed=d + M, ldg=synth.round_up(d, 64))
    _, w8, w4, idx8, idx4 = both_indices(host, d, scales)
    assert torch.equal(w8[:1], w4[:1])
    vals, raw = nibbles(idx4, d)
    assert np.array_equal(vals, idx8[:d].cpu().numpy())
    if d % 2:
        assert raw[-1] >> 4 == 0, "the unused high nibble of the last byte"
    # nothing past the layout's (d + 1) / 2 bytes is written
    assert bool((idx4[(d + 1) // 2:] == 0xEE).all())


@pytest.mark.parametrize("name", list(SCALE_SETS))
def test_sixteen_scales_and_every_value(name):
    """K up to 16 (index values up to 15, the full nibble) against the oracle."""
    scales = SCALE_SETS[name]
    d, M = 30_011, 3
    host = synth.mixed_rows(M, d, seed=len(scales), ldg=synth.round_up(d, 64))
    _, _, w4, _, idx4 = both_indices(host, d, scales)
    ref = O.pipeline(host, scales, 1, d=d, W=np.float32(w4[0].item()))
    vals, _ = nibbles(idx4, d)
    assert np.array_equal(vals, ref["idx"])


def run_streamed(host, d, scales, seed, index_bits):
    g = torch.from_numpy(np.ascontiguousarray(host)).to(DEV)
    st = Step(d, host.shape[0], scales, device=DEV, streamed=True, index_bits=index_bits)
    st.run(g, seed)
    torch.cuda.synchronize()
    return st


@pytest.mark.parametrize("d", [1, 9, 511, 513, 1001, 4097, 65_539, 200_003])
@pytest.mark.parametrize("name", ["K2", "K8", "crowded", "K16"])
def test_streamed_step_matches_oracle_and_byte_index(d, name):
    scales = SCALE_SETS[name]
    M = 4
    host = synth.mixed_rows(M, d, seed=d, ldg=synth.round_up(d, 64))
    a = run_streamed(host, d, scales, 21, 4)
    b = run_streamed(host, d, scales, 21, 8)
    assert torch.equal(a.w[:1], b.w[:1])
    assert np.array_equal(a.index_host(), b.idx[:d].cpu().numpy())
    assert torch.equal(a.sum[:d], b.sum[:d])
    assert torch.equal(a.out[:d].view(torch.int32), b.out[:d].view(torch.int32))
    ref = O.pipeline(host, scales, 21, d=d, W=np.float32(a.w[0].item()))
    assert np.array_equal(a.index_host(), ref["idx"])
    assert np.array_equal(a.sum[:d].cpu().numpy(), ref["sum"])
    assert np.array_equal(a.out[:d].cpu().numpy().view(np.int32), ref["out"].view(np.int32))


@pytest.mark.parametrize("cap", [8, 24])
def test_capped_grids(cap):
    """Waves and blocks striding over several tiles and octets."""
    d, M = 300_007, 16
    scales = SCALE_SETS["K8"]
    host = synth.mixed_rows(M, d, seed=cap, ldg=synth.round_up(d, 64))
    uq.uq_set_grid_cap(cap)
    try:
        a = run_streamed(host, d, scales, cap, 4)
    finally:
        uq.uq_set_grid_cap(0)
    ref = O.pipeline(host, scales, cap, d=d, W=np.float32(a.w[0].item()))
    assert np.array_equal(a.index_host(), ref["idx"])
    assert np.array_equal(a.sum[:d].cpu().numpy(), ref["sum"])
    assert np.array_equal(a.out[:d].cpu().numpy().view(np.int32), ref["out"].view(np.int32))


@pytest.mark.parametrize("rows", [1, 3])
@pytest.mark.parametrize("reconstruct", [False, True])
def test_quantize_sum_calls_equal_byte_index(rows, reconstruct):
    """One call of `rows` rows onto sums already stored (accumulate = 1), with
    and without the reconstruction: the two index layouts give the same sums
    and outputs."""
    d, M = 70_001, 6
    scales = SCALE_SETS["K4"]
    host = synth.mixed_rows(M, d, seed=rows, ldg=synth.round_up(d, 64))
    g, w8, _, idx8, idx4 = both_indices(host, d, scales)
    start = torch.randint(-1000, 1000, (round_up(d, 64),), dtype=torch.int32, device=DEV)
    res = []
    for call, idx in ((uq.uq_quantize_sum, idx8), (uq.uq_quantize_sum_idx4, idx4)):
        s = start.clone()
        out = torch.zeros(round_up(d, 64), dtype=torch.float32, device=DEV) if reconstruct else None
        call(g[1:1 + rows], d, rows, g.stride(0), 1, w8, scales, len(scales), idx, 5, 1, s, M, out)
        torch.cuda.synchronize()
        res.append((s, out))
    assert torch.equal(res[0][0][:d], res[1][0][:d])
    if reconstruct:
        assert torch.equal(res[0][1][:d].view(torch.int32), res[1][1][:d].view(torch.int32))
