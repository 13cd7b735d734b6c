"""uq_shared_scale_noalloc, the variant of uq_shared_scale for callers that
cannot allocate device memory, through the C ABI: the same W (bit for bit)
and the same shared scale index as uq_shared_scale with a workspace, on two
calls in a row (the second with a smaller input, on the same static scratch)
for one scale, for several scales with 2 to 16 rows (the row maxima's keys
in the scratch), with more than 16 rows and with one row; W within one binary32 ulp
of the oracle's and the index equal to the oracle's given that W.
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

DEV = torch.device("cuda:0")


def both_ways(g, d, M, scales):
    K = len(scales)
    idx_pad = synth.round_up(max(d, 1), 256)
    w_ws = torch.full((4,), -3.0, device=DEV)
    w_na = torch.full((4,), -5.0, device=DEV)
    idx_ws = torch.full((idx_pad,), 0xEE, dtype=torch.uint8, device=DEV) if K > 1 else None
    idx_na = torch.full((idx_pad,), 0xDD, dtype=torch.uint8, device=DEV) if K > 1 else None
    ws_bytes = uq.uq_workspace_bytes(d, M)
    ws = torch.zeros(ws_bytes // 8, dtype=torch.float64, device=DEV)
    uq.uq_shared_scale(g, d, M, g.stride(0), scales, K, w_ws, idx_ws, ws, ws_bytes)
    uq.uq_shared_scale_noalloc(g, d, M, g.stride(0), scales, K, w_na, idx_na)
    torch.cuda.synchronize()
    W = np.float32(w_ws[0].item())
    assert np.float32(w_na[0].item()).view(np.int32) == W.view(np.int32)
    if K > 1:
        assert torch.equal(idx_na[:d], idx_ws[:d])
    return W, None if idx_na is None else idx_na[:d].cpu().numpy()


def check_oracle(host, d, scales, W, idx):
    W_own, _ = O.shared_scale(host, d)
    assert abs(int(W.view(np.int32)) - int(W_own.view(np.int32))) <= 1
    if len(scales) > 1:
        assert np.array_equal(idx, O.scale_index_shared(host, W, scales, d))


# (rows, first d, second d, scales): one scale; several scales with 2 to 16
# rows (the fused pass, whose row maxima's keys fill most of the scratch at
# the first size); more than 16 rows; one row
CASES = [
    (8, 3_000_017, 1_000_003, [127.0]),
    (8, 32_000_000, 2_500_001, synth.scales_for(8, 4)),
    (16, 4_000_037, 65_539, synth.scales_for(4, 4)),
    (17, 1_000_003, 10_007, synth.scales_for(8, 4)),
    (1, 777_777, 4_097, synth.scales_for(8, 8)),
]


@pytest.mark.parametrize("M,d1,d2,scales", CASES, ids=["s127-M8", "K4-M8-fused-large", "K4-M16-fused",
                                                      "K4-M17", "K8-M1"])
def test_noalloc_equals_workspace_call(M, d1, d2, scales):
    for d, seed in ((d1, 1), (d2, 2)):
        host = synth.mixed_rows(M, d, seed=seed, ldg=synth.round_up(d, 64))
        g = torch.from_numpy(host).to(DEV)
        W, idx = both_ways(g, d, M, scales)
        check_oracle(host, d, scales, W, idx)


def test_noalloc_small_and_empty_inputs():
    """Below one norm chunk, a ragged tail, and d = 0 (W = 0)."""
    for d in (1, 5, 4_099, 0):
        M = 3
        host = synth.mixed_rows(M, max(d, 1), seed=d, ldg=64 * ((max(d, 1) + 63) // 64))
        g = torch.from_numpy(host).to(DEV)
        W, idx = both_ways(g, d, M, synth.scales_for(8, 3))
        if d == 0:
            assert W == 0.0
        else:
            check_oracle(host, d, synth.scales_for(8, 3), W, idx)


def test_noalloc_beyond_the_limit_is_refused_and_launches_nothing():
    d, M = 34_000_000, 8
    # whole buffers, although the call is refused before any launch
    g = torch.zeros((M, d), device=DEV)
    w = torch.full((4,), 9.0, device=DEV)
    idx = torch.zeros(d, dtype=torch.uint8, device=DEV)
    with pytest.raises(uq.UQError) as e:
        uq.uq_shared_scale_noalloc(g, d, M, g.stride(0), synth.scales_for(8, 2), 2, w, idx)
    assert e.value.status == uq.UQ_EWORKSPACE
    torch.cuda.synchronize()
    assert w[0].item() == 9.0
