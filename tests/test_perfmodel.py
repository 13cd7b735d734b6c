"""The analytic scaling model: collective costs, the choice between an
int16 all-reduce and an all-gather of packed codes, and the byte counts of
the local kernels."""
import math

import pytest

from paper_2109_12497_amd import perfmodel as pm

FLAT = pm.Network("no latency", 100.0, 0.0)


def test_ring_collectives():
    net = pm.Network("x", 100.0, 3.0)
    assert net.ring_allreduce_s(1e9, 1) == 0.0 and net.ring_allgather_s(1e9, 1) == 0.0
    P, n = 8, 4e8
    assert math.isclose(net.ring_allreduce_s(n, P), 2 * (P - 1) * (3e-6 + n / (P * 100e9)))
    assert math.isclose(net.ring_allgather_s(n, P), (P - 1) * (3e-6 + n / 100e9))
    # the bandwidth term of a ring all-reduce tends to 2 n / B
    assert FLAT.ring_allreduce_s(n, 10_000) == pytest.approx(2 * n / 100e9, rel=1e-3)


@pytest.mark.parametrize("bits", [2, 4])
def test_packed_allgather_wins_below_32_over_bits_gpus(bits):
    """Bandwidth terms: (P - 1) d b / 8 / B against 4 (P - 1) d / (P B)."""
    d = 10 ** 8
    sc = pm.Scheme("packed", bits)
    cross = 32 // bits
    for P in (2, cross - 1, cross + 1, 4 * cross):
        gather = FLAT.ring_allgather_s(d * bits / 8, P)
        reduce16 = FLAT.ring_allreduce_s(2 * d, P)
        assert (gather < reduce16) == (P < cross), P
        # plus the exchange of W (one fp32)
        assert math.isclose(pm.comm_s(d, P, sc, FLAT), min(gather, reduce16) + FLAT.ring_allreduce_s(4, P))


def test_int16_codes_halve_the_fp32_exchange():
    d, P = 10 ** 8, 8
    fp32 = pm.comm_s(d, P, pm.SCHEMES[0], FLAT)
    int16 = FLAT.ring_allreduce_s(2 * d, P)
    assert math.isclose(fp32, 2 * int16)


def test_local_bytes():
    d = 10 ** 9
    rate = pm.LOCAL_TBPS * 1e12
    assert pm.local_s(d, pm.Scheme("fp32", None)) == 0.0
    assert math.isclose(pm.local_s(d, pm.Scheme("8", 8)), d * 17 / rate)
    assert math.isclose(pm.local_s(d, pm.Scheme("8m", 8, True)), d * 24 / rate)
    assert math.isclose(pm.local_s(d, pm.Scheme("4", 4)), d * 16.5 / rate)


def test_compression_pays_on_slow_links_and_little_on_xgmi():
    d = 138_357_544  # VGG-16
    eth, xgmi7 = pm.NETWORKS["eth-10g"], pm.NETWORKS["xgmi-7rings"]
    for sc in pm.SCHEMES[1:]:
        # one scale: int16 sums (or packed codes) against fp32; several scales
        # also exchange the shared index, 3 bytes per coordinate in all
        want = 1.3 if sc.several_scales else 1.9
        assert pm.step_s(d, 32, pm.SCHEMES[0], eth) / pm.step_s(d, 32, sc, eth) > want, sc.name
    # over seven xGMI rings at P = 2 the 8-bit exchange saves about what the
    # local work costs: the two steps are within 10% of each other
    ratio = pm.step_s(d, 2, pm.SCHEMES[0], xgmi7) / pm.step_s(d, 2, pm.SCHEMES[1], xgmi7)
    assert 0.9 < ratio < 1.1, ratio
