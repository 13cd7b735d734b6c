"""Pins for the oracle's sub-byte codes: two's complement fields of 4 or 2
bits, low bits first (the packing discussed in Sec. 5 and Appendix A)."""
import itertools
import json
import os

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
GOLD = json.load(open(os.path.join(HERE, "golden", "packed_codes.json")))


@pytest.mark.parametrize("case", GOLD["cases"], ids=lambda c: f"{c['bits']}bit")
def test_hand_packed_examples(orc, case):
    codes = np.array(case["codes"], dtype=np.int8)
    want = np.array([int(x, 16) for x in case["bytes"]], dtype=np.uint8)
    assert np.array_equal(orc.pack_codes(codes, case["bits"]), want)
    assert np.array_equal(orc.unpack_codes(want, codes.size, case["bits"]), codes)


@pytest.mark.parametrize("bits,lo,hi", [(4, -8, 7), (2, -2, 1)])
def test_round_trip_every_value_every_position(orc, bits, lo, hi):
    per = 8 // bits
    vals = list(range(lo, hi + 1))
    for combo in itertools.product(vals, repeat=per):
        codes = np.array(combo * 3 + combo[:1], dtype=np.int8)  # several bytes and a ragged tail
        packed = orc.pack_codes(codes, bits)
        assert packed.size == (codes.size + per - 1) // per
        assert np.array_equal(orc.unpack_codes(packed, codes.size, bits), codes)


@pytest.mark.parametrize("bits,s", [(4, 7), (2, 1)])
def test_packed_sum_equals_int8_sum(orc, bits, s):
    rng = np.random.default_rng(bits)
    rows, n = 9, 1001
    codes = rng.integers(-s, s + 1, size=(rows, n)).astype(np.int8)
    per = 8 // bits
    ldp = (n + per - 1) // per + 5
    packed = np.zeros((rows, ldp), dtype=np.uint8)
    for r in range(rows):
        p = orc.pack_codes(codes[r], bits)
        packed[r, :p.size] = p
    assert np.array_equal(orc.sum_packed(packed, n, bits), codes.astype(np.int64).sum(axis=0))


def test_quantiser_codes_fit_the_field(orc):
    """|code| <= s_min: s = 7 codes fit 4 bits, s = 1 codes fit 2 bits."""
    rng = np.random.default_rng(2)
    v = rng.normal(size=5000).astype(np.float32)
    W, _ = orc.shared_scale(v.reshape(1, -1))
    for s, bits in ((7.0, 4), (1.0, 2)):
        c = orc.quantize(v, W, [s], seed=3)
        assert np.array_equal(orc.unpack_codes(orc.pack_codes(c, bits), c.size, bits), c)
