"""The oracle's multi-threaded driver changes no byte of any result.

Each row's norm stays one sequential index-order sum and every later step is
a pure function of its coordinate (Sec. 3.1-3.2, Algorithms 1-2), so the rows
and fixed coordinate chunks may run on any number of host threads: W, the
row sums, the scale index, the codes, the sums and the reconstruction must be
identical to the single-threaded pipeline for 1 and for N threads, for any
chunk length, and a window starting at i0 must equal that slice of the whole.
"""
import numpy as np
import pytest

import synth


@pytest.mark.parametrize("scales", [[127.0], synth.scales_for(8, 4), [7.0, 112.0]], ids=["s127", "K4", "K2"])
@pytest.mark.parametrize("chunk", [1 << 20, 65_536, 9_999])
def test_threads_give_identical_bytes(orc, scales, chunk):
    d, M = 300_007, 6
    g = synth.mixed_rows(M, d, seed=chunk, ldg=synth.round_up(d, 64))
    ref = orc.pipeline(g, scales, 41, d=d)
    for threads in (1, 3, 8):
        got = orc.pipeline_threaded(g, scales, 41, d=d, threads=threads, chunk=chunk)
        assert got["W_oracle"].view(np.int32) == ref["W_oracle"].view(np.int32)
        assert np.array_equal(got["sumsq"].view(np.int64), ref["sumsq"].view(np.int64))
        if len(scales) > 1:
            assert np.array_equal(got["idx"], ref["idx"])
        else:
            assert got["idx"] is None
        assert np.array_equal(got["codes"], ref["codes"])
        assert np.array_equal(got["sum"], ref["sum"])
        assert np.array_equal(got["out"].view(np.int32), ref["out"].view(np.int32))


def test_given_scale_and_worker_offset(orc):
    d, M = 50_001, 3
    g = synth.gaussian_rows(M, d, seed=2, ldg=synth.round_up(d, 64))
    W = np.float32(0.0625)
    ref = orc.pipeline(g, synth.scales_for(8, 3), 5, d=d, W=W, worker0=7)
    got = orc.pipeline_threaded(g, synth.scales_for(8, 3), 5, d=d, W=W, worker0=7, threads=4, chunk=4_096)
    assert got["W"] == W and got["W_oracle"] == ref["W_oracle"]
    for k in ("idx", "codes", "sum"):
        assert np.array_equal(got[k], ref[k]), k
    assert np.array_equal(got["out"].view(np.int32), ref["out"].view(np.int32))


@pytest.mark.parametrize("i0", [0, 1, 8, 4_093, 123_456])
def test_window_is_a_slice_of_the_whole(orc, i0):
    """The window's Philox counters follow the absolute coordinate i0 + j."""
    d, M, n = 200_000, 4, 20_011
    scales = synth.scales_for(8, 4)
    g = synth.mixed_rows(M, d, seed=9, ldg=d)
    W = orc.shared_scale(g, d)[0]
    whole = orc.pipeline(g, scales, 77, d=d, W=W)
    part = orc.window(np.ascontiguousarray(g[:, i0:i0 + n]), W, scales, 77, i0=i0, threads=3, chunk=5_000)
    assert np.array_equal(part["idx"], whole["idx"][i0:i0 + n])
    assert np.array_equal(part["codes"], whole["codes"][:, i0:i0 + n])
    assert np.array_equal(part["sum"], whole["sum"][i0:i0 + n])
    assert np.array_equal(part["out"].view(np.int32), whole["out"][i0:i0 + n].view(np.int32))


def test_default_thread_count_is_bounded():
    from oracle import oracle as O

    assert 1 <= O.default_threads() <= 16
