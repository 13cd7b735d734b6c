"""The scale tables' device arithmetic against the host's IEEE operations,
bitwise: inv_k = RN32(s_k / W) and deq_k = RN32(W / (M s_k)) are formed as a
binary64 quotient rounded to binary32 (correctly rounded, since 53 >= 2*24 + 2),
and W = RN32(sqrt(S)) from the binary64 sum of squares.  The helper library
(tests/kat/uq_tables.hip) runs the library's own device function on arrays;
it is built by __graft_entry__.build() (tests/kat/tables_helper.py) with the
library's compiler flags."""
import ctypes
import os

import numpy as np
import pytest

LIB = os.path.join(os.path.dirname(os.path.abspath(__file__)), "kat", "libuq_tables.so")

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

DEV = torch.device("cuda:0")


@pytest.fixture(scope="module")
def helper():
    if not os.path.exists(LIB):
        pytest.fail(f"{LIB} is not built; run __graft_entry__.build()")
    L = ctypes.CDLL(LIB)
    P, i64 = ctypes.c_void_p, ctypes.c_int64
    L.uqt_div_rn32.argtypes = [P, P, P, i64, P]
    L.uqt_sqrt_rn32.argtypes = [P, P, i64, P]
    return L


def _bits(x: np.ndarray) -> np.ndarray:
    return x.view(np.uint32 if x.dtype == np.float32 else np.uint64)


def _same(got: np.ndarray, want: np.ndarray) -> np.ndarray:
    """Bitwise equal, any NaN matching any NaN."""
    return (_bits(got) == _bits(want)) | (np.isnan(got) & np.isnan(want))


def _random_floats(rng, n, lo_exp, hi_exp):
    """Positive binary32 values with uniformly random exponents and mantissas."""
    e = rng.integers(lo_exp, hi_exp + 1, n)
    m = rng.integers(0, 1 << 23, n)
    return ((e.astype(np.uint32) << 23) | m.astype(np.uint32)).view(np.float32)


def test_table_division_is_correctly_rounded(helper):
    rng = np.random.default_rng(2109)
    n = 1 << 20
    # numerators: scale values (integers exactly representable in binary32, and
    # M * s_k products) and arbitrary floats; denominators: W over the whole
    # normal and subnormal range, and M * s_k
    ints = rng.integers(1, 1 << 24, n).astype(np.float32)
    anyf = _random_floats(rng, n, 1, 254)
    subn = (rng.integers(1, 1 << 23, n).astype(np.uint32)).view(np.float32)
    a = np.where(rng.random(n) < 0.5, ints, anyf).astype(np.float32)
    b = np.where(rng.random(n) < 0.8, _random_floats(rng, n, 1, 254), subn).astype(np.float32)
    # the other direction (W / (M s_k)) and edge cases: zero, infinity, NaN,
    # the largest and smallest floats, exact powers of two
    special = np.array([0.0, np.inf, np.nan, 1.0, 2.0 ** -149, 2.0 ** -126, np.finfo(np.float32).max,
                        127.0, 32512.0, 0.7], dtype=np.float32)
    sa, sb = np.meshgrid(special, special)
    a = np.concatenate([a, b, sa.ravel()]).astype(np.float32)
    b = np.concatenate([b, ints, sb.ravel()]).astype(np.float32)
    ta, tb = torch.from_numpy(a).to(DEV), torch.from_numpy(b).to(DEV)
    tq = torch.empty_like(ta)
    assert helper.uqt_div_rn32(ta.data_ptr(), tb.data_ptr(), tq.data_ptr(), a.size,
                               torch.cuda.current_stream().cuda_stream) == 0
    got = tq.cpu().numpy()
    with np.errstate(divide="ignore", invalid="ignore", over="ignore", under="ignore"):
        want = (a / b).astype(np.float32)  # numpy float32 division: IEEE round to nearest even
    ok = _same(got, want)
    assert ok.all(), f"{(~ok).sum()} of {a.size} quotients differ, e.g. {a[~ok][:3]} / {b[~ok][:3]}"


def test_norm_square_root_is_correctly_rounded(helper):
    rng = np.random.default_rng(2110)
    n = 1 << 20
    # sums of squares: binary64 values across the range the norms take (from
    # squares of subnormal floats to sums near the binary32 overflow)
    e = rng.integers(1023 - 300, 1023 + 260, n).astype(np.uint64)
    m = rng.integers(0, 1 << 52, n, dtype=np.uint64)
    s = ((e << np.uint64(52)) | m).view(np.float64)
    special = np.array([0.0, np.inf, np.nan, 1.0, 2.0 ** -298, float(np.finfo(np.float32).max) ** 2,
                        (float(np.finfo(np.float32).max) ** 2) * 1.0000001], dtype=np.float64)
    s = np.concatenate([s, special])
    ts = torch.from_numpy(s).to(DEV)
    tw = torch.empty(s.size, dtype=torch.float32, device=DEV)
    assert helper.uqt_sqrt_rn32(ts.data_ptr(), tw.data_ptr(), s.size, torch.cuda.current_stream().cuda_stream) == 0
    got = tw.cpu().numpy()
    with np.errstate(over="ignore", invalid="ignore"):
        want = np.sqrt(s).astype(np.float32)  # correctly rounded binary64 sqrt, then one rounding
    ok = _same(got, want)
    assert ok.all(), f"{(~ok).sum()} of {s.size} roots differ, e.g. {s[~ok][:3]}"
