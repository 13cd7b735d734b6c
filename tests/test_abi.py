"""The C ABI contract, checked without a GPU.

The library must load, export every function include/uq.h declares, and
reject every invalid argument with the documented status before it touches
the HIP runtime (so these calls are safe on a machine with no GPU).
"""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "uq.h")

uq = pytest.importorskip("paper_2109_12497_amd", reason="libuq.so not built")
L = uq.lib

A = 0x10000  # a 16-byte aligned stand-in address; never dereferenced by a rejected call
S127 = [127.0]
S4 = [127.0, 2032.0, 32512.0, 520192.0]


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\*?\s+\*?(uq_[a-z_]+)\s*\(", text, re.M)))


def test_header_declares_the_five_calls():
    names = declared_functions()
    for name in ("uq_shared_scale", "uq_quantize_single", "uq_quantize_multi", "uq_sum_codes", "uq_dequantize",
                 "uq_workspace_bytes", "uq_strerror", "uq_last_error"):
        assert name in names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(uq.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_probe_library_is_separate():
    """The bandwidth-probe kernels live in their own library: libuq does not
    export them, libuq_probe.so does, and its argument checks need no GPU."""
    import os

    lib = ctypes.CDLL(uq.LIB_PATH)
    probe = ctypes.CDLL(os.path.join(os.path.dirname(uq.LIB_PATH), "libuq_probe.so"))
    for name in ("uqp_read", "uqp_read_write8", "uqp_read_out_floats"):
        assert hasattr(probe, name) and not hasattr(lib, name), name
    probe.uqp_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p]
    probe.uqp_read_out_floats.argtypes = [ctypes.c_int64]
    probe.uqp_read_out_floats.restype = ctypes.c_int64
    assert probe.uqp_read(None, 512, None, None) == -1
    assert probe.uqp_read(16, 500, 16, None) == -1   # not a multiple of 512
    assert probe.uqp_read_out_floats(512) == 256


def test_strerror_and_workspace():
    assert uq.uq_strerror(0) == "success"
    for status in (-1, -2, -3, -4, -5):
        assert uq.uq_strerror(status) not in ("success", "unknown status")
    assert uq.uq_strerror(12345) == "unknown status"
    assert uq.uq_workspace_bytes(0, 1) >= 8
    for d, M in ((1, 1), (2 ** 20, 4), (11_173_962, 8), (2 ** 30, 16), (2 ** 30, 17), (5, 300)):
        b = uq.uq_workspace_bytes(d, M)
        assert b % 256 == 0 and b >= 8 * M
        if 2 <= M <= 16:
            # several scales with 2 to 16 rows: d 16-bit keys of the row
            # maxima, one fp64 partial per row and 1024 coordinates, their
            # sums per 16384 partials, M row sums, and the index pass's
            # constants (a 256-entry table of 8 bytes, two words per scale
            # for at most 16 scales, one flag), and up to 4 KiB to align the
            # keys
            tiles = -(-d // 1024)
            consts = 256 * 8 + 2 * 4 * 16 + 4
            assert 2 * d <= b <= 2 * d + 8 * M * (tiles + -(-tiles // 16384) + 1) + consts + 4096 + 6 * 256
        else:
            assert b <= 8 * M * 1024 + 256
    assert uq.uq_workspace_bytes(2 ** 30, 17) <= 17 * 1024 * 8 + 256


def _hs(vals):
    return uq._HostScales(vals).array


def status_shared(g=A, d=100, M=2, ldg=128, scales=S127, K=1, w=A, idx=A, ws=A, ws_bytes=1 << 20):
    hs = uq._HostScales(scales)
    return L.uq_shared_scale(g, d, M, ldg, hs.ptr, K, w, idx, ws, ws_bytes, None)


def status_qs(g=A, d=100, rows=2, ldg=128, worker0=0, w=A, s=127, seed=1, codes=A, ldc=128):
    return L.uq_quantize_single(g, d, rows, ldg, worker0, w, s, seed, codes, ldc, None)


def status_qm(g=A, d=100, rows=2, ldg=128, worker0=0, w=A, scales=S4, K=4, idx=A, seed=1, codes=A, ldc=128):
    hs = uq._HostScales(scales)
    return L.uq_quantize_multi(g, d, rows, ldg, worker0, w, hs.ptr, K, idx, seed, codes, ldc, None)


def status_sum(codes=A, d=100, rows=2, ldc=128, acc=0, sum_=A):
    return L.uq_sum_codes(codes, d, rows, ldc, acc, sum_, None)


def status_deq(sum_=A, d=100, M=2, w=A, scales=S127, K=1, idx=None, out=A):
    hs = uq._HostScales(scales)
    return L.uq_dequantize(sum_, d, M, w, hs.ptr, K, idx, out, None)


E = dict(inval=uq.UQ_EINVAL, range=uq.UQ_ERANGE, align=uq.UQ_EALIGN, ws=uq.UQ_EWORKSPACE)


@pytest.mark.parametrize("kw,want", [
    (dict(g=None), "inval"), (dict(d=-1), "inval"), (dict(M=0), "inval"), (dict(M=70000), "range"),
    (dict(ldg=64), "inval"), (dict(ldg=130), "align"), (dict(g=A + 4), "align"), (dict(w=None), "inval"),
    (dict(w=A + 2), "align"), (dict(ws=None), "inval"), (dict(ws=A + 8), "align"), (dict(ws_bytes=8), "ws"),
    (dict(K=0), "range"), (dict(K=17, scales=[float(i + 1) for i in range(17)]), "range"),
    (dict(K=2, scales=[3.0, 3.0]), "range"), (dict(K=2, scales=[3.0, 2.5]), "range"),
    (dict(K=2, scales=[3.5, 7.0]), "range"), (dict(K=2, scales=[0.0, 7.0]), "range"),
    (dict(K=2, scales=[128.0, 256.0]), "range"), (dict(K=2, scales=[7.0, float("inf")]), "range"),
    (dict(K=2, scales=[7.0, float("nan")]), "range"), (dict(K=2, scales=S4[:2], idx=None), "inval"),
    (dict(K=2, scales=S4[:2], idx=A + 1), "align"), (dict(K=2, scales=None), "inval"),
])
def test_shared_scale_rejects(kw, want):
    assert status_shared(**kw) == E[want]
    assert uq.uq_last_error() != ""


def status_shared4(g=A, d=100, M=2, ldg=128, scales=S4, K=4, w=A, idx=A, ws=A, ws_bytes=1 << 20):
    hs = uq._HostScales(scales)
    return L.uq_shared_scale_idx4(g, d, M, ldg, hs.ptr, K, w, idx, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,want", [
    # one scale has no index to hold
    (dict(K=1, scales=S127), "inval"), (dict(K=1, scales=None, idx=None), "inval"),
    # then the checks of uq_shared_scale
    (dict(g=None), "inval"), (dict(M=0), "inval"), (dict(ldg=130), "align"), (dict(w=None), "inval"),
    (dict(ws=None), "inval"), (dict(ws_bytes=8), "ws"), (dict(idx=None), "inval"), (dict(idx=A + 1), "align"),
    (dict(K=17, scales=[float(i + 1) for i in range(17)]), "range"), (dict(K=2, scales=[3.0, 2.5]), "range"),
])
def test_shared_scale_idx4_rejects(kw, want):
    assert status_shared4(**kw) == E[want]
    assert uq.uq_last_error() != ""


def status_noalloc(g=A, d=100, M=2, ldg=128, scales=S127, K=1, w=A, idx=A):
    hs = uq._HostScales(scales)
    return L.uq_shared_scale_noalloc(g, d, M, ldg, hs.ptr, K, w, idx, None)


@pytest.mark.parametrize("kw,want", [
    (dict(g=None), "inval"), (dict(d=-1), "inval"), (dict(M=0), "inval"), (dict(M=70000), "range"),
    (dict(ldg=64), "inval"), (dict(ldg=130), "align"), (dict(g=A + 4), "align"), (dict(w=None), "inval"),
    (dict(w=A + 2), "align"), (dict(K=0), "range"), (dict(K=2, scales=[3.0, 3.0]), "range"),
    (dict(K=2, scales=S4[:2], idx=None), "inval"), (dict(K=2, scales=S4[:2], idx=A + 1), "align"),
    (dict(K=2, scales=None), "inval"),
    # beyond the static scratch: the row maxima's keys of 40 million
    # coordinates (several scales, 8 rows), or 8 KiB of norm partials for each
    # of 9000 rows
    (dict(d=40_000_000, ldg=40_000_000, M=8, K=4, scales=S4), "ws"),
    (dict(d=1 << 30, ldg=1 << 30, M=9000), "ws"),
])
def test_shared_scale_noalloc_rejects(kw, want):
    assert status_noalloc(**kw) == E[want]
    assert uq.uq_last_error() != ""


def test_shared_scale_noalloc_limit_is_the_header_s():
    import re

    m = re.search(r"#define UQ_NOALLOC_SCRATCH_BYTES \(\(size_t\)(\d+) << (\d+)\)", open(HEADER).read())
    assert m and int(m.group(1)) << int(m.group(2)) == uq.UQ_NOALLOC_SCRATCH_BYTES == 64 << 20
    # the same sizes with a workspace argument are accepted by the checks
    need = uq.uq_workspace_bytes(40_000_000, 8)
    assert need > uq.UQ_NOALLOC_SCRATCH_BYTES


@pytest.mark.parametrize("M", [1, 2, 8, 16, 17])
def test_shared_scale_needs_the_full_workspace(M):
    """The workspace of uq_workspace_bytes(d, M) covers any K; one 256-byte
    line less is refused before anything is launched (with 2 to 16 rows the
    size includes the 2 d bytes of the row maxima's keys of the fused pass)."""
    d = 100_003
    need = uq.uq_workspace_bytes(d, M)
    assert (need >= 2 * d) == (2 <= M <= 16)
    for K, scales, idx in ((1, S127, A), (4, S4, A)):
        assert status_shared(d=d, M=M, ldg=100_032, scales=scales, K=K, idx=idx, ws_bytes=need - 256) == E["ws"]


@pytest.mark.parametrize("kw,want", [
    (dict(s=0), "range"), (dict(s=128), "range"), (dict(g=None), "inval"), (dict(codes=None), "inval"),
    (dict(w=None), "inval"), (dict(d=-5), "inval"), (dict(rows=0), "inval"), (dict(rows=65536), "range"),
    (dict(ldg=96), "inval"), (dict(ldg=102), "align"), (dict(ldc=120), "align"), (dict(ldc=96), "inval"),
    (dict(codes=A + 8), "align"), (dict(g=A + 8), "align"), (dict(worker0=-1), "range"),
    (dict(worker0=2 ** 31 - 1, rows=2), "range"),
])
def test_quantize_single_rejects(kw, want):
    assert status_qs(**kw) == E[want]


@pytest.mark.parametrize("kw,want", [
    (dict(idx=None), "inval"), (dict(idx=A + 4), "align"), (dict(K=0), "range"),
    (dict(scales=[127.0, 100.0, 200.0, 300.0]), "range"), (dict(scales=None), "inval"),
    (dict(rows=0), "inval"), (dict(w=None), "inval"),
])
def test_quantize_multi_rejects(kw, want):
    assert status_qm(**kw) == E[want]


@pytest.mark.parametrize("kw,want", [
    (dict(codes=None), "inval"), (dict(sum_=None), "inval"), (dict(rows=0), "inval"),
    (dict(rows=(1 << 24) + 1), "range"), (dict(acc=2), "inval"), (dict(ldc=120), "align"),
    (dict(ldc=64), "inval"), (dict(sum_=A + 4), "align"), (dict(d=-1), "inval"),
])
def test_sum_codes_rejects(kw, want):
    assert status_sum(**kw) == E[want]


@pytest.mark.parametrize("kw,want", [
    (dict(sum_=None), "inval"), (dict(out=None), "inval"), (dict(w=None), "inval"), (dict(M=0), "inval"),
    (dict(idx=A), "inval"), (dict(K=4, scales=S4, idx=None), "inval"), (dict(out=A + 4), "align"),
    (dict(M=3, K=2, scales=[7.0, 11184811.0], idx=A), "range"),  # 3 * 11184811 = 2^25 + 1
    (dict(M=2 ** 24 + 1), "range"), (dict(M=20_000_000, scales=[127.0]), "range"),
    (dict(K=4, scales=S4, idx=A + 2), "align"),
])
def test_dequantize_rejects(kw, want):
    assert status_deq(**kw) == E[want]


def status_sumdeq(codes=A, d=100, rows=2, ldc=128, bits=8, acc=0, sum_=A, M=2, w=A, scales=S127, K=1, idx=None,
                  out=A):
    hs = uq._HostScales(scales)
    return L.uq_sum_dequantize(codes, d, rows, ldc, bits, acc, sum_, M, w, hs.ptr, K, idx, out, None)


@pytest.mark.parametrize("kw,want", [
    # the sum's checks
    (dict(codes=None), "inval"), (dict(sum_=None), "inval"), (dict(rows=0), "inval"),
    (dict(rows=(1 << 24) + 1), "range"), (dict(acc=2), "inval"), (dict(ldc=120), "align"),
    (dict(ldc=64), "inval"), (dict(sum_=A + 4), "align"), (dict(d=-1), "inval"),
    (dict(bits=3), "range"), (dict(bits=16), "range"), (dict(bits=4, ldc=48), "inval"),
    # the reconstruction's checks
    (dict(out=None), "inval"), (dict(w=None), "inval"), (dict(M=0), "inval"), (dict(idx=A), "inval"),
    (dict(K=4, scales=S4, idx=None), "inval"), (dict(out=A + 4), "align"),
    (dict(M=3, K=2, scales=[7.0, 11184811.0], idx=A), "range"), (dict(M=20_000_000, scales=[127.0]), "range"),
    (dict(K=4, scales=S4, idx=A + 2), "align"),
])
def test_sum_dequantize_rejects(kw, want):
    assert status_sumdeq(**kw) == E[want]


def status_qsum(g=A, d=100, rows=2, ldg=128, worker0=0, w=A, scales=S4, K=4, idx=A, seed=1, acc=0, sum_=A,
                M=2, out=A):
    hs = uq._HostScales(scales)
    return L.uq_quantize_sum(g, d, rows, ldg, worker0, w, hs.ptr, K, idx, seed, acc, sum_, M, out, None)


@pytest.mark.parametrize("kw,want", [
    # the quantiser's checks
    (dict(g=None), "inval"), (dict(w=None), "inval"), (dict(w=A + 2), "align"), (dict(d=-1), "inval"),
    (dict(rows=0), "inval"), (dict(rows=65536), "range"), (dict(ldg=96), "inval"), (dict(ldg=102), "align"),
    (dict(g=A + 8), "align"), (dict(worker0=-1), "range"), (dict(worker0=2 ** 31 - 1, rows=2), "range"),
    (dict(idx=None), "inval"), (dict(idx=A + 4), "align"), (dict(K=0), "range"), (dict(scales=None), "inval"),
    (dict(scales=[127.0, 100.0, 200.0, 300.0]), "range"), (dict(K=1, scales=[128.0]), "range"),
    # the sum's checks
    (dict(sum_=None), "inval"), (dict(sum_=A + 4), "align"), (dict(acc=2), "inval"), (dict(acc=-1), "inval"),
    # the reconstruction's checks, only when out is given
    (dict(M=0), "inval"), (dict(out=A + 4), "align"), (dict(M=20_000_000, K=1, scales=[127.0]), "range"),
    (dict(M=3, K=2, scales=[7.0, 11184811.0]), "range"),
])
def test_quantize_sum_rejects(kw, want):
    assert status_qsum(**kw) == E[want]
    assert uq.uq_last_error() != ""


def status_qsum4(g=A, d=100, rows=2, ldg=128, worker0=0, w=A, scales=S4, K=4, idx=A, seed=1, acc=0, sum_=A,
                 M=2, out=A):
    hs = uq._HostScales(scales)
    return L.uq_quantize_sum_idx4(g, d, rows, ldg, worker0, w, hs.ptr, K, idx, seed, acc, sum_, M, out, None)


@pytest.mark.parametrize("kw,want", [
    (dict(K=1, scales=S127), "inval"),
    (dict(g=None), "inval"), (dict(rows=0), "inval"), (dict(ldg=102), "align"), (dict(worker0=-1), "range"),
    (dict(idx=None), "inval"), (dict(idx=A + 4), "align"), (dict(scales=[127.0, 100.0, 200.0, 300.0]), "range"),
    (dict(sum_=None), "inval"), (dict(acc=2), "inval"), (dict(M=0), "inval"), (dict(out=A + 4), "align"),
])
def test_quantize_sum_idx4_rejects(kw, want):
    assert status_qsum4(**kw) == E[want]
    assert uq.uq_last_error() != ""


def test_quantize_sum_idx4_accepts_a_valid_no_op():
    """d = 0 with several scales passes every check and launches nothing."""
    assert status_qsum4(d=0, out=None) == uq.UQ_OK


def test_quantize_sum_reconstruction_checks_only_with_out():
    """Without an output the worker count is not read, and one scale does not
    read the index: such calls pass every check.  d = 0 makes them valid
    no-ops that launch nothing, so this holds on any host."""
    for kw in (dict(out=None, M=0), dict(out=None, M=20_000_000, K=1, scales=[127.0]),
               dict(K=1, scales=[127.0], idx=None), dict(K=1, scales=[127.0], idx=A + 1)):
        assert status_qsum(d=0, **kw) == uq.UQ_OK, kw
    assert status_qsum(d=0, M=0) == uq.UQ_EINVAL


def status_iqs(g=A, d=100, M=2, ldg=128, w=A, scales=S4, K=4, seed=1, idx=A, sum_=A, out=A):
    hs = uq._HostScales(scales)
    return L.uq_index_quantize_sum(g, d, M, ldg, w, hs.ptr, K, seed, idx, sum_, out, None)


@pytest.mark.parametrize("kw,want", [
    (dict(g=None), "inval"), (dict(w=None), "inval"), (dict(w=A + 2), "align"), (dict(d=-1), "inval"),
    (dict(M=0), "inval"), (dict(M=17), "range"), (dict(ldg=96), "inval"), (dict(ldg=102), "align"),
    (dict(g=A + 8), "align"), (dict(idx=None), "inval"), (dict(idx=A + 4), "align"), (dict(K=0), "range"),
    (dict(scales=None), "inval"), (dict(scales=[127.0, 100.0, 200.0, 300.0]), "range"),
    (dict(sum_=None), "inval"), (dict(sum_=A + 4), "align"), (dict(out=None), "inval"),
    (dict(out=A + 4), "align"), (dict(M=3, K=2, scales=[7.0, 11184811.0]), "range"),
    (dict(K=1, scales=[128.0]), "range"),
])
def test_index_quantize_sum_rejects(kw, want):
    assert status_iqs(**kw) == E[want]
    assert uq.uq_last_error() != ""


def test_index_quantize_sum_accepts_valid_no_ops():
    """d = 0 passes every check and launches nothing; one scale is valid (the
    index is then 0 everywhere)."""
    assert status_iqs(d=0) == uq.UQ_OK
    assert status_iqs(d=0, K=1, scales=[127.0]) == uq.UQ_OK
    assert status_iqs(d=0, M=16) == uq.UQ_OK


def status_iq(g=A, d=1000, M=4, ldg=1024, w=A, scales=(7.0, 112.0, 1792.0, 28672.0), K=4, seed=5, bits=4,
              idx=A, codes=A, ldc=512):
    hs = uq._HostScales(list(scales)) if scales is not None else None
    return L.uq_index_quantize(g, d, M, ldg, w, hs.ptr if hs else None, K, seed, bits, idx, codes, ldc, None)


@pytest.mark.parametrize("kw,want", [
    (dict(g=None), "inval"), (dict(w=None), "inval"), (dict(w=A + 2), "align"), (dict(d=-1), "inval"),
    (dict(M=0), "inval"), (dict(M=17), "range"), (dict(ldg=96), "inval"), (dict(ldg=1026), "align"),
    (dict(g=A + 8), "align"), (dict(idx=None), "inval"), (dict(idx=A + 4), "align"), (dict(K=0), "range"),
    (dict(scales=None), "inval"), (dict(bits=3), "range"), (dict(bits=16), "range"),
    (dict(scales=(8.0, 128.0), K=2), "range"), (dict(bits=2, scales=(3.0, 48.0), K=2), "range"),
    (dict(bits=8, scales=(128.0, 2048.0), K=2), "range"), (dict(codes=None), "inval"), (dict(codes=A + 4), "align"),
    (dict(ldc=496), "inval"), (dict(ldc=504), "align"), (dict(bits=8, ldc=992), "inval"),
])
def test_index_quantize_rejects(kw, want):
    """Argument checks of the index-forming quantiser with stored codes; d =
    1000 needs 500 bytes per row of 4-bit codes, 1000 of int8 codes."""
    assert status_iq(**kw) == E[want]
    assert uq.uq_last_error() != ""


def test_index_quantize_accepts_valid_no_ops():
    assert status_iq(d=0) == uq.UQ_OK
    assert status_iq(d=0, bits=8, scales=(127.0, 2032.0), K=2) == uq.UQ_OK
    assert status_iq(d=0, bits=2, scales=(1.0, 16.0), K=2, M=16) == uq.UQ_OK


def test_binding_raises_with_detail():
    with pytest.raises(uq.UQError) as e:
        uq.uq_quantize_single(A, 100, 2, 128, 0, A, 200, 1, A, 128, stream=0)
    assert e.value.status == uq.UQ_ERANGE and "s = 200" in str(e.value)


# GlobalRandK entry points -------------------------------------------------

def status_sel(d=1000, K=10, sel=A, ws=A, ws_bytes=1 << 20):
    return L.uq_randk_select(d, K, 7, sel, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,want", [
    (dict(d=0), "inval"), (dict(d=2 ** 32), "inval"), (dict(K=0), "range"), (dict(K=1001), "range"),
    (dict(sel=None), "inval"), (dict(sel=A + 4), "align"),
    (dict(ws=None), "inval"), (dict(ws=A + 8), "align"), (dict(ws_bytes=64), "ws"),
])
def test_randk_select_rejects(kw, want):
    assert status_sel(**kw) == E[want]


@pytest.mark.parametrize("kw,want", [
    (dict(g=None), "inval"), (dict(M=0), "inval"), (dict(K=0), "range"), (dict(K=101), "range"),
    (dict(ldg=50), "inval"), (dict(lds=10), "inval"), (dict(lds=30), "align"), (dict(sel=None), "inval"),
    (dict(sub=A + 4), "align"),
])
def test_gather_rejects(kw, want):
    args = dict(g=A, d=100, M=2, ldg=128, sel=A, K=20, sub=A, lds=32)
    args.update(kw)
    assert L.uq_gather(args["g"], args["d"], args["M"], args["ldg"], args["sel"], args["K"], args["sub"],
                       args["lds"], None) == E[want]


@pytest.mark.parametrize("kw,want", [
    (dict(vals=None), "inval"), (dict(sel=None), "inval"), (dict(out=None), "inval"), (dict(K=0), "range"),
    (dict(K=101), "range"), (dict(d=0), "inval"), (dict(out=A + 4), "align"),
])
def test_scatter_rejects(kw, want):
    args = dict(vals=A, sel=A, K=20, out=A, d=100)
    args.update(kw)
    assert L.uq_scatter(args["vals"], args["sel"], args["K"], args["out"], args["d"], None) == E[want]


def test_randk_workspace_fixed_and_aligned():
    b = uq.uq_randk_workspace_bytes(10 ** 6, 10_000)
    assert b % 256 == 0 and 32 * 1024 < b < 8 * 1024 * 1024
    assert uq.uq_randk_workspace_bytes(2 ** 32 - 1, 2 ** 31) == b


# Packed codes ---------------------------------------------------------------

def status_qp(g=A, d=100, rows=2, ldg=128, worker0=0, w=A, scales=[7.0], K=1, idx=None, bits=4, packed=A, ldp=64):
    hs = uq._HostScales(scales)
    return L.uq_quantize_packed(g, d, rows, ldg, worker0, w, hs.ptr, K, idx, 1, bits, packed, ldp, None)


@pytest.mark.parametrize("kw,want", [
    (dict(bits=8), "range"), (dict(bits=3), "range"), (dict(scales=[15.0]), "range"),
    (dict(bits=2, scales=[3.0]), "range"), (dict(ldp=48), "inval"), (dict(ldp=72), "align"),
    (dict(packed=None), "inval"), (dict(K=2, scales=[7.0, 112.0], idx=None), "inval"), (dict(rows=0), "inval"),
])
def test_quantize_packed_rejects(kw, want):
    assert status_qp(**kw) == E[want]


@pytest.mark.parametrize("kw,want", [
    (dict(bits=8), "range"), (dict(ldp=16), "inval"), (dict(ldp=56), "align"), (dict(sum_=None), "inval"),
    (dict(acc=3), "inval"), (dict(rows=0), "inval"),
])
def test_sum_packed_rejects(kw, want):
    args = dict(packed=A, d=100, rows=2, ldp=64, bits=4, acc=0, sum_=A)
    args.update(kw)
    assert L.uq_sum_packed(args["packed"], args["d"], args["rows"], args["ldp"], args["bits"], args["acc"],
                           args["sum_"], None) == E[want]


@pytest.mark.parametrize("blocks", [-1, 1, 7, (1 << 22) + 1, 1 << 40])
def test_grid_cap_rejects(blocks):
    assert L.uq_set_grid_cap(blocks) == uq.UQ_EINVAL
    assert b"grid cap" in L.uq_last_error()


def test_grid_cap_accepts_the_range_and_restores():
    for blocks in (8, 1000, 1 << 22, 0):
        assert L.uq_set_grid_cap(blocks) == uq.UQ_OK
    uq.uq_set_grid_cap(0)
    with pytest.raises(uq.UQError):
        uq.uq_set_grid_cap(3)


@pytest.mark.parametrize("mode", [-1, 5, 100])
def test_randk_mode_rejects(mode):
    assert L.uq_set_randk_mode(mode) == uq.UQ_EINVAL
    assert b"GlobalRandK mode" in L.uq_last_error()


def test_randk_mode_accepts_and_restores():
    for mode in (0, 2, 3, 4, 1):
        assert L.uq_set_randk_mode(mode) == uq.UQ_OK


def test_host_scale_arrays_are_shared_and_bounded():
    """The binding builds a scale set's host array once and reuses it; the
    cache of arrays stays bounded."""
    a = uq._host_scales([127.0, 2032.0])
    assert a is uq._host_scales((127.0, 2032.0))
    assert list(a.array) == [127.0, 2032.0]
    assert uq._host_scales([7.0]) is not a
    for k in range(400):
        uq._host_scales([float(k + 1)])
    assert len(uq._scale_arrays) <= 256
    assert uq._host_scales(None).ptr is None
