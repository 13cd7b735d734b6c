"""The bandwidth-probe kernels (libuq_probe.so) compute what they claim, so
that the achievable-bandwidth figures rest on kernels that touch every byte."""
import ctypes
import os

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2109_12497_amd as uq  # noqa: E402


def probe_lib():
    lib = ctypes.CDLL(os.path.join(os.path.dirname(uq.LIB_PATH), "libuq_probe.so"))
    P, i64 = ctypes.c_void_p, ctypes.c_int64
    lib.uqp_read.argtypes = [P, i64, P, P]
    lib.uqp_read_write8.argtypes = [P, i64, P, P]
    lib.uqp_read_out_floats.argtypes = [i64]
    lib.uqp_read_out_floats.restype = i64
    lib.uqp_rows_read.argtypes = [P, i64, ctypes.c_int32, i64, P, P]
    lib.uqp_rows_out_floats.argtypes = [i64, ctypes.c_int32]
    lib.uqp_rows_out_floats.restype = i64
    lib.uqp_accumulate.argtypes = [P, P, P, i64, P]
    lib.uqp_copy.argtypes = [P, P, i64, P]
    lib.uqp_keys_index.argtypes = [P, i64, P, ctypes.c_int32, P]
    return lib


@pytest.mark.parametrize("n", [512, 512 * 1000, 512 * (1 << 14) + 512])
def test_probe_kernels(n):
    lib = probe_lib()
    g = torch.randn(n, device="cuda")
    codes = torch.zeros(n, dtype=torch.uint8, device="cuda")
    out = torch.zeros(int(lib.uqp_read_out_floats(n)), device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    assert lib.uqp_read_write8(g.data_ptr(), n, codes.data_ptr(), s) == 0
    assert lib.uqp_read(g.data_ptr(), n, out.data_ptr(), s) == 0
    torch.cuda.synchronize()
    top = (g.cpu().numpy().view(np.uint32) >> 24).astype(np.uint8)
    assert np.array_equal(codes.cpu().numpy(), top)
    # the read kernel's per-thread sums add up to the sum of all elements
    assert abs(float(out.double().sum()) - float(g.double().sum())) <= 1e-3 * max(1.0, float(g.abs().sum()))


@pytest.mark.parametrize("d,M", [(512, 1), (512 * 300, 3), (65536 * 2 + 1024, 4)])
def test_row_accumulate_and_copy_probes(d, M):
    lib = probe_lib()
    s = torch.cuda.current_stream().cuda_stream
    ldg = d + 64
    g = torch.randn((M, ldg), device="cuda") * 100
    out = torch.zeros(int(lib.uqp_rows_out_floats(d, M)), device="cuda")
    assert lib.uqp_rows_read(g.data_ptr(), d, M, ldg, out.data_ptr(), s) == 0
    idx = torch.randint(0, 256, (d,), dtype=torch.uint8, device="cuda")
    acc = torch.randint(-1000, 1000, (d,), dtype=torch.int32, device="cuda")
    before = acc.clone()
    assert lib.uqp_accumulate(g.data_ptr(), idx.data_ptr(), acc.data_ptr(), d, s) == 0
    dst = torch.zeros(d, device="cuda")
    assert lib.uqp_copy(g.data_ptr(), dst.data_ptr(), d, s) == 0
    torch.cuda.synchronize()
    rows = g[:, :d].double().sum(dim=1)
    got = out.double().reshape(M, -1).sum(dim=1)
    assert torch.allclose(got, rows, rtol=1e-4, atol=1e-2 * d ** 0.5)
    want = before + idx.to(torch.int32) + g[0, :d].to(torch.int32)  # truncation toward zero, as the probe
    assert torch.equal(acc, want)
    assert torch.equal(dst, g[0, :d])
    # out-of-range arguments are refused before any launch
    assert lib.uqp_rows_read(g.data_ptr(), d, M, d - 4, out.data_ptr(), s) == -1
    assert lib.uqp_accumulate(g.data_ptr(), idx.data_ptr(), acc.data_ptr(), d + 1, s) == -1


@pytest.mark.parametrize("octs", [2, 4, 8])
@pytest.mark.parametrize("d", [512, 512 * 77, 512 * 5000 + 512])
def test_keys_index_probe(d, octs):
    """Every key read and its low byte written, whatever the octets per thread
    (tiles past d partly filled)."""
    lib = probe_lib()
    s = torch.cuda.current_stream().cuda_stream
    keys = torch.randint(0, 1 << 16, (d,), dtype=torch.int32, device="cuda").to(torch.int16)
    idx = torch.zeros(d + 64, dtype=torch.uint8, device="cuda")
    assert lib.uqp_keys_index(keys.data_ptr(), d, idx.data_ptr(), octs, s) == 0
    torch.cuda.synchronize()
    want = (keys.cpu().numpy().view(np.uint16) & 0xFF).astype(np.uint8)
    got = idx.cpu().numpy()
    assert np.array_equal(got[:d], want)
    assert not got[d:].any()
    assert lib.uqp_keys_index(keys.data_ptr(), d, idx.data_ptr(), 3, s) == -1
