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
