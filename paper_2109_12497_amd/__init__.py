"""Python binding of libuq, the MI355X quantiser library (arXiv 2109.12497).

Argument marshalling only: every entry point has the name, argument order and
meaning of its C declaration in include/uq.h.  Device arrays may be passed as
torch tensors on the GPU (their data pointers are used) or as raw integer
addresses; `scales` is a Python sequence (a host array); `stream` defaults to
torch's current stream.  A nonzero status raises UQError.

Importing this package loads the compiled library and fails loudly if it is
not built: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libuq.so")

UQ_OK, UQ_EINVAL, UQ_ERANGE, UQ_EALIGN, UQ_EWORKSPACE, UQ_EHIP = 0, -1, -2, -3, -4, -5
UQ_MAX_SCALES = 16
UQ_NOALLOC_SCRATCH_BYTES = 64 << 20


class UQError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"libuq status {status}: {message}")
        self.status = status


def _hip_runtimes_mapped() -> set:
    try:
        with open("/proc/self/maps") as f:
            return {line.split()[-1] for line in f if "libamdhip64.so" in line}
    except OSError:
        return set()


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() (hipcc for gfx950)")
    # One HIP runtime per process: torch ships its own libamdhip64 (same
    # soname as the system one).  Loading torch first makes the dynamic
    # linker bind libuq to that already-loaded runtime, so the tensors and
    # streams torch hands over and the kernels libuq launches share a device
    # context.
    import torch  # noqa: F401

    L = ctypes.CDLL(LIB_PATH)
    runtimes = _hip_runtimes_mapped()
    if len(runtimes) > 1:
        raise ImportError(f"two HIP runtimes are mapped in this process: {sorted(runtimes)}")
    P, i32, i64, u64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_size_t
    L.uq_shared_scale.argtypes = [P, i64, i32, i64, P, i32, P, P, P, sz, P]
    L.uq_shared_scale_idx4.argtypes = [P, i64, i32, i64, P, i32, P, P, P, sz, P]
    L.uq_shared_scale_noalloc.argtypes = [P, i64, i32, i64, P, i32, P, P, P]
    L.uq_workspace_bytes.argtypes = [i64, i32]
    L.uq_workspace_bytes.restype = sz
    L.uq_quantize_single.argtypes = [P, i64, i32, i64, i32, P, i32, u64, P, i64, P]
    L.uq_quantize_multi.argtypes = [P, i64, i32, i64, i32, P, P, i32, P, u64, P, i64, P]
    L.uq_sum_codes.argtypes = [P, i64, i32, i64, i32, P, P]
    L.uq_dequantize.argtypes = [P, i64, i32, P, P, i32, P, P, P]
    L.uq_sum_dequantize.argtypes = [P, i64, i32, i64, i32, i32, P, i32, P, P, i32, P, P, P]
    L.uq_quantize_packed.argtypes = [P, i64, i32, i64, i32, P, P, i32, P, u64, i32, P, i64, P]
    L.uq_quantize_sum.argtypes = [P, i64, i32, i64, i32, P, P, i32, P, u64, i32, P, i32, P, P]
    L.uq_quantize_sum_idx4.argtypes = [P, i64, i32, i64, i32, P, P, i32, P, u64, i32, P, i32, P, P]
    L.uq_index_quantize_sum.argtypes = [P, i64, i32, i64, P, P, i32, u64, P, P, P, P]
    L.uq_index_quantize.argtypes = [P, i64, i32, i64, P, P, i32, u64, i32, P, P, i64, P]
    L.uq_sum_packed.argtypes = [P, i64, i32, i64, i32, i32, P, P]
    L.uq_randk_workspace_bytes.argtypes = [i64, i64]
    L.uq_randk_workspace_bytes.restype = sz
    L.uq_randk_select.argtypes = [i64, i64, u64, P, P, sz, P]
    L.uq_gather.argtypes = [P, i64, i32, i64, P, i64, P, i64, P]
    L.uq_scatter.argtypes = [P, P, i64, P, i64, P]
    L.uq_set_grid_cap.argtypes = [i64]
    L.uq_set_randk_mode.argtypes = [i32]
    L.uq_strerror.argtypes = [ctypes.c_int]
    L.uq_strerror.restype = ctypes.c_char_p
    L.uq_last_error.argtypes = []
    L.uq_last_error.restype = ctypes.c_char_p
    for name in ("uq_shared_scale", "uq_shared_scale_idx4", "uq_shared_scale_noalloc", "uq_quantize_single",
                 "uq_quantize_multi", "uq_sum_codes", "uq_dequantize", "uq_sum_dequantize", "uq_quantize_packed",
                 "uq_sum_packed", "uq_quantize_sum", "uq_quantize_sum_idx4",
                 "uq_index_quantize_sum", "uq_index_quantize",
                 "uq_randk_select", "uq_gather",
                 "uq_scatter", "uq_set_grid_cap", "uq_set_randk_mode"):
        getattr(L, name).restype = ctypes.c_int
    return L


lib = _load()


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream):
    if stream is None:
        import torch

        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


class _HostScales:
    """Keeps a ctypes float array alive for the duration of a call."""

    def __init__(self, scales):
        if scales is None:
            self.array = None
            self.ptr = None
        else:
            vals = [float(s) for s in scales]
            self.array = (ctypes.c_float * max(1, len(vals)))(*vals)
            self.ptr = ctypes.cast(self.array, ctypes.c_void_p)


_scale_arrays: dict = {}


def _host_scales(scales) -> _HostScales:
    """The ctypes array of a scale set, built once per distinct set (the
    arrays are read-only to the library, so they can be shared)."""
    if scales is None:
        return _HostScales(None)
    key = tuple(scales)
    hs = _scale_arrays.get(key)
    if hs is None:
        if len(_scale_arrays) >= 256:
            _scale_arrays.clear()
        hs = _scale_arrays[key] = _HostScales(key)
    return hs


def _check(status: int) -> None:
    if status != UQ_OK:
        raise UQError(status, f"{lib.uq_strerror(status).decode()}: {lib.uq_last_error().decode()}")


def uq_set_grid_cap(blocks: int) -> None:
    """Test hook: cap the streaming passes' grids at `blocks` blocks (0: the default)."""
    _check(lib.uq_set_grid_cap(blocks))


def uq_set_randk_mode(mode: int) -> None:
    """Test hook: 1 bracket (default), 0 histogram passes, 2 bracket forced to miss."""
    _check(lib.uq_set_randk_mode(mode))


def uq_workspace_bytes(d: int, M: int) -> int:
    return int(lib.uq_workspace_bytes(d, M))


def uq_shared_scale(g, d, M, ldg, scales, K, w, idx, ws, ws_bytes, stream=None) -> None:
    hs = _host_scales(scales)
    _check(lib.uq_shared_scale(_ptr(g), d, M, ldg, hs.ptr, K, _ptr(w), _ptr(idx), _ptr(ws), ws_bytes,
                               _stream(stream)))


def uq_shared_scale_idx4(g, d, M, ldg, scales, K, w, idx4, ws, ws_bytes, stream=None) -> None:
    hs = _host_scales(scales)
    _check(lib.uq_shared_scale_idx4(_ptr(g), d, M, ldg, hs.ptr, K, _ptr(w), _ptr(idx4), _ptr(ws), ws_bytes,
                                    _stream(stream)))


def uq_shared_scale_noalloc(g, d, M, ldg, scales, K, w, idx, stream=None) -> None:
    hs = _host_scales(scales)
    _check(lib.uq_shared_scale_noalloc(_ptr(g), d, M, ldg, hs.ptr, K, _ptr(w), _ptr(idx), _stream(stream)))


def uq_quantize_single(g, d, rows, ldg, worker0, w, s, seed, codes, ldc, stream=None) -> None:
    _check(lib.uq_quantize_single(_ptr(g), d, rows, ldg, worker0, _ptr(w), s, seed, _ptr(codes), ldc,
                                  _stream(stream)))


def uq_quantize_multi(g, d, rows, ldg, worker0, w, scales, K, idx, seed, codes, ldc, stream=None) -> None:
    hs = _host_scales(scales)
    _check(lib.uq_quantize_multi(_ptr(g), d, rows, ldg, worker0, _ptr(w), hs.ptr, K, _ptr(idx), seed,
                                 _ptr(codes), ldc, _stream(stream)))


def uq_sum_codes(codes, d, rows, ldc, accumulate, sum, stream=None) -> None:
    _check(lib.uq_sum_codes(_ptr(codes), d, rows, ldc, accumulate, _ptr(sum), _stream(stream)))


def uq_dequantize(sum, d, M, w, scales, K, idx, out, stream=None) -> None:
    hs = _host_scales(scales)
    _check(lib.uq_dequantize(_ptr(sum), d, M, _ptr(w), hs.ptr, K, _ptr(idx), _ptr(out), _stream(stream)))


def uq_sum_dequantize(codes, d, rows, ldc, bits, accumulate, sum, M, w, scales, K, idx, out, stream=None) -> None:
    hs = _host_scales(scales)
    _check(lib.uq_sum_dequantize(_ptr(codes), d, rows, ldc, bits, accumulate, _ptr(sum), M, _ptr(w), hs.ptr, K,
                                 _ptr(idx), _ptr(out), _stream(stream)))


def uq_quantize_packed(g, d, rows, ldg, worker0, w, scales, K, idx, seed, bits, packed, ldp, stream=None) -> None:
    hs = _host_scales(scales)
    _check(lib.uq_quantize_packed(_ptr(g), d, rows, ldg, worker0, _ptr(w), hs.ptr, K, _ptr(idx), seed, bits,
                                  _ptr(packed), ldp, _stream(stream)))


def uq_quantize_sum(g, d, rows, ldg, worker0, w, scales, K, idx, seed, accumulate, sum, M, out,
                    stream=None) -> None:
    hs = _host_scales(scales)
    _check(lib.uq_quantize_sum(_ptr(g), d, rows, ldg, worker0, _ptr(w), hs.ptr, K, _ptr(idx), seed, accumulate,
                               _ptr(sum), M, _ptr(out), _stream(stream)))


def uq_quantize_sum_idx4(g, d, rows, ldg, worker0, w, scales, K, idx4, seed, accumulate, sum, M, out,
                         stream=None) -> None:
    hs = _host_scales(scales)
    _check(lib.uq_quantize_sum_idx4(_ptr(g), d, rows, ldg, worker0, _ptr(w), hs.ptr, K, _ptr(idx4), seed,
                                    accumulate, _ptr(sum), M, _ptr(out), _stream(stream)))


def uq_index_quantize_sum(g, d, M, ldg, w, scales, K, seed, idx, sum, out, stream=None) -> None:
    hs = _host_scales(scales)
    _check(lib.uq_index_quantize_sum(_ptr(g), d, M, ldg, _ptr(w), hs.ptr, K, seed, _ptr(idx), _ptr(sum), _ptr(out),
                                     _stream(stream)))


def uq_index_quantize(g, d, M, ldg, w, scales, K, seed, bits, idx, codes, ldc, stream=None) -> None:
    hs = _host_scales(scales)
    _check(lib.uq_index_quantize(_ptr(g), d, M, ldg, _ptr(w), hs.ptr, K, seed, bits, _ptr(idx), _ptr(codes), ldc,
                                 _stream(stream)))


def uq_sum_packed(packed, d, rows, ldp, bits, accumulate, sum, stream=None) -> None:
    _check(lib.uq_sum_packed(_ptr(packed), d, rows, ldp, bits, accumulate, _ptr(sum), _stream(stream)))


def uq_randk_workspace_bytes(d: int, K: int) -> int:
    return int(lib.uq_randk_workspace_bytes(d, K))


def uq_randk_select(d, K, seed, sel, ws, ws_bytes, stream=None) -> None:
    _check(lib.uq_randk_select(d, K, seed, _ptr(sel), _ptr(ws), ws_bytes, _stream(stream)))


def uq_gather(g, d, M, ldg, sel, K, sub, lds, stream=None) -> None:
    _check(lib.uq_gather(_ptr(g), d, M, ldg, _ptr(sel), K, _ptr(sub), lds, _stream(stream)))


def uq_scatter(vals, sel, K, out, d, stream=None) -> None:
    _check(lib.uq_scatter(_ptr(vals), _ptr(sel), K, _ptr(out), d, _stream(stream)))


def uq_strerror(status: int) -> str:
    return lib.uq_strerror(status).decode()


def uq_last_error() -> str:
    return lib.uq_last_error().decode()
