"""TEST INFRASTRUCTURE ONLY: ctypes view of the C oracle (uq_oracle.c).

The oracle is the plain CPU reference for the unbiased max-norm quantisers of
arXiv 2109.12497 (Sec. 3.1-3.2, Algorithms 1-2).  Only the test suite, the
smoke check and the benchmark's CPU-baseline leg use it.  It shares no code
with the HIP library.  All arrays here are numpy arrays on the host.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(HERE, "uq_oracle.c")
# UQ_ORACLE_LIB lets the mutation test load a deliberately broken copy.
LIB_PATH = os.environ.get("UQ_ORACLE_LIB", os.path.join(HERE, "liboracle.so"))
CFLAGS = ["-O2", "-std=c99", "-ffp-contract=off", "-fno-fast-math", "-shared", "-fPIC"]

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no contraction, IEEE arithmetic)."""
    if force or not os.path.exists(LIB_PATH):
        tmp = LIB_PATH + ".tmp"
        subprocess.run(["gcc", *CFLAGS, SOURCE, "-o", tmp, "-lm"], check=True)
        os.replace(tmp, LIB_PATH)
    return LIB_PATH


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build(force=True)
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.c_void_p
        i64, i32, u32, u64, f32 = (ctypes.c_int64, ctypes.c_int32, ctypes.c_uint32,
                                   ctypes.c_uint64, ctypes.c_float)
        L.orc_philox4x32_10.argtypes = [P, P, P]
        L.orc_philox4x32_10.restype = None
        L.orc_uniform_word.argtypes = [u64, u32, u64]
        L.orc_uniform_word.restype = u32
        L.orc_sum_of_squares.argtypes = [P, i64]
        L.orc_sum_of_squares.restype = ctypes.c_double
        L.orc_max_norm.argtypes = [P, i32]
        L.orc_max_norm.restype = f32
        L.orc_shared_scale.argtypes = [P, i64, i32, i64, P]
        L.orc_shared_scale.restype = f32
        L.orc_tables.argtypes = [f32, P, i32, i32, P, P]
        L.orc_tables.restype = ctypes.c_int
        L.orc_scale_index_worker.argtypes = [P, i64, f32, P, i32, P]
        L.orc_scale_index_worker.restype = None
        L.orc_scale_index_shared.argtypes = [P, i64, i32, i64, f32, P, i32, P, P]
        L.orc_scale_index_shared.restype = None
        L.orc_quantize.argtypes = [P, i64, i64, u32, f32, P, i32, P, u64, P]
        L.orc_quantize.restype = None
        L.orc_sum_codes.argtypes = [P, i64, i32, i64, P]
        L.orc_sum_codes.restype = None
        L.orc_dequantize.argtypes = [P, i64, i32, f32, P, i32, P, P]
        L.orc_dequantize.restype = None
        L.orc_pack_codes.argtypes = [P, i64, i32, P]
        L.orc_pack_codes.restype = None
        L.orc_unpack_codes.argtypes = [P, i64, i32, P]
        L.orc_unpack_codes.restype = None
        L.orc_sum_packed.argtypes = [P, i64, i32, i64, i32, P]
        L.orc_sum_packed.restype = None
        L.orc_randk_keys.argtypes = [u64, i64, i64, P, P]
        L.orc_randk_keys.restype = None
        L.orc_randk_select.argtypes = [i64, i64, u64, P, P]
        L.orc_randk_select.restype = None
        _lib = L
    return _lib


def _ptr(a: np.ndarray | None):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"] or a.ndim == 1, "oracle arrays must be contiguous"
    return a.ctypes.data


def _scales(scales) -> np.ndarray:
    s = np.ascontiguousarray(np.asarray(scales, dtype=np.float32).reshape(-1))
    assert 1 <= s.size <= 16
    return s


def philox(ctr, key) -> np.ndarray:
    c = np.ascontiguousarray(np.asarray(ctr, dtype=np.uint32))
    k = np.ascontiguousarray(np.asarray(key, dtype=np.uint32))
    out = np.zeros(4, dtype=np.uint32)
    lib().orc_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def uniform_word(seed: int, worker: int, i: int) -> int:
    return int(lib().orc_uniform_word(seed, worker, i))


def sum_of_squares(v: np.ndarray) -> float:
    v = np.ascontiguousarray(v, dtype=np.float32)
    return float(lib().orc_sum_of_squares(_ptr(v), v.size))


def shared_scale(g: np.ndarray, d: int | None = None):
    """g: [M, ldg] float32.  Returns (W as np.float32, per-row sums of squares)."""
    g = np.ascontiguousarray(g, dtype=np.float32)
    M, ldg = g.shape
    d = ldg if d is None else d
    S = np.zeros(M, dtype=np.float64)
    W = lib().orc_shared_scale(_ptr(g), d, M, ldg, _ptr(S))
    return np.float32(W), S


def tables(W, scales, M: int = 1):
    s = _scales(scales)
    inv = np.zeros(s.size, dtype=np.float32)
    deq = np.zeros(s.size, dtype=np.float32)
    zero = lib().orc_tables(np.float32(W), _ptr(s), s.size, M, _ptr(inv), _ptr(deq))
    return bool(zero), inv, deq


def scale_index_worker(v: np.ndarray, W, scales) -> np.ndarray:
    v = np.ascontiguousarray(v, dtype=np.float32)
    s = _scales(scales)
    out = np.zeros(v.size, dtype=np.uint8)
    lib().orc_scale_index_worker(_ptr(v), v.size, np.float32(W), _ptr(s), s.size, _ptr(out))
    return out


def scale_index_shared(g: np.ndarray, W, scales, d: int | None = None) -> np.ndarray:
    g = np.ascontiguousarray(g, dtype=np.float32)
    M, ldg = g.shape
    d = ldg if d is None else d
    s = _scales(scales)
    idx = np.zeros(d, dtype=np.uint8)
    scratch = np.zeros(d, dtype=np.uint8)
    lib().orc_scale_index_shared(_ptr(g), d, M, ldg, np.float32(W), _ptr(s), s.size,
                                 _ptr(idx), _ptr(scratch))
    return idx


def quantize(v: np.ndarray, W, scales, seed: int, worker: int = 0, i0: int = 0,
             idx: np.ndarray | None = None) -> np.ndarray:
    """Codes of worker `worker` for coordinates i0 .. i0+len(v)-1."""
    v = np.ascontiguousarray(v, dtype=np.float32).reshape(-1)
    s = _scales(scales)
    if idx is not None:
        idx = np.ascontiguousarray(idx, dtype=np.uint8).reshape(-1)
        assert idx.size == v.size
    out = np.zeros(v.size, dtype=np.int8)
    lib().orc_quantize(_ptr(v), v.size, i0, worker, np.float32(W), _ptr(s), s.size,
                       _ptr(idx), seed, _ptr(out))
    return out


def sum_codes(codes: np.ndarray, d: int | None = None) -> np.ndarray:
    codes = np.ascontiguousarray(codes, dtype=np.int8)
    if codes.ndim == 1:
        codes = codes.reshape(1, -1)
    rows, ldc = codes.shape
    d = ldc if d is None else d
    out = np.zeros(d, dtype=np.int32)
    lib().orc_sum_codes(_ptr(codes), d, rows, ldc, _ptr(out))
    return out


def dequantize(sums: np.ndarray, M: int, W, scales, idx: np.ndarray | None = None) -> np.ndarray:
    sums = np.ascontiguousarray(sums, dtype=np.int32).reshape(-1)
    s = _scales(scales)
    if idx is not None:
        idx = np.ascontiguousarray(idx, dtype=np.uint8).reshape(-1)
    out = np.zeros(sums.size, dtype=np.float32)
    lib().orc_dequantize(_ptr(sums), sums.size, M, np.float32(W), _ptr(s), s.size,
                         _ptr(idx), _ptr(out))
    return out


def pipeline(g: np.ndarray, scales, seed: int, d: int | None = None, W=None,
             worker0: int = 0) -> dict:
    """Algorithm 1 (one scale) or Algorithm 2 (several scales), all M workers.

    g: [M, ldg] float32.  If W is given it replaces the oracle's own shared
    scale for every later step (used to check the device's later stages on
    the device's own scale).  Returns W, idx (None for one scale), codes
    [M, d] int8, sum [d] int32 and out [d] float32.
    """
    g = np.ascontiguousarray(g, dtype=np.float32)
    M, ldg = g.shape
    d = ldg if d is None else d
    s = _scales(scales)
    W_own, S = shared_scale(g, d)
    W = W_own if W is None else np.float32(W)
    idx = scale_index_shared(g, W, s, d) if s.size > 1 else None
    codes = np.zeros((M, d), dtype=np.int8)
    for m in range(M):
        codes[m] = quantize(g[m, :d], W, s, seed, worker=worker0 + m, i0=0, idx=idx)
    sums = sum_codes(codes, d)
    out = dequantize(sums, M, W, s, idx)
    return {"W": W, "W_oracle": W_own, "sumsq": S, "idx": idx, "codes": codes,
            "sum": sums, "out": out}


# ---------------------------------------------------------------------------
# The same steps on several host threads.  Every per-coordinate step is a pure
# function of its coordinate, and each row's norm is still one sequential
# index-order sum, so splitting the rows and fixed coordinate chunks over
# threads changes no byte of any result; the C calls release the GIL.
# ---------------------------------------------------------------------------

def default_threads() -> int:
    """Host threads for the parallel driver: the cores this process may use,
    at most 16."""
    return max(1, min(16, len(os.sched_getaffinity(0))))


def _run_jobs(jobs, threads: int) -> None:
    if threads <= 1 or len(jobs) <= 1:
        for job in jobs:
            job()
        return
    from concurrent.futures import ThreadPoolExecutor

    with ThreadPoolExecutor(max_workers=threads) as ex:
        for f in [ex.submit(job) for job in jobs]:
            f.result()


def _chunks(n: int, chunk: int):
    return [(c, min(n, c + chunk)) for c in range(0, n, chunk)]


def shared_scale_threaded(g: np.ndarray, d: int | None = None, threads: int = 1):
    """shared_scale with the rows on `threads` threads (each row's sum of
    squares sequential in index order, as there)."""
    g = np.ascontiguousarray(g, dtype=np.float32)
    M, ldg = g.shape
    d = ldg if d is None else d
    L = lib()
    S = np.zeros(M, dtype=np.float64)
    base = g.ctypes.data

    def norm(m):
        S[m] = L.orc_sum_of_squares(base + 4 * m * ldg, d)

    _run_jobs([lambda m=m: norm(m) for m in range(M)], threads)
    return np.float32(L.orc_max_norm(_ptr(S), M)), S


def window(g: np.ndarray, W, scales, seed: int, i0: int = 0, n: int | None = None, worker0: int = 0,
           threads: int = 1, chunk: int = 1 << 20) -> dict:
    """The steps after the shared scale for coordinates i0 .. i0+n-1, given W:
    g [M, >= n] holds those coordinates of every worker.  Returns idx (None
    for one scale), codes [M, n], sum [n] and out [n], as pipeline does."""
    g = np.ascontiguousarray(g, dtype=np.float32)
    M, ldg = g.shape
    n = ldg if n is None else n
    s = _scales(scales)
    K = s.size
    W = np.float32(W)
    L = lib()
    gp, sp = g.ctypes.data, _ptr(s)
    parts = _chunks(n, chunk)
    idx = np.zeros(n, dtype=np.uint8) if K > 1 else None
    if idx is not None:
        ip = idx.ctypes.data

        def index(c0, c1):
            scratch = np.zeros(c1 - c0, dtype=np.uint8)
            L.orc_scale_index_shared(gp + 4 * c0, c1 - c0, M, ldg, W, sp, K, ip + c0, _ptr(scratch))

        _run_jobs([lambda a=a, b=b: index(a, b) for a, b in parts], threads)
    codes = np.zeros((M, n), dtype=np.int8)
    cp = codes.ctypes.data

    def quant(m, c0, c1):
        L.orc_quantize(gp + 4 * (m * ldg + c0), c1 - c0, i0 + c0, worker0 + m, W, sp, K,
                       None if idx is None else ip + c0, seed, cp + m * n + c0)

    _run_jobs([lambda m=m, a=a, b=b: quant(m, a, b) for m in range(M) for a, b in parts], threads)
    sums = np.zeros(n, dtype=np.int32)
    out = np.zeros(n, dtype=np.float32)
    up, op = sums.ctypes.data, out.ctypes.data

    def add_and_reconstruct(c0, c1):
        L.orc_sum_codes(cp + c0, c1 - c0, M, n, up + 4 * c0)
        L.orc_dequantize(up + 4 * c0, c1 - c0, M, W, sp, K, None if idx is None else ip + c0, op + 4 * c0)

    _run_jobs([lambda a=a, b=b: add_and_reconstruct(a, b) for a, b in parts], threads)
    return {"idx": idx, "codes": codes, "sum": sums, "out": out}


def pipeline_threaded(g: np.ndarray, scales, seed: int, d: int | None = None, W=None, worker0: int = 0,
                      threads: int | None = None, chunk: int = 1 << 20) -> dict:
    """pipeline() with the rows (norm) and fixed coordinate chunks (every
    later step) spread over `threads` host threads; byte for byte the same
    result for any thread count."""
    g = np.ascontiguousarray(g, dtype=np.float32)
    M, ldg = g.shape
    d = ldg if d is None else d
    threads = default_threads() if threads is None else threads
    W_own, S = shared_scale_threaded(g, d, threads)
    W = W_own if W is None else np.float32(W)
    r = window(g, W, scales, seed, i0=0, n=d, worker0=worker0, threads=threads, chunk=chunk)
    r.update(W=W, W_oracle=W_own, sumsq=S)
    return r


# ---------------------------------------------------------------------------
# Sub-byte codes
# ---------------------------------------------------------------------------

def pack_codes(codes: np.ndarray, bits: int) -> np.ndarray:
    codes = np.ascontiguousarray(codes, dtype=np.int8).reshape(-1)
    per = 8 // bits
    out = np.zeros((codes.size + per - 1) // per, dtype=np.uint8)
    lib().orc_pack_codes(_ptr(codes), codes.size, bits, _ptr(out))
    return out


def unpack_codes(packed: np.ndarray, n: int, bits: int) -> np.ndarray:
    packed = np.ascontiguousarray(packed, dtype=np.uint8).reshape(-1)
    out = np.zeros(n, dtype=np.int8)
    lib().orc_unpack_codes(_ptr(packed), n, bits, _ptr(out))
    return out


def sum_packed(packed: np.ndarray, n: int, bits: int) -> np.ndarray:
    """packed: [rows, ldp] uint8; the int32 sum of the rows' first n codes."""
    packed = np.ascontiguousarray(packed, dtype=np.uint8)
    if packed.ndim == 1:
        packed = packed.reshape(1, -1)
    rows, ldp = packed.shape
    out = np.zeros(n, dtype=np.int32)
    lib().orc_sum_packed(_ptr(packed), n, rows, ldp, bits, _ptr(out))
    return out


# ---------------------------------------------------------------------------
# GlobalRandK (Sec. 3.3-3.4)
# ---------------------------------------------------------------------------

def randk_keys(seed: int, i0: int, n: int):
    """(hi, lo) 32-bit selection keys of coordinates i0 .. i0+n-1."""
    hi = np.zeros(n, dtype=np.uint32)
    lo = np.zeros(n, dtype=np.uint32)
    lib().orc_randk_keys(seed, i0, n, _ptr(hi), _ptr(lo))
    return hi, lo


def randk_select(d: int, K: int, seed: int) -> np.ndarray:
    """The K coordinates with the smallest (key, index), ascending (uint32)."""
    assert 0 < K <= d < 2 ** 32
    out = np.zeros(K, dtype=np.uint32)
    scratch = np.zeros(d * 12, dtype=np.uint8)
    lib().orc_randk_select(d, K, seed, _ptr(out), _ptr(scratch))
    return out


def randk_pipeline(g: np.ndarray, K: int, scales, seed: int, d: int | None = None, W=None,
                   worker0: int = 0) -> dict:
    """GlobalRandK step: select K coordinates, run Algorithm 1/2 on the
    gathered [M, K] sub-vectors, write the reconstruction back (0 elsewhere)."""
    g = np.ascontiguousarray(g, dtype=np.float32)
    M, ldg = g.shape
    d = ldg if d is None else d
    sel = randk_select(d, K, seed)
    sub = np.ascontiguousarray(g[:, sel.astype(np.int64)])
    r = pipeline(sub, scales, seed, d=K, W=W, worker0=worker0)
    full = np.zeros(d, dtype=np.float32)
    full[sel.astype(np.int64)] = r["out"]
    r.update(sel=sel, sub=sub, full=full)
    return r
