"""One aggregation step of Algorithm 1 / Algorithm 2 through the C ABI.

`Step` owns the device buffers of a fixed problem shape and issues the
library calls in the order of the algorithms (Sec. 3.1-3.2):
shared scale (+ shared index) -> quantise -> integer sum -> reconstruct,
the last two as one call (uq_sum_dequantize) unless fused=False.
No arithmetic of the method happens here.
"""
from __future__ import annotations

import numpy as np
import torch

from . import (_stream, uq_dequantize, uq_gather, uq_index_quantize, uq_index_quantize_sum, uq_quantize_multi, uq_quantize_packed,
               uq_quantize_single, uq_quantize_sum, uq_quantize_sum_idx4, uq_randk_select, uq_randk_workspace_bytes,
               uq_scatter, uq_shared_scale, uq_shared_scale_idx4, uq_sum_codes, uq_sum_dequantize, uq_sum_packed,
               uq_workspace_bytes)


def round_up(x: int, m: int) -> int:
    return (x + m - 1) // m * m


class Step:
    """Buffers and call sequence for M workers' gradients g [M, ldg] fp32.

    streamed=False: every worker's codes are materialised ([M, ldc] int8) and
    summed by one call.  streamed=True: one code row is reused; each worker is
    quantised and accumulated into the int32 sum in turn.
    bits = 4 or 2: the codes are held packed ([M, ldc] bytes, ldc >= d*bits/8).
    fused=True: the last sum call also reconstructs (uq_sum_dequantize);
    False: uq_sum_codes / uq_sum_packed, then uq_dequantize.
    quant_sum=True: the codes are added into the sum as they are formed
    (uq_quantize_sum) and never stored: one call per worker when streamed
    (the last one also reconstructs), one call for all workers otherwise.
    The default is True for a streamed step with fused=True, else False.
    index_in_pass=True (resident rows, several scales, M <= 16): the shared
    index is formed inside the call that quantises every row, from the rows
    it holds (uq_index_quantize_sum with quant_sum, else uq_index_quantize,
    which stores the codes), so the shared-scale call forms W only.  The
    default is True when those conditions hold with quant_sum or with packed
    codes; int8 codes stored keep the separate index pass unless asked.
    index_bits=4 (several scales, quant_sum, index not formed in the pass):
    the shared index is held as 4-bit fields, two coordinates a byte
    (uq_shared_scale_idx4, uq_quantize_sum_idx4), so each call that reads it
    reads half the bytes; index_host() gives its values either way.
    """

    def __init__(self, d: int, M: int, scales, device="cuda", streamed: bool = False, ldc: int | None = None,
                 bits: int = 8, fused: bool = True, quant_sum: bool | None = None,
                 index_in_pass: bool | None = None, index_bits: int = 8):
        self.d, self.M = d, M
        self.fused = fused
        self.quant_sum = (streamed and fused) if quant_sum is None else quant_sum
        assert not (self.quant_sum and not fused), "quant_sum reconstructs in the same pass (fused)"
        self.scales = [float(s) for s in scales]
        self.K = len(self.scales)
        can = not streamed and self.K > 1 and 1 <= M <= 16
        default = can and (self.quant_sum or bits != 8)
        self.index_in_pass = default if index_in_pass is None else index_in_pass
        assert not (self.index_in_pass and not can), "index_in_pass needs resident rows, K > 1, M <= 16"
        self.streamed = streamed
        self.bits = bits
        assert index_bits in (8, 4), "index_bits is 8 or 4"
        assert index_bits == 8 or (self.quant_sum and self.K > 1 and not self.index_in_pass), \
            "the 4-bit index serves the quantise-and-sum with several scales and a separate index pass"
        self.index_bits = index_bits
        row_bytes = (max(d, 1) * bits + 7) // 8
        self.ldc = round_up(row_bytes, 256) if ldc is None else ldc
        self.device = torch.device(device)
        if self.device.type == "cuda" and self.device.index is None:
            self.device = torch.device("cuda", torch.cuda.current_device())
        self.w = torch.zeros(4, dtype=torch.float32, device=device)  # W lives in w[0]
        idx_bytes = max(d, 1) if index_bits == 8 else (max(d, 1) + 1) // 2
        self.idx = torch.zeros(round_up(idx_bytes, 256), dtype=torch.uint8, device=device) if self.K > 1 else None
        self.ws_bytes = uq_workspace_bytes(d, M)
        self.ws = torch.zeros(self.ws_bytes // 8, dtype=torch.float64, device=device)
        rows = 1 if streamed else M
        # the fused quantise-and-sum stores no codes
        self.codes = None if self.quant_sum else torch.zeros((rows, self.ldc), dtype=torch.int8, device=device)
        self.sum = torch.zeros(round_up(max(d, 1), 64), dtype=torch.int32, device=device)
        self.out = torch.zeros(round_up(max(d, 1), 64), dtype=torch.float32, device=device)

    # -- the four stages -------------------------------------------------------
    def shared_scale(self, g, stream=None, w_only: bool = False):
        if w_only:
            # W does not depend on the scales: the one-scale call forms it alone
            uq_shared_scale(g, self.d, self.M, g.stride(0), self.scales[:1], 1, self.w, None, self.ws,
                            self.ws_bytes, stream)
        elif self.index_bits == 4:
            uq_shared_scale_idx4(g, self.d, self.M, g.stride(0), self.scales, self.K, self.w, self.idx, self.ws,
                                 self.ws_bytes, stream)
        else:
            uq_shared_scale(g, self.d, self.M, g.stride(0), self.scales, self.K, self.w, self.idx, self.ws,
                            self.ws_bytes, stream)

    def quantize(self, g, seed: int, rows: int | None = None, worker0: int = 0, codes=None, stream=None):
        rows = self.M if rows is None else rows
        codes = self.codes if codes is None else codes
        if self.bits != 8:
            uq_quantize_packed(g, self.d, rows, g.stride(0), worker0, self.w, self.scales, self.K, self.idx, seed,
                               self.bits, codes, codes.stride(0), stream)
        elif self.K == 1:
            uq_quantize_single(g, self.d, rows, g.stride(0), worker0, self.w, int(self.scales[0]), seed, codes,
                               codes.stride(0), stream)
        else:
            uq_quantize_multi(g, self.d, rows, g.stride(0), worker0, self.w, self.scales, self.K, self.idx, seed,
                              codes, codes.stride(0), stream)

    def sum_codes(self, rows: int | None = None, accumulate: int = 0, codes=None, stream=None):
        rows = self.M if rows is None else rows
        codes = self.codes if codes is None else codes
        if self.bits != 8:
            uq_sum_packed(codes, self.d, rows, codes.stride(0), self.bits, accumulate, self.sum, stream)
        else:
            uq_sum_codes(codes, self.d, rows, codes.stride(0), accumulate, self.sum, stream)

    def quantize_sum(self, g, seed: int, rows: int | None = None, worker0: int = 0, accumulate: int = 0,
                     reconstruct: bool = True, stream=None):
        rows = self.M if rows is None else rows
        call = uq_quantize_sum_idx4 if self.index_bits == 4 else uq_quantize_sum
        call(g, self.d, rows, g.stride(0), worker0, self.w, self.scales, self.K, self.idx, seed, accumulate,
             self.sum, self.M, self.out if reconstruct else None, stream)

    def index_host(self, i0: int = 0, i1: int | None = None) -> np.ndarray:
        """The shared index k*_i for i in [i0, i1) as host uint8 values (the
        4-bit layout's fields read out: the low nibble of byte i / 2 for even
        i, the high one for odd i)."""
        i1 = self.d if i1 is None else i1
        if self.index_bits == 8:
            return self.idx[i0:i1].cpu().numpy()
        b = self.idx[i0 // 2:(i1 + 1) // 2].cpu().numpy()
        fields = np.stack([b & 0xF, b >> 4], axis=1).reshape(-1)
        return fields[i0 - 2 * (i0 // 2):i0 - 2 * (i0 // 2) + (i1 - i0)]

    def index_quantize(self, g, seed: int, stream=None):
        uq_index_quantize(g, self.d, self.M, g.stride(0), self.w, self.scales, self.K, seed, self.bits, self.idx,
                          self.codes, self.codes.stride(0), stream)

    def index_quantize_sum(self, g, seed: int, stream=None):
        uq_index_quantize_sum(g, self.d, self.M, g.stride(0), self.w, self.scales, self.K, seed, self.idx, self.sum,
                              self.out, stream)

    def dequantize(self, stream=None):
        uq_dequantize(self.sum, self.d, self.M, self.w, self.scales, self.K, self.idx, self.out, stream)

    def sum_dequantize(self, rows: int | None = None, accumulate: int = 0, codes=None, stream=None):
        rows = self.M if rows is None else rows
        codes = self.codes if codes is None else codes
        uq_sum_dequantize(codes, self.d, rows, codes.stride(0), self.bits, accumulate, self.sum, self.M, self.w,
                          self.scales, self.K, self.idx, self.out, stream)

    # -- the whole step ----------------------------------------------------------
    def run(self, g, seed: int, stream=None):
        """g: [M, ldg] float32 on the device.  Returns the output view [d]."""
        assert g.dtype == torch.float32 and g.device == self.device and g.shape[0] == self.M
        assert g.stride(1) == 1 and g.shape[1] >= self.d
        stream = _stream(stream)  # resolved once for the step's calls
        self.shared_scale(g, stream, w_only=self.index_in_pass)
        if self.index_in_pass and self.quant_sum:
            self.index_quantize_sum(g, seed, stream=stream)
        elif self.index_in_pass:
            self.index_quantize(g, seed, stream=stream)
            if self.fused:
                self.sum_dequantize(stream=stream)
            else:
                self.sum_codes(stream=stream)
        elif self.quant_sum and self.streamed:
            for m in range(self.M):
                self.quantize_sum(g[m:m + 1], seed, rows=1, worker0=m, accumulate=1 if m > 0 else 0,
                                  reconstruct=m == self.M - 1, stream=stream)
        elif self.quant_sum:
            self.quantize_sum(g, seed, stream=stream)
        elif self.streamed:
            for m in range(self.M):
                self.quantize(g[m:m + 1], seed, rows=1, worker0=m, stream=stream)
                acc = 1 if m > 0 else 0
                if self.fused and m == self.M - 1:
                    self.sum_dequantize(rows=1, accumulate=acc, stream=stream)
                else:
                    self.sum_codes(rows=1, accumulate=acc, stream=stream)
        else:
            self.quantize(g, seed, stream=stream)
            if self.fused:
                self.sum_dequantize(stream=stream)
            else:
                self.sum_codes(stream=stream)
        if not self.fused:
            self.dequantize(stream)
        return self.out[:self.d]


class RandKStep:
    """GlobalRandK step (Sec. 3.3-3.4): select k coordinates shared by all
    workers, gather them into [M, k] sub-vectors, run Algorithm 1/2 on those
    with `Step`, and scatter the reconstruction into the d-vector (0 elsewhere)."""

    def __init__(self, d: int, M: int, k: int, scales, device="cuda"):
        self.d, self.M, self.k = d, M, k
        self.inner = Step(k, M, scales, device=device)
        dev = self.inner.device
        self.sel = torch.zeros(round_up(k, 64), dtype=torch.int32, device=dev)  # uint32 indices
        self.sub = torch.zeros((M, round_up(k, 64)), dtype=torch.float32, device=dev)
        self.rk_ws_bytes = uq_randk_workspace_bytes(d, k)
        self.rk_ws = torch.zeros(self.rk_ws_bytes // 8, dtype=torch.float64, device=dev)
        self.out = torch.zeros(round_up(max(d, 1), 64), dtype=torch.float32, device=dev)

    def select(self, seed: int, stream=None):
        uq_randk_select(self.d, self.k, seed, self.sel, self.rk_ws, self.rk_ws_bytes, stream)

    def gather(self, g, stream=None):
        uq_gather(g, self.d, self.M, g.stride(0), self.sel, self.k, self.sub, self.sub.stride(0), stream)

    def scatter(self, stream=None):
        uq_scatter(self.inner.out, self.sel, self.k, self.out, self.d, stream)

    def run(self, g, seed: int, stream=None):
        assert g.dtype == torch.float32 and g.shape[0] == self.M and g.stride(1) == 1
        stream = _stream(stream)  # resolved once for the step's calls
        self.select(seed, stream)
        self.gather(g, stream)
        self.inner.run(self.sub, seed, stream)
        self.scatter(stream)
        return self.out[:self.d]


def capture(step, g, seed: int):
    """Record step.run(g, seed) into a HIP graph (torch's graph API over the
    stream the library launches on).  Replaying it redoes the whole step on
    the same buffers; the library's kernels issue no memsets or allocations."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step.run(g, seed)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step.run(g, seed)
    torch.cuda.synchronize()
    return graph
