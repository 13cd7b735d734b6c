"""Analytic per-step time of quantised data-parallel aggregation on P MI355X
GPUs, one worker per GPU, for the exchanges of Algorithms 1-2 (Sec. 3.1-3.2)
and GlobalRandK (Sec. 3.3-3.4), against the uncompressed fp32 all-reduce.

The paper studies scaling with a performance model taken from prior work
(Sec. 5.6) on V100 nodes and Ethernet; this module is a model of the same kind
with MI355X parameters: the local work is the measured streaming throughput of
this library's kernels, the exchanges are bandwidth-latency models of ring
collectives.

Per step, with d coordinates and P GPUs:
  local   norm (4 B per coordinate), quantise (5 B; 6 B with several scales),
          reconstruction (8 B; 9 B), index pass with several scales (5 B),
          all at `local_tbps`;
  scale   all-reduce MAX of one fp32: latency only;
  index   with several scales, all-reduce MIN of d uint8;
  codes   all-reduce SUM: the wire carries int16 partial sums (int8 overflows
          once P * s_min > 127; int16 is exact while P * s_min <= 32767), or
          with sub-byte codes an all-gather of the packed codes followed by a
          local sum, whichever is cheaper;
  fp32    the uncompressed baseline: one all-reduce SUM of d fp32 and no
          local quantisation work.
A ring all-reduce of n bytes costs 2 (P - 1) (alpha + n / (P B)); a ring
all-gather of P blocks of n bytes costs (P - 1) (alpha + n / B), with B the
per-direction bandwidth of the links the ring uses and alpha the per-step
latency.  Computation and communication are not overlapped (a conservative
bound; overlap with the backward pass would hide part of either).
"""
from __future__ import annotations

from dataclasses import dataclass


@dataclass(frozen=True)
class Network:
    name: str
    bandwidth_gbps: float   # per direction, GB/s, of the links one ring uses
    latency_us: float       # per ring step

    def ring_allreduce_s(self, nbytes: float, P: int) -> float:
        if P <= 1:
            return 0.0
        return 2 * (P - 1) * (self.latency_us * 1e-6 + nbytes / (P * self.bandwidth_gbps * 1e9))

    def ring_allgather_s(self, nbytes_per_gpu: float, P: int) -> float:
        if P <= 1:
            return 0.0
        return (P - 1) * (self.latency_us * 1e-6 + nbytes_per_gpu / (self.bandwidth_gbps * 1e9))


# xGMI inside an MI355X node: seven point-to-point links of about 153 GB/s per
# GPU; one ring uses one link per hop, rings over disjoint links add up.  A
# 400 Gb/s NIC per GPU between nodes; the paper's 10 Gb/s Ethernet for
# comparison.  Latencies are typical orders of magnitude, not measurements.
NETWORKS = {
    "xgmi-1ring": Network("xGMI, one ring", 153.0, 2.0),
    "xgmi-7rings": Network("xGMI, seven rings", 7 * 153.0, 2.0),
    "nic-400g": Network("400 Gb/s NIC per GPU", 50.0, 5.0),
    "eth-10g": Network("10 Gb/s Ethernet", 1.25, 20.0),
}

# Streaming rate of this library's kernels on one MI355X (the measured norm,
# quantise and sum + reconstruction kernels run at 6.3-7.1 TB/s, the fused
# norm and index passes at 5.2-5.8).
LOCAL_TBPS = 6.4


@dataclass(frozen=True)
class Scheme:
    name: str
    bits: int | None        # code bits (None: uncompressed fp32)
    several_scales: bool = False
    randk: int | None = None  # GlobalRandK sample size


SCHEMES = [
    Scheme("fp32 all-reduce", None),
    Scheme("8-bit codes, one scale", 8),
    Scheme("8-bit codes, several scales", 8, True),
    Scheme("4-bit codes, one scale", 4),
    Scheme("2-bit codes, one scale", 2),
    Scheme("GlobalRandK 10000, 8-bit", 8, False, 10_000),
]


def local_s(d: int, scheme: Scheme, local_tbps: float = LOCAL_TBPS) -> float:
    """Per-GPU kernel time of one step (one worker row)."""
    if scheme.bits is None:
        return 0.0
    n = scheme.randk if scheme.randk else d
    code = scheme.bits / 8
    per = 4 + (4 + code) + 8            # norm, quantise, reconstruction
    if scheme.several_scales:
        per += 5 + 1 + 1                # index pass, index read by quantise and reconstruction
    t = n * per / (local_tbps * 1e12)
    if scheme.randk:
        t += 2 * d * 4 / (local_tbps * 1e12)  # zero fill and scatter into the d-vector
    return t


def comm_s(d: int, P: int, scheme: Scheme, net: Network) -> float:
    """Exchange time of one step."""
    if scheme.bits is None:
        return net.ring_allreduce_s(4 * d, P)
    n = scheme.randk if scheme.randk else d
    t = net.ring_allreduce_s(4, P)                       # W (MAX)
    if scheme.several_scales:
        t += net.ring_allreduce_s(n, P)                  # shared index (MIN)
    summed = net.ring_allreduce_s(2 * n, P)              # int16 partial sums
    gathered = net.ring_allgather_s(n * scheme.bits / 8, P)  # packed codes, summed locally
    return t + min(summed, gathered)


def step_s(d: int, P: int, scheme: Scheme, net: Network, local_tbps: float = LOCAL_TBPS) -> float:
    return local_s(d, scheme, local_tbps) + comm_s(d, P, scheme, net)


def table(d: int, P_values=(2, 8, 32, 128), networks=None, schemes=None) -> list[dict]:
    networks = NETWORKS if networks is None else networks
    schemes = SCHEMES if schemes is None else schemes
    rows = []
    for key, net in networks.items():
        for P in P_values:
            base = step_s(d, P, schemes[0], net)
            for sc in schemes:
                t = step_s(d, P, sc, net)
                rows.append(dict(network=key, P=P, scheme=sc.name, ms=t * 1e3,
                                 speedup=base / t if t > 0 else float("inf")))
    return rows


def main() -> int:
    import argparse

    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--d", type=int, default=138_357_544, help="coordinates (default: VGG-16)")
    args = ap.parse_args()
    rows = table(args.d)
    print(f"d = {args.d:,}")
    print(f"{'network':12s} {'P':>4s}  {'scheme':30s} {'ms/step':>9s} {'vs fp32':>8s}")
    for r in rows:
        print(f"{r['network']:12s} {r['P']:4d}  {r['scheme']:30s} {r['ms']:9.3f} {r['speedup']:8.2f}")
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
