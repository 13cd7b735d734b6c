"""Seeded synthetic gradients shaped like the paper's workloads.

This module holds input generation only: no step of the quantisers.  It is
shared by the tests, the smoke check and the benchmark, and both the HIP
path and the CPU oracle consume what it produces.

Workloads (flat fp32 gradients of M simulated workers, row-major [M][ldg]):
  * small-gaussian : d = 2^20, M = 4, i.i.d. N(0, 1e-3^2), one scale s = 127.
  * resnet18       : d = 11,173,962 (62 CIFAR ResNet-18 tensors), M = 8,
                     per-tensor Laplace(0, b_l), b_l = 10^U(-5,-2), s = 127.
  * resnet50       : d = 25,557,032 (161 ResNet-50 tensors), M = 8,
                     per-tensor N(0, sigma_l^2), sigma_l = 10^U(-6,-2), then
                     every coordinate of every worker x100 with prob. 0.01;
                     K = 4 scales 127 * 16^k (8-bit codes).
  * vgg16          : d = 138,357,544 (32 VGG-16 tensors), M = 16; the fully
                     connected tensors N(0, 1e-4^2), the convolutional ones
                     N(0, 1e-3^2); one scale s = 7, or K = 4 scales 7 * 16^k.
  * student-t      : d = 2^30, M = 16, 1e-4 * t_3; K = 8 scales 127 * 16^k,
                     workers streamed through an int32 accumulator.
  * *-4bit, *-2bit : the same gradients with the codes held packed (s = 7
                     in 4 bits, s = 1 in 2 bits).
  * *-grandk*      : the same gradients with GlobalRandK sparsification of
                     10000 coordinates (one scale, or two scales 127, 2032).

Per-tensor parameters come from numpy.random.default_rng(seed) and are shared
by the workers; worker m's values come from a torch generator seeded
seed * 1000 + m on the device the tensor is made on.
"""
from __future__ import annotations

import math

import numpy as np


# ---------------------------------------------------------------------------
# Parameter-tensor sizes of the three architectures, in registration order.
# ---------------------------------------------------------------------------

def resnet18_cifar_sizes() -> list[int]:
    """CIFAR ResNet-18: 3x3 stem, four stages of two basic blocks, 10-way fc."""
    sizes = [3 * 64 * 9, 64, 64]  # stem conv, BN weight, BN bias
    cin = 64
    for width in (64, 128, 256, 512):
        for b in range(2):
            sizes += [cin * width * 9, width, width, width * width * 9, width, width]
            if b == 0 and cin != width:
                sizes += [cin * width, width, width]  # 1x1 shortcut + BN
            cin = width
    sizes += [512 * 10, 10]
    return sizes


def resnet50_sizes() -> list[int]:
    """ImageNet ResNet-50: 7x7 stem, bottleneck stages (3, 4, 6, 3), 1000-way fc."""
    sizes = [3 * 64 * 49, 64, 64]
    cin = 64
    for width, blocks in ((64, 3), (128, 4), (256, 6), (512, 3)):
        for b in range(blocks):
            sizes += [cin * width, width, width,
                      width * width * 9, width, width,
                      width * width * 4, width * 4, width * 4]
            if b == 0:
                sizes += [cin * width * 4, width * 4, width * 4]  # downsample + BN
            cin = width * 4
    sizes += [2048 * 1000, 1000]
    return sizes


def vgg16_sizes() -> list[tuple[int, bool]]:
    """ImageNet VGG-16: 13 3x3 convolutions and 3 fully connected layers,
    each a weight and a bias.  Returns (size, is_fully_connected)."""
    out = []
    cin = 3
    for width in (64, 64, 128, 128, 256, 256, 256, 512, 512, 512, 512, 512, 512):
        out += [(cin * width * 9, False), (width, False)]
        cin = width
    for fin, fout in ((25088, 4096), (4096, 4096), (4096, 1000)):
        out += [(fin * fout, True), (fout, True)]
    return out


def scales_for(bits: int, K: int) -> list[float]:
    """s_0 = 2^(bits-1) - 1 (a signed `bits`-bit code), s_k = s_0 * 16^k."""
    s0 = 2 ** (bits - 1) - 1
    return [float(s0 * 16 ** k) for k in range(K)]


WORKLOADS = {
    "small-gaussian": dict(d=2 ** 20, M=4, scales=scales_for(8, 1), seed=1, kind="gaussian"),
    "resnet18": dict(d=11_173_962, M=8, scales=scales_for(8, 1), seed=2, kind="resnet18"),
    "resnet50": dict(d=25_557_032, M=8, scales=scales_for(8, 4), seed=3, kind="resnet50"),
    "vgg16-single": dict(d=138_357_544, M=16, scales=scales_for(4, 1), seed=4, kind="vgg16"),
    "vgg16-multi": dict(d=138_357_544, M=16, scales=scales_for(4, 4), seed=4, kind="vgg16"),
    "student-t": dict(d=2 ** 30, M=16, scales=scales_for(8, 8), seed=5, kind="student-t",
                      streamed=True),
    # the same codes held as 4-bit / 2-bit fields
    "vgg16-single-4bit": dict(d=138_357_544, M=16, scales=scales_for(4, 1), seed=4, kind="vgg16", bits=4),
    "vgg16-multi-4bit": dict(d=138_357_544, M=16, scales=scales_for(4, 4), seed=4, kind="vgg16", bits=4),
    "resnet18-2bit": dict(d=11_173_962, M=8, scales=scales_for(2, 1), seed=2, kind="resnet18", bits=2),
    # GlobalRandK (Sec. 3.3-3.4) with the paper's K = 10000 sampled coordinates
    "resnet18-grandk": dict(d=11_173_962, M=8, scales=scales_for(8, 1), seed=2, kind="resnet18", randk=10_000),
    "resnet50-grandk-ts": dict(d=25_557_032, M=8, scales=scales_for(8, 2), seed=3, kind="resnet50",
                               randk=10_000),
}


def round_up(x: int, m: int) -> int:
    return (x + m - 1) // m * m


def leading_dims(d: int) -> tuple[int, int]:
    """(ldg, ldc): gradient rows padded to 64 floats, code rows to 256 bytes."""
    return round_up(max(d, 1), 64), round_up(max(d, 1), 256)


def layer_plan(kind: str, d: int, seed: int):
    """Per-tensor (start, size, parameter) for the block-structured workloads."""
    rng = np.random.default_rng(seed)
    if kind == "resnet18":
        sizes = resnet18_cifar_sizes()
        params = 10.0 ** rng.uniform(-5, -2, size=len(sizes))
    elif kind == "resnet50":
        sizes = resnet50_sizes()
        params = 10.0 ** rng.uniform(-6, -2, size=len(sizes))
    elif kind == "vgg16":
        spec = vgg16_sizes()
        sizes = [s for s, _ in spec]
        params = np.array([1e-4 if fc else 1e-3 for _, fc in spec])
    else:
        return [(0, d, None)]
    assert sum(sizes) == d, (kind, sum(sizes), d)
    plan, start = [], 0
    for size, p in zip(sizes, params):
        plan.append((start, size, float(p)))
        start += size
    return plan


def fill_worker(row, kind: str, d: int, seed: int, worker: int, plan=None, chunk: int = 1 << 26):
    """Fill row[:d] (a torch float32 tensor) with worker `worker`'s gradient."""
    import torch

    dev = row.device
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed * 1000 + worker)
    plan = plan if plan is not None else layer_plan(kind, d, seed)
    for start, size, p in plan:
        for c0 in range(0, size, chunk):
            n = min(chunk, size - c0)
            dst = row[start + c0:start + c0 + n]
            if kind == "gaussian":
                dst.normal_(0.0, 1e-3, generator=gen)
            elif kind == "resnet18":
                # Laplace(0, b): a sign times b * Exp(1), with Exp(1) = -log(1 - U)
                mag = torch.empty(n, device=dev, dtype=torch.float32).exponential_(1.0, generator=gen)
                sgn = torch.randint(0, 2, (n,), device=dev, generator=gen, dtype=torch.int8)
                dst.copy_(mag * p)
                dst.mul_(sgn.to(torch.float32) * 2 - 1)
            elif kind == "resnet50":
                dst.normal_(0.0, p, generator=gen)
                hit = torch.rand(n, device=dev, generator=gen) < 0.01
                dst.mul_(torch.where(hit, 100.0, 1.0))
            elif kind == "vgg16":
                dst.normal_(0.0, p, generator=gen)
            elif kind == "student-t":
                z = torch.randn(n, device=dev, generator=gen)
                chi2 = torch.zeros(n, device=dev)
                for _ in range(3):
                    e = torch.randn(n, device=dev, generator=gen)
                    chi2.add_(e * e)
                dst.copy_(z / torch.sqrt(chi2 / 3.0) * 1e-4)
            else:
                raise ValueError(kind)


def make_gradients(name_or_cfg, device="cuda", rows=None, d=None):
    """Allocate [M, ldg] float32 on `device` (padding zero) and fill every worker.

    `d` overrides the workload's dimension (only for the gaussian and
    student-t kinds, which have no layer structure); `rows` limits the number
    of workers generated.
    """
    import torch

    cfg = dict(WORKLOADS[name_or_cfg]) if isinstance(name_or_cfg, str) else dict(name_or_cfg)
    if d is not None:
        assert cfg["kind"] in ("gaussian", "student-t")
        cfg["d"] = d
    M = cfg["M"] if rows is None else rows
    ldg, _ = leading_dims(cfg["d"])
    g = torch.zeros((M, ldg), dtype=torch.float32, device=device)
    plan = layer_plan(cfg["kind"], cfg["d"], cfg["seed"])
    for m in range(M):
        fill_worker(g[m], cfg["kind"], cfg["d"], cfg["seed"], m, plan)
    return g, cfg


def gaussian_rows(M: int, d: int, seed: int, sigma: float = 1e-3, ldg: int | None = None) -> np.ndarray:
    """Small host-side N(0, sigma^2) rows (numpy), padded with zeros to ldg."""
    rng = np.random.default_rng(seed)
    ldg = d if ldg is None else ldg
    g = np.zeros((M, ldg), dtype=np.float32)
    g[:, :d] = rng.normal(0.0, sigma, size=(M, d)).astype(np.float32)
    return g


def mixed_rows(M: int, d: int, seed: int, ldg: int | None = None) -> np.ndarray:
    """Small host-side rows exercising the edge cases: per-block scales over six
    decades, exact zeros, negative zeros, denormals, a coordinate equal to a
    whole row's norm (one-hot row) and outliers."""
    rng = np.random.default_rng(seed)
    ldg = d if ldg is None else ldg
    g = np.zeros((M, ldg), dtype=np.float32)
    for m in range(M):
        sig = 10.0 ** rng.uniform(-6, 0, size=max(1, d // 97 + 1))
        blocks = np.repeat(sig, 97)[:d]
        row = rng.normal(0.0, 1.0, size=d) * blocks
        row[rng.random(d) < 0.05] = 0.0
        row[rng.random(d) < 0.01] *= 100.0
        g[m, :d] = row.astype(np.float32)
        neg0 = rng.random(d) < 0.01
        g[m, :d][neg0] = np.float32(-0.0)
        den = rng.random(d) < 0.005
        g[m, :d][den] = (rng.integers(1, 1 << 20, size=int(den.sum())) * (2.0 ** -149)).astype(np.float32)
    if M > 1 and d > 0:
        g[M - 1, :d] = 0.0
        g[M - 1, d // 2] = np.float32(-math.pi)  # one-hot row: |v_i| equals its row norm
    return g
