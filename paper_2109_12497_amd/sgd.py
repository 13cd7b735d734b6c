"""Data-parallel projected SGD with quantised gradient aggregation on a
synthetic least-squares problem: the setting of the convergence results of
arXiv 2109.12497 (Theorem 1 and Corollary 1 restated from prior work,
Theorems 2-3 for the max-norm quantisers).

f(theta) = 1/(2N) ||A theta - b||^2 is convex and L-smooth with
L = lambda_max(A^T A / N).  Worker m holds a shard (A_m, b_m) of N/M rows and
contributes its shard gradient g_m(theta) = A_m^T (A_m theta - b_m) / (N/M);
their mean is the full gradient.  Each step aggregates the M shard gradients
through a quantised all-reduce (shared max-norm scale, stochastic rounding,
integer sum, dequantisation) or, as the baseline, their plain fp32 mean, and
takes a projected step on the ball ||theta - theta_0|| <= R.

The only randomness is the quantiser's, so the aggregated gradient's variance
is the quantisation variance.  By Lemma 1 (Lemma 2 with s_hat = min_k s_k)
each worker adds at most min(n/s^2, sqrt(n)/s) W^2 with W the shared norm;
independent workers averaged give
    sigma^2 <= min(n/s_hat^2, sqrt(n)/s_hat) * W_max^2 / M,
with W_max a bound of every shard gradient's norm on the ball.  Theorem 1 with
that variance (constant step 1/(L + 1/gamma), gamma = (R/sigma) sqrt(2/T))
bounds the averaged iterate's suboptimality by
    R sqrt(2 sigma^2 / T) + L R^2 / T,
which is the content of Theorems 2-3 for this problem.

The aggregator is a callable (grads [M, ldg] fp32 device tensor, d, seed) ->
[d] fp32 tensor.  `QuantisedAggregate` runs the library's four calls; the
baseline is `mean_aggregate`.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import torch

from .step import Step


@dataclass
class LeastSquares:
    A: torch.Tensor        # [M, rows, n] float64
    b: torch.Tensor        # [M, rows] float64
    H: torch.Tensor        # [M, n, n] float64: A_m^T A_m / rows
    c: torch.Tensor        # [M, n] float64: A_m^T b_m / rows
    L: float               # lambda_max of the mean of H
    R: float               # radius of the feasible ball around theta0 = 0
    theta_star: torch.Tensor  # minimiser of f over the ball (inside it)
    f_star: float
    W_max: float           # bound of ||g_m(theta)|| over the ball and m

    @property
    def n(self) -> int:
        return self.A.shape[2]

    @property
    def M(self) -> int:
        return self.A.shape[0]


def make_problem(n: int, M: int, rows: int, seed: int, device="cpu", noise: float = 0.1) -> LeastSquares:
    """Gaussian features with a per-worker scale and shift (heterogeneous
    shards), b = A theta_true + noise."""
    gen = torch.Generator(device="cpu").manual_seed(seed)
    theta_true = torch.randn(n, generator=gen, dtype=torch.float64)
    scale = 0.5 + torch.rand(M, 1, 1, generator=gen, dtype=torch.float64)
    shift = 0.05 * torch.randn(M, 1, n, generator=gen, dtype=torch.float64)
    A = torch.randn(M, rows, n, generator=gen, dtype=torch.float64) * scale + shift
    b = A @ theta_true + noise * torch.randn(M, rows, generator=gen, dtype=torch.float64)
    H = A.transpose(1, 2) @ A / rows
    c = (A.transpose(1, 2) @ b.unsqueeze(2)).squeeze(2) / rows
    Hbar, cbar = H.mean(0), c.mean(0)
    L = float(torch.linalg.eigvalsh(Hbar)[-1])
    theta_star = torch.linalg.solve(Hbar, cbar)
    R = 2.0 * float(theta_star.norm())
    # ||g_m(theta)|| <= ||H_m||_2 ||theta|| + ||c_m|| <= ||H_m||_2 R + ||c_m||
    W_max = max(float(torch.linalg.eigvalsh(H[m])[-1]) * R + float(c[m].norm()) for m in range(M))
    p = LeastSquares(A=A.to(device), b=b.to(device), H=H.to(device), c=c.to(device), L=L, R=R,
                     theta_star=theta_star.to(device), f_star=0.0, W_max=W_max)
    p.f_star = loss(p, p.theta_star)
    return p


def loss(p: LeastSquares, theta: torch.Tensor) -> float:
    r = p.A @ theta - p.b
    return float((r * r).sum() / (2 * r.numel()))


def shard_gradients(p: LeastSquares, theta: torch.Tensor, out: torch.Tensor) -> None:
    """out[m, :n] = fp32(H_m theta - c_m)."""
    out[:, :p.n].copy_(torch.matmul(p.H, theta) - p.c)


def project(p: LeastSquares, theta: torch.Tensor) -> torch.Tensor:
    nrm = float(theta.norm())
    return theta if nrm <= p.R else theta * (p.R / nrm)


def variance_bound(p: LeastSquares, scales) -> float:
    """Lemma 1 / 2 excess second moment of one worker, averaged over M
    independent workers; 0 for the unquantised mean (scales None)."""
    if scales is None:
        return 0.0
    s_hat = float(min(scales))
    n = p.n
    return min(n / s_hat ** 2, math.sqrt(n) / s_hat) * p.W_max ** 2 / p.M


def theorem_step(p: LeastSquares, sigma2: float, T: int) -> tuple[float, float]:
    """(eta, bound): the constant step 1/(L + 1/gamma), gamma = (R/sigma) sqrt(2/T),
    and the resulting bound R sqrt(2 sigma^2/T) + L R^2/T of the averaged iterate."""
    if sigma2 <= 0.0:
        return 1.0 / p.L, p.L * p.R ** 2 / T
    gamma = p.R / math.sqrt(sigma2) * math.sqrt(2.0 / T)
    return 1.0 / (p.L + 1.0 / gamma), p.R * math.sqrt(2.0 * sigma2 / T) + p.L * p.R ** 2 / T


def mean_aggregate(grads: torch.Tensor, d: int, seed: int) -> torch.Tensor:
    return grads[:, :d].mean(0)


class QuantisedAggregate:
    """The library's aggregation: shared scale -> quantise every worker ->
    integer sum -> dequantise (1/M folded in)."""

    def __init__(self, d: int, M: int, scales, device):
        self.step = Step(d, M, scales, device=device)

    def __call__(self, grads: torch.Tensor, d: int, seed: int) -> torch.Tensor:
        self.step.run(grads, seed)
        return self.step.out[:d]


def run_sgd(p: LeastSquares, aggregate, T: int, eta: float, seed: int, ldg: int | None = None) -> dict:
    """T projected SGD steps from theta0 = 0.  Returns the suboptimality of
    the averaged iterate (1/T) sum_{t=1..T} theta_t (the quantity Theorems 1-3
    bound), of the last iterate, and of the mean of the last T/2 iterates."""
    n, M = p.n, p.M
    device = p.A.device
    ldg = n if ldg is None else ldg
    grads = torch.zeros((M, ldg), dtype=torch.float32, device=device)
    theta = torch.zeros(n, dtype=torch.float64, device=device)
    avg = torch.zeros_like(theta)
    tail = torch.zeros_like(theta)
    for t in range(T):
        shard_gradients(p, theta, grads)
        g = aggregate(grads, n, seed * 1_000_003 + t).to(torch.float64)
        theta = project(p, theta - eta * g)
        avg += theta
        if t >= T // 2:
            tail += theta
    avg /= T
    tail /= T - T // 2
    return dict(gap_avg=loss(p, avg) - p.f_star, gap_last=loss(p, theta) - p.f_star,
                gap_tail=loss(p, tail) - p.f_star)


# Quantiser settings compared by the convergence table: None is the fp32 mean.
CONFIGS = {
    "fp32 mean": None,
    "s=1": [1.0],
    "s=7": [7.0],
    "s=127": [127.0],
    "multi 1,16,256,4096": [1.0, 16.0, 256.0, 4096.0],
    "multi 7,112,1792,28672": [7.0, 112.0, 1792.0, 28672.0],
}


def convergence_table(p: LeastSquares, make_aggregate, T: int, seeds=(0, 1, 2), configs=None) -> dict:
    """For every setting: the Theorem 1-3 bound and mean averaged-iterate gap
    at the theorem's step, and the mean tail gap at the common step 1/(2L).
    make_aggregate(scales) returns an aggregator (scales None: the mean)."""
    configs = CONFIGS if configs is None else configs
    table = {}
    for name, scales in configs.items():
        agg = make_aggregate(scales)
        sigma2 = variance_bound(p, scales)
        eta, bound = theorem_step(p, sigma2, T)
        thm = [run_sgd(p, agg, T, eta, seed=s)["gap_avg"] for s in seeds]
        fixed = [run_sgd(p, agg, T, 0.5 / p.L, seed=s)["gap_tail"] for s in seeds]
        table[name] = dict(sigma2_bound=sigma2, eta=eta, bound=bound, gap_avg=sum(thm) / len(thm),
                           gap_tail_fixed_step=sum(fixed) / len(fixed))
    return table


def main() -> int:
    import argparse
    import json

    ap = argparse.ArgumentParser(description="convergence table of quantised data-parallel SGD on one GPU")
    ap.add_argument("--n", type=int, default=1000)
    ap.add_argument("--M", type=int, default=8)
    ap.add_argument("--rows", type=int, default=4000)
    ap.add_argument("--T", type=int, default=300)
    ap.add_argument("--seed", type=int, default=1)
    args = ap.parse_args()
    dev = torch.device("cuda", torch.cuda.current_device())
    p = make_problem(args.n, args.M, args.rows, args.seed, device=dev)

    def make(scales):
        return mean_aggregate if scales is None else QuantisedAggregate(p.n, p.M, scales, dev)

    table = convergence_table(p, make, args.T)
    print(json.dumps(dict(n=p.n, M=p.M, rows=args.rows, T=args.T, L=p.L, R=p.R, W_max=p.W_max, f_star=p.f_star,
                          table=table), indent=1))
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
