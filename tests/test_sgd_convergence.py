"""Convergence of quantised data-parallel SGD (Theorems 1-3) on a synthetic
least-squares problem, with the oracle as the aggregator.

Checks: the averaged iterate's gap stays under the Theorem 1 bound evaluated
with the Lemma 1 / 2 variance, and at a common step the gap orders as the
quantisers' variance does (more levels or several scales: smaller gap).
"""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2109_12497_amd import sgd


def oracle_aggregate(scales):
    if scales is None:
        return sgd.mean_aggregate

    def agg(grads, d, seed):
        return torch.from_numpy(O.pipeline(grads.numpy(), scales, seed, d=d)["out"].copy())

    return agg


def check_table(table):
    for name, row in table.items():
        assert row["gap_avg"] >= -1e-9 and row["gap_avg"] <= row["bound"], (name, row)
    g = {k: v["gap_tail_fixed_step"] for k, v in table.items()}
    assert g["s=1"] > 2 * g["s=7"] > 4 * g["s=127"]
    assert g["s=127"] > g["fp32 mean"]
    # several scales: the coordinates below W s_0 / s_1 take the finer scale,
    # so the noise floor drops (by more as n grows and that fraction rises)
    assert g["multi 7,112,1792,28672"] < g["s=7"] / 1.5
    assert g["multi 1,16,256,4096"] < g["s=1"] / 1.5


@pytest.fixture(scope="module")
def problem():
    return sgd.make_problem(n=256, M=4, rows=1024, seed=1)


def test_problem_constants(problem):
    p = problem
    # the minimiser is inside the ball and has zero full gradient
    assert float(p.theta_star.norm()) < p.R
    g = torch.zeros((p.M, p.n), dtype=torch.float32)
    sgd.shard_gradients(p, p.theta_star, g)
    assert float(g.double().mean(0).norm()) < 1e-5 * float(g.double().norm())
    # W_max bounds every shard gradient norm on the ball (spot check on its surface)
    rng = np.random.default_rng(0)
    for _ in range(8):
        u = torch.from_numpy(rng.normal(size=p.n))
        sgd.shard_gradients(p, u / u.norm() * p.R, g)
        assert float(g.double().norm(dim=1).max()) <= p.W_max


def test_unquantised_step_is_gradient_descent(problem):
    """With the fp32 mean and step 1/L the run is plain projected gradient
    descent on a strongly convex problem: the last gap is tiny."""
    r = sgd.run_sgd(problem, sgd.mean_aggregate, T=400, eta=1.0 / problem.L, seed=0)
    assert r["gap_last"] < 1e-9


def test_convergence_table_oracle(problem):
    check_table(sgd.convergence_table(problem, oracle_aggregate, T=400))
