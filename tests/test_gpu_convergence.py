"""Convergence of quantised data-parallel SGD through the HIP path (the
library's four calls aggregate the workers' gradients at every step)."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

from oracle import oracle as O  # noqa: E402
from paper_2109_12497_amd import sgd  # noqa: E402

from test_sgd_convergence import check_table  # noqa: E402

DEV = torch.device("cuda:0")


@pytest.fixture(scope="module")
def problem():
    return sgd.make_problem(n=1000, M=8, rows=4000, seed=2, device=DEV)


def make(p):
    def f(scales):
        return sgd.mean_aggregate if scales is None else sgd.QuantisedAggregate(p.n, p.M, scales, DEV)
    return f


def test_aggregate_is_the_quantised_mean(problem):
    """One aggregation on the device equals the oracle's on the same inputs."""
    p = problem
    theta = torch.zeros(p.n, dtype=torch.float64, device=DEV)
    g = torch.zeros((p.M, p.n), dtype=torch.float32, device=DEV)
    sgd.shard_gradients(p, theta, g)
    for scales in ([7.0], [7.0, 112.0, 1792.0, 28672.0]):
        out = sgd.QuantisedAggregate(p.n, p.M, scales, DEV)(g, p.n, 12345).cpu().numpy()
        ref = O.pipeline(g.cpu().numpy(), scales, 12345, d=p.n)["out"]
        assert np.array_equal(out.view(np.int32), ref.view(np.int32))


def test_convergence_table_gpu(problem):
    check_table(sgd.convergence_table(problem, make(problem), T=300))
