"""End to end on the CPU: RelaySGD as a training loop on heterogeneous
quadratics, with the oracle's round.

Worker i minimises f_i(x) = |x - b_i|^2 / 2, with optima b_i far apart (the
paper's data heterogeneity); the global optimum of the average objective is
mean_i b_i.  A fixed point of Alg. 1 with every worker at the same x, and
counters saturated, has x = (1/n) sum_k (x - lr (x - b_k)), that is x =
mean_i b_i: RelaySGD with a constant step reaches the exact optimum,
whatever the heterogeneity (Section 4: Theorem 1's rate does not depend on
it).  Gossip averaging with the same step (D-SGD, eq. DP-SGD of Section 3,
with Metropolis-Hastings weights) settles at a point biased by the
heterogeneity; it runs beside as a contrast, so the test cannot pass for a
trivial reason.
"""
import numpy as np
import pytest

import oracle
from oracle.double import DoubleOracle
import workloads as wl


def problem(n, d, seed=0):
    rng = np.random.default_rng(seed)
    return rng.standard_normal((n, d)) + 3.0 * np.arange(n)[:, None]


def relaysgd(n, edges, b, lr, beta, rounds, edges_b=None):
    x = np.zeros_like(b)
    mom = np.zeros_like(b)
    o = (oracle.Oracle(n, b.shape[1], edges, np.float64) if edges_b is None
         else DoubleOracle(n, b.shape[1], edges, edges_b, np.float64))
    for _ in range(rounds):
        o.round(x, x - b, mom if beta else None, lr, beta)
    if edges_b is None:
        o.close()
    else:
        o.a.close()
        o.b.close()
    return x


def gossip(n, edges, b, lr, rounds):
    """D-SGD with Metropolis-Hastings weights: x <- W (x - lr (x - b))."""
    deg = np.zeros(n, int)
    for u, v in edges:
        deg[u] += 1
        deg[v] += 1
    W = np.zeros((n, n))
    for u, v in edges:
        W[u, v] = W[v, u] = 1.0 / (1 + max(deg[u], deg[v]))
    W[np.arange(n), np.arange(n)] = 1.0 - W.sum(1)
    x = np.zeros_like(b)
    for _ in range(rounds):
        x = W @ (x - lr * (x - b))
    return x


@pytest.mark.parametrize("name,n,edges,edges_b,lr,beta,rounds", [
    ("chain16 SGD", 16, wl.chain_edges(16), None, 0.5, 0.0, 500),
    ("chain16 Nesterov", 16, wl.chain_edges(16), None, 0.1, 0.9, 800),
    ("random tree of 64", 64, wl.random_tree_edges(64, seed=3), None, 0.5, 0.0, 700),
    ("double binary trees of 16", 16, *wl.double_binary_tree_edges(16), 0.5, 0.0, 500),
])
def test_relaysgd_reaches_the_exact_optimum(name, n, edges, edges_b, lr, beta, rounds):
    b = problem(n, 6)
    opt = b.mean(0)
    x = relaysgd(n, edges, b, lr, beta, rounds, edges_b)
    assert np.abs(x - opt).max() < 1e-10, name
    if edges_b is None and beta == 0.0:
        bias = np.abs(gossip(n, edges, b, lr, rounds) - opt).max()
        assert bias > 1e-2, (name, bias)
