"""Pins of the oracle's consensus distance (oracle/metrics.py) against what
the definition and the paper fix, independent of its own formula: exact
rational arithmetic on tiny inputs through the pairwise form, the two-worker
closed form, invariances, and the linear convergence of Alg. 1's consensus
distance with lr = 0 (Section 4)."""
from fractions import Fraction
from itertools import product

import numpy as np

import oracle
from oracle.metrics import consensus_distance
import workloads as wl


def _pairwise_exact(x):
    """(1/(2 n^2)) * sum_{i,j} ||x_i - x_j||^2 in exact rationals: the same
    quantity written through pairwise distances, no average formed."""
    n, d = x.shape
    rows = [[Fraction(float(v)) for v in r] for r in x]
    tot = Fraction(0)
    for i, j in product(range(n), range(n)):
        tot += sum((rows[i][c] - rows[j][c]) ** 2 for c in range(d))
    return tot / (2 * n * n)


def test_identical_rows_have_zero_distance():
    row = np.random.default_rng(1).standard_normal(37).astype(np.float32)
    x = np.tile(row, (9, 1))
    assert consensus_distance(x) == (0.0, 0.0)


def test_two_workers_closed_form():
    # n = 2: xbar = (a + b) / 2, so Xi = ||a - b||^2 / 4 and the largest
    # deviation is max |a - b| / 2.
    rng = np.random.default_rng(2)
    a, b = rng.standard_normal((2, 11)).astype(np.float32)
    dist, spread = consensus_distance(np.stack([a, b]))
    diff = a.astype(np.float64) - b.astype(np.float64)
    assert abs(dist - (diff @ diff) / 4) <= 1e-15 * (diff @ diff)
    assert spread == np.abs(diff).max() / 2


def test_pairwise_form_exactly_on_tiny_inputs():
    rng = np.random.default_rng(3)
    for n, d in [(1, 3), (3, 1), (5, 7), (6, 4)]:
        x = (rng.standard_normal((n, d)) * 4).astype(np.float32)
        want = _pairwise_exact(x)
        got, _ = consensus_distance(x)
        assert abs(Fraction(got) - want) <= Fraction(1, 10**12) * max(want, Fraction(1)), (n, d)


def test_shift_and_scale():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((8, 50))
    base, spread = consensus_distance(x)
    shifted, s2 = consensus_distance(x + rng.standard_normal(50))
    assert abs(shifted - base) <= 1e-12 * base and abs(s2 - spread) <= 1e-12 * spread
    scaled, s3 = consensus_distance(3.0 * x)
    assert abs(scaled - 9.0 * base) <= 1e-12 * base and abs(s3 - 3.0 * spread) <= 1e-12 * spread


def test_alg1_pulls_models_together_at_a_linear_rate():
    """With lr = 0, Alg. 1 is a consensus algorithm whose consensus distance
    converges linearly (Section 4's key lemma): on a random tree of 12
    workers each window of 20 rounds after the first shrinks the distance by
    more than 3x, and 200 rounds take it below 1e-6 of its start."""
    n, d = 12, 64
    edges = wl.random_tree_edges(n, seed=5)
    x = np.random.default_rng(6).standard_normal((n, d))
    o = oracle.Oracle(n, d, edges, np.float64)
    zero = np.zeros_like(x)
    seen = [consensus_distance(x)[0]]
    for t in range(1, 201):
        o.round(x, zero, None, 0.0, 0.0)
        if t % 20 == 0:
            seen.append(consensus_distance(x)[0])
    o.close()
    assert all(b < a / 3 for a, b in zip(seen[1:], seen[2:])), seen
    assert seen[-1] < 1e-6 * seen[0], seen
