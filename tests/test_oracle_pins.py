"""Pins of the oracle to facts other than itself (CPU only).

Each test checks the oracle against something the paper or mathematics fixes:
a 3-worker chain worked by hand from Alg. 1, closed forms for counters and
messages, the delayed-average form of the update (eq. RelaySum/Model with the
delays Alg. 1 actually realises), textbook special cases (n=1 is Nesterov SGD
as torch.optim.SGD implements it; n=2 is all-reduce; a star's centre holds
the exact mean), invariants, and exhaustive brute force over every labelled
tree with up to 6 workers.
"""
from fractions import Fraction as F

import numpy as np
import pytest

import golden
import oracle
from oracle.exact import ExactRelaySum
import treeutil
import workloads as wl

CHAIN3 = np.array([[0, 1], [1, 2]], dtype=np.int32)


def frac_rows(a):
    return [[F(v) for v in row] for row in a]


# --------------------------------------------------------------------------
# 1. Hand-worked 3-worker chain (Alg. 1 with App. D.2's momentum, derived
#    with pencil and paper; the paper prints no numeric example).  Workers
#    0-1-2, d = 1.  The exact values live in tests/golden with their source.
# --------------------------------------------------------------------------

# Directed edges listed as (src, dst), the order of the fixture's m and c.
EDGE_ORDER = [(0, 1), (1, 0), (1, 2), (2, 1)]


def _hand_case(case):
    return {
        "x0": case["x0"], "g": case["g"], "lr": case["lr"], "beta": case["beta"],
        "rounds": [(r["m"], r["x"]) for r in case["rounds"]],
        "mom": [r["mom"] for r in case["rounds"]] if case["beta"] != 0 else None,
        "counts": [(r["c"], r["nbar"]) for r in case["rounds"]],
    }


_HAND = golden.chain3_hand_worked()
HAND_A = _hand_case(_HAND["lr0"])        # x0 = (1, 2, 4), lr = 0, no momentum
HAND_B = _hand_case(_HAND["nesterov"])   # g = (2, 0, -2), lr = beta = 1/2
# Counters are the same in both examples.
HAND_COUNTS = HAND_A["counts"]
assert HAND_B["counts"] == HAND_COUNTS


@pytest.mark.parametrize("case", [HAND_A, HAND_B], ids=["lr0", "nesterov"])
def test_hand_worked_chain3_exact(case):
    ex = ExactRelaySum(3, 1, CHAIN3)
    x = [[F(v)] for v in case["x0"]]
    mom = [[F(0)] for _ in range(3)]
    g = [[F(v)] for v in case["g"]]
    for r, (msgs, xs) in enumerate(case["rounds"]):
        x, mom_new = ex.round(x, g, mom if case["beta"] != 0 else None, case["lr"], case["beta"])
        if case["beta"] != 0:
            mom = mom_new
            assert tuple(row[0] for row in mom) == case["mom"][r]
        assert tuple(ex.msg[e][0] for e in EDGE_ORDER) == msgs
        assert tuple(row[0] for row in x) == xs
        assert tuple(ex.cnt[e] for e in EDGE_ORDER) == HAND_COUNTS[r][0]
        assert tuple(ex.nbar) == HAND_COUNTS[r][1]


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
@pytest.mark.parametrize("case", [HAND_A, HAND_B], ids=["lr0", "nesterov"])
def test_hand_worked_chain3_c_oracle(case, dtype):
    o = oracle.Oracle(3, 1, CHAIN3, dtype=dtype)
    x = np.array([[v] for v in case["x0"]], dtype=dtype)
    g = np.array([[v] for v in case["g"]], dtype=dtype)
    mom = np.zeros((3, 1), dtype=dtype)
    # float32 keeps 24 bits: values like 7/3 are rounded, a few ulps at most.
    tol = 1e-14 if dtype == np.float64 else 4e-7
    for r, (msgs, xs) in enumerate(case["rounds"]):
        o.round(x, g, mom if case["beta"] != 0 else None, float(case["lr"]), float(case["beta"]))
        got_m = [float(o.message(s, t)[0]) for s, t in EDGE_ORDER]
        np.testing.assert_allclose(got_m, [float(v) for v in msgs], rtol=tol, atol=tol)
        np.testing.assert_allclose(x[:, 0], [float(v) for v in xs], rtol=tol, atol=tol)
        if case["beta"] != 0:
            np.testing.assert_allclose(mom[:, 0], [float(v) for v in case["mom"][r]], rtol=0, atol=0)
        assert [o.count(s, t) for s, t in EDGE_ORDER] == list(HAND_COUNTS[r][0])
        assert list(o.nbars()) == list(HAND_COUNTS[r][1])


# --------------------------------------------------------------------------
# 2. Closed forms for counters: c_{i->j}^{(t)} counts the workers on i's side
#    of (i,j) within t hops of i; nbar_i^{(t+1)} counts workers within t+1 hops.
# --------------------------------------------------------------------------

TOPOLOGIES = {
    "chain4": wl.chain_edges(4),
    "heap16": wl.heap_edges(16),
    "chain16": wl.chain_edges(16),
    "star7": wl.star_edges(7, centre=3),
    "prufer40": wl.random_tree_edges(40, seed=3),
    "prufer256": wl.random_tree_edges(256, seed=0),
}


@pytest.mark.parametrize("name", list(TOPOLOGIES))
def test_counts_closed_form(name):
    edges = TOPOLOGIES[name]
    n = edges.shape[0] + 1
    tau = treeutil.hop_distances(n, edges)
    diam = int(tau.max())
    o = oracle.Oracle(n, 1, edges, dtype=np.float32)
    x = np.zeros((n, 1), np.float32)
    g = np.zeros((n, 1), np.float32)
    sides = {}
    for t in range(diam + 3):
        o.round(x, g, None, 0.0, 0.0)
        for u, v in edges:
            for i, j in ((int(u), int(v)), (int(v), int(u))):
                if (i, j) not in sides:
                    sides[(i, j)] = treeutil.side(n, edges, i, j)
                want = sum(1 for k in sides[(i, j)] if tau[i, k] <= t)
                assert o.count(i, j) == want, (t, i, j)
        nb = o.nbars()
        for i in range(n):
            assert nb[i] == treeutil.closed_form_nbar(tau, i, t)
        if t + 1 >= diam:
            # after diameter rounds every worker counts all n models
            assert (nb == n).all()
    assert o.count(0, 0) == -1


# --------------------------------------------------------------------------
# 3. The update is a uniform average of delayed half-steps and each message
#    is a sum of delayed half-steps over one side of its edge: exact check in
#    rational arithmetic on random data, and in double on the C oracle.
# --------------------------------------------------------------------------


def _random_rational(rng, shape):
    return np.array([F(int(v), 8) for v in rng.integers(-64, 65, size=int(np.prod(shape)))],
                    dtype=object).reshape(shape)


@pytest.mark.parametrize("name", ["chain4", "star7", "prufer40"])
def test_delayed_average_identity_exact(name):
    edges = TOPOLOGIES[name]
    n = edges.shape[0] + 1
    if n > 10:
        edges = wl.random_tree_edges(9, seed=11)
        n = 9
    tau = treeutil.hop_distances(n, edges)
    rng = np.random.default_rng(5)
    d = 2
    ex = ExactRelaySum(n, d, edges)
    x = _random_rational(rng, (n, d))
    lr = F(1, 4)
    hist = []
    for t in range(int(tau.max()) + 4):
        g = _random_rational(rng, (n, d))
        # plain SGD half-step of this round, the input the relay averages
        hist.append([x[k] - lr * g[k] for k in range(n)])
        x_new, _ = ex.round(x.tolist(), g.tolist(), None, lr, 0)
        x = np.array(x_new, dtype=object)
        for i in range(n):
            assert list(x[i]) == list(treeutil.delayed_average(tau, hist, i, t))
        for u, v in edges:
            for i, j in ((int(u), int(v)), (int(v), int(u))):
                want = treeutil.delayed_message(n, edges, tau, hist, i, j, t)
                assert list(ex.msg[(i, j)]) == list(want)


def test_delayed_average_identity_c_oracle_double():
    n, d = 24, 5
    edges = wl.random_tree_edges(n, seed=7)
    tau = treeutil.hop_distances(n, edges)
    rng = np.random.default_rng(1)
    o = oracle.Oracle(n, d, edges, dtype=np.float64)
    x = rng.standard_normal((n, d))
    mom = np.zeros((n, d))
    hist = []
    lr, beta = 0.05, 0.9
    buf = np.zeros((n, d))
    for t in range(int(tau.max()) + 5):
        g = rng.standard_normal((n, d))
        buf = beta * buf + g
        hist.append(x - lr * (g + beta * buf))
        o.round(x, g, mom, lr, beta)
        np.testing.assert_allclose(mom, buf, rtol=1e-15, atol=1e-15)
        for i in range(n):
            np.testing.assert_allclose(x[i], treeutil.delayed_average(tau, hist, i, t),
                                       rtol=1e-12, atol=1e-12)
        for u, v in edges[:6]:
            for i, j in ((int(u), int(v)), (int(v), int(u))):
                np.testing.assert_allclose(
                    o.message(i, j), treeutil.delayed_message(n, edges, tau, hist, i, j, t),
                    rtol=1e-12, atol=1e-12)


def test_delayed_average_identity_on_the_256_worker_tree():
    """The binary64 oracle on the Pruefer tree of the 256-worker workload
    (diameter 44) follows the delayed-average identity for every worker,
    every round, through the warm-up and past the diameter, with Nesterov
    momentum; the identity is evaluated here from the hop distances alone."""
    edges = wl.workload("prufer256").edges
    n, d = 256, 3
    tau = treeutil.hop_distances(n, edges)
    delta = np.maximum(tau - 1, 0)
    rng = np.random.default_rng(256)
    o = oracle.Oracle(n, d, edges, dtype=np.float64)
    x = rng.standard_normal((n, d))
    mom = np.zeros((n, d))
    buf = np.zeros((n, d))
    hist = []
    lr, beta = 0.05, 0.9
    workers = np.arange(n)
    for t in range(int(tau.max()) + 3):
        g = rng.standard_normal((n, d))
        buf = beta * buf + g
        hist.append(x - lr * (g + beta * buf))
        o.round(x, g, mom, lr, beta)
        h = np.array(hist)                       # [t+1, n, d]
        for i in range(n):
            arrived = delta[i] <= t
            want = h[t - delta[i][arrived], workers[arrived]].sum(axis=0) / arrived.sum()
            np.testing.assert_allclose(x[i], want, rtol=1e-11, atol=1e-11,
                                       err_msg=f"worker {i}, round {t}")
        assert (o.nbars() == (tau <= t + 1).sum(axis=1)).all(), f"nbar, round {t}"
    o.close()


@pytest.mark.parametrize("n", [2, 3, 4, 5, 6])
def test_every_labelled_tree_brute_force(n):
    """All n^(n-2) labelled trees: counts and averages against brute force."""
    rng = np.random.default_rng(n)
    d = 3
    for edges in wl.all_labelled_trees(n):
        tau = treeutil.hop_distances(n, edges)
        o = oracle.Oracle(n, d, edges, dtype=np.float64)
        x = rng.standard_normal((n, d))
        hist = []
        for t in range(int(tau.max()) + 2):
            g = rng.standard_normal((n, d))
            hist.append(x - 0.1 * g)
            o.round(x, g, None, 0.1, 0.0)
            for i in range(n):
                assert o.nbar(i) == treeutil.closed_form_nbar(tau, i, t)
                np.testing.assert_allclose(x[i], treeutil.delayed_average(tau, hist, i, t),
                                           rtol=1e-13, atol=1e-13)
        o.close()


# --------------------------------------------------------------------------
# 4. Special cases that reduce to textbook routines.
# --------------------------------------------------------------------------


def test_single_worker_is_torch_nesterov_sgd():
    """n = 1: no edges, nbar = 1, the round is one step of Nesterov SGD
    (App. D.2), which torch.optim.SGD(nesterov=True, dampening=0) implements."""
    import torch
    d = 257
    rng = np.random.default_rng(2)
    x0 = rng.standard_normal((1, d))
    o = oracle.Oracle(1, d, np.zeros((0, 2), np.int32), dtype=np.float64)
    x = x0.copy()
    mom = np.zeros((1, d))
    p = torch.nn.Parameter(torch.tensor(x0, dtype=torch.float64))
    opt = torch.optim.SGD([p], lr=0.03, momentum=0.9, dampening=0.0, nesterov=True)
    for t in range(30):
        g = rng.standard_normal((1, d))
        o.round(x, g, mom, 0.03, 0.9)
        p.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        assert o.nbar(0) == 1
        np.testing.assert_allclose(x, p.detach().numpy(), rtol=1e-12, atol=1e-13)


def test_single_worker_plain_sgd_float32_is_exact():
    """n = 1 without momentum: x - lr*g rounded once, then divided by 1."""
    d = 1000
    rng = np.random.default_rng(3)
    x = rng.standard_normal((1, d)).astype(np.float32)
    g = rng.standard_normal((1, d)).astype(np.float32)
    want = (x - np.float32(0.1) * g).astype(np.float32)
    o = oracle.Oracle(1, d, np.zeros((0, 2), np.int32), dtype=np.float32)
    o.round(x, g, None, 0.1, 0.0)
    assert np.array_equal(x, want)


def test_two_workers_is_allreduce():
    """n = 2: both workers hold the exact mean of the two half-steps after
    every round, including the first (the all-reduce average of Section 3)."""
    edges = np.array([[1, 0]], np.int32)
    rng = np.random.default_rng(4)
    ex = ExactRelaySum(2, 2, edges)
    x = _random_rational(rng, (2, 2))
    for t in range(6):
        g = _random_rational(rng, (2, 2))
        xh = [x[k] - F(1, 2) * g[k] for k in range(2)]
        x_new, _ = ex.round(x.tolist(), g.tolist(), None, F(1, 2), 0)
        x = np.array(x_new, dtype=object)
        mean = (xh[0] + xh[1]) / 2
        assert list(x[0]) == list(mean) and list(x[1]) == list(mean)


def test_star_centre_holds_exact_mean():
    """Star: the centre is one hop from everyone, so after each round it holds
    the mean of all current half-steps."""
    n = 6
    edges = wl.star_edges(n, centre=2)
    rng = np.random.default_rng(6)
    ex = ExactRelaySum(n, 1, edges)
    x = _random_rational(rng, (n, 1))
    for t in range(4):
        g = _random_rational(rng, (n, 1))
        xh = [x[k] - F(1, 3) * g[k] for k in range(n)]
        x_new, _ = ex.round(x.tolist(), g.tolist(), None, F(1, 3), 0)
        x = np.array(x_new, dtype=object)
        assert x[2][0] == sum(v[0] for v in xh) / n


def test_identical_workers_first_round_is_single_worker_step():
    """Identical x0 and gradients on every worker: after round 0 every worker
    holds the one-worker Nesterov step (all messages carry the same half-step
    and nbar counts them).  From round 1 on the average mixes half-steps of
    different ages (delays max(tau-1, 0)), so the workers leave the
    one-worker trajectory: the second check pins that too."""
    edges = wl.random_tree_edges(7, seed=2)
    rng = np.random.default_rng(8)
    ex = ExactRelaySum(7, 2, edges)
    single = ExactRelaySum(1, 2, np.zeros((0, 2), np.int32))
    row = _random_rational(rng, (1, 2))
    x = [list(row[0]) for _ in range(7)]
    mom = [[F(0), F(0)] for _ in range(7)]
    xs, ms = [list(row[0])], [[F(0), F(0)]]
    grow = _random_rational(rng, (1, 2))
    x, mom = ex.round(x, [list(grow[0])] * 7, mom, F(1, 5), F(3, 4))
    xs, ms = single.round(xs, [list(grow[0])], ms, F(1, 5), F(3, 4))
    for i in range(7):
        assert x[i] == xs[0] and mom[i] == ms[0]
    grow = _random_rational(rng, (1, 2))
    x, mom = ex.round(x, [list(grow[0])] * 7, mom, F(1, 5), F(3, 4))
    xs, ms = single.round(xs, [list(grow[0])], ms, F(1, 5), F(3, 4))
    leaf = next(i for i in range(7) if len(ex.nb[i]) == 1 and
                sum(len(ex.nb[j]) for j in ex.nb[i]) > 1)
    assert x[leaf] != xs[0]
    assert mom[leaf] == ms[0]


def test_constant_models_stay_constant_float32():
    """Row-stochastic averaging: lr = 0 and equal models leave every model
    unchanged, bit for bit (1.25*k/k is exact in binary32 for small k)."""
    edges = wl.random_tree_edges(50, seed=9)
    o = oracle.Oracle(50, 33, edges, dtype=np.float32)
    x = np.full((50, 33), 1.25, np.float32)
    g = np.random.default_rng(0).standard_normal((50, 33)).astype(np.float32)
    mom = np.zeros((50, 33), np.float32)
    for _ in range(20):
        o.round(x, g, mom, 0.0, 0.9)
        assert (x == np.float32(1.25)).all()


def test_identical_x0_lr0_is_stable_float32():
    """Identical x0 and lr = 0: exactly stable in rationals; in binary32 the
    drift after 50 rounds stays at the rounding level."""
    edges = wl.chain_edges(16)
    d = 4096
    row = np.random.default_rng(1).standard_normal((1, d)).astype(np.float32) * np.float32(0.01)
    x = np.repeat(row, 16, axis=0)
    o = oracle.Oracle(16, d, edges, dtype=np.float32)
    g = np.zeros((16, d), np.float32)
    for _ in range(50):
        o.round(x, g, None, 0.0, 0.0)
    rel = np.abs(x - row).max() / np.abs(row).max()
    assert rel < 1e-6


# --------------------------------------------------------------------------
# 5. Cross-precision: the float32 oracle against the float64 one.
# --------------------------------------------------------------------------


def test_float32_one_round_within_rounding_of_float64():
    """One round from binary32 inputs: each binary32 result differs from the
    double result by at most the rounding of its few operations, i.e. a few
    units of 2^-24 relative to the largest magnitude that enters it."""
    n, d = 64, 2000
    edges = wl.random_tree_edges(n, seed=4)
    rng = np.random.default_rng(10)
    x32 = rng.standard_normal((n, d)).astype(np.float32)
    g32 = rng.standard_normal((n, d)).astype(np.float32)
    m32 = rng.standard_normal((n, d)).astype(np.float32)
    x64, g64, m64 = x32.astype(np.float64), g32.astype(np.float64), m32.astype(np.float64)
    o32 = oracle.Oracle(n, d, edges, np.float32)
    o64 = oracle.Oracle(n, d, edges, np.float64)
    o32.round(x32, g32, m32, 0.05, 0.9)
    o64.round(x64, g64, m64, 0.05, 0.9)
    # mom: two ops on values of size ~|m|+|g|
    assert np.abs(m32 - m64).max() <= 2 * 2.0 ** -24 * np.abs(m64).max() * 2
    scale = max(np.abs(x64).max(), 1.0) * (1 + max(len(a) for a in _nbrs(n, edges)))
    assert np.abs(x32 - x64).max() <= 16 * 2.0 ** -24 * scale


def _nbrs(n, edges):
    return [sorted(s) for s in treeutil.adjacency(n, edges)]


def test_float32_many_rounds_close_to_float64():
    """300 rounds on a 64-worker random tree: binary32 stays within 1e-5 of
    double, max-norm relative per worker (rounding only; a wrong term would
    be off by O(1))."""
    n, d = 64, 500
    edges = wl.random_tree_edges(n, seed=5)
    rng = np.random.default_rng(11)
    x64 = rng.standard_normal((n, d))
    x32 = x64.astype(np.float32)
    x64 = x32.astype(np.float64)
    m32 = np.zeros((n, d), np.float32)
    m64 = np.zeros((n, d))
    o32 = oracle.Oracle(n, d, edges, np.float32)
    o64 = oracle.Oracle(n, d, edges, np.float64)
    for t in range(300):
        g32 = rng.standard_normal((n, d)).astype(np.float32)
        lr = 0.0 if t < 200 else 0.01
        o32.round(x32, g32, m32, lr, 0.9)
        o64.round(x64, g32.astype(np.float64), m64, lr, 0.9)
    err = np.abs(x32 - x64).max(axis=1) / np.abs(x64).max(axis=1)
    assert err.max() < 1e-5


def test_oracle_rejects_non_trees():
    with pytest.raises(ValueError):
        oracle.Oracle(3, 1, [[0, 1], [1, 0]])            # duplicate
    with pytest.raises(ValueError):
        oracle.Oracle(4, 1, [[0, 1], [1, 2], [2, 0]])    # cycle, 3 ≠ n-1 ... disconnected
    with pytest.raises(ValueError):
        oracle.Oracle(3, 1, [[0, 0], [1, 2]])            # self loop
    with pytest.raises(ValueError):
        oracle.Oracle(3, 1, [[0, 3], [1, 2]])            # out of range
    with pytest.raises(ValueError):
        oracle.Oracle(3, 1, [[0, 1]])                    # too few edges


def test_oracle_threads_do_not_change_results():
    n, d = 16, 300_000
    edges = wl.heap_edges(n)
    rng = np.random.default_rng(12)
    x0 = rng.standard_normal((n, d)).astype(np.float32)
    g = rng.standard_normal((n, d)).astype(np.float32)
    outs = []
    before = oracle.get_threads()
    for k in (1, 4):
        oracle.set_threads(k)
        o = oracle.Oracle(n, d, edges, np.float32)
        x = x0.copy()
        mom = np.zeros_like(x)
        for _ in range(3):
            o.round(x, g, mom, 0.05, 0.9)
        outs.append((x, mom))
    oracle.set_threads(before)
    assert np.array_equal(outs[0][0], outs[1][0]) and np.array_equal(outs[0][1], outs[1][1])
