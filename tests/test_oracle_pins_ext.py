"""Pins of the extended oracle round (CPU only): the robust update and lost
messages (Section 5.4, eq. robust), RelaySGD/Grad (Alg. 4), RelaySum for
mean estimation (Alg. 3) and the Adam local step (App. D.3).

The independent reference is parcel routing: every quantity a worker puts
into the relay is followed hop by hop along its tree path, one hop per round,
and is lost with any lost message on the way (tests/treeutil.arrivals).
"""
from fractions import Fraction as F

import numpy as np
import pytest
import torch

import oracle
import treeutil
import workloads as wl


def _drops(rng, n, edges, rounds, p):
    """Random lost messages: {round: {(src, dst), ...}} with probability p each."""
    out = {}
    for r in range(rounds):
        lost = set()
        for u, v in np.asarray(edges).reshape(-1, 2):
            for a, b in ((int(u), int(v)), (int(v), int(u))):
                if rng.random() < p:
                    lost.add((a, b))
        out[r] = lost
    return out


def _mask(n, lost):
    m = np.zeros((n, n), np.uint8)
    for a, b in lost:
        m[a, b] = 1
    return m


def test_round_ex_model_equals_round_bit_for_bit():
    n, d = 20, 777
    edges = wl.random_tree_edges(n, seed=2)
    rng = np.random.default_rng(0)
    x0 = rng.standard_normal((n, d)).astype(np.float32)
    a, b = oracle.Oracle(n, d, edges), oracle.Oracle(n, d, edges)
    xa, xb = x0.copy(), x0.copy()
    ma, mb = np.zeros_like(x0), np.zeros_like(x0)
    for t in range(12):
        g = rng.standard_normal((n, d)).astype(np.float32)
        a.round(xa, g, ma, 0.05, 0.9)
        b.round_ex(xb, g, mb, update="model", lr=0.05, beta1=0.9)
        assert np.array_equal(xa.view(np.uint32), xb.view(np.uint32))
        assert np.array_equal(ma.view(np.uint32), mb.view(np.uint32))
        assert list(a.nbars()) == list(b.nbars())


@pytest.mark.parametrize("update", ["model", "robust"])
@pytest.mark.parametrize("p_drop", [0.0, 0.1, 0.4])
def test_lost_messages_match_parcel_routing(update, p_drop):
    """Model and robust updates with lost messages against parcel routing:
    x_i = (sum of arrived half-steps) / #arrived, or, robust,
    (sum of arrived + (n - #arrived) x_i^(t)) / n; nbar_i = #arrived."""
    n, d, rounds = 9, 3, 12
    edges = wl.random_tree_edges(n, seed=5)
    rng = np.random.default_rng(int(p_drop * 100) + (update == "robust"))
    drops = _drops(rng, n, edges, rounds, p_drop)
    o = oracle.Oracle(n, d, edges, np.float64)
    x = rng.standard_normal((n, d))
    hist = []
    for t in range(rounds):
        g = rng.standard_normal((n, d))
        x_old = x.copy()
        hist.append(x - 0.1 * g)          # plain SGD half-steps of round t
        o.round_ex(x, g, update=update, lr=0.1, dropped=_mask(n, drops[t]))
        for i in range(n):
            arr = treeutil.arrivals(n, edges, i, t, drops)
            tot = sum(hist[s][k] for k, s in arr)
            assert o.nbar(i) == len(arr)
            if update == "model":
                want = tot / len(arr)
            else:
                want = (tot + (n - len(arr)) * x_old[i]) / n
            np.testing.assert_allclose(x[i], want, rtol=1e-12, atol=1e-12)


def test_lost_message_counters_match_parcel_routing():
    n, rounds = 10, 14
    edges = wl.random_tree_edges(n, seed=8)
    rng = np.random.default_rng(3)
    drops = _drops(rng, n, edges, rounds, 0.2)
    o = oracle.Oracle(n, 1, edges, np.float64)
    x = np.zeros((n, 1))
    g = np.zeros((n, 1))
    for t in range(rounds):
        o.round_ex(x, g, update="model", dropped=_mask(n, drops[t]))
        for u, v in edges:
            for i, j in ((int(u), int(v)), (int(v), int(u))):
                if (i, j) in drops[t]:
                    assert o.count(i, j) == 0
                    continue
                # parcels that cross i -> j in round t: those reaching j in
                # round t from workers on i's side of the edge
                side = treeutil.side(n, edges, i, j)
                arr = treeutil.arrivals(n, edges, j, t, drops)
                want = sum(1 for k, _ in arr if k in side)
                assert o.count(i, j) == want, (t, i, j)


def test_robust_without_losses_equals_alg1_once_counters_saturate():
    n, d = 16, 500
    edges = wl.heap_edges(n)
    diam = treeutil.diameter(n, edges)
    rng = np.random.default_rng(4)
    x0 = rng.standard_normal((n, d)).astype(np.float32)
    a, b = oracle.Oracle(n, d, edges), oracle.Oracle(n, d, edges)
    xa, xb = x0.copy(), x0.copy()
    ma, mb = np.zeros_like(x0), np.zeros_like(x0)
    for t in range(diam + 6):
        g = rng.standard_normal((n, d)).astype(np.float32)
        a.round_ex(xa, g, ma, update="model", lr=0.05, beta1=0.9)
        b.round_ex(xb, g, mb, update="robust", lr=0.05, beta1=0.9)
        if t + 1 >= diam:
            assert (a.nbars() == n).all()
            # saturated: both copies restart from identical models
            xb[:] = xa
    # one more round from equal state: (acc + 0*x)/n == acc/n bit for bit
    g = rng.standard_normal((n, d)).astype(np.float32)
    a.round_ex(xa, g, ma, update="model", lr=0.05, beta1=0.9)
    b.round_ex(xb, g, mb, update="robust", lr=0.05, beta1=0.9)
    assert np.array_equal(xa.view(np.uint32), xb.view(np.uint32))


def test_robust_keeps_constant_models_constant_with_losses():
    """Missing models are replaced by x_i^(t): with equal models and lr = 0 the
    robust update returns them unchanged even when messages are lost."""
    n, d = 12, 40
    edges = wl.random_tree_edges(n, seed=6)
    rng = np.random.default_rng(7)
    drops = _drops(rng, n, edges, 10, 0.3)
    o = oracle.Oracle(n, d, edges, np.float32)
    x = np.full((n, d), 0.75, np.float32)
    g = rng.standard_normal((n, d)).astype(np.float32)
    for t in range(10):
        o.round_ex(x, g, update="robust", lr=0.0, dropped=_mask(n, drops[t]))
        assert (x == np.float32(0.75)).all()


def test_grad_relay_matches_parcel_routing_and_spreads_exactly():
    """Alg. 4: x_i gains (1/n) of every update that reaches it; after the
    diameter, with no new updates, every worker holds x0 + (1/n) * (sum of all
    updates), exactly (rational arithmetic)."""
    n, d = 7, 2
    edges = wl.random_tree_edges(n, seed=9)
    diam = treeutil.diameter(n, edges)
    rng = np.random.default_rng(10)
    o = oracle.Oracle(n, d, edges, np.float64)
    x0 = rng.integers(-8, 9, (n, d)).astype(np.float64)
    x = x0.copy()
    ups = []
    for t in range(6 + diam):
        g = rng.integers(-8, 9, (n, d)).astype(np.float64) if t < 6 else np.zeros((n, d))
        ups.append(-0.25 * g)
        x_before = x.copy()
        o.round_ex(x, g, update="grad", lr=0.25)
        for i in range(n):
            arr = treeutil.arrivals(n, edges, i, t, {})
            want = x_before[i] + sum(ups[s][k] for k, s in arr) / n
            np.testing.assert_allclose(x[i], want, rtol=1e-13, atol=1e-13)
    total = sum(ups)                       # [n, d], summed over rounds
    # every worker received every update: x_i = x0_i + (1/n) sum_k sum_s u_k^(s)
    np.testing.assert_allclose(x, x0 + total.sum(axis=0)[None] / n, rtol=0, atol=1e-12)


def test_mean_estimation_matches_parcel_routing():
    """Alg. 3: y_i sums every sample that has reached i, s_i counts them,
    x_i = y_i / s_i; with constant samples the estimate is exact."""
    n, d, rounds = 8, 3, 10
    edges = wl.random_tree_edges(n, seed=12)
    rng = np.random.default_rng(13)
    o = oracle.Oracle(n, d, edges, np.float64)
    x = np.zeros((n, d))
    y = np.zeros((n, d))
    samples = []
    for t in range(rounds):
        smp = rng.standard_normal((n, d))
        samples.append(smp)
        o.round_ex(x, smp, y, update="mean")
        for i in range(n):
            got = []
            for r in range(t + 1):
                got += treeutil.arrivals(n, edges, i, r, {})
            tot = sum(samples[s][k] for k, s in got)
            assert o.samples(i) == len(got)
            np.testing.assert_allclose(y[i], tot, rtol=1e-12, atol=1e-12)
            np.testing.assert_allclose(x[i], tot / len(got), rtol=1e-12, atol=1e-12)
    o2 = oracle.Oracle(n, d, edges, np.float32)
    x = np.zeros((n, d), np.float32)
    y = np.zeros((n, d), np.float32)
    c = np.full((n, d), 1.5, np.float32)
    for t in range(6):
        o2.round_ex(x, c, y, update="mean")
        assert (x == np.float32(1.5)).all()


def test_single_worker_adam_is_torch_adam():
    """n = 1: the round is one step of PyTorch's Adam (App. D.3)."""
    d = 301
    rng = np.random.default_rng(14)
    x0 = rng.standard_normal((1, d))
    o = oracle.Oracle(1, d, np.zeros((0, 2), np.int32), np.float64)
    x = x0.copy()
    m, v = np.zeros((1, d)), np.zeros((1, d))
    p = torch.nn.Parameter(torch.tensor(x0, dtype=torch.float64))
    opt = torch.optim.Adam([p], lr=1e-3, betas=(0.9, 0.999), eps=1e-8)
    for t in range(1, 41):
        g = rng.standard_normal((1, d))
        o.round_ex(x, g, m, v, update="model", optimizer="adam", lr=1e-3, beta1=0.9,
                   beta2=0.999, eps=1e-8, adam_step=t)
        p.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        np.testing.assert_allclose(x, p.detach().numpy(), rtol=1e-12, atol=1e-14)
        st = opt.state[p]
        np.testing.assert_allclose(m, st["exp_avg"].numpy(), rtol=1e-12, atol=1e-15)
        np.testing.assert_allclose(v, st["exp_avg_sq"].numpy(), rtol=1e-12, atol=1e-15)


def test_adam_state_is_local_and_relay_unchanged():
    """Relay-Adam: every worker's Adam state evolves as torch's on its own
    gradients, and the models follow the delayed-average identity of Alg. 1
    applied to the Adam half-steps."""
    n, d = 5, 4
    edges = wl.chain_edges(n)
    tau = treeutil.hop_distances(n, edges)
    rng = np.random.default_rng(15)
    o = oracle.Oracle(n, d, edges, np.float64)
    x = rng.standard_normal((n, d))
    m, v = np.zeros((n, d)), np.zeros((n, d))
    ps = [torch.zeros(d, dtype=torch.float64, requires_grad=True) for _ in range(n)]
    opts = [torch.optim.Adam([p], lr=0.01, betas=(0.8, 0.99), eps=1e-6) for p in ps]
    hist = []
    for t in range(1, 9):
        g = rng.standard_normal((n, d))
        half = np.empty((n, d))
        for i in range(n):
            with torch.no_grad():
                ps[i].copy_(torch.tensor(x[i]))
            ps[i].grad = torch.tensor(g[i])
            opts[i].step()
            half[i] = ps[i].detach().numpy()
        hist.append(half)
        o.round_ex(x, g, m, v, update="model", optimizer="adam", lr=0.01, beta1=0.8,
                   beta2=0.99, eps=1e-6, adam_step=t)
        for i in range(n):
            np.testing.assert_allclose(m[i], opts[i].state[ps[i]]["exp_avg"].numpy(), rtol=1e-12)
            np.testing.assert_allclose(x[i], treeutil.delayed_average(tau, hist, i, t - 1),
                                       rtol=1e-11, atol=1e-12)


def test_double_trees_with_one_tree_twice_equal_single_tree():
    """Section 3's double binary trees split the coordinates by parity; with
    the same tree as A and B the round is the single-tree round, bit for bit."""
    from oracle.double import DoubleOracle
    n, d = 11, 301
    edges = wl.random_tree_edges(n, seed=21)
    rng = np.random.default_rng(22)
    x0 = rng.standard_normal((n, d)).astype(np.float32)
    one = oracle.Oracle(n, d, edges)
    two = DoubleOracle(n, d, edges, edges)
    xa, xb = x0.copy(), x0.copy()
    ma, mb = np.zeros_like(x0), np.zeros_like(x0)
    for t in range(8):
        g = rng.standard_normal((n, d)).astype(np.float32)
        one.round_ex(xa, g, ma, update="robust", lr=0.05, beta1=0.9)
        two.round_ex(xb, g, mb, update="robust", lr=0.05, beta1=0.9)
        assert np.array_equal(xa.view(np.uint32), xb.view(np.uint32))
        assert np.array_equal(ma.view(np.uint32), mb.view(np.uint32))


def test_double_trees_each_parity_is_the_delayed_average_on_its_tree():
    """Two different trees (Section 3): odd coordinates are the uniform
    average of half-steps delayed by tree A's hop distances, even ones by
    tree B's (fp64, Nesterov momentum).  A swapped parity, a swapped tree or
    a coordinate relayed on both trees fails it."""
    from oracle.double import DoubleOracle
    n, d = 12, 7
    ea, eb = wl.double_binary_tree_edges(n)
    ta, tb = treeutil.hop_distances(n, ea), treeutil.hop_distances(n, eb)
    assert not np.array_equal(ta, tb)
    rng = np.random.default_rng(31)
    o = DoubleOracle(n, d, ea, eb, np.float64)
    x = rng.standard_normal((n, d))
    mom = np.zeros((n, d))
    buf = np.zeros((n, d))
    lr, beta = 0.05, 0.9
    hist = []
    for t in range(int(max(ta.max(), tb.max())) + 4):
        g = rng.standard_normal((n, d))
        buf = beta * buf + g
        hist.append(x - lr * (g + beta * buf))
        o.round(x, g, mom, lr, beta)
        np.testing.assert_allclose(mom, buf, rtol=1e-15, atol=1e-15)
        for i in range(n):
            want_a = treeutil.delayed_average(ta, hist, i, t)
            want_b = treeutil.delayed_average(tb, hist, i, t)
            np.testing.assert_allclose(x[i, 1::2], want_a[1::2], rtol=1e-12, atol=1e-12)
            np.testing.assert_allclose(x[i, 0::2], want_b[0::2], rtol=1e-12, atol=1e-12)
    o.close()


def test_double_trees_counters_follow_each_tree():
    from oracle.double import DoubleOracle
    n = 16
    ea, eb = wl.double_binary_tree_edges(n)
    o = DoubleOracle(n, 6, ea, eb, np.float64)
    x = np.zeros((n, 6))
    g = np.zeros((n, 6))
    ta, tb = treeutil.hop_distances(n, ea), treeutil.hop_distances(n, eb)
    for t in range(8):
        o.round(x, g, None, 0.0, 0.0)
        for i in range(n):
            assert o.a.nbar(i) == treeutil.closed_form_nbar(ta, i, t)
            assert o.b.nbar(i) == treeutil.closed_form_nbar(tb, i, t)


@pytest.mark.parametrize("update,optimizer,kw", [
    ("robust", "adam", dict(lr=1e-2, beta1=0.9, beta2=0.999, eps=1e-8)),
    ("grad", "sgd", dict(lr=0.1)),
    ("mean", "sgd", dict()),
])
def test_extended_round_threads_do_not_change_results(update, optimizer, kw):
    """The extended round is parallel over coordinates only: 1 and 4 threads
    give the same bits, with lost messages."""
    n, d = 10, 200_000
    edges = wl.random_tree_edges(n, seed=21)
    rng = np.random.default_rng(22)
    x0 = rng.standard_normal((n, d)).astype(np.float32)
    g = rng.standard_normal((n, d)).astype(np.float32)
    masks = [(rng.random((n, n)) < 0.2).astype(np.uint8) for _ in range(3)]
    outs = []
    before = oracle.get_threads()
    for k in (1, 4):
        oracle.set_threads(k)
        o = oracle.Oracle(n, d, edges, np.float32)
        x = x0.copy()
        s1, s2 = np.zeros_like(x), np.zeros_like(x)
        for t in range(3):
            o.round_ex(x, g, s1, s2, update=update, optimizer=optimizer, adam_step=t + 1,
                       dropped=masks[t], **kw)
        outs.append((x, s1, s2))
        o.close()
    oracle.set_threads(before)
    for a, b in zip(*outs):
        assert np.array_equal(a, b)


def round_to_float32(q):
    """The binary32 number nearest to the rational q >= 0 (ties to even), by
    integer arithmetic: q = m * 2^e with 2^23 <= m < 2^24 rounded to an
    integer m."""
    if q == 0:
        return np.float32(0.0)
    e = q.numerator.bit_length() - q.denominator.bit_length() - 24
    while q / F(2) ** e >= 2 ** 24:
        e += 1
    while q / F(2) ** e < 2 ** 23:
        e -= 1
    m = q / F(2) ** e
    r = m.numerator // m.denominator
    rem = m - r
    if rem > F(1, 2) or (rem == F(1, 2) and r % 2 == 1):
        r += 1
    return np.float32(np.ldexp(np.float64(r), e))   # exact: r has at most 25 bits


def chain_sample_counts(n, rounds):
    """s_i of Alg. 3 on a chain after `rounds` rounds without losses: round t
    adds nbar_i = 1 + min(i, t+1) + min(n-1-i, t+1), the workers within t+1
    hops."""
    i = np.arange(n, dtype=np.int64)
    s = np.zeros(n, np.int64)
    for t in range(rounds):
        s += 1 + np.minimum(i, t + 1) + np.minimum(n - 1 - i, t + 1)
    return s


def test_round_to_float32_pins():
    assert round_to_float32(F(1, 3)) == np.float32(1) / np.float32(3)
    assert round_to_float32(F(2 ** 24 + 1)) == np.float32(2 ** 24)        # tie to even
    assert round_to_float32(F(2 ** 24 + 3)) == np.float32(2 ** 24 + 4)    # tie to even
    assert round_to_float32(F(7, 10)) == np.float32(0.7)


def test_mean_estimation_divides_exactly_up_to_two_to_the_24():
    """Alg. 3 with sample counts just under 2^24 (a chain of 1024 workers,
    16,639 rounds): s_i follows the hop-distance closed form, and with 0/1
    samples (y_i an integer, exact in binary32 while it stays at most s_i)
    the binary32 estimate is exactly y_i / s_i rounded once, i.e. the integer
    divisor converts exactly.  16,639 is the last round count whose bound of
    the sample counts, the sum over rounds t of min(n, 1 + 2(t+1)) (the
    workers within t+1 hops on a tree of degree 2), stays within 2^24."""
    n, d = 1024, 2
    rounds, bound = 0, 0
    while bound + min(n, 1 + 2 * (rounds + 1)) <= 1 << 24:
        bound += min(n, 1 + 2 * (rounds + 1))
        rounds += 1
    assert rounds == 16639 and bound == (1 << 24) - 1
    rng = np.random.default_rng(24)
    g = rng.integers(0, 2, (n, d)).astype(np.float32)
    o = oracle.Oracle(n, d, wl.chain_edges(n), np.float32)
    x = np.zeros((n, d), np.float32)
    y = np.zeros((n, d), np.float32)
    for t in range(rounds):
        o.round_ex(x, g, y, update="mean")
    s = np.array([o.samples(i) for i in range(n)], np.int64)
    o.close()
    assert np.array_equal(s, chain_sample_counts(n, rounds))
    assert (1 << 24) - 2048 < s.max() <= 1 << 24
    assert np.array_equal(y, np.floor(y)) and (y <= s[:, None]).all()
    for i in range(0, n, 37):
        for c in range(d):
            want = round_to_float32(F(int(y[i, c]), int(s[i])))
            assert x[i, c] == want, (i, c)
