"""Seeded random sweep over the combinations the dispatch has to get right:
tree size (tile kernel up to 32 workers; cluster and double-tree kernels
from 33, stars behind a hub kernel; the two-pass path for double trees
beyond their kernels' ranges; and a band of 330-4096 workers, where single
trees take the cluster kernels, brooms with a hub of 13 among them behind a
hub kernel),
single or double binary trees, 16-byte or 4-byte aligned rows, d of any
residue, every update rule and local optimizer, with and without lost
messages.  Every case is compared with the oracle bit for bit, every round
(100 seeded cases, plus 20 in the large band and 16 preferential-attachment
trees of 33 to 3,000 workers with hubs), and the sweep as a whole must
reach every kernel path the library still takes."""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2110_04175_amd as rs
from oracle.double import DoubleOracle
import workloads as wl
from parity import assert_params_close, bit_mismatches

pytestmark = pytest.mark.gpu

RULES = [
    ("model", "sgd", dict(lr=0.1)),
    ("model", "sgd", dict(lr=0.1, beta1=0.9)),
    ("model", "adam", dict(lr=1e-2, beta1=0.9, beta2=0.999, eps=1e-8)),
    ("robust", "sgd", dict(lr=0.1, beta1=0.5)),
    ("robust", "adam", dict(lr=1e-2, beta1=0.8, beta2=0.99, eps=1e-6)),
    ("grad", "sgd", dict(lr=0.2)),
    ("mean", "sgd", dict()),
]


def _cases(count=100, seed=2110):
    rng = np.random.default_rng(seed)
    out = []
    for k in range(count):
        band = rng.integers(0, 4)
        n = int([rng.integers(1, 33), rng.integers(33, 130), rng.integers(130, 257),
                 rng.integers(257, 330)][band])
        double = bool(rng.random() < 0.35) and n >= 2 and n <= 140
        d = int(rng.choice([1, 2, 3, 5, 63, 64, 255, 256, 257, 511, 512, 513, 1024, 1500, 2052]))
        offset = int(rng.choice([0, 0, 1, 2]))
        rule = int(rng.integers(0, len(RULES)))
        p_drop = float(rng.choice([0.0, 0.0, 0.2]))
        topo = str(rng.choice(["random", "chain", "heap", "star"]))
        out.append((k, n, d, offset, double, rule, p_drop, topo))
    return out


CASES = _cases()


def _large_cases(count=20, seed=4175):
    """Single trees of 330 to 4096 workers with short models (the oracle's
    cost grows with n * d)."""
    rng = np.random.default_rng(seed)
    out = []
    for k in range(count):
        n = int(rng.integers(330, 4097))
        d = int(rng.choice([1, 3, 4, 61, 128, 257, 300]))
        offset = int(rng.choice([0, 0, 1]))
        rule = int(rng.integers(0, len(RULES)))
        p_drop = float(rng.choice([0.0, 0.2]))
        topo = str(rng.choice(["random", "random", "chain", "heap", "broom"]))
        out.append((100 + k, n, d, offset, False, rule, p_drop, topo))
    return out


LARGE = _large_cases()


def _hub_cases(count=16, seed=2021):
    """Preferential-attachment trees of 33 to 3,000 workers: workers of 9 to
    about 70 neighbours go through every class of hub kernel ahead of the
    cluster kernel."""
    rng = np.random.default_rng(seed)
    out = []
    for k in range(count):
        n = int(rng.integers(33, 3001))
        d = int(rng.choice([1, 3, 4, 61, 128, 257, 300]))
        offset = int(rng.choice([0, 0, 1]))
        rule = int(rng.integers(0, len(RULES)))
        p_drop = float(rng.choice([0.0, 0.2]))
        out.append((200 + k, n, d, offset, False, rule, p_drop, "pa"))
    return out


HUBS = _hub_cases()


def _edges(topo, n, seed):
    if topo == "chain":
        return wl.chain_edges(n)
    if topo == "heap":
        return wl.heap_edges(n)
    if topo == "star":
        return wl.star_edges(n)
    if topo == "broom":
        return wl.broom_edges(n)
    if topo == "pa":
        return wl.preferential_attachment_edges(n, seed)
    return wl.random_tree_edges(n, seed=seed)


def _pair(k, n):
    """Every third double case pairs a star with a chain (a hub of n - 1
    neighbours: the double-tree or sequential double-tree kernel up to 64
    workers, the per-tree two-pass path beyond);
    the others are the paper's double binary trees."""
    if k % 3 == 0 and n > 2:
        return wl.star_edges(n), wl.chain_edges(n)
    return wl.double_binary_tree_edges(n)


def test_sweep_reaches_every_kernel_path():
    paths = set()
    for k, n, d, offset, double, rule, p_drop, topo in CASES + LARGE + HUBS:
        if double:
            ea, eb = _pair(k, n)
            h = rs.RelaySum(n, d, ea, edges_b=eb)
        else:
            h = rs.RelaySum(n, d, _edges(topo, n, seed=k))
        paths.add(h.path)
        h.close()
    assert paths == set(rs.PATHS) - set(rs.RETIRED_PATHS), sorted(paths)


@pytest.mark.parametrize("k,n,d,offset,double,rule,p_drop,topo", CASES + LARGE + HUBS,
                         ids=[f"case{c[0]}" for c in CASES + LARGE + HUBS])
def test_random_case(k, n, d, offset, double, rule, p_drop, topo):
    update, optimizer, kw = RULES[rule]
    sys.__stderr__.write(f"[gpu] random case {k}: n={n} d={d} offset={offset} double={double} "
                         f"{update}/{optimizer} p_drop={p_drop} {topo}\n")
    sys.__stderr__.flush()
    rng = np.random.default_rng(1000 + k)
    if double:
        ea, eb = _pair(k, n)
        o = DoubleOracle(n, d, ea, eb, np.float32)
        h = rs.RelaySum(n, d, ea, edges_b=eb)
        e2a = 2 * (n - 1)
    else:
        edges = _edges(topo, n, seed=k)
        o = oracle.Oracle(n, d, edges, np.float32)
        h = rs.RelaySum(n, d, edges)
    slots = [h.directed_edge(s) for s in range(h.num_directed_edges)]
    dev = torch.device("cuda")
    uses_s1 = optimizer == "adam" or kw.get("beta1", 0.0) != 0.0 or update == "mean"
    uses_s2 = optimizer == "adam"
    x0 = rng.standard_normal((n, d)).astype(np.float32)
    if update == "mean":
        x0[:] = 0

    def dev_buf(arr):
        b = torch.zeros(n * d + offset, dtype=torch.float32, device=dev)
        v = b[offset:].view(n, d)
        v.copy_(torch.from_numpy(arr))
        return b, v

    bx, x = dev_buf(x0)
    b1, s1 = dev_buf(np.zeros_like(x0)) if uses_s1 else (None, None)
    b2, s2 = dev_buf(np.zeros_like(x0)) if uses_s2 else (None, None)
    xo = x0.copy()
    o1 = np.zeros_like(x0) if uses_s1 else None
    o2 = np.zeros_like(x0) if uses_s2 else None
    rounds = 6
    for t in range(rounds):
        g = rng.standard_normal((n, d)).astype(np.float32)
        bg, gd = dev_buf(g)
        drop_dev, okw = None, {}
        if p_drop:
            if double:
                ma = (rng.random((n, n)) < p_drop).astype(np.uint8)
                mb = (rng.random((n, n)) < p_drop).astype(np.uint8)
                per = [(ma if s < e2a else mb)[i, j] for s, (i, j) in enumerate(slots)]
                okw = dict(dropped_a=ma, dropped_b=mb)
            else:
                m = (rng.random((n, n)) < p_drop).astype(np.uint8)
                per = [m[i, j] for i, j in slots]
                okw = dict(dropped=m)
            if per:
                drop_dev = torch.tensor(per, dtype=torch.uint8, device=dev)
        else:
            okw = dict(dropped_a=None, dropped_b=None) if double else dict(dropped=None)
        rs.relaysum_step_ex(h.h, x, gd, s1, s2, update=update, optimizer=optimizer,
                            adam_step=t + 1, dropped=drop_dev, **kw)
        o.round_ex(xo, g, o1, o2, update=update, optimizer=optimizer, adam_step=t + 1,
                   **okw, **kw)
        torch.cuda.synchronize()
        xg = x.cpu().numpy()
        assert_params_close(xg, xo, f"case {k} x round {t}")
        assert bit_mismatches(xg, xo) == 0, f"case {k}: x not bit-identical at round {t}"
        if uses_s1:
            assert bit_mismatches(s1.cpu().numpy(), o1) == 0, f"case {k}: state1 at round {t}"
        if uses_s2:
            assert bit_mismatches(s2.cpu().numpy(), o2) == 0, f"case {k}: state2 at round {t}"
        nbar, _ = h.counts()
        want = np.concatenate([o.a.nbars(), o.b.nbars()]) if double else o.nbars()
        assert np.array_equal(nbar, want), f"case {k}: nbar at round {t}"
    h.close()
    o.close()
    torch.cuda.synchronize()
