"""GPU parity for double binary trees (Section 3): a relaysum_create_double
handle against the double-tree oracle (two single-tree oracles over the odd
and even coordinates), bit for bit, for every update rule and local
optimizer, with and without lost messages.  Shapes cover the fused
double-tree kernel (up to 32 workers, one and two workers per wave, ragged
last tile), the kernel that relays the two trees in turn through LDS (33 to
64 workers), the double-tree cluster kernels (more than 64 workers, the
boundary workers completed by a second launch) and, for pairs of trees with
a hub of more than 32 neighbours (a star with a chain), the per-tree
two-pass path with its hub kernels, each on 16-byte aligned rows, on rows
only 4-byte aligned and with d % 4 != 0 (a partial last chunk; d odd gives
tree B one more coordinate)."""
import sys

import numpy as np
import pytest
import torch

import paper_2110_04175_amd as rs
import treeutil
import workloads as wl
from oracle.double import DoubleOracle
from parity import assert_params_close, bit_mismatches

pytestmark = pytest.mark.gpu

RULES = [
    ("model", "sgd", dict(lr=0.1)),
    ("model", "sgd", dict(lr=0.1, beta1=0.9)),
    ("model", "adam", dict(lr=1e-2, beta1=0.9, beta2=0.999, eps=1e-8)),
    ("robust", "sgd", dict(lr=0.1)),
    ("robust", "sgd", dict(lr=0.05, beta1=0.9)),
    ("robust", "adam", dict(lr=1e-2, beta1=0.8, beta2=0.99, eps=1e-6)),
    ("grad", "sgd", dict(lr=0.2)),
    ("mean", "sgd", dict()),
]
RULE_IDS = ["model-sgd", "model-nesterov", "model-adam", "robust-sgd", "robust-nesterov",
            "robust-adam", "grad", "mean"]

# name: (n, d, row offset in floats)
SHAPES = {
    "dbt16-fused": (16, 3000, 0),        # 5.9 tiles of 512 coordinates
    "dbt32-fused-pw2": (32, 2048, 0),    # two workers per wave
    "dbt7-fused": (7, 520, 0),           # one full tile and an 8-coordinate tail
    "dbt16-d3002": (16, 3002, 0),        # d % 4 != 0: a partial last chunk
    "dbt9-odd-d": (9, 1001, 0),          # d odd: tree B carries one more coordinate
    "dbt9-misaligned": (9, 1000, 1),     # 4-byte aligned rows only
    "dbt20-odd-off2": (20, 4003, 2),     # both: partial chunk on rows 8 bytes off
    "dbt40-seq": (40, 1500, 0),          # trees relayed in turn through LDS
    "dbt64-seq": (64, 2056, 0),          # four workers per wave, ragged tile
    "dbt40-seq-misaligned": (40, 1500, 1),   # on 4-byte aligned rows
    "dbt64-seq-odd": (64, 2051, 3),      # partial chunk, rows 12 bytes off
    "dbt33-seq": (33, 520, 0),           # one worker in the third slot of wave 0
    "dbt65-cluster": (65, 1500, 0),      # double-tree cluster kernels
    "dbt100-cluster": (100, 1000, 0),
    "dbt90-cluster-odd": (90, 2051, 1),  # partial chunk, 4-byte aligned rows
    "dbt200-cluster": (200, 1030, 0),    # more than 128 workers
    "dbt130-cluster-odd": (130, 1001, 1),   # d odd on 4-byte aligned rows
    "sc65-twopass": (65, 1500, 0),       # star + chain: per-tree two-pass path, hub kernels
    "sc100-twopass-odd": (100, 2051, 1), # partial chunk, 4-byte aligned rows
    "sc130-twopass": (130, 1000, 0),     # star + chain beyond 128 workers: two-pass per tree
    "sc130-twopass-odd": (130, 1001, 1),   # the same with d odd on 4-byte aligned rows
}


def pair_edges(shape, n):
    """The shape's two trees: the paper's double binary trees, or ("sc") a
    star for tree A and a chain for tree B."""
    if shape.startswith("sc"):
        return wl.star_edges(n), wl.chain_edges(n)
    return wl.double_binary_tree_edges(n)


def announce(msg):
    sys.__stderr__.write(f"[gpu] {msg}\n")
    sys.__stderr__.flush()


def per_slot(mask_a, mask_b, slots, e2a):
    return np.array([(mask_a if s < e2a else mask_b)[i, j] for s, (i, j) in enumerate(slots)],
                    np.uint8)


def expected_path(n, d, hub=False):
    """The double-tree kernels' ranges (relaysum.h, relaysum_path); `hub`: a
    tree has a worker of more than 32 neighbours."""
    if n <= 32:
        return "dtree"
    if d == 0:
        return "two_pass"
    if n <= 64:
        return "dtree_seq"
    return "two_pass" if hub else "cluster_dtree"


def run_double(shape, update, optimizer, kw, p_drop, seed=0, rounds=None):
    n, d, offset = SHAPES[shape]
    ea, eb = pair_edges(shape, n)
    diam = max(treeutil.diameter(n, ea), treeutil.diameter(n, eb))
    rounds = rounds or diam + 3
    announce(f"double {shape} {update}/{optimizer} {kw} p_drop={p_drop} n={n} d={d} "
             f"rounds={rounds}")
    rng = np.random.default_rng(seed)
    dev = torch.device("cuda")
    x0 = rng.standard_normal((n, d)).astype(np.float32)
    if update == "mean":
        x0[:] = 0
    uses_s1 = optimizer == "adam" or kw.get("beta1", 0.0) != 0.0 or update == "mean"
    uses_s2 = optimizer == "adam"

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
    o = DoubleOracle(n, d, ea, eb, np.float32)
    with rs.RelaySum(n, d, ea, edges_b=eb) as h:
        assert h.path == expected_path(n, d, hub=shape.startswith("sc") and n > 33), h.path
        assert h.num_trees == 2
        e2a = 2 * (n - 1)
        assert h.num_directed_edges == 2 * e2a
        slots = [h.directed_edge(s) for s in range(h.num_directed_edges)]
        for t in range(rounds):
            g = rng.standard_normal((n, d)).astype(np.float32)
            bg, gd = dev_buf(g)
            ma = mb = None
            drop_dev = None
            if p_drop:
                ma = (rng.random((n, n)) < p_drop).astype(np.uint8)
                mb = (rng.random((n, n)) < p_drop).astype(np.uint8)
                drop_dev = torch.from_numpy(per_slot(ma, mb, slots, e2a)).to(dev)
            step = t + 1
            rs.relaysum_step_ex(h.h, x, gd, s1, s2, update=update, optimizer=optimizer,
                                adam_step=step, dropped=drop_dev, **kw)
            o.round_ex(xo, g, o1, o2, update=update, optimizer=optimizer, adam_step=step,
                       dropped_a=ma, dropped_b=mb, **kw)
            torch.cuda.synchronize()
            xg = x.cpu().numpy()
            assert_params_close(xg, xo, f"{shape} {update} x round {t}")
            assert bit_mismatches(xg, xo) == 0, f"x not bit-identical at round {t}"
            if uses_s1:
                assert bit_mismatches(s1.cpu().numpy(), o1) == 0, f"state1 differs at round {t}"
            if uses_s2:
                assert bit_mismatches(s2.cpu().numpy(), o2) == 0, f"state2 differs at round {t}"
            nbar, cnt = h.counts()
            assert np.array_equal(nbar[:n], o.a.nbars()), f"tree A nbar differs at round {t}"
            assert np.array_equal(nbar[n:], o.b.nbars()), f"tree B nbar differs at round {t}"
            want = [(o.a if s < e2a else o.b).count(i, j) for s, (i, j) in enumerate(slots)]
            assert np.array_equal(cnt, want), f"edge counters differ at round {t}"
            if update == "mean":
                smp = h.samples()
                assert list(smp[:n]) == [o.a.samples(i) for i in range(n)]
                assert list(smp[n:]) == [o.b.samples(i) for i in range(n)]
            if t == rounds - 1:
                for s_ in list(range(3)) + list(range(e2a, e2a + 3)):
                    i, j = slots[s_]
                    tree = o.a if s_ < e2a else o.b
                    got = h.message(s_)
                    assert len(got) == (d // 2 if s_ < e2a else (d + 1) // 2)
                    assert bit_mismatches(got[None], tree.message(i, j)[None]) == 0
    o.close()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("shape", list(SHAPES))
@pytest.mark.parametrize("rule", range(len(RULES)), ids=RULE_IDS)
def test_double_trees_rule(rule, shape):
    update, optimizer, kw = RULES[rule]
    run_double(shape, update, optimizer, kw, 0.0, seed=rule)


@pytest.mark.parametrize("shape", ["dbt16-fused", "dbt32-fused-pw2", "dbt9-odd-d",
                                   "dbt20-odd-off2", "dbt40-seq", "dbt64-seq",
                                   "dbt64-seq-odd", "dbt100-cluster", "dbt90-cluster-odd",
                                   "dbt200-cluster", "sc100-twopass-odd", "sc130-twopass-odd"])
@pytest.mark.parametrize("rule", [1, 4, 5, 7], ids=[RULE_IDS[i] for i in (1, 4, 5, 7)])
def test_double_trees_with_lost_messages(rule, shape):
    update, optimizer, kw = RULES[rule]
    run_double(shape, update, optimizer, kw, 0.15, seed=200 + rule)


@pytest.mark.parametrize("n,d", [(1, 64), (2, 8), (2, 3), (16, 0), (5, 1)])
def test_double_trees_degenerate(n, d):
    """One worker (no edges), two workers, d = 0 (counters only), d = 1
    (tree A carries nothing)."""
    ea, eb = wl.double_binary_tree_edges(n)
    rng = np.random.default_rng(n * 100 + d)
    x0 = rng.standard_normal((n, d)).astype(np.float32)
    xo = x0.copy()
    mo = np.zeros_like(x0)
    x = torch.from_numpy(x0).cuda()
    mom = torch.zeros_like(x)
    o = DoubleOracle(n, d, ea, eb, np.float32)
    with rs.RelaySum(n, d, ea, edges_b=eb) as h:
        assert h.path == expected_path(n, d), h.path
        for t in range(4):
            g = rng.standard_normal((n, d)).astype(np.float32)
            h.step(x, torch.from_numpy(g).cuda(), mom, 0.1, 0.9)
            o.round(xo, g, mo, 0.1, 0.9)
            torch.cuda.synchronize()
            assert bit_mismatches(x.cpu().numpy(), xo) == 0
            nbar, _ = h.counts()
            assert np.array_equal(nbar, np.concatenate([o.a.nbars(), o.b.nbars()]))
    o.close()


@pytest.mark.parametrize("name", ["dbtree16", "dbtree64", "dbtree200"])
def test_double_tree_workloads_full_size_sampled(name):
    """The double-tree workloads at full size, in the launch shape the
    benchmark times (fused kernel at 16 workers, sequential kernel at 64,
    clusters at 200), checked
    on sampled coordinate pairs against the oracle."""
    w = wl.workload(name)
    announce(f"workload {name} full size, sampled parity")
    dev = torch.device("cuda")
    # sample whole even/odd pairs so both trees are covered; the oracle runs
    # each tree on its own sampled coordinates
    base = wl.sample_columns(w.d // 2, 2048, tile=256) * 2   # 256 carried coordinates per kernel tile
    idx_np = np.unique(np.concatenate([base, base + 1]))
    idx_np = idx_np[idx_np < w.d]
    odd = idx_np[idx_np % 2 == 1]
    even = idx_np[idx_np % 2 == 0]
    from oracle import Oracle
    oa = Oracle(w.n, len(odd), w.edges, np.float32)
    ob = Oracle(w.n, len(even), w.edges_b, np.float32)
    state = {}
    x = w.x0(dev)
    mom = torch.zeros_like(x)
    cols = {"a": torch.from_numpy(odd).to(dev), "b": torch.from_numpy(even).to(dev)}
    xs = {k: x.index_select(1, c).cpu().numpy().copy() for k, c in cols.items()}
    ms = {k: np.zeros_like(v) for k, v in xs.items()}
    mism = 0
    with rs.RelaySum(w.n, w.d, w.edges, edges_b=w.edges_b) as h:
        assert h.path == expected_path(w.n, w.d), h.path
        for t in range(w.rounds):
            g = w.grad(t, dev, state)
            h.step(x, g, mom, w.lr(t), w.beta)
            for k, o in (("a", oa), ("b", ob)):
                o.round(xs[k], g.index_select(1, cols[k]).cpu().numpy(), ms[k], w.lr(t), w.beta)
                xg = x.index_select(1, cols[k]).cpu().numpy()
                assert_params_close(xg, xs[k], f"{name} tree {k} x round {t}")
                mism += bit_mismatches(xg, xs[k])
                mism += bit_mismatches(mom.index_select(1, cols[k]).cpu().numpy(), ms[k])
            del g
            nbar, _ = h.counts()
            assert np.array_equal(nbar, np.concatenate([oa.nbars(), ob.nbars()]))
    announce(f"{name}: bit mismatches = {mism}")
    assert mism == 0
    oa.close()
    ob.close()
    del x, mom
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
