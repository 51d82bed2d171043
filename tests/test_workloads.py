"""Seeded input generators: topologies and streams (CPU)."""
import itertools

import numpy as np
import pytest
import torch

import workloads as wl
import treeutil


def prufer_encode(n, edges):
    """Textbook encoding: repeatedly remove the smallest leaf, record its neighbour."""
    adj = treeutil.adjacency(n, edges)
    removed = set()
    seq = []
    for _ in range(n - 2):
        leaf = min(i for i in range(n) if i not in removed and len(adj[i]) == 1)
        (nb,) = adj[leaf]
        seq.append(nb)
        adj[nb].discard(leaf)
        removed.add(leaf)
    return seq


@pytest.mark.parametrize("n", [3, 4, 5, 6])
def test_prufer_decode_is_a_bijection(n):
    trees = list(wl.all_labelled_trees(n))
    assert len(trees) == n ** (n - 2)   # Cayley's formula
    keys = set()
    for seq in itertools.product(range(n), repeat=n - 2):
        e = wl.prufer_decode(seq, n)
        assert e.shape == (n - 1, 2)
        treeutil.hop_distances(n, e)   # connected
        assert prufer_encode(n, e) == list(seq)
        keys.add(frozenset(frozenset(map(int, x)) for x in e))
    assert len(keys) == n ** (n - 2)


def test_topologies():
    assert treeutil.diameter(4, wl.chain_edges(4)) == 3
    assert treeutil.diameter(16, wl.heap_edges(16)) == 7
    assert treeutil.diameter(16, wl.chain_edges(16)) == 15
    e = wl.random_tree_edges(256, 0)
    assert e.shape == (255, 2)
    tau = treeutil.hop_distances(256, e)
    assert 20 <= tau.max() <= 80
    assert np.array_equal(e, wl.random_tree_edges(256, 0))
    b = wl.broom_edges(40)
    assert b.shape == (39, 2) and treeutil.diameter(40, b) == 28
    assert np.bincount(b.ravel(), minlength=40).max() == 13


def test_streams_are_seeded_and_independent():
    a = wl.normal((3, 5), 0, "grad", 7)
    b = wl.normal((3, 5), 0, "grad", 7)
    c = wl.normal((3, 5), 0, "grad", 8)
    assert torch.equal(a, b) and not torch.equal(a, c)
    assert a.dtype == torch.float32


def test_workloads_shapes_and_recipes():
    ws = wl.workloads()
    assert list(ws) == ["chain4", "heap16", "chain16", "prufer256", "chain16_bert"]
    for w in ws.values():
        small = w.with_d(64)
        x0 = small.x0()
        g0 = small.grad(0)
        assert x0.shape == (w.n, 64) and g0.shape == (w.n, 64)
        assert w.edges.shape == (w.n - 1, 2)
    c1 = ws["chain4"].with_d(20000)
    g = c1.grad(3)
    assert np.allclose(g.mean(dim=1).numpy(), [0, 1, 2, 3], atol=0.05)
    # identical x0 across workers where the recipe says so
    for name in ("heap16", "chain16", "chain16_bert"):
        x0 = ws[name].with_d(100).x0()
        assert torch.equal(x0[0], x0[-1])
    assert ws["prufer256"].lr(299) == 0.0 and ws["prufer256"].lr(300) == 0.01


def test_algorithmic_bytes():
    # chain n=16, d=9.75M, momentum: 4*d*(5*16 + 4*15) = 5.46 GB
    assert wl.algorithmic_bytes(16, 9_750_000, 15, 0.9) == 4 * 9_750_000 * 140
    assert wl.algorithmic_bytes(4, 1000, 3, 0.0) == 4 * 1000 * 24


def test_sample_columns():
    idx = wl.sample_columns(1_000_000, 4096)
    assert len(idx) == 4096 and np.all(np.diff(idx) > 0)
    assert idx[0] == 0 and idx[-1] == 999_999
    assert np.array_equal(wl.sample_columns(100), np.arange(100))


@pytest.mark.parametrize("d", [9_750_000, 110_000_000, 1_000_000, 270_000])
def test_sample_columns_cover_tile_edges_across_the_row(d):
    """Both sides of kernel-tile (512k) and ring-tile (4096k) boundaries are
    sampled over the whole row, not only near its start."""
    idx = set(wl.sample_columns(d, 4096).tolist())
    for step in (512, 4096):
        pairs = [b for b in range(step, d, step) if b - 1 in idx and b in idx]
        assert len(pairs) >= min(100, (d - 1) // step)
        assert max(pairs) >= 0.95 * d - step and min(pairs) <= 0.05 * d + step


@pytest.mark.parametrize("n", [2, 3, 7, 8, 15, 16, 17, 33, 64])
def test_double_binary_trees_are_complementary(n):
    """Both are trees of degree <= 3, and no worker is internal (degree >= 2)
    in both (Section 3: internal nodes of one tree are leaves of the other)."""
    a, b = wl.double_binary_tree_edges(n)
    for e in (a, b):
        assert e.shape == (n - 1, 2)
        treeutil.hop_distances(n, e)          # connected
    da = np.bincount(a.ravel(), minlength=n)
    db = np.bincount(b.ravel(), minlength=n)
    assert da.max() <= 3 and db.max() <= 3
    if n >= 3:
        assert not np.any((da >= 2) & (db >= 2))


def test_next_workloads_recipes():
    names = wl.all_workload_names()
    assert names[5:] == ["chain16_adam", "chain16_robust10", "chain16_grad", "chain16_mean",
                         "dbtree16", "dbtree64", "broom1000", "random8192", "dbtree200", "pa2000",
                         "chain64"]
    pa = wl.workload("pa2000")
    deg = np.bincount(pa.edges.ravel(), minlength=pa.n)
    assert pa.edges.shape == (1999, 2) and sorted(deg)[-5:] == [33, 34, 36, 36, 41]
    treeutil.hop_distances(pa.n, pa.edges)   # connected
    b = wl.workload("broom1000")
    assert np.bincount(b.edges.ravel(), minlength=b.n).max() == 13
    r8 = wl.workload("random8192")
    assert r8.n == 8192 and r8.edges.shape == (8191, 2)
    d2 = wl.workload("dbtree200")
    assert d2.double and d2.n == 200 and d2.bytes_per_round() == wl.algorithmic_bytes(200, d2.d, 199, 0.9)
    c64 = wl.workload("chain64")
    assert not c64.double and c64.n == 64 and np.array_equal(c64.edges, wl.chain_edges(64))
    assert c64.bytes_per_round() == wl.algorithmic_bytes(64, 9_750_000, 63, 0.9)
    w64 = wl.workload("dbtree64")
    assert w64.double and w64.n == 64 and w64.edges.shape == (63, 2)
    w = wl.workload("dbtree16")
    assert w.double and w.n == 16 and w.d == 9_750_000
    ea, eb = wl.double_binary_tree_edges(16)
    assert np.array_equal(w.edges, ea) and np.array_equal(w.edges_b, eb)
    # each coordinate rides one tree: same per-coordinate bytes as a chain of 16
    assert w.bytes_per_round() == wl.algorithmic_bytes(16, w.d, 15, 0.9)
    small = w.with_d(64)
    assert small.double and small.x0().shape == (16, 64)
    r = wl.workload("chain16_robust10")
    assert r.drop_mask(3).shape == (16, 16)
    assert np.array_equal(r.drop_mask(3), r.drop_mask(3))
    rd = wl.Workload(**{**r.__dict__, "edges_b": eb})
    assert rd.drop_mask(3).shape == (2, 16, 16)
    assert rd.bytes_per_round() == r.bytes_per_round() + 2 * 15
