"""GPU parity at the size limits of the C ABI: the most workers a handle takes
(n = RELAYSUM_MAX_WORKERS = 2^24) and rows longer than 2^31 floats.

Neither fits the oracle whole (it keeps an n x n table of message slots, and
a 2^31-float row is 8.6 GB), so each test checks what a smaller oracle run
fixes exactly:

* Locality of the relay on a chain (Alg. 1): after R rounds worker i's model
  and momentum depend only on the workers within R hops of it, and its
  counters only on the workers within R hops.  A chain cut out around i,
  with at least R+2 workers on each side (or the real end of the chain),
  therefore gives bit-identical results for i, and the oracle runs that
  window.  The counters of every slot follow the chain's closed form.
* Independence of coordinates: every operation of a round is elementwise in
  the model coordinate, so the oracle run on a few sampled columns of a
  2-worker chain gives those columns of the full-length round.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2110_04175_amd as rs
import workloads as wl
from parity import bit_mismatches


def announce(msg: str) -> None:
    sys.__stderr__.write(f"[gpu] {msg}\n")
    sys.__stderr__.flush()


def _chain_counts(n: int, t: int):
    """Closed-form counters of a chain after rounds 0..t, in the library's
    slot order (directed edges sorted by source, then destination).

    c_{i->i+1} counts the workers i, i-1, ... within t hops of i (the message
    leaving i in round t has relayed t rounds); c_{i->i-1} likewise towards
    the other end; nbar_i = 1 + the counters received."""
    deg = np.full(n, 2, np.int64)
    deg[0] = deg[-1] = 1
    src = np.repeat(np.arange(n, dtype=np.int64), deg)
    # Worker i sends to i-1 first (when it exists), then to i+1.
    first = np.zeros(len(src), bool)
    first[np.concatenate(([0], np.cumsum(deg)[:-1]))] = True
    down = first & (src > 0)                  # i -> i-1
    dst = np.where(down, src - 1, src + 1)
    dst[-1] = n - 2                            # the last worker's only edge
    cnt = np.where(dst == src + 1, np.minimum(t + 1, src + 1), np.minimum(t + 1, n - src))
    i = np.arange(n)
    nbar = 1 + np.minimum(t + 1, i) + np.minimum(t + 1, n - 1 - i)
    return src, dst, cnt.astype(np.int32), nbar.astype(np.int32)


def test_chain_counts_closed_form_matches_oracle():
    """The closed form used below, against the oracle on a short chain."""
    n = 9
    o = oracle.Oracle(n, 1, wl.chain_edges(n), np.float32)
    x = np.zeros((n, 1), np.float32)
    g = np.zeros_like(x)
    for t in range(n + 1):
        o.round(x, g, None, 0.0, 0.0)
        src, dst, cnt, nbar = _chain_counts(n, t)
        assert np.array_equal(nbar, o.nbars()), t
        assert [o.count(int(a), int(b)) for a, b in zip(src, dst)] == cnt.tolist(), t
    o.close()


@pytest.mark.gpu
def test_most_workers():
    """n = 2^24 workers on a chain (the largest tree a handle takes), d = 5,
    Nesterov momentum, 3 rounds, on the cluster kernels (2^20 clusters)."""
    n, d, rounds, lr, beta = rs.RELAYSUM_MAX_WORKERS, 5, 3, 0.1, 0.9
    announce(f"most workers: chain n={n} d={d} rounds={rounds}")
    rng = np.random.default_rng(24)
    x0 = rng.standard_normal((n, d), dtype=np.float32)
    grads = [np.random.default_rng([24, t]).standard_normal((n, d), dtype=np.float32)
             for t in range(rounds)]
    dev = torch.device("cuda")
    x = torch.from_numpy(x0).to(dev)
    mom = torch.zeros_like(x)
    edges = wl.chain_edges(n)
    with rs.RelaySum(n, d, edges) as h:
        assert h.path == "cluster", h.path
        src, dst, _, _ = _chain_counts(n, 0)
        for s in (0, 1, 2, 3, 4, n, n + 1, 2 * n - 4, 2 * n - 3):
            assert h.directed_edge(s) == (int(src[s]), int(dst[s])), s
        for t in range(rounds):
            h.step(x, torch.from_numpy(grads[t]).to(dev), mom, lr, beta)
            nbar, cnt = h.counts()
            _, _, want_cnt, want_nbar = _chain_counts(n, t)
            assert np.array_equal(nbar, want_nbar), f"nbar round {t}"
            assert np.array_equal(cnt, want_cnt), f"edge counters round {t}"
        xg = x.cpu().numpy()
        mg = mom.cpu().numpy()
    del x, mom
    torch.cuda.empty_cache()

    margin = rounds + 2
    picks = [0, 1, 2, 3, 7, n // 2, n // 2 + 1, (1 << 23) + 12345, n - 8, n - 4, n - 3,
             n - 2, n - 1]
    picks += rng.integers(0, n, 8).tolist()
    for i in picks:
        lo, hi = max(0, i - margin), min(n - 1, i + margin)
        m = hi - lo + 1
        o = oracle.Oracle(m, d, wl.chain_edges(m), np.float32)
        xo = x0[lo:hi + 1].copy()
        mo = np.zeros_like(xo)
        for t in range(rounds):
            o.round(xo, np.ascontiguousarray(grads[t][lo:hi + 1]), mo, lr, beta)
        assert o.nbars()[i - lo] == 1 + min(rounds, i) + min(rounds, n - 1 - i)
        o.close()
        assert bit_mismatches(xg[i:i + 1], xo[i - lo:i - lo + 1]) == 0, f"x of worker {i}"
        assert bit_mismatches(mg[i:i + 1], mo[i - lo:i - lo + 1]) == 0, f"mom of worker {i}"


@pytest.mark.gpu
def test_longest_rows():
    """Rows of d = 2^31 + 3 floats (past 32-bit coordinate and byte offsets;
    d % 4 = 3, so worker 1's row is only 4-byte aligned and every row ends in
    a partial chunk): a 2-worker chain, Nesterov momentum, 2 rounds, checked
    on sampled coordinates around the 2^29, 2^30 and 2^31 float boundaries and
    at both ends of the row."""
    n, d, rounds, lr, beta = 2, (1 << 31) + 3, 2, 0.05, 0.9
    need = (3 * n * d + 4 * (n - 1) * (d + 4096)) * 4
    free, _ = torch.cuda.mem_get_info()
    if free < need + (8 << 30):
        pytest.skip(f"needs {need / 2**30:.0f} GiB of free device memory, {free / 2**30:.0f} free")
    announce(f"longest rows: chain n={n} d={d} rounds={rounds}")
    dev = torch.device("cuda")
    gen = torch.Generator(device=dev)
    gen.manual_seed(31)
    x = torch.empty((n, d), dtype=torch.float32, device=dev)
    x.normal_(generator=gen)
    g = torch.empty_like(x)
    mom = torch.zeros_like(x)
    cols = []
    for b in (0, 1 << 29, 1 << 30, 1 << 31):
        cols += range(max(0, b - 9), min(d, b + 9))
    cols += range(d - 12, d)
    cols += np.random.default_rng(31).integers(0, d, 64).tolist()
    cols = np.unique(np.array(cols, np.int64))
    idx = torch.from_numpy(cols).to(dev)
    xo = x.index_select(1, idx).cpu().numpy()
    mo = np.zeros_like(xo)
    o = oracle.Oracle(n, len(cols), wl.chain_edges(n), np.float32)
    with rs.RelaySum(n, d, wl.chain_edges(n)) as h:
        for t in range(rounds):
            g.normal_(generator=gen)
            h.step(x, g, mom, lr, beta)
            o.round(xo, g.index_select(1, idx).cpu().numpy(), mo, lr, beta)
        xg = x.index_select(1, idx).cpu().numpy()
        mg = mom.index_select(1, idx).cpu().numpy()
        nbar, cnt = h.counts()
    o.close()
    del x, g, mom
    torch.cuda.empty_cache()
    assert nbar.tolist() == [2, 2] and cnt.tolist() == [1, 1]
    assert bit_mismatches(xg, xo) == 0, "x differs from the oracle on sampled coordinates"
    assert bit_mismatches(mg, mo) == 0, "mom differs from the oracle on sampled coordinates"
