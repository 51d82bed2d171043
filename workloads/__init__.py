"""Seeded synthetic inputs for RelaySum rounds: tree topologies and the
per-round model / gradient tensors of the five benchmark workloads.

This module is shared by the HIP path's tests and bench and by the oracle's
tests.  It holds no arithmetic of the method itself (no local step, no
message relay, no averaging): only graph construction and random draws.

Stand-ins for the paper's workloads (Section 5 and Appendix B): the
parameter-vector lengths d stand for model sizes (a VGG-11-sized flat vector,
a BERT-base-sized one), n=16 is the paper's worker count, per-worker gradient
means mu_i stand for its Dirichlet label heterogeneity, and chains, balanced
binary trees and a uniformly random labelled tree stand for the trees it runs
on (chains, double binary trees, spanning trees of arbitrary graphs).  No
dataset item is reproduced; every value is drawn from a seeded generator.

Readings of the workload text:
  * N(a, b): b is a standard deviation.
  * Where a per-worker mean mu_i is not said to be a vector it is a scalar.
  * The random labelled tree decodes a Pruefer sequence drawn uniformly from
    [0, n)^(n-2) with numpy PCG64, by the usual smallest-leaf rule.
  * Seed 0 everywhere.  Each (tag, round) pair has its own generator, seeded
    from numpy's SeedSequence, so any round can be produced on its own.
"""
from __future__ import annotations

import heapq
from dataclasses import dataclass, field
from typing import Callable, Dict, List, Optional, Sequence, Tuple

import numpy as np

# ----------------------------------------------------------------------------
# Topologies.  An edge list is an int32 array of shape (n-1, 2), 0-based.
# ----------------------------------------------------------------------------


def chain_edges(n: int) -> np.ndarray:
    """Chain 0-1-...-(n-1) (the paper's chain, Section 3)."""
    i = np.arange(max(n - 1, 0), dtype=np.int32)
    return np.stack([i, i + 1], axis=1)


def heap_edges(n: int) -> np.ndarray:
    """Balanced binary tree in heap order: node i's parent is (i-1)//2."""
    return np.array([((i - 1) // 2, i) for i in range(1, n)], dtype=np.int32).reshape(-1, 2)


def star_edges(n: int, centre: int = 0) -> np.ndarray:
    """Star: every worker attached to `centre`."""
    return np.array([(centre, i) for i in range(n) if i != centre], dtype=np.int32).reshape(-1, 2)


def broom_edges(n: int, bristles: int = 12) -> np.ndarray:
    """Broom: a chain 0 - 1 - ... - (n - bristles - 1) whose last worker also
    carries the `bristles` leaves n - bristles .. n - 1 (a worker of degree
    bristles + 1 on a long handle)."""
    h = n - bristles
    assert h >= 1, "a broom needs a handle of at least one worker"
    handle = [(i, i + 1) for i in range(h - 1)]
    leaves = [(h - 1, j) for j in range(h, n)]
    return np.array(handle + leaves, dtype=np.int32).reshape(-1, 2)


def preferential_attachment_edges(n: int, seed: int) -> np.ndarray:
    """Seeded preferential-attachment tree: worker k >= 2 joins an existing
    worker chosen with probability proportional to its degree (worker 1
    joins worker 0), so a few workers become hubs, as in spanning trees of
    scale-free networks."""
    rng = np.random.default_rng(seed)
    ends = []        # every edge end once: a draw from it is degree-proportional
    edges = []
    for k in range(1, n):
        p = 0 if k == 1 else ends[int(rng.integers(len(ends)))]
        edges.append((p, k))
        ends += [p, k]
    return np.array(edges, dtype=np.int32).reshape(-1, 2)


def _inorder_tree(lo: int, hi: int, parent, out) -> None:
    """Balanced binary tree over the ranks [lo, hi) in in-order numbering:
    the root is the rank whose offset from lo, plus one, has the most
    trailing zero bits, so leaves fall on even offsets."""
    if lo >= hi:
        return
    best, best_z = lo, -1
    for r in range(lo, hi):
        v = r - lo + 1
        z = (v & -v).bit_length()
        if z > best_z:
            best, best_z = r, z
    if parent is not None:
        out.append((parent, best))
    _inorder_tree(lo, best, best, out)
    _inorder_tree(best + 1, hi, best, out)


def double_binary_tree_edges(n: int):
    """Two complementary balanced binary trees on n workers (Section 3's double
    binary trees, after Sanders et al.): tree A numbers the workers in-order,
    so its leaves are the even ranks; tree B is tree A with every rank shifted
    by one (mod n), so the workers internal in one tree are leaves in the
    other.  Returns (edges_a, edges_b)."""
    a = []
    _inorder_tree(0, n, None, a)
    b = [((u + 1) % n, (v + 1) % n) for u, v in a]
    return (np.array(a, dtype=np.int32).reshape(-1, 2),
            np.array(b, dtype=np.int32).reshape(-1, 2))


def prufer_decode(seq: Sequence[int], n: int) -> np.ndarray:
    """Tree with the given Pruefer sequence (length n-2, entries in [0, n)).

    Smallest-leaf decoding: repeatedly join the smallest current leaf to the
    next sequence entry.  Every labelled tree on n >= 2 nodes has exactly one
    sequence, so drawing the sequence uniformly draws the tree uniformly.
    """
    if n == 1:
        return np.zeros((0, 2), dtype=np.int32)
    if n == 2:
        return np.array([[0, 1]], dtype=np.int32)
    seq = [int(s) for s in seq]
    assert len(seq) == n - 2 and all(0 <= s < n for s in seq)
    degree = [1] * n
    for s in seq:
        degree[s] += 1
    leaves = [i for i in range(n) if degree[i] == 1]
    heapq.heapify(leaves)
    edges = []
    for s in seq:
        leaf = heapq.heappop(leaves)
        edges.append((leaf, s))
        degree[s] -= 1
        if degree[s] == 1:
            heapq.heappush(leaves, s)
    u = heapq.heappop(leaves)
    v = heapq.heappop(leaves)
    edges.append((u, v))
    return np.array(edges, dtype=np.int32)


def random_tree_edges(n: int, seed: int = 0) -> np.ndarray:
    """Uniform random labelled tree on n nodes from a seeded Pruefer sequence."""
    if n <= 2:
        return prufer_decode([], n)
    rng = np.random.default_rng(seed)
    return prufer_decode(rng.integers(0, n, n - 2), n)


def all_labelled_trees(n: int):
    """Every labelled tree on n nodes (n^(n-2) of them), via all Pruefer sequences."""
    import itertools
    if n <= 2:
        yield prufer_decode([], n)
        return
    for seq in itertools.product(range(n), repeat=n - 2):
        yield prufer_decode(seq, n)


# ----------------------------------------------------------------------------
# Seeded streams.
# ----------------------------------------------------------------------------

_TAGS = {"x0": 1, "grad": 2, "mu": 3, "perm": 4, "drop": 5, "misc": 6}


def stream_seed(seed: int, tag: str, *idx: int) -> int:
    """A 63-bit seed for the stream (seed, tag, idx...), independent per tuple."""
    ss = np.random.SeedSequence([seed, _TAGS[tag], *[int(i) for i in idx]])
    return int(ss.generate_state(1, dtype=np.uint64)[0] & np.uint64(0x7FFFFFFFFFFFFFFF))


def normal(shape, seed: int, tag: str, *idx: int, device="cpu", std: float = 1.0,
           mean=0.0):
    """float32 tensor of N(mean, std) draws from stream (seed, tag, idx...).

    Draws come from torch's generator on `device`; a given (device, stream)
    always yields the same values.  `mean` may be a scalar or a tensor that
    broadcasts against `shape`.
    """
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(stream_seed(seed, tag, *idx))
    z = torch.randn(tuple(shape), generator=gen, device=device, dtype=torch.float32)
    if std != 1.0:
        z.mul_(std)
    if isinstance(mean, (int, float)):
        if mean != 0.0:
            z.add_(mean)
    else:
        z.add_(mean)
    return z


# ----------------------------------------------------------------------------
# The five benchmark workloads.
# ----------------------------------------------------------------------------


@dataclass
class Workload:
    """One synthetic RelaySGD workload: a tree, sizes, and seeded inputs."""

    name: str
    description: str
    n: int
    d: int
    edges: np.ndarray
    rounds: int
    beta: float
    lr_of_round: Callable[[int], float]
    _x0: Callable = field(repr=False, default=None)
    _grad: Callable = field(repr=False, default=None)
    seed: int = 0
    checkpoints: Tuple[int, ...] = ()
    update: str = "model"        # model | robust | grad | mean
    optimizer: str = "sgd"       # sgd (beta = Nesterov momentum, 0 = none) | adam
    beta2: float = 0.0
    eps: float = 0.0
    drop_prob: float = 0.0       # probability that a directed message is lost
    edges_b: Optional[np.ndarray] = None   # double binary trees: tree B (even coordinates)

    @property
    def double(self) -> bool:
        """Double binary trees: odd coordinates relayed on `edges`, even on `edges_b`."""
        return self.edges_b is not None

    def lr(self, t: int) -> float:
        return float(self.lr_of_round(t))

    def drop_mask(self, t: int) -> Optional[np.ndarray]:
        """[n, n] uint8: (k, i) = 1 when the message k -> i of round t is lost
        ([2, n, n] on double trees: tree A's mask, then tree B's)."""
        if self.drop_prob <= 0.0:
            return None
        rng = np.random.default_rng(np.random.SeedSequence([self.seed, _TAGS["drop"], t]))
        shape = (2, self.n, self.n) if self.double else (self.n, self.n)
        return (rng.random(shape) < self.drop_prob).astype(np.uint8)

    def bytes_per_round(self) -> int:
        """Algorithmic HBM bytes of one round (see algorithmic_bytes)."""
        return algorithmic_bytes(self.n, self.d, self.n - 1, self.beta, self.update,
                                 self.optimizer, self.drop_prob > 0,
                                 trees=2 if self.double else 1)

    def x0(self, device="cpu"):
        """Initial models, float32 [n, d] (row i is worker i)."""
        return self._x0(self, device)

    def grad(self, t: int, device="cpu", state: Optional[dict] = None):
        """Round-t gradients, float32 [n, d].  `state` caches fixed draws (mu)."""
        if state is None:
            state = {}
        return self._grad(self, t, device, state)

    def with_d(self, d: int) -> "Workload":
        """Same workload at a different vector length (small CPU cases)."""
        w = Workload(**{**self.__dict__})
        w.d = int(d)
        w.name = f"{self.name}@d={d}"
        return w


def _x0_iid(std):
    def f(w, device):
        return normal((w.n, w.d), w.seed, "x0", device=device, std=std)
    return f


def _x0_identical(std):
    def f(w, device):
        row = normal((1, w.d), w.seed, "x0", device=device, std=std)
        return row.expand(w.n, w.d).contiguous()
    return f


def _grad_mean_index(std):
    """g_i ~ N(i, std): worker i's mean is its index."""
    def f(w, t, device, state):
        import torch
        mu = torch.arange(w.n, dtype=torch.float32, device=device).reshape(w.n, 1)
        return normal((w.n, w.d), w.seed, "grad", t, device=device, std=std, mean=mu)
    return f


def _grad_scalar_mu(mu_std, std):
    """g_i ~ N(mu_i, std) with a fixed scalar mu_i ~ N(0, mu_std) per worker."""
    def f(w, t, device, state):
        key = ("mu", str(device))
        if key not in state:
            state[key] = normal((w.n, 1), w.seed, "mu", device=device, std=mu_std)
        return normal((w.n, w.d), w.seed, "grad", t, device=device, std=std,
                      mean=state[key])
    return f


def _grad_vector_mu(mu_std, std):
    """g_i ~ mu_i + N(0, std), mu_i ~ N(0, mu_std) a fixed vector of length d."""
    def f(w, t, device, state):
        key = ("mu", str(device), w.d)
        if key not in state:
            state[key] = normal((w.n, w.d), w.seed, "mu", device=device, std=mu_std)
        return normal((w.n, w.d), w.seed, "grad", t, device=device, std=std,
                      mean=state[key])
    return f


def _grad_standard():
    def f(w, t, device, state):
        return normal((w.n, w.d), w.seed, "grad", t, device=device)
    return f


def workloads() -> Dict[str, Workload]:
    """The five workloads, keyed by short name."""
    ws = [
        Workload(
            name="chain4",
            description="chain of n=4 workers, d=1,000 fp32, x0 iid N(0,1), "
                        "g_i ~ N(i,1), lr=0.1, no momentum, 20 rounds, seed 0",
            n=4, d=1000, edges=chain_edges(4), rounds=20, beta=0.0,
            lr_of_round=lambda t: 0.1, _x0=_x0_iid(1.0),
            _grad=_grad_mean_index(1.0), checkpoints=tuple(range(1, 21))),
        Workload(
            name="heap16",
            description="balanced binary tree n=16 (parent (i-1)//2), d=270,000 "
                        "fp32, identical x0 ~ N(0,0.01), g_i ~ N(mu_i,1) with "
                        "scalar mu_i ~ N(0,1), lr=0.05, momentum 0.9, 100 rounds",
            n=16, d=270_000, edges=heap_edges(16), rounds=100, beta=0.9,
            lr_of_round=lambda t: 0.05, _x0=_x0_identical(0.01),
            _grad=_grad_scalar_mu(1.0, 1.0), checkpoints=(1, 2, 7, 8, 50, 100)),
        Workload(
            name="chain16",
            description="chain n=16, d=9,750,000 fp32 (VGG-11-sized), identical "
                        "x0 ~ N(0,0.01), g_i ~ mu_i + N(0,0.1) with vector "
                        "mu_i ~ N(0,1) of length d, lr=0.1, momentum 0.9, 50 rounds",
            n=16, d=9_750_000, edges=chain_edges(16), rounds=50, beta=0.9,
            lr_of_round=lambda t: 0.1, _x0=_x0_identical(0.01),
            _grad=_grad_vector_mu(1.0, 0.1), checkpoints=(1, 15, 16, 50)),
        Workload(
            name="prufer256",
            description="uniform random labelled tree n=256 (seeded Pruefer "
                        "sequence), d=1,000,000 fp32, x0 iid N(0,1), g ~ N(0,1), "
                        "lr=0 for rounds 0..299 then 0.01, momentum 0.9, 400 rounds",
            n=256, d=1_000_000, edges=random_tree_edges(256, 0), rounds=400,
            beta=0.9, lr_of_round=lambda t: 0.0 if t < 300 else 0.01,
            _x0=_x0_iid(1.0), _grad=_grad_standard(),
            checkpoints=(1, 50, 300, 400)),
        Workload(
            name="chain16_bert",
            description="chain n=16, d=110,000,000 fp32 (BERT-base-sized), "
                        "identical x0 ~ N(0,0.02), g_i ~ N(mu_i,0.1) with scalar "
                        "mu_i ~ N(0,0.5), lr=0.01, momentum 0.9, 10 rounds",
            n=16, d=110_000_000, edges=chain_edges(16), rounds=10, beta=0.9,
            lr_of_round=lambda t: 0.01, _x0=_x0_identical(0.02),
            _grad=_grad_scalar_mu(0.5, 0.1), checkpoints=(1, 5, 10)),
    ]
    return {w.name: w for w in ws}


def _next_workloads() -> List[Workload]:
    """Workloads of the other update rules, at the chain16 size."""
    base = dict(n=16, d=9_750_000, edges=chain_edges(16), _x0=_x0_identical(0.01),
                checkpoints=(1, 15, 16))
    return [
        Workload(
            name="chain16_adam",
            description="Relay-Adam: chain n=16, d=9,750,000 fp32, identical x0 ~ "
                        "N(0,0.01), g_i ~ mu_i + N(0,0.1) with vector mu_i ~ N(0,1), "
                        "Adam lr=1e-3, betas (0.9, 0.999), eps 1e-8, 20 rounds",
            rounds=20, beta=0.9, lr_of_round=lambda t: 1e-3, optimizer="adam",
            beta2=0.999, eps=1e-8, _grad=_grad_vector_mu(1.0, 0.1), **base),
        Workload(
            name="chain16_robust10",
            description="robust update with 10% of messages lost per round: chain "
                        "n=16, d=9,750,000 fp32, identical x0 ~ N(0,0.01), g_i ~ mu_i "
                        "+ N(0,0.1) with vector mu_i ~ N(0,1), lr=0.1, momentum 0.9, "
                        "20 rounds",
            rounds=20, beta=0.9, lr_of_round=lambda t: 0.1, update="robust",
            drop_prob=0.1, _grad=_grad_vector_mu(1.0, 0.1), **base),
        Workload(
            name="chain16_grad",
            description="RelaySGD/Grad: chain n=16, d=9,750,000 fp32, identical x0 ~ "
                        "N(0,0.01), g_i ~ mu_i + N(0,0.1) with vector mu_i ~ N(0,1), "
                        "lr=0.1, 20 rounds",
            rounds=20, beta=0.0, lr_of_round=lambda t: 0.1, update="grad",
            _grad=_grad_vector_mu(1.0, 0.1), **base),
        Workload(
            name="chain16_mean",
            description="RelaySum mean estimation: chain n=16, d=9,750,000 fp32, "
                        "samples ~ N(1,1) per round, 20 rounds",
            rounds=20, beta=0.0, lr_of_round=lambda t: 0.0, update="mean",
            _grad=_samples_normal(1.0, 1.0), **base),
        Workload(
            name="dbtree16",
            description="double binary trees n=16 (in-order tree A for the odd "
                        "coordinates, its rank-shifted complement B for the even "
                        "ones), d=9,750,000 fp32, identical x0 ~ N(0,0.01), g_i ~ "
                        "mu_i + N(0,0.1) with vector mu_i ~ N(0,1), lr=0.1, "
                        "momentum 0.9, 20 rounds",
            rounds=20, beta=0.9, lr_of_round=lambda t: 0.1,
            _grad=_grad_vector_mu(1.0, 0.1),
            **{**base, "edges": double_binary_tree_edges(16)[0],
               "edges_b": double_binary_tree_edges(16)[1]}),
        Workload(
            name="dbtree64",
            description="double binary trees n=64 (in-order tree A for the odd "
                        "coordinates, its rank-shifted complement B for the even "
                        "ones), d=9,750,000 fp32, identical x0 ~ N(0,0.01), g_i ~ "
                        "N(mu_i,0.1) with scalar mu_i ~ N(0,1), lr=0.1, momentum 0.9, "
                        "20 rounds",
            n=64, d=9_750_000, edges=double_binary_tree_edges(64)[0],
            edges_b=double_binary_tree_edges(64)[1], rounds=20, beta=0.9,
            lr_of_round=lambda t: 0.1, _x0=_x0_identical(0.01),
            _grad=_grad_scalar_mu(1.0, 0.1), checkpoints=(1, 10, 20)),
        Workload(
            name="broom1000",
            description="broom of n=1,000 workers (a chain of 988 with 12 bristles on its "
                        "last worker: degree 13), d=300,000 fp32, identical x0 ~ N(0,0.01), "
                        "g_i ~ N(mu_i,0.1) with scalar mu_i ~ N(0,1), lr=0.1, momentum 0.9, "
                        "20 rounds",
            n=1000, d=300_000, edges=broom_edges(1000), edges_b=None, rounds=20, beta=0.9,
            lr_of_round=lambda t: 0.1, _x0=_x0_identical(0.01),
            _grad=_grad_scalar_mu(1.0, 0.1), checkpoints=(1, 10, 20)),
        Workload(
            name="random8192",
            description="uniform random labelled tree of n=8,192 workers (seeded Pruefer "
                        "sequence), d=40,000 fp32, x0 iid N(0,1), g ~ N(0,1), lr=0.01, "
                        "momentum 0.9, 20 rounds",
            n=8192, d=40_000, edges=random_tree_edges(8192, 0), edges_b=None, rounds=20,
            beta=0.9, lr_of_round=lambda t: 0.01, _x0=_x0_iid(1.0), _grad=_grad_standard(),
            checkpoints=(1, 10, 20)),
        Workload(
            name="dbtree200",
            description="double binary trees n=200 (in-order tree A for the odd "
                        "coordinates, its rank-shifted complement B for the even "
                        "ones), d=1,000,000 fp32, identical x0 ~ N(0,0.01), g_i ~ "
                        "N(mu_i,0.1) with scalar mu_i ~ N(0,1), lr=0.1, momentum 0.9, "
                        "20 rounds",
            n=200, d=1_000_000, edges=double_binary_tree_edges(200)[0],
            edges_b=double_binary_tree_edges(200)[1], rounds=20, beta=0.9,
            lr_of_round=lambda t: 0.1, _x0=_x0_identical(0.01),
            _grad=_grad_scalar_mu(1.0, 0.1), checkpoints=(1, 10, 20)),
        Workload(
            name="pa2000",
            description="preferential-attachment tree of n=2,000 workers (each new worker "
                        "joins an existing one with probability proportional to its degree; "
                        "seed 0: 5 hubs of 33 to 41 neighbours), d=150,000 fp32, identical "
                        "x0 ~ N(0,0.01), g_i ~ N(mu_i,0.1) with scalar mu_i ~ N(0,1), lr=0.1, "
                        "momentum 0.9, 20 rounds",
            n=2000, d=150_000, edges=preferential_attachment_edges(2000, 0), edges_b=None,
            rounds=20, beta=0.9, lr_of_round=lambda t: 0.1, _x0=_x0_identical(0.01),
            _grad=_grad_scalar_mu(1.0, 0.1), checkpoints=(1, 10, 20)),
        Workload(
            name="chain64",
            description="chain n=64 (the scaling runs' largest chain), d=9,750,000 fp32, "
                        "identical x0 ~ N(0,0.01), g_i ~ N(mu_i,0.1) with scalar "
                        "mu_i ~ N(0,1), lr=0.1, momentum 0.9, 20 rounds",
            n=64, d=9_750_000, edges=chain_edges(64), edges_b=None, rounds=20, beta=0.9,
            lr_of_round=lambda t: 0.1, _x0=_x0_identical(0.01),
            _grad=_grad_scalar_mu(1.0, 0.1), checkpoints=(1, 10, 20)),
    ]


def _samples_normal(mean, std):
    def f(w, t, device, state):
        return normal((w.n, w.d), w.seed, "grad", t, device=device, std=std, mean=mean)
    return f


def workload(name: str) -> Workload:
    ws = workloads()
    if name in ws:
        return ws[name]
    for w in _next_workloads():
        if w.name == name:
            return w
    raise KeyError(name)


def all_workload_names() -> List[str]:
    return list(workloads()) + [w.name for w in _next_workloads()]


def algorithmic_bytes(n: int, d: int, num_edges: int, beta: float, update: str = "model",
                      optimizer: str = "sgd", drops: bool = False, trees: int = 1) -> int:
    """Bytes one round must move through HBM at minimum.

    Per coordinate, in floats: x read and written (2n; mean estimation only
    writes its estimate, n), g read (n), the optimizer state read and written
    (momentum 2n, Adam 4n, mean-estimation sums 2n), and every directed
    edge's previous message read and new message written (4E).  With
    momentum that is 4*d*(5n + 4E) bytes, without 4*d*(3n + 4E).  Lost
    messages add the 2E-byte mask per tree.  On double binary trees each
    coordinate travels on one tree of E edges, so the per-coordinate figure
    is the same.
    """
    if update == "mean":
        rows = 4 * n
    elif update == "grad":
        rows = 3 * n
    elif optimizer == "adam":
        rows = 7 * n
    else:
        rows = 5 * n if beta != 0.0 else 3 * n
    per_coord = rows + 4 * num_edges
    return 4 * int(d) * per_coord + (2 * num_edges * trees if drops else 0)


def sample_columns(d: int, count: int = 4096, seed: int = 0, tile: int = 512,
                   ring_tile: int = 4096) -> np.ndarray:
    """Sorted coordinate indices for sampled parity at full size.

    Always includes the first and last 256 coordinates (the row ends and a
    ragged tail), both sides of kernel-tile boundaries (multiples of `tile`)
    and of ring-tile boundaries (multiples of `ring_tile`) spread evenly over
    the whole of [0, d), and uniform random coordinates to fill the rest.
    For double binary trees pass carried coordinates of one tree (a kernel
    tile carries 256 of them).
    """
    d = int(d)
    if d <= count:
        return np.arange(d, dtype=np.int64)
    picks = set(range(min(256, d)))
    picks.update(range(max(0, d - 256), d))

    def boundaries(step: int, budget: int) -> None:
        last = (d - 1) // step              # boundaries step*k, k = 1..last
        if last < 1 or budget < 1:
            return
        ks = np.unique(np.linspace(1, last, num=min(last, budget)).round().astype(np.int64))
        for b in (ks * step).tolist():
            picks.update((b - 1, b))

    boundaries(tile, count // 4)
    boundaries(ring_tile, count // 8)
    rng = np.random.default_rng(np.random.SeedSequence([seed, _TAGS["misc"], d]))
    while len(picks) < count:
        picks.update(rng.integers(0, d, count - len(picks)).tolist())
    return np.array(sorted(picks), dtype=np.int64)
