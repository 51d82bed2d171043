"""End to end on the GPU: RelaySGD as a training loop on heterogeneous
quadratics f_i(x) = |x - b_i|^2 / 2, the gradient x - b_i computed from the
current models every round (torch on the device; numpy for the oracle; one
IEEE subtraction, so both sides see the same gradients).  Each kernel path
runs the loop through relaysum_step; the models must equal the float32
oracle's bit for bit at every checkpoint and end at the global optimum
mean_i b_i (the exact fixed point of Alg. 1 with a constant step; see
test_end_to_end.py)."""
import sys

import numpy as np
import pytest
import torch

import oracle
from oracle.double import DoubleOracle
import paper_2110_04175_amd as rs
import workloads as wl
from parity import bit_mismatches

pytestmark = pytest.mark.gpu

CASES = {
    "tile, chain of 16": (16, 4096, wl.chain_edges(16), None, 0.5, 0.0, 400),
    "tile, chain of 16, Nesterov": (16, 4096, wl.chain_edges(16), None, 0.1, 0.9, 600),
    "double-tree kernel, 16 workers": (16, 4096, *wl.double_binary_tree_edges(16), 0.5, 0.0, 400),
    "sequential double-tree kernel, 40 workers": (40, 2048, *wl.double_binary_tree_edges(40), 0.5, 0.0, 400),
    "double-tree cluster kernels, 100 workers": (100, 2048, *wl.double_binary_tree_edges(100), 0.5, 0.0, 500),
    "two-pass path, a star and a binary tree of 80": (80, 2048, wl.star_edges(80), wl.heap_edges(80), 0.5, 0.0, 300),
    "hub kernels, broom of 64 with a hub of 41": (64, 2048, wl.broom_edges(64, bristles=40), None, 0.5, 0.0, 500),
    "cluster kernels, random tree of 64": (64, 2048, wl.random_tree_edges(64, seed=3), None, 0.5, 0.0, 500),
    "cluster kernels, random tree of 300": (300, 64, wl.random_tree_edges(300, seed=4), None, 0.5, 0.0, 400),
    # A hub of 261 workers on a 40-worker handle: diameter 40, like the random tree's.
    "hub kernels, broom of 300": (300, 64, wl.broom_edges(300, bristles=260), None, 0.5, 0.0, 400),
}


PATHS = {"tile": "tile", "double-tree kernel": "dtree", "sequential double-tree kernel": "dtree_seq",
         "cluster kernels": "cluster", "hub kernels": "cluster", "two-pass path": "two_pass",
         "double-tree cluster kernels": "cluster_dtree"}


@pytest.mark.parametrize("name", list(CASES))
def test_quadratic_training_loop(name):
    n, d, edges, edges_b, lr, beta, rounds = CASES[name]
    sys.__stderr__.write(f"[gpu] training loop {name}: n={n} d={d} rounds={rounds}\n")
    sys.__stderr__.flush()
    rng = np.random.default_rng(11)
    b = (rng.standard_normal((n, d)) + 3.0 * np.arange(n)[:, None]).astype(np.float32)
    dev = torch.device("cuda")
    bd = torch.from_numpy(b).to(dev)
    x = torch.zeros((n, d), dtype=torch.float32, device=dev)
    mom = torch.zeros_like(x) if beta else None
    xo = np.zeros((n, d), np.float32)
    mo = np.zeros((n, d), np.float32) if beta else None
    o = (oracle.Oracle(n, d, edges, np.float32) if edges_b is None
         else DoubleOracle(n, d, edges, edges_b, np.float32))
    with rs.RelaySum(n, d, edges, edges_b=edges_b) as h:
        assert h.path == PATHS[name.split(",")[0]], h.path
        for t in range(rounds):
            h.step(x, x - bd, mom, lr, beta)
            o.round(xo, xo - b, mo, lr, beta)
            if t % 100 == 99 or t == rounds - 1:
                assert bit_mismatches(x.cpu().numpy(), xo) == 0, f"{name}: round {t}"
    opt = b.astype(np.float64).mean(0)
    err = np.abs(x.cpu().numpy().astype(np.float64) - opt).max()
    assert err < 1e-4 * np.abs(opt).max(), (name, err)
