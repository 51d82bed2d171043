"""Rounds captured into a HIP graph, and handles that share a kernel.

relaysum_create resolves every rule's kernel and launch attributes, so a
round only launches kernels: the two rounds of a ring period (parity t&1 and
its successor) can be captured into a HIP graph and replayed.  Every replay
is checked bit for bit against the same rounds run eagerly on a second
handle, with eager work (fresh gradients drawn on the device) and a
synchronisation between replays.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2110_04175_amd as rs
import workloads as wl
from parity import bit_mismatches

pytestmark = pytest.mark.gpu


def announce(msg: str) -> None:
    sys.__stderr__.write(f"[gpu] {msg}\n")
    sys.__stderr__.flush()


# (name, n, d, trees, rule): one case per kernel path; trees is "random",
# "chain", "heap", "broom", "pa" (preferential attachment) or "double".
CASES = [
    ("tile kernel", 16, 100_000, "random", "model"),
    ("tile kernel, Alg. 3 sample counts", 9, 30_000, "random", "mean"),
    ("tile kernel, spill sub-tiles", 16, 266_144, "heap", "model"),
    ("double-tree kernel", 20, 50_000, "double", "model"),
    ("cluster kernels behind a hub kernel", 100, 20_000, "broom", "model"),
    ("cluster kernels", 70, 20_000, "chain", "model"),
    ("cluster kernels after a counter launch", 100, 20_000, "random", "model"),
    ("cluster kernels, Alg. 3 sample counts", 40, 9_000, "chain", "mean"),
    ("double trees relayed in turn through LDS", 64, 20_000, "double", "model"),
    ("double-tree cluster kernels", 100, 20_000, "double", "model"),
    ("double-tree cluster kernels, Alg. 3 sample counts", 130, 4_000, "double", "mean"),
    ("two-pass path, a star and a chain", 100, 20_000, "starchain", "model"),
    ("two-pass path, a star and a chain, Alg. 3 sample counts", 90, 3_000, "starchain", "mean"),
    ("cluster kernels, 300 workers", 300, 4_000, "random", "model"),
    ("cluster kernels behind a hub kernel, 300 workers", 300, 4_000, "broom", "model"),
    ("cluster kernels behind hub kernels of every degree class", 2000, 1_000, "pa", "model"),
]
PATHS = {"tile kernel": "tile", "double-tree kernel": "dtree",
         "cluster kernels": "cluster", "double trees relayed in turn through LDS": "dtree_seq",
         "two-pass path": "two_pass", "cluster kernels behind a hub kernel": "cluster",
         "cluster kernels behind hub kernels of every degree class": "cluster",
         "double-tree cluster kernels": "cluster_dtree"}


def _round(h, x, g, s1, rule):
    if rule == "model":
        h.step(x, g, s1, 0.05, 0.9)
    else:
        h.step_ex(x, g, s1, None, update="mean")


@pytest.mark.parametrize("name,n,d,trees,rule", CASES)
def test_graph_replays_match_eager_rounds(name, n, d, trees, rule):
    announce(f"graph capture: {name} n={n} d={d}")
    dev = torch.device("cuda")
    edges_b = None
    if trees == "double":
        edges, edges_b = wl.double_binary_tree_edges(n)
    elif trees == "starchain":
        edges, edges_b = wl.star_edges(n), wl.chain_edges(n)
    elif trees == "chain":
        edges = wl.chain_edges(n)
    elif trees == "heap":
        edges = wl.heap_edges(n)
    elif trees == "pa":
        edges = wl.preferential_attachment_edges(n, 1)   # workers of 9 to 68 neighbours
    elif trees == "broom":
        edges = wl.broom_edges(n, bristles=40)   # a hub of 41: a hub kernel
    else:
        edges = wl.random_tree_edges(n, seed=n)
    gen = torch.Generator(device=dev)
    gen.manual_seed(1000 + n)
    x0 = torch.randn(n, d, device=dev, generator=gen)
    xe, xg = x0.clone(), x0.clone()
    se, sg = torch.zeros_like(x0), torch.zeros_like(x0)
    g = torch.zeros_like(x0)
    he = rs.RelaySum(n, d, edges, edges_b=edges_b)
    hg = rs.RelaySum(n, d, edges, edges_b=edges_b)
    assert he.path == PATHS[name.split(",")[0].split(" after")[0]], he.path
    graph = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        _round(hg, xg, g, sg, rule)
        _round(hg, xg, g, sg, rule)
    torch.cuda.synchronize()
    assert hg.t == 2
    assert torch.equal(xg, x0), "capture must record the rounds, not run them"
    for r in range(6):
        g.normal_(generator=gen)
        graph.replay()
        _round(he, xe, g, se, rule)
        _round(he, xe, g, se, rule)
        torch.cuda.synchronize()
        assert torch.equal(xg, xe), f"{name}: x differs after replay {r}"
        assert torch.equal(sg, se), f"{name}: state differs after replay {r}"
        ne, ce = he.counts()
        ng, cg = hg.counts()
        assert np.array_equal(ng, ne) and np.array_equal(cg, ce), f"{name}: counters, replay {r}"
        if rule == "mean":
            assert np.array_equal(hg.samples(), he.samples())
    he.close()
    hg.close()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def test_handles_sharing_a_kernel():
    """A long grid (which reserves extra LDS to keep one workgroup per CU) and
    a short grid that run the same tile kernel, stepped alternately: each
    launch keeps its own LDS size.  Both against the oracle."""
    n = 16
    edges = wl.chain_edges(n)
    dev = torch.device("cuda")
    runs = []
    for d in (1_048_576, 500_000):    # 2048 tiles (capped) and 977 tiles (not capped)
        rng = np.random.default_rng(d)
        x0 = rng.standard_normal((n, d)).astype(np.float32)
        runs.append(dict(d=d, x=torch.from_numpy(x0).to(dev), mom=torch.zeros(n, d, device=dev),
                         xo=x0.copy(), mo=np.zeros((n, d), np.float32),
                         o=oracle.Oracle(n, d, edges, np.float32), h=rs.RelaySum(n, d, edges)))
    for t in range(3):
        for run in runs:
            announce(f"shared kernel: d={run['d']} round {t}")
            g = np.random.default_rng([run["d"], t]).standard_normal((n, run["d"])).astype(np.float32)
            run["h"].step(run["x"], torch.from_numpy(g).to(dev), run["mom"], 0.05, 0.9)
            run["o"].round(run["xo"], g, run["mo"], 0.05, 0.9)
            torch.cuda.synchronize()
            assert bit_mismatches(run["x"].cpu().numpy(), run["xo"]) == 0
            assert bit_mismatches(run["mom"].cpu().numpy(), run["mo"]) == 0
    for run in runs:
        run["h"].close()
        run["o"].close()
    del runs
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _hip():
    """The HIP runtime torch has mapped (the library binds to the same one)."""
    import ctypes
    with open("/proc/self/maps") as f:
        path = next(ln.split()[-1] for ln in f if "libamdhip64" in ln)
    return ctypes.CDLL(path)


@pytest.mark.parametrize("n,trees", [(16, "random"), (100, "random"), (300, "broom")])
def test_state_calls_refuse_capture(n, trees):
    """reset, poison_next, save/load_state and the synchronising accessors
    return INVALID_ARG while the handle's stream is capturing, and record
    nothing into the graph."""
    import ctypes
    announce(f"state calls under capture: n={n}")
    hip = _hip()
    d = 1000
    edges = wl.random_tree_edges(n, seed=n) if trees == "random" else wl.broom_edges(n, bristles=40)
    stream = torch.cuda.Stream()
    x = torch.zeros(n, d, device="cuda")
    g = torch.zeros_like(x)
    with rs.RelaySum(n, d, edges, stream=stream) as h:
        h.step(x, g, None, 0.1, 0.0)
        snap = h.save_state()
        torch.cuda.synchronize()
        s = ctypes.c_void_p(stream.cuda_stream)
        assert hip.hipStreamBeginCapture(s, 2) == 0          # hipStreamCaptureModeRelaxed
        calls = [h.reset, h.poison_next, h.save_state, lambda: h.load_state(snap), h.counts,
                 h.samples, lambda: h.message(0)]
        codes = []
        for call in calls:
            try:
                call()
                codes.append(0)
            except rs.RelaySumError as e:
                codes.append(e.code)
        graph = ctypes.c_void_p()
        assert hip.hipStreamEndCapture(s, ctypes.byref(graph)) == 0
        nodes = ctypes.c_size_t(123)
        assert hip.hipGraphGetNodes(graph, None, ctypes.byref(nodes)) == 0
        hip.hipGraphDestroy(graph)
        assert codes == [rs.RELAYSUM_ERR_INVALID_ARG] * len(calls)
        assert nodes.value == 0
        # The handle is untouched and works after the capture.
        assert h.t == 1
        h.reset()
        h.step(x, g, None, 0.1, 0.0)
        torch.cuda.synchronize()
        assert h.t == 1
