"""GPU parity: the HIP RelaySum round against the oracle, through the C ABI.

Bar: counters bit-exact; x and momentum within 1e-6 max-norm relative per
worker (and, since both sides follow the same binary32 operation order, bit
identical where the test says so).  Inputs are seeded and synthetic; none
comes from the HIP path.
"""
import ctypes
import sys

import numpy as np
import pytest
import torch

import golden
import oracle
import paper_2110_04175_amd as rs
import treeutil
import workloads as wl
from parity import REL_TOL, assert_params_close, bit_mismatches

pytestmark = pytest.mark.gpu


def announce(msg: str) -> None:
    sys.__stderr__.write(f"[gpu] {msg}\n")
    sys.__stderr__.flush()


def _free():
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _slot_table(h: rs.RelaySum):
    return [h.directed_edge(s) for s in range(h.num_directed_edges)]


def check_counts(h: rs.RelaySum, o: oracle.Oracle, slots, where=""):
    nbar, cnt = h.counts()
    assert np.array_equal(nbar, o.nbars()), f"nbar differs {where}"
    want = np.array([o.count(s, t) for s, t in slots], dtype=np.int32)
    assert np.array_equal(cnt, want), f"edge counters differ {where}"


def run_case(n, d, edges, rounds, lr, beta, x0, grad, *, exact=True, check_msgs=True,
             offset=0, name=""):
    """Run `rounds` rounds on the GPU and on the float32 oracle; compare every round.

    x0: float32 numpy [n, d]; grad(t) -> float32 numpy [n, d]; lr(t) -> float.
    offset > 0 places x at a 4*offset-byte offset inside a larger buffer.
    """
    dev = torch.device("cuda")
    announce(f"{name}: n={n} d={d} rounds={rounds} beta={beta} offset={offset}")
    buf = torch.zeros(n * d + offset, dtype=torch.float32, device=dev)
    x = buf[offset:].view(n, d)
    x.copy_(torch.from_numpy(x0))
    mom = torch.zeros((n, d), dtype=torch.float32, device=dev) if beta != 0.0 else None
    xo = x0.copy()
    mo = np.zeros((n, d), np.float32)
    o = oracle.Oracle(n, d, edges, np.float32)
    with rs.RelaySum(n, d, edges) as h:
        slots = _slot_table(h)
        for t in range(rounds):
            g = grad(t)
            gd = torch.from_numpy(g).to(dev)
            h.step(x, gd, mom, lr(t), beta)
            o.round(xo, g, mo if beta != 0.0 else None, lr(t), beta)
            torch.cuda.synchronize()
            xg = x.cpu().numpy()
            assert_params_close(xg, xo, f"{name} x round {t}")
            if exact:
                assert bit_mismatches(xg, xo) == 0, f"{name} x not bit-identical at round {t}"
            if beta != 0.0:
                mg = mom.cpu().numpy()
                assert_params_close(mg, mo, f"{name} mom round {t}")
                if exact:
                    assert bit_mismatches(mg, mo) == 0, f"{name} mom not bit-identical round {t}"
            check_counts(h, o, slots, f"{name} round {t}")
            if check_msgs and d > 0:
                for s, (i, j) in enumerate(slots):
                    got = h.message(s)
                    want = o.message(i, j)
                    if exact:
                        assert bit_mismatches(got[None], want[None]) == 0, (name, t, i, j)
                    else:
                        assert_params_close(got[None], want[None], f"{name} m_{i}->{j}")
        assert h.t == rounds
    o.close()
    del x, buf, mom
    _free()


def _rng_inputs(seed, n, d, sigma=1.0):
    rng = np.random.default_rng(seed)
    x0 = rng.standard_normal((n, d)).astype(np.float32)
    means = rng.standard_normal((n, 1)).astype(np.float32)

    def grad(t):
        r = np.random.default_rng([seed, t])
        return (means + sigma * r.standard_normal((n, d))).astype(np.float32)
    return x0, grad


# ---------------------------------------------------------------------------


@pytest.mark.parametrize("name", ["lr0", "nesterov"])
def test_hand_worked_chain3_on_gpu(name):
    """The 3-worker chain worked by hand from Alg. 1 (tests/golden): the GPU
    reaches the exact values up to binary32 rounding, and the exact counters."""
    case = golden.chain3_hand_worked()[name]
    edges = np.array([[0, 1], [1, 2]], np.int32)
    x = torch.tensor([[float(v)] for v in case["x0"]], device="cuda")
    g = torch.tensor([[float(v)] for v in case["g"]], device="cuda")
    mom = torch.zeros_like(x)
    announce(f"hand-worked chain3 {name}")
    with rs.RelaySum(3, 1, edges) as h:
        # slots ordered by (src, dst): 0->1, 1->0, 1->2, 2->1, the fixture's order
        assert [h.directed_edge(s) for s in range(4)] == [(0, 1), (1, 0), (1, 2), (2, 1)]
        for r in case["rounds"]:
            h.step(x, g, mom, float(case["lr"]), float(case["beta"]))
            np.testing.assert_allclose(x.cpu().numpy()[:, 0], [float(v) for v in r["x"]],
                                       rtol=3e-7, atol=1e-7)
            nbar, cnt = h.counts()
            assert tuple(nbar) == r["nbar"] and tuple(cnt) == r["c"]
            np.testing.assert_allclose([h.message(s)[0] for s in range(4)],
                                       [float(v) for v in r["m"]], rtol=3e-7, atol=1e-7)
            if "mom" in r:
                assert [float(v) for v in mom.cpu().numpy()[:, 0]] == [float(v) for v in r["mom"]]


SMALL_CASES = []
_r = np.random.default_rng(2024)
for _k in range(24):
    _n = int(_r.integers(1, 41))
    _d = int(_r.choice([1, 3, 4, 63, 64, 65, 255, 256, 257, 1000, 1023, 2052, 4099]))
    _beta = float(_r.choice([0.0, 0.9, 0.5]))
    SMALL_CASES.append((_k, _n, _d, _beta))


@pytest.mark.parametrize("k,n,d,beta", SMALL_CASES)
def test_random_small_trees_bit_exact(k, n, d, beta):
    edges = wl.random_tree_edges(n, seed=100 + k)
    x0, grad = _rng_inputs(k, n, d)
    lr_val = float(np.float32(0.01 + 0.01 * k))
    rounds = treeutil.diameter(n, edges) + 3 if n > 1 else 3
    run_case(n, d, edges, min(rounds, 30), lambda t: lr_val, beta, x0, grad,
             name=f"random tree #{k}")


@pytest.mark.parametrize("topo,n", [("chain", 2), ("chain", 16), ("heap", 16), ("star", 9),
                                    ("chain", 32), ("heap", 33), ("star", 64)])
def test_named_topologies_bit_exact(topo, n):
    edges = {"chain": wl.chain_edges, "heap": wl.heap_edges, "star": wl.star_edges}[topo](n)
    d = 1000
    x0, grad = _rng_inputs(n, n, d)
    run_case(n, d, edges, treeutil.diameter(n, edges) + 2, lambda t: 0.05, 0.9, x0, grad,
             name=f"{topo}{n}")


def test_single_worker():
    x0, grad = _rng_inputs(1, 1, 777)
    run_case(1, 777, np.zeros((0, 2), np.int32), 5, lambda t: 0.1, 0.9, x0, grad, name="n=1")
    run_case(1, 776, np.zeros((0, 2), np.int32), 5, lambda t: 0.1, 0.0, x0[:, :776].copy(),
             lambda t: grad(t)[:, :776].copy(), name="n=1 sgd")


def test_rows_at_4_byte_alignment():
    n, d = 7, 1024
    edges = wl.random_tree_edges(n, seed=1)
    x0, grad = _rng_inputs(3, n, d)
    run_case(n, d, edges, 6, lambda t: 0.1, 0.9, x0, grad, offset=1, name="x at +4 bytes")


def test_zero_length_models_relay_counters():
    n = 12
    edges = wl.random_tree_edges(n, seed=4)
    tau = treeutil.hop_distances(n, edges)
    announce("d=0 counters only")
    with rs.RelaySum(n, 0, edges) as h:
        for t in range(int(tau.max()) + 2):
            rs.relaysum_step(h.h, None, None, None, 0.1, 0.0)
            nbar, _ = h.counts()
            assert [int(v) for v in nbar] == [treeutil.closed_form_nbar(tau, i, t)
                                              for i in range(n)]


@pytest.mark.parametrize("n,d,beta", [(400, 1000, 0.9), (400, 257, 0.0), (1000, 64, 0.9)])
def test_large_brooms_cluster_path_with_hub_kernels(n, d, beta):
    """Brooms with n/10 leaves on one worker (a hub of 41 or 101
    neighbours): the hub kernels form the hub's payload and messages ahead
    of the cluster kernel, whose members read them from the ring, and the
    completion launch finishes the hub's sum."""
    edges = wl.broom_edges(n, bristles=n // 10)
    with rs.RelaySum(n, d, edges) as h:
        assert h.path == "cluster", h.path
    x0, grad = _rng_inputs(n, n, d)
    run_case(n, d, edges, 8, lambda t: 0.02, beta, x0, grad, check_msgs=(n < 500),
             name=f"broom with a hub n={n}")


@pytest.mark.parametrize("n,d,offset", [(2500, 1_537, 0), (3000, 2_049, 1)])
def test_large_trees_with_short_ring_tiles(n, d, offset):
    """Single trees of more than 2048 workers keep 512-float ring tiles:
    several ring tiles per message, a partial last one, 4-byte rows."""
    edges = wl.random_tree_edges(n, seed=n)
    with rs.RelaySum(n, d, edges) as h:
        assert h.path == "cluster", h.path
    x0, grad = _rng_inputs(n + d, n, d)
    run_case(n, d, edges, 4, lambda t: 0.02, 0.9, x0, grad, check_msgs=True, offset=offset,
             name=f"cluster n={n} d={d}")


@pytest.mark.parametrize("n,seed,d", [(1000, 1, 1000), (2000, 1, 257)])
def test_hub_trees_cluster_path(n, seed, d):
    """Preferential-attachment trees (hubs of up to 53 and 68 neighbours):
    their workers of more than 8 neighbours join no cluster and go through
    the hub kernels of 16, 32 and 64 neighbours, the worker of 68 through
    the blocked one, ahead of the cluster kernel."""
    edges = wl.preferential_attachment_edges(n, seed)
    deg = np.bincount(edges.ravel(), minlength=n)
    assert deg.max() > 32 and ((deg > 8) & (deg <= 64)).sum() > 10
    with rs.RelaySum(n, d, edges) as h:
        assert h.path == "cluster", h.path
    x0, grad = _rng_inputs(n + seed, n, d)
    run_case(n, d, edges, 6, lambda t: 0.02, 0.9, x0, grad, check_msgs=(n <= 1000),
             name=f"pa{n} cluster with hubs")


def test_very_large_trees():
    """Trees of any size run: 5,000 workers of a random tree (the cluster
    kernels after the many-workgroup counter launch) and of a broom with a hub
    of 501 (the cluster kernels behind the blocked hub kernel) against the
    oracle, and a chain of 12,000 workers against its
    closed-form counters (nbar_i after round t counts the workers within t+1
    hops)."""
    n = 5000
    for edges, path in ((wl.random_tree_edges(n, seed=77), "cluster"),
                        (wl.broom_edges(n, bristles=500), "cluster")):
        with rs.RelaySum(n, 16, edges) as h:
            assert h.path == path, h.path
        x0, grad = _rng_inputs(77, n, 16)
        run_case(n, 16, edges, 4, lambda t: 0.05, 0.9, x0, grad, check_msgs=False,
                 name=f"{path} n=5000")
    n, d = 12000, 8
    announce(f"chain n={n} counters")
    x = torch.randn(n, d, device="cuda")
    g = torch.randn(n, d, device="cuda")
    with rs.RelaySum(n, d, wl.chain_edges(n)) as h:
        assert h.path == "cluster", h.path
        for t in range(5):
            h.step(x, g, None, 0.1, 0.0)
            nbar, _ = h.counts()
            i = np.arange(n)
            want = np.minimum(i, t + 1) + np.minimum(n - 1 - i, t + 1) + 1
            assert np.array_equal(nbar, want), t
    assert bool(torch.isfinite(x).all())


@pytest.mark.parametrize("n", [33, 100, 256, 300, 1000])
def test_random_trees(n):
    """Random trees of 33 to 1000 workers (degrees 4 to 8) take the cluster
    kernels after a counter launch, with up to 8 previous messages per worker
    in registers."""
    edges = wl.random_tree_edges(n, seed=n + 1)
    x0, grad = _rng_inputs(n, n, 700)
    run_case(n, 700, edges, 6, lambda t: 0.02, 0.9, x0, grad, check_msgs=(n <= 100),
             name=f"random tree n={n}")


@pytest.mark.parametrize("topo,n,d,offset", [("chain", 33, 2_000, 0), ("chain", 47, 1_001, 1),
                                             ("chain", 256, 600, 0), ("heap", 255, 513, 2),
                                             ("heap", 63, 4_100, 0), ("chain", 700, 300, 0),
                                             ("heap", 4096, 40, 1)])
def test_cluster_kernels(topo, n, d, offset):
    """Chains and binary trees of more than 32 workers (degrees at most 3)
    run as clusters of at most 16 workers: cluster sizes that leave waves
    idle (33, 47 workers), full clusters (256), 4-byte rows with partial last
    chunks, the boundary workers completed by the second launch, and trees
    of more than 256 workers, whose counters come from a launch before (a
    chain of 700, a binary tree of 4096)."""
    edges = {"chain": wl.chain_edges, "heap": wl.heap_edges}[topo](n)
    x0, grad = _rng_inputs(n + d, n, d)
    run_case(n, d, edges, 5, lambda t: 0.03, 0.9, x0, grad, check_msgs=(n <= 64), offset=offset,
             name=f"cluster {topo} n={n}")


@pytest.mark.parametrize("topo,n,d,offset", [("random", 17, 9_001, 1), ("random", 32, 4_099, 0),
                                             ("random", 33, 1_025, 1), ("random", 256, 513, 0),
                                             ("broom", 48, 1_025, 1), ("broom", 256, 513, 2)])
def test_unaligned_rows_fast_paths(topo, n, d, offset):
    """Rows only 4-byte aligned or d % 4 != 0: the tile kernel with 16-byte
    chunks at 4-byte alignment and a float-by-float tail (17 and 32 workers),
    the cluster kernels' float-by-float boundary launch (random trees of 33
    and 256 workers, and brooms of 48 and 256 workers behind a hub kernel,
    whose members read the hub's messages float by float), several tiles and
    a ragged tail."""
    if topo == "broom":
        edges = wl.broom_edges(n, bristles=40)   # a hub of 41 neighbours: a hub kernel
    else:
        edges = wl.random_tree_edges(n, seed=n + 11)
    x0, grad = _rng_inputs(n + 11, n, d)
    run_case(n, d, edges, 5, lambda t: 0.03, 0.9, x0, grad, check_msgs=(n <= 33),
             offset=offset, name=f"unaligned rows n={n} d={d}")


@pytest.mark.parametrize("n,d,offset", [(16, 2_500_001, 0), (32, 1_000_003, 1),
                                        (32, 1_000_000, 0), (16, 2_000_000, 2)])
def test_tile_kernel_streaming_sizes(n, d, offset):
    """Rounds whose working set exceeds half the 256 MB MALL take the tile
    kernel's non-temporal variant (smaller ones, as in every other tile test,
    the cache-allocating one): d % 4 != 0 (every row's last chunk partial),
    with rows only 4-byte aligned, 16-byte aligned rows with two workers per
    wave, and d % 4 == 0 on rows 8 bytes off 16-byte alignment; every
    coordinate against the oracle."""
    edges = wl.random_tree_edges(n, seed=n + 23)
    x0, grad = _rng_inputs(n + 23, n, d)
    run_case(n, d, edges, 3, lambda t: 0.05, 0.9, x0, grad, check_msgs=False, offset=offset,
             name=f"streaming tile kernel n={n} d={d}")


@pytest.mark.parametrize("topo,n", [("star", 60), ("broom", 64), ("broom", 200), ("star", 130)])
def test_hub_topologies_cluster_path(topo, n):
    """Trees with a hub take the cluster kernels behind the hub kernels,
    which form a hub's payload and out-messages first: a centre of degree
    59 (the 64-neighbour class; its leaves, 16 to a cluster, read its
    messages from the ring), brooms (a chain of 24 or 160 workers whose last
    worker carries 40 more leaves: the 64-neighbour class on a long handle)
    and a centre of degree 129 (the kernel for more than 64 neighbours, in
    blocks of 64)."""
    edges = wl.star_edges(n) if topo == "star" else wl.broom_edges(n, bristles=40)
    x0, grad = _rng_inputs(n + 7, n, 1028)
    with rs.RelaySum(n, 1028, edges) as h:
        assert h.path == "cluster", h.path
    run_case(n, 1028, edges, 5, lambda t: 0.05, 0.9, x0, grad, check_msgs=(n <= 64),
             name=f"hub kernels {topo} n={n}")


def test_denormal_inputs_bit_exact():
    n, d = 5, 512
    edges = wl.chain_edges(n)
    rng = np.random.default_rng(9)
    tiny = np.float32(1e-39)   # binary32 subnormal
    x0 = (rng.standard_normal((n, d)) * tiny).astype(np.float32)
    g0 = (rng.standard_normal((n, d)) * tiny).astype(np.float32)
    assert (np.abs(x0[x0 != 0]) < np.finfo(np.float32).tiny).all()
    run_case(n, d, edges, 6, lambda t: 0.5, 0.9, x0, lambda t: g0, name="subnormals")


def test_reset_and_determinism():
    n, d = 16, 4096
    edges = wl.heap_edges(n)
    x0, grad = _rng_inputs(5, n, d)
    announce("reset/determinism")
    outs = []
    with rs.RelaySum(n, d, edges) as h:
        for rep in range(2):
            x = torch.from_numpy(x0).cuda()
            mom = torch.zeros_like(x)
            for t in range(9):
                h.step(x, torch.from_numpy(grad(t)).cuda(), mom, 0.05, 0.9)
            outs.append((x.cpu().numpy(), mom.cpu().numpy(), h.counts()))
            h.reset()
            assert h.t == 0
            nbar, cnt = h.counts()
            assert (nbar == 0).all() and (cnt == 0).all()
    assert np.array_equal(outs[0][0], outs[1][0]) and np.array_equal(outs[0][1], outs[1][1])
    _free()


def test_side_stream():
    n, d = 8, 3000
    edges = wl.chain_edges(n)
    x0, grad = _rng_inputs(6, n, d)
    announce("side stream")
    s = torch.cuda.Stream()
    res = []
    for use_side in (False, True):
        with rs.RelaySum(n, d, edges) as h:
            x = torch.from_numpy(x0).cuda()
            mom = torch.zeros_like(x)
            gs = [torch.from_numpy(grad(t)).cuda() for t in range(5)]
            torch.cuda.synchronize()
            if use_side:
                h.set_stream(s)
                with torch.cuda.stream(s):
                    for t in range(5):
                        h.step(x, gs[t], mom, 0.1, 0.9)
                s.synchronize()
            else:
                for t in range(5):
                    h.step(x, gs[t], mom, 0.1, 0.9)
            res.append(x.cpu().numpy())
    assert np.array_equal(res[0], res[1])


def test_step_argument_errors():
    n, d = 4, 64
    announce("argument errors")
    with rs.RelaySum(n, d, wl.chain_edges(n)) as h:
        x = torch.zeros((n, d), device="cuda")
        g = torch.zeros((n, d), device="cuda")
        with pytest.raises(rs.RelaySumError) as e:
            rs.relaysum_step(h.h, x, g, None, 0.1, 0.9)         # momentum buffer missing
        assert e.value.code == rs.RELAYSUM_ERR_INVALID_ARG
        with pytest.raises(rs.RelaySumError) as e:
            rs.relaysum_step(h.h, x, None, None, 0.1, 0.0)      # no gradient
        assert e.value.code == rs.RELAYSUM_ERR_INVALID_ARG
        with pytest.raises(rs.RelaySumError) as e:
            rs.relaysum_step(h.h, x.data_ptr() + 2, g, None, 0.1, 0.0)   # not 4-byte aligned
        assert e.value.code == rs.RELAYSUM_ERR_INVALID_ARG
        assert h.t == 0   # failed calls do not advance the round
        with pytest.raises(rs.RelaySumError):
            h.directed_edge(6)


class _PtrAttr(ctypes.Structure):
    """hipPointerAttribute_t."""
    _fields_ = [("type", ctypes.c_int), ("device", ctypes.c_int),
                ("devicePointer", ctypes.c_void_p), ("hostPointer", ctypes.c_void_p),
                ("isManaged", ctypes.c_int), ("allocationFlags", ctypes.c_uint)]


def test_arrays_outside_device_memory_are_refused():
    """Host memory (pinned or pageable), a loss mask in host memory and device
    buffers too short for n*d floats are refused before any kernel runs.  Each
    case is first confirmed with the runtime's own pointer queries, so that a
    wrong acceptance could never reach a kernel with such a pointer."""
    hip = ctypes.CDLL("libamdhip64.so")
    hip.hipPointerGetAttributes.argtypes = [ctypes.POINTER(_PtrAttr), ctypes.c_void_p]
    hip.hipMemGetAddressRange.argtypes = [ctypes.POINTER(ctypes.c_void_p),
                                          ctypes.POINTER(ctypes.c_size_t), ctypes.c_void_p]
    n, d = 4, 1024
    announce("arrays outside device memory")

    def kind(ptr):
        at = _PtrAttr()
        rc = hip.hipPointerGetAttributes(ctypes.byref(at), ctypes.c_void_p(ptr))
        hip.hipGetLastError()
        return None if rc != 0 else at.type

    def refused(call, what):
        with pytest.raises(rs.RelaySumError) as e:
            call()
        assert e.value.code == rs.RELAYSUM_ERR_INVALID_ARG
        assert what in str(e.value), str(e.value)

    with rs.RelaySum(n, d, wl.chain_edges(n)) as h:
        x = torch.zeros((n, d), device="cuda")
        g = torch.zeros((n, d), device="cuda")
        mom = torch.zeros((n, d), device="cuda")
        assert kind(x.data_ptr()) == 2   # device memory
        pinned = torch.zeros((n, d), pin_memory=True)
        assert kind(pinned.data_ptr()) == 1   # host memory
        refused(lambda: rs.relaysum_step(h.h, pinned.data_ptr(), g, mom, 0.1, 0.9), "x is not")
        refused(lambda: rs.relaysum_step(h.h, x, g, pinned.data_ptr(), 0.1, 0.9), "state1 is not")
        pageable = torch.zeros((n, d))
        assert kind(pageable.data_ptr()) in (None, 0, 1)
        refused(lambda: rs.relaysum_step(h.h, x, pageable.data_ptr(), mom, 0.1, 0.9), "g is not")
        mask = torch.zeros(2 * (n - 1), dtype=torch.uint8, pin_memory=True)
        assert kind(mask.data_ptr()) == 1
        refused(lambda: rs.relaysum_step_ex(h.h, x, g, mom, None, update="robust", lr=0.1,
                                            beta1=0.9, dropped=mask.data_ptr()), "dropped is not")
        # A device pointer whose n*d floats would run 4 bytes past the end of
        # the allocation that holds it.
        big = torch.zeros(1 << 20, device="cuda")
        base, size = ctypes.c_void_p(), ctypes.c_size_t()
        assert hip.hipMemGetAddressRange(ctypes.byref(base), ctypes.byref(size),
                                         ctypes.c_void_p(big.data_ptr())) == 0
        assert base.value and size.value >= n * d * 4
        short = base.value + size.value - n * d * 4 + 4
        refused(lambda: rs.relaysum_step(h.h, short, g, mom, 0.1, 0.9), "x is not")
        refused(lambda: rs.relaysum_step(h.h, x, short, mom, 0.1, 0.9), "g is not")
        refused(lambda: rs.relaysum_step_static(n, d, wl.chain_edges(n), 0, pinned.data_ptr(), g,
                                                mom, 0.1, 0.9), "x is not")
        assert h.t == 0
        h.step(x, g, mom, 0.1, 0.9)    # the same handle still runs on device arrays
        torch.cuda.synchronize()
        assert h.t == 1


# ---------------------------------------------------------------------------
# The five workloads.  chain4 and heap16: every coordinate, every round.
# chain16, prufer256, chain16_bert: full-size GPU runs in the launch shape the
# benchmark times, checked on sampled coordinates (each coordinate of the
# round is independent, so the oracle runs on the sampled columns alone).
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("name", ["chain4", "heap16"])
def test_workload_full_compare(name):
    w = wl.workload(name)
    announce(f"workload {name} full")
    dev = torch.device("cuda")
    state = {}
    x = w.x0(dev)
    mom = torch.zeros_like(x) if w.beta != 0 else None
    xo = x.cpu().numpy().copy()
    mo = np.zeros_like(xo)
    o = oracle.Oracle(w.n, w.d, w.edges, np.float32)
    with rs.RelaySum(w.n, w.d, w.edges) as h:
        slots = _slot_table(h)
        for t in range(w.rounds):
            g = w.grad(t, dev, state)
            h.step(x, g, mom, w.lr(t), w.beta)
            o.round(xo, g.cpu().numpy(), mo if w.beta != 0 else None, w.lr(t), w.beta)
            xg = x.cpu().numpy()
            assert_params_close(xg, xo, f"{name} x round {t}")
            assert bit_mismatches(xg, xo) == 0
            if w.beta != 0:
                assert_params_close(mom.cpu().numpy(), mo, f"{name} mom round {t}")
            check_counts(h, o, slots, f"{name} round {t}")
    o.close()
    _free()


FULL_SIZE_PATHS = {"chain16": "tile", "prufer256": "cluster", "chain16_bert": "tile",
                   "chain64": "cluster", "broom1000": "cluster", "random8192": "cluster",
                   "pa2000": "cluster"}


@pytest.mark.parametrize("name", list(FULL_SIZE_PATHS))
def test_workload_full_size_sampled(name):
    w = wl.workload(name)
    announce(f"workload {name} full size, sampled parity")
    dev = torch.device("cuda")
    idx_np = wl.sample_columns(w.d, 4096)
    idx = torch.from_numpy(idx_np).to(dev)
    state = {}
    x = w.x0(dev)
    mom = torch.zeros_like(x)
    xo = x.index_select(1, idx).cpu().numpy().copy()
    mo = np.zeros_like(xo)
    o = oracle.Oracle(w.n, len(idx_np), w.edges, np.float32)
    tau = treeutil.hop_distances(w.n, w.edges)
    diam = int(tau.max())
    worst = 0.0
    mism = 0
    with rs.RelaySum(w.n, w.d, w.edges) as h:
        assert h.path == FULL_SIZE_PATHS[name], h.path
        slots = _slot_table(h)
        for t in range(w.rounds):
            g = w.grad(t, dev, state)
            h.step(x, g, mom, w.lr(t), w.beta)
            o.round(xo, g.index_select(1, idx).cpu().numpy(), mo, w.lr(t), w.beta)
            del g
            xg = x.index_select(1, idx).cpu().numpy()
            mg = mom.index_select(1, idx).cpu().numpy()
            assert_params_close(xg, xo, f"{name} x round {t}")
            assert_params_close(mg, mo, f"{name} mom round {t}")
            worst = max(worst, float(np.max(np.abs(xg.astype(np.float64) - xo))))
            mism += bit_mismatches(xg, xo) + bit_mismatches(mg, mo)
            check_counts(h, o, slots, f"{name} round {t}")
            if t + 1 >= diam:
                assert (h.counts()[0] == w.n).all()
        # a few full messages of the last round, sampled
        for s in (0, len(slots) // 2, len(slots) - 1):
            i, j = slots[s]
            got = h.message(s)[idx_np]
            assert bit_mismatches(got[None], o.message(i, j)[None]) == 0
    announce(f"{name}: max |x_gpu - x_oracle| = {worst:.3e}, bit mismatches = {mism}")
    assert mism == 0
    o.close()
    del x, mom
    _free()
