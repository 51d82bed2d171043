"""GPU parity for every update rule and local optimizer, with and without
lost messages: the HIP round (relaysum_step_ex) against the oracle's
extended round, bit for bit, on the 128-bit tile path (chain of 16, heap of
16), the 32-bit tile path (misaligned rows), the cluster kernels with
counters relayed per workgroup (a chain of 70 workers; a binary tree of 100
on 4-byte rows with a partial last chunk) and with counters from a launch
before (random trees of 40, 130 and 300 workers, 16-byte and 4-byte rows) and
behind the hub kernels (brooms of 48, 130 and 300 workers with a hub of 41,
a broom of 400 with a hub of 101 and preferential-attachment trees of 1000,
16-byte and 4-byte rows; trees of 2,100 workers in clusters of 32), and tile-kernel grids just past the workgroups resident at
once, whose excess coordinates run as spill sub-tiles.  Each shape asserts
the kernel path its name promises."""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2110_04175_amd as rs
import treeutil
import workloads as wl
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
SHAPES = {
    "chain16": (16, wl.chain_edges(16), 3000, 0),
    "heap16": (16, wl.heap_edges(16), 2052, 0),
    "rand9-misaligned": (9, wl.random_tree_edges(9, seed=3), 1001, 1),
    "broom48-hubs": (48, wl.broom_edges(48, bristles=40), 1500, 0),
    "broom130-hubs": (130, wl.broom_edges(130, bristles=40), 1028, 0),
    "broom48-hubs-misaligned": (48, wl.broom_edges(48, bristles=40), 1501, 1),
    "rand40-cluster": (40, wl.random_tree_edges(40, seed=4), 1500, 0),
    "rand130-cluster-misaligned": (130, wl.random_tree_edges(130, seed=5), 1027, 1),
    "chain70-cluster": (70, wl.chain_edges(70), 1500, 0),
    "heap100-cluster-misaligned": (100, wl.heap_edges(100), 1027, 1),
    "rand300-cluster": (300, wl.random_tree_edges(300, seed=6), 600, 0),
    "broom300-hubs": (300, wl.broom_edges(300, bristles=40), 600, 0),
    "broom300-hubs-misaligned": (300, wl.broom_edges(300, bristles=40), 601, 1),
    # Short grids just past a whole number of dispatch rounds (256 or 512
    # workgroups resident at once for 16 waves per workgroup, depending on
    # the rule's registers; 768 or 1024 for 8): the tile kernel's spill
    # sub-tiles take the excess.
    "heap16-spill512": (16, wl.heap_edges(16), 266_144, 0),
    "heap16-spill256-misaligned": (16, wl.heap_edges(16), 135_075, 1),
    "star16-spill512": (16, wl.star_edges(16), 270_000, 0),
    "rand8-spill1024-misaligned": (8, wl.random_tree_edges(8, seed=8), 530_001, 1),
    "rand8-spill768": (8, wl.random_tree_edges(8, seed=9), 400_000, 0),
    "chain32-spill256": (32, wl.chain_edges(32), 140_000, 0),
    # preferential attachment: workers of 9 to 53 neighbours through the hub
    # kernels ahead of the cluster kernel
    "pa1000-hubs": (1000, wl.preferential_attachment_edges(1000, 1), 300, 0),
    "pa1000-hubs-misaligned": (1000, wl.preferential_attachment_edges(1000, 1), 301, 1),
    # a hub of 101 neighbours: the blocked hub kernel (blocks of 64 out-messages),
    # whose completion walks 101 messages
    "broom400-bighub": (400, wl.broom_edges(400, bristles=100), 300, 0),
    "broom400-bighub-misaligned": (400, wl.broom_edges(400, bristles=100), 301, 1),
    # 2,048 workers or more: clusters of 32, two members per wave (with hubs,
    # and on 4-byte rows with a partial last chunk)
    "pa2100-hubs": (2100, wl.preferential_attachment_edges(2100, 3), 300, 0),
    "rand2100-cluster-misaligned": (2100, wl.random_tree_edges(2100, seed=12), 130, 1),
    # three dispatch rounds of 256 workgroups and a spill (rules whose
    # registers leave one 16-wave workgroup per CU)
    "rand16-spill3x256": (16, wl.random_tree_edges(16, seed=10), 398_216, 0),
}


def announce(msg):
    sys.__stderr__.write(f"[gpu] {msg}\n")
    sys.__stderr__.flush()


def shape_path(shape):
    """The kernel path a shape's name promises."""
    for tag, path in (("-cluster", "cluster"), ("-hubs", "cluster"), ("-bighub", "cluster")):
        if tag in shape:
            return path
    return "tile"


def run_rule(shape, update, optimizer, kw, p_drop, rounds=None, seed=0):
    n, edges, d, offset = SHAPES[shape]
    diam = treeutil.diameter(n, edges)
    rounds = rounds or diam + 3
    announce(f"{shape} {update}/{optimizer} {kw} p_drop={p_drop} n={n} d={d} rounds={rounds}")
    rng = np.random.default_rng(seed)
    dev = torch.device("cuda")
    x0 = rng.standard_normal((n, d)).astype(np.float32)
    uses_s1 = optimizer == "adam" or kw.get("beta1", 0.0) != 0.0 or update == "mean"
    uses_s2 = optimizer == "adam"

    def dev_buf(arr):
        b = torch.zeros(n * d + offset, dtype=torch.float32, device=dev)
        v = b[offset:].view(n, d)
        v.copy_(torch.from_numpy(arr))
        return b, v

    bx, x = dev_buf(x0 if update != "mean" else np.zeros_like(x0))
    b1, s1 = dev_buf(np.zeros_like(x0)) if uses_s1 else (None, None)
    b2, s2 = dev_buf(np.zeros_like(x0)) if uses_s2 else (None, None)
    xo = (x0 if update != "mean" else np.zeros_like(x0)).copy()
    o1 = np.zeros_like(x0) if uses_s1 else None
    o2 = np.zeros_like(x0) if uses_s2 else None
    o = oracle.Oracle(n, d, edges, np.float32)
    with rs.RelaySum(n, d, edges) as h:
        assert h.path == shape_path(shape), h.path
        slots = [h.directed_edge(s) for s in range(h.num_directed_edges)]
        for t in range(rounds):
            g = rng.standard_normal((n, d)).astype(np.float32)
            bg, gd = dev_buf(g)
            mask = (rng.random((n, n)) < p_drop).astype(np.uint8) if p_drop else None
            drop_dev = None
            if mask is not None:
                per_slot = np.array([mask[i, j] for i, j in slots], np.uint8)
                drop_dev = torch.from_numpy(per_slot).to(dev)
            step = t + 1
            rs.relaysum_step_ex(h.h, x, gd, s1, s2, update=update, optimizer=optimizer,
                                adam_step=step, dropped=drop_dev, **kw)
            o.round_ex(xo, g, o1, o2, update=update, optimizer=optimizer, adam_step=step,
                       dropped=mask, **kw)
            torch.cuda.synchronize()
            xg = x.cpu().numpy()
            assert_params_close(xg, xo, f"{shape} {update} x round {t}")
            assert bit_mismatches(xg, xo) == 0, f"x not bit-identical at round {t}"
            if uses_s1:
                assert bit_mismatches(s1.cpu().numpy(), o1) == 0, f"state1 differs at round {t}"
            if uses_s2:
                assert bit_mismatches(s2.cpu().numpy(), o2) == 0, f"state2 differs at round {t}"
            nbar, cnt = h.counts()
            assert np.array_equal(nbar, o.nbars()), f"nbar differs at round {t}"
            assert np.array_equal(cnt, [o.count(i, j) for i, j in slots])
            if update == "mean":
                assert list(h.samples()) == [o.samples(i) for i in range(n)]
            if t == rounds - 1:
                for s_, (i, j) in enumerate(slots[:6]):
                    assert bit_mismatches(h.message(s_)[None], o.message(i, j)[None]) == 0
    o.close()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("shape", list(SHAPES))
@pytest.mark.parametrize("rule", range(len(RULES)), ids=RULE_IDS)
def test_rule_without_losses(rule, shape):
    update, optimizer, kw = RULES[rule]
    run_rule(shape, update, optimizer, kw, 0.0, seed=rule)


@pytest.mark.parametrize("shape", ["chain16", "heap16", "rand9-misaligned", "broom48-hubs",
                                   "broom130-hubs", "broom48-hubs-misaligned", "chain70-cluster",
                                   "heap100-cluster-misaligned", "rand40-cluster",
                                   "rand130-cluster-misaligned",
                                   "rand300-cluster", "broom300-hubs",
                                   "broom300-hubs-misaligned", "heap16-spill512",
                                   "heap16-spill256-misaligned", "chain32-spill256",
                                   "pa1000-hubs", "broom400-bighub", "pa2100-hubs",
                                   "rand2100-cluster-misaligned"])
@pytest.mark.parametrize("rule", [0, 1, 2, 3, 4, 5, 7], ids=[RULE_IDS[i] for i in (0, 1, 2, 3, 4, 5, 7)])
def test_rule_with_lost_messages(rule, shape):
    update, optimizer, kw = RULES[rule]
    run_rule(shape, update, optimizer, kw, 0.15, seed=100 + rule)


def test_step_ex_argument_errors():
    n, d = 4, 64
    with rs.RelaySum(n, d, wl.chain_edges(n)) as h:
        x = torch.zeros((n, d), device="cuda")
        g = torch.zeros((n, d), device="cuda")
        for kw in (dict(update="grad", beta1=0.9), dict(update="grad", optimizer="adam"),
                   dict(update="model", optimizer="adam", adam_step=0),
                   dict(update="mean")):
            with pytest.raises(rs.RelaySumError) as e:
                rs.relaysum_step_ex(h.h, x, g, None, None, **kw)
            assert e.value.code == rs.RELAYSUM_ERR_INVALID_ARG
        # loss masks of the wrong length, type or device never reach a kernel
        for bad in (torch.zeros(5, dtype=torch.uint8, device="cuda"),
                    torch.zeros(6, dtype=torch.int32, device="cuda"),
                    torch.zeros(6, dtype=torch.uint8)):
            with pytest.raises((ValueError, TypeError)):
                h.step_ex(x, g, update="robust", lr=0.1, dropped=bad)
        assert h.t == 0
        # arrays that share bytes would mix a round's inputs with its outputs
        buf = torch.zeros(2 * n * d, device="cuda")
        a, b = buf[: n * d].view(n, d), buf[d: d + n * d].view(n, d)
        for args in ((x, x, None, None), (a, b, None, None)):
            with pytest.raises(rs.RelaySumError) as e:
                rs.relaysum_step_ex(h.h, *args, update="model", lr=0.1)
            assert e.value.code == rs.RELAYSUM_ERR_INVALID_ARG
        with pytest.raises(rs.RelaySumError):
            h.step_ex(x, g, a, b, update="model", optimizer="adam", lr=0.1, adam_step=1)
        assert h.t == 0
        h.step_ex(x, g, buf[: n * d].view(n, d), buf[n * d:].view(n, d), update="model",
                  optimizer="adam", lr=0.1, adam_step=1)    # adjacent, not shared: accepted
        torch.cuda.synchronize()
        assert h.t == 1


@pytest.mark.parametrize("name", ["chain16_adam", "chain16_robust10", "chain16_grad",
                                  "chain16_mean"])
def test_rule_workloads_full_size_sampled(name):
    """The workloads of the other rules at full size, in the launch shape the
    benchmark times, checked on sampled coordinates against the oracle."""
    w = wl.workload(name)
    announce(f"workload {name} full size, sampled parity")
    dev = torch.device("cuda")
    idx_np = wl.sample_columns(w.d, 4096)
    idx = torch.from_numpy(idx_np).to(dev)
    state = {}
    adam = w.optimizer == "adam"
    x = w.x0(dev) if w.update != "mean" else torch.zeros((w.n, w.d), device=dev)
    s1 = torch.zeros_like(x) if (adam or w.beta != 0 or w.update == "mean") else None
    s2 = torch.zeros_like(x) if adam else None
    xo = x.index_select(1, idx).cpu().numpy().copy()
    o1 = np.zeros_like(xo) if s1 is not None else None
    o2 = np.zeros_like(xo) if s2 is not None else None
    o = oracle.Oracle(w.n, len(idx_np), w.edges, np.float32)
    mism = 0
    with rs.RelaySum(w.n, w.d, w.edges) as h:
        slots = [h.directed_edge(s) for s in range(h.num_directed_edges)]
        for t in range(w.rounds):
            g = w.grad(t, dev, state)
            mask = w.drop_mask(t)
            drop = None
            if mask is not None:
                drop = torch.from_numpy(np.array([mask[i, j] for i, j in slots], np.uint8)).to(dev)
            kw = dict(update=w.update, optimizer=w.optimizer, lr=w.lr(t), beta1=w.beta,
                      beta2=w.beta2, eps=w.eps, adam_step=t + 1)
            h.step_ex(x, g, s1, s2, dropped=drop, **kw)
            o.round_ex(xo, g.index_select(1, idx).cpu().numpy(), o1, o2, dropped=mask, **kw)
            del g
            xg = x.index_select(1, idx).cpu().numpy()
            assert_params_close(xg, xo, f"{name} x round {t}")
            mism += bit_mismatches(xg, xo)
            if s1 is not None:
                mism += bit_mismatches(s1.index_select(1, idx).cpu().numpy(), o1)
            nbar, cnt = h.counts()
            assert np.array_equal(nbar, o.nbars())
            assert np.array_equal(cnt, [o.count(i, j) for i, j in slots])
    announce(f"{name}: bit mismatches = {mism}")
    assert mism == 0
    o.close()
    del x, s1, s2
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def test_mean_estimation_up_to_the_divisor_limit():
    """Alg. 3 on a chain of 1024 workers for the 16,639 rounds the library's
    bound of the sample counts allows (the sum over rounds of the workers
    within t+1 hops stays within 2^24, where s_i converts to binary32
    exactly), then the next round is refused with INVALID_ARG and changes
    nothing, also on a handle resumed from a snapshot.  With 0/1 samples
    every sum is an exact integer, so the closed forms check the GPU:
    worker k's sample of round r reaches i after delta_ik = max(|i-k|-1, 0)
    rounds, so after T rounds s_i = sum_k max(0, T - delta_ik), y_i =
    sum_k g_k max(0, T - delta_ik), and x_i = y_i / s_i rounded once."""
    from test_oracle_pins_ext import round_to_float32
    from fractions import Fraction as F
    n, d, rounds = 1024, 8, 16639
    edges = wl.chain_edges(n)
    announce(f"mean estimation to the divisor limit: chain n={n} d={d} rounds={rounds}")
    rng = np.random.default_rng(1024)
    g_np = rng.integers(0, 2, (n, d)).astype(np.float32)
    dev = torch.device("cuda")
    g = torch.from_numpy(g_np).to(dev)
    x = torch.zeros(n, d, device=dev)
    y = torch.zeros(n, d, device=dev)
    with rs.RelaySum(n, d, edges) as h:
        for t in range(rounds):
            h.step_ex(x, g, y, update="mean")
        torch.cuda.synchronize()
        s = h.samples()
        i = np.arange(n)
        w = np.maximum(0, rounds - np.maximum(np.abs(i[:, None] - i[None, :]) - 1, 0))   # [i, k]
        assert np.array_equal(s, w.sum(axis=1))
        assert s.max() <= 1 << 24
        yg, xg = y.cpu().numpy(), x.cpu().numpy()
        assert np.array_equal(yg.astype(np.int64), w @ g_np.astype(np.int64))
        for r in range(0, n, 31):
            for c in range(d):
                assert xg[r, c] == round_to_float32(F(int(yg[r, c]), int(s[r]))), (r, c)
        snap = h.save_state()
        with pytest.raises(rs.RelaySumError) as e:
            h.step_ex(x, g, y, update="mean")
        assert e.value.code == rs.RELAYSUM_ERR_INVALID_ARG and h.t == rounds
        torch.cuda.synchronize()
        assert np.array_equal(x.cpu().numpy(), xg) and np.array_equal(y.cpu().numpy(), yg)
        # Other rules do not add samples, so they still run.
        h.step_ex(x, g, update="grad", lr=0.0)
    with rs.RelaySum(n, d, edges) as h2:
        h2.load_state(snap)
        with pytest.raises(rs.RelaySumError):
            h2.step_ex(x, g, y, update="mean")
