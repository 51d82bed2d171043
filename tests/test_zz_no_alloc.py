"""relaysum_step_static, the entry point that allocates nothing, against
relaysum_step on a handle: bit-identical models and momentum after every
round, for two runs in a row on one GPU, the second on a smaller input (a
new run must not see what the first left in the static buffer)."""
import ctypes

import numpy as np
import pytest

import paper_2110_04175_amd as rs
import workloads as wl

pytestmark = pytest.mark.gpu


def _bits(t):
    return t.cpu().numpy().view(np.uint32)


def _run_both(n, d, edges, rounds, lr, beta, seed):
    import torch
    dev = torch.device("cuda:0")
    gen = torch.Generator(device=dev).manual_seed(seed)
    x0 = torch.randn(n, d, generator=gen, device=dev)
    xs, xh = x0.clone(), x0.clone()
    ms = torch.zeros_like(x0) if beta != 0 else None
    mh = torch.zeros_like(x0) if beta != 0 else None
    stream = torch.cuda.current_stream()
    with rs.RelaySum(n, d, edges, stream=stream) as h:
        for t in range(rounds):
            g = torch.randn(n, d, generator=gen, device=dev)
            rs.relaysum_step_static(n, d, edges, t, xs, g, ms, lr, beta, stream=stream)
            h.step(xh, g, mh, lr, beta)
            torch.cuda.synchronize()
            assert np.array_equal(_bits(xs), _bits(xh)), f"x differs after round {t}"
            if beta != 0:
                assert np.array_equal(_bits(ms), _bits(mh)), f"mom differs after round {t}"
    return xs


def test_static_entry_matches_handle_two_runs_second_smaller():
    # Run 1: a 16-worker heap, d with a ragged tail spanning many tiles and
    # ring tiles, Nesterov momentum.
    print("static entry: run 1, heap16 d=100003", flush=True)
    _run_both(16, 100_003, wl.heap_edges(16), rounds=5, lr=0.05, beta=0.9, seed=1)
    # Run 2, right after on the same GPU: smaller (9 workers of a random
    # tree, d = 3001, plain SGD, no momentum buffer).
    print("static entry: run 2, random9 d=3001", flush=True)
    _run_both(9, 3001, wl.random_tree_edges(9, seed=4), rounds=4, lr=0.1, beta=0.0, seed=2)


def test_static_entry_two_pairs_of_workers_per_wave():
    # 32 workers: two workers per wave of the tile kernel.
    print("static entry: chain32 d=5000", flush=True)
    _run_both(32, 5000, wl.chain_edges(32), rounds=3, lr=0.1, beta=0.9, seed=3)


def test_static_entry_refuses_what_it_cannot_hold():
    import torch
    dev = torch.device("cuda:0")
    edges = wl.chain_edges(4)
    x = torch.zeros(4, 8, device=dev)
    g = torch.zeros_like(x)
    # Round 3 of a run whose round 2 is not in the buffer.
    rs.relaysum_step_static(4, 8, edges, 0, x, g, None, 0.1, 0.0)
    with pytest.raises(rs.RelaySumError) as e:
        rs.relaysum_step_static(4, 8, edges, 3, x, g, None, 0.1, 0.0)
    assert e.value.code == rs.RELAYSUM_ERR_INVALID_ARG
    # Round 1 of another tree.
    with pytest.raises(rs.RelaySumError) as e:
        rs.relaysum_step_static(4, 8, wl.star_edges(4), 1, x, g, None, 0.1, 0.0)
    assert e.value.code == rs.RELAYSUM_ERR_INVALID_ARG
    # More state than the 64 MiB buffer holds (checked before any launch).
    lib = rs.load_library()
    rc = lib.relaysum_step_static(16, 300_000, None, 0, 0, None, None, None,
                                  ctypes.c_float(0.1), ctypes.c_float(0.0), None)
    assert rc == rs.RELAYSUM_ERR_NOT_A_TREE
    e16 = np.ascontiguousarray(np.asarray(wl.chain_edges(16), np.int32))
    rc = lib.relaysum_step_static(16, 300_000, e16.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                  15, 0, 1 << 20, 2 << 40, None, ctypes.c_float(0.1),
                                  ctypes.c_float(0.0), None)
    assert rc == rs.RELAYSUM_ERR_INVALID_ARG
    assert b"static buffer" in lib.relaysum_last_error(None)
    torch.cuda.synchronize()
