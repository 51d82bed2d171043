#!/usr/bin/env python3
"""Benchmark: RelaySGD rounds/s of the HIP RelaySum round on one MI355X.

A step is one full round (local Nesterov step, message + counter relay,
count-corrected average) for all workers, i.e. one relaysum_step launch, with
every input already resident in HBM.  Default workload: chain of n=16
workers, d=9,750,000 fp32 (a VGG-11-sized flat vector), lr=0.1, momentum 0.9.

Prints ONE JSON line.  The K timed steps run in 5 back-to-back segments,
each between its own pair of HIP events on the stream the kernels run on;
`ms_per_step` and `value` come from the median segment.  The `roofline`
object prices the round's algorithmic bytes, 4*d*(5n+4E) with momentum,
against MI355X's 8 TB/s HBM peak at that duration.  `cpu_baseline` times the float32 oracle on the host on a
bounded slice of the same workload (coordinates are independent, so a slice
of d' coordinates costs d'/d of a round) and scales it to full rounds/s.

    python bench.py [--steps K] [--warmup W] [--workload chain16]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "RelaySGD rounds/s at n=16,d=9.75M fp32; achieved HBM GB/s vs peak"
HBM_PEAK_GBPS = 8000.0
PROFILES = os.path.join(ROOT, "profiles")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2110_04175_amd", "csrc", f)
                  for f in ("relaysum.hip", "tree_plan.hpp")]


def log(msg: str) -> None:
    sys.stderr.write(msg + "\n")
    sys.stderr.flush()


def code_digest() -> str:
    """sha256 of the library's sources (the kernels and the host code that
    plans their launches) with comments and whitespace removed: it changes
    when the code does, not when a comment does."""
    text = ""
    for path in KERNEL_SOURCES:
        with open(path) as f:
            text += f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    text = re.sub(r"\s+", "", text)
    return hashlib.sha256(text.encode()).hexdigest()


def measured_traffic(workload: str):
    """HBM bytes per launch from committed rocprofv3 counter runs, or None.

    profiles/*_<workload>_counters.json holds FETCH_SIZE and WRITE_SIZE (KiB
    per dispatch) for the round's kernel, the same counters for a plain
    device copy of known size (to turn counter units into bytes), and the
    digest of the kernel code they were taken on (code_digest); a changed
    kernel makes them stale, and then this is None.
    """
    import glob
    files = sorted(glob.glob(os.path.join(PROFILES, f"*_{workload}_counters.json")))
    if not files:
        return None
    try:
        with open(files[0]) as f:
            c = json.load(f)
    except (OSError, ValueError):
        return None
    if c.get("workload") != workload or c.get("kernel_code_sha256") != code_digest():
        return None
    try:
        copy_bytes = float(c["copy"]["bytes_read"])
        fetch_scale = copy_bytes / (float(c["copy"]["FETCH_SIZE_KiB"]) * 1024.0)
        write_scale = float(c["copy"]["bytes_written"]) / (float(c["copy"]["WRITE_SIZE_KiB"]) * 1024.0)
        fetch = float(c["kernel"]["FETCH_SIZE_KiB"]) * 1024.0 * fetch_scale
        write = float(c["kernel"]["WRITE_SIZE_KiB"]) * 1024.0 * write_scale
    except (KeyError, ValueError, ZeroDivisionError):
        return None
    return fetch + write


def _slot_mask(mask, slots):
    """Per-slot loss flags (library order) from an [n, n] (src, dst) mask, or
    from a [2, n, n] pair of masks on double trees (tree A's slots first)."""
    import numpy as np
    if mask.ndim == 2:
        return np.array([mask[i, j] for i, j in slots], np.uint8)
    half = len(slots) // 2
    return np.array([mask[s // half if half else 0, i, j] for s, (i, j) in enumerate(slots)],
                    np.uint8)


def cpu_baseline(w, budget_s: float = 12.0):
    """The float32 oracle, as it stands, on a slice of the workload's coordinates."""
    import numpy as np
    import oracle
    threads = host_threads()
    oracle.set_threads(threads)
    d_sample = min(w.d, 1 << 21)
    ws = w.with_d(d_sample)
    x = ws.x0("cpu").numpy().copy()
    g = ws.grad(0, "cpu").numpy()
    s1 = np.zeros_like(x)
    s2 = np.zeros_like(x)
    mask = w.drop_mask(0)
    if w.double:
        from oracle.double import DoubleOracle
        o = DoubleOracle(w.n, d_sample, w.edges, w.edges_b, np.float32)
        drops = dict(dropped_a=None if mask is None else mask[0],
                     dropped_b=None if mask is None else mask[1])
    else:
        o = oracle.Oracle(w.n, d_sample, w.edges, np.float32)
        drops = dict(dropped=mask)

    def one(t):
        o.round_ex(x, g, s1, s2, update=w.update, optimizer=w.optimizer, lr=w.lr(t) or 0.01,
                   beta1=w.beta, beta2=w.beta2, eps=w.eps, adam_step=t + 1, **drops)

    def timed(budget):
        rounds = 0
        t0 = time.perf_counter()
        while True:
            one(rounds + 1)
            rounds += 1
            el = time.perf_counter() - t0
            if (el >= budget and rounds >= 2) or rounds >= 1000:
                return rounds, el

    one(0)                                   # warm-up (page faults)
    rounds, el = timed(budget_s)
    cores = int(oracle.get_threads())
    # The same oracle on one thread (coordinates are independent, so the
    # thread count changes no result), for the per-core rate.
    oracle.set_threads(1)
    rounds1, el1 = timed(budget_s / 3)
    oracle.set_threads(threads)
    o.close()
    scale = w.d / d_sample
    return {
        "value": rounds / el / scale,
        "unit": "rounds/s",
        "cores": cores,
        "kind": "oracle",
        "sample": f"{rounds} rounds of the float32 oracle on the first {d_sample} of "
                  f"{w.d} coordinates of all {w.n} workers ({el:.1f} s), scaled by "
                  f"{w.d}/{d_sample}",
        "value_1_thread": rounds1 / el1 / scale,
        "host": host_cpu(),
    }


def host_threads() -> int:
    """Host cores this process may run on (its CPU affinity), or fewer when
    OMP_NUM_THREADS asks for fewer (a shared host may set it to the
    process's share of the CPU)."""
    try:
        cores = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        cores = os.cpu_count() or 1
    omp = os.environ.get("OMP_NUM_THREADS", "")
    if omp.isdigit() and int(omp) > 0:
        cores = min(cores, int(omp))
    return max(1, cores)


def host_cpu() -> str:
    """The host's CPU model name (as lscpu reports it), or '' if unknown."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return ""


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=300)
    ap.add_argument("--reps", type=int, default=5,
                    help="the K timed steps are split into this many equal segments, each "
                         "timed on its own; the median segment gives ms_per_step")
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="chain16",
                    help="chain4 | heap16 | chain16 | prufer256 | chain16_bert | chain16_adam | "
                         "chain16_robust10 | chain16_grad | chain16_mean | dbtree16 | dbtree64 | "
                         "chain64 | broom1000 | random8192 | dbtree200 | pa2000")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--copy-check", action="store_true",
                    help="also time a plain 2 GiB device copy (context for the roofline)")
    ap.add_argument("--graph", type=int, default=0, metavar="K",
                    help="capture K rounds (K even) into one HIP graph and time its replays "
                         "(steps must be a multiple of K); default: one relaysum_step call per round")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU only: the RelaySum round of all n workers is "
              "simulated on a single device (no collectives); use --gpus 1.",
              file=sys.stderr)
        return 2

    import numpy as np
    import torch
    import paper_2110_04175_amd as rs
    import workloads as wl

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    w = wl.workload(args.workload)
    dev = torch.device("cuda:0")
    if args.graph:
        if args.graph < 2 or args.graph % 2 or args.steps % args.graph:
            print("--graph K needs an even K >= 2 that divides --steps", file=sys.stderr)
            return 2
        if w.optimizer == "adam":
            print("--graph: Adam's bias corrections change every round, so its rounds "
                  "cannot be replayed from one graph", file=sys.stderr)
            return 2
    log(f"[bench] workload {w.name}: {w.description}")
    x = w.x0(dev)
    g = w.grad(0, dev, {})
    adam = w.optimizer == "adam"
    s1 = torch.zeros_like(x) if (adam or w.beta != 0 or w.update == "mean") else None
    s2 = torch.zeros_like(x) if adam else None
    lr = w.lr(0) if w.lr(0) != 0 else 0.01
    stream = torch.cuda.Stream(device=dev)
    torch.cuda.synchronize()

    h = rs.RelaySum(w.n, w.d, w.edges, stream=stream, edges_b=w.edges_b)
    kernel_path = h.path
    mask = w.drop_mask(0)
    drop = None
    if mask is not None:
        slots = [h.directed_edge(s) for s in range(h.num_directed_edges)]
        drop = torch.from_numpy(_slot_mask(mask, slots)).to(dev)
    plain = w.update == "model" and not adam and drop is None
    step_no = [0]

    def step():
        step_no[0] += 1
        if plain:
            h.step(x, g, s1, lr, w.beta)
        else:
            h.step_ex(x, g, s1, s2, update=w.update, optimizer=w.optimizer, lr=lr,
                      beta1=w.beta, beta2=w.beta2, eps=w.eps, adam_step=step_no[0],
                      dropped=drop)

    with torch.cuda.stream(stream):
        for _ in range(args.warmup):
            step()
    stream.synchronize()
    log(f"[bench] warmup {args.warmup} done")
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    if args.graph:
        # K rounds (a whole number of ring periods) recorded once; each
        # replay runs them with one launch.
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=stream):
            for _ in range(args.graph):
                step()
        graph.replay()
        stream.synchronize()
        with torch.cuda.stream(stream):
            start.record(stream)
            for _ in range(args.steps // args.graph):
                graph.replay()
            end.record(stream)
    else:
        # K steps in `reps` back-to-back segments, each between its own pair of
        # events on the launch stream; nothing else runs in between.
        reps = max(1, min(args.reps, args.steps))
        sizes = [args.steps // reps + (1 if r < args.steps % reps else 0) for r in range(reps)]
        marks = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
        with torch.cuda.stream(stream):
            start.record(stream)
            marks[0] = start
            for r, k in enumerate(sizes):
                for _ in range(k):
                    step()
                marks[r + 1].record(stream)
            end = marks[-1]
    end.synchronize()
    torch.cuda.synchronize()
    ms_total = start.elapsed_time(end)
    ms_per_step = ms_total / args.steps
    seg_ms = None
    if not args.graph:
        seg_ms = [marks[r].elapsed_time(marks[r + 1]) / sizes[r] for r in range(len(sizes))]
        ms_per_step = sorted(seg_ms)[len(seg_ms) // 2]
    assert bool(torch.isfinite(x).all()), "non-finite models after the timed rounds"
    log(f"[bench] {args.steps} steps in {ms_total:.2f} ms")
    h.close()

    num_edges = w.n - 1
    alg_bytes = w.bytes_per_round()
    achieved = alg_bytes / (ms_per_step * 1e-3) / 1e9
    traffic = measured_traffic(w.name)
    if traffic is not None:
        traffic = round(traffic)
    roofline = {
        "bound": "hbm",
        "achieved": round(achieved, 1),
        "peak": HBM_PEAK_GBPS,
        "unit": "GB/s",
        "frac": round(achieved / HBM_PEAK_GBPS, 4),
        "traffic": traffic,
    }

    if args.copy_check:
        a = torch.empty(1 << 29, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        s0 = torch.cuda.Event(enable_timing=True)
        s1 = torch.cuda.Event(enable_timing=True)
        s0.record()
        for _ in range(20):
            b.copy_(a)
        s1.record()
        s1.synchronize()
        gbps = 2 * a.numel() * 4 * 20 / (s0.elapsed_time(s1) * 1e-3) / 1e9
        log(f"[bench] plain device copy (2 GiB read + 2 GiB written): {gbps:.0f} GB/s")
        del a, b

    del x, g, s1, s2
    torch.cuda.empty_cache()
    cpu = None
    if not args.no_cpu_baseline:
        log("[bench] timing the oracle on the host ...")
        cpu = cpu_baseline(w, args.cpu_seconds)
        log(f"[bench] oracle: {cpu['value']:.4f} rounds/s on {cpu['cores']} threads")

    rounds_per_s = 1e3 / ms_per_step          # the median segment's rate
    metric = METRIC if w.name == "chain16" else \
        f"RelaySGD rounds/s on workload {w.name} (n={w.n}, d={w.d}) fp32; achieved HBM GB/s vs peak"
    out = {
        "metric": metric,
        "value": round(rounds_per_s, 2),
        "unit": "rounds/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "timing": {
            "segments_ms_per_step": [round(v, 5) for v in seg_ms] if seg_ms else None,
            "all_steps_ms_per_step": round(ms_total / args.steps, 5),
            "all_steps_rounds_per_s": round(args.steps / (ms_total * 1e-3), 2),
        },
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": w.description,
            "n": w.n, "d": w.d, "trees": 2 if w.double else 1, "tree_edges": num_edges,
            "lr": lr, "beta": w.beta,
            "update": w.update, "optimizer": w.optimizer, "lost_message_prob": w.drop_prob,
            "algorithmic_bytes_per_round": alg_bytes,
            "launch": (f"HIP graph of {args.graph} rounds per replay" if args.graph
                       else "one relaysum_step call per round"),
            "kernel_path": kernel_path,
        },
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
