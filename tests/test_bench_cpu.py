"""bench.py's host logic (CPU): the one-GPU contract, the digest that ties
committed counters to the kernel code, the counter-to-bytes scaling and the
per-slot loss masks of double trees."""
import json
import os
import subprocess
import sys

import numpy as np

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_code_digest_ignores_comments_and_whitespace(tmp_path, monkeypatch):
    def digest(text, plan="int g(int y) { return y; }\n"):
        p = tmp_path / "k.hip"
        p.write_text(text)
        q = tmp_path / "plan.hpp"
        q.write_text(plan)
        monkeypatch.setattr(bench, "KERNEL_SOURCES", [str(p), str(q)])
        return bench.code_digest()

    a = digest("int f(int x) { return x + 1; }  // one\n")
    b = digest("/* header\n comment */\nint f(int x)\n{\n    return x + 1;\n}\n")
    c = digest("int f(int x) { return x + 2; }\n")
    e = digest("int f(int x) { return x + 1; }\n", plan="int g(int y) { return y + 1; }\n")
    assert a == b and a != c and a != e


def _write_counters(folder, workload, sha, kernel_fetch_kib, kernel_write_kib):
    copy_bytes = 1 << 31
    rec = {
        "workload": workload,
        "kernel_code_sha256": sha,
        # a copy kernel of known size: FETCH_SIZE counts half the bytes read,
        # WRITE_SIZE all the bytes written
        "copy": {"bytes_read": copy_bytes, "bytes_written": copy_bytes,
                 "FETCH_SIZE_KiB": copy_bytes / 2 / 1024, "WRITE_SIZE_KiB": copy_bytes / 1024},
        "kernel": {"FETCH_SIZE_KiB": kernel_fetch_kib, "WRITE_SIZE_KiB": kernel_write_kib},
    }
    (folder / f"relaysum_tile_{workload}_counters.json").write_text(json.dumps(rec))


def test_measured_traffic_scales_by_the_copy_and_goes_stale(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    assert bench.measured_traffic("chain16") is None            # no counters
    _write_counters(tmp_path, "chain16", bench.code_digest(), 1000.0, 500.0)
    assert bench.measured_traffic("chain16") == 1000 * 1024 * 2 + 500 * 1024
    assert bench.measured_traffic("chain4") is None              # other workload
    _write_counters(tmp_path, "chain16", "0" * 64, 1000.0, 500.0)
    assert bench.measured_traffic("chain16") is None             # kernel changed since


def test_committed_counters_are_well_formed():
    files = [f for f in os.listdir(bench.PROFILES) if f.endswith("_counters.json")]
    assert files
    for f in files:
        rec = json.load(open(os.path.join(bench.PROFILES, f)))
        assert f.endswith(f"_{rec['workload']}_counters.json")
        assert len(rec["kernel_code_sha256"]) == 64
        for part in ("copy", "kernel"):
            assert float(rec[part]["FETCH_SIZE_KiB"]) > 0 and float(rec[part]["WRITE_SIZE_KiB"]) > 0


def test_slot_masks_follow_library_slot_order():
    n = 4
    mask = np.zeros((n, n), np.uint8)
    mask[1, 2] = 1
    slots = [(0, 1), (1, 0), (1, 2), (2, 1), (2, 3), (3, 2)]
    assert bench._slot_mask(mask, slots).tolist() == [0, 0, 1, 0, 0, 0]
    # double trees: tree A's slots first, each looked up in its own mask
    pair = np.zeros((2, n, n), np.uint8)
    pair[0, 0, 1] = 1
    pair[1, 0, 1] = 0
    pair[1, 3, 2] = 1
    both = slots + slots
    assert bench._slot_mask(pair, both).tolist() == [1, 0, 0, 0, 0, 0] + [0, 0, 0, 0, 0, 1]
