"""The C ABI used from C: tests/c_abi/relaysum_abi_check links
librelaysum.so and the HIP runtime only (no Python, no torch), runs the
hand-worked 3-worker chain from tests/golden, the error codes of invalid
calls, a double-tree handle against two single-tree handles, and a run
resumed from a snapshot against a straight one.  It runs
as a child process with its own HIP runtime."""
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
BIN = os.path.join(HERE, "c_abi", "relaysum_abi_check")
FIXTURE = os.path.join(HERE, "golden", "chain3_alg1_hand_worked.txt")


def test_c_consumer_of_the_abi():
    if not os.path.exists(BIN):
        pytest.fail(f"{BIN} is missing: run __graft_entry__.build() first")
    sys.__stderr__.write("[gpu] C ABI consumer check\n")
    sys.__stderr__.flush()
    r = subprocess.run([BIN, FIXTURE], capture_output=True, text=True, timeout=120)
    print(r.stdout)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "checks passed" in r.stdout and "FAILED" not in r.stdout
