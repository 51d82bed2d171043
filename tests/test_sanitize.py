"""CPU builds under AddressSanitizer and UndefinedBehaviorSanitizer.

* The library's host-side tree code (tree validation, CSR form, cluster
  plan; paper_2110_04175_amd/csrc/tree_plan.hpp) against its invariants on
  every labelled tree of up to 7 workers and on chains, stars, brooms, heaps
  and random trees up to 5,000 workers (tests/sanitize/plan_check.cpp): every
  worker in exactly one cluster of at most `cap` workers, LDS slots and ring
  positions bijective, the boundary workers exactly the ends of the cut edges.
* The oracle (tests/sanitize/oracle_check.c): every rule and optimizer with
  and without lost messages, in float and double; the sanitized build must
  give the same output bits as a plain build.
"""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g"]


def _compile(cmd):
    r = subprocess.run(cmd, cwd=os.path.join(HERE, "sanitize"), capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]


def _run(exe):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, r.stderr[-4000:]
    return r.stdout


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_tree_plan_invariants_under_sanitizers(tmp_path):
    exe = str(tmp_path / "plan_check")
    _compile(["g++", "-std=c++17", "-O1", *SAN, "-I", os.path.join(ROOT, "include"),
              "-o", exe, "plan_check.cpp"])
    out = _run(exe)
    assert out.startswith("ok "), out
    assert int(out.split()[1]) > 18000


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_under_sanitizers_matches_plain_build(tmp_path):
    flags = ["-std=c11", "-ffp-contract=off", "-fno-fast-math"]
    san, plain = str(tmp_path / "oracle_san"), str(tmp_path / "oracle_plain")
    _compile(["gcc", *flags, "-O1", *SAN, "-o", san, "oracle_check.c", "-lm"])
    _compile(["gcc", *flags, "-O2", "-o", plain, "oracle_check.c", "-lm"])
    a, b = _run(san), _run(plain)
    assert a.startswith("digest ") and a == b, (a, b)
