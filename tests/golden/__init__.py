"""Readers of the fixtures in this folder (exact values with their sources)."""
from __future__ import annotations

import os
from fractions import Fraction

HERE = os.path.dirname(os.path.abspath(__file__))


def _fracs(text):
    return tuple(Fraction(v) for v in text.split())


def chain3_hand_worked():
    """Cases of chain3_alg1_hand_worked.txt: {name: {"x0", "g", "lr", "beta",
    "rounds": [{"m", "c", "nbar", "x", "mom"?}, ...]}} with Fraction values
    (c and nbar as ints)."""
    cases, cur = {}, None
    with open(os.path.join(HERE, "chain3_alg1_hand_worked.txt")) as f:
        for raw in f:
            line = raw.strip()
            if not line or line.startswith("#"):
                continue
            if line.startswith("case "):
                cur = {"rounds": []}
                cases[line.split()[1]] = cur
            elif line.startswith("round "):
                fields = [p.strip() for p in line.split("|")[1:]]
                rec = {}
                for fld in fields:
                    key, val = (s.strip() for s in fld.split("="))
                    vals = _fracs(val)
                    rec[key] = tuple(int(v) for v in vals) if key in ("c", "nbar") else vals
                cur["rounds"].append(rec)
            else:
                key, val = (s.strip() for s in line.split("="))
                vals = _fracs(val)
                cur[key] = vals if key in ("x0", "g") else vals[0]
    return cases
