"""RelaySum on double binary trees (test infrastructure only).

Section 3 of the paper: the odd coordinates of every model travel on tree A,
the even ones on tree B (0-based coordinates).  Coordinates are independent
in every step of a round, so a round on double trees is exactly one round on
tree A over the odd coordinates plus one round on tree B over the even ones;
this class composes two single-tree oracles that way.
"""
from __future__ import annotations

import numpy as np

from . import Oracle


class DoubleOracle:
    def __init__(self, n: int, d: int, edges_a, edges_b, dtype=np.float32):
        self.n, self.d = int(n), int(d)
        self.odd = np.arange(1, self.d, 2)
        self.even = np.arange(0, self.d, 2)
        self.a = Oracle(n, len(self.odd), edges_a, dtype)
        self.b = Oracle(n, len(self.even), edges_b, dtype)
        self.dtype = np.dtype(dtype)

    def _split(self, arr, cols):
        return None if arr is None else np.ascontiguousarray(arr[:, cols])

    def round_ex(self, x, g, s1=None, s2=None, *, dropped_a=None, dropped_b=None, **kw):
        for tree, cols, dropped in ((self.a, self.odd, dropped_a), (self.b, self.even, dropped_b)):
            xs, gs = self._split(x, cols), self._split(g, cols)
            s1s, s2s = self._split(s1, cols), self._split(s2, cols)
            tree.round_ex(xs, gs, s1s, s2s, dropped=dropped, **kw)
            x[:, cols] = xs
            if s1 is not None:
                s1[:, cols] = s1s
            if s2 is not None:
                s2[:, cols] = s2s

    def round(self, x, g, mom, lr, beta):
        self.round_ex(x, g, mom, None, update="model", lr=lr, beta1=beta)

    def close(self):
        self.a.close()
        self.b.close()
