"""RelaySum round in exact rational arithmetic (test infrastructure only).

Alg. 1 of the paper (RelaySum/Model) with the Nesterov-momentum local step of
Appendix D.2, written with pure-Python loops over ``fractions.Fraction`` so
that tiny cases carry no rounding at all.  Models are lists of d-tuples.
"""
from __future__ import annotations

from fractions import Fraction
from typing import Dict, List, Sequence, Tuple


def neighbours(n: int, edges) -> List[List[int]]:
    """N_i for every worker, ascending (Section 3, Setup)."""
    nb = [[] for _ in range(n)]
    for u, v in edges:
        nb[int(u)].append(int(v))
        nb[int(v)].append(int(u))
    return [sorted(x) for x in nb]


class ExactRelaySum:
    """State of Alg. 1 for n workers; every number is a Fraction."""

    def __init__(self, n: int, d: int, edges):
        self.n, self.d = n, d
        self.nb = neighbours(n, edges)
        zero = tuple(Fraction(0) for _ in range(d))
        # Alg. 1 input: m^{(-1)} = 0 and c^{(-1)} = 0 on every directed edge.
        self.msg: Dict[Tuple[int, int], tuple] = {
            (i, j): zero for i in range(n) for j in self.nb[i]}
        self.cnt: Dict[Tuple[int, int], int] = {(i, j): 0 for i in range(n) for j in self.nb[i]}
        self.nbar = [0] * n
        self.t = 0
        self.last_xh = None

    def round(self, x: Sequence[Sequence], g: Sequence[Sequence], mom, lr, beta):
        """One iteration for every worker.  Returns (x_new, mom_new)."""
        n, d = self.n, self.d
        lr, beta = Fraction(lr), Fraction(beta)
        x = [[Fraction(v) for v in row] for row in x]
        g = [[Fraction(v) for v in row] for row in g]
        mom = [[Fraction(v) for v in row] for row in mom] if mom is not None else None

        # Local half-step (Alg. 1's local step; Nesterov momentum, App. D.2).
        xh = []
        new_mom = None if mom is None else []
        for i in range(n):
            if beta != 0:
                m_i = [beta * mom[i][c] + g[i][c] for c in range(d)]
                new_mom.append(m_i)
                xh.append([x[i][c] - lr * (g[i][c] + beta * m_i[c]) for c in range(d)])
            else:
                if new_mom is not None:
                    new_mom.append(list(mom[i]))
                xh.append([x[i][c] - lr * g[i][c] for c in range(d)])

        # Relay: m_{i->j} = xh_i + sum_{k in N_i \ j} m_{k->i}^{(t-1)}, and counters.
        msg, cnt = {}, {}
        for i in range(n):
            for j in self.nb[i]:
                others = [k for k in self.nb[i] if k != j]
                msg[(i, j)] = tuple(xh[i][c] + sum((self.msg[(k, i)][c] for k in others),
                                                   Fraction(0)) for c in range(d))
                cnt[(i, j)] = 1 + sum(self.cnt[(k, i)] for k in others)

        # Count-corrected average.
        x_new = []
        for i in range(n):
            nb_i = 1 + sum(cnt[(j, i)] for j in self.nb[i])
            self.nbar[i] = nb_i
            x_new.append([(xh[i][c] + sum((msg[(j, i)][c] for j in self.nb[i]), Fraction(0)))
                          / nb_i for c in range(d)])
        self.msg, self.cnt = msg, cnt
        self.last_xh = xh
        self.t += 1
        return x_new, new_mom
