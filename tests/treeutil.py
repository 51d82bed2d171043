"""Tree facts used to pin the oracle, written independently of it.

Nothing here relays messages: these are hop distances, the two sides of an
edge, and the closed forms that Alg. 1's recurrences reach (each follows
from Alg. 1 by induction on the round t).
"""
from __future__ import annotations

from collections import deque
from fractions import Fraction

import numpy as np


def adjacency(n, edges):
    adj = [set() for _ in range(n)]
    for u, v in np.asarray(edges).reshape(-1, 2):
        adj[int(u)].add(int(v))
        adj[int(v)].add(int(u))
    return adj


def hop_distances(n, edges):
    """tau[i][k]: fewest hops between workers i and k (tau_ii = 0)."""
    adj = adjacency(n, edges)
    tau = np.full((n, n), -1, dtype=np.int64)
    for s in range(n):
        tau[s, s] = 0
        q = deque([s])
        while q:
            u = q.popleft()
            for v in adj[u]:
                if tau[s, v] < 0:
                    tau[s, v] = tau[s, u] + 1
                    q.append(v)
    assert (tau >= 0).all(), "graph is not connected"
    return tau


def diameter(n, edges):
    return int(hop_distances(n, edges).max())


def side(n, edges, i, j):
    """Workers on i's side of edge (i, j): the part of the tree that still
    contains i once the edge is removed."""
    adj = adjacency(n, edges)
    seen = {i}
    q = deque([i])
    while q:
        u = q.popleft()
        for v in adj[u]:
            if (u, v) == (i, j):
                continue
            if v not in seen:
                seen.add(v)
                q.append(v)
    return seen


def closed_form_count(n, edges, tau, i, j, t):
    """c_{i->j} sent in round t: workers on i's side within t hops of i."""
    return sum(1 for k in side(n, edges, i, j) if tau[i, k] <= t)


def closed_form_nbar(tau, i, t):
    """nbar_i^{(t+1)} used after round t: workers within t+1 hops of i."""
    return int((tau[i] <= t + 1).sum())


def delayed_average(tau, xh_history, i, t):
    """x_i^{(t+1)} as the uniform average of delayed half-steps.

    Alg. 1 delivers a half-step of worker k to worker i after
    delta_ik = max(tau_ik - 1, 0) rounds, so
        x_i^{(t+1)} = sum_{k: delta_ik <= t} xh_k^{(t - delta_ik)} / #{k: delta_ik <= t}.
    xh_history[s][k] is worker k's half-step of round s (any element type
    supporting + and /, e.g. Fraction tuples or numpy arrays).
    """
    n = tau.shape[0]
    terms = []
    for k in range(n):
        delta = max(int(tau[i, k]) - 1, 0)
        if delta <= t:
            terms.append(xh_history[t - delta][k])
    total = terms[0]
    for v in terms[1:]:
        total = total + v
    return total / len(terms)


def delayed_message(n, edges, tau, xh_history, i, j, t):
    """m_{i->j} sent in round t: sum of xh_k^{(t - tau_ik)} over i's side,
    for the k that are within t hops of i."""
    total = None
    for k in sorted(side(n, edges, i, j)):
        if tau[i, k] <= t:
            v = xh_history[t - int(tau[i, k])][k]
            total = v if total is None else total + v
    return total


def tree_path(n, edges, k, i):
    """Workers on the tree path from k to i, both ends included."""
    adj = adjacency(n, edges)
    parent = {k: None}
    q = deque([k])
    while q:
        u = q.popleft()
        for v in adj[u]:
            if v not in parent:
                parent[v] = u
                q.append(v)
    path = [i]
    while path[-1] != k:
        path.append(parent[path[-1]])
    return path[::-1]


def arrivals(n, edges, i, t, dropped_by_round):
    """Parcels that reach worker i's update in round t, as (k, s) pairs.

    A parcel is what worker k puts into the relay in round s (a half-step,
    an update or a sample).  It crosses one tree hop per round: the hop h of
    its path k = p_0, p_1, ..., p_tau = i is the message p_{h-1} -> p_h of
    round s + h - 1, and it reaches i in round s + tau - 1 (round s when
    k = i).  It arrives only if none of those messages was lost.
    dropped_by_round[r] is a set of lost (src, dst) messages of round r.
    """
    out = [(i, t)]
    for k in range(n):
        if k == i:
            continue
        p = tree_path(n, edges, k, i)
        tau = len(p) - 1
        s = t - tau + 1
        if s < 0:
            continue
        ok = all((p[h - 1], p[h]) not in dropped_by_round.get(s + h - 1, ())
                 for h in range(1, tau + 1))
        if ok:
            out.append((k, s))
    return out
