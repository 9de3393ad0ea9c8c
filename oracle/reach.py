"""Reachability and minimum depth under causal pi-Attention -- TEST INFRASTRUCTURE.

Section 3.4 of the paper (reachability analysis, minimum depth, Proposition 1)
and the receptive-field figure of Appendix B.  Stacking L attention layers
composes the per-layer working-set graphs: position j can influence query i
after L layers iff there is a chain i = p_0 -> p_1 -> ... -> p_L = j with
p_{l+1} in W_{p_l}.  Everything here is brute force on small N, built on the
oracle's own index set, so that the paper's closed forms can be checked
against it.
"""
from __future__ import annotations

import math
from collections import deque

import numpy as np

from . import index_set


def adjacency(n: int, k: int, pi: int) -> np.ndarray:
    """A[i, j] = True iff j is in W_i (one layer of causal pi-Attention)."""
    idx = index_set(n, k, pi)
    A = np.zeros((n, n), dtype=bool)
    rows = np.repeat(np.arange(n), idx.shape[1])
    cols = idx.reshape(-1)
    ok = cols >= 0
    A[rows[ok], cols[ok]] = True
    return A


def reach(n: int, k: int, pi: int, L: int) -> np.ndarray:
    """R[i, j] = True iff j reaches query i through L stacked layers."""
    A = adjacency(n, k, pi).astype(np.int64)
    R = np.eye(n, dtype=np.int64)
    for _ in range(L):
        R = np.minimum(R @ A, 1)
    return R.astype(bool)


def reach_closed_form(n: int, k: int, pi: int, L: int) -> np.ndarray:
    """The set of eq. (reachable): { i - a - pi*b : 0 <= b <= L, 0 <= a <= k(L-b) },
    truncated to [0, i] (the boundary truncation Proposition 1 allows)."""
    R = np.zeros((n, n), dtype=bool)
    for i in range(n):
        for b in range(L + 1):
            for a in range(k * (L - b) + 1):
                j = i - a - pi * b
                if 0 <= j <= i:
                    R[i, j] = True
    return R


def span(n: int, k: int, pi: int, L: int) -> int:
    """Largest lag i - j over reachable pairs (the R(L) of eq. rf_pi)."""
    R = reach(n, k, pi, L)
    i, j = np.nonzero(R)
    return int((i - j).max())


def coverage(n: int, k: int, pi: int, L: int) -> float:
    """Fraction of the n x n (query, source) grid that is reachable after L layers."""
    return float(reach(n, k, pi, L).sum()) / float(n * n)


def lmin_bfs(d_max: int, k: int, pi: int) -> np.ndarray:
    """Minimum number of layers whose per-layer backward hops (one of
    0..k, or pi) sum to exactly d, for d in [0, d_max]; -1 if unreachable
    within d_max layers.  Breadth-first search over the lag."""
    hops = set(range(k + 1))
    if pi > 0:
        hops.add(pi)
    depth = np.full(d_max + 1, -1, dtype=np.int64)
    depth[0] = 0
    q = deque([0])
    while q:
        d = q.popleft()
        for h in hops:
            e = d + h
            if h > 0 and e <= d_max and depth[e] < 0:
                depth[e] = depth[d] + 1
                q.append(e)
    return depth


def lmin_printed(d: int, k: int, pi: int) -> int:
    """eq. (lmin) exactly as printed: min over b >= 0 of b + ceil(max(0, d - b pi) / k).
    b beyond ceil(d/pi) cannot lower the value, so the search stops there."""
    bmax = d // pi + 1 if pi > 0 else 0
    return min(b + math.ceil(max(0, d - b * pi) / k) for b in range(bmax + 1))


def lmin_exact_lag(d: int, k: int, pi: int) -> int:
    """Reading of eq. (lmin) for an exact lag d: the number of pi-hops b may
    not exceed d // pi (hops only move backward, so overshoot is final)."""
    bmax = d // pi if pi > 0 else 0
    return min(b + math.ceil((d - b * pi) / k) for b in range(bmax + 1))
