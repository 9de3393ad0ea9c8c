"""The oracle against its pins (CPU only)."""
import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle import reach
from tests import oracle_pins as P

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


@pytest.mark.parametrize("pin", P.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(oracle.lib())


def test_fig_rf_app_coverage():
    """Appendix B receptive-field figure: 39.1% (window) -> 51.0% (with pi)."""
    g = json.load(open(os.path.join(GOLDEN, "rf_app.json")))
    n, k, L = g["N"], g["k"], g["L"]
    loc = 100 * reach.coverage(n, k, 0, L)
    withpi = 100 * reach.coverage(n, k, g["pi"], L)
    assert round(loc, g["printed_decimals"]) == g["coverage_local_pct"]
    assert round(withpi, g["printed_decimals"]) == g["coverage_pi_pct"]
    # with the partner the whole causal triangle is reached
    assert reach.reach(n, k, g["pi"], L).sum() == n * (n + 1) // 2


@pytest.mark.parametrize("k,pi,L", [(4, 16, 6), (2, 5, 4), (3, 3, 5), (1, 7, 3)])
def test_span_bound(k, pi, L):
    """eq. (rf_pi) / Prop. 1: R(L) <= L(k+pi); by brute force the exact span is
    L*max(k, pi) (so the bound holds but is not attained when k, pi > 0)."""
    n = L * (k + pi) + 10
    s = reach.span(n, k, pi, L)
    assert s <= L * (k + pi)
    assert s == L * max(k, pi)


@pytest.mark.parametrize("k,L", [(2, 3), (4, 6), (3, 4)])
def test_local_only_unreachable(k, L):
    """eq. (unreachable): with the window alone a lag d > kL is never reached,
    and every lag d <= kL is (eq. rf_local)."""
    n = k * L + 12
    R = reach.reach(n, k, 0, L)
    i = n - 1
    for d in range(0, i + 1):
        assert R[i, i - d] == (d <= k * L)


@pytest.mark.parametrize("k,pi", [(1, 2), (1, 5), (2, 7), (3, 4), (4, 16), (4, 9)])
def test_minimum_depth(k, pi):
    """eq. (lmin) for an exact lag: BFS over per-layer hops equals
    min_{0 <= b <= d//pi} [b + ceil((d - b pi)/k)], and equals the first depth
    at which the composed graphs connect the pair.  The printed form (b
    unbounded) is the depth to reach a lag >= d: it never exceeds the exact
    value and differs where a pi-hop overshoots."""
    dmax = 3 * pi + 5
    bfs = reach.lmin_bfs(dmax, k, pi)
    for d in range(dmax + 1):
        assert bfs[d] == reach.lmin_exact_lag(d, k, pi), d
        assert reach.lmin_printed(d, k, pi) <= bfs[d]
    n = dmax + 2
    i = n - 1
    first = {}
    for L in range(0, int(bfs.max()) + 1):
        R = reach.reach(n, k, pi, L) if L else np.eye(n, dtype=bool)
        for d in range(dmax + 1):
            if d not in first and R[i, i - d]:
                first[d] = L
    for d in range(dmax + 1):
        assert first[d] == bfs[d]


def test_lmin_printed_overshoot_example():
    """k=4, pi=16, d=5: the printed form gives 1 (one pi-hop overshoots to lag
    16) while an exact lag of 5 needs 2 layers."""
    assert reach.lmin_printed(5, 4, 16) == 1
    assert reach.lmin_exact_lag(5, 4, 16) == 2
    assert reach.lmin_bfs(5, 4, 16)[5] == 2


def test_local_depth_is_ceil():
    """Local-only depth is ceil(d/k) (Sec. 3.4)."""
    bfs = reach.lmin_bfs(50, 4, 0)
    assert all(bfs[d] == math.ceil(d / 4) for d in range(51))
