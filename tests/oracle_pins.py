"""Pins for the fp64 oracle: checks against what the paper and the mathematics
fix, independent of the oracle's own formulas.

Each ``pin_*`` takes an oracle library handle and raises AssertionError on a
mismatch, so the same battery runs against the real oracle (test_oracle.py)
and against builds with a planted mistake (test_oracle_mutants.py), which it
must reject.
"""
from __future__ import annotations

import json
import math
import os

import numpy as np

import oracle
from oracle import reach

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
EPS = json.load(open(os.path.join(GOLDEN, "defaults.json")))["eps"]


# ---------------------------------------------------------------------------
# independent references
# ---------------------------------------------------------------------------
def scan_membership(n: int, k: int, pi: int, causal: bool = True) -> np.ndarray:
    """Brute-force membership scan: M[t, j] for every pair, straight from the
    set definitions (eq. Nr, eq. Npi, eq. U; bidirectional: |j - t| <= k and
    the partners t -/+ pi, App. B hyper-parameter table); positions outside
    the sequence are never visited."""
    M = np.zeros((n, n), dtype=bool)
    for t in range(n):
        for j in range(n):
            if causal:
                in_window = max(0, t - k) <= j <= t
                is_partner = j == t - pi
            else:
                in_window = abs(j - t) <= k
                is_partner = j == t - pi or j == t + pi
            M[t, j] = in_window or is_partner
    return M


def rand_qkv(rng, B, H, N, D, dtype=np.float32):
    return [rng.standard_normal((B, H, N, D)).astype(dtype) for _ in range(3)]


def textbook_causal(q, k, v, scale, causal=True):
    """Dense scaled-dot-product attention (eqs. alpha and attn), causal or
    over every position, fp64."""
    q, k, v = (np.asarray(x, np.float64) for x in (q, k, v))
    N = q.shape[-2]
    S = (q @ np.swapaxes(k, -1, -2)) * scale
    if causal:
        S = np.where(np.tril(np.ones((N, N), bool)), S, -np.inf)
    S = S - S.max(-1, keepdims=True)
    P = np.exp(S)
    P /= P.sum(-1, keepdims=True)
    return P @ v


def logsumexp_masked(S, M):
    S = np.where(M, S, -np.inf)
    mx = S.max(-1, keepdims=True)
    return (mx + np.log(np.exp(S - mx).sum(-1, keepdims=True)))[..., 0]


def multiplicative_fusion(q, k, v, gate, kk, pi, scale, causal=True, alpha_t=None):
    """eq. (alphahat_adapt) in its multiplicative form: weights
    omega_tj * exp(z_tj) normalised over U(t), omega = alpha~ on the window and
    1 - alpha~ on a partner; mask from the brute-force scan.  fp64, dense.
    ``alpha_t`` [B, H, N], when given, is used as alpha~ directly (``gate``
    is then ignored)."""
    q, k, v = (np.asarray(x, np.float64) for x in (q, k, v))
    B, H, N, D = q.shape
    M = scan_membership(N, kk, pi, causal)
    window = np.zeros((N, N), bool)
    for t in range(N):
        window[t, max(0, t - kk):(t + 1 if causal else t + kk + 1)] = True
    if alpha_t is None:
        g = np.asarray(gate, np.float64)
        g = np.broadcast_to(g[None, :, None] if g.shape == (H,) else g, (B, H, N))
        a_t = EPS + (1 - 2 * EPS) / (1 + np.exp(-g))           # [B,H,N]
    else:
        a_t = np.asarray(alpha_t, np.float64)
    omega = np.where(window[None, None], a_t[..., None], (1 - a_t)[..., None])
    Z = (q @ np.swapaxes(k, -1, -2)) * scale
    W = np.where(M[None, None], omega * np.exp(Z), 0.0)
    W /= W.sum(-1, keepdims=True)
    return W @ v, W


# ---------------------------------------------------------------------------
# pins
# ---------------------------------------------------------------------------
IDX_CASES = [(1, 0, 0), (1, 3, 5), (7, 0, 1), (9, 2, 5), (16, 3, 3), (16, 3, 2), (16, 3, 4),
             (20, 4, 16), (33, 5, 0), (40, 50, 7), (40, 6, 39), (40, 6, 40), (64, 8, 16)]


def pin_index_set_scan(L):
    """Working-set indices equal the brute-force membership scan, slot order
    is window offsets -k..0 then the partner, and no index exceeds t."""
    for n, k, pi in IDX_CASES:
        idx = oracle.index_set(n, k, pi, L)
        m = k + 1 + (1 if pi > k else 0)
        assert idx.shape == (n, m), (n, k, pi, idx.shape)
        M = scan_membership(n, k, pi)
        for t in range(n):
            got = idx[t][idx[t] >= 0]
            assert len(set(got.tolist())) == len(got), "duplicate entry"
            assert sorted(got.tolist()) == np.nonzero(M[t])[0].tolist(), (n, k, pi, t)
            assert (got <= t).all()
            for s in range(k + 1):
                assert idx[t, s] == (t - k + s if t - k + s >= 0 else -1)
            if m == k + 2:
                assert idx[t, k + 1] == (t - pi if t >= pi else -1)


def pin_working_set_sizes(L):
    """|W_t| = min(t, k) + 1 + [pi > k and t >= pi] summed in closed form."""
    for n, k, pi in [(256, 32, 64), (4096, 128, 256), (1000, 7, 3), (300, 299, 500)]:
        idx = oracle.index_set(n, k, pi, L)
        total = int((idx >= 0).sum())
        if n > k:
            closed = (k + 1) * (k + 2) // 2 + (n - k - 1) * (k + 1)
        else:
            closed = n * (n + 1) // 2
        closed += max(0, n - pi) if pi > k else 0
        assert total == closed, (n, k, pi, total, closed)


def pin_dense_reduction(L):
    """k >= N-1: every j <= t is in the window with one common prior, which
    cancels in the softmax, so the result is dense causal attention (Sec. 3.1)
    for any gate; lse = log alpha~ + logsumexp(z)."""
    rng = np.random.default_rng(11)
    B, H, N, D = 2, 3, 37, 16
    q, k, v = rand_qkv(rng, B, H, N, D)
    gate = rng.uniform(-3, 3, H).astype(np.float32)
    scale = 1 / math.sqrt(D)
    ref = textbook_causal(q, k, v, scale)
    for kk, pi in [(N - 1, 5), (N + 10, 0), (N - 1, N + 3)]:
        out, lse = oracle.forward(q, k, v, gate, kk, pi, want_lse=True, L=L)
        assert np.abs(out - ref).max() <= 1e-12, (kk, pi, np.abs(out - ref).max())
        S = (q.astype(np.float64) @ np.swapaxes(k, -1, -2).astype(np.float64)) * scale
        a_t = EPS + (1 - 2 * EPS) / (1 + np.exp(-gate.astype(np.float64)))
        lse_ref = np.log(a_t)[None, :, None] + logsumexp_masked(S, np.tril(np.ones((N, N), bool)))
        assert np.abs(lse - lse_ref).max() <= 1e-12


def pin_local_reduction(L):
    """pi <= k (partner already in the window), or t < pi: plain sliding-window
    attention (eq. Nr), independent of the gate."""
    rng = np.random.default_rng(12)
    B, H, N, D = 1, 2, 40, 8
    q, k, v = rand_qkv(rng, B, H, N, D)
    kk = 5
    M = np.zeros((N, N), bool)
    for t in range(N):
        M[t, max(0, t - kk):t + 1] = True
    S = (q.astype(np.float64) @ np.swapaxes(k, -1, -2).astype(np.float64)) / math.sqrt(D)
    S = np.where(M, S, -np.inf)
    P = np.exp(S - S.max(-1, keepdims=True))
    P /= P.sum(-1, keepdims=True)
    ref = P @ v.astype(np.float64)
    for pi in (0, 1, 3, kk):
        for g in (-4.0, 0.0, 2.5):
            out = oracle.forward(q, k, v, np.full(H, g, np.float32), kk, pi, L=L)
            assert np.abs(out - ref).max() <= 1e-12, (pi, g)
    # pi > k, but rows t < pi have no partner
    pi = 17
    out = oracle.forward(q, k, v, np.array([1.5, -2.0], np.float32), kk, pi, L=L)
    assert np.abs(out[:, :, :pi] - ref[:, :, :pi]).max() <= 1e-12
    assert np.abs(out[:, :, pi:] - ref[:, :, pi:]).max() > 1e-6


def pin_basic_union_g0(L):
    """g = 0 gives alpha~ = 1/2 for both branches: the prior cancels and the
    result is the basic union softmax (eqs. alpha_u, beta), which is also fixed
    fusion with alpha = 0.5 (Variant 2)."""
    rng = np.random.default_rng(13)
    B, H, N, D = 1, 2, 48, 8
    q, k, v = rand_qkv(rng, B, H, N, D)
    kk, pi = 4, 11
    M = scan_membership(N, kk, pi)
    S = (q.astype(np.float64) @ np.swapaxes(k, -1, -2).astype(np.float64)) / math.sqrt(D)
    S = np.where(M, S, -np.inf)
    P = np.exp(S - S.max(-1, keepdims=True))
    P /= P.sum(-1, keepdims=True)
    ref = P @ v.astype(np.float64)
    out = oracle.forward(q, k, v, np.zeros(H, np.float32), kk, pi, L=L)
    assert np.abs(out - ref).max() <= 1e-12


def pin_multiplicative_form(L):
    """General adaptive fusion equals eq. (alphahat_adapt) written
    multiplicatively, per-head and per-query gates, weights included."""
    rng = np.random.default_rng(14)
    B, H, N, D = 2, 2, 45, 8
    q, k, v = rand_qkv(rng, B, H, N, D)
    for kk, pi in [(3, 9), (6, 7), (2, 20)]:
        for gate in (rng.uniform(-2, 2, H).astype(np.float32),
                     rng.uniform(-4, 4, (B, H, N)).astype(np.float32)):
            ref, W = multiplicative_fusion(q, k, v, gate, kk, pi, 1 / math.sqrt(D))
            out, P = oracle.forward(q, k, v, gate, kk, pi, want_probs=True, L=L)
            assert np.abs(out - ref).max() <= 1e-12, (kk, pi, np.abs(out - ref).max())
            idx = oracle.index_set(N, kk, pi, L)
            for t in (0, 1, kk, pi, N - 1):
                for b in range(B):
                    for h in range(H):
                        for s in range(idx.shape[1]):
                            j = idx[t, s]
                            want = W[b, h, t, j] if j >= 0 else 0.0
                            assert abs(P[b, h, t, s] - want) <= 1e-12


def pin_gate_limits(L):
    """alpha -> 1 (g -> +inf): partner weight relative to a window key is
    eps/(1-eps) * exp(z_p - z_j); alpha -> 0: (1-eps)/eps * exp(z_p - z_j)
    (Sec. 3.5: the clip keeps both priors inside [eps, 1-eps])."""
    rng = np.random.default_rng(15)
    B, H, N, D = 1, 2, 30, 8
    q, k, v = rand_qkv(rng, B, H, N, D)
    kk, pi = 3, 10
    gate = np.array([60.0, -60.0], np.float32)
    _, P = oracle.forward(q, k, v, gate, kk, pi, want_probs=True, L=L)
    q64, k64 = q.astype(np.float64), k.astype(np.float64)
    for t in range(pi, N):
        for h, ratio in ((0, EPS / (1 - EPS)), (1, (1 - EPS) / EPS)):
            zp = q64[0, h, t] @ k64[0, h, t - pi] / math.sqrt(D)
            zs = q64[0, h, t] @ k64[0, h, t] / math.sqrt(D)
            got = P[0, h, t, kk + 1] / P[0, h, t, kk]
            want = ratio * math.exp(zp - zs)
            assert abs(got / want - 1) <= 1e-9, (t, h, got, want)


def pin_sum_to_one_and_row0(L):
    """Weights over W_t sum to 1; row t = 0 attends only to itself, so y_0 = v_0
    exactly; t = 1 has the two-element closed form."""
    rng = np.random.default_rng(16)
    B, H, N, D = 2, 2, 50, 8
    q, k, v = rand_qkv(rng, B, H, N, D)
    gate = rng.uniform(-1, 1, (B, H, N)).astype(np.float32)
    out, P = oracle.forward(q, k, v, gate, 6, 13, want_probs=True, L=L)
    assert np.abs(P.sum(-1) - 1).max() <= 1e-12
    assert (P >= 0).all()
    assert np.array_equal(out[:, :, 0], v[:, :, 0].astype(np.float64))
    q64, k64, v64 = (x.astype(np.float64) for x in (q, k, v))
    for b in range(B):
        for h in range(H):
            z0 = q64[b, h, 1] @ k64[b, h, 0] / math.sqrt(D)
            z1 = q64[b, h, 1] @ k64[b, h, 1] / math.sqrt(D)
            y = (math.exp(z0) * v64[b, h, 0] + math.exp(z1) * v64[b, h, 1]) / (math.exp(z0) + math.exp(z1))
            assert np.abs(out[b, h, 1] - y).max() <= 1e-12


def pin_causality(L):
    """Perturbing or NaN-poisoning positions > t changes no output at t."""
    rng = np.random.default_rng(17)
    B, H, N, D = 1, 2, 64, 8
    q, k, v = rand_qkv(rng, B, H, N, D)
    gate = rng.uniform(-1, 1, H).astype(np.float32)
    base = oracle.forward(q, k, v, gate, 5, 12, L=L)
    for cut in (0, 7, 31, 63):
        q2, k2, v2 = q.copy(), k.copy(), v.copy()
        q2[:, :, cut + 1:] = np.nan
        k2[:, :, cut + 1:] = np.nan
        v2[:, :, cut + 1:] = np.inf
        out = oracle.forward(q2, k2, v2, gate, 5, 12, L=L)
        assert np.array_equal(out[:, :, :cut + 1], base[:, :, :cut + 1]), cut


def pin_head_batch_independence(L):
    """Permuting heads (with their gates) and batches permutes the outputs."""
    rng = np.random.default_rng(18)
    B, H, N, D = 2, 4, 24, 8
    q, k, v = rand_qkv(rng, B, H, N, D)
    gate = rng.uniform(-1, 1, H).astype(np.float32)
    out = oracle.forward(q, k, v, gate, 3, 7, L=L)
    ph, pb = np.array([2, 0, 3, 1]), np.array([1, 0])
    out2 = oracle.forward(q[pb][:, ph], k[pb][:, ph], v[pb][:, ph], gate[ph], 3, 7, L=L)
    assert np.array_equal(out2, out[pb][:, ph])


def pin_decode_matches_last_row(L):
    """A decode step at t = len is the forward's row t over the sequence whose
    row t is the new key/value (Sec. 3.5, online working set); the step writes
    that row into the cache."""
    rng = np.random.default_rng(19)
    S, H, D, cap = 3, 2, 8, 64
    kk, pi = 5, 13
    lens = np.array([0, 20, 47], np.int32)
    Kc = rng.standard_normal((S, H, cap, D)).astype(np.float32)
    Vc = rng.standard_normal((S, H, cap, D)).astype(np.float32)
    qn, kn, vn = (rng.standard_normal((S, H, D)).astype(np.float32) for _ in range(3))
    gate = rng.uniform(-1, 1, (S, H)).astype(np.float32)
    K2, V2 = Kc.copy(), Vc.copy()
    out, lse = oracle.decode_step(lens, qn, kn, vn, K2, V2, gate, kk, pi, want_lse=True, L=L)
    for s in range(S):
        t = int(lens[s])
        assert np.array_equal(K2[s, :, t], kn[s]) and np.array_equal(V2[s, :, t], vn[s])
        keep = np.ones(cap, bool)
        keep[t] = False
        assert np.array_equal(K2[s][:, keep], Kc[s][:, keep])
        seqK, seqV = K2[s:s + 1, :, :t + 1], V2[s:s + 1, :, :t + 1]
        seqQ = np.zeros_like(seqK)
        seqQ[0, :, t] = qn[s]
        g = np.broadcast_to(gate[s][None, :, None], (1, H, t + 1)).astype(np.float32).copy()
        ref, lref = oracle.forward(seqQ, seqK, seqV, g, kk, pi, want_lse=True, L=L)
        assert np.array_equal(out[s], ref[0, :, t])
        assert np.array_equal(lse[s], lref[0, :, t])
    # and the last row agrees with the multiplicative form on the full sequence
    s = 2
    t = int(lens[s])
    seqQ = np.zeros((1, H, t + 1, D), np.float32)
    seqQ[0, :, t] = qn[s]
    ref, _ = multiplicative_fusion(seqQ, K2[s:s + 1, :, :t + 1], V2[s:s + 1, :, :t + 1],
                                   np.broadcast_to(gate[s][None, :, None], (1, H, t + 1)),
                                   kk, pi, 1 / math.sqrt(D))
    assert np.abs(out[s] - ref[0, :, t]).max() <= 1e-12


def pin_clamp_reading(L):
    """Reading of the logit clamp (hyper-parameter table, L_c = 20): clamp the
    fused logits of valid entries to [-L_c, L_c]; with every |delta| < L_c the
    clamp changes nothing."""
    rng = np.random.default_rng(20)
    B, H, N, D = 1, 2, 30, 8
    q, k, v = rand_qkv(rng, B, H, N, D)
    gate = rng.uniform(-1, 1, H).astype(np.float32)
    a = oracle.forward(q, k, v, gate, 4, 9, L=L)
    b = oracle.forward(q, k, v, gate, 4, 9, clamp=20.0, L=L)
    assert np.array_equal(a, b)
    big = oracle.forward(q, k, v, gate, 4, 9, scale=40.0, clamp=20.0, L=L)
    _, P = oracle.forward(q, k, v, gate, 4, 9, scale=40.0, clamp=20.0, want_probs=True, L=L)
    idx = oracle.index_set(N, 4, 9, L)
    Z = (q.astype(np.float64) @ np.swapaxes(k, -1, -2).astype(np.float64)) * 40.0
    a_t = EPS + (1 - 2 * EPS) / (1 + np.exp(-gate.astype(np.float64)))
    for h in range(H):
        for t in range(N):
            js = idx[t]
            dl = np.array([Z[0, h, t, j] + (math.log(a_t[h]) if s <= 4 else math.log(1 - a_t[h]))
                           for s, j in enumerate(js) if j >= 0])
            dl = np.clip(dl, -20.0, 20.0)
            w = np.exp(dl - dl.max())
            w /= w.sum()
            got = P[0, h, t][js >= 0]
            assert np.abs(got - w).max() <= 1e-12
            assert np.abs(big[0, h, t] - w @ v[0, h, js[js >= 0]].astype(np.float64)).max() <= 1e-12


# ---------------------------------------------------------------------------
# bidirectional mode (eq. Nr bidirectional case; partners t -/+ pi)
# ---------------------------------------------------------------------------
BIDIR_IDX_CASES = [(1, 0, 0), (1, 3, 5), (7, 0, 1), (9, 2, 5), (16, 3, 3), (16, 3, 4), (20, 4, 16),
                   (33, 5, 0), (40, 50, 7), (40, 6, 39), (40, 6, 40), (64, 8, 16), (12, 2, 11)]


def pin_bidir_index_set_scan(L):
    """Bidirectional working sets equal the brute-force scan; slot order is
    window offsets -k..k, then t - pi, then t + pi (App. A offset list)."""
    for n, k, pi in BIDIR_IDX_CASES:
        idx = oracle.index_set(n, k, pi, L, causal=False)
        m = 2 * k + 1 + (2 if pi > k else 0)
        assert idx.shape == (n, m), (n, k, pi, idx.shape)
        M = scan_membership(n, k, pi, causal=False)
        for t in range(n):
            got = idx[t][idx[t] >= 0]
            assert len(set(got.tolist())) == len(got), "duplicate entry"
            assert sorted(got.tolist()) == np.nonzero(M[t])[0].tolist(), (n, k, pi, t)
            for s in range(2 * k + 1):
                j = t - k + s
                assert idx[t, s] == (j if 0 <= j < n else -1)
            if pi > k:
                assert idx[t, 2 * k + 1] == (t - pi if t >= pi else -1)
                assert idx[t, 2 * k + 2] == (t + pi if t + pi < n else -1)


def pin_bidir_working_set_sizes(L):
    """sum_t |W_t| in closed form: window n(2k+1) - k(k+1) for n > k (n^2
    otherwise), plus 2 max(0, n - pi) partners when pi > k."""
    for n, k, pi in [(256, 32, 64), (4096, 128, 256), (1000, 7, 3), (300, 299, 500), (50, 60, 70)]:
        idx = oracle.index_set(n, k, pi, L, causal=False)
        total = int((idx >= 0).sum())
        closed = n * (2 * k + 1) - k * (k + 1) if n > k else n * n
        closed += 2 * max(0, n - pi) if pi > k else 0
        assert total == closed, (n, k, pi, total, closed)


def pin_bidir_dense_reduction(L):
    """k >= N-1, bidirectional: every position is in the window, the prior
    cancels, and the result is dense (unmasked) softmax attention (eqs. alpha,
    attn) for any gate; lse = log alpha~ + logsumexp(z) over all positions."""
    rng = np.random.default_rng(31)
    B, H, N, D = 2, 2, 29, 16
    q, k, v = rand_qkv(rng, B, H, N, D)
    gate = rng.uniform(-3, 3, (B, H, N)).astype(np.float32)
    scale = 1 / math.sqrt(D)
    ref = textbook_causal(q, k, v, scale, causal=False)
    S = (q.astype(np.float64) @ np.swapaxes(k, -1, -2).astype(np.float64)) * scale
    a_t = EPS + (1 - 2 * EPS) / (1 + np.exp(-gate.astype(np.float64)))
    lse_ref = np.log(a_t) + logsumexp_masked(S, np.ones((N, N), bool))
    for kk, pi in [(N - 1, 5), (N + 10, 0), (N - 1, N + 3)]:
        out, lse = oracle.forward(q, k, v, gate, kk, pi, want_lse=True, L=L, causal=False)
        assert np.abs(out - ref).max() <= 1e-12, (kk, pi, np.abs(out - ref).max())
        assert np.abs(lse - lse_ref).max() <= 1e-12


def pin_bidir_local_reduction(L):
    """pi <= k, bidirectional: both partners lie in the window, so the result is
    plain bidirectional sliding-window attention, independent of the gate."""
    rng = np.random.default_rng(32)
    B, H, N, D = 1, 2, 40, 8
    q, k, v = rand_qkv(rng, B, H, N, D)
    kk = 5
    M = np.abs(np.arange(N)[:, None] - np.arange(N)[None, :]) <= kk
    S = (q.astype(np.float64) @ np.swapaxes(k, -1, -2).astype(np.float64)) / math.sqrt(D)
    S = np.where(M, S, -np.inf)
    P = np.exp(S - S.max(-1, keepdims=True))
    P /= P.sum(-1, keepdims=True)
    ref = P @ v.astype(np.float64)
    for pi in (0, 1, 3, kk):
        for g in (-4.0, 0.0, 2.5):
            out = oracle.forward(q, k, v, np.full(H, g, np.float32), kk, pi, L=L, causal=False)
            assert np.abs(out - ref).max() <= 1e-12, (pi, g)


def pin_bidir_multiplicative_form(L):
    """Bidirectional adaptive fusion equals the multiplicative form of eq.
    (alphahat_adapt) with both partners priced 1 - alpha~; g = 0 reduces it to
    the basic union softmax (eqs. alpha_u, beta)."""
    rng = np.random.default_rng(33)
    B, H, N, D = 2, 2, 45, 8
    q, k, v = rand_qkv(rng, B, H, N, D)
    for kk, pi in [(3, 9), (6, 7), (2, 20), (4, 44)]:
        for gate in (rng.uniform(-2, 2, H).astype(np.float32),
                     rng.uniform(-4, 4, (B, H, N)).astype(np.float32), np.zeros(H, np.float32)):
            ref, W = multiplicative_fusion(q, k, v, gate, kk, pi, 1 / math.sqrt(D), causal=False)
            out, P = oracle.forward(q, k, v, gate, kk, pi, want_probs=True, L=L, causal=False)
            assert np.abs(out - ref).max() <= 1e-12, (kk, pi, np.abs(out - ref).max())
            idx = oracle.index_set(N, kk, pi, L, causal=False)
            for t in (0, 1, kk, pi, N - 1 - pi, N - 1):
                if not 0 <= t < N:
                    continue
                for s in range(idx.shape[1]):
                    j = idx[t, s]
                    want = W[:, :, t, j] if j >= 0 else 0.0
                    assert np.abs(P[:, :, t, s] - want).max() <= 1e-12


def pin_bidir_time_reversal(L):
    """Reversing the sequence (q, k, v and a per-query gate) reverses the
    bidirectional output: the window is symmetric and the partners t -/+ pi
    trade places."""
    rng = np.random.default_rng(34)
    B, H, N, D = 1, 3, 37, 8
    q, k, v = rand_qkv(rng, B, H, N, D)
    gate = rng.uniform(-2, 2, (B, H, N)).astype(np.float32)
    for kk, pi in [(2, 7), (4, 30), (3, 3), (0, 1)]:
        out = oracle.forward(q, k, v, gate, kk, pi, L=L, causal=False)
        rev = oracle.forward(q[:, :, ::-1], k[:, :, ::-1], v[:, :, ::-1], gate[:, :, ::-1], kk, pi,
                             L=L, causal=False)
        assert np.abs(rev[:, :, ::-1] - out).max() <= 1e-12, (kk, pi)


def pin_bidir_gate_limits(L):
    """g -> +inf: each partner's weight relative to the self entry tends to
    eps/(1-eps) exp(z_p - z_t); g -> -inf: (1-eps)/eps exp(z_p - z_t)."""
    rng = np.random.default_rng(35)
    B, H, N, D = 1, 2, 30, 8
    q, k, v = rand_qkv(rng, B, H, N, D)
    kk, pi = 3, 10
    gate = np.array([60.0, -60.0], np.float32)
    _, P = oracle.forward(q, k, v, gate, kk, pi, want_probs=True, L=L, causal=False)
    q64, k64 = q.astype(np.float64), k.astype(np.float64)
    for t in range(N):
        for h, ratio in ((0, EPS / (1 - EPS)), (1, (1 - EPS) / EPS)):
            zs = q64[0, h, t] @ k64[0, h, t] / math.sqrt(D)
            for slot, j in ((2 * kk + 1, t - pi), (2 * kk + 2, t + pi)):
                if not 0 <= j < N:
                    assert P[0, h, t, slot] == 0.0
                    continue
                zp = q64[0, h, t] @ k64[0, h, j] / math.sqrt(D)
                got = P[0, h, t, slot] / P[0, h, t, kk]
                assert abs(got / (ratio * math.exp(zp - zs)) - 1) <= 1e-9, (t, h, j)


def pin_gate_mlp_composition(L):
    """App. A module, written with torch fp64 layers: gate = Sigmoid(Linear(
    GELU(Linear(x)))), alpha~ = alpha (1 - 2 eps) + eps, union attention in
    its multiplicative form.  Equals oracle.forward on the logits
    oracle.gate_logits(u, W2, b2), u = GELU(Linear(x)) (rounded to float32,
    the operator's input), for causal and bidirectional windows."""
    import torch
    import torch.nn.functional as F
    rng = np.random.default_rng(40)
    B, T, d, h = 2, 37, 32, 4
    dh, D = d // 2, d // h
    f32 = lambda a: np.asarray(a, np.float32)
    x = torch.tensor(rng.standard_normal((B, T, d)))
    W1, b1 = torch.tensor(rng.standard_normal((dh, d)) / math.sqrt(d)), torch.tensor(rng.standard_normal(dh) * 0.1)
    W2 = torch.tensor(f32(rng.standard_normal((h, dh)) / math.sqrt(dh)), dtype=torch.float64)
    b2 = torch.tensor(f32(rng.standard_normal(h)), dtype=torch.float64)
    u = F.gelu(F.linear(x, W1, b1)).float().double()           # the operator's input u
    a = torch.sigmoid(F.linear(u, W2, b2))                     # [B, T, h]
    a_t = (a * (1 - 2 * EPS) + EPS).permute(0, 2, 1).numpy()   # [B, h, T]
    g = oracle.gate_logits(u.float().numpy(), W2.float().numpy(), b2.float().numpy())
    assert g.shape == (B, h, T)
    q, k, v = rand_qkv(rng, B, h, T, D)
    for causal in (True, False):
        for kk, pi in [(2, 5), (3, 3), (1, 9)]:
            ref, _ = multiplicative_fusion(q, k, v, None, kk, pi, 1 / math.sqrt(D), causal, alpha_t=a_t)
            out = oracle.forward(q, k, v, g, kk, pi, L=L, causal=causal)
            assert np.abs(out - ref).max() <= 1e-12, (causal, kk, pi, np.abs(out - ref).max())


ALL_PINS = [pin_index_set_scan, pin_working_set_sizes, pin_dense_reduction, pin_local_reduction,
            pin_basic_union_g0, pin_multiplicative_form, pin_gate_limits, pin_sum_to_one_and_row0,
            pin_causality, pin_head_batch_independence, pin_decode_matches_last_row,
            pin_clamp_reading, pin_bidir_index_set_scan, pin_bidir_working_set_sizes,
            pin_bidir_dense_reduction, pin_bidir_local_reduction, pin_bidir_multiplicative_form,
            pin_bidir_time_reversal, pin_bidir_gate_limits, pin_gate_mlp_composition]


def pin_reachability(L):
    """Composing the per-layer working-set graphs reproduces eq. (reachable)
    exactly (up to truncation at position 0), for many (k, pi, L)."""
    for kk in (1, 2, 3):
        for pi in (kk + 1, 2 * kk + 3, 7):
            for depth in (1, 2, 3):
                n = 40
                idx = oracle.index_set(n, kk, pi, L)
                A = np.zeros((n, n), np.int64)
                for t in range(n):
                    for j in idx[t]:
                        if j >= 0:
                            A[t, j] = 1
                R = np.eye(n, dtype=np.int64)
                for _ in range(depth):
                    R = np.minimum(R @ A, 1)
                assert np.array_equal(R.astype(bool), reach.reach_closed_form(n, kk, pi, depth)), (kk, pi, depth)


ALL_PINS.append(pin_reachability)


# ---------------------------------------------------------------------------
# backward pins
# ---------------------------------------------------------------------------
def _loss(L, q, k, v, gate, kk, pi, dout, clamp=0.0, causal=True):
    y = oracle.forward(q, k, v, gate, kk, pi, clamp=clamp, L=L, causal=causal)
    return float(np.sum(y * np.asarray(dout, np.float64)))


def _central_difference(L, arrays, which, idx, h, kk, pi, dout, clamp=0.0, causal=True):
    """d loss / d arrays[which][idx] by a central difference whose two steps
    are the exact float32 increments actually applied (the oracle takes
    float32 inputs)."""
    x = arrays[which]
    base = np.float32(x[idx])
    up, dn = np.float32(base + np.float32(h)), np.float32(base - np.float32(h))
    a, b = float(up) - float(base), float(base) - float(dn)
    xs = [arr.copy() for arr in arrays]
    xs[which][idx] = up
    f_up = _loss(L, *xs, kk, pi, dout, clamp, causal)
    xs[which][idx] = dn
    f_dn = _loss(L, *xs, kk, pi, dout, clamp, causal)
    return (f_up - f_dn) / (a + b)


def pin_backward_finite_differences(L):
    """The oracle gradients (Sec. 3.5 eqs. jac, ddelta_da, dalpha_da) equal
    central differences of the oracle's own forward, for q, k, v and the gate
    logit, with the partner inside and outside the window, with per-head
    and per-query gates, causal and bidirectional."""
    rng = np.random.default_rng(11)
    for (B, H, N, D, kk, pi, per_query, causal) in [
            (1, 2, 24, 8, 4, 8, False, True), (2, 1, 20, 8, 3, 3, True, True), (1, 1, 17, 16, 2, 5, True, True),
            (1, 2, 22, 8, 3, 7, True, False), (1, 1, 15, 8, 2, 2, False, False)]:
        q, k, v = rand_qkv(rng, B, H, N, D)
        gate = (rng.uniform(-1, 1, (B, H, N)) if per_query else rng.uniform(-1, 1, H)).astype(np.float32)
        dout = rng.standard_normal((B, H, N, D)).astype(np.float32)
        dq, dk, dv, dg = oracle.backward(q, k, v, gate, kk, pi, dout, L=L, causal=causal)
        grads = [dq, dk, dv]
        arrays = [q, k, v, gate]
        for which in range(4):
            for _ in range(6 if which < 3 else 4):
                idx = tuple(int(rng.integers(0, n)) for n in arrays[which].shape)
                fd = _central_difference(L, arrays, which, idx, 2.0 ** -8, kk, pi, dout, causal=causal)
                if which < 3:
                    an = grads[which][idx]
                elif per_query:
                    an = dg[idx]
                else:  # a per-head gate collects the gradient of every query of head h
                    an = dg[:, idx[0], :].sum()
                assert abs(fd - an) <= 5e-5 + 1e-3 * abs(an), (B, H, N, D, kk, pi, causal, which, idx, fd, an)


def pin_backward_dense_reduction(L):
    """With k >= N-1 and no partner the prior cancels and pi-Attention is dense
    causal attention (Sec. 3.2): q, k, v gradients equal torch autograd of the
    textbook softmax attention in fp64, and the gate gradient vanishes (the
    softmax Jacobian's rows sum to zero, eq. jac)."""
    import torch
    rng = np.random.default_rng(5)
    B, H, N, D = 2, 2, 19, 8
    q, k, v = rand_qkv(rng, B, H, N, D)
    gate = rng.uniform(-2, 2, H).astype(np.float32)
    dout = rng.standard_normal((B, H, N, D)).astype(np.float32)
    scale = 1.0 / math.sqrt(D)
    for causal in (True, False):   # bidirectional: no mask at all
        dq, dk, dv, dg = oracle.backward(q, k, v, gate, N - 1, 0, dout, L=L, causal=causal)
        tq, tk, tv = (torch.tensor(x, dtype=torch.float64, requires_grad=True) for x in (q, k, v))
        S = (tq @ tk.transpose(-1, -2)) * scale
        if causal:
            S = S.masked_fill(~torch.tril(torch.ones(N, N, dtype=torch.bool)), float("-inf"))
        y = torch.softmax(S, dim=-1) @ tv
        y.backward(torch.tensor(dout, dtype=torch.float64))
        for got, ref in ((dq, tq.grad), (dk, tk.grad), (dv, tv.grad)):
            assert np.allclose(got, ref.numpy(), rtol=1e-10, atol=1e-12), causal
        assert np.abs(dg).max() < 1e-12


def pin_backward_clamp_limits(L):
    """Logit clamp (App. B reading): a clamp that never binds changes no
    gradient; a clamp that binds everywhere cuts every path through the
    logits (dq = dk = 0, gate gradient 0) and leaves uniform weights, so dv_j
    is the mean of dL/dy over the queries whose working set holds j."""
    rng = np.random.default_rng(9)
    B, H, N, D, kk, pi = 1, 2, 18, 8, 3, 7
    q, k, v = rand_qkv(rng, B, H, N, D)
    gate = rng.uniform(-1, 1, H).astype(np.float32)
    dout = rng.standard_normal((B, H, N, D)).astype(np.float32)
    free = oracle.backward(q, k, v, gate, kk, pi, dout, L=L)
    loose = oracle.backward(q, k, v, gate, kk, pi, dout, clamp=1e6, L=L)
    for a, b in zip(free, loose):
        assert np.array_equal(a, b)
    dq, dk, dv, dg = oracle.backward(q, k, v, gate, kk, pi, dout, clamp=1e-7, L=L)
    assert not dq.any() and not dk.any() and not dg.any()
    M = scan_membership(N, kk, pi).astype(np.float64)           # [t, j]
    W = M / M.sum(-1, keepdims=True)
    ref = np.einsum("tj,bhtd->bhjd", W, np.asarray(dout, np.float64))
    assert np.allclose(dv, ref, atol=1e-5)


ALL_PINS += [pin_backward_finite_differences, pin_backward_dense_reduction, pin_backward_clamp_limits]
