"""The gradient bar of every backward parity test, and the forward state the
backward is fed.

Inputs.  pi_attn_backward takes the forward's output y and its lse besides
q, k, v, the gate and dL/dy.  The tests hand it the oracle's forward state:
y rounded to the input dtype and lse rounded to float32.  So every input of
the backward is seeded or computed by the oracle, and no expected value
depends on the HIP forward (whose own parity is tested elsewhere).

Row term (Sec. 3.5, eq. jac).  The exact gradient uses
r*_t = sum_j alpha^_tj dL/dalpha^_tj = <dL/dy_t, y*_t>, y* the exact output.
The float32 passes, the banded bf16 passes (k > 16) and the shard passes
form dq with the row term of the output they are given,
r_t = <dL/dy_t, y_t> (the query pass needs r before its sweep over W_t
ends); the small-window bf16 passes (k <= 16) accumulate r* themselves.
Where dq takes r_t, in real arithmetic
    dq_t = dq*_t + scale (r*_t - r_t) Y_t,
    Y_t  = sum of alpha^_tj k_j over the entries of W_t the clamp does not
           saturate,
and dk, dv and the gate gradient use r* (the query pass writes it back as the
key pass's row term).  The expected dq carries that term, computed here in
fp64 from the oracle's y*, weights and keys and from the y that was passed.

Bar, per gradient tensor G against its expected value E (fp64):
  float32: max |G - E| <= 1e-4 max(1, max |E|)  (a float32 sum of at most
           2k + 3 terms of that scale errs by well under it);
  bf16:    max |G - E| <= 2e-2 max(1, max |E|) and
           ||G - E||_2 <= 5e-3 ||E||_2 + 1e-5 sqrt(size(G)),
the forward's bf16 bar, plus an RMS floor of 1e-5: float32 rounding of sums
of unit-scale terms (2^-24 relative each), which is all that a gradient
equal to zero in exact arithmetic shows (dq of a one-entry working set, the
gate gradient when every entry of W_t carries the same prior).
"""
from __future__ import annotations

import math

import numpy as np
import torch

import oracle
import paper_2511_10696_amd as pa
from paper_2511_10696_amd import workloads as W

F32_TOL = 1e-4
BF16_MAXABS, BF16_RELL2, RMS_FLOOR = 2e-2, 5e-3, 1e-5
SMALLK_MAX = 16   # bf16 with k <= 16 takes the small-window passes (include/pi_attn.h)


def np32(t):
    return t.detach().float().cpu().numpy()


def forward_state(q, k, v, gate, kw, pi, scale=None, clamp=0.0, causal=True):
    """The oracle's forward output and lse, rounded to what the backward
    takes (y in q's dtype, lse in float32, on q's device), and y in fp64."""
    y, lse = oracle.forward(q, k, v, gate, kw, pi, scale=scale, clamp=clamp, want_lse=True, causal=causal)
    out = torch.from_numpy(y.astype(np.float32)).to(q.device).to(q.dtype)
    lse_t = torch.from_numpy(lse.astype(np.float32)).to(q.device)
    return out, lse_t, y


def weighted_keys(q, k, gate, kw, pi, scale=None, clamp=0.0, causal=True):
    """Y_t = sum_j alpha^_tj k_j over the entries of W_t whose fused logit the
    clamp does not saturate (all of them without the clamp), fp64 [B,H,N,D]."""
    if clamp <= 0.0:
        return oracle.forward(q, k, k, gate, kw, pi, scale=scale, causal=causal)
    # the clamp saturates the entries whose unclamped fused logit has
    # |delta| >= clamp; delta = log alpha^ + lse of the unclamped softmax
    _, probs = oracle.forward(q, k, k, gate, kw, pi, scale=scale, clamp=clamp, want_probs=True, causal=causal)
    _, lse_u, probs_u = oracle.forward(q, k, k, gate, kw, pi, scale=scale, want_lse=True, want_probs=True,
                                       causal=causal)
    B, H, N, D = q.shape
    idx = oracle.index_set(N, kw, pi, causal=causal)
    with np.errstate(divide="ignore"):
        delta = np.log(probs_u) + lse_u[..., None]
    keep = (np.abs(delta) < clamp) & (idx >= 0)[None, None]
    w = np.where(keep, probs, 0.0)
    kf = np32(k).astype(np.float64)
    rows = np.maximum(idx, 0)
    Y = np.empty((B, H, N, D))
    for b in range(B):
        for h in range(H):
            Y[b, h] = np.einsum("tm,tmd->td", w[b, h], kf[b, h][rows])
    return Y


def dq_row_term_shift(dout, out, y_exact, Y, scale):
    """scale (r*_t - r_t) Y_t with r* = <dL/dy, y*> and r = <dL/dy, y>."""
    d = np32(dout).astype(np.float64)
    r_star = (d * y_exact).sum(-1)
    r_used = (d * np32(out).astype(np.float64)).sum(-1)
    return scale * (r_star - r_used)[..., None] * Y


def takes_row_term_from_out(dtype, kw, shard=False):
    return shard or dtype == torch.float32 or kw > SMALLK_MAX


def assert_grad(got, exp, what, dtype):
    got, exp = np.asarray(got, np.float64), np.asarray(exp, np.float64)
    assert got.shape == exp.shape, (what, got.shape, exp.shape)
    assert np.isfinite(got).all(), f"{what}: non-finite"
    scale = max(1.0, float(np.abs(exp).max())) if exp.size else 1.0
    err = float(np.abs(got - exp).max()) if exp.size else 0.0
    if dtype == torch.float32:
        assert err <= F32_TOL * scale, f"{what}: max-abs {err:.3g} (scale {scale:.3g})"
        return
    assert err <= BF16_MAXABS * scale, f"{what}: max-abs {err:.3g} (scale {scale:.3g})"
    ne, nr = float(np.linalg.norm(got - exp)), float(np.linalg.norm(exp))
    bound = BF16_RELL2 * nr + RMS_FLOOR * math.sqrt(exp.size)
    assert ne <= bound, f"{what}: ||err|| {ne:.3g} > {bound:.3g} (rel-L2 {ne / max(nr, 1e-300):.3g})"


def expected_grads(q, k, v, gate, kw, pi, dout, out, y_exact, scale=None, clamp=0.0, causal=True,
                   row_term_from_out=True):
    """The oracle's gradients (dq, dk, dv, per-query dgate), dq carrying the
    row-term shift where the path forms dq with the row term of `out`."""
    if scale is None:
        scale = 1.0 / math.sqrt(q.shape[-1])
    rq, rk, rv, rg = oracle.backward(q, k, v, gate, kw, pi, dout, scale=scale, clamp=clamp, causal=causal)
    if row_term_from_out:
        Y = weighted_keys(q, k, gate, kw, pi, scale=scale, clamp=clamp, causal=causal)
        rq = rq + dq_row_term_shift(dout, out, y_exact, Y, scale)
    return rq, rk, rv, rg


def check_backward(q, k, v, gate, kw, pi, seed, causal=True, clamp=0.0, scale=None, per_head_sum=True, extra=None):
    """Run pi_attn_backward on the oracle's forward state and hold every
    gradient to the bar; also the per-head gate reduction for an [H] gate.
    Returns the GPU gradients (dq, dk, dv, per-query dgate)."""
    out, lse, y = forward_state(q, k, v, gate, kw, pi, scale=scale, clamp=clamp, causal=causal)
    dout = W.cotangent(q.shape, q.dtype, seed, q.device)
    grads = pa.pi_attn_backward(q, k, v, gate, kw, pi, out, lse, dout, logit_clamp=clamp, scale=scale,
                                gate_grad_per_query=True, causal=causal)
    torch.cuda.synchronize()
    exp = expected_grads(q, k, v, gate, kw, pi, dout, out, y, scale=scale, clamp=clamp, causal=causal,
                         row_term_from_out=takes_row_term_from_out(q.dtype, kw))
    for name, got, e in zip(("dq", "dk", "dv", "dgate"), grads, exp):
        assert_grad(np32(got), e, name, q.dtype)
        if extra is not None:
            extra(name, np32(got), e)
    if per_head_sum and gate.dim() == 1:   # the per-head reduction the binding does by default
        *_, dgh = pa.pi_attn_backward(q, k, v, gate, kw, pi, out, lse, dout, logit_clamp=clamp, scale=scale,
                                      causal=causal)
        torch.cuda.synchronize()
        rg = exp[3]
        tol = F32_TOL if q.dtype == torch.float32 else BF16_MAXABS
        bound = tol * np.maximum(1.0, np.abs(rg).sum(axis=(0, 2)))
        assert (np.abs(np32(dgh) - rg.sum(axis=(0, 2))) <= bound).all(), "per-head dgate"
    return grads
