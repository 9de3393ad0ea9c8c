"""GPU parity of the backward (pi_attn_backward through the C ABI) against
the fp64 oracle gradients on the same seeded inputs and cotangent.

The backward is fed the oracle's forward state (y in the input dtype, lse
in float32) and every gradient is held to the bar stated in
tests/grad_check.py: float32 max-abs within 1e-4 * max(1, max|ref|); bf16
max-abs within 2e-2 * max(1, max|ref|) and L2 error within
5e-3 ||ref|| + 1e-5 sqrt(size), with dq's expected value carrying the
documented row-term shift of the paths that form dq with <dL/dy, y> from
the output they are given.  The gate gradient is compared per query; a
per-head gate's sum over (b, t) is then held to the same factor times the
sum of the per-query magnitudes.
"""
import numpy as np
import pytest
import torch

import paper_2511_10696_amd as pa
from paper_2511_10696_amd import workloads as W
from tests.grad_check import assert_grad, check_backward, np32  # noqa: F401

pytestmark = pytest.mark.gpu


def run_case(q, k, v, gate, kw, pi, seed, clamp=0.0, scale=None, causal=True):
    return check_backward(q, k, v, gate, kw, pi, seed, causal=causal, clamp=clamp, scale=scale)


def inputs(B, H, N, D, dtype, seed, per_query_gate=False):
    cfg = W.ForwardConfig("custom", B, H, N, D, 0, 0, dtype)
    return W.forward_inputs(cfg, seed, "cuda", per_query_gate)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_backward_f32_tiny(device, seed):
    cfg = W.FORWARD["tiny"]
    q, k, v, gate = W.forward_inputs(cfg, seed, device)
    run_case(q, k, v, gate, cfg.k, cfg.pi, seed)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("B,H,N,D,k,pi,pq", [
    (1, 2, 300, 64, 32, 64, False),      # several tiles, ragged tail
    (1, 2, 200, 128, 16, 40, True),      # D = 128, per-query gate
    (2, 1, 130, 64, 5, 3, False),        # pi <= k: no partner slot
    (1, 2, 70, 128, 100, 7, True),       # k >= N: dense causal plus nothing
    (1, 1, 1, 64, 4, 16, False),         # a single position
    (1, 1, 40, 64, 0, 0, False),         # k = 0: self only
    (1, 1, 45, 64, 3, 44, True),         # partner only for the last position
])
def test_backward_shapes(device, dtype, B, H, N, D, k, pi, pq):
    q, kk, v, gate = inputs(B, H, N, D, dtype, 7, pq)
    run_case(q, kk, v, gate, k, pi, 7)


def test_backward_bf16_mid(device):
    """One D = 128 head pair at the 32K workload's window and period."""
    q, kk, v, gate = inputs(1, 2, 4096, 128, torch.bfloat16, 3)
    run_case(q, kk, v, gate, 512, 1024, 3)


def test_backward_bf16_fwd4k(device):
    cfg = W.FORWARD["fwd4k"]
    q, kk, v, gate = W.forward_inputs(cfg, 0, device)
    run_case(q, kk, v, gate, cfg.k, cfg.pi, 0)


def _clamp_placement():
    """A gate logit g and clamp L such that, for scores on the grid
    Z = (1/128) Z, no fused logit z + log omega (omega = alpha~ on the window,
    1 - alpha~ on the partner) lies within 1e-3 of +-L."""
    eps = 1e-4
    g = np.linspace(-2.0, 2.0, 801)[:, None]
    L = np.arange(0.75, 2.5, 1.0 / 2048)[None, :]
    at = eps + (1 - 2 * eps) / (1 + np.exp(-g))
    worst = np.full(np.broadcast(g, L).shape, 1.0)
    for b in (np.log(at), np.log1p(-at)):
        for edge in (L - b, -L - b):
            frac = np.mod(edge * 128.0, 1.0)
            worst = np.minimum(worst, np.minimum(frac, 1.0 - frac) / 128.0)
    i, j = np.unravel_index(np.argmax(worst), worst.shape)
    return float(worst[i, j]), float(g[i, 0]), float(L[0, j])


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_backward_clamp(device, dtype):
    """Clamp on: saturated logits pass no gradient.  Inputs are multiples of
    1/4 in [-2, 2] and scale = 1/8, so every score is a multiple of 1/128;
    the gate and the clamp are placed so that no fused logit comes within
    1e-3 of +-clamp (both sides disagreeing on a saturation would otherwise
    be decided by rounding)."""
    B, H, N, D, kw, pi = 1, 2, 150, 64, 20, 33
    gen = torch.Generator(device="cuda").manual_seed(5)
    q, kk, v = (torch.randint(-8, 9, (B, H, N, D), generator=gen, device="cuda").float().div(4).to(dtype)
                for _ in range(3))
    margin, g, clamp = _clamp_placement()
    assert margin > 1e-3
    gate = torch.full((H,), g, device="cuda")
    run_case(q, kk, v, gate, kw, pi, 5, clamp=clamp, scale=0.125)


@pytest.mark.parametrize("B,H,N", [(2, 3, 1000), (1, 40, 70001), (3, 1, 1), (2, 5, 0)])
def test_gate_grad_per_head(device, B, H, N):
    """pi_attn_gate_grad_per_head sums the per-query gate gradients over b
    and t: against an fp64 sum of the same values, within 1e-6 of the summed
    magnitudes (fp64 sums, one float32 rounding at the end); zeros when
    there are no queries; deterministic."""
    import ctypes
    g = torch.Generator(device="cuda").manual_seed(B * 1000 + H)
    dg = torch.randn(B, H, N, generator=g, device="cuda") * 3
    out = torch.full((H,), float("nan"), device="cuda")
    lib = pa.library()
    st = lib.pi_attn_gate_grad_per_head(B, H, N, ctypes.c_void_p(dg.data_ptr()), ctypes.c_void_p(out.data_ptr()),
                                        None)
    assert st == 0
    torch.cuda.synchronize()
    ref = np32(dg).astype(np.float64).sum(axis=(0, 2))
    bound = 1e-6 * np.maximum(1.0, np.abs(np32(dg)).astype(np.float64).sum(axis=(0, 2)))
    assert (np.abs(np32(out) - ref) <= bound).all()
    out2 = torch.empty_like(out)
    lib.pi_attn_gate_grad_per_head(B, H, N, ctypes.c_void_p(dg.data_ptr()), ctypes.c_void_p(out2.data_ptr()), None)
    torch.cuda.synchronize()
    assert torch.equal(out, out2)


def _fused_logits(q, k, gate, kw, pi, causal):
    """The unclamped fused logits of every entry of W_t (oracle, fp64)."""
    import oracle
    _, lse, probs = oracle.forward(q, k, k, gate, kw, pi, want_lse=True, want_probs=True, causal=causal)
    idx = oracle.index_set(q.shape[2], kw, pi, causal=causal)
    with np.errstate(divide="ignore"):
        delta = np.log(probs) + lse[..., None]
    return delta[np.broadcast_to((idx >= 0)[None, None], delta.shape)]


@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("clamped", [False, True])
def test_backward_bf16_three_rows(device, causal, clamped):
    """B1 H2 N3 D128 k150 pi1: three rows, dense, the banded passes.  The
    exact dq of such a tensor is small against |dL/dy| |y|, so the row term
    taken from the bf16 output moves dq by about 1% of its norm; the
    expected dq carries that shift and the rest is held to the bf16 bar.
    With the clamp, the clamp is the one of a fixed list that leaves every
    fused logit farthest from +-clamp (at least 1e-3, checked here, so both
    sides cut the same entries) while cutting at least one."""
    seed = 467447612    # the random-sweep case that first showed the shift (dq rel-L2 0.92%)
    q, kk, v, gate = inputs(1, 2, 3, 128, torch.bfloat16, seed)
    clamp = 0.0
    if clamped:
        d = _fused_logits(q, kk, gate, 150, 1, causal)
        cands = [c for c in np.arange(0.5, 3.0, 0.0625) if (np.abs(d) >= c).any()]
        margins = [float(np.abs(np.abs(d) - c).min()) for c in cands]
        clamp = float(cands[int(np.argmax(margins))])
        assert max(margins) > 1e-3
    run_case(q, kk, v, gate, 150, 1, seed, clamp=clamp, causal=causal)


def _config_heads(cfg, causal, n_pairs, seed):
    """The backward at a workload's full shape, launched as the benchmark
    launches it (every head, per-head gates), checked on n_pairs seeded
    (b, h) pairs in full: heads are independent, so each checked pair gets
    the oracle's forward state and its gradients are compared whole."""
    from tests.grad_check import expected_grads, forward_state
    q, k, v, gate = W.forward_inputs(cfg, 0, "cuda")
    out, lse = pa.pi_attn_forward(q, k, v, gate, cfg.k, cfg.pi, return_lse=True, causal=causal)
    rng = np.random.default_rng(seed)
    flat = rng.choice(cfg.B * cfg.H, n_pairs, replace=False)
    pairs = [(int(f) // cfg.H, int(f) % cfg.H) for f in flat]
    dout = W.cotangent(q.shape, q.dtype, 0, "cuda")
    sl = {}
    for b, h in pairs:
        qs, ks, vs = (x[b:b + 1, h:h + 1] for x in (q, k, v))
        gs = gate[h:h + 1]
        ostate, lstate, y = forward_state(qs, ks, vs, gs, cfg.k, cfg.pi, causal=causal)
        out[b, h] = ostate[0, 0]
        lse[b, h] = lstate[0, 0]
        sl[(b, h)] = (qs, ks, vs, gs, ostate, y)
    grads = pa.pi_attn_backward(q, k, v, gate, cfg.k, cfg.pi, out, lse, dout, gate_grad_per_query=True,
                                causal=causal)
    torch.cuda.synchronize()
    for (b, h), (qs, ks, vs, gs, ostate, y) in sl.items():
        exp = expected_grads(qs, ks, vs, gs, cfg.k, cfg.pi, dout[b:b + 1, h:h + 1], ostate, y, causal=causal,
                             row_term_from_out=True)
        for name, got, e in zip(("dq", "dk", "dv", "dgate"), grads, exp):
            assert_grad(np32(got[b:b + 1, h:h + 1]), e, f"{name} b{b} h{h}", torch.bfloat16)


@pytest.mark.parametrize("causal", [True, False])
def test_backward_config_fwd32k(device, causal):
    """The benchmarked backward: fwd32k (B1 H32 N32768 D128 k512 pi1024),
    two whole heads against the oracle."""
    _config_heads(W.FORWARD["fwd32k"], causal, 2, 11)


def test_backward_config_fwd16k(device):
    """fwd16k (B2 H32 N16384 D128 k256 pi512, heavy-hitter keys): two whole
    (b, h) pairs against the oracle."""
    _config_heads(W.FORWARD["fwd16k"], True, 2, 12)
