"""GPU parity of the backward (pi_attn_backward through the C ABI) against
the fp64 oracle gradients on the same seeded inputs and cotangent.

Float32 inputs run float32 kernels and are held to a float32 bar: every
gradient entry within 1e-4 * max(1, max |ref|) of the oracle (a float32 sum
of at most k + 2 terms of size <= that scale errs by about
(k + 2) * 2^-24 * scale <= 3.1e-5 * scale at k = 512).  bf16 inputs take the
bf16 forward's output y in the row term <dL/dy, y> and feed bf16-rounded
softmax gradients to the MFMA products (2^-9 relative each), so they are
held to the forward's bf16 bar per gradient tensor: max-abs within
2e-2 * scale and relative L2 within 5e-3.  The gate gradient is compared per
query; a per-head gate's sum over (b, t) is then held to the same factor
times the sum of the per-query magnitudes.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2511_10696_amd as pa
from paper_2511_10696_amd import workloads as W

pytestmark = pytest.mark.gpu

GRAD_TOL = 1e-4
BF16_GRAD_MAXABS, BF16_GRAD_RELL2 = 2e-2, 5e-3


def np32(t):
    return t.detach().float().cpu().numpy()


def assert_grad(got, ref, what, dtype=torch.float32):
    got, ref = np.asarray(got, np.float64), np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.isfinite(got).all(), f"{what}: non-finite"
    scale = max(1.0, float(np.abs(ref).max()))
    err = float(np.abs(got - ref).max())
    if dtype == torch.float32:
        assert err <= GRAD_TOL * scale, f"{what}: max-abs {err:.3g} (scale {scale:.3g})"
        return
    rel = float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30))
    assert err <= BF16_GRAD_MAXABS * scale, f"{what}: max-abs {err:.3g} (scale {scale:.3g})"
    assert rel <= BF16_GRAD_RELL2 or err <= 1e-3 * scale, f"{what}: rel-L2 {rel:.3g}"


def run_case(q, k, v, gate, kw, pi, seed, clamp=0.0, scale=None):
    out, lse = pa.pi_attn_forward(q, k, v, gate, kw, pi, return_lse=True, logit_clamp=clamp, scale=scale)
    dout = W.cotangent(q.shape, q.dtype, seed, q.device)
    dq, dk, dv, dg = pa.pi_attn_backward(q, k, v, gate, kw, pi, out, lse, dout, logit_clamp=clamp,
                                         scale=scale, gate_grad_per_query=True)
    torch.cuda.synchronize()
    rq, rk, rv, rg = oracle.backward(q, k, v, gate, kw, pi, dout, scale=scale, clamp=clamp)
    for name, got, ref in (("dq", dq, rq), ("dk", dk, rk), ("dv", dv, rv), ("dgate", dg, rg)):
        assert_grad(np32(got), ref, name, q.dtype)
    if gate.dim() == 1:   # the per-head reduction the binding does by default
        *_, dgh = pa.pi_attn_backward(q, k, v, gate, kw, pi, out, lse, dout, logit_clamp=clamp, scale=scale)
        tol = GRAD_TOL if q.dtype == torch.float32 else BF16_GRAD_MAXABS
        bound = tol * np.maximum(1.0, np.abs(rg).sum(axis=(0, 2)))
        assert (np.abs(np32(dgh) - rg.sum(axis=(0, 2))) <= bound).all(), "per-head dgate"


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
