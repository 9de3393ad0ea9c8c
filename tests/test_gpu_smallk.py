"""GPU parity of the small-window path (k <= 16, the paper's default k = 4,
pi = 16) and of the gated forward (gate logits from the gate MLP's last
layer) against the fp64 oracle, through the C ABI.  Bars as in the causal
tests: bf16 outputs max-abs <= 2e-2 and relative L2 <= 5e-3, float32
max-abs <= 1e-4, lse within 1e-3.  The gate logits are an fp32 sum of dh
bf16 products and are held to 1e-5 of sum |u w2| + 1e-6.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2511_10696_amd as pa
from paper_2511_10696_amd import workloads as W
from tests.test_gpu_parity import LSE_TOL, assert_close, np32

pytestmark = pytest.mark.gpu


def inputs(B, H, N, D, dtype, seed, per_query_gate=False):
    cfg = W.ForwardConfig("custom", B, H, N, D, 0, 0, dtype)
    return W.forward_inputs(cfg, seed, "cuda", per_query_gate)


SHAPES = [
    (2, 3, 100, 64, 4, 16),       # the paper's default window and period, ragged tail
    (1, 2, 257, 128, 4, 16),      # D = 128
    (1, 1, 1, 64, 4, 16),         # a single position
    (1, 2, 70, 64, 0, 0),         # self only
    (1, 2, 90, 64, 16, 40),       # the largest window of the path
    (1, 40, 65, 64, 2, 8),        # more heads than one group
    (1, 3, 200, 128, 8, 3),       # pi <= k: no partner slot
    (1, 2, 300, 64, 4, 1000),     # partner beyond the sequence
    (2, 5, 1000, 64, 3, 64),
    (1, 2, 33, 128, 16, 32),      # tile boundary, band wider than the tile
]


@pytest.mark.parametrize("B,H,N,D,k,pi", SHAPES)
@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("pq", [False, True])
def test_forward_shapes(device, B, H, N, D, k, pi, causal, pq):
    q, k_, v, gate = inputs(B, H, N, D, torch.bfloat16, 7, pq)
    out, lse = pa.pi_attn_forward(q, k_, v, gate, k, pi, return_lse=True, causal=causal)
    torch.cuda.synchronize()
    ref, lref = oracle.forward(q, k_, v, gate, k, pi, want_lse=True, causal=causal)
    assert_close(np32(out), ref, torch.bfloat16, f"{(B, H, N, D, k, pi, causal)}")
    assert np.abs(np32(lse) - lref).max() <= LSE_TOL


def test_self_only_is_exact(device):
    q, k, v, gate = inputs(1, 3, 150, 64, torch.bfloat16, 3)
    for causal in (True, False):
        out = pa.pi_attn_forward(q, k, v, gate, 0, 0, causal=causal)
        torch.cuda.synchronize()
        assert torch.equal(out, v)


@pytest.mark.parametrize("causal", [True, False])
def test_clamp(device, causal):
    cfg = W.ForwardConfig("hh", 1, 2, 300, 64, 4, 16, torch.bfloat16, heavy_frac=0.05, heavy_mult=8.0)
    q, k, v, gate = W.forward_inputs(cfg, 2, device, per_query_gate=True)
    for clamp in (20.0, 3.0):
        out, lse = pa.pi_attn_forward(q, k, v, gate, 4, 16, scale=0.5, logit_clamp=clamp, return_lse=True,
                                      causal=causal)
        torch.cuda.synchronize()
        ref, lref = oracle.forward(q, k, v, gate, 4, 16, scale=0.5, clamp=clamp, want_lse=True, causal=causal)
        assert_close(np32(out), ref, torch.bfloat16, f"clamp {clamp}")
        assert np.abs(np32(lse) - lref).max() <= LSE_TOL * 10


def test_strided_layout(device):
    """[B, N, H, D] storage viewed as [B, H, N, D]: same result as contiguous."""
    B, H, N, D = 2, 3, 300, 64
    g = torch.Generator(device="cuda").manual_seed(9)
    base = [torch.randn(B, N, H, D, generator=g, device="cuda").to(torch.bfloat16) for _ in range(3)]
    q, k, v = (x.permute(0, 2, 1, 3) for x in base)
    gate = torch.rand(H, generator=g, device="cuda") * 2 - 1
    out_s = torch.empty(B, N, H, D, dtype=torch.bfloat16, device="cuda").permute(0, 2, 1, 3)
    pa.pi_attn_forward(q, k, v, gate, 4, 16, out=out_s)
    out_c = pa.pi_attn_forward(q.contiguous(), k.contiguous(), v.contiguous(), gate, 4, 16)
    torch.cuda.synchronize()
    assert torch.equal(out_s, out_c)


@pytest.mark.parametrize("causal", [True, False])
def test_causality_and_determinism(device, causal):
    q, k, v, gate = inputs(1, 2, 400, 64, torch.bfloat16, 11)
    a = pa.pi_attn_forward(q, k, v, gate, 4, 16, causal=causal)
    b = pa.pi_attn_forward(q, k, v, gate, 4, 16, causal=causal)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    if causal:   # NaN after `cut` never reaches rows <= cut
        for cut in (0, 31, 32, 200):
            q2, k2, v2 = q.clone(), k.clone(), v.clone()
            for x in (q2, k2, v2):
                x[:, :, cut + 1:] = float("nan")
            c = pa.pi_attn_forward(q2, k2, v2, gate, 4, 16)
            torch.cuda.synchronize()
            assert torch.equal(c[:, :, :cut + 1], a[:, :, :cut + 1]), cut


def sampled_rows(cfg, rng):
    B, H, N = cfg.B, cfg.H, cfg.N
    bh = rng.choice(B * H, size=2, replace=False)
    rows = [np.arange(N) + x * N for x in bh]
    edge = np.concatenate([np.arange(64), np.arange(N - 64, N)])
    rows += [edge + x * N for x in range(B * H)]
    rows.append(rng.choice(B * H * N, 2048, replace=False))
    return np.unique(np.concatenate(rows))


@pytest.mark.parametrize("causal", [True, False])
def test_config_smallk8k_sampled(device, causal):
    cfg = W.FORWARD["smallk8k"]
    q, k, v, gate = W.forward_inputs(cfg, 0, device, per_query_gate=True)
    out, lse = pa.pi_attn_forward(q, k, v, gate, cfg.k, cfg.pi, return_lse=True, causal=causal)
    torch.cuda.synchronize()
    rows = sampled_rows(cfg, np.random.default_rng(0))
    ref, lref = oracle.forward(q, k, v, gate, cfg.k, cfg.pi, rows=rows, want_lse=True, causal=causal)
    assert_close(np32(out).reshape(-1, cfg.D)[rows], ref, torch.bfloat16, "smallk8k")
    assert np.abs(np32(lse).reshape(-1)[rows] - lref).max() <= LSE_TOL


# ---------------------------------------------------------------------------
# gated forward: the gate MLP's last layer inside the operator
# ---------------------------------------------------------------------------
def check_gated(q, k, v, u, w2, b2, kw, pi, causal, rows=None, **kw2):
    out, g, lse = pa.pi_attn_forward_gated(q, k, v, u, w2, b2, kw, pi, return_lse=True, causal=causal, **kw2)
    torch.cuda.synchronize()
    gref = oracle.gate_logits(u, w2, np.zeros(w2.shape[0]) if b2 is None else b2)
    bound = 1e-5 * (np.abs(np32(u)) @ np.abs(np32(w2)).T).transpose(0, 2, 1) + 1e-6
    assert (np.abs(np32(g) - gref) <= bound).all(), float(np.abs(np32(g) - gref).max())
    ref, lref = oracle.forward(q, k, v, gref, kw, pi, rows=rows, want_lse=True, causal=causal,
                               scale=kw2.get("scale"), clamp=kw2.get("logit_clamp", 0.0))
    D = q.shape[-1]
    got = np32(out) if rows is None else np32(out).reshape(-1, D)[rows]
    gl = np32(lse) if rows is None else np32(lse).reshape(-1)[rows]
    assert_close(got, ref, q.dtype, "gated")
    assert np.abs(gl - lref).max() <= LSE_TOL
    return g


@pytest.mark.parametrize("B,H,N,D,k,pi,dh", [
    (2, 3, 100, 64, 4, 16, 96),       # default window and period
    (1, 40, 70, 64, 2, 8, 64),        # heads in two groups of the gate product
    (1, 2, 33, 128, 3, 12, 24),       # dh not a multiple of 16
    (1, 2, 300, 64, 30, 100, 32),     # k > 16: gate kernel, then the banded forward
])
@pytest.mark.parametrize("causal", [True, False])
def test_gated_forward(device, B, H, N, D, k, pi, dh, causal):
    cfg = W.ForwardConfig("custom", B, H, N, D, k, pi, torch.bfloat16)
    q, k_, v, _ = W.forward_inputs(cfg, 4, device)
    u, w2, b2 = W.gate_mlp_inputs(cfg, 4, device, dh=dh)
    check_gated(q, k_, v, u, w2, b2, k, pi, causal)
    check_gated(q, k_, v, u, w2, None, k, pi, causal)


def test_gated_forward_f32(device):
    cfg = W.ForwardConfig("custom", 1, 3, 90, 64, 4, 16, torch.float32)
    q, k, v, _ = W.forward_inputs(cfg, 5, device)
    u, w2, b2 = W.gate_mlp_inputs(cfg, 5, device, dh=40)
    check_gated(q, k, v, u, w2, b2, 4, 16, True)


def test_gated_config_smallk8k(device):
    cfg = W.FORWARD["smallk8k"]
    q, k, v, _ = W.forward_inputs(cfg, 0, device)
    u, w2, b2 = W.gate_mlp_inputs(cfg, 0, device)
    rows = sampled_rows(cfg, np.random.default_rng(1))
    check_gated(q, k, v, u, w2, b2, cfg.k, cfg.pi, True, rows=rows)


def test_gated_logits_feed_the_backward(device):
    """The gate logits the gated forward writes are laid out as the per-query
    gate of pi_attn_backward: they match the oracle's logits, and the
    backward on those logits (rounded to float32 by the oracle side) meets
    the gradient bar."""
    from tests.grad_check import check_backward
    cfg = W.ForwardConfig("custom", 1, 2, 200, 64, 4, 16, torch.bfloat16)
    q, k, v, _ = W.forward_inputs(cfg, 6, device)
    u, w2, b2 = W.gate_mlp_inputs(cfg, 6, device)
    _, g = pa.pi_attn_forward_gated(q, k, v, u, w2, b2, 4, 16)
    torch.cuda.synchronize()
    gref = oracle.gate_logits(u, w2, b2)
    assert g.shape == gref.shape and g.is_contiguous()
    bound = 1e-5 * (np.abs(np32(u)) @ np.abs(np32(w2)).T).transpose(0, 2, 1) + 1e-6
    assert (np.abs(np32(g) - gref) <= bound).all()
    gate = torch.from_numpy(gref.astype(np.float32)).to(device)
    check_backward(q, k, v, gate, 4, 16, 6)
