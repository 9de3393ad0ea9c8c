"""GPU tests of the sequence-shard calls: a sequence split into shards,
each shard's forward run on its queries with its k/v rows plus the halo
before (and, bidirectional, after) it, reproduces the whole-sequence
forward; the backward split the same way (each shard's query pass, the row
terms gathered as a neighbour would send them, each shard's key pass over
its keys with the query rows that reach them) reproduces the whole-sequence
gradients.

Shards whose first query (key) is a multiple of 128 run the same tiles in
the same order as the whole-sequence call, so their results must be
bit-identical to its rows.  Other shard boundaries are held to the bf16 bar
against the oracle.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2511_10696_amd as pa
from paper_2511_10696_amd import workloads as W
from tests.test_gpu_parity import LSE_TOL, assert_close, np32

pytestmark = pytest.mark.gpu


def halo_rows(nseq, k, pi, causal, qpos0, nq, align=True):
    """The k/v rows [lo, hi) a shard needs (the library's documented minimum,
    or the plain halo max(k, pi) rounded down to 32 when align)."""
    par = pi > k
    lo = max(0, qpos0 - k) & ~31
    if par:
        lo = min(lo, max(0, qpos0 - pi))
    if align:
        lo = lo & ~31
    hi = qpos0 + nq if causal else min(nseq, qpos0 + nq + (max(k, pi) if par else k))
    return lo, hi


def run_shards(q, k, v, gate, kw, pi, bounds, causal, pq, **fw):
    B, H, N, D = q.shape
    outs, lses = [], []
    for s0, s1 in bounds:
        lo, hi = halo_rows(N, kw, pi, causal, s0, s1 - s0)
        g = gate[:, :, s0:s1] if pq else gate
        o, l = pa.pi_attn_forward_shard(q[:, :, s0:s1], k[:, :, lo:hi], v[:, :, lo:hi], g, kw, pi, N, s0, lo,
                                        return_lse=True, causal=causal, **fw)
        outs.append(o)
        lses.append(l)
    return torch.cat(outs, dim=2), torch.cat(lses, dim=2)


@pytest.mark.parametrize("B,H,N,D,kw,pi,nshard", [
    (1, 2, 4096, 128, 512, 1024, 4),
    (2, 3, 2048, 64, 128, 256, 8),
    (1, 2, 1536, 128, 40, 100, 3),       # k, pi not multiples of 32
    (1, 1, 1024, 64, 200, 150, 2),       # pi <= k: no partner
])
@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("pq", [False, True])
def test_aligned_shards_are_bit_identical(device, B, H, N, D, kw, pi, nshard, causal, pq):
    cfg = W.ForwardConfig("custom", B, H, N, D, kw, pi, torch.bfloat16)
    q, k, v, gate = W.forward_inputs(cfg, 3, device, per_query_gate=pq)
    full, lfull = pa.pi_attn_forward(q, k, v, gate, kw, pi, return_lse=True, causal=causal)
    step = N // nshard
    assert step % 128 == 0
    bounds = [(i * step, (i + 1) * step) for i in range(nshard)]
    out, lse = run_shards(q, k, v, gate, kw, pi, bounds, causal, pq)
    torch.cuda.synchronize()
    assert torch.equal(out, full)
    assert torch.equal(lse, lfull)


@pytest.mark.parametrize("causal", [True, False])
def test_unaligned_shards_against_the_oracle(device, causal):
    B, H, N, D, kw, pi = 1, 2, 1000, 64, 48, 130
    cfg = W.ForwardConfig("custom", B, H, N, D, kw, pi, torch.bfloat16)
    q, k, v, gate = W.forward_inputs(cfg, 4, device, per_query_gate=True)
    bounds = [(0, 37), (37, 300), (300, 301), (301, 777), (777, 1000)]
    out, lse = run_shards(q, k, v, gate, kw, pi, bounds, causal, True)
    torch.cuda.synchronize()
    ref, lref = oracle.forward(q, k, v, gate, kw, pi, want_lse=True, causal=causal)
    assert_close(np32(out), ref, torch.bfloat16, "unaligned shards")
    assert np.abs(np32(lse) - lref).max() <= LSE_TOL


def test_minimal_halo_and_clamp(device):
    """The exact minimum k/v range of the header (not rounded further) and a
    binding logit clamp: rows equal the whole-sequence forward's."""
    B, H, N, D, kw, pi = 1, 2, 2048, 128, 96, 300
    cfg = W.ForwardConfig("hh", B, H, N, D, kw, pi, torch.bfloat16, heavy_frac=0.05, heavy_mult=8.0)
    q, k, v, gate = W.forward_inputs(cfg, 5, device)
    full = pa.pi_attn_forward(q, k, v, gate, kw, pi, scale=0.5, logit_clamp=3.0)
    s0, s1 = 1024, 1536
    lo, hi = halo_rows(N, kw, pi, True, s0, s1 - s0, align=False)
    out = pa.pi_attn_forward_shard(q[:, :, s0:s1], k[:, :, lo:hi], v[:, :, lo:hi], gate, kw, pi, N, s0, lo,
                                   scale=0.5, logit_clamp=3.0)
    torch.cuda.synchronize()
    assert torch.equal(out, full[:, :, s0:s1])


def test_shard_of_the_benchmark_workload(device):
    """fwd32k split eight ways as a sequence-sharded run would split it: the
    last rank's shard (queries [28672, 32768), k/v from 27648) against the
    whole-sequence forward."""
    cfg = W.FORWARD["fwd32k"]
    q, k, v, gate = W.forward_inputs(cfg, 0, device)
    N = cfg.N
    s0 = N - N // 8
    lo, hi = halo_rows(N, cfg.k, cfg.pi, True, s0, N - s0)
    assert lo == s0 - cfg.pi
    out = pa.pi_attn_forward_shard(q[:, :, s0:].contiguous(), k[:, :, lo:].contiguous(), v[:, :, lo:].contiguous(),
                                   gate, cfg.k, cfg.pi, N, s0, lo)
    full = pa.pi_attn_forward(q, k, v, gate, cfg.k, cfg.pi)
    torch.cuda.synchronize()
    assert torch.equal(out, full[:, :, s0:])


# ---------------------------------------------------------------------------
# backward over shards: the query pass per shard, the row terms gathered (the
# halo a neighbour would send), then the key pass per shard
# ---------------------------------------------------------------------------
def q_rows_for_keys(nseq, k, pi, causal, kpos0, nk):
    reach = max(k, pi) if pi > k else k
    return (kpos0 if causal else max(0, kpos0 - reach)), min(nseq, kpos0 + nk + reach)


def sharded_backward(q, k, v, gate, kw, pi, out, lse, dout, bounds, causal, pq):
    B, H, N, D = q.shape
    dqs, dgs, rts = [], [], []
    for s0, s1 in bounds:
        lo, hi = halo_rows(N, kw, pi, causal, s0, s1 - s0)
        g = gate[:, :, s0:s1] if pq else gate
        dq, dg, rt = pa.pi_attn_backward_shard_q(q[:, :, s0:s1], k[:, :, lo:hi], v[:, :, lo:hi], g, kw, pi, N, s0, lo,
                                                 out[:, :, s0:s1], lse[:, :, s0:s1].contiguous(), dout[:, :, s0:s1],
                                                 causal=causal)
        dqs.append(dq)
        dgs.append(dg)
        rts.append(rt)
    rowterm = torch.cat(rts, dim=2)
    dks, dvs = [], []
    for s0, s1 in bounds:
        qlo, qhi = q_rows_for_keys(N, kw, pi, causal, s0, s1 - s0)
        g = gate[:, :, qlo:qhi] if pq else gate
        dk, dv = pa.pi_attn_backward_shard_kv(q[:, :, qlo:qhi], k[:, :, s0:s1], v[:, :, s0:s1], g, kw, pi, N, s0, qlo,
                                              lse[:, :, qlo:qhi].contiguous(), rowterm[:, :, qlo:qhi].contiguous(),
                                              dout[:, :, qlo:qhi], causal=causal)
        dks.append(dk)
        dvs.append(dv)
    return tuple(torch.cat(x, dim=2) for x in (dqs, dks, dvs, dgs))


@pytest.mark.parametrize("B,H,N,D,kw,pi,nshard", [
    (1, 2, 4096, 128, 512, 1024, 4),
    (2, 3, 2048, 64, 128, 256, 8),
    (1, 2, 1536, 128, 40, 100, 3),
    (1, 1, 1024, 64, 200, 150, 2),       # pi <= k: no partner
])
@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("pq", [False, True])
def test_backward_shards_are_bit_identical(device, B, H, N, D, kw, pi, nshard, causal, pq):
    cfg = W.ForwardConfig("custom", B, H, N, D, kw, pi, torch.bfloat16)
    q, k, v, gate = W.forward_inputs(cfg, 6, device, per_query_gate=pq)
    out, lse = pa.pi_attn_forward(q, k, v, gate, kw, pi, return_lse=True, causal=causal)
    dout = W.cotangent(q.shape, q.dtype, 6, device)
    whole = pa.pi_attn_backward(q, k, v, gate, kw, pi, out, lse, dout, gate_grad_per_query=True, causal=causal)
    step = N // nshard
    bounds = [(i * step, (i + 1) * step) for i in range(nshard)]
    got = sharded_backward(q, k, v, gate, kw, pi, out, lse, dout, bounds, causal, pq)
    torch.cuda.synchronize()
    for name, a, b in zip(("dq", "dk", "dv", "dgate"), got, whole):
        assert torch.equal(a, b), name


@pytest.mark.parametrize("causal", [True, False])
def test_backward_unaligned_shards_against_the_oracle(device, causal):
    from tests.grad_check import assert_grad, expected_grads, forward_state
    B, H, N, D, kw, pi = 1, 2, 700, 64, 40, 130
    cfg = W.ForwardConfig("custom", B, H, N, D, kw, pi, torch.bfloat16)
    q, k, v, gate = W.forward_inputs(cfg, 7, device, per_query_gate=True)
    out, lse, y = forward_state(q, k, v, gate, kw, pi, causal=causal)
    dout = W.cotangent(q.shape, q.dtype, 7, device)
    bounds = [(0, 100), (100, 101), (101, 450), (450, 700)]
    got = sharded_backward(q, k, v, gate, kw, pi, out, lse, dout, bounds, causal, True)
    torch.cuda.synchronize()
    exp = expected_grads(q, k, v, gate, kw, pi, dout, out, y, causal=causal, row_term_from_out=True)
    for name, a, e in zip(("dq", "dk", "dv", "dgate"), got, exp):
        assert_grad(np32(a), e, name, torch.bfloat16)


@pytest.mark.parametrize("causal", [True, False])
def test_clamped_shards_are_bit_identical(device, causal):
    """A binding logit clamp through the sharded forward and both sharded
    backward passes: equal to the whole-sequence results."""
    B, H, N, D, kw, pi = 1, 2, 2048, 128, 96, 300
    cfg = W.ForwardConfig("hh", B, H, N, D, kw, pi, torch.bfloat16, heavy_frac=0.05, heavy_mult=8.0)
    q, k, v, gate = W.forward_inputs(cfg, 8, device, per_query_gate=True)
    fw = dict(scale=0.5, logit_clamp=3.0)
    out, lse = pa.pi_attn_forward(q, k, v, gate, kw, pi, return_lse=True, causal=causal, **fw)
    bounds = [(0, 512), (512, 1024), (1024, 1536), (1536, 2048)]
    sout, slse = run_shards(q, k, v, gate, kw, pi, bounds, causal, True, **fw)
    dout = W.cotangent(q.shape, q.dtype, 8, device)
    whole = pa.pi_attn_backward(q, k, v, gate, kw, pi, out, lse, dout, gate_grad_per_query=True, causal=causal, **fw)
    dqs, dgs, rts = [], [], []
    for s0, s1 in bounds:
        lo, hi = halo_rows(N, kw, pi, causal, s0, s1 - s0)
        dq, dg, rt = pa.pi_attn_backward_shard_q(q[:, :, s0:s1], k[:, :, lo:hi], v[:, :, lo:hi], gate[:, :, s0:s1],
                                                 kw, pi, N, s0, lo, out[:, :, s0:s1], lse[:, :, s0:s1].contiguous(),
                                                 dout[:, :, s0:s1], causal=causal, **fw)
        dqs.append(dq)
        dgs.append(dg)
        rts.append(rt)
    rowterm = torch.cat(rts, dim=2)
    dks, dvs = [], []
    for s0, s1 in bounds:
        qlo, qhi = q_rows_for_keys(N, kw, pi, causal, s0, s1 - s0)
        dk, dv = pa.pi_attn_backward_shard_kv(q[:, :, qlo:qhi], k[:, :, s0:s1], v[:, :, s0:s1], gate[:, :, qlo:qhi],
                                              kw, pi, N, s0, qlo, lse[:, :, qlo:qhi].contiguous(),
                                              rowterm[:, :, qlo:qhi].contiguous(), dout[:, :, qlo:qhi],
                                              causal=causal, **fw)
        dks.append(dk)
        dvs.append(dv)
    torch.cuda.synchronize()
    assert torch.equal(sout, out) and torch.equal(slse, lse)
    got = [torch.cat(x, dim=2) for x in (dqs, dks, dvs, dgs)]
    for name, a, b in zip(("dq", "dk", "dv", "dgate"), got, whole):
        assert torch.equal(a, b), name
