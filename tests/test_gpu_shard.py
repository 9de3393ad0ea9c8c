"""GPU tests of pi_attn_forward_shard: a sequence split into shards, each
shard's forward run on its queries with its k/v rows plus the halo before
(and, bidirectional, after) it, reproduces the whole-sequence forward.

Shards whose first query is a multiple of 128 and whose k/v rows start at a
multiple of 32 run the same tiles in the same order as the whole-sequence
call, so their outputs and lse must be bit-identical to its rows.  Other
shard boundaries are held to the bf16 bar against the oracle.
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
