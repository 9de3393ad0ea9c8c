"""Guard bands around every output of every entry point.

Each output buffer (attention outputs, lse, gradients, row terms, the index
table, decode caches, lengths, per-head gate gradients) is a view into a
larger allocation whose 4 KiB margins on both sides are filled with a
byte pattern (0xff, a NaN, for float32 and bf16 outputs; 0x5a for int32
outputs, whose -1 is a legitimate value).  Shapes are
ragged: sequence lengths off the 128-query tiling, tail tiles shorter than
a 32-row block, shard cuts off the tile grid.  After each call the margins
must be bit-unchanged (nothing writes past an output), and the output
itself, pre-filled with the same pattern, must hold no pattern left over
where the call defines every element (every element is written).  Invalid
positions are masked, never touched (App. A).
"""
import numpy as np
import pytest
import torch

import paper_2511_10696_amd as pa
from paper_2511_10696_amd import workloads as W

pytestmark = pytest.mark.gpu

MARGIN = 4096


class Guarded:
    """A tensor of `shape` and `dtype` inside a byte buffer with MARGIN
    pattern bytes before and after it."""

    def __init__(self, shape, dtype):
        es = torch.empty((), dtype=dtype).element_size()
        self.fill = 0x5A if dtype == torch.int32 else 0xFF
        self.nbytes = int(np.prod(shape)) * es
        self.buf = torch.full((MARGIN + self.nbytes + MARGIN,), self.fill, dtype=torch.uint8, device="cuda")
        self.t = self.buf[MARGIN:MARGIN + self.nbytes].view(dtype).view(shape)

    def margins_intact(self):
        f = self.fill
        return bool((self.buf[:MARGIN] == f).all()) and bool((self.buf[MARGIN + self.nbytes:] == f).all())

    def all_written(self):
        """No element still holds the fill pattern."""
        inner = self.buf[MARGIN:MARGIN + self.nbytes]
        es = self.t.element_size()
        return not bool((inner.view(-1, es) == self.fill).all(dim=1).any())


def check(*gs, written=True):
    torch.cuda.synchronize()
    for g in gs:
        assert g.margins_intact(), "a margin was written"
        if written:
            assert g.all_written(), "an output element was not written"


def inputs(B, H, N, D, dtype, seed, pq=False):
    cfg = W.ForwardConfig("custom", B, H, N, D, 0, 0, dtype)
    return W.forward_inputs(cfg, seed, "cuda", per_query_gate=pq)


@pytest.mark.parametrize("n,k,pi,causal", [(1000, 33, 100, True), (77, 5, 16, False), (1, 4, 16, True)])
def test_index_set(device, n, k, pi, causal):
    m = pa.pi_attn_ws_width(k, pi, causal)
    idx = Guarded((n, m), torch.int32)
    pa.pi_attn_index_set(n, k, pi, out=idx.t, causal=causal)
    check(idx)


FWD_CASES = [
    # B, H, N, D, k, pi, dtype, causal, per-query gate
    (1, 2, 1000, 128, 64, 200, torch.bfloat16, True, False),    # banded, tail tile of 104 queries
    (2, 3, 333, 64, 100, 150, torch.bfloat16, False, True),     # banded bidirectional
    (1, 3, 1001, 64, 4, 16, torch.bfloat16, True, True),        # small window, tail of 9 tokens
    (2, 2, 97, 128, 16, 40, torch.bfloat16, False, False),      # small window bidirectional
    (1, 2, 300, 64, 32, 64, torch.float32, True, False),        # float32
    (1, 1, 1, 128, 512, 1024, torch.bfloat16, True, False),     # one position
]


@pytest.mark.parametrize("case", FWD_CASES)
def test_forward(device, case):
    B, H, N, D, k, pi, dtype, causal, pq = case
    q, kk, v, gate = inputs(B, H, N, D, dtype, 1, pq)
    out, lse = Guarded((B, H, N, D), dtype), Guarded((B, H, N), torch.float32)
    pa.pi_attn_forward(q, kk, v, gate, k, pi, out=out.t, lse=lse.t, causal=causal)
    check(out, lse)


@pytest.mark.parametrize("k,causal", [(4, True), (40, False)])
def test_forward_gated(device, k, causal):
    B, H, N, D = 2, 3, 211, 64
    cfg = W.ForwardConfig("custom", B, H, N, D, k, 3 * k, torch.bfloat16)
    q, kk, v, _ = W.forward_inputs(cfg, 2, "cuda")
    u, w2, b2 = W.gate_mlp_inputs(cfg, 2, "cuda", dh=96)
    out, lse, g = Guarded((B, H, N, D), torch.bfloat16), Guarded((B, H, N), torch.float32), Guarded(
        (B, H, N), torch.float32)
    pa.pi_attn_forward_gated(q, kk, v, u, w2, b2, k, 3 * k, out=out.t, lse=lse.t, gate_out=g.t, causal=causal)
    check(out, lse, g)


BWD_CASES = [
    (1, 2, 1000, 128, 64, 200, torch.bfloat16, True, False),    # banded passes
    (1, 2, 333, 64, 100, 150, torch.bfloat16, False, True),
    (2, 2, 1001, 64, 4, 16, torch.bfloat16, True, True),        # small-window passes
    (1, 3, 97, 128, 16, 40, torch.bfloat16, False, False),
    (1, 2, 300, 64, 32, 64, torch.float32, False, True),        # float32 passes
]


@pytest.mark.parametrize("case", BWD_CASES)
def test_backward(device, case):
    B, H, N, D, k, pi, dtype, causal, pq = case
    q, kk, v, gate = inputs(B, H, N, D, dtype, 3, pq)
    y, l = pa.pi_attn_forward(q, kk, v, gate, k, pi, return_lse=True, causal=causal)
    dout = W.cotangent(q.shape, q.dtype, 3, "cuda")
    f32 = torch.float32
    gs = [Guarded((B, H, N, D), f32) for _ in range(3)] + [Guarded((B, H, N), f32) for _ in range(2)]
    pa.pi_attn_backward(q, kk, v, gate, k, pi, y, l, dout, gate_grad_per_query=True, causal=causal,
                        dq=gs[0].t, dk=gs[1].t, dv=gs[2].t, dgate=gs[3].t, rowterm=gs[4].t)
    check(*gs)
    # the no-allocation entry point into guarded outputs
    ns = [Guarded((B, H, N, D), f32) for _ in range(3)] + [Guarded((B, H, N), f32)]
    pa.pi_attn_backward_noalloc(q, kk, v, gate, k, pi, y, l, dout, *(g.t for g in ns), causal=causal)
    check(*ns)
    if gate.dim() == 1:   # the per-head gate reduction
        gh = Guarded((H,), f32)
        st = pa.library().pi_attn_gate_grad_per_head(B, H, N, pa._ptr(gs[3].t), pa._ptr(gh.t), None)
        assert st == 0
        check(gh)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_decode(device, dtype):
    S, H, D, cap, k, pi = 5, 3, 128, 300, 37, 100
    g = torch.Generator(device="cuda").manual_seed(4)
    kc, vc = Guarded((S, H, cap, D), dtype), Guarded((S, H, cap, D), dtype)
    kc.t.copy_(torch.randn(S, H, cap, D, generator=g, device="cuda").to(dtype))
    vc.t.copy_(torch.randn(S, H, cap, D, generator=g, device="cuda").to(dtype))
    lens = torch.tensor([0, 1, 150, 298, cap - 1], dtype=torch.int32, device="cuda")
    qn, kn, vn = (torch.randn(S, H, D, generator=g, device="cuda").to(dtype) for _ in range(3))
    gate = torch.rand(H, generator=g, device="cuda") * 2 - 1
    out, lse, lo = Guarded((S, H, D), dtype), Guarded((S, H), torch.float32), Guarded((S,), torch.int32)
    kc0, vc0 = kc.t.clone(), vc.t.clone()
    pa.pi_attn_decode_step(lens, qn, kn, vn, kc.t, vc.t, gate, k, pi, len_out=lo.t, out=out.t, lse=lse.t)
    check(out, lse, lo)
    check(kc, vc, written=False)
    # only row len_in[s] of each (s, h) changed
    for s in range(S):
        t = int(lens[s])
        keep = torch.ones(cap, dtype=torch.bool, device="cuda")
        keep[t] = False
        assert torch.equal(kc.t[s][:, keep], kc0[s][:, keep]) and torch.equal(vc.t[s][:, keep], vc0[s][:, keep])


@pytest.mark.parametrize("causal", [True, False])
def test_shards(device, causal):
    """A sequence cut at 100, 357 and 700 (off the 128-query grid): each
    shard's forward, query pass and key pass into guarded outputs."""
    from tests.test_gpu_shard import halo_rows, q_rows_for_keys
    B, H, N, D, kw, pi = 1, 2, 900, 64, 40, 130
    q, k, v, gate = inputs(B, H, N, D, torch.bfloat16, 5, pq=True)
    y, l = pa.pi_attn_forward(q, k, v, gate, kw, pi, return_lse=True, causal=causal)
    dout = W.cotangent(q.shape, q.dtype, 5, "cuda")
    bounds = [(0, 100), (100, 357), (357, 700), (700, 900)]
    f32 = torch.float32
    rts = []
    for s0, s1 in bounds:
        n = s1 - s0
        lo, hi = halo_rows(N, kw, pi, causal, s0, n)
        out, lse = Guarded((B, H, n, D), torch.bfloat16), Guarded((B, H, n), f32)
        pa.pi_attn_forward_shard(q[:, :, s0:s1], k[:, :, lo:hi], v[:, :, lo:hi], gate[:, :, s0:s1], kw, pi, N, s0,
                                 lo, out=out.t, lse=lse.t, causal=causal)
        dq, dg, rt = Guarded((B, H, n, D), f32), Guarded((B, H, n), f32), Guarded((B, H, n), f32)
        pa.pi_attn_backward_shard_q(q[:, :, s0:s1], k[:, :, lo:hi], v[:, :, lo:hi], gate[:, :, s0:s1], kw, pi, N,
                                    s0, lo, y[:, :, s0:s1], l[:, :, s0:s1].contiguous(), dout[:, :, s0:s1],
                                    causal=causal, dq=dq.t, dgate=dg.t, rowterm=rt.t)
        check(out, lse, dq, dg, rt)
        rts.append(rt.t.clone())
    rowterm = torch.cat(rts, dim=2)
    for s0, s1 in bounds:
        n = s1 - s0
        qlo, qhi = q_rows_for_keys(N, kw, pi, causal, s0, n)
        dk, dv = Guarded((B, H, n, D), f32), Guarded((B, H, n, D), f32)
        pa.pi_attn_backward_shard_kv(q[:, :, qlo:qhi], k[:, :, s0:s1], v[:, :, s0:s1], gate[:, :, qlo:qhi], kw, pi,
                                     N, s0, qlo, l[:, :, qlo:qhi].contiguous(), rowterm[:, :, qlo:qhi].contiguous(),
                                     dout[:, :, qlo:qhi], causal=causal, dk=dk.t, dv=dv.t)
        check(dk, dv)
