"""A seeded sweep of random small configurations through every path: the
forward (float32 and bf16; causal and bidirectional; per-head and per-query
gates; with and without the logit clamp; k on both sides of the
small-window threshold; pi below, at and above k), the backward (bf16) and
the index set, each against the oracle at its bar; random sequence shards
(boundaries on or off the 128-query tile grid) through the shard calls; and
random decode steps (per-sequence lengths from 0 to cap - 1), and longer
banded backward problems with partners outside the window.  The cases
are drawn once from fixed seeds, so every run checks the same ones."""
import numpy as np
import pytest
import torch

import oracle
import paper_2511_10696_amd as pa
from paper_2511_10696_amd import workloads as W
from tests.grad_check import assert_grad, check_backward, expected_grads, forward_state
from tests.test_gpu_parity import LSE_TOL, assert_close, np32
from tests.test_gpu_shard import run_shards, sharded_backward

pytestmark = pytest.mark.gpu


def draw_cases(n, seed):
    rng = np.random.default_rng(seed)
    cases = []
    for _ in range(n):
        N = int(rng.integers(1, 420))
        k = int(rng.choice([0, 1, 3, 4, 8, 15, 16, 17, 31, 64, 150, 500]))
        pi = int(rng.choice([0, 1, k, k + 1, 2 * k + 3, 97, 300]))
        cases.append(dict(B=int(rng.integers(1, 3)), H=int(rng.integers(1, 4)), N=N, D=int(rng.choice([64, 128])),
                          k=k, pi=pi, causal=bool(rng.integers(0, 2)), pq=bool(rng.integers(0, 2)),
                          clamp=float(rng.choice([0.0, 0.0, 2.5])), seed=int(rng.integers(0, 1 << 30))))
    return cases


CASES = draw_cases(40, 20261202)


def ident(c):
    return "B{B}H{H}N{N}D{D}k{k}pi{pi}{m}{g}{cl}".format(
        m="c" if c["causal"] else "b", g="q" if c["pq"] else "h", cl=f"L{c['clamp']}" if c["clamp"] else "", **c)


@pytest.mark.parametrize("c", CASES, ids=ident)
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_forward_sweep(device, c, dtype):
    cfg = W.ForwardConfig("custom", c["B"], c["H"], c["N"], c["D"], c["k"], c["pi"], dtype)
    q, k, v, gate = W.forward_inputs(cfg, c["seed"], device, per_query_gate=c["pq"])
    out, lse = pa.pi_attn_forward(q, k, v, gate, c["k"], c["pi"], logit_clamp=c["clamp"], return_lse=True,
                                  causal=c["causal"])
    torch.cuda.synchronize()
    ref, lref = oracle.forward(q, k, v, gate, c["k"], c["pi"], clamp=c["clamp"], want_lse=True, causal=c["causal"])
    assert_close(np32(out), ref, dtype, ident(c))
    assert np.abs(np32(lse) - lref).max() <= LSE_TOL * (10 if c["clamp"] else 1)


@pytest.mark.parametrize("c", CASES[:24], ids=ident)
def test_backward_sweep(device, c):
    if c["clamp"]:
        pytest.skip("the clamp's gradient cut is a discontinuity; clamp cases are placed by hand elsewhere")
    cfg = W.ForwardConfig("custom", c["B"], c["H"], c["N"], c["D"], c["k"], c["pi"], torch.bfloat16)
    q, k, v, gate = W.forward_inputs(cfg, c["seed"], device, per_query_gate=c["pq"])
    check_backward(q, k, v, gate, c["k"], c["pi"], c["seed"], causal=c["causal"], per_head_sum=False)


def draw_partner_cases(n, seed):
    """Banded (k > 16) problems whose partners lie outside the window (pi > k),
    with sequences long enough that whole partner runs of 128 queries occur."""
    rng = np.random.default_rng(seed)
    cases = []
    for _ in range(n):
        k = int(rng.choice([17, 24, 31, 40, 64, 100, 150, 300]))
        pi = max(k + 1, int(rng.choice([k + 1, k + 5, 2 * k + 3, 97, 300, 700])))
        cases.append(dict(B=int(rng.integers(1, 3)), H=int(rng.integers(1, 3)), N=int(rng.integers(40, 1600)),
                          D=int(rng.choice([64, 128])), k=k, pi=pi, causal=bool(rng.integers(0, 2)),
                          pq=bool(rng.integers(0, 2)), clamp=0.0, seed=int(rng.integers(0, 1 << 30))))
    return cases


PARTNER_CASES = draw_partner_cases(12, 20261203)


@pytest.mark.parametrize("c", PARTNER_CASES, ids=ident)
def test_backward_partner_sweep(device, c):
    cfg = W.ForwardConfig("custom", c["B"], c["H"], c["N"], c["D"], c["k"], c["pi"], torch.bfloat16)
    q, k, v, gate = W.forward_inputs(cfg, c["seed"], device, per_query_gate=c["pq"])
    check_backward(q, k, v, gate, c["k"], c["pi"], c["seed"], causal=c["causal"], per_head_sum=False)


@pytest.mark.parametrize("c", CASES, ids=ident)
def test_index_set_sweep(device, c):
    idx = pa.pi_attn_index_set(c["N"], c["k"], c["pi"], causal=c["causal"])
    torch.cuda.synchronize()
    ref = oracle.index_set(c["N"], c["k"], c["pi"], causal=c["causal"])
    assert np.array_equal(idx.cpu().numpy(), ref)


# ---------------------------------------------------------------------------
# sequence shards: forward and both backward passes over random boundaries
# ---------------------------------------------------------------------------
def draw_shard_cases(n, seed):
    rng = np.random.default_rng(seed)
    cases = []
    for _ in range(n):
        aligned = bool(rng.integers(0, 2))
        N = int(rng.integers(2, 12)) * 128 if aligned else int(rng.integers(50, 1600))
        kw = int(rng.choice([17, 31, 40, 64, 100, 128, 200, 300]))
        pi = int(rng.choice([1, kw, kw + 1, 2 * kw, 2 * kw + 5, 333]))
        ns = int(rng.integers(2, 6))
        if aligned:
            cuts = sorted(set(int(x) * 128 for x in rng.integers(1, N // 128, size=ns - 1)))
        else:
            cuts = sorted(set(int(x) for x in rng.integers(1, N, size=ns - 1)))
        edges = [0] + cuts + [N]
        cases.append(dict(N=N, D=int(rng.choice([64, 128])), k=kw, pi=pi, causal=bool(rng.integers(0, 2)),
                          pq=bool(rng.integers(0, 2)), aligned=aligned,
                          bounds=[(a, b) for a, b in zip(edges, edges[1:]) if b > a],
                          seed=int(rng.integers(0, 1 << 30))))
    return cases


SHARD_CASES = draw_shard_cases(48, 31337)


def shard_ident(c):
    return "N{N}D{D}k{k}pi{pi}{m}{g}-".format(m="c" if c["causal"] else "b", g="q" if c["pq"] else "h", **c) + \
        "_".join(str(b) for _, b in c["bounds"][:-1])


@pytest.mark.parametrize("c", SHARD_CASES, ids=shard_ident)
def test_shard_sweep(device, c):
    """Shards on the tile grid reproduce the whole-sequence forward, lse and
    gradients bit for bit; other boundaries meet the bars against the
    oracle."""
    kw, pi, causal, pq = c["k"], c["pi"], c["causal"], c["pq"]
    cfg = W.ForwardConfig("custom", 1, 2, c["N"], c["D"], kw, pi, torch.bfloat16)
    q, k, v, gate = W.forward_inputs(cfg, c["seed"], device, per_query_gate=pq)
    full, lfull = pa.pi_attn_forward(q, k, v, gate, kw, pi, return_lse=True, causal=causal)
    out, lse = run_shards(q, k, v, gate, kw, pi, c["bounds"], causal, pq)
    dout = W.cotangent(q.shape, q.dtype, c["seed"], device)
    if c["aligned"]:
        got = sharded_backward(q, k, v, gate, kw, pi, full, lfull, dout, c["bounds"], causal, pq)
        whole = pa.pi_attn_backward(q, k, v, gate, kw, pi, full, lfull, dout, gate_grad_per_query=True,
                                    causal=causal)
        torch.cuda.synchronize()
        assert torch.equal(out, full) and torch.equal(lse, lfull)
        for name, a, b in zip(("dq", "dk", "dv", "dgate"), got, whole):
            assert torch.equal(a, b), name
        return
    torch.cuda.synchronize()
    ref, lref = oracle.forward(q, k, v, gate, kw, pi, want_lse=True, causal=causal)
    assert_close(np32(out), ref, torch.bfloat16, shard_ident(c))
    assert np.abs(np32(lse) - lref).max() <= LSE_TOL
    # the gradients on the oracle's forward state
    ostate, lstate, y = forward_state(q, k, v, gate, kw, pi, causal=causal)
    got = sharded_backward(q, k, v, gate, kw, pi, ostate, lstate, dout, c["bounds"], causal, pq)
    torch.cuda.synchronize()
    exp = expected_grads(q, k, v, gate, kw, pi, dout, ostate, y, causal=causal, row_term_from_out=True)
    for name, a, e in zip(("dq", "dk", "dv", "dgate"), got, exp):
        assert_grad(np32(a), e, f"{name} {shard_ident(c)}", torch.bfloat16)


# ---------------------------------------------------------------------------
# decode steps
# ---------------------------------------------------------------------------
def draw_decode_cases(n, seed):
    rng = np.random.default_rng(seed)
    cases = []
    for _ in range(n):
        S, cap = int(rng.integers(1, 9)), int(rng.integers(1, 3000))
        kw = int(rng.choice([0, 1, 5, 16, 17, 37, 100, 512, 1500]))
        lens = rng.integers(0, cap, size=S)
        lens[0] = min(int(lens[0]), int(rng.choice([0, cap - 1])))
        cases.append(dict(S=S, H=int(rng.integers(1, 5)), D=int(rng.choice([64, 128])), cap=cap, k=kw,
                          pi=int(rng.choice([0, 1, kw, kw + 1, 2 * kw, 777, 2000])),
                          clamp=float(rng.choice([0.0, 0.0, 2.5])), bf16=bool(rng.integers(0, 3)),
                          lens=[int(x) for x in lens], seed=int(rng.integers(0, 1 << 30))))
    return cases


DECODE_CASES = draw_decode_cases(100, 2718)


def decode_ident(c):
    return "S{S}H{H}D{D}cap{cap}k{k}pi{pi}{cl}{dt}".format(
        cl=f"L{c['clamp']}" if c["clamp"] else "", dt="bf16" if c["bf16"] else "f32", **c)


@pytest.mark.parametrize("c", DECODE_CASES, ids=decode_ident)
def test_decode_sweep(device, c):
    S, H, D, cap = c["S"], c["H"], c["D"], c["cap"]
    dtype = torch.bfloat16 if c["bf16"] else torch.float32
    g = torch.Generator(device="cuda").manual_seed(c["seed"])
    kc = torch.randn(S, H, cap, D, generator=g, device="cuda").to(dtype)
    vc = torch.randn(S, H, cap, D, generator=g, device="cuda").to(dtype)
    gate = torch.rand(S, H, generator=g, device="cuda") * 2 - 1
    lens_np = np.array(c["lens"], np.int32)
    lens = torch.tensor(lens_np, device="cuda")
    qn, kn, vn = (torch.randn(S, H, D, generator=g, device="cuda").to(dtype) for _ in range(3))
    kc_ref, vc_ref = np32(kc), np32(vc)
    lse = torch.empty(S, H, dtype=torch.float32, device="cuda")
    out = pa.pi_attn_decode_step(lens, qn, kn, vn, kc, vc, gate, c["k"], c["pi"], logit_clamp=c["clamp"], lse=lse)
    torch.cuda.synchronize()
    ref, lref = oracle.decode_step(lens_np, qn, kn, vn, kc_ref, vc_ref, gate, c["k"], c["pi"], clamp=c["clamp"],
                                   want_lse=True)
    assert_close(np32(out), ref, dtype, decode_ident(c))
    assert np.abs(np32(lse) - lref).max() <= LSE_TOL * (10 if c["clamp"] else 1)
    for s in range(S):
        assert torch.equal(kc[s, :, lens_np[s]], kn[s]) and torch.equal(vc[s, :, lens_np[s]], vn[s])
