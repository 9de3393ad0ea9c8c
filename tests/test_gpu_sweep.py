"""A seeded sweep of random small configurations through every path: the
forward (float32 and bf16; causal and bidirectional; per-head and per-query
gates; with and without the logit clamp; k on both sides of the
small-window threshold; pi below, at and above k), the backward (bf16) and
the index set, each against the oracle at its bar.  The cases are drawn
once from a fixed seed, so every run checks the same ones."""
import numpy as np
import pytest
import torch

import oracle
import paper_2511_10696_amd as pa
from paper_2511_10696_amd import workloads as W
from tests.test_gpu_backward import assert_grad
from tests.test_gpu_parity import LSE_TOL, assert_close, np32

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
    out, lse = pa.pi_attn_forward(q, k, v, gate, c["k"], c["pi"], return_lse=True, causal=c["causal"])
    dout = W.cotangent(q.shape, q.dtype, c["seed"], device)
    grads = pa.pi_attn_backward(q, k, v, gate, c["k"], c["pi"], out, lse, dout, gate_grad_per_query=True,
                                causal=c["causal"])
    torch.cuda.synchronize()
    refs = oracle.backward(q, k, v, gate, c["k"], c["pi"], dout, causal=c["causal"])
    for name, got, ref in zip(("dq", "dk", "dv", "dgate"), grads, refs):
        assert_grad(np32(got), ref, f"{name} {ident(c)}", torch.bfloat16)


@pytest.mark.parametrize("c", CASES, ids=ident)
def test_index_set_sweep(device, c):
    idx = pa.pi_attn_index_set(c["N"], c["k"], c["pi"], causal=c["causal"])
    torch.cuda.synchronize()
    ref = oracle.index_set(c["N"], c["k"], c["pi"], causal=c["causal"])
    assert np.array_equal(idx.cpu().numpy(), ref)
