"""The no-allocation backward, pi_attn_backward_noalloc, through the C ABI,
against pi_attn_backward on the same inputs.  Both run the same kernels and
differ only in where the row terms live (the library's fixed per-device
array against a caller workspace), so the gradients must be bit-identical.
Each case makes two no-allocation calls in a row, the second on a smaller
problem, so that the array still holds the first call's row terms when the
second one runs; one case fills the array exactly (B*H*N = 4194304)."""
import pytest
import torch

import paper_2511_10696_amd as pa
from paper_2511_10696_amd import workloads as W

pytestmark = pytest.mark.gpu

MAX_ROWS = 1 << 22


def problem(B, H, N, D, kw, pi, dtype, seed, causal, pq):
    cfg = W.ForwardConfig("custom", B, H, N, D, kw, pi, dtype)
    q, k, v, gate = W.forward_inputs(cfg, seed, "cuda", per_query_gate=pq)
    out, lse = pa.pi_attn_forward(q, k, v, gate, kw, pi, return_lse=True, causal=causal)
    dout = W.cotangent(q.shape, q.dtype, seed, "cuda")
    return q, k, v, gate, kw, pi, out, lse, dout, causal


def noalloc(q, k, v, gate, kw, pi, out, lse, dout, causal):
    B, H, N, D = q.shape
    f32 = dict(dtype=torch.float32, device=q.device)
    dq, dk, dv = (torch.full((B, H, N, D), float("nan"), **f32) for _ in range(3))
    dg = torch.full((B, H, N), float("nan"), **f32)
    return pa.pi_attn_backward_noalloc(q, k, v, gate, kw, pi, out, lse, dout, dq, dk, dv, dg, causal=causal)


def with_workspace(q, k, v, gate, kw, pi, out, lse, dout, causal):
    return pa.pi_attn_backward(q, k, v, gate, kw, pi, out, lse, dout, gate_grad_per_query=True, causal=causal)


CASES = {
    # name: (first problem, second, smaller problem)
    "bf16-banded-causal": ((1, 4, 3000, 128, 512, 1024, torch.bfloat16, 1, True, False),
                           (1, 2, 700, 64, 40, 100, torch.bfloat16, 2, True, True)),
    "bf16-banded-bidirectional": ((2, 3, 1500, 64, 100, 300, torch.bfloat16, 3, False, True),
                                  (1, 1, 200, 128, 20, 50, torch.bfloat16, 4, False, False)),
    "bf16-small-window": ((2, 4, 2000, 64, 4, 16, torch.bfloat16, 5, True, True),
                          (1, 2, 100, 128, 4, 16, torch.bfloat16, 6, False, False)),
    "float32": ((1, 2, 500, 64, 32, 64, torch.float32, 7, True, False),
                (1, 1, 100, 128, 8, 20, torch.float32, 8, False, True)),
    "array-full": ((1, 64, MAX_ROWS // 64, 64, 20, 50, torch.bfloat16, 9, True, False),
                   (1, 3, 333, 64, 20, 50, torch.bfloat16, 10, True, False)),
}


@pytest.mark.parametrize("name", list(CASES))
def test_noalloc_matches_workspace_backward(device, name):
    for spec in CASES[name]:
        args = problem(*spec)
        got = noalloc(*args)
        ref = with_workspace(*args)
        torch.cuda.synchronize()
        for what, a, b in zip(("dq", "dk", "dv", "dgate"), got, ref):
            assert torch.equal(a, b), f"{name} {spec[:6]}: {what}"
        del args, got, ref


def test_noalloc_rejects_oversize_before_launching(device):
    """B*H*N one past the array: ESCRATCH, and the outputs stay untouched."""
    import ctypes
    B, H, N, D = 1, 1, MAX_ROWS + 1, 64
    lib = pa.library()
    dq = torch.full((4,), 7.0, device="cuda")
    vp = ctypes.c_void_p(dq.data_ptr())
    st = lib.pi_attn_backward_noalloc(1, B, H, N, D, 20, 50, 1, vp, vp, vp, N * D, N * D, D, vp, 0, 1, 0,
                                      0.125, 0.0, vp, vp, vp, N * D, N * D, D, vp, vp, vp, vp, None)
    torch.cuda.synchronize()
    assert st == -4 and "4194304" in pa.pi_attn_strerror(st)
    assert torch.equal(dq, torch.full((4,), 7.0, device="cuda"))
