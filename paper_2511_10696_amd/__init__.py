"""MI355X (gfx950) pi-Attention operator: Python binding of libpi_attn.so.

The binding only marshals arguments (device pointers, strides, the current
HIP stream) into the C ABI declared in ``include/pi_attn.h``; every step of
the operator runs in the library's HIP kernels.  There is no fallback: if the
library is missing or the tensors are not on the GPU, the calls raise.

Entry points (same names as the C ABI; ``causal=False`` selects the
bidirectional mode, window |j - t| <= k and partners t -/+ pi):
    pi_attn_index_set(n, k, pi, causal=True)                  -> int32 [n, m] (device)
    pi_attn_forward(q, k, v, gate, k_window, pi, causal=True) -> out [B,H,N,D] (and lse)
    pi_attn_forward_gated(q, k, v, u, w2, b2, k_window, pi)   -> out, gate logits [B,H,N]
    pi_attn_backward(q, k, v, gate, k_window, pi, out, lse, dout, causal=True)
    pi_attn_decode_step(len_in, q_new, k_new, v_new, k_cache, v_cache, gate, k, pi)
"""
from __future__ import annotations

import ctypes
import os
import threading

__all__ = ["pi_attn_index_set", "pi_attn_forward", "pi_attn_forward_gated", "pi_attn_backward",
           "pi_attn_backward_noalloc",
           "pi_attn_decode_step", "pi_attn_ws_width",
           "pi_attn_forward_shard", "pi_attn_backward_shard_q", "pi_attn_backward_shard_kv",
           "pi_attn_strerror", "library", "LIB_PATH", "EXPORTED_SYMBOLS", "PiAttnError"]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libpi_attn.so")
EXPORTED_SYMBOLS = ("pi_attn_strerror", "pi_attn_ws_width", "pi_attn_default_scale", "pi_attn_index_set",
                    "pi_attn_forward", "pi_attn_forward_gated", "pi_attn_decode_step", "pi_attn_backward",
                    "pi_attn_gate_grad_per_head", "pi_attn_forward_shard", "pi_attn_backward_shard_q",
                    "pi_attn_backward_shard_kv", "pi_attn_backward_noalloc")

PI_ATTN_F32, PI_ATTN_BF16 = 0, 1

_lock = threading.Lock()
_lib = None


class PiAttnError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: status {status} ({pi_attn_strerror(status)})")
        self.status = status


def library() -> ctypes.CDLL:
    """Load libpi_attn.so (built by ``paper_2511_10696_amd.build``)."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2511_10696_amd.build`")
            lib = ctypes.CDLL(LIB_PATH)
            i32, i64, f32, vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_void_p
            lib.pi_attn_strerror.argtypes = [ctypes.c_int]
            lib.pi_attn_strerror.restype = ctypes.c_char_p
            lib.pi_attn_ws_width.argtypes = [i32, i32, i32]
            lib.pi_attn_ws_width.restype = i32
            lib.pi_attn_default_scale.argtypes = [i32]
            lib.pi_attn_default_scale.restype = f32
            lib.pi_attn_index_set.argtypes = [i32, i32, i32, i32, vp, vp]
            lib.pi_attn_index_set.restype = ctypes.c_int
            lib.pi_attn_forward.argtypes = ([i32] * 8 + [vp, vp, vp, i64, i64, i64, vp, i64, i64, i64,
                                                        f32, f32, vp, i64, i64, i64, vp, vp])
            lib.pi_attn_forward.restype = ctypes.c_int
            lib.pi_attn_forward_gated.argtypes = ([i32] * 8 + [vp, vp, vp, i64, i64, i64, vp, i64, i64, i32, vp, vp,
                                                              f32, f32, vp, i64, i64, i64, vp, vp, vp])
            lib.pi_attn_forward_gated.restype = ctypes.c_int
            lib.pi_attn_decode_step.argtypes = ([i32] * 7 + [vp, vp, vp, vp, vp, vp, vp, vp, i64, i64,
                                                            f32, f32, vp, vp, vp])
            lib.pi_attn_decode_step.restype = ctypes.c_int
            lib.pi_attn_backward.argtypes = ([i32] * 8 + [vp, vp, vp, i64, i64, i64, vp, i64, i64, i64,
                                                         f32, f32, vp, vp, vp, i64, i64, i64,
                                                         vp, vp, vp, vp, vp, vp])
            lib.pi_attn_backward.restype = ctypes.c_int
            lib.pi_attn_backward_noalloc.argtypes = ([i32] * 8 + [vp, vp, vp, i64, i64, i64, vp, i64, i64, i64,
                                                                 f32, f32, vp, vp, vp, i64, i64, i64,
                                                                 vp, vp, vp, vp, vp])
            lib.pi_attn_backward_noalloc.restype = ctypes.c_int
            lib.pi_attn_gate_grad_per_head.argtypes = [i32, i32, i32, vp, vp, vp]
            lib.pi_attn_gate_grad_per_head.restype = ctypes.c_int
            lib.pi_attn_forward_shard.argtypes = ([i32] * 12 + [vp, i64, i64, i64, vp, vp, i64, i64, i64,
                                                                vp, i64, i64, i64, f32, f32, vp, i64, i64, i64, vp, vp])
            lib.pi_attn_forward_shard.restype = ctypes.c_int
            lib.pi_attn_backward_shard_q.argtypes = ([i32] * 12 + [vp, i64, i64, i64, vp, vp, i64, i64, i64,
                                                                   vp, i64, i64, i64, f32, f32, vp, vp, vp, i64, i64,
                                                                   i64, vp, vp, vp, vp])
            lib.pi_attn_backward_shard_q.restype = ctypes.c_int
            lib.pi_attn_backward_shard_kv.argtypes = ([i32] * 12 + [vp, i64, i64, i64, vp, vp, i64, i64, i64,
                                                                    vp, i64, i64, i64, f32, f32, vp, vp, vp, i64, i64,
                                                                    i64, vp, vp, vp])
            lib.pi_attn_backward_shard_kv.restype = ctypes.c_int
            _lib = lib
    return _lib


def pi_attn_strerror(status: int) -> str:
    return library().pi_attn_strerror(int(status)).decode()


def pi_attn_ws_width(k: int, pi: int, causal: bool = True) -> int:
    return int(library().pi_attn_ws_width(int(k), int(pi), int(bool(causal))))


def _torch():
    import torch
    return torch


def _stream_handle(stream, device):
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return ctypes.c_void_p(stream.cuda_stream)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dtype_code(dt):
    torch = _torch()
    if dt == torch.float32:
        return PI_ATTN_F32
    if dt == torch.bfloat16:
        return PI_ATTN_BF16
    raise TypeError(f"unsupported dtype {dt} (float32 or bfloat16)")


def _require_cuda(*ts):
    for t in ts:
        if t is not None and not t.is_cuda:
            raise RuntimeError("pi_attn tensors must be on the GPU (no CPU path exists)")


def _out_f32(torch, given, shape, device, name):
    """A caller's float32 output buffer (checked: contiguous, the shape), or a new one."""
    if given is None:
        return torch.empty(shape, dtype=torch.float32, device=device)
    _require_cuda(given)
    if given.dtype != torch.float32 or tuple(given.shape) != tuple(shape) or not given.is_contiguous():
        raise ValueError(f"{name} must be a contiguous float32 tensor of shape {tuple(shape)}")
    return given


def _scale(scale, D: int) -> float:
    """The given score scale, or the library's default 1/sqrt(D)."""
    return float(library().pi_attn_default_scale(int(D))) if scale is None else float(scale)


def _check(status: int, where: str):
    if status != 0:
        raise PiAttnError(status, where)


def pi_attn_index_set(n: int, k: int, pi: int, out=None, device=None, stream=None, causal: bool = True):
    """W_t for t in [0, n) as a device int32 tensor [n, m] (m = pi_attn_ws_width(k, pi, causal)):
    window columns hold t-k.. (k+1 causal, 2k+1 bidirectional), then t-pi and
    (bidirectional) t+pi when pi > k; -1 outside [0, n)."""
    torch = _torch()
    m = pi_attn_ws_width(k, pi, causal)
    if m < 0:
        raise PiAttnError(-1, "pi_attn_index_set")
    if out is None:
        out = torch.empty((n, m), dtype=torch.int32, device=device or "cuda")
    _require_cuda(out)
    if out.dtype != torch.int32 or tuple(out.shape) != (n, m) or not out.is_contiguous():
        raise ValueError(f"out must be a contiguous int32 tensor of shape {(n, m)}")
    _check(library().pi_attn_index_set(n, k, pi, int(bool(causal)), _ptr(out), _stream_handle(stream, out.device)),
           "pi_attn_index_set")
    return out


def pi_attn_forward(q, k, v, gate, k_window: int, pi: int, scale: float | None = None,
                    logit_clamp: float = 0.0, out=None, return_lse: bool = False, lse=None, stream=None,
                    causal: bool = True):
    """pi-Attention forward (causal, or bidirectional with ``causal=False``).

    q, k, v: [B, H, N, D] float32 or bfloat16 on the GPU, identical strides,
    last dimension contiguous.  gate: float32 pre-sigmoid gate logits, [H]
    (per head) or [B, H, N] (per query), any strides.  Returns out
    [B, H, N, D] in the input dtype (and lse [B, H, N] float32 on request).
    """
    torch = _torch()
    _require_cuda(q, k, v, gate, out, lse)
    if q.dim() != 4 or k.shape != q.shape or v.shape != q.shape:
        raise ValueError("q, k, v must share one [B, H, N, D] shape")
    if k.dtype != q.dtype or v.dtype != q.dtype:
        raise TypeError("q, k, v must share one dtype")
    if k.stride() != q.stride() or v.stride() != q.stride():
        raise ValueError("q, k, v must share strides (use .contiguous())")
    if q.stride(3) != 1:
        raise ValueError("the head dimension must be contiguous")
    B, H, N, D = q.shape
    if gate.dtype != torch.float32:
        raise TypeError("gate logits must be float32")
    if tuple(gate.shape) == (H,):
        g = gate.view(1, H, 1).expand(B, H, N)
    elif tuple(gate.shape) == (B, H, N):
        g = gate
    else:
        raise ValueError(f"gate must be [H] or [B, H, N], got {tuple(gate.shape)}")
    if out is None:
        out = torch.empty_like(q, memory_format=torch.contiguous_format)
    if out.shape != q.shape or out.dtype != q.dtype or out.stride(3) != 1:
        raise ValueError("out must match q's shape and dtype with a contiguous last dimension")
    if return_lse and lse is None:
        lse = torch.empty((B, H, N), dtype=torch.float32, device=q.device)
    if lse is not None and (lse.dtype != torch.float32 or tuple(lse.shape) != (B, H, N)
                            or not lse.is_contiguous()):
        raise ValueError("lse must be a contiguous float32 [B, H, N] tensor")
    scale = _scale(scale, D)
    st = library().pi_attn_forward(
        _dtype_code(q.dtype), B, H, N, D, int(k_window), int(pi), int(bool(causal)),
        _ptr(q), _ptr(k), _ptr(v), q.stride(0), q.stride(1), q.stride(2),
        _ptr(g), g.stride(0), g.stride(1), g.stride(2), float(scale), float(logit_clamp),
        _ptr(out), out.stride(0), out.stride(1), out.stride(2), _ptr(lse),
        _stream_handle(stream, q.device))
    _check(st, "pi_attn_forward")
    return (out, lse) if (return_lse or lse is not None) else out


def pi_attn_forward_shard(q, k, v, gate, k_window: int, pi: int, nseq: int, qpos0: int, kvpos0: int,
                          scale: float | None = None, logit_clamp: float = 0.0, out=None, return_lse: bool = False,
                          lse=None, stream=None, causal: bool = True):
    """The forward over one shard of a sequence of ``nseq`` positions: q
    [B, H, nq, D] holds the queries at absolute positions
    [qpos0, qpos0 + nq), k and v [B, H, nkv, D] the rows from absolute
    position ``kvpos0`` on (the shard plus its halo; see
    pi_attn_forward_shard in include/pi_attn.h for the rows required).
    bfloat16 only.  gate: [H] or [B, H, nq].  Returns out [B, H, nq, D]
    (and lse [B, H, nq])."""
    torch = _torch()
    _require_cuda(q, k, v, gate, out, lse)
    if q.dim() != 4 or k.dim() != 4 or k.shape != v.shape or k.stride() != v.stride():
        raise ValueError("q [B, H, nq, D] and k, v [B, H, nkv, D] with k and v sharing strides")
    B, H, nq, D = q.shape
    if k.shape[0] != B or k.shape[1] != H or k.shape[3] != D:
        raise ValueError("k and v must share q's B, H and D")
    nkv = k.shape[2]
    if q.dtype != torch.bfloat16 or k.dtype != q.dtype or v.dtype != q.dtype:
        raise TypeError("q, k, v must be bfloat16")
    if q.stride(3) != 1 or k.stride(3) != 1:
        raise ValueError("the head dimension must be contiguous")
    if gate.dtype != torch.float32:
        raise TypeError("gate logits must be float32")
    if tuple(gate.shape) == (H,):
        g = gate.view(1, H, 1).expand(B, H, nq)
    elif tuple(gate.shape) == (B, H, nq):
        g = gate
    else:
        raise ValueError(f"gate must be [H] or [B, H, nq], got {tuple(gate.shape)}")
    if out is None:
        out = torch.empty_like(q, memory_format=torch.contiguous_format)
    if out.shape != q.shape or out.dtype != q.dtype or out.stride(3) != 1:
        raise ValueError("out must match q's shape and dtype with a contiguous last dimension")
    if return_lse and lse is None:
        lse = torch.empty((B, H, nq), dtype=torch.float32, device=q.device)
    if lse is not None and (lse.dtype != torch.float32 or tuple(lse.shape) != (B, H, nq)
                            or not lse.is_contiguous()):
        raise ValueError("lse must be a contiguous float32 [B, H, nq] tensor")
    scale = _scale(scale, D)
    st = library().pi_attn_forward_shard(
        PI_ATTN_BF16, B, H, D, int(k_window), int(pi), int(bool(causal)), int(nseq), int(qpos0), nq, int(kvpos0),
        nkv, _ptr(q), q.stride(0), q.stride(1), q.stride(2), _ptr(k), _ptr(v), k.stride(0), k.stride(1),
        k.stride(2), _ptr(g), g.stride(0), g.stride(1), g.stride(2), float(scale), float(logit_clamp),
        _ptr(out), out.stride(0), out.stride(1), out.stride(2), _ptr(lse), _stream_handle(stream, q.device))
    _check(st, "pi_attn_forward_shard")
    return (out, lse) if return_lse else out


def _shard_gate(torch, gate, B, H, n):
    if gate.dtype != torch.float32:
        raise TypeError("gate logits must be float32")
    if tuple(gate.shape) == (H,):
        return gate.view(1, H, 1).expand(B, H, n)
    if tuple(gate.shape) == (B, H, n):
        return gate
    raise ValueError(f"gate must be [H] or [B, H, {n}], got {tuple(gate.shape)}")


def pi_attn_backward_shard_q(q, k, v, gate, k_window: int, pi: int, nseq: int, qpos0: int, kvpos0: int, out, lse,
                             dout, scale: float | None = None, logit_clamp: float = 0.0, stream=None,
                             causal: bool = True, dq=None, dgate=None, rowterm=None):
    """Query pass of the backward over one shard: q, out, dout [B, H, nq, D]
    (bfloat16) at absolute positions [qpos0, qpos0 + nq), k and v
    [B, H, nkv, D] from absolute position ``kvpos0`` (the forward shard's
    rows), lse [B, H, nq].  Returns float32 dq [B, H, nq, D], the per-query
    gate gradient and the row terms [B, H, nq]."""
    torch = _torch()
    _require_cuda(q, k, v, gate, out, dout, lse)
    B, H, nq, D = q.shape
    if out.shape != q.shape or dout.shape != q.shape or out.stride() != dout.stride():
        raise ValueError("out and dout must match q's shape and share strides")
    if k.shape != v.shape or k.stride() != v.stride() or k.shape[:2] != q.shape[:2] or k.shape[3] != D:
        raise ValueError("k, v [B, H, nkv, D] with shared strides")
    g = _shard_gate(torch, gate, B, H, nq)
    dq = _out_f32(torch, dq, (B, H, nq, D), q.device, "dq")
    dg = _out_f32(torch, dgate, (B, H, nq), q.device, "dgate")
    rt = _out_f32(torch, rowterm, (B, H, nq), q.device, "rowterm")
    scale = _scale(scale, D)
    st = library().pi_attn_backward_shard_q(
        _dtype_code(q.dtype), B, H, D, int(k_window), int(pi), int(bool(causal)), int(nseq), int(qpos0), nq,
        int(kvpos0), k.shape[2], _ptr(q), q.stride(0), q.stride(1), q.stride(2), _ptr(k), _ptr(v), k.stride(0),
        k.stride(1), k.stride(2), _ptr(g), g.stride(0), g.stride(1), g.stride(2), float(scale), float(logit_clamp),
        _ptr(lse), _ptr(out), _ptr(dout), dout.stride(0), dout.stride(1), dout.stride(2), _ptr(dq), _ptr(dg),
        _ptr(rt), _stream_handle(stream, q.device))
    _check(st, "pi_attn_backward_shard_q")
    return dq, dg, rt


def pi_attn_backward_shard_kv(q, k, v, gate, k_window: int, pi: int, nseq: int, kpos0: int, qpos0: int, lse, rowterm,
                              dout, scale: float | None = None, logit_clamp: float = 0.0, stream=None,
                              causal: bool = True, dk=None, dv=None):
    """Key pass of the backward over one shard: k, v [B, H, nk, D] (bfloat16)
    the keys at absolute positions [kpos0, kpos0 + nk); q, dout
    [B, H, nqh, D], lse, rowterm [B, H, nqh] (contiguous float32) and gate
    the query rows held from absolute position ``qpos0`` (the shard's own and
    the halo rows).  Returns float32 dk, dv [B, H, nk, D]."""
    torch = _torch()
    _require_cuda(q, k, v, gate, dout, lse, rowterm)
    B, H, nk, D = k.shape
    if v.shape != k.shape or v.stride() != k.stride():
        raise ValueError("k and v must share shape and strides")
    if q.dim() != 4 or q.shape[:2] != k.shape[:2] or q.shape[3] != D or dout.shape != q.shape:
        raise ValueError("q, dout [B, H, nqh, D]")
    nqh = q.shape[2]
    for name, x in (("lse", lse), ("rowterm", rowterm)):
        if x.dtype != torch.float32 or tuple(x.shape) != (B, H, nqh) or not x.is_contiguous():
            raise ValueError(f"{name} must be a contiguous float32 [B, H, nqh] tensor")
    g = _shard_gate(torch, gate, B, H, nqh)
    dk = _out_f32(torch, dk, (B, H, nk, D), k.device, "dk")
    dv = _out_f32(torch, dv, (B, H, nk, D), k.device, "dv")
    scale = _scale(scale, D)
    st = library().pi_attn_backward_shard_kv(
        _dtype_code(k.dtype), B, H, D, int(k_window), int(pi), int(bool(causal)), int(nseq), int(kpos0), nk,
        int(qpos0), nqh, _ptr(q), q.stride(0), q.stride(1), q.stride(2), _ptr(k), _ptr(v), k.stride(0),
        k.stride(1), k.stride(2), _ptr(g), g.stride(0), g.stride(1), g.stride(2), float(scale), float(logit_clamp),
        _ptr(lse), _ptr(rowterm), _ptr(dout), dout.stride(0), dout.stride(1), dout.stride(2), _ptr(dk), _ptr(dv),
        _stream_handle(stream, k.device))
    _check(st, "pi_attn_backward_shard_kv")
    return dk, dv


def pi_attn_forward_gated(q, k, v, u, w2, b2, k_window: int, pi: int, scale: float | None = None,
                          logit_clamp: float = 0.0, out=None, return_lse: bool = False, lse=None,
                          gate_out=None, stream=None, causal: bool = True):
    """pi-Attention forward with the gate logits computed from the gate MLP's
    last layer: g[b, h, t] = <u[b, t], w2[h]> + b2[h] (App. A gate module).

    q, k, v as in pi_attn_forward; u [B, N, dh] (the GELU output, q's dtype,
    last dimension contiguous), w2 [H, dh] (q's dtype, contiguous: a Linear
    weight as stored), b2 [H] float32 or None.  Returns (out, gate_logits
    [B, H, N] float32) and lse on request; gate_logits is the ``gate`` that
    pi_attn_backward takes.
    """
    torch = _torch()
    _require_cuda(q, k, v, u, w2, b2, out, lse, gate_out)
    if q.dim() != 4 or k.shape != q.shape or v.shape != q.shape:
        raise ValueError("q, k, v must share one [B, H, N, D] shape")
    if k.dtype != q.dtype or v.dtype != q.dtype or u.dtype != q.dtype or w2.dtype != q.dtype:
        raise TypeError("q, k, v, u and w2 must share one dtype")
    if k.stride() != q.stride() or v.stride() != q.stride():
        raise ValueError("q, k, v must share strides (use .contiguous())")
    if q.stride(3) != 1:
        raise ValueError("the head dimension must be contiguous")
    B, H, N, D = q.shape
    if u.dim() != 3 or u.shape[0] != B or u.shape[1] != N or u.stride(2) != 1:
        raise ValueError("u must be [B, N, dh] with a contiguous last dimension")
    dh = u.shape[2]
    if tuple(w2.shape) != (H, dh) or not w2.is_contiguous():
        raise ValueError(f"w2 must be a contiguous [H, dh] = {(H, dh)} tensor")
    if b2 is not None and (b2.dtype != torch.float32 or tuple(b2.shape) != (H,) or not b2.is_contiguous()):
        raise ValueError("b2 must be a contiguous float32 [H] tensor or None")
    if out is None:
        out = torch.empty_like(q, memory_format=torch.contiguous_format)
    if out.shape != q.shape or out.dtype != q.dtype or out.stride(3) != 1:
        raise ValueError("out must match q's shape and dtype with a contiguous last dimension")
    if gate_out is None:
        gate_out = torch.empty((B, H, N), dtype=torch.float32, device=q.device)
    if gate_out.dtype != torch.float32 or tuple(gate_out.shape) != (B, H, N) or not gate_out.is_contiguous():
        raise ValueError("gate_out must be a contiguous float32 [B, H, N] tensor")
    if return_lse and lse is None:
        lse = torch.empty((B, H, N), dtype=torch.float32, device=q.device)
    if lse is not None and (lse.dtype != torch.float32 or tuple(lse.shape) != (B, H, N)
                            or not lse.is_contiguous()):
        raise ValueError("lse must be a contiguous float32 [B, H, N] tensor")
    scale = _scale(scale, D)
    st = library().pi_attn_forward_gated(
        _dtype_code(q.dtype), B, H, N, D, int(k_window), int(pi), int(bool(causal)),
        _ptr(q), _ptr(k), _ptr(v), q.stride(0), q.stride(1), q.stride(2),
        _ptr(u), u.stride(0), u.stride(1), dh, _ptr(w2), _ptr(b2), float(scale), float(logit_clamp),
        _ptr(out), out.stride(0), out.stride(1), out.stride(2), _ptr(lse), _ptr(gate_out),
        _stream_handle(stream, q.device))
    _check(st, "pi_attn_forward_gated")
    return (out, gate_out, lse) if (return_lse or lse is not None) else (out, gate_out)


def pi_attn_backward(q, k, v, gate, k_window: int, pi: int, out, lse, dout, scale: float | None = None,
                     logit_clamp: float = 0.0, gate_grad_per_query: bool = False, stream=None,
                     causal: bool = True, dq=None, dk=None, dv=None, dgate=None, rowterm=None):
    """Gradients of the pi-Attention forward for dL/dy = ``dout``.

    q, k, v, gate, k_window, pi, scale, logit_clamp and causal as passed to
    pi_attn_forward; ``out`` and ``lse`` are what that forward call returned
    ([B, H, N, D] in q's dtype, [B, H, N] float32); ``dout`` has out's shape,
    dtype and strides.  Returns float32
    (dq, dk, dv) [B, H, N, D] and dgate shaped like ``gate`` (summed over
    b and t for a per-head gate), or [B, H, N] per query when
    ``gate_grad_per_query``.  dq, dk, dv, dgate (per query) and the row-term
    workspace rowterm may be passed as contiguous float32 buffers to fill.
    """
    torch = _torch()
    _require_cuda(q, k, v, gate, out, dout, lse)
    if (q.dim() != 4 or k.shape != q.shape or v.shape != q.shape or dout.shape != q.shape
            or out.shape != q.shape):
        raise ValueError("q, k, v, out, dout must share one [B, H, N, D] shape")
    if k.dtype != q.dtype or v.dtype != q.dtype or dout.dtype != q.dtype or out.dtype != q.dtype:
        raise TypeError("q, k, v, out, dout must share one dtype")
    if out.stride() != dout.stride():
        dout = dout.contiguous()
        out = out.contiguous()
    if k.stride() != q.stride() or v.stride() != q.stride():
        raise ValueError("q, k, v must share strides (use .contiguous())")
    if q.stride(3) != 1 or dout.stride(3) != 1:
        raise ValueError("the head dimension must be contiguous")
    B, H, N, D = q.shape
    if gate.dtype != torch.float32:
        raise TypeError("gate logits must be float32")
    if tuple(gate.shape) == (H,):
        g = gate.view(1, H, 1).expand(B, H, N)
    elif tuple(gate.shape) == (B, H, N):
        g = gate
    else:
        raise ValueError(f"gate must be [H] or [B, H, N], got {tuple(gate.shape)}")
    if lse.dtype != torch.float32 or tuple(lse.shape) != (B, H, N) or not lse.is_contiguous():
        raise ValueError("lse must be the contiguous float32 [B, H, N] lse of the forward")
    f32 = dict(dtype=torch.float32, device=q.device)
    dq, dk, dv = (_out_f32(torch, x, (B, H, N, D), q.device, n) for x, n in ((dq, "dq"), (dk, "dk"), (dv, "dv")))
    dg = _out_f32(torch, dgate, (B, H, N), q.device, "dgate")
    rowterm = _out_f32(torch, rowterm, (B, H, N), q.device, "rowterm")
    scale = _scale(scale, D)
    st = library().pi_attn_backward(
        _dtype_code(q.dtype), B, H, N, D, int(k_window), int(pi), int(bool(causal)),
        _ptr(q), _ptr(k), _ptr(v), q.stride(0), q.stride(1), q.stride(2),
        _ptr(g), g.stride(0), g.stride(1), g.stride(2), float(scale), float(logit_clamp), _ptr(lse),
        _ptr(out), _ptr(dout), dout.stride(0), dout.stride(1), dout.stride(2),
        _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dg), _ptr(rowterm), _stream_handle(stream, q.device))
    _check(st, "pi_attn_backward")
    if tuple(gate.shape) == (H,) and not gate_grad_per_query:
        dgh = torch.empty((H,), **f32)
        _check(library().pi_attn_gate_grad_per_head(B, H, N, _ptr(dg), _ptr(dgh), _stream_handle(stream, q.device)),
               "pi_attn_gate_grad_per_head")
        dg = dgh
    return dq, dk, dv, dg


def pi_attn_backward_noalloc(q, k, v, gate, k_window: int, pi: int, out, lse, dout, dq, dk, dv, dgate,
                             scale: float | None = None, logit_clamp: float = 0.0, stream=None,
                             causal: bool = True):
    """pi_attn_backward into caller-owned outputs with no workspace: the row
    terms live in the library's fixed per-device array (B*H*N <= 4194304;
    calls that overlap in time on one device race on it).  dq, dk, dv
    [B, H, N, D] and dgate [B, H, N] (per query) are contiguous float32
    tensors that the call overwrites; out and dout must share strides.
    Nothing is allocated here or in the library."""
    torch = _torch()
    _require_cuda(q, k, v, gate, out, dout, lse, dq, dk, dv, dgate)
    if (q.dim() != 4 or k.shape != q.shape or v.shape != q.shape or dout.shape != q.shape
            or out.shape != q.shape):
        raise ValueError("q, k, v, out, dout must share one [B, H, N, D] shape")
    if k.dtype != q.dtype or v.dtype != q.dtype or dout.dtype != q.dtype or out.dtype != q.dtype:
        raise TypeError("q, k, v, out, dout must share one dtype")
    if out.stride() != dout.stride() or k.stride() != q.stride() or v.stride() != q.stride():
        raise ValueError("q, k, v must share strides, and out and dout must share strides")
    if q.stride(3) != 1 or dout.stride(3) != 1:
        raise ValueError("the head dimension must be contiguous")
    B, H, N, D = q.shape
    if gate.dtype != torch.float32:
        raise TypeError("gate logits must be float32")
    if tuple(gate.shape) == (H,):
        gs = (0, gate.stride(0), 0)
    elif tuple(gate.shape) == (B, H, N):
        gs = gate.stride()
    else:
        raise ValueError(f"gate must be [H] or [B, H, N], got {tuple(gate.shape)}")
    if lse.dtype != torch.float32 or tuple(lse.shape) != (B, H, N) or not lse.is_contiguous():
        raise ValueError("lse must be the contiguous float32 [B, H, N] lse of the forward")
    for name, t, shape in (("dq", dq, (B, H, N, D)), ("dk", dk, (B, H, N, D)), ("dv", dv, (B, H, N, D)),
                           ("dgate", dgate, (B, H, N))):
        if t.dtype != torch.float32 or tuple(t.shape) != shape or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous float32 {list(shape)} tensor")
    scale = _scale(scale, D)
    st = library().pi_attn_backward_noalloc(
        _dtype_code(q.dtype), B, H, N, D, int(k_window), int(pi), int(bool(causal)),
        _ptr(q), _ptr(k), _ptr(v), q.stride(0), q.stride(1), q.stride(2),
        _ptr(gate), gs[0], gs[1], gs[2], float(scale), float(logit_clamp), _ptr(lse),
        _ptr(out), _ptr(dout), dout.stride(0), dout.stride(1), dout.stride(2),
        _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dgate), _stream_handle(stream, q.device))
    _check(st, "pi_attn_backward_noalloc")
    return dq, dk, dv, dgate


def pi_attn_decode_step(len_in, q_new, k_new, v_new, k_cache, v_cache, gate, k: int, pi: int,
                        scale: float | None = None, logit_clamp: float = 0.0, len_out=None,
                        out=None, lse=None, stream=None):
    """One decode step: appends k_new/v_new [S, H, D] as row len_in[s] of the
    caches [S, H, cap, D] and attends q_new over W_t.  Returns out [S, H, D]."""
    torch = _torch()
    _require_cuda(len_in, q_new, k_new, v_new, k_cache, v_cache, gate, len_out, out, lse)
    S, H, cap, D = k_cache.shape
    for name, t in (("q_new", q_new), ("k_new", k_new), ("v_new", v_new)):
        if tuple(t.shape) != (S, H, D) or not t.is_contiguous() or t.dtype != k_cache.dtype:
            raise ValueError(f"{name} must be a contiguous [S, H, D] tensor of the cache dtype")
    if v_cache.shape != k_cache.shape or v_cache.dtype != k_cache.dtype:
        raise ValueError("k_cache and v_cache must match")
    if not (k_cache.is_contiguous() and v_cache.is_contiguous()):
        raise ValueError("caches must be contiguous")
    if len_in.dtype != torch.int32 or tuple(len_in.shape) != (S,) or not len_in.is_contiguous():
        raise ValueError("len_in must be a contiguous int32 [S] tensor")
    if gate.dtype != torch.float32:
        raise TypeError("gate logits must be float32")
    if tuple(gate.shape) == (H,):
        gss, gsh = 0, gate.stride(0)
    elif tuple(gate.shape) == (S, H):
        gss, gsh = gate.stride(0), gate.stride(1)
    else:
        raise ValueError("decode gate must be [H] or [S, H]")
    if out is None:
        out = torch.empty_like(q_new)
    if tuple(out.shape) != (S, H, D) or out.dtype != k_cache.dtype or not out.is_contiguous():
        raise ValueError("out must be a contiguous [S, H, D] tensor of the cache dtype")
    if lse is not None and (lse.dtype != torch.float32 or tuple(lse.shape) != (S, H) or not lse.is_contiguous()):
        raise ValueError("lse must be a contiguous float32 [S, H] tensor")
    if len_out is not None and (len_out.dtype != torch.int32 or tuple(len_out.shape) != (S,)
                                or not len_out.is_contiguous()):
        raise ValueError("len_out must be a contiguous int32 [S] tensor")
    scale = _scale(scale, D)
    st = library().pi_attn_decode_step(
        _dtype_code(k_cache.dtype), S, H, D, cap, int(k), int(pi), _ptr(len_in), _ptr(len_out),
        _ptr(q_new), _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache), _ptr(gate), gss, gsh,
        float(scale), float(logit_clamp), _ptr(out), _ptr(lse), _stream_handle(stream, q_new.device))
    _check(st, "pi_attn_decode_step")
    return out
