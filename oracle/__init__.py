"""fp64 CPU oracle for pi-Attention (causal and bidirectional) -- TEST
INFRASTRUCTURE ONLY.

Nothing in the product path (the HIP library and its Python binding) may
import, link or call this package.  Its users are the tests, the smoke check
and the CPU-baseline leg of the benchmark.  It shares no code with the HIP
path: the C source ``pi_oracle.c`` is compiled here with gcc into
``liboracle.so`` and called through ctypes.

What it computes is stated, with the paper passages it follows, in the
header of ``pi_oracle.c``; ``reach.py`` holds the reachability and
minimum-depth analysis (Sec. 3.4).
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "pi_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None

EPS = 1e-4  # gate clip of Variant 3 (Sec. 3.5)


def build(src: str = _SRC, out: str = _LIB_PATH) -> str:
    """Compile the oracle with gcc (plain -O2, no fast-math)."""
    tmp = f"{out}.{os.getpid()}.tmp"   # per process: concurrent builds must not collide
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
           "-Wall", "-o", tmp, src, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def _declare(lib: ctypes.CDLL) -> ctypes.CDLL:
    i64, dbl, vp = ctypes.c_int64, ctypes.c_double, ctypes.c_void_p
    lib.oracle_ws_width.argtypes = [ctypes.c_int] * 3
    lib.oracle_ws_width.restype = ctypes.c_int
    lib.oracle_index_set.argtypes = [ctypes.c_int] * 4 + [vp]
    lib.oracle_index_set.restype = None
    lib.oracle_forward_rows.argtypes = (
        [ctypes.c_int] * 7 + [vp, vp, vp, vp, i64, i64, i64, dbl, dbl, vp, i64, vp, vp, vp])
    lib.oracle_forward_rows.restype = None
    lib.oracle_backward.argtypes = (
        [ctypes.c_int] * 7 + [vp, vp, vp, vp, i64, i64, i64, dbl, dbl, vp, vp, vp, vp, vp])
    lib.oracle_backward.restype = None
    lib.oracle_decode_step.argtypes = (
        [ctypes.c_int] * 6 + [vp, vp, vp, vp, vp, vp, vp, i64, i64, dbl, dbl, vp, vp])
    lib.oracle_decode_step.restype = ctypes.c_int
    return lib


def load_library(path: str) -> ctypes.CDLL:
    """Load an oracle build from ``path`` (tests load planted-mistake builds)."""
    return _declare(ctypes.CDLL(path))


def lib() -> ctypes.CDLL:
    """The oracle library; built on first use if no current build exists."""
    global _lib
    with _lock:
        if _lib is None:
            if (not os.path.exists(_LIB_PATH)
                    or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC)):
                build()
            _lib = load_library(_LIB_PATH)
    return _lib


def _ptr(a: np.ndarray | None):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _f32(a) -> np.ndarray:
    """Exact widening to a contiguous float32 numpy array (bf16 -> f32 is exact)."""
    if hasattr(a, "detach"):  # torch tensor
        a = a.detach()
        if a.dtype != __import__("torch").float32:
            a = a.float()
        a = a.cpu().numpy()
    a = np.ascontiguousarray(a)
    if a.dtype != np.float32:
        if a.dtype == np.float64 and not np.array_equal(a.astype(np.float32).astype(np.float64), a):
            raise ValueError("oracle inputs must be exactly representable in float32")
        a = a.astype(np.float32)
    return a


def _f64(a) -> np.ndarray:
    """Contiguous float64 numpy array (gate logits)."""
    if hasattr(a, "detach"):
        a = a.detach().cpu().double().numpy()
    return np.ascontiguousarray(a, dtype=np.float64)


def _gate_strides(gate: np.ndarray, B: int, H: int, N: int):
    """Element strides (gsb, gsh, gsn) for a per-head [H] or per-query [B,H,N] gate."""
    if gate.shape == (H,):
        return 0, 1, 0
    if gate.shape == (B, H, N):
        return H * N, N, 1
    raise ValueError(f"gate must be [H] or [B,H,N], got {gate.shape}")


def ws_width(k: int, pi: int, L=None, causal: bool = True) -> int:
    L = L or lib()
    return int(L.oracle_ws_width(k, pi, int(bool(causal))))


def index_set(n: int, k: int, pi: int, L=None, causal: bool = True) -> np.ndarray:
    """W_t for t in [0, n) as an [n, m] int32 array in slot order (see pi_oracle.c)."""
    L = L or lib()
    m = ws_width(k, pi, L, causal)
    idx = np.empty((n, m), dtype=np.int32)
    L.oracle_index_set(n, k, pi, int(bool(causal)), _ptr(idx))
    return idx


def forward(q, k_, v, gate, k: int, pi: int, scale: float | None = None,
            clamp: float = 0.0, rows=None, want_lse=False, want_probs=False, L=None,
            causal: bool = True):
    """Oracle forward over q, k, v [B,H,N,D] with gate logits [H] or [B,H,N]
    (``causal=False``: bidirectional window and both partners t -/+ pi).

    Returns out [B,H,N,D] float64 (or [len(rows), D] when ``rows`` lists flat
    query rows (b*H+h)*N+t), plus lse and per-slot probabilities on request.
    """
    L = L or lib()
    q, k_, v, gate = _f32(q), _f32(k_), _f32(v), _f64(gate)
    B, H, N, D = q.shape
    assert k_.shape == q.shape and v.shape == q.shape
    gsb, gsh, gsn = _gate_strides(gate, B, H, N)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    m = ws_width(k, pi, L, causal)
    if rows is None:
        nr, rows_arr = B * H * N, None
        out_shape = (B, H, N, D)
    else:
        rows_arr = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
        if rows_arr.size and (rows_arr.min() < 0 or rows_arr.max() >= B * H * N):
            raise ValueError("row index out of range")
        nr = rows_arr.size
        out_shape = (nr, D)
    out = np.empty((nr, D), dtype=np.float64)
    lse = np.empty(nr, dtype=np.float64) if want_lse else None
    probs = np.empty((nr, m), dtype=np.float64) if want_probs else None
    if nr:
        L.oracle_forward_rows(B, H, N, D, k, pi, int(bool(causal)), _ptr(q), _ptr(k_), _ptr(v), _ptr(gate),
                              gsb, gsh, gsn, float(scale), float(clamp),
                              _ptr(rows_arr), nr, _ptr(out), _ptr(lse), _ptr(probs))
    res = [out.reshape(out_shape)]
    if want_lse:
        res.append(lse.reshape(out_shape[:-1]))
    if want_probs:
        res.append(probs.reshape(out_shape[:-1] + (m,)))
    return res[0] if len(res) == 1 else tuple(res)


def backward(q, k_, v, gate, k: int, pi: int, dout, scale: float | None = None,
             clamp: float = 0.0, L=None, causal: bool = True):
    """Oracle gradients for a loss L with dL/dy = ``dout`` [B,H,N,D].

    Returns (dq, dk, dv) [B,H,N,D] and dgate [B,H,N] (dL/dg of the gate logit
    as seen by each query; a per-head gate's gradient is the sum over its
    queries), all float64.  See the backward block of pi_oracle.c's header.
    """
    L = L or lib()
    q, k_, v, gate, dout = _f32(q), _f32(k_), _f32(v), _f64(gate), _f32(dout)
    B, H, N, D = q.shape
    assert k_.shape == q.shape and v.shape == q.shape and dout.shape == q.shape
    gsb, gsh, gsn = _gate_strides(gate, B, H, N)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    dq, dk, dv = (np.empty((B, H, N, D), dtype=np.float64) for _ in range(3))
    dg = np.empty((B, H, N), dtype=np.float64)
    if B * H * N:
        L.oracle_backward(B, H, N, D, k, pi, int(bool(causal)), _ptr(q), _ptr(k_), _ptr(v), _ptr(gate), gsb, gsh, gsn,
                          float(scale), float(clamp), _ptr(dout), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dg))
    return dq, dk, dv, dg


def decode_step(len_in, q_new, k_new, v_new, k_cache, v_cache, gate, k: int, pi: int,
                scale: float | None = None, clamp: float = 0.0, want_lse=False, L=None):
    """Oracle decode step.  ``k_cache``/``v_cache`` are float32 numpy arrays
    [S,H,cap,D] updated in place (row len_in[s] <- new key/value).  Returns
    out [S,H,D] float64 (and lse [S,H])."""
    L = L or lib()
    for c in (k_cache, v_cache):
        if not (isinstance(c, np.ndarray) and c.dtype == np.float32 and c.flags.c_contiguous):
            raise TypeError("caches must be contiguous float32 numpy arrays (updated in place)")
    S, H, cap, D = k_cache.shape
    q_new, k_new, v_new, gate = _f32(q_new), _f32(k_new), _f32(v_new), _f64(gate)
    len_in = np.ascontiguousarray(np.asarray(len_in, dtype=np.int32))
    if gate.shape == (H,):
        gss, gsh = 0, 1
    elif gate.shape == (S, H):
        gss, gsh = H, 1
    else:
        raise ValueError("decode gate must be [H] or [S,H]")
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    out = np.empty((S, H, D), dtype=np.float64)
    lse = np.empty((S, H), dtype=np.float64) if want_lse else None
    rc = L.oracle_decode_step(S, H, D, cap, k, pi, _ptr(len_in), _ptr(q_new), _ptr(k_new),
                              _ptr(v_new), _ptr(k_cache), _ptr(v_cache), _ptr(gate), gss, gsh,
                              float(scale), float(clamp), _ptr(out), _ptr(lse))
    if rc != 0:
        raise ValueError("len_in out of range [0, cap)")
    return (out, lse) if want_lse else out


def gate_logits(u, w2, b2) -> np.ndarray:
    """Variant-3 gate logits from the gate MLP's hidden activations (the App. A
    gate module is Linear(d, d/2), GELU, Linear(d/2, h), Sigmoid; ``u`` is the
    GELU output [B, N, dh], ``w2`` [H, dh] (the Linear weight as stored) and
    ``b2`` [H] the last Linear layer, whose output is the pre-sigmoid gate
    logit): g[b, h, t] = sum_c u[b, t, c] w2[h, c] + b2[h], in fp64.
    Returns [B, H, N]."""
    u, w2, b2 = (np.asarray(_f32(x), np.float64) for x in (u, w2, b2))
    g = u @ w2.T + b2          # [B, N, H]
    return np.ascontiguousarray(np.transpose(g, (0, 2, 1)))


def num_threads() -> int:
    """OpenMP threads the oracle uses (OMP_NUM_THREADS, else all available cores)."""
    env = os.environ.get("OMP_NUM_THREADS")
    if env and env.strip().isdigit():
        return int(env)
    return len(os.sched_getaffinity(0))
