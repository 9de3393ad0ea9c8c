"""Seeded synthetic workloads (shapes, distributions) and their generators.

This module holds no arithmetic of the attention method: it only draws the
input tensors.  Tests and the benchmark hand the same tensors to the HIP
path and (after a device-to-host copy) to the CPU oracle, so parity never
depends on two random number generators agreeing.

Workloads (one GPU):
  tiny    B1  H2  N256   D64  k32  pi64   float32
  fwd4k   B4  H16 N4096  D64  k128 pi256  bf16, q scaled by 1/sqrt(D)
  fwd16k  B2  H32 N16384 D128 k256 pi512  bf16, 1% of key rows x8 (heavy hitters)
  fwd32k  B1  H32 N32768 D128 k512 pi1024 bf16
  smallk8k B8 H16 N8192  D64  k4   pi16   bf16, the paper's default window and period
          (Sec. 4, App. B) at its 8K efficiency context; gate from the gate MLP's
          last layer (hidden width d/2 = 512)
  decode  S64 H32 D128 k512 pi1024, bf16 KV cache of 32768 rows, 1000 appended steps
q, k, v ~ N(0, 1) drawn in float32 then rounded to the dtype; per-head gate
logits ~ U(-1, 1) in float32.  The paper's own efficiency runs use trained
models on WikiText-103; these synthetic tensors stand in for them.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import torch

EFF_K, EFF_PI = 4, 16   # the paper's default window radius and period


@dataclass(frozen=True)
class ForwardConfig:
    name: str
    B: int
    H: int
    N: int
    D: int
    k: int
    pi: int
    dtype: torch.dtype
    q_scale: float = 1.0          # multiply q by this after drawing (exact power of two here)
    heavy_frac: float = 0.0       # fraction of key rows per (b, h) multiplied by heavy_mult
    heavy_mult: float = 1.0


@dataclass(frozen=True)
class DecodeConfig:
    name: str
    S: int
    H: int
    D: int
    k: int
    pi: int
    cache_len: int                # rows present before the first step
    steps: int
    dtype: torch.dtype = torch.bfloat16
    extra: dict = field(default_factory=dict)

    @property
    def cap(self) -> int:
        # room for every appended step, rounded up to a multiple of 64 rows
        return ((self.cache_len + self.steps + 63) // 64) * 64


FORWARD = {
    "tiny": ForwardConfig("tiny", 1, 2, 256, 64, 32, 64, torch.float32),
    "fwd4k": ForwardConfig("fwd4k", 4, 16, 4096, 64, 128, 256, torch.bfloat16, q_scale=1.0 / 8.0),
    "fwd16k": ForwardConfig("fwd16k", 2, 32, 16384, 128, 256, 512, torch.bfloat16,
                            heavy_frac=0.01, heavy_mult=8.0),
    "fwd32k": ForwardConfig("fwd32k", 1, 32, 32768, 128, 512, 1024, torch.bfloat16),
    "smallk8k": ForwardConfig("smallk8k", 8, 16, 8192, 64, EFF_K, EFF_PI, torch.bfloat16),
}
DECODE = {
    "decode": DecodeConfig("decode", 64, 32, 128, 512, 1024, 32768, 1000),
}


def _gen(device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def forward_inputs(cfg: ForwardConfig, seed: int = 0, device="cuda", per_query_gate: bool = False):
    """q, k, v [B, H, N, D] (cfg.dtype, contiguous) and float32 gate logits
    ([H], or [B, H, N] when per_query_gate)."""
    g = _gen(device, seed)
    shape = (cfg.B, cfg.H, cfg.N, cfg.D)
    out = []
    for which in range(3):
        x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
        if which == 0 and cfg.q_scale != 1.0:
            x.mul_(cfg.q_scale)
        if which == 1 and cfg.heavy_frac > 0:
            n_heavy = int(math.floor(cfg.heavy_frac * cfg.N))
            for b in range(cfg.B):
                for h in range(cfg.H):
                    rows = torch.randperm(cfg.N, generator=g, device=device)[:n_heavy]
                    x[b, h, rows] *= cfg.heavy_mult
        out.append(x.to(cfg.dtype))
        del x
    gshape = (cfg.B, cfg.H, cfg.N) if per_query_gate else (cfg.H,)
    gate = torch.rand(gshape, generator=g, device=device, dtype=torch.float32) * 2.0 - 1.0
    return out[0], out[1], out[2], gate


def gate_mlp_inputs(cfg: ForwardConfig, seed: int = 0, device="cuda", dh: int | None = None):
    """Operands of the gate MLP's last layer: u [B, N, dh] (GELU of N(0, 1),
    the hidden activations), w2 [H, dh] ~ N(0, 1/dh) (both cfg.dtype) and
    b2 [H] ~ U(-0.1, 0.1) float32; dh defaults to d/2 = H*D/2."""
    dh = dh or cfg.H * cfg.D // 2
    g = _gen(device, seed + 2000003)
    x = torch.randn((cfg.B, cfg.N, dh), generator=g, device=device, dtype=torch.float32)
    u = torch.nn.functional.gelu(x).to(cfg.dtype)
    del x
    w2 = (torch.randn((cfg.H, dh), generator=g, device=device, dtype=torch.float32) / math.sqrt(dh)).to(cfg.dtype)
    b2 = torch.rand((cfg.H,), generator=g, device=device, dtype=torch.float32) * 0.2 - 0.1
    return u, w2, b2


def cotangent(shape, dtype, seed: int = 0, device="cuda"):
    """Seeded dL/dy for the backward: N(0, 1) in ``dtype`` (its own stream,
    seed offset so it never repeats the q/k/v draws of the same seed)."""
    g = _gen(device, seed + 1000003)
    return torch.randn(tuple(shape), generator=g, device=device, dtype=torch.float32).to(dtype)


def decode_state(cfg: DecodeConfig, seed: int = 0, device="cuda"):
    """Caches [S, H, cap, D] with rows [0, cache_len) ~ N(0,1) and the rest
    zero, the int32 lengths [S] (= cache_len), and per-head gate logits."""
    g = _gen(device, seed)
    shape = (cfg.S, cfg.H, cfg.cap, cfg.D)
    caches = []
    for _ in range(2):
        c = torch.zeros(shape, dtype=cfg.dtype, device=device)
        for s in range(cfg.S):
            c[s, :, :cfg.cache_len] = torch.randn((cfg.H, cfg.cache_len, cfg.D), generator=g,
                                                  device=device, dtype=torch.float32).to(cfg.dtype)
        caches.append(c)
    lens = torch.full((cfg.S,), cfg.cache_len, dtype=torch.int32, device=device)
    gate = torch.rand((cfg.H,), generator=g, device=device, dtype=torch.float32) * 2.0 - 1.0
    return caches[0], caches[1], lens, gate


def decode_tokens(cfg: DecodeConfig, steps: int, seed: int = 1, device="cuda"):
    """New q, k, v rows for `steps` steps: [steps, S, H, D] each."""
    g = _gen(device, seed)
    shape = (steps, cfg.S, cfg.H, cfg.D)
    return tuple(torch.randn(shape, generator=g, device=device, dtype=torch.float32).to(cfg.dtype)
                 for _ in range(3))
