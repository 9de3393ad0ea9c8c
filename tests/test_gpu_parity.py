"""GPU parity: the HIP path, called through the C ABI, against the fp64 CPU
oracle on the same seeded inputs (device-to-host copies of exactly the bytes
the kernels consumed).

Bars: index sets bit-exact; float32 outputs max-abs <= 1e-4; bfloat16 outputs
max-abs <= 2e-2 and relative L2 <= 5e-3 (against the fp64 oracle).
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2511_10696_amd as pa
from paper_2511_10696_amd import workloads as W
from tests.oracle_pins import IDX_CASES

pytestmark = pytest.mark.gpu

F32_TOL = 1e-4
BF16_MAXABS, BF16_RELL2 = 2e-2, 5e-3
LSE_TOL = 1e-3


def np32(t):
    return t.detach().float().cpu().numpy()


def assert_close(got, ref, dtype, what=""):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    err = np.abs(got - ref)
    if dtype == torch.float32:
        assert err.max() <= F32_TOL, f"{what}: max-abs {err.max():.3g}"
    else:
        rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)
        assert err.max() <= BF16_MAXABS, f"{what}: max-abs {err.max():.3g}"
        assert rel <= BF16_RELL2, f"{what}: rel-L2 {rel:.3g}"


def run_forward(q, k, v, gate, kw, pi, **kw2):
    out, lse = pa.pi_attn_forward(q, k, v, gate, kw, pi, return_lse=True, **kw2)
    torch.cuda.synchronize()
    return out, lse


def rand_inputs(B, H, N, D, dtype, seed, per_query_gate=False, device="cuda"):
    cfg = W.ForwardConfig("custom", B, H, N, D, 0, 0, dtype)
    return W.forward_inputs(cfg, seed, device, per_query_gate)


# ---------------------------------------------------------------------------
# index sets
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("n,k,pi", IDX_CASES + [(256, 32, 64), (4096, 128, 256), (16384, 256, 512),
                                                (32768, 512, 1024), (1000, 0, 0), (70, 70, 3)])
def test_index_set_bit_exact(device, n, k, pi):
    got = pa.pi_attn_index_set(n, k, pi).cpu().numpy()
    ref = oracle.index_set(n, k, pi)
    assert got.dtype == np.int32 and np.array_equal(got, ref)


# ---------------------------------------------------------------------------
# forward, float32
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_forward_f32_tiny(device, seed):
    cfg = W.FORWARD["tiny"]
    q, k, v, gate = W.forward_inputs(cfg, seed, device)
    out, lse = run_forward(q, k, v, gate, cfg.k, cfg.pi)
    ref, lref = oracle.forward(q, k, v, gate, cfg.k, cfg.pi, want_lse=True)
    assert_close(np32(out), ref, torch.float32, "tiny")
    assert np.abs(np32(lse) - lref).max() <= LSE_TOL


@pytest.mark.parametrize("B,H,N,D,k,pi", [(1, 2, 70, 128, 5, 13), (2, 1, 33, 64, 0, 0), (1, 1, 40, 64, 7, 3),
                                          (1, 2, 50, 128, 60, 7), (1, 1, 1, 64, 4, 16)])
def test_forward_f32_shapes(device, B, H, N, D, k, pi):
    q, k_, v, gate = rand_inputs(B, H, N, D, torch.float32, 5, per_query_gate=True)
    out, lse = run_forward(q, k_, v, gate, k, pi)
    ref, lref = oracle.forward(q, k_, v, gate, k, pi, want_lse=True)
    assert_close(np32(out), ref, torch.float32)
    assert np.abs(np32(lse) - lref).max() <= LSE_TOL


# ---------------------------------------------------------------------------
# forward, bfloat16 (banded MFMA kernel)
# ---------------------------------------------------------------------------
BF16_SHAPES = [
    # several query tiles, ragged tails, partner inside and outside the band
    (1, 2, 300, 64, 37, 100),
    (2, 3, 517, 128, 64, 129),
    (1, 2, 640, 128, 130, 260),
    (1, 1, 1, 64, 4, 16),           # single position
    (1, 1, 127, 128, 4, 16),        # less than one query tile, small k (paper default)
    (1, 2, 200, 64, 0, 0),          # self only
    (1, 2, 333, 128, 40, 40),       # pi == k: no separate partner
    (1, 1, 300, 64, 299, 17),       # k >= N-1: dense causal
    (1, 1, 257, 128, 5, 256),       # partner exists only for the last row
    (2, 2, 1100, 64, 100, 1000),    # partner period beyond several tiles
]


@pytest.mark.parametrize("B,H,N,D,k,pi", BF16_SHAPES)
@pytest.mark.parametrize("per_query_gate", [False, True])
def test_forward_bf16_shapes(device, B, H, N, D, k, pi, per_query_gate):
    q, k_, v, gate = rand_inputs(B, H, N, D, torch.bfloat16, 7, per_query_gate)
    out, lse = run_forward(q, k_, v, gate, k, pi)
    ref, lref = oracle.forward(q, k_, v, gate, k, pi, want_lse=True)
    assert_close(np32(out), ref, torch.bfloat16, f"{(B, H, N, D, k, pi)}")
    assert np.abs(np32(lse) - lref).max() <= LSE_TOL


def test_forward_bf16_self_only_is_exact(device):
    """k = 0, no partner: each query attends only to itself, weight exactly 1."""
    q, k, v, gate = rand_inputs(1, 2, 300, 128, torch.bfloat16, 3)
    out, _ = run_forward(q, k, v, gate, 0, 0)
    assert torch.equal(out, v)


def test_forward_bf16_row0_is_v0(device):
    q, k, v, gate = rand_inputs(2, 3, 200, 64, torch.bfloat16, 4)
    out, _ = run_forward(q, k, v, gate, 16, 40)
    assert torch.equal(out[:, :, 0], v[:, :, 0])


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_forward_bf16_config_4k(device, seed):
    cfg = W.FORWARD["fwd4k"]
    q, k, v, gate = W.forward_inputs(cfg, seed, device)
    out, lse = run_forward(q, k, v, gate, cfg.k, cfg.pi)
    ref, lref = oracle.forward(q, k, v, gate, cfg.k, cfg.pi, want_lse=True)
    assert_close(np32(out), ref, torch.bfloat16, "fwd4k")
    assert np.abs(np32(lse) - lref).max() <= LSE_TOL


def sampled_rows(cfg, rng):
    """Every query of two seeded (b, h) pairs, plus in every head the rows
    t < pi + 256, the last 512 rows and the rows at query-tile boundaries."""
    B, H, N = cfg.B, cfg.H, cfg.N
    bh = rng.choice(B * H, size=2, replace=False)
    rows = [np.arange(N) + x * N for x in bh]
    early = np.concatenate([np.arange(min(N, cfg.pi + 256)), np.arange(max(0, N - 512), N)])
    bounds = np.unique(np.concatenate([np.arange(0, N, 128), np.arange(127, N, 128),
                                       np.arange(63, N, 128), np.arange(64, N, 128)]))
    bounds = rng.choice(bounds, size=min(256, bounds.size), replace=False)
    for x in range(B * H):
        rows.append(early + x * N)
        rows.append(bounds + x * N)
    return np.unique(np.concatenate(rows))


@pytest.mark.parametrize("name", ["fwd16k", "fwd32k"])
def test_forward_bf16_config_sampled(device, name):
    cfg = W.FORWARD[name]
    q, k, v, gate = W.forward_inputs(cfg, 0, device)
    out, lse = run_forward(q, k, v, gate, cfg.k, cfg.pi)
    rows = sampled_rows(cfg, np.random.default_rng(0))
    ref, lref = oracle.forward(q, k, v, gate, cfg.k, cfg.pi, rows=rows, want_lse=True)
    got = np32(out).reshape(-1, cfg.D)[rows]
    assert_close(got, ref, torch.bfloat16, name)
    assert np.abs(np32(lse).reshape(-1)[rows] - lref).max() <= LSE_TOL


@pytest.mark.parametrize("name,kw", [("fwd32k", dict(k=32767, pi=1024)), ("fwd32k", dict(k=512, pi=0))])
def test_forward_bf16_dense_and_local_only(device, name, kw):
    """The same shape as dense causal attention (k = N-1) and window-only (pi = 0)."""
    cfg = W.FORWARD[name]
    q, k, v, gate = W.forward_inputs(cfg, 1, device)
    out, lse = run_forward(q, k, v, gate, kw["k"], kw["pi"])
    rng = np.random.default_rng(1)
    rows = np.unique(np.concatenate([rng.choice(cfg.B * cfg.H * cfg.N, 384, replace=False),
                                     np.arange(130), cfg.N - 1 - np.arange(130)]))
    ref, lref = oracle.forward(q, k, v, gate, kw["k"], kw["pi"], rows=rows, want_lse=True)
    assert_close(np32(out).reshape(-1, cfg.D)[rows], ref, torch.bfloat16)
    assert np.abs(np32(lse).reshape(-1)[rows] - lref).max() <= LSE_TOL


def test_forward_bf16_logit_clamp(device):
    """Clamp of the fused logits (L_c = 20) on heavy-hitter keys whose logits exceed it."""
    cfg = W.ForwardConfig("hh", 1, 2, 700, 128, 50, 120, torch.bfloat16, heavy_frac=0.05, heavy_mult=8.0)
    q, k, v, gate = W.forward_inputs(cfg, 2, device, per_query_gate=True)
    for clamp in (20.0, 3.0):
        out, lse = run_forward(q, k, v, gate, cfg.k, cfg.pi, logit_clamp=clamp, scale=0.5)
        ref, lref = oracle.forward(q, k, v, gate, cfg.k, cfg.pi, scale=0.5, clamp=clamp, want_lse=True)
        assert_close(np32(out), ref, torch.bfloat16, f"clamp {clamp}")
        assert np.abs(np32(lse) - lref).max() <= LSE_TOL * 10


def test_forward_strided_layout(device):
    """[B, N, H, D] storage viewed as [B, H, N, D]: same result as contiguous."""
    B, H, N, D = 2, 3, 300, 64
    g = torch.Generator(device="cuda").manual_seed(9)
    base = [torch.randn(B, N, H, D, generator=g, device="cuda").to(torch.bfloat16) for _ in range(3)]
    q, k, v = (x.permute(0, 2, 1, 3) for x in base)
    gate = torch.rand(H, generator=g, device="cuda") * 2 - 1
    out_strided = torch.empty(B, N, H, D, dtype=torch.bfloat16, device="cuda").permute(0, 2, 1, 3)
    pa.pi_attn_forward(q, k, v, gate, 20, 50, out=out_strided)
    out_c = pa.pi_attn_forward(q.contiguous(), k.contiguous(), v.contiguous(), gate, 20, 50)
    torch.cuda.synchronize()
    assert torch.equal(out_strided, out_c)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_forward_causality(device, dtype):
    """Perturbing positions after `cut` leaves rows <= cut bit-identical.
    Keys and queries after the cut become NaN; values after the cut become
    large finite numbers inside the cut's 128-query tile and NaN beyond it
    (a masked weight is exactly 0, and 0 times a finite value adds nothing)."""
    B, H, N, D, k, pi = 1, 2, 600, 128, 70, 150
    q, kk, v, gate = rand_inputs(B, H, N, D, dtype, 11)
    base, _ = run_forward(q, kk, v, gate, k, pi)
    for cut in (0, 130, 255, 383, 598):
        q2, k2, v2 = q.clone(), kk.clone(), v.clone()
        q2[:, :, cut + 1:] = float("nan")
        k2[:, :, cut + 1:] = float("nan")
        tile_end = (cut // 128 + 1) * 128
        v2[:, :, cut + 1:tile_end] = 1e4
        v2[:, :, tile_end:] = float("nan")
        out, _ = run_forward(q2, k2, v2, gate, k, pi)
        assert torch.equal(out[:, :, :cut + 1], base[:, :, :cut + 1]), cut


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_forward_deterministic(device, dtype):
    q, k, v, gate = rand_inputs(2, 4, 1000, 128, dtype, 12)
    a, la = run_forward(q, k, v, gate, 100, 300)
    b, lb = run_forward(q, k, v, gate, 100, 300)
    assert torch.equal(a, b) and torch.equal(la, lb)


def test_forward_head_permutation(device):
    q, k, v, gate = rand_inputs(1, 4, 400, 64, torch.bfloat16, 13)
    perm = torch.tensor([2, 0, 3, 1], device="cuda")
    a, _ = run_forward(q, k, v, gate, 30, 90)
    b, _ = run_forward(q[:, perm].contiguous(), k[:, perm].contiguous(), v[:, perm].contiguous(),
                       gate[perm].contiguous(), 30, 90)
    assert torch.equal(a[:, perm], b)


# ---------------------------------------------------------------------------
# decode step
# ---------------------------------------------------------------------------
def decode_small(dtype, D, seed=21):
    S, H, cap, k, pi = 4, 2, 320, 37, 100
    g = torch.Generator(device="cuda").manual_seed(seed)
    kc = torch.randn(S, H, cap, D, generator=g, device="cuda").to(dtype)
    vc = torch.randn(S, H, cap, D, generator=g, device="cuda").to(dtype)
    lens = torch.tensor([0, 50, 100, 250], dtype=torch.int32, device="cuda")
    gate = torch.rand(S, H, generator=g, device="cuda") * 2 - 1
    return S, H, cap, k, pi, kc, vc, lens, gate, g


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("D", [64, 128])
def test_decode_steps_small(device, dtype, D):
    S, H, cap, k, pi, kc, vc, lens, gate, g = decode_small(dtype, D)
    len_a, len_b = lens.clone(), torch.empty_like(lens)
    for step in range(6):
        qn, kn, vn = (torch.randn(S, H, D, generator=g, device="cuda").to(dtype) for _ in range(3))
        before_k = kc.clone()
        lse = torch.empty(S, H, dtype=torch.float32, device="cuda")
        out = pa.pi_attn_decode_step(len_a, qn, kn, vn, kc, vc, gate, k, pi, len_out=len_b, lse=lse)
        torch.cuda.synchronize()
        t = len_a.cpu().numpy()
        assert np.array_equal(len_b.cpu().numpy(), t + 1)
        kc_ref = np32(before_k)
        vc_ref = np32(vc)   # rows != t are unchanged by the step; the oracle rewrites row t
        ref, lref = oracle.decode_step(t, qn, kn, vn, kc_ref, vc_ref, gate, k, pi, want_lse=True)
        assert_close(np32(out), ref, dtype, f"step {step}")
        assert np.abs(np32(lse) - lref).max() <= LSE_TOL
        for s in range(S):
            assert torch.equal(kc[s, :, t[s]], kn[s]) and torch.equal(vc[s, :, t[s]], vn[s])
        mask = torch.ones(cap, dtype=torch.bool, device="cuda")
        for s in range(S):
            mask[:] = True
            mask[int(t[s])] = False
            assert torch.equal(kc[s][:, mask], before_k[s][:, mask])
        len_a, len_b = len_b, len_a


def test_decode_idempotent_and_len_out_optional(device):
    S, H, cap, k, pi, kc, vc, lens, gate, g = decode_small(torch.bfloat16, 128)
    qn, kn, vn = (torch.randn(S, H, 128, generator=g, device="cuda").to(torch.bfloat16) for _ in range(3))
    a = pa.pi_attn_decode_step(lens, qn, kn, vn, kc, vc, gate, k, pi)
    b = pa.pi_attn_decode_step(lens, qn, kn, vn, kc, vc, gate, k, pi)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    assert torch.equal(lens.cpu(), torch.tensor([0, 50, 100, 250], dtype=torch.int32))


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_decode_length_out_of_range(device, dtype):
    """A length outside [0, cap) yields NaN for that sequence and no cache write."""
    S, H, cap, k, pi, kc, vc, lens, gate, g = decode_small(dtype, 128)
    lens = torch.tensor([5, cap, -1, 7], dtype=torch.int32, device="cuda")
    len_out = torch.empty_like(lens)
    qn, kn, vn = (torch.randn(S, H, 128, generator=g, device="cuda").to(dtype) for _ in range(3))
    kc0, vc0 = kc.clone(), vc.clone()
    out = pa.pi_attn_decode_step(lens, qn, kn, vn, kc, vc, gate, k, pi, len_out=len_out)
    torch.cuda.synchronize()
    assert torch.isnan(out[1]).all() and torch.isnan(out[2]).all()
    assert torch.isfinite(out[0]).all() and torch.isfinite(out[3]).all()
    assert torch.equal(kc[1], kc0[1]) and torch.equal(kc[2], kc0[2]) and torch.equal(vc[1], vc0[1])
    assert len_out.cpu().tolist() == [6, cap, -1, 8]


def test_decode_config(device):
    """The decode workload (64 sequences, 32 heads, 32768 cached rows, k=512,
    pi=1024): 1000 consecutive steps.  Every appended cache row equals its
    token bit for bit; at steps 0, 1, 499 and 999 every (s, h) pair, and at
    16 seeded steps 64 seeded pairs, against the oracle.  The oracle's cache
    for step i holds only rows [t - pi, t] (t = 32768 + i, all its working
    set can reach), built from the seeded initial cache and the seeded
    tokens of the earlier steps, never from the caches the kernel wrote."""
    cfg = W.DECODE["decode"]
    kc, vc, lens, gate = W.decode_state(cfg, 0, device)
    qs, ks, vs = W.decode_tokens(cfg, cfg.steps, 1, device)
    L0, P = cfg.cache_len, cfg.pi
    assert cfg.steps <= P    # every step's reach [t - pi, t) starts inside the initial cache
    k0 = kc[:, :, L0 - P:L0].float().cpu().numpy()    # initial rows [L0 - pi, L0), fp32 (exact)
    v0 = vc[:, :, L0 - P:L0].float().cpu().numpy()
    len_buf = [lens, torch.empty_like(lens)]
    rng = np.random.default_rng(3)
    full_steps = [0, 1, 499, cfg.steps - 1]
    some_steps = sorted(set(rng.choice(cfg.steps, 16, replace=False).tolist()) - set(full_steps))
    outs = {}
    for step in range(cfg.steps):
        out = pa.pi_attn_decode_step(len_buf[step % 2], qs[step], ks[step], vs[step], kc, vc, gate,
                                     cfg.k, cfg.pi, len_out=len_buf[(step + 1) % 2])
        if step in full_steps or step in some_steps:
            outs[step] = out.clone()
    torch.cuda.synchronize()
    assert (len_buf[cfg.steps % 2] == L0 + cfg.steps).all()
    assert torch.equal(kc[:, :, L0:L0 + cfg.steps], ks.permute(1, 2, 0, 3))
    assert torch.equal(vc[:, :, L0:L0 + cfg.steps], vs.permute(1, 2, 0, 3))
    ks_h, vs_h = ks.float().cpu().numpy(), vs.float().cpu().numpy()    # [steps, S, H, D]

    def reach(step, s_idx, h_idx):
        """Cache rows [t - pi, t) of the listed pairs as the step saw them:
        [S', H', pi + 1, D], the last row left for the oracle's own write."""
        a = P - step
        kk = np.empty((len(s_idx), len(h_idx), P + 1, cfg.D), np.float32)
        vv = np.empty_like(kk)
        kk[:, :, :a] = k0[np.ix_(s_idx, h_idx)][:, :, step:]
        vv[:, :, :a] = v0[np.ix_(s_idx, h_idx)][:, :, step:]
        kk[:, :, a:P] = ks_h[:step][:, s_idx][:, :, h_idx].transpose(1, 2, 0, 3)
        vv[:, :, a:P] = vs_h[:step][:, s_idx][:, :, h_idx].transpose(1, 2, 0, 3)
        return kk, vv

    all_s, all_h = np.arange(cfg.S), np.arange(cfg.H)
    for step in full_steps:
        kk, vv = reach(step, all_s, all_h)
        t_rel = np.full(cfg.S, P, np.int32)   # t sits at row pi of the reach
        ref = oracle.decode_step(t_rel, qs[step], ks[step], vs[step], kk, vv, gate, cfg.k, cfg.pi)
        assert_close(np32(outs[step]), ref, torch.bfloat16, f"step {step}, all pairs")
    for step in some_steps:
        for s, h in zip(rng.choice(cfg.S, 64), rng.choice(cfg.H, 64)):
            s, h = int(s), int(h)
            kk, vv = reach(step, [s], [h])
            ref = oracle.decode_step(np.array([P], np.int32), qs[step, s:s + 1, h:h + 1],
                                     ks[step, s:s + 1, h:h + 1], vs[step, s:s + 1, h:h + 1],
                                     kk, vv, gate[h:h + 1], cfg.k, cfg.pi)
            assert_close(np32(outs[step][s:s + 1, h:h + 1]), ref, torch.bfloat16, f"step {step} s{s} h{h}")
