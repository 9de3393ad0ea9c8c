"""Host-side pieces of the benchmark: algorithmic work counts and the
refusal to run on more than one GPU."""
import subprocess
import sys

import bench
from paper_2511_10696_amd import workloads as W


def test_attended_keys_match_closed_form():
    # sum over t of |W_t| per (b, h): window min(t,k)+1 plus the partner for t >= pi
    per_bh = {"tiny": 8112, "fwd4k": 523968, "fwd16k": 4193664, "fwd32k": 16710400, "smallk8k": 49126}
    for name, cfg in W.FORWARD.items():
        keys, flops, nbytes = bench.forward_algorithmic(cfg)
        assert keys == per_bh[name] * cfg.B * cfg.H
        assert flops == 4 * cfg.D * keys
        assert nbytes == 4 * cfg.B * cfg.H * cfg.N * cfg.D * 2


def test_decode_bytes_per_step():
    cfg = W.DECODE["decode"]
    keys, nbytes = bench.decode_algorithmic(cfg, cfg.cache_len)
    assert keys == 514 * cfg.S * cfg.H
    assert nbytes == (2 * 513 + 6) * cfg.D * 2 * cfg.S * cfg.H


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, "bench.py", "--gpus", "2"], capture_output=True, text=True,
                       cwd=bench.ROOT)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_bidirectional_attended_keys_match_the_index_sets():
    import oracle
    for name in ("tiny", "fwd4k"):
        cfg = W.FORWARD[name]
        keys, flops, _ = bench.forward_algorithmic(cfg, causal=False)
        idx = oracle.index_set(cfg.N, cfg.k, cfg.pi, causal=False)
        assert keys == int((idx >= 0).sum()) * cfg.B * cfg.H
        assert flops == 4 * cfg.D * keys


def test_shard_accounting():
    """One rank's share of fwd32k sharded eight ways: every query of the last
    shard attends k + 1 window keys and its partner; the bytes are its q and
    out plus the k/v rows held (shard and pi halo)."""
    cfg = W.FORWARD["fwd32k"]
    s0, lo = cfg.N - cfg.N // 8, cfg.N - cfg.N // 8 - cfg.pi
    keys, flops, nbytes = bench.shard_algorithmic(cfg, s0, cfg.N, lo)
    assert keys == (cfg.N - s0) * (cfg.k + 2) * cfg.B * cfg.H
    assert flops == 4 * cfg.D * keys
    assert nbytes == cfg.B * cfg.H * cfg.D * 2 * (2 * (cfg.N - s0) + 2 * (cfg.N - lo))


def test_cpu_baseline_legs_on_a_small_problem():
    """The CPU-baseline leg on small stand-ins: the all-core forward, the
    one-thread slice extrapolated to every head, and ten decode steps over
    the rows each step can reach."""
    import dataclasses
    import torch
    cfg = W.ForwardConfig("small", 1, 2, 300, 64, 32, 64, torch.bfloat16)
    host = W.forward_inputs(cfg, 0, "cpu")
    dcfg = dataclasses.replace(W.DECODE["decode"], S=2, H=2, D=64, k=16, pi=40, cache_len=100, steps=10)
    g = torch.Generator().manual_seed(0)
    k0, v0 = (torch.randn(2, 2, 40, 64, generator=g).to(torch.bfloat16) for _ in range(2))
    qs, ks, vs = (torch.randn(10, 2, 2, 64, generator=g).to(torch.bfloat16) for _ in range(3))
    res = bench.cpu_baseline(cfg, host, dcfg, (k0, v0, qs, ks, vs, torch.zeros(2)))
    assert res["kind"] == "oracle" and res["value"] > 0 and res["cores"] >= 1
    st = res["single_thread_extrapolated"]
    assert st["cores"] == 1 and st["value"] > 0 and "extrapolated" in st["sample"]
    assert res["decode"]["steps"] == 10 and res["decode"]["us_per_step"] > 0
