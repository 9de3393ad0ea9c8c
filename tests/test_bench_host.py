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
