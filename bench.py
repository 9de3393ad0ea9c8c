"""Benchmark of the pi-Attention hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W]

Workload (the metric's configuration): full-sequence causal forward, B=1,
H=32, N=32768, D=128, k=512, pi=1024, bf16 q/k/v ~ N(0,1), per-head gate
logits ~ U(-1,1).  One step = one pi_attn_forward over the whole sequence.
Also timed in the same run: the KV-cached decode step (64 sequences, 32
heads, 32768 cached rows, k=512, pi=1024, 1000 consecutive steps), the
bidirectional forward on the same shape, one rank's share of the sequence
sharded eight ways (pi_attn_forward_shard), the backward (pi_attn_backward,
causal and bidirectional) on that shape with a seeded dL/dy, and the fp64
CPU oracle on a bounded sample of the forward workload.

The forward is also timed cold: single launches, each after a 1 GiB device
fill that evicts the L2s and the last-level cache (reported beside the
steady-state figure, which is the headline).  The decode step reports the mean
over its 1000 steps and, from a second pass over the same steps with an event
after each, the median and p99 of the per-step times.

Every timed loop is preceded by a settling phase (the same launches, untimed,
for at least SETTLE_S seconds, so the GPU clocks have left their idle state)
and by the warm-up launches; the timed region is exactly the stated number
of launches between two HIP events on the launch stream.

Prints ONE JSON line.  value = query positions per second (B*N per step) of
the forward, inputs resident in HBM.
"""
from __future__ import annotations

import argparse
import dataclasses
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA, TFLOP/s
PROFILE_TRAFFIC = os.path.join(ROOT, "profiles", "forward_bf16_fwd32k_counters.txt")
DECODE_TRAFFIC = os.path.join(ROOT, "profiles", "decode_bf16_s64_counters.txt")
BIDIR_TRAFFIC = os.path.join(ROOT, "profiles", "forward_bf16_bidir_fwd32k_counters.txt")
BACKWARD_TRAFFIC = {True: os.path.join(ROOT, "profiles", "backward_bf16_fwd32k_counters.txt"),
                    False: os.path.join(ROOT, "profiles", "backward_bf16_bidir_fwd32k_counters.txt")}
SMALLK_TRAFFIC = {"gated": os.path.join(ROOT, "profiles", "smallk_bf16_gated_smallk8k_counters.txt"),
                  "gated_bidirectional": os.path.join(ROOT, "profiles",
                                                      "smallk_bf16_gated_bidir_smallk8k_counters.txt"),
                  "per_head_gate": os.path.join(ROOT, "profiles", "smallk_bf16_smallk8k_counters.txt"),
                  "backward": os.path.join(ROOT, "profiles", "smallk_bwd_bf16_smallk8k_counters.txt"),
                  "backward_bidirectional": os.path.join(ROOT, "profiles",
                                                         "smallk_bwd_bf16_bidir_smallk8k_counters.txt")}
FORWARD_SOURCES = ("forward_bf16.hip", "pi_common.h", "kernels.h")
SMALLK_SOURCES = ("smallk_bf16.hip", "smallk_common.h", "smallk.h", "pi_common.h", "kernels.h")
SMALLK_BWD_SOURCES = ("smallk_bwd_bf16.hip", "smallk_common.h", "smallk.h", "backward.hip", "pi_common.h",
                      "kernels.h")
BACKWARD_SOURCES = ("backward_bf16.hip", "backward_kv_bf16.hip", "backward.hip", "pi_common.h", "kernels.h")


def csrc_digest(names):
    return source_digest([os.path.join(ROOT, "paper_2511_10696_amd", "csrc", f) for f in names])
COPY_PROBE_BYTES = 1 << 30      # plain device copy used to calibrate the HBM byte counters
SETTLE_S = 0.3                  # untimed run-in before each timed loop (clock ramp)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--cold-reps", type=int, default=10,
                    help="single forward launches timed after an L2/last-level-cache flush")
    ap.add_argument("--decode-steps", type=int, default=1000)
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--backward-steps", type=int, default=20)
    ap.add_argument("--no-backward", action="store_true")
    ap.add_argument("--no-bidirectional", action="store_true")
    ap.add_argument("--no-smallk", action="store_true")
    ap.add_argument("--no-shard", action="store_true")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip the fwd32k dense-causal and local-only comparisons and the fwd4k/fwd16k forwards")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--pmc-probe", action="store_true",
                    help="run 3 launches of each timed kernel (forward, bidirectional forward, backward "
                         "both ways, decode step) and 3 plain 1 GiB device copies, then exit (for "
                         "hardware-counter runs)")
    return ap.parse_args()


def forward_algorithmic(cfg, causal=True):
    """Algorithmic work of one forward: attended keys (sum of |W_t|, closed
    form), FLOPs (QK + PV, 2 FLOP per MAC), bytes (q, k, v read once, out
    written once)."""
    n, k, pi = cfg.N, cfg.k, cfg.pi
    if causal:
        keys = (k + 1) * (k + 2) // 2 + (n - k - 1) * (k + 1) if n > k else n * (n + 1) // 2
        keys += max(0, n - pi) if pi > k else 0
    else:
        keys = n * (2 * k + 1) - k * (k + 1) if n > k else n * n
        keys += 2 * max(0, n - pi) if pi > k else 0
    keys *= cfg.B * cfg.H
    flops = 4 * cfg.D * keys
    es = 2
    nbytes = 4 * cfg.B * cfg.H * cfg.N * cfg.D * es
    return keys, flops, nbytes


def shard_algorithmic(cfg, s0, s1, lo):
    """Algorithmic work of the causal forward of one sequence shard: queries
    [s0, s1) against the k/v rows [lo, s1) held (the shard and its halo):
    attended keys summed per query, FLOPs (QK + PV), bytes (q and out of the
    shard, k and v of the rows held, each once)."""
    k, pi = cfg.k, cfg.pi
    keys = sum(min(t, k) + 1 + (1 if pi > k and t >= pi else 0) for t in range(s0, s1)) * cfg.B * cfg.H
    es = 2
    nbytes = cfg.B * cfg.H * cfg.D * es * (2 * (s1 - s0) + 2 * (s1 - lo))
    return keys, 4 * cfg.D * keys, nbytes


def smallk_algorithmic(cfg, causal=True, gated=True):
    """Algorithmic work of one small-window forward: the attention's keys,
    FLOPs and bytes, plus (gated) the gate MLP's last layer: u [B, N, dh] and
    w2 [H, dh] read once, the logits [B, H, N] float32 written, 2 dh FLOPs
    per (b, h, t)."""
    keys, flops, nbytes = forward_algorithmic(cfg, causal)
    if gated:
        dh = cfg.H * cfg.D // 2
        flops += 2 * dh * cfg.B * cfg.H * cfg.N
        nbytes += 2 * (cfg.B * cfg.N * dh + cfg.H * dh) + 4 * cfg.B * cfg.H * cfg.N
    return keys, flops, nbytes


def time_launches(torch, fn, steps, warmup, stream):
    """Settle (>= SETTLE_S s of fn, untimed), `warmup` more launches, then
    exactly `steps` launches between two HIP events on `stream`.  Returns
    (ms per launch, wall seconds of the timed region, settle seconds)."""
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < SETTLE_S:
        for _ in range(4):
            fn()
        torch.cuda.synchronize()
    settle = time.perf_counter() - t0
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_wall = time.perf_counter()
    e0.record(stream)
    for _ in range(steps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    return e0.elapsed_time(e1) / steps, t_wall, settle


FLUSH_BYTES = 1 << 30    # written between cold launches: 4x the 256 MB last-level cache plus the L2s


def hip_clocks(dev_index):
    """Peak shader and memory clocks (MHz) the HIP runtime reports for the device."""
    import ctypes
    try:
        hip = ctypes.CDLL("libamdhip64.so")
    except OSError:
        return {}
    out = {}
    for name, attr in (("sclk_peak_mhz", "hipDeviceAttributeClockRate"),
                       ("mclk_peak_mhz", "hipDeviceAttributeMemoryClockRate")):
        code = HIP_DEVICE_ATTRIBUTES[attr]
        val = ctypes.c_int(0)
        if hip.hipDeviceGetAttribute(ctypes.byref(val), code, dev_index) == 0:
            out[name] = round(val.value / 1e3, 1)   # kHz -> MHz
    return out


# hipDeviceAttribute_t values of the two clock queries (hip/hip_runtime_api.h, ROCm 7)
HIP_DEVICE_ATTRIBUTES = {"hipDeviceAttributeClockRate": 5, "hipDeviceAttributeMemoryClockRate": 60}


def device_info(torch, dev):
    pr = torch.cuda.get_device_properties(dev)
    return {"name": pr.name, "arch": getattr(pr, "gcnArchName", None), "compute_units": pr.multi_processor_count,
            "hbm_bytes": pr.total_memory, "hbm_peak_gbs": HBM_PEAK_GBS, "mfma_bf16_peak_tflops": MFMA_BF16_PEAK_TFLOPS,
            **hip_clocks(dev.index or 0)}


def time_cold(torch, fn, reps, stream):
    """Median and minimum ms of `reps` single launches, each after a 1 GiB
    device fill (untimed) that evicts the inputs from the L2s and the
    last-level cache, so every launch reads its inputs from HBM."""
    flush = torch.empty(FLUSH_BYTES // 4, dtype=torch.float32, device=stream.device)
    times = []
    for i in range(reps):
        flush.fill_(float(i))
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        fn()
        e1.record(stream)
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
    del flush
    times.sort()
    return times[len(times) // 2], times[0]


def roofline_of(flops, nbytes, sec, kernel, traffic=None, counters=None):
    """Roofline record of one launch: the bound is whichever of the HBM and
    MFMA times of its algorithmic work is larger; `counters` (from the
    committed counter summary of the same kernel sources) adds the measured
    MFMA busy fraction, DRAM rate and clock."""
    tflops, gbs = flops / sec / 1e12, nbytes / sec / 1e9
    hbm = nbytes / (HBM_PEAK_GBS * 1e9) >= flops / (MFMA_BF16_PEAK_TFLOPS * 1e12)
    r = {"bound": "hbm" if hbm else "mfma", "kernel": kernel,
         "achieved": round(gbs if hbm else tflops, 2),
         "peak": HBM_PEAK_GBS if hbm else MFMA_BF16_PEAK_TFLOPS,
         "unit": "GB/s" if hbm else "TFLOP/s",
         "frac": round((gbs / HBM_PEAK_GBS) if hbm else (tflops / MFMA_BF16_PEAK_TFLOPS), 4),
         "traffic": traffic}
    if counters:
        r.update(counters)
    mf = {"achieved": round(tflops, 2), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
          "frac": round(tflops / MFMA_BF16_PEAK_TFLOPS, 4), "flops_per_launch": flops,
          "bytes_per_launch": nbytes}
    return r, mf


def backward_algorithmic(cfg, causal=True):
    """Algorithmic work of one backward: per attended key 10*D FLOPs (the
    scores recomputed, dP = dO V^T, dV, dQ and dK: five D-long products,
    2 FLOP per MAC); bytes: q, k, v, dO read once (input dtype), lse read,
    dq, dk, dv (float32) and the per-query gate gradient written."""
    keys, _, _ = forward_algorithmic(cfg, causal)
    rows = cfg.B * cfg.H * cfg.N
    nbytes = rows * (4 * cfg.D * 2 + 3 * cfg.D * 4 + 4 + 4)
    return keys, 10 * cfg.D * keys, nbytes


def decode_algorithmic(cfg, t):
    """Per decode step: cache rows read (window t-k..t-1 plus partner) for K
    and V, plus q/k/v of the new token read, the appended row and out written."""
    rows = min(t, cfg.k) + (1 if (cfg.pi > cfg.k and t >= cfg.pi) else 0)
    es = 2
    per_sh = (2 * rows + 3 + 2 + 1) * cfg.D * es
    keys = (rows + 1) * cfg.S * cfg.H
    return keys, per_sh * cfg.S * cfg.H


def source_digest(paths):
    h = hashlib.sha256()
    for p in paths:
        h.update(open(p, "rb").read())
    return h.hexdigest()[:16]


def read_profile(digest, path):
    """The key = value fields of a committed rocprofv3 counter summary, or
    None when it is missing or was taken on other kernel sources (its
    source_digest differs from `digest`)."""
    if not os.path.exists(path):
        return None
    rec = {}
    for line in open(path):
        if "=" in line and not line.lstrip().startswith("#"):
            key, val = line.split("=", 1)
            rec[key.strip()] = val.strip()
    return rec if rec.get("source_digest") == digest else None


def measured_traffic(digest, path=PROFILE_TRAFFIC):
    """HBM bytes per launch (calibrated FETCH_SIZE + WRITE_SIZE) from the
    committed rocprofv3 counter summary; valid only for the kernel source it
    was taken on, so None once the source digest differs."""
    rec = read_profile(digest, path)
    if rec is None or "hbm_bytes_per_launch" not in rec:
        return None
    return int(float(rec["hbm_bytes_per_launch"]))


def measured_counters(digest, path, sec):
    """Counter figures of the same summary for the bench line: the MFMA busy
    fraction (SQ_VALU_MFMA_BUSY_CYCLES over the SIMD-cycles of the kernel's
    active time), the LDS bank-conflict fraction, an upper bound on the
    shader clock the kernel ran at (GRBM_GUI_ACTIVE cycles, whose counting
    window can extend past the dispatch, over its traced duration; taken
    from dispatches of at least 300 us only), and the measured DRAM rate
    (the counted HBM bytes over this run's launch time).  Empty when the
    summary does not match the kernel sources."""
    rec = read_profile(digest, path)
    if rec is None:
        return {}
    out = {}
    for key in ("mfma_busy", "lds_bank_conflict", "sclk_mhz_max"):
        if key in rec:
            out[key] = float(rec[key])
    if "hbm_bytes_per_launch" in rec:
        out["dram_gbs"] = round(float(rec["hbm_bytes_per_launch"]) / sec / 1e9, 2)
    return out


def pmc_probe(W, pa, torch, dev):
    """Launch each kernel a few times (and a plain copy of known size) so a
    counter run can read per-dispatch HBM bytes and calibrate them."""
    cfg = W.FORWARD["fwd32k"]
    q, k, v, gate = W.forward_inputs(cfg, 0, dev)
    out = torch.empty_like(q)
    for _ in range(3):
        pa.pi_attn_forward(q, k, v, gate, cfg.k, cfg.pi, out=out)
    torch.cuda.synchronize()
    print(f"probe: 3 x forward fwd32k", flush=True)
    for _ in range(3):
        pa.pi_attn_forward(q, k, v, gate, cfg.k, cfg.pi, out=out, causal=False)
    torch.cuda.synchronize()
    print(f"probe: 3 x bidirectional forward fwd32k", flush=True)
    dout = W.cotangent(q.shape, q.dtype, 0, dev)
    for causal in (True, False):
        y, lse = pa.pi_attn_forward(q, k, v, gate, cfg.k, cfg.pi, return_lse=True, causal=causal)
        for _ in range(3):
            pa.pi_attn_backward(q, k, v, gate, cfg.k, cfg.pi, y, lse, dout, causal=causal)
        torch.cuda.synchronize()
        print(f"probe: 3 x backward fwd32k causal={causal}", flush=True)
        del y, lse
    del q, k, v, out, dout
    scfg = W.FORWARD["smallk8k"]
    q, k, v, gate = W.forward_inputs(scfg, 0, dev)
    u, w2, b2 = W.gate_mlp_inputs(scfg, 0, dev)
    out = torch.empty_like(q)
    for _ in range(3):
        pa.pi_attn_forward(q, k, v, gate, scfg.k, scfg.pi, out=out)
    for causal in (True, False):
        for _ in range(3):
            pa.pi_attn_forward_gated(q, k, v, u, w2, b2, scfg.k, scfg.pi, out=out, causal=causal)
    torch.cuda.synchronize()
    print("probe: 3 x small-window forward, 3 x gated (causal, bidirectional) smallk8k", flush=True)
    dout = W.cotangent(q.shape, q.dtype, 0, dev)
    for causal in (True, False):
        y, lse = pa.pi_attn_forward(q, k, v, gate, scfg.k, scfg.pi, return_lse=True, causal=causal)
        for _ in range(3):
            pa.pi_attn_backward(q, k, v, gate, scfg.k, scfg.pi, y, lse, dout, causal=causal)
        torch.cuda.synchronize()
        print(f"probe: 3 x small-window backward smallk8k causal={causal}", flush=True)
        del y, lse
    del q, k, v, u, w2, out, dout
    dcfg = W.DECODE["decode"]
    kc, vc, lens, dgate = W.decode_state(dcfg, 0, dev)
    qs, ks, vs = W.decode_tokens(dcfg, 3, 1, dev)
    lbuf = [lens, torch.empty_like(lens)]
    for i in range(3):
        pa.pi_attn_decode_step(lbuf[i % 2], qs[i], ks[i], vs[i], kc, vc, dgate, dcfg.k, dcfg.pi,
                               len_out=lbuf[(i + 1) % 2])
    torch.cuda.synchronize()
    print(f"probe: 3 x decode step", flush=True)
    del kc, vc, qs, ks, vs
    src = torch.ones(COPY_PROBE_BYTES // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(f"probe: 3 x device copy of {COPY_PROBE_BYTES} bytes", flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported: a multi-GPU run of this "
              "operator is one process per GPU over its own (b, h) slice (no communication) or its own "
              "sequence shard, so one GPU's throughput is the measured figure", file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2511_10696_amd as pa
    from paper_2511_10696_amd import workloads as W

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.pmc_probe:
        pmc_probe(W, pa, torch, dev)
        return
    stream = torch.cuda.current_stream(dev)
    cfg = W.FORWARD["fwd32k"]
    q, k, v, gate = W.forward_inputs(cfg, 0, dev)
    out = torch.empty_like(q)

    # ---- causal forward (the metric) ---------------------------------------
    ms, t_wall, settle = time_launches(
        torch, lambda: pa.pi_attn_forward(q, k, v, gate, cfg.k, cfg.pi, out=out), args.steps, args.warmup, stream)
    sec = ms / 1e3
    value = cfg.B * cfg.N / sec
    cold_ms, cold_min = time_cold(torch, lambda: pa.pi_attn_forward(q, k, v, gate, cfg.k, cfg.pi, out=out),
                                  args.cold_reps, stream)
    keys, flops, nbytes = forward_algorithmic(cfg)
    digest = csrc_digest(FORWARD_SOURCES)
    roofline, roofline_mfma = roofline_of(flops, nbytes, sec, "forward_bf16_kernel<128,false,false,false>",
                                          measured_traffic(digest), measured_counters(digest, PROFILE_TRAFFIC, sec))
    host_inputs = [x.cpu() for x in (q, k, v, gate)]   # the exact bytes the kernel consumed, for the CPU baseline

    # ---- bidirectional forward, same shape ----------------------------------
    bidir = None
    if not args.no_bidirectional:
        bms, _, _ = time_launches(
            torch, lambda: pa.pi_attn_forward(q, k, v, gate, cfg.k, cfg.pi, out=out, causal=False),
            args.steps, args.warmup, stream)
        bkeys, bflops, bbytes = forward_algorithmic(cfg, causal=False)
        brl, bmf = roofline_of(bflops, bbytes, bms / 1e3, "forward_bf16_kernel<128,false,true,false>",
                               measured_traffic(digest, BIDIR_TRAFFIC),
                               measured_counters(digest, BIDIR_TRAFFIC, bms / 1e3))
        bidir = {"workload": "fwd32k bidirectional: B1 H32 N32768 D128 k512 pi1024 bf16 (window |j-t|<=k, "
                             "partners t-pi and t+pi)",
                 "steps": args.steps, "ms_per_step": round(bms, 5),
                 "query_positions_per_s": round(cfg.B * cfg.N / (bms / 1e3), 1),
                 "attended_keys_per_s": round(bkeys / (bms / 1e3), 1),
                 "roofline": brl, "roofline_mfma": bmf}
    # ---- at the same shape: dense causal attention (k = N - 1) and the
    # local window alone (pi = 0, no partner) -----------------------------------
    variants = None
    if not args.no_variants:
        variants = {}
        for name, kk, pp, steps in (("dense_causal", cfg.N - 1, 0, 5), ("local_only", cfg.k, 0, args.steps)):
            vcfg = dataclasses.replace(cfg, name=name, k=kk, pi=pp)
            vms, _, _ = time_launches(torch, lambda: pa.pi_attn_forward(q, k, v, gate, kk, pp, out=out), steps,
                                      1, stream)
            vkeys, vflops, vbytes = forward_algorithmic(vcfg)
            vrl, vmf = roofline_of(vflops, vbytes, vms / 1e3, "forward_bf16_kernel<128,false,false,false>")
            variants[name] = {"workload": f"fwd32k shape, causal, k={kk} pi={pp}", "steps": steps,
                              "ms_per_step": round(vms, 5),
                              "query_positions_per_s": round(cfg.B * cfg.N / (vms / 1e3), 1),
                              "attended_keys_per_s": round(vkeys / (vms / 1e3), 1),
                              "roofline": vrl, "roofline_mfma": vmf}
    del q, k, v, out
    torch.cuda.empty_cache()
    if variants is not None:
        for cname in ("fwd4k", "fwd16k"):
            ccfg = W.FORWARD[cname]
            cq, ck, cv, cg = W.forward_inputs(ccfg, 0, dev)
            cout = torch.empty_like(cq)
            cfn = lambda: pa.pi_attn_forward(cq, ck, cv, cg, ccfg.k, ccfg.pi, out=cout)
            cms, _, _ = time_launches(torch, cfn, args.steps, args.warmup, stream)
            ccold, ccold_min = time_cold(torch, cfn, args.cold_reps, stream)
            ckeys, cflops, cbytes = forward_algorithmic(ccfg)
            crl, cmf = roofline_of(cflops, cbytes, cms / 1e3, f"forward_bf16_kernel<{ccfg.D},false,false,false>")
            variants[cname] = {"workload": f"{cname}: causal B{ccfg.B} H{ccfg.H} N{ccfg.N} D{ccfg.D} k{ccfg.k} "
                                           f"pi{ccfg.pi} bf16", "steps": args.steps, "ms_per_step": round(cms, 5),
                               "query_positions_per_s": round(ccfg.B * ccfg.N / (cms / 1e3), 1),
                               "attended_keys_per_s": round(ckeys / (cms / 1e3), 1),
                               "roofline": crl, "roofline_mfma": cmf,
                               "cold": {"ms_per_step_median": round(ccold, 5), "ms_per_step_min": round(ccold_min, 5),
                                        "reps": args.cold_reps,
                                        "roofline_frac_median": round(cbytes / (ccold / 1e3) / 1e9 / HBM_PEAK_GBS, 4)}}
            del cq, ck, cv, cg, cout
            torch.cuda.empty_cache()

    # ---- small window (the paper's default k = 4, pi = 16) -------------------
    smallk = None
    if not args.no_smallk:
        smallk = bench_smallk(W, pa, torch, dev, stream, args.steps, args.warmup)

    # ---- one rank's share of a sequence-sharded fwd32k ----------------------
    shard = None
    if not args.no_shard:
        shard = bench_shard(cfg, W, pa, torch, dev, stream, args.steps, args.warmup)

    # ---- decode step --------------------------------------------------------
    decode = decode_host = None
    if not args.no_decode:
        dcfg = W.DECODE["decode"]
        nsteps = args.decode_steps
        kc, vc, lens, dgate = W.decode_state(dcfg, 0, dev)
        qs, ks, vs = W.decode_tokens(dcfg, nsteps, 1, dev)
        if not args.no_cpu_baseline:   # the rows the oracle's first ten steps can reach, as the GPU holds them
            L0, P = dcfg.cache_len, dcfg.pi
            decode_host = (kc[:, :, L0 - P:L0].cpu(), vc[:, :, L0 - P:L0].cpu(), qs[:10].cpu(), ks[:10].cpu(),
                           vs[:10].cpu(), dgate.cpu())
        lbuf = [lens, torch.empty_like(lens)]
        dout = torch.empty((dcfg.S, dcfg.H, dcfg.D), dtype=dcfg.dtype, device=dev)
        # settle and warm up on a scratch copy of the lengths (row cache_len is
        # rewritten by every such step); the timed loop starts from cache_len
        warm_len = [lens.clone(), torch.empty_like(lens)]
        time_launches(torch, lambda: pa.pi_attn_decode_step(warm_len[0], qs[0], ks[0], vs[0], kc, vc, dgate, dcfg.k,
                                                            dcfg.pi, len_out=warm_len[1], out=dout), 1, 3, stream)
        si = [0]

        def step():
            i = si[0]
            pa.pi_attn_decode_step(lbuf[i % 2], qs[i], ks[i], vs[i], kc, vc, dgate, dcfg.k, dcfg.pi,
                                   len_out=lbuf[(i + 1) % 2], out=dout)
            si[0] += 1
        lens0 = lens.clone()
        d0, d1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        d0.record(stream)
        for _ in range(nsteps):
            step()
        d1.record(stream)
        torch.cuda.synchronize()
        dms = d0.elapsed_time(d1) / nsteps
        # the same steps again from the same lengths, an event after each, for
        # the per-step distribution (the events add a little time per step,
        # so the mean above is taken without them)
        lbuf[0].copy_(lens0)
        si[0] = 0
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(nsteps + 1)]
        ev[0].record(stream)
        for i in range(nsteps):
            step()
            ev[i + 1].record(stream)
        torch.cuda.synchronize()
        per = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(nsteps))
        dkeys, dbytes = decode_algorithmic(dcfg, dcfg.cache_len)
        ddigest = source_digest([os.path.join(ROOT, "paper_2511_10696_amd", "csrc", f)
                                 for f in ("decode_bf16.hip", "pi_common.h", "kernels.h")])
        dtraffic = measured_traffic(ddigest, DECODE_TRAFFIC)
        dcounters = measured_counters(ddigest, DECODE_TRAFFIC, dms / 1e3)
        dgbs = dbytes / (dms / 1e3) / 1e9
        decode = {"workload": "decode S64 H32 D128 k512 pi1024 cache32768 bf16", "steps": nsteps,
                  "ms_per_step": round(dms, 5), "us_per_step": round(dms * 1e3, 2),
                  "us_per_step_p50": round(per[len(per) // 2] * 1e3, 2),
                  "us_per_step_p99": round(per[min(len(per) - 1, (99 * len(per)) // 100)] * 1e3, 2),
                  "queries_per_s": round(dcfg.S / (dms / 1e3), 1),
                  "roofline": {"bound": "hbm", "kernel": "decode_bf16_kernel<128>",
                               "achieved": round(dgbs, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                               "frac": round(dgbs / HBM_PEAK_GBS, 4), "bytes_per_step": dbytes,
                               "traffic": dtraffic, **dcounters}}
        del kc, vc, qs, ks, vs
        torch.cuda.empty_cache()

    # ---- backward -----------------------------------------------------------
    backward = backward_bidir = None
    if not args.no_backward:
        backward = bench_backward(cfg, W, pa, torch, dev, stream, args.backward_steps, True)
        if not args.no_bidirectional:
            backward_bidir = bench_backward(cfg, W, pa, torch, dev, stream, args.backward_steps, False)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(cfg, host_inputs, W.DECODE["decode"], decode_host)
    del host_inputs

    rec = {
        "metric": "pi-Attn fwd queries/s at N=32K + decode step latency; % HBM/MFMA roofline",
        "value": round(value, 1),
        "unit": "query positions/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "fwd32k: causal pi-Attention forward B1 H32 N32768 D128 k512 pi1024 bf16",
                   "B": cfg.B, "H": cfg.H, "N": cfg.N, "D": cfg.D, "k": cfg.k, "pi": cfg.pi,
                   "parallelism": "single-gpu"},
        "head_queries_per_s": round(cfg.B * cfg.H * cfg.N / sec, 1),
        "attended_keys_per_s": round(keys / sec, 1),
        "roofline": roofline,
        "roofline_mfma": roofline_mfma,
        "settle_s": round(settle, 3),
        "cold": {"ms_per_step_median": round(cold_ms, 5), "ms_per_step_min": round(cold_min, 5),
                 "reps": args.cold_reps,
                 "note": "single launches, each after a 1 GiB device fill that evicts the L2s and the "
                         "last-level cache; the headline value is the steady-state (hot) loop"},
        "device": device_info(torch, dev),
        "bidirectional": bidir,
        "variants": variants,
        "smallk": smallk,
        "sequence_shard": shard,
        "decode": decode,
        "backward": backward,
        "backward_bidirectional": backward_bidir,
        "cpu_baseline": cpu,
        "wall_s_timed": round(t_wall, 3),
    }
    print(json.dumps(rec))


def bench_smallk(W, pa, torch, dev, stream, steps, warmup):
    """The small-window gather path on smallk8k: the gated forward (gate MLP's
    last layer fused), causal and bidirectional, the forward with given
    per-head gate logits, and the backward (causal and bidirectional)."""
    cfg = W.FORWARD["smallk8k"]
    q, k, v, gate = W.forward_inputs(cfg, 0, dev)
    u, w2, b2 = W.gate_mlp_inputs(cfg, 0, dev)
    out = torch.empty_like(q)
    g = torch.empty((cfg.B, cfg.H, cfg.N), dtype=torch.float32, device=dev)
    res = {"workload": "smallk8k: B8 H16 N8192 D64 k4 pi16 bf16, gate MLP hidden width 512",
           "steps": steps}
    for name, causal, gated in (("gated", True, True), ("gated_bidirectional", False, True),
                                ("per_head_gate", True, False)):
        if gated:
            fn = lambda c=causal: pa.pi_attn_forward_gated(q, k, v, u, w2, b2, cfg.k, cfg.pi, out=out, gate_out=g,
                                                           causal=c)
        else:
            fn = lambda c=causal: pa.pi_attn_forward(q, k, v, gate, cfg.k, cfg.pi, out=out, causal=c)
        ms, _, _ = time_launches(torch, fn, steps, warmup, stream)
        keys, flops, nbytes = smallk_algorithmic(cfg, causal, gated)
        mode = "false" if causal else "true"
        rl, mf = roofline_of(flops, nbytes, ms / 1e3,
                             f"smallk_bf16_kernel<64,{mode},{'true' if gated else 'false'},4>",
                             measured_traffic(csrc_digest(SMALLK_SOURCES), SMALLK_TRAFFIC[name]),
                             measured_counters(csrc_digest(SMALLK_SOURCES), SMALLK_TRAFFIC[name], ms / 1e3))
        res[name] = {"us_per_step": round(ms * 1e3, 2),
                     "query_positions_per_s": round(cfg.B * cfg.N / (ms / 1e3), 1),
                     "attended_keys_per_s": round(keys / (ms / 1e3), 1),
                     "bytes_per_step": nbytes, "roofline": rl}
    del u, w2, out, g
    for name, causal in (("backward", True), ("backward_bidirectional", False)):
        y, lse = pa.pi_attn_forward(q, k, v, gate, cfg.k, cfg.pi, return_lse=True, causal=causal)
        dout = W.cotangent(q.shape, q.dtype, 0, dev)
        ms, _, _ = time_launches(
            torch, lambda c=causal: pa.pi_attn_backward(q, k, v, gate, cfg.k, cfg.pi, y, lse, dout, causal=c),
            steps, warmup, stream)
        keys, flops, nbytes = backward_algorithmic(cfg, causal)
        mode = "false" if causal else "true"
        rl, _ = roofline_of(flops, nbytes, ms / 1e3,
                            f"smallk_bwd_q_kernel<64,{mode},4> + smallk_bwd_kv_kernel<64,{mode},4>",
                            measured_traffic(csrc_digest(SMALLK_BWD_SOURCES), SMALLK_TRAFFIC[name]),
                            measured_counters(csrc_digest(SMALLK_BWD_SOURCES), SMALLK_TRAFFIC[name], ms / 1e3))
        res[name] = {"us_per_step": round(ms * 1e3, 2),
                     "query_positions_per_s": round(cfg.B * cfg.N / (ms / 1e3), 1),
                     "bytes_per_step": nbytes, "roofline": rl}
        del y, lse, dout
    del q, k, v
    torch.cuda.empty_cache()
    return res


def bench_shard(cfg, W, pa, torch, dev, stream, steps, warmup, nshard=8, rank=6):
    """One rank's share of the fwd32k sequence sharded ``nshard`` ways (an
    interior rank: halos on both sides), held as contiguous tensors as the
    rank would hold them: the forward over its queries with the pi halo rows
    of k/v before them, and the backward's two passes -- the query pass over
    its queries, the key pass over its keys with the query rows that reach
    them (its own and the max(k, pi) rows after them, whose lse and row terms
    a neighbour would send)."""
    q, k, v, gate = W.forward_inputs(cfg, 0, dev)
    n = cfg.N
    s0, s1 = rank * n // nshard, (rank + 1) * n // nshard
    reach = max(cfg.k, cfg.pi)
    lo = max(0, s0 - reach)              # k/v rows held by the forward and the query pass
    qhi = min(n, s1 + reach)             # query rows held by the key pass
    qs, ks, vs = (x[:, :, a:b].contiguous() for x, a, b in ((q, s0, s1), (k, lo, s1), (v, lo, s1)))
    out = torch.empty_like(qs)
    ms, _, _ = time_launches(
        torch, lambda: pa.pi_attn_forward_shard(qs, ks, vs, gate, cfg.k, cfg.pi, n, s0, lo, out=out),
        steps, warmup, stream)
    keys, flops, nbytes = shard_algorithmic(cfg, s0, s1, lo)
    rl, mf = roofline_of(flops, nbytes, ms / 1e3, "forward_bf16_kernel<128,false,false,false> (one shard)")
    res = {"workload": (f"fwd32k sequence-sharded {nshard} ways, rank {rank}'s share: queries [{s0}, {s1}), "
                        f"k/v rows [{lo}, {s1}) (its own and the pi = {cfg.pi} halo rows), B1 H32 D128 k512"),
           "steps": steps, "us_per_step": round(ms * 1e3, 2),
           "query_positions_per_s": round(cfg.B * (s1 - s0) / (ms / 1e3), 1),
           "attended_keys_per_s": round(keys / (ms / 1e3), 1), "roofline": rl, "roofline_mfma": mf}
    # backward: the forward's lse and output over the query rows the key pass
    # holds, their row terms from a query pass over the same rows (what the
    # neighbour's query pass and the halo exchange would deliver)
    kv_lo = max(0, s0 - reach)
    qh, kh, vh = (x[:, :, a:b].contiguous() for x, a, b in ((q, s0, qhi), (k, kv_lo, qhi), (v, kv_lo, qhi)))
    outh, lseh = pa.pi_attn_forward_shard(qh, kh, vh, gate, cfg.k, cfg.pi, n, s0, kv_lo, return_lse=True)
    douth = W.cotangent(qh.shape, qh.dtype, 0, dev)
    _, _, rth = pa.pi_attn_backward_shard_q(qh, kh, vh, gate, cfg.k, cfg.pi, n, s0, kv_lo, outh, lseh, douth)
    nq = s1 - s0
    out_s, lse_s, dout_s = outh[:, :, :nq].contiguous(), lseh[:, :, :nq].contiguous(), douth[:, :, :nq].contiguous()
    k_own, v_own = ks[:, :, s0 - lo:].contiguous(), vs[:, :, s0 - lo:].contiguous()

    def backward():
        pa.pi_attn_backward_shard_q(qs, ks, vs, gate, cfg.k, cfg.pi, n, s0, lo, out_s, lse_s, dout_s)
        pa.pi_attn_backward_shard_kv(qh, k_own, v_own, gate, cfg.k, cfg.pi, n, s0, s0, lseh, rth, douth)
    bms, _, _ = time_launches(torch, backward, max(1, steps // 5), 2, stream)
    res["backward"] = {"us_per_step": round(bms * 1e3, 2),
                       "note": "the query pass over the rank's queries and the key pass over its keys, one each"}
    del q, k, v, qs, ks, vs, out, qh, kh, vh, outh, lseh, douth, rth
    torch.cuda.empty_cache()
    return res


def bench_backward(cfg, W, pa, torch, dev, stream, steps, causal):
    """pi_attn_backward on the forward workload (lse from one forward call,
    a seeded dL/dy); inputs resident, settled and warmed up, then ``steps``."""
    q, k, v, gate = W.forward_inputs(cfg, 0, dev)
    out, lse = pa.pi_attn_forward(q, k, v, gate, cfg.k, cfg.pi, return_lse=True, causal=causal)
    dout = W.cotangent(q.shape, q.dtype, 0, dev)
    ms, _, _ = time_launches(
        torch, lambda: pa.pi_attn_backward(q, k, v, gate, cfg.k, cfg.pi, out, lse, dout, causal=causal),
        steps, 2, stream)
    keys, flops, nbytes = backward_algorithmic(cfg, causal)
    del q, k, v, out, dout, lse
    torch.cuda.empty_cache()
    mode = "false" if causal else "true"
    kernels = f"backward_q_bf16_kernel<128,false,{mode}> + backward_kv_bf16_kernel<128,false,{mode}>"
    rl, mf = roofline_of(flops, nbytes, ms / 1e3, kernels,
                         measured_traffic(csrc_digest(BACKWARD_SOURCES), BACKWARD_TRAFFIC[causal]),
                         measured_counters(csrc_digest(BACKWARD_SOURCES), BACKWARD_TRAFFIC[causal], ms / 1e3))
    return {"workload": ("backward of fwd32k" + ("" if causal else " bidirectional")
                         + ": B1 H32 N32768 D128 k512 pi1024 bf16 in, fp32 gradients"),
            "steps": steps, "ms_per_step": round(ms, 4), "roofline": rl, "roofline_mfma": mf}


ONE_THREAD_CHILD = """
import sys, time
import numpy as np
sys.path.insert(0, sys.argv[1])
import oracle
d = np.load(sys.argv[2])
t = time.perf_counter()
oracle.forward(d["q"], d["k"], d["v"], d["gate"], int(d["kw"]), int(d["pi"]))
print(time.perf_counter() - t)
"""


def cpu_baseline(cfg, host_inputs, dcfg=None, decode_host=None):
    """The fp64 oracle, as it stands, on the host's cores, fed host copies of
    exactly the bytes the GPU consumed: (1) the whole fwd32k forward on all
    cores, in query positions/s; (2) one (b, h) slice on one thread,
    scaled by B*H and labelled extrapolated; (3) ten consecutive decode
    steps of the decode workload on all cores, per step, over the rows each
    step's working set can reach (pi + 1 per (s, h))."""
    import subprocess
    import tempfile

    import numpy as np

    import oracle
    q, k, v, gate = host_inputs
    t = time.perf_counter()
    oracle.forward(q, k, v, gate, cfg.k, cfg.pi)
    dt = time.perf_counter() - t
    res = {"value": round(cfg.B * cfg.N / dt, 1), "unit": "query positions/s",
           "cores": oracle.num_threads(), "kind": "oracle",
           "sample": f"the whole fwd32k forward ({cfg.B * cfg.H} heads x {cfg.N} queries), fp64, {dt:.2f} s, "
                     "on a device-to-host copy of the kernel's inputs",
           "head_rows_per_s": round(cfg.B * cfg.H * cfg.N / dt, 1)}
    with tempfile.TemporaryDirectory() as td:
        path = os.path.join(td, "slice.npz")
        np.savez(path, q=q[:1, :1].float().numpy(), k=k[:1, :1].float().numpy(), v=v[:1, :1].float().numpy(),
                 gate=gate[:1].double().numpy(), kw=cfg.k, pi=cfg.pi)
        env = dict(os.environ, OMP_NUM_THREADS="1")
        r = subprocess.run([sys.executable, "-c", ONE_THREAD_CHILD, ROOT, path], env=env, capture_output=True,
                           text=True, timeout=600)
    if r.returncode == 0:
        dt1 = float(r.stdout.strip().splitlines()[-1])
        res["single_thread_extrapolated"] = {
            "value": round(cfg.N / (dt1 * cfg.B * cfg.H) * cfg.B, 1), "unit": "query positions/s", "cores": 1,
            "sample": f"one (b, h) slice of fwd32k ({cfg.N} queries) on one thread in {dt1:.2f} s, "
                      f"extrapolated to all {cfg.B * cfg.H} heads"}
    if decode_host is not None:
        k0, v0, qs, ks, vs, gate_d = decode_host
        steps = qs.shape[0]
        P = dcfg.pi
        shape = (dcfg.S, dcfg.H, P + steps, dcfg.D)
        kk = np.zeros(shape, np.float32)
        vv = np.zeros(shape, np.float32)
        kk[:, :, :P] = k0.float().numpy()
        vv[:, :, :P] = v0.float().numpy()
        per = []
        for i in range(steps):
            lens = np.full(dcfg.S, P + i, np.int32)
            t = time.perf_counter()
            oracle.decode_step(lens, qs[i], ks[i], vs[i], kk, vv, gate_d, dcfg.k, dcfg.pi)
            per.append(time.perf_counter() - t)
        us = sum(per) / steps * 1e6
        res["decode"] = {"us_per_step": round(us, 1), "queries_per_s": round(dcfg.S / (us / 1e6), 1),
                         "steps": steps, "cores": oracle.num_threads(),
                         "sample": f"{steps} consecutive steps of the decode workload from 32768 cached rows, "
                                   f"{dcfg.S} sequences x {dcfg.H} heads, fp64, over the pi + 1 rows each "
                                   "(s, h) can reach"}
    return res


if __name__ == "__main__":
    main()
