"""The C ABI on the host: the library loads, exports every entry point that
include/pi_attn.h declares, and rejects invalid arguments before touching the
GPU (none of these calls enqueues work, so they run without a GPU)."""
import ctypes
import os
import re

import pytest

import paper_2511_10696_amd as pa

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pi_attn.h")

EINVAL, EUNSUP, ESCRATCH = -1, -2, -4


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(pa.LIB_PATH):
        from paper_2511_10696_amd import build
        build.build()
    return pa.library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pi_attn_\w+)\s*\(", text)))


def test_header_declares_the_entry_points():
    assert declared_functions() == sorted(pa.EXPORTED_SYMBOLS)


def test_every_declared_symbol_is_exported(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name
        assert ctypes.cast(getattr(lib, name), ctypes.c_void_p).value


def test_strerror(lib):
    for st in (0, -1, -2, -3, -4, -99):
        assert isinstance(pa.pi_attn_strerror(st), str) and pa.pi_attn_strerror(st)


@pytest.mark.parametrize("k,pi,m", [(0, 0, 1), (4, 16, 6), (4, 4, 5), (4, 3, 5), (512, 1024, 514),
                                    (128, 256, 130), (3, 0, 4), (-1, 2, -1), (2, -1, -1)])
def test_ws_width(lib, k, pi, m):
    assert pa.pi_attn_ws_width(k, pi) == m


@pytest.mark.parametrize("k,pi,m", [(0, 0, 1), (4, 16, 11), (4, 4, 9), (4, 3, 9), (512, 1024, 1027),
                                    (0, 1, 3), (-1, 2, -1), (2, -1, -1), (1 << 30, (1 << 30) + 1, -1)])
def test_ws_width_bidirectional(lib, k, pi, m):
    assert pa.pi_attn_ws_width(k, pi, causal=False) == m


def fwd(lib, **kw):
    a = dict(dtype=1, B=1, H=2, N=256, D=64, k=32, pi=64, causal=1, q=16, kk=16, v=16, sb=32768, sh=16384,
             sn=64, gate=16, gsb=0, gsh=1, gsn=0, scale=0.125, clamp=0.0, out=16, osb=32768, osh=16384, osn=64,
             lse=None, stream=None)
    a.update(kw)
    vp = lambda x: None if x is None else ctypes.c_void_p(x)
    return lib.pi_attn_forward(a["dtype"], a["B"], a["H"], a["N"], a["D"], a["k"], a["pi"], a["causal"],
                               vp(a["q"]),
                               vp(a["kk"]), vp(a["v"]), a["sb"], a["sh"], a["sn"], vp(a["gate"]), a["gsb"],
                               a["gsh"], a["gsn"], a["scale"], a["clamp"], vp(a["out"]), a["osb"], a["osh"],
                               a["osn"], vp(a["lse"]), vp(a["stream"]))


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=7), EUNSUP), (dict(D=96), EUNSUP), (dict(D=256), EUNSUP),
    (dict(B=-1), EINVAL), (dict(N=-5), EINVAL), (dict(k=-1), EINVAL), (dict(pi=-2), EINVAL),
    (dict(q=None), EINVAL), (dict(kk=None), EINVAL), (dict(v=None), EINVAL), (dict(gate=None), EINVAL),
    (dict(out=None), EINVAL), (dict(q=24), EINVAL), (dict(out=8), EINVAL), (dict(sn=68), EINVAL),
    (dict(sn=-64), EINVAL), (dict(osn=4), EINVAL), (dict(gate=18), EINVAL), (dict(gsn=-1), EINVAL),
    (dict(scale=0.0), EINVAL), (dict(scale=-1.0), EINVAL), (dict(scale=float("inf")), EINVAL),
    (dict(scale=float("nan")), EINVAL), (dict(clamp=float("nan")), EINVAL), (dict(lse=2), EINVAL),
    (dict(dtype=0, sn=66), EINVAL),
    # bf16: one query tile's (min(k, N) + 256) key rows must span < 2 GiB
    (dict(sn=1 << 22, sh=1 << 32, sb=1 << 33, k=32), EUNSUP),
    (dict(N=1 << 16, k=1 << 16, sn=1 << 14, sh=1 << 30, sb=1 << 31), EUNSUP),
    # bidirectional: (2 min(k, N) + 256) rows
    (dict(causal=0, N=1 << 16, k=40000, sn=1 << 14, sh=1 << 30, sb=1 << 31), EUNSUP),
])
def test_forward_rejects(lib, kw, code):
    assert fwd(lib, **kw) == code


@pytest.mark.parametrize("kw", [dict(N=0), dict(B=0), dict(H=0), dict(N=0, q=None, out=None)])
def test_forward_empty_is_noop(lib, kw):
    assert fwd(lib, **kw) == 0


def gated(lib, **kw):
    a = dict(dtype=1, B=1, H=2, N=256, D=64, k=4, pi=16, causal=1, q=16, kk=16, v=16, sb=32768, sh=16384, sn=64,
             u=16, usb=256 * 64, usn=64, dh=64, w2=16, b2=16, scale=0.125, clamp=0.0, out=16, osb=32768, osh=16384,
             osn=64, lse=None, gate_out=16, stream=None)
    a.update(kw)
    vp = lambda x: None if x is None else ctypes.c_void_p(x)
    return lib.pi_attn_forward_gated(a["dtype"], a["B"], a["H"], a["N"], a["D"], a["k"], a["pi"], a["causal"],
                                     vp(a["q"]), vp(a["kk"]), vp(a["v"]), a["sb"], a["sh"], a["sn"], vp(a["u"]),
                                     a["usb"], a["usn"], a["dh"], vp(a["w2"]), vp(a["b2"]), a["scale"], a["clamp"],
                                     vp(a["out"]), a["osb"], a["osh"], a["osn"], vp(a["lse"]), vp(a["gate_out"]),
                                     vp(a["stream"]))


# every case has exactly one fault, so nothing is ever launched
@pytest.mark.parametrize("kw,code", [
    (dict(dtype=4), EUNSUP), (dict(D=32), EUNSUP), (dict(B=-1), EINVAL), (dict(k=-1), EINVAL),
    (dict(dh=0), EINVAL), (dict(dh=12), EINVAL), (dict(u=None), EINVAL), (dict(u=8), EINVAL),
    (dict(w2=None), EINVAL), (dict(w2=24), EINVAL), (dict(b2=18), EINVAL), (dict(gate_out=None), EINVAL),
    (dict(gate_out=2), EINVAL), (dict(usn=4), EINVAL), (dict(usb=-64), EINVAL), (dict(q=None), EINVAL),
    (dict(out=8), EINVAL), (dict(lse=6), EINVAL), (dict(scale=0.0), EINVAL), (dict(clamp=float("nan")), EINVAL),
    (dict(dtype=0, dh=6), EINVAL),
    (dict(causal=0, N=1 << 16, k=40000, sn=1 << 14, sh=1 << 30, sb=1 << 31), EUNSUP),
])
def test_forward_gated_rejects(lib, kw, code):
    assert gated(lib, **kw) == code


@pytest.mark.parametrize("kw", [dict(N=0), dict(H=0), dict(N=0, u=None, gate_out=None)])
def test_forward_gated_empty_is_noop(lib, kw):
    assert gated(lib, **kw) == 0


def bwd(lib, **kw):
    a = dict(dtype=1, B=1, H=2, N=256, D=64, k=32, pi=64, causal=1, q=16, kk=16, v=16, sb=32768, sh=16384,
             sn=64, gate=16, gsb=0, gsh=1, gsn=0, scale=0.125, clamp=0.0, lse=16, out=16, dout=16, osb=32768,
             osh=16384, osn=64, dq=16, dk=16, dv=16, dg=16, rt=16, stream=None)
    a.update(kw)
    vp = lambda x: None if x is None else ctypes.c_void_p(x)
    return lib.pi_attn_backward(a["dtype"], a["B"], a["H"], a["N"], a["D"], a["k"], a["pi"], a["causal"],
                                vp(a["q"]),
                                vp(a["kk"]), vp(a["v"]), a["sb"], a["sh"], a["sn"], vp(a["gate"]), a["gsb"],
                                a["gsh"], a["gsn"], a["scale"], a["clamp"], vp(a["lse"]), vp(a["out"]), vp(a["dout"]),
                                a["osb"], a["osh"], a["osn"], vp(a["dq"]), vp(a["dk"]), vp(a["dv"]),
                                vp(a["dg"]), vp(a["rt"]), vp(a["stream"]))


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=5), EUNSUP), (dict(D=32), EUNSUP), (dict(B=-1), EINVAL), (dict(k=-1), EINVAL),
    (dict(lse=None), EINVAL), (dict(out=None), EINVAL), (dict(out=8), EINVAL),
    (dict(dout=None), EINVAL), (dict(dq=None), EINVAL), (dict(dk=None), EINVAL),
    (dict(dv=None), EINVAL), (dict(dg=None), EINVAL), (dict(rt=None), EINVAL), (dict(q=None), EINVAL),
    (dict(lse=18), EINVAL), (dict(dq=20), EINVAL), (dict(dout=24), EINVAL), (dict(osn=4), EINVAL),
    (dict(scale=0.0), EINVAL), (dict(clamp=float("nan")), EINVAL), (dict(gsh=-1), EINVAL),
    (dict(causal=0, N=1 << 16, k=40000, sn=1 << 14, sh=1 << 30, sb=1 << 31), EUNSUP),
])
def test_backward_rejects(lib, kw, code):
    assert bwd(lib, **kw) == code


@pytest.mark.parametrize("kw", [dict(N=0), dict(B=0), dict(N=0, lse=None, dq=None)])
def test_backward_empty_is_noop(lib, kw):
    assert bwd(lib, **kw) == 0


def bwd_noalloc(lib, **kw):
    a = dict(dtype=1, B=1, H=2, N=256, D=64, k=32, pi=64, causal=1, q=16, kk=16, v=16, sb=32768, sh=16384,
             sn=64, gate=16, gsb=0, gsh=1, gsn=0, scale=0.125, clamp=0.0, lse=16, out=16, dout=16, osb=32768,
             osh=16384, osn=64, dq=16, dk=16, dv=16, dg=16, stream=None)
    a.update(kw)
    vp = lambda x: None if x is None else ctypes.c_void_p(x)
    return lib.pi_attn_backward_noalloc(a["dtype"], a["B"], a["H"], a["N"], a["D"], a["k"], a["pi"], a["causal"],
                                        vp(a["q"]), vp(a["kk"]), vp(a["v"]), a["sb"], a["sh"], a["sn"],
                                        vp(a["gate"]), a["gsb"], a["gsh"], a["gsn"], a["scale"], a["clamp"],
                                        vp(a["lse"]), vp(a["out"]), vp(a["dout"]), a["osb"], a["osh"], a["osn"],
                                        vp(a["dq"]), vp(a["dk"]), vp(a["dv"]), vp(a["dg"]), vp(a["stream"]))


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=5), EUNSUP), (dict(D=32), EUNSUP), (dict(B=-1), EINVAL), (dict(N=-3), EINVAL),
    (dict(k=-1), EINVAL), (dict(lse=None), EINVAL), (dict(out=8), EINVAL), (dict(dq=None), EINVAL),
    (dict(dg=None), EINVAL), (dict(dq=20), EINVAL), (dict(scale=0.0), EINVAL), (dict(gsh=-1), EINVAL),
    # B*H*N above the fixed row-term array (4194304 entries): rejected before anything else
    (dict(B=1, H=1, N=(1 << 22) + 1), ESCRATCH), (dict(B=2, H=1024, N=2049), ESCRATCH),
    (dict(B=1, H=32, N=(1 << 17) + 1, q=None), ESCRATCH),
    (dict(B=1, H=32, N=1 << 17, q=None), EINVAL),     # exactly the maximum: past the size check
])
def test_backward_noalloc_rejects(lib, kw, code):
    assert bwd_noalloc(lib, **kw) == code


@pytest.mark.parametrize("kw", [dict(N=0), dict(B=0, H=1 << 20), dict(N=0, lse=None, dq=None)])
def test_backward_noalloc_empty_is_noop(lib, kw):
    assert bwd_noalloc(lib, **kw) == 0


def shard(lib, **kw):
    # a valid-looking causal shard: queries [1024, 1536) of 4096, k/v from 512
    a = dict(dtype=1, B=1, H=2, D=64, k=128, pi=512, causal=1, nseq=4096, qpos0=1024, nq=512, kvpos0=512, nkv=1024,
             q=16, sb=65536, sh=32768, sn=64, kk=16, v=16, ksb=131072, ksh=65536, ksn=64, gate=16, gsb=0, gsh=1,
             gsn=0, scale=0.125, clamp=0.0, out=16, osb=65536, osh=32768, osn=64, lse=None, stream=None)
    a.update(kw)
    vp = lambda x: None if x is None else ctypes.c_void_p(x)
    return lib.pi_attn_forward_shard(a["dtype"], a["B"], a["H"], a["D"], a["k"], a["pi"], a["causal"], a["nseq"],
                                     a["qpos0"], a["nq"], a["kvpos0"], a["nkv"], vp(a["q"]), a["sb"], a["sh"],
                                     a["sn"], vp(a["kk"]), vp(a["v"]), a["ksb"], a["ksh"], a["ksn"], vp(a["gate"]),
                                     a["gsb"], a["gsh"], a["gsn"], a["scale"], a["clamp"], vp(a["out"]), a["osb"],
                                     a["osh"], a["osn"], vp(a["lse"]), vp(a["stream"]))


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=0), EUNSUP), (dict(D=32), EUNSUP), (dict(nseq=-1), EINVAL), (dict(qpos0=-1), EINVAL),
    (dict(nq=4000), EINVAL),                       # queries past the sequence
    (dict(kvpos0=544), EINVAL),                    # halo short of the partner t - pi of the first query
    (dict(k=600, pi=0, kvpos0=448), EINVAL),       # halo short of the 32-aligned window start (424 -> 416)
    (dict(nkv=1023), EINVAL),                      # k/v rows end before the last query
    (dict(causal=0, nkv=1535), EINVAL),            # bidirectional: k/v must reach the last query + pi (2048)
    (dict(kvpos0=3500, nkv=1000), EINVAL),         # k/v rows past the sequence
    (dict(kk=None), EINVAL), (dict(v=8), EINVAL), (dict(ksn=4), EINVAL), (dict(gate=None), EINVAL),
    (dict(q=None), EINVAL), (dict(out=8), EINVAL), (dict(scale=0.0), EINVAL), (dict(lse=2), EINVAL),
])
def test_forward_shard_rejects(lib, kw, code):
    assert shard(lib, **kw) == code


@pytest.mark.parametrize("kw", [dict(nq=0), dict(B=0), dict(H=0, q=None, kk=None)])
def test_forward_shard_empty_is_noop(lib, kw):
    assert shard(lib, **kw) == 0


def shard_q(lib, **kw):
    # a valid-looking causal query pass: queries [1024, 1536) of 4096, k/v from 512
    a = dict(dtype=1, B=1, H=2, D=64, k=128, pi=512, causal=1, nseq=4096, qpos0=1024, nq=512, kvpos0=512, nkv=1024,
             q=16, sb=65536, sh=32768, sn=64, kk=16, v=16, ksb=131072, ksh=65536, ksn=64, gate=16, gsb=0, gsh=1,
             gsn=0, scale=0.125, clamp=0.0, lse=16, out=16, dout=16, osb=65536, osh=32768, osn=64, dq=16, dg=16,
             rt=16, stream=None)
    a.update(kw)
    vp = lambda x: None if x is None else ctypes.c_void_p(x)
    return lib.pi_attn_backward_shard_q(
        a["dtype"], a["B"], a["H"], a["D"], a["k"], a["pi"], a["causal"], a["nseq"], a["qpos0"], a["nq"],
        a["kvpos0"], a["nkv"], vp(a["q"]), a["sb"], a["sh"], a["sn"], vp(a["kk"]), vp(a["v"]), a["ksb"], a["ksh"],
        a["ksn"], vp(a["gate"]), a["gsb"], a["gsh"], a["gsn"], a["scale"], a["clamp"], vp(a["lse"]), vp(a["out"]),
        vp(a["dout"]), a["osb"], a["osh"], a["osn"], vp(a["dq"]), vp(a["dg"]), vp(a["rt"]), vp(a["stream"]))


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=0), EUNSUP), (dict(kvpos0=544), EINVAL), (dict(nq=4000), EINVAL), (dict(nkv=1023), EINVAL),
    (dict(lse=None), EINVAL), (dict(out=None), EINVAL), (dict(dout=None), EINVAL), (dict(dq=None), EINVAL),
    (dict(dg=None), EINVAL), (dict(rt=None), EINVAL), (dict(dq=20), EINVAL), (dict(kk=None), EINVAL),
    (dict(gate=None), EINVAL), (dict(qpos0=-1), EINVAL),
])
def test_backward_shard_q_rejects(lib, kw, code):
    assert shard_q(lib, **kw) == code


def test_backward_shard_q_empty_is_noop(lib):
    assert shard_q(lib, nq=0) == 0


def shard_kv(lib, **kw):
    # a valid-looking causal key pass: keys [1024, 1536) of 4096, query rows [1024, 2048) held
    a = dict(dtype=1, B=1, H=2, D=64, k=128, pi=512, causal=1, nseq=4096, kpos0=1024, nk=512, qpos0=1024, nqh=1024,
             q=16, sb=131072, sh=65536, sn=64, kk=16, v=16, ksb=65536, ksh=32768, ksn=64, gate=16, gsb=0, gsh=1,
             gsn=0, scale=0.125, clamp=0.0, lse=16, rt=16, dout=16, osb=131072, osh=65536, osn=64, dk=16, dv=16,
             stream=None)
    a.update(kw)
    vp = lambda x: None if x is None else ctypes.c_void_p(x)
    return lib.pi_attn_backward_shard_kv(
        a["dtype"], a["B"], a["H"], a["D"], a["k"], a["pi"], a["causal"], a["nseq"], a["kpos0"], a["nk"],
        a["qpos0"], a["nqh"], vp(a["q"]), a["sb"], a["sh"], a["sn"], vp(a["kk"]), vp(a["v"]), a["ksb"], a["ksh"],
        a["ksn"], vp(a["gate"]), a["gsb"], a["gsh"], a["gsn"], a["scale"], a["clamp"], vp(a["lse"]), vp(a["rt"]),
        vp(a["dout"]), a["osb"], a["osh"], a["osn"], vp(a["dk"]), vp(a["dv"]), vp(a["stream"]))


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=0), EUNSUP), (dict(qpos0=1056, nqh=992), EINVAL),   # queries held start after the first key
    (dict(nqh=1023), EINVAL),                                       # short of the last key + pi
    (dict(causal=0), EINVAL),                                       # bidirectional: from the first key - pi
    (dict(nk=4000), EINVAL), (dict(kk=None), EINVAL), (dict(q=None), EINVAL), (dict(dout=None), EINVAL),
    (dict(lse=None), EINVAL), (dict(rt=None), EINVAL), (dict(dk=None), EINVAL), (dict(dv=8), EINVAL),
    (dict(gate=None), EINVAL), (dict(osn=4), EINVAL),
])
def test_backward_shard_kv_rejects(lib, kw, code):
    assert shard_kv(lib, **kw) == code


def test_backward_shard_kv_empty_is_noop(lib):
    assert shard_kv(lib, nk=0) == 0


def ggh(lib, **kw):
    a = dict(B=2, H=3, N=100, dg=16, out=16, stream=None)
    a.update(kw)
    vp = lambda x: None if x is None else ctypes.c_void_p(x)
    return lib.pi_attn_gate_grad_per_head(a["B"], a["H"], a["N"], vp(a["dg"]), vp(a["out"]), vp(a["stream"]))


@pytest.mark.parametrize("kw,code", [
    (dict(B=-1), EINVAL), (dict(H=-1), EINVAL), (dict(N=-1), EINVAL), (dict(out=None), EINVAL),
    (dict(out=2), EINVAL), (dict(dg=None), EINVAL), (dict(dg=6), EINVAL),
    (dict(B=1 << 16, H=1 << 8, N=1 << 8), EINVAL),
])
def test_gate_grad_per_head_rejects(lib, kw, code):
    assert ggh(lib, **kw) == code


@pytest.mark.parametrize("kw", [dict(H=0), dict(H=0, dg=None, out=None)])
def test_gate_grad_per_head_no_heads_is_noop(lib, kw):
    assert ggh(lib, **kw) == 0


def dec(lib, **kw):
    a = dict(dtype=1, S=2, H=2, D=128, cap=64, k=4, pi=8, len_in=64, len_out=128, q=16, kn=16, vn=16,
             kc=16, vc=16, gate=16, gss=0, gsh=1, scale=0.1, clamp=0.0, out=16, lse=None, stream=None)
    a.update(kw)
    vp = lambda x: None if x is None else ctypes.c_void_p(x)
    return lib.pi_attn_decode_step(a["dtype"], a["S"], a["H"], a["D"], a["cap"], a["k"], a["pi"],
                                   vp(a["len_in"]), vp(a["len_out"]), vp(a["q"]), vp(a["kn"]), vp(a["vn"]),
                                   vp(a["kc"]), vp(a["vc"]), vp(a["gate"]), a["gss"], a["gsh"], a["scale"],
                                   a["clamp"], vp(a["out"]), vp(a["lse"]), vp(a["stream"]))


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=3), EUNSUP), (dict(D=32), EUNSUP), (dict(S=-1), EINVAL), (dict(cap=0), EINVAL),
    (dict(k=-1), EINVAL), (dict(len_in=None), EINVAL), (dict(len_out=64), EINVAL), (dict(len_in=66), EINVAL),
    (dict(len_out=68), EINVAL), (dict(len_out=60), EINVAL),    # partial overlaps of the two [S] ranges
    (dict(q=None), EINVAL), (dict(kc=None), EINVAL), (dict(vc=8), EINVAL), (dict(out=4), EINVAL),
    (dict(gate=None), EINVAL), (dict(gsh=-1), EINVAL), (dict(scale=0.0), EINVAL), (dict(lse=1), EINVAL),
])
def test_decode_rejects(lib, kw, code):
    assert dec(lib, **kw) == code


@pytest.mark.parametrize("kw", [dict(S=0), dict(H=0)])
def test_decode_empty_is_noop(lib, kw):
    assert dec(lib, **kw) == 0


@pytest.mark.parametrize("causal", [1, 0])
def test_index_set_rejects(lib, causal):
    assert lib.pi_attn_index_set(-1, 2, 3, causal, ctypes.c_void_p(16), None) == EINVAL
    assert lib.pi_attn_index_set(5, -2, 3, causal, ctypes.c_void_p(16), None) == EINVAL
    assert lib.pi_attn_index_set(5, 2, -3, causal, ctypes.c_void_p(16), None) == EINVAL
    assert lib.pi_attn_index_set(5, 2, 3, causal, None, None) == EINVAL
    assert lib.pi_attn_index_set(5, 2, 3, causal, ctypes.c_void_p(2), None) == EINVAL
    assert lib.pi_attn_index_set(1 << 30, 8, 16, causal, ctypes.c_void_p(16), None) == EINVAL
    if not causal:   # n * (2k + 3) entries pass 2^31 where n * (k + 2) does not
        assert lib.pi_attn_index_set(1 << 27, 8, 16, causal, ctypes.c_void_p(16), None) == EINVAL
    assert lib.pi_attn_index_set(0, 2, 3, causal, None, None) == 0


def test_binding_refuses_cpu_tensors(lib):
    import torch
    q = torch.zeros(1, 1, 4, 64)
    with pytest.raises(RuntimeError, match="GPU"):
        pa.pi_attn_forward(q, q, q, torch.zeros(1), 2, 3)


def test_product_does_not_import_oracle():
    """The product package must not reach the oracle (test infrastructure)."""
    pkg = os.path.join(ROOT, "paper_2511_10696_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert not re.search(r"^\s*(import|from)\s+oracle\b", text, flags=re.M), f
                assert "pi_oracle" not in text and "liboracle" not in text, f


def test_build_rejects_scratch_users():
    """The build's spill check reads the compiler's resource remarks."""
    from paper_2511_10696_amd import build
    ok = ("x.hip:1:1: remark: Function Name: _Z1kv [-Rpass-analysis=kernel-resource-usage]\n"
          "x.hip:1:1: remark:     ScratchSize [bytes/lane]: 0 [-Rpass-analysis=kernel-resource-usage]\n")
    bad = ok.replace("_Z1kv", "_Z1jv").replace("]: 0 ", "]: 28 ")
    assert build.scratch_users(ok) == []
    assert build.scratch_users(ok + bad) == ["_Z1jv (28 bytes/lane)"]


@pytest.mark.parametrize("D", [64, 128, 1, 0, -3])
def test_default_scale(lib, D):
    """1/sqrt(D) (Sec. 3.2, eq. z), rounded to float32; 0 for D < 1."""
    import math
    import numpy as np
    got = pa.library().pi_attn_default_scale(D)
    assert got == (float(np.float32(1.0 / math.sqrt(D))) if D >= 1 else 0.0)
