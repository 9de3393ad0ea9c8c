// api.hip -- the C ABI (include/pi_attn.h): argument validation and dispatch.
// Nothing here allocates; every launch goes on the caller's stream.
#include <math.h>
#include <algorithm>
#include <mutex>
#include <stdint.h>

#include "../../include/pi_attn.h"
#include "kernels.h"
#include "pi_common.h"
#include "smallk.h"

using namespace pi_attn;

namespace {

constexpr int64_t kMaxRows = (int64_t)1 << 31;   // B*H*N (and S*H) limit

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

int elem_size(int32_t dtype) { return dtype == PI_ATTN_F32 ? 4 : dtype == PI_ATTN_BF16 ? 2 : 0; }

bool stride16(int64_t stride_elems, int es) { return stride_elems >= 0 && ((stride_elems * es) & 15) == 0; }

int from_hip(hipError_t e) { return e == hipSuccess ? PI_ATTN_OK : PI_ATTN_EHIP; }

// The bf16 kernels address the key/value rows one tile of 128 queries (or
// keys) can reach -- at most k + 256 of them, 2k + 256 bidirectional --
// with 32-bit byte offsets.
bool tile_span_ok(int32_t k, int32_t N, bool causal, int64_t sn, int es) {
    const int64_t rows = (causal ? 1 : 2) * (int64_t)std::min(k, N) + 256;
    return rows * sn * es < ((int64_t)1 << 31);
}

// Checks shared by the full-sequence calls (forward, gated forward,
// backward): dtype, sizes, head dimension, scale and clamp, the q/k/v/out
// pointers, their alignment and strides, and the bf16 tile span.  Returns a
// status; on PI_ATTN_OK, `empty` tells whether the problem has no rows (then
// nothing else is checked and the call is a no-op), and p holds the shared
// fields.
int check_sequence(int32_t dtype, int32_t B, int32_t H, int32_t N, int32_t D, int32_t k, int32_t pi, int32_t causal,
                   const void *q, const void *kk, const void *v, int64_t sb, int64_t sh, int64_t sn, float scale,
                   float logit_clamp, const void *out, int64_t osb, int64_t osh, int64_t osn, FwdParams &p,
                   bool &empty) {
    const int es = elem_size(dtype);
    empty = false;
    if (es == 0) return PI_ATTN_EUNSUPPORTED;
    if (B < 0 || H < 0 || N < 0 || k < 0 || pi < 0) return PI_ATTN_EINVAL;
    if (D != 64 && D != 128) return PI_ATTN_EUNSUPPORTED;
    if (!isfinite(scale) || scale <= 0.0f || isnan(logit_clamp)) return PI_ATTN_EINVAL;
    const int64_t rows = (int64_t)B * H * N;
    if (rows >= kMaxRows) return PI_ATTN_EINVAL;
    if (rows == 0) {
        empty = true;
        return PI_ATTN_OK;
    }
    if (!q || !kk || !v || !out) return PI_ATTN_EINVAL;
    if (!aligned16(q) || !aligned16(kk) || !aligned16(v) || !aligned16(out)) return PI_ATTN_EINVAL;
    if (!stride16(sb, es) || !stride16(sh, es) || !stride16(sn, es)) return PI_ATTN_EINVAL;
    if (!stride16(osb, es) || !stride16(osh, es) || !stride16(osn, es)) return PI_ATTN_EINVAL;
    if (dtype == PI_ATTN_BF16 && !tile_span_ok(k, N, causal != 0, sn, es)) return PI_ATTN_EUNSUPPORTED;
    p.B = B; p.H = H; p.N = N; p.D = D; p.k = k; p.pi = pi; p.causal = causal != 0;
    p.q = q; p.k_ptr = kk; p.v = v;
    p.sb = sb; p.sh = sh; p.sn = sn;
    p.scale = scale;
    p.clamp = logit_clamp > 0.0f ? logit_clamp : 0.0f;
    p.qpos0 = 0; p.kvpos0 = 0; p.kvend = N; p.nseq = N; p.qend = N;
    p.ksb = sb; p.ksh = sh; p.ksn = sn;
    return PI_ATTN_OK;
}

// Shard of a sequence of nseq positions: the queries [qpos0, qpos0 + nq)
// and k/v rows held from kvpos0 (nkv of them).  True when the rows held
// cover everything the query tiles stage or read: from the 32-aligned
// window start of the first query (and its partner t - pi) to the last query
// (causal) or max(k, pi) rows past it (bidirectional), within the sequence.
bool shard_kv_covered(int32_t k, int32_t pi, bool causal, int32_t nseq, int32_t qpos0, int32_t nq, int32_t kvpos0,
                      int32_t nkv) {
    const bool par = pi > k;
    int64_t lo = window_lo(qpos0, k) & ~31;
    if (par) lo = std::min<int64_t>(lo, std::max(0, qpos0 - pi));
    const int64_t qend = (int64_t)qpos0 + nq;
    const int64_t hi = causal ? qend : std::min<int64_t>(nseq, qend + (par ? std::max(k, pi) : k));
    return kvpos0 <= lo && (int64_t)kvpos0 + nkv >= hi;
}

// The positions of a shard call: non-negative and inside the sequence.
bool shard_positions_ok(int32_t nseq, int32_t p0, int32_t n0, int32_t p1, int32_t n1) {
    if (nseq < 0 || p0 < 0 || n0 < 0 || p1 < 0 || n1 < 0) return false;
    return (int64_t)p0 + n0 <= nseq && (int64_t)p1 + n1 <= nseq;
}

// Row terms of pi_attn_backward_noalloc: one fixed array per device in
// place of the caller's workspace.  Host code never uses its name as an
// address; the device address comes from hipGetSymbolAddress.
constexpr int64_t kScratchRows = (int64_t)1 << 22;   // float32 row terms: 16 MiB
static __device__ __align__(256) float scratch[kScratchRows];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float *g_scratch[kMaxDevices];   // address of `scratch` on each device (null until looked up)

// The address of the current device's copy of `scratch`, looked up on the
// first call on that device (with it current) and kept.
int scratch_of_current_device(float **ptr) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return PI_ATTN_EHIP;
    if (dev < 0 || dev >= kMaxDevices) return PI_ATTN_EUNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        void *addr = nullptr;
        if (hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch)) != hipSuccess || !addr) return PI_ATTN_EHIP;
        g_scratch[dev] = static_cast<float *>(addr);
    }
    *ptr = g_scratch[dev];
    return PI_ATTN_OK;
}

}  // namespace

extern "C" {

const char *pi_attn_strerror(int status) {
    switch (status) {
        case PI_ATTN_OK: return "ok";
        case PI_ATTN_EINVAL: return "invalid argument (null pointer, negative size or stride, misalignment)";
        case PI_ATTN_EUNSUPPORTED:
            return "unsupported configuration (head dimension must be 64 or 128; dtype f32/bf16; bf16: "
                   "(k + 256) rows of keys, (2k + 256) bidirectional, must span under 2 GiB)";
        case PI_ATTN_EHIP: return "HIP runtime refused the launch";
        case PI_ATTN_ESCRATCH:
            return "problem too large for the no-allocation backward's fixed row-term array (B*H*N > 4194304)";
        default: return "unknown status";
    }
}

int32_t pi_attn_ws_width(int32_t k, int32_t pi, int32_t causal) {
    if (k < 0 || pi < 0) return -1;
    const int64_t m = ws_width(k, pi, causal != 0);
    return m > INT32_MAX ? -1 : (int32_t)m;
}

float pi_attn_default_scale(int32_t D) { return D < 1 ? 0.0f : 1.0f / sqrtf((float)D); }

int pi_attn_index_set(int32_t n, int32_t k, int32_t pi, int32_t causal, int32_t *idx, void *stream) {
    if (n < 0 || k < 0 || pi < 0) return PI_ATTN_EINVAL;
    if ((int64_t)n * ws_width(k, pi, causal != 0) >= kMaxRows) return PI_ATTN_EINVAL;
    if (n == 0) return PI_ATTN_OK;
    if (!idx || !aligned4(idx)) return PI_ATTN_EINVAL;
    return from_hip(launch_index_set(n, k, pi, causal != 0, idx, (hipStream_t)stream));
}

int pi_attn_forward(int32_t dtype, int32_t B, int32_t H, int32_t N, int32_t D, int32_t k, int32_t pi,
                    int32_t causal, const void *q, const void *kk, const void *v, int64_t sb, int64_t sh, int64_t sn,
                    const float *gate, int64_t gsb, int64_t gsh, int64_t gsn, float scale, float logit_clamp,
                    void *out, int64_t osb, int64_t osh, int64_t osn, float *lse, void *stream) {
    FwdParams p{};
    bool empty;
    const int status = check_sequence(dtype, B, H, N, D, k, pi, causal, q, kk, v, sb, sh, sn, scale, logit_clamp,
                                      out, osb, osh, osn, p, empty);
    if (status != PI_ATTN_OK || empty) return status;
    if (!gate || !aligned4(gate) || gsb < 0 || gsh < 0 || gsn < 0) return PI_ATTN_EINVAL;
    if (lse && !aligned4(lse)) return PI_ATTN_EINVAL;
    p.gate = gate; p.gsb = gsb; p.gsh = gsh; p.gsn = gsn;
    p.out = out; p.osb = osb; p.osh = osh; p.osn = osn;
    p.lse = lse;
    const hipStream_t st = (hipStream_t)stream;
    if (dtype != PI_ATTN_BF16) return from_hip(launch_forward_f32(p, st));
    // a window of a few keys: the gather path; otherwise the banded MFMA path
    return from_hip(k <= kSmallK ? launch_forward_smallk(p, nullptr, st) : launch_forward_bf16(p, st));
}

int pi_attn_forward_gated(int32_t dtype, int32_t B, int32_t H, int32_t N, int32_t D, int32_t k, int32_t pi,
                          int32_t causal, const void *q, const void *kk, const void *v, int64_t sb, int64_t sh,
                          int64_t sn, const void *u, int64_t usb, int64_t usn, int32_t dh, const void *w2,
                          const float *b2, float scale, float logit_clamp, void *out, int64_t osb, int64_t osh,
                          int64_t osn, float *lse, float *gate_out, void *stream) {
    if (dh < 1) return PI_ATTN_EINVAL;
    FwdParams p{};
    bool empty;
    const int status = check_sequence(dtype, B, H, N, D, k, pi, causal, q, kk, v, sb, sh, sn, scale, logit_clamp,
                                      out, osb, osh, osn, p, empty);
    if (status != PI_ATTN_OK || empty) return status;
    const int es = elem_size(dtype);
    if (!u || !w2 || !gate_out || !aligned16(u) || !aligned16(w2)) return PI_ATTN_EINVAL;
    if (!stride16(usb, es) || !stride16(usn, es) || ((int64_t)dh * es) % 16 != 0) return PI_ATTN_EINVAL;
    if ((b2 && !aligned4(b2)) || !aligned4(gate_out) || (lse && !aligned4(lse))) return PI_ATTN_EINVAL;
    p.gate = gate_out; p.gsb = (int64_t)H * N; p.gsh = N; p.gsn = 1;   // the logits this call computes
    p.out = out; p.osb = osb; p.osh = osh; p.osn = osn;
    p.lse = lse;
    GateMlp m{};
    m.u = u; m.usb = usb; m.usn = usn; m.dh = dh; m.w2 = w2; m.b2 = b2; m.gate_out = gate_out;
    const hipStream_t st = (hipStream_t)stream;
    if (dtype == PI_ATTN_BF16 && k <= kSmallK) return from_hip(launch_forward_smallk(p, &m, st));
    // otherwise: the logits first, then the forward that reads them
    const hipError_t e = launch_gate_logits(p, m, dtype == PI_ATTN_BF16 ? 1 : 0, st);
    if (e != hipSuccess) return PI_ATTN_EHIP;
    return from_hip(dtype == PI_ATTN_BF16 ? launch_forward_bf16(p, st) : launch_forward_f32(p, st));
}

}  // extern "C"

namespace {

// Validation of pi_attn_backward's arguments other than the row-term
// workspace; fills p on PI_ATTN_OK (empty: nothing to do).
int prepare_backward(int32_t dtype, int32_t B, int32_t H, int32_t N, int32_t D, int32_t k, int32_t pi,
                     int32_t causal, const void *q, const void *kk, const void *v, int64_t sb, int64_t sh,
                     int64_t sn, const float *gate, int64_t gsb, int64_t gsh, int64_t gsn, float scale,
                     float logit_clamp, const float *lse, const void *out, const void *dout, int64_t osb, int64_t osh,
                     int64_t osn, float *dq, float *dk, float *dv, float *dgate, BwdParams &p, bool &empty) {
    FwdParams &f = p.f;
    // out shares dout's strides; it stands in for the forward output in the shared checks
    const int status = check_sequence(dtype, B, H, N, D, k, pi, causal, q, kk, v, sb, sh, sn, scale, logit_clamp,
                                      out, osb, osh, osn, f, empty);
    if (status != PI_ATTN_OK || empty) return status;
    if (!gate || !lse || !dout || !dq || !dk || !dv || !dgate) return PI_ATTN_EINVAL;
    if (!aligned16(dout) || !aligned4(gate) || gsb < 0 || gsh < 0 || gsn < 0) return PI_ATTN_EINVAL;
    if (!aligned4(lse) || !aligned16(dq) || !aligned16(dk) || !aligned16(dv) || !aligned4(dgate))
        return PI_ATTN_EINVAL;
    f.gate = gate; f.gsb = gsb; f.gsh = gsh; f.gsn = gsn;
    p.dtype = dtype == PI_ATTN_BF16 ? 1 : 0;
    p.lse = lse;
    p.out = out; p.dout = dout; p.osb = osb; p.osh = osh; p.osn = osn;
    p.dq = dq; p.dk = dk; p.dv = dv; p.dgate = dgate;
    return PI_ATTN_OK;
}

}  // namespace

extern "C" {

int pi_attn_backward(int32_t dtype, int32_t B, int32_t H, int32_t N, int32_t D, int32_t k, int32_t pi,
                     int32_t causal, const void *q, const void *kk, const void *v, int64_t sb, int64_t sh, int64_t sn,
                     const float *gate, int64_t gsb, int64_t gsh, int64_t gsn, float scale, float logit_clamp,
                     const float *lse, const void *out, const void *dout, int64_t osb, int64_t osh,
                     int64_t osn, float *dq,
                     float *dk, float *dv, float *dgate, float *rowterm, void *stream) {
    BwdParams p{};
    bool empty;
    const int status = prepare_backward(dtype, B, H, N, D, k, pi, causal, q, kk, v, sb, sh, sn, gate, gsb, gsh, gsn,
                                        scale, logit_clamp, lse, out, dout, osb, osh, osn, dq, dk, dv, dgate, p,
                                        empty);
    if (status != PI_ATTN_OK || empty) return status;
    if (!rowterm || !aligned4(rowterm)) return PI_ATTN_EINVAL;
    p.rowterm = rowterm;
    return from_hip(launch_backward(p, (hipStream_t)stream));
}

int pi_attn_backward_noalloc(int32_t dtype, int32_t B, int32_t H, int32_t N, int32_t D, int32_t k, int32_t pi,
                             int32_t causal, const void *q, const void *kk, const void *v, int64_t sb, int64_t sh,
                             int64_t sn, const float *gate, int64_t gsb, int64_t gsh, int64_t gsn, float scale,
                             float logit_clamp, const float *lse, const void *out, const void *dout, int64_t osb,
                             int64_t osh, int64_t osn, float *dq, float *dk, float *dv, float *dgate, void *stream) {
    if (B < 0 || H < 0 || N < 0) return PI_ATTN_EINVAL;
    if ((int64_t)B * H * N > kScratchRows) return PI_ATTN_ESCRATCH;
    BwdParams p{};
    bool empty;
    int status = prepare_backward(dtype, B, H, N, D, k, pi, causal, q, kk, v, sb, sh, sn, gate, gsb, gsh, gsn, scale,
                                  logit_clamp, lse, out, dout, osb, osh, osn, dq, dk, dv, dgate, p, empty);
    if (status != PI_ATTN_OK || empty) return status;
    status = scratch_of_current_device(&p.rowterm);
    if (status != PI_ATTN_OK) return status;
    // every path writes each row term before it reads it: nothing to clear
    return from_hip(launch_backward(p, (hipStream_t)stream));
}

int pi_attn_decode_step(int32_t dtype, int32_t S, int32_t H, int32_t D, int32_t cap, int32_t k, int32_t pi,
                        const int32_t *len_in, int32_t *len_out, const void *q_new, const void *k_new,
                        const void *v_new, void *k_cache, void *v_cache, const float *gate, int64_t gss,
                        int64_t gsh, float scale, float logit_clamp, void *out, float *lse, void *stream) {
    const int es = elem_size(dtype);
    if (es == 0) return PI_ATTN_EUNSUPPORTED;
    if (S < 0 || H < 0 || cap < 1 || k < 0 || pi < 0) return PI_ATTN_EINVAL;
    if (D != 64 && D != 128) return PI_ATTN_EUNSUPPORTED;
    if (!isfinite(scale) || scale <= 0.0f || isnan(logit_clamp)) return PI_ATTN_EINVAL;
    const int64_t n = (int64_t)S * H;
    if (n >= kMaxRows) return PI_ATTN_EINVAL;
    if (n == 0) return PI_ATTN_OK;
    if (!len_in || !q_new || !k_new || !v_new || !k_cache || !v_cache || !gate || !out) return PI_ATTN_EINVAL;
    if (len_out) {   // len_out must not overlap len_in: other work-groups of the step still read it
        const uintptr_t a = reinterpret_cast<uintptr_t>(len_in), b = reinterpret_cast<uintptr_t>(len_out);
        const uintptr_t bytes = (uintptr_t)S * sizeof(int32_t);
        if (a < b + bytes && b < a + bytes) return PI_ATTN_EINVAL;
    }
    if (!aligned4(len_in) || (len_out && !aligned4(len_out))) return PI_ATTN_EINVAL;
    if (!aligned16(q_new) || !aligned16(k_new) || !aligned16(v_new) || !aligned16(k_cache) ||
        !aligned16(v_cache) || !aligned16(out))
        return PI_ATTN_EINVAL;
    if (!aligned4(gate) || gss < 0 || gsh < 0) return PI_ATTN_EINVAL;
    if (lse && !aligned4(lse)) return PI_ATTN_EINVAL;

    DecodeParams p{};   // decode is causal
    p.S = S; p.H = H; p.D = D; p.cap = cap; p.k = k; p.pi = pi;
    p.len_in = len_in; p.len_out = len_out;
    p.q_new = q_new; p.k_new = k_new; p.v_new = v_new;
    p.k_cache = k_cache; p.v_cache = v_cache;
    p.gate = gate; p.gss = gss; p.gsh = gsh;
    p.scale = scale;
    p.clamp = logit_clamp > 0.0f ? logit_clamp : 0.0f;
    p.out = out; p.lse = lse;
    const hipStream_t st = (hipStream_t)stream;
    return from_hip(dtype == PI_ATTN_BF16 ? launch_decode_bf16(p, st) : launch_decode_f32(p, st));
}

int pi_attn_forward_shard(int32_t dtype, int32_t B, int32_t H, int32_t D, int32_t k, int32_t pi, int32_t causal,
                          int32_t nseq, int32_t qpos0, int32_t nq, int32_t kvpos0, int32_t nkv, const void *q,
                          int64_t sb, int64_t sh, int64_t sn, const void *kk, const void *v, int64_t ksb, int64_t ksh,
                          int64_t ksn, const float *gate, int64_t gsb, int64_t gsh, int64_t gsn, float scale,
                          float logit_clamp, void *out, int64_t osb, int64_t osh, int64_t osn, float *lse,
                          void *stream) {
    if (dtype != PI_ATTN_BF16) return PI_ATTN_EUNSUPPORTED;
    if (!shard_positions_ok(nseq, qpos0, nq, kvpos0, nkv)) return PI_ATTN_EINVAL;
    if (B < 0 || H < 0 || k < 0 || pi < 0) return PI_ATTN_EINVAL;
    if ((int64_t)B * H * nkv >= kMaxRows) return PI_ATTN_EINVAL;
    // the query checks of a whole-sequence forward over the nq query rows
    // (the k/v pointers are checked against the k/v strides below)
    FwdParams p{};
    bool empty;
    const int status = check_sequence(dtype, B, H, nq, D, k, pi, causal, q, q, q, sb, sh, sn, scale, logit_clamp, out,
                                      osb, osh, osn, p, empty);
    if (status != PI_ATTN_OK || empty) return status;
    const int es = 2;
    if (!kk || !v || !aligned16(kk) || !aligned16(v)) return PI_ATTN_EINVAL;
    if (!stride16(ksb, es) || !stride16(ksh, es) || !stride16(ksn, es)) return PI_ATTN_EINVAL;
    if (!tile_span_ok(k, nseq, causal != 0, ksn, es)) return PI_ATTN_EUNSUPPORTED;
    if (!shard_kv_covered(k, pi, causal != 0, nseq, qpos0, nq, kvpos0, nkv)) return PI_ATTN_EINVAL;
    if (!gate || !aligned4(gate) || gsb < 0 || gsh < 0 || gsn < 0) return PI_ATTN_EINVAL;
    if (lse && !aligned4(lse)) return PI_ATTN_EINVAL;
    p.k_ptr = kk; p.v = v;
    p.ksb = ksb; p.ksh = ksh; p.ksn = ksn;
    p.qpos0 = qpos0; p.kvpos0 = kvpos0; p.kvend = kvpos0 + nkv; p.nseq = nseq;
    p.gate = gate; p.gsb = gsb; p.gsh = gsh; p.gsn = gsn;
    p.out = out; p.osb = osb; p.osh = osh; p.osn = osn;
    p.lse = lse;
    return from_hip(launch_forward_bf16(p, (hipStream_t)stream));
}

int pi_attn_backward_shard_q(int32_t dtype, int32_t B, int32_t H, int32_t D, int32_t k, int32_t pi,
                             int32_t causal, int32_t nseq, int32_t qpos0, int32_t nq, int32_t kvpos0, int32_t nkv,
                             const void *q, int64_t sb, int64_t sh, int64_t sn, const void *kk, const void *v,
                             int64_t ksb, int64_t ksh, int64_t ksn, const float *gate, int64_t gsb, int64_t gsh,
                             int64_t gsn, float scale, float logit_clamp, const float *lse, const void *out,
                             const void *dout, int64_t osb, int64_t osh, int64_t osn, float *dq, float *dgate,
                             float *rowterm, void *stream) {
    if (dtype != PI_ATTN_BF16) return PI_ATTN_EUNSUPPORTED;
    if (!shard_positions_ok(nseq, qpos0, nq, kvpos0, nkv)) return PI_ATTN_EINVAL;
    if (B < 0 || H < 0 || k < 0 || pi < 0) return PI_ATTN_EINVAL;
    if ((int64_t)B * H * nkv >= kMaxRows) return PI_ATTN_EINVAL;
    BwdParams p{};
    FwdParams &f = p.f;
    bool empty;
    const int status = check_sequence(dtype, B, H, nq, D, k, pi, causal, q, q, q, sb, sh, sn, scale, logit_clamp, out,
                                      osb, osh, osn, f, empty);
    if (status != PI_ATTN_OK || empty) return status;
    if (!kk || !v || !aligned16(kk) || !aligned16(v)) return PI_ATTN_EINVAL;
    if (!stride16(ksb, 2) || !stride16(ksh, 2) || !stride16(ksn, 2)) return PI_ATTN_EINVAL;
    if (!tile_span_ok(k, nseq, causal != 0, ksn, 2)) return PI_ATTN_EUNSUPPORTED;
    if (!shard_kv_covered(k, pi, causal != 0, nseq, qpos0, nq, kvpos0, nkv)) return PI_ATTN_EINVAL;
    if (!gate || !lse || !dout || !dq || !dgate || !rowterm) return PI_ATTN_EINVAL;
    if (!aligned16(dout) || !aligned4(gate) || gsb < 0 || gsh < 0 || gsn < 0) return PI_ATTN_EINVAL;
    if (!aligned4(lse) || !aligned16(dq) || !aligned4(dgate) || !aligned4(rowterm)) return PI_ATTN_EINVAL;
    f.k_ptr = kk; f.v = v;
    f.ksb = ksb; f.ksh = ksh; f.ksn = ksn;
    f.qpos0 = qpos0; f.kvpos0 = kvpos0; f.kvend = kvpos0 + nkv; f.nseq = nseq; f.qend = qpos0 + nq;
    f.gate = gate; f.gsb = gsb; f.gsh = gsh; f.gsn = gsn;
    p.dtype = 1;
    p.lse = lse;
    p.out = out; p.dout = dout; p.osb = osb; p.osh = osh; p.osn = osn;
    p.dq = dq; p.dgate = dgate; p.rowterm = rowterm;
    return from_hip(launch_backward_q_bf16(p, (hipStream_t)stream));
}

int pi_attn_backward_shard_kv(int32_t dtype, int32_t B, int32_t H, int32_t D, int32_t k, int32_t pi,
                              int32_t causal, int32_t nseq, int32_t kpos0, int32_t nk, int32_t qpos0, int32_t nqh,
                              const void *q, int64_t sb, int64_t sh, int64_t sn, const void *kk, const void *v,
                              int64_t ksb, int64_t ksh, int64_t ksn, const float *gate, int64_t gsb, int64_t gsh,
                              int64_t gsn, float scale, float logit_clamp, const float *lse, const float *rowterm,
                              const void *dout, int64_t osb, int64_t osh, int64_t osn, float *dk, float *dv,
                              void *stream) {
    if (dtype != PI_ATTN_BF16) return PI_ATTN_EUNSUPPORTED;
    if (!shard_positions_ok(nseq, kpos0, nk, qpos0, nqh)) return PI_ATTN_EINVAL;
    if (B < 0 || H < 0 || k < 0 || pi < 0) return PI_ATTN_EINVAL;
    if ((int64_t)B * H * nqh >= kMaxRows) return PI_ATTN_EINVAL;
    // the keys' checks through the whole-sequence ones over the nk key rows
    // (their strides and pointers; q and dL/dy are checked below)
    BwdParams p{};
    FwdParams &f = p.f;
    bool empty;
    const int status = check_sequence(dtype, B, H, nk, D, k, pi, causal, kk, kk, v, ksb, ksh, ksn, scale,
                                      logit_clamp, kk, ksb, ksh, ksn, f, empty);
    if (status != PI_ATTN_OK || empty) return status;
    if (!q || !dout || !aligned16(q) || !aligned16(dout)) return PI_ATTN_EINVAL;
    if (!stride16(sb, 2) || !stride16(sh, 2) || !stride16(sn, 2)) return PI_ATTN_EINVAL;
    if (!stride16(osb, 2) || !stride16(osh, 2) || !stride16(osn, 2)) return PI_ATTN_EINVAL;
    if (!tile_span_ok(k, nseq, causal != 0, sn, 2) || !tile_span_ok(k, nseq, causal != 0, osn, 2))
        return PI_ATTN_EUNSUPPORTED;
    // the query rows held must include every query whose working set holds
    // one of the keys: from max(k, pi) rows before the first key
    // (bidirectional; the keys themselves when causal) to max(k, pi) rows
    // past the last one (k when pi <= k), within the sequence
    const int reach = pi > k ? std::max(k, pi) : k;
    const int64_t lo = causal ? kpos0 : std::max(0, kpos0 - reach);
    const int64_t hi = std::min<int64_t>(nseq, (int64_t)kpos0 + nk + reach);
    if (qpos0 > lo || (int64_t)qpos0 + nqh < hi) return PI_ATTN_EINVAL;
    if (!gate || !lse || !rowterm || !dk || !dv) return PI_ATTN_EINVAL;
    if (!aligned4(gate) || gsb < 0 || gsh < 0 || gsn < 0) return PI_ATTN_EINVAL;
    if (!aligned4(lse) || !aligned4(rowterm) || !aligned16(dk) || !aligned16(dv)) return PI_ATTN_EINVAL;
    f.q = q; f.sb = sb; f.sh = sh; f.sn = sn;
    f.k_ptr = kk; f.v = v; f.ksb = ksb; f.ksh = ksh; f.ksn = ksn;
    f.qpos0 = qpos0; f.kvpos0 = kpos0; f.kvend = kpos0 + nk; f.nseq = nseq; f.qend = qpos0 + nqh;
    f.gate = gate; f.gsb = gsb; f.gsh = gsh; f.gsn = gsn;
    p.dtype = 1;
    p.lse = lse;
    p.dout = dout; p.osb = osb; p.osh = osh; p.osn = osn;
    p.dk = dk; p.dv = dv; p.rowterm = const_cast<float *>(rowterm);
    return from_hip(launch_backward_kv_bf16(p, (hipStream_t)stream));
}

int pi_attn_gate_grad_per_head(int32_t B, int32_t H, int32_t N, const float *dgate, float *out, void *stream) {
    if (B < 0 || H < 0 || N < 0) return PI_ATTN_EINVAL;
    if ((int64_t)B * H * N >= kMaxRows) return PI_ATTN_EINVAL;
    if (H == 0) return PI_ATTN_OK;
    if (!out || !aligned4(out)) return PI_ATTN_EINVAL;
    if ((int64_t)B * N > 0 && (!dgate || !aligned4(dgate))) return PI_ATTN_EINVAL;
    return from_hip(launch_gate_grad_per_head(B, H, N, dgate, out, (hipStream_t)stream));
}

}  // extern "C"
