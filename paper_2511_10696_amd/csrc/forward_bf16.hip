// forward_bf16.hip -- banded MFMA forward of pi-Attention, bf16 in, fp32
// accumulate, for head dimension D = 64 or 128, causal or bidirectional.
//
// Work decomposition.  One work-group (4 wavefronts) owns a query tile of
// BM = 128 consecutive positions [t0, t0+128) of one (b, h); wavefront w owns
// the 32 queries q0 = t0 + 32w + [0, 32).  The window keys of the tile,
// [max(0, t0-k), t0+127] (bidirectional: up to t0+127+k), form a band that is
// streamed through LDS in 64-row tiles (two 32-key blocks, aligned to
// multiples of 32); each wavefront works on the blocks that meet its own band
// [q0 - k, q0 + 31] (bidirectional: [q0 - k, q0 + 31 + k]).  Two work-groups
// share a CU, so each SIMD interleaves two wavefronts.
//
// MFMA layout (v_mfma_f32_32x32x16_bf16).  Scores are computed transposed,
// S^T = K Q^T: A = 32 key rows x 16 dims read from LDS, B = Q^T kept in
// registers for the whole tile, C = 32 keys x 32 queries, so lane l holds the
// scores of query l%32 for keys 8i + 4(l/32) + j in accumulator slot 4i+j;
// the softmax row reductions are in-lane plus one exchange between the two
// halves of the wavefront.  The output is O^T = V^T P^T on the same
// instruction: B = P^T is taken straight from the score registers (slots
// 8c..8c+7 feed key chunk c, with the key order permuted inside the chunk)
// and A = V^T comes from the LDS transpose read (ds_read_b64_tr_b16) of the
// row-major value tile, with the same permutation.
//
// Tiles go from global memory straight into LDS (buffer loads with the LDS
// destination, no staging registers), the next tile while the two blocks
// of the current one are consumed, row-major.  K rows have their
// 16-byte chunks XOR-swizzled (chunk ^ (r mod chunks-per-row)): the
// fragment reads (16 lanes, 16 rows, one chunk each) hit 16 distinct groups
// of 4 banks.  V rows are padded by 64 bytes at D = 128: the transpose reads
// (4 rows, 64 bytes each per 32 lanes) then hit 64 distinct banks, whereas a
// chunk swizzle (chunk ^ 2(r mod 4), kept at D = 64, whose LDS budget has no
// room for padding) leaves them two-way conflicted when the LDS serves
// 8-byte reads 32 lanes at a time (23.9% conflict cycles by the counters at
// fwd32k, none with the padding, same time).  The global side uses buffer loads whose
// descriptor range ends at the tile's last usable row: the hardware range
// check zero-fills rows past it, and offsets are 32-bit with no per-load
// clamping or 64-bit address arithmetic.
//
// The long-range partner (Sec. 3.4, eq. Npi; Sec. 3.5, eq. online_ws): the
// partner rows of a wavefront's 32 queries are 32 consecutive rows shifted by
// pi, read straight from global memory in the layout of the query fragments.
// Its score (a per-lane dot product of the two) seeds the online softmax:
// running max = partner logit, running sum = 1, accumulator = partner value.
// The bidirectional mode scores the second partner t + pi the same way and
// seeds the state with both.
//
// Online softmax with a lazily updated maximum: a lane raises its reference
// maximum m only when a block's maximum exceeds it by more than 2^8 (exp2
// units); otherwise probabilities exp2(s - m) <= 256 are accumulated against
// the stale m, which changes nothing in exact arithmetic (numerator and
// denominator share the reference) and keeps the rescale of the accumulators
// out of the common path.
//
// Normalisation.  The value product takes the probabilities rounded to bf16,
// so the output is divided by the sum of those rounded values (accumulated
// with v_dot2c_f32_bf16, two per instruction): the weights actually applied
// to V sum to one, and a query whose attention sits on one key returns that
// key's value row exactly, whatever the rounding of its stale-maximum
// probability.  The lse, when requested, is taken from a second, fp32 sum of
// the unrounded values (a separate instantiation keeps it off the common
// path).
#include "kernels.h"
#include "pi_common.h"

namespace pi_attn {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

constexpr int WAVES = 4;
constexpr int NT = 64 * WAVES;   // threads per work-group
constexpr int BM = 32 * WAVES;   // queries per work-group
constexpr int TK = 64;           // key rows per LDS tile (two 32-key blocks)
constexpr float kTau = 8.0f;     // lazy-max threshold, log2 units

template <int D>
struct Tile {
    static constexpr int CPR = D / 8;   // 16-byte chunks per row
    static constexpr int ROW_BYTES = 2 * D;
    static constexpr int BYTES = TK * ROW_BYTES;
    // V rows: padded by 64 bytes at D = 128 (not swizzled), XOR-swizzled at D = 64
    static constexpr bool VPAD = D == 128;
    static constexpr int VROW = VPAD ? 2 * D + 64 : 2 * D;
    static constexpr int VBYTES = TK * VROW;
};

// One LDS tile buffer: 64 key rows and 64 value rows.  The kernel declares
// two of them (double buffering) as separate objects.
template <int D>
struct TileBuf {
    alignas(16) unsigned char k[Tile<D>::BYTES];
    alignas(16) unsigned char v[Tile<D>::VBYTES];
};

__device__ inline int k_swz(int row, int chunk, int cpr) { return chunk ^ (row & (cpr - 1)); }
__device__ inline int v_swz(int row, int chunk) { return chunk ^ ((row & 3) << 1); }


// Fetch tile rows [row0, row0 + TK) (counted from the window start) into
// LDS buffer tb with buffer loads that write LDS directly: 16 bytes per
// lane, the 64 lanes of one instruction filling 1 KB of consecutive LDS,
// each lane's source offset chosen so that the bytes land in the tile's
// layout.  Instruction u fills bytes [1024u, 1024u + 1024) of the K or the V
// buffer; wavefront w issues u = w, w + WAVES, ...  K: LDS chunk pc of row r
// holds global chunk k_swz(r, pc).  V: D = 128 rows are padded to VROW and
// the pad chunks take an out-of-range offset (written as zeros); D = 64 rows
// hold global chunk v_swz(r, pc) at chunk pc.  Offsets past the rows the
// descriptor covers read as zeros.
template <int D>
struct Fetch {
    static constexpr int KI = TK * Tile<D>::CPR / 64;   // instructions per K tile
    static constexpr int VU = Tile<D>::VROW / 16;       // LDS chunks per V row
    static constexpr int VI = TK * VU / 64;             // instructions per V tile
};

template <int D>
__device__ inline void tile_fetch(TileBuf<D> &tb, u32x4 rk, u32x4 rv, int rowb, int row0, int w, int lane) {
    using T = Tile<D>;
    using F = Fetch<D>;
    static_assert(F::KI % WAVES == 0 && TK * T::CPR % 64 == 0 && TK * F::VU % 64 == 0, "tile fetch shape");
#pragma unroll
    for (int u0 = 0; u0 < F::KI; u0 += WAVES) {
        const int u = u0 + w, pidx = 64 * u + lane;
        const int row = pidx / T::CPR, pc = pidx % T::CPR;
        const int off = (row0 + row) * rowb + k_swz(row, pc, T::CPR) * 16;
        lds_fetch16(rk, off, tb.k + 1024 * u);
    }
#pragma unroll
    for (int u0 = 0; u0 < F::VI; u0 += WAVES) {
        const int u = u0 + w;
        if (u < F::VI) {   // wave-uniform
            const int pidx = 64 * u + lane;
            const int row = pidx / F::VU, pc = pidx % F::VU;
            const int off = T::VPAD ? (pc < T::CPR ? (row0 + row) * rowb + pc * 16 : kOutOfRange)
                                    : (row0 + row) * rowb + v_swz(row, pc) * 16;
            lds_fetch16(rv, off, tb.v + 1024 * u);
        }
    }
}

// The value held by the other half of the wavefront (lane l ^ 32).
__device__ inline float other_half(float x) {
    const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(__lane_id() < 32 ? p[1] : p[0]);
}

__device__ inline float max16(const f32x16 &a) {
    float m0 = fmaxf(fmaxf(a[0], a[1]), a[2]), m1 = fmaxf(fmaxf(a[3], a[4]), a[5]);
    float m2 = fmaxf(fmaxf(a[6], a[7]), a[8]), m3 = fmaxf(fmaxf(a[9], a[10]), a[11]);
    float m4 = fmaxf(fmaxf(a[12], a[13]), a[14]);
    return fmaxf(fmaxf(fmaxf(m0, m1), fmaxf(m2, m3)), fmaxf(m4, a[15]));
}

// Per-wavefront state: lane (c, g) = (l % 32, l / 32) belongs to query q0 + c.
template <int D>
struct Wave {
    static constexpr int DB = D / 32;   // 32-dim output blocks
    static constexpr int KS = D / 16;   // 16-dim k-steps of the score MFMA
    bf16x8 qf[KS];                      // B operand: Q[t][16s + 8g .. +8]
    f32x16 o[DB];                       // O^T accumulators: dims 32db + 8i + 4g + j
    float m;                            // reference (lazy) maximum, log2 units
    float l;                            // this lane's part of the running sum (kept for the lse)
    float lb;                           // the same sum over the bf16-rounded probabilities
};

// s + the sum of the eight bf16 values of p.
__device__ inline float sum_bf16x8(const bf16x8 &p, float s) {
    const bf16x2 one = {(__bf16)1.0f, (__bf16)1.0f};
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(p, p, 0, 1), one, s, false);
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(p, p, 2, 3), one, s, false);
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(p, p, 4, 5), one, s, false);
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(p, p, 6, 7), one, s, false);
    return s;
}

// acc + <a, b> over eight bf16 pairs (packed products, fp32 sums).
__device__ inline float dot_bf16x8(const bf16x8 &a, const bf16x8 &b, float acc) {
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(a, a, 0, 1), __builtin_shufflevector(b, b, 0, 1),
                                          acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(a, a, 2, 3), __builtin_shufflevector(b, b, 2, 3),
                                          acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(a, a, 4, 5), __builtin_shufflevector(b, b, 4, 5),
                                          acc, false);
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(a, a, 6, 7), __builtin_shufflevector(b, b, 6, 7),
                                           acc, false);
}

// Scores of one 32-key block -> log2-unit logits (masked to -inf on edge
// blocks), running state update, and bf16 probabilities for the value product.
template <int D, bool CLAMP, bool BIDIR, bool LSE>
__device__ inline void softmax_block(Wave<D> &ws, f32x16 &s, bool edge, int j0, int t, int kw, int N, bool t_ok,
                                     float c2, float scale, float bias, float clampv, int g, bf16x8 pb[2]) {
    if constexpr (CLAMP) {
#pragma unroll
        for (int e = 0; e < 16; ++e) s[e] = fminf(fmaxf(s[e] * scale + bias, -clampv), clampv) * kLog2e;
    }
    if (edge) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int j = j0 + 8 * (e >> 2) + 4 * g + (e & 3);
            bool ok;
            if constexpr (BIDIR) {
                ok = t_ok && j < N && j - t <= kw && t - j <= kw;
            } else {
                ok = t_ok && j <= t && j >= t - kw;
            }
            s[e] = ok ? s[e] : -INFINITY;
        }
    }
    float mx = max16(s);
    mx = fmaxf(mx, other_half(mx));
    if constexpr (!CLAMP) mx *= c2;
    // Only lanes whose own maximum moved update their reference (the others
    // scale by exactly 1), so a query's result never depends on the data of
    // the other queries sharing the wavefront.
    const bool need = mx > ws.m + kTau;
    if (__builtin_amdgcn_ballot_w64(need)) {
        const float m_new = need ? mx : ws.m;
        const float alpha = need ? __builtin_amdgcn_exp2f(ws.m - m_new) : 1.0f;
        ws.m = m_new;
        if constexpr (LSE) ws.l *= alpha;
        ws.lb *= alpha;
#pragma unroll
        for (int db = 0; db < Wave<D>::DB; ++db) ws.o[db] *= alpha;
    }
    const float mu = ws.m == -INFINITY ? 0.0f : ws.m;
    float lsum = 0.0f;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            float v;
            if constexpr (CLAMP) {
                v = s[8 * c + e] - mu;
            } else {
                v = __builtin_fmaf(s[8 * c + e], c2, -mu);
            }
            const float p = __builtin_amdgcn_exp2f(v);
            if constexpr (LSE) lsum += p;
            pb[c][e] = (__bf16)p;
        }
    }
    if constexpr (LSE) ws.l += lsum;
    ws.lb = sum_bf16x8(pb[1], sum_bf16x8(pb[0], ws.lb));
}

template <int D, bool CLAMP, bool BIDIR, bool LSE>
__global__ __launch_bounds__(NT, D == 64 ? 4 : 2) void forward_bf16_kernel(FwdParams p, int n_qt, int64_t n_logical) {
    using T = Tile<D>;
    using W = Wave<D>;
    __shared__ TileBuf<D> tA, tB;
    const int64_t logical = xcd_remap(blockIdx.x, n_logical);
    if (logical < 0) return;
    const int qt = (int)(logical % n_qt);
    const int64_t bh = logical / n_qt;
    const int h = (int)(bh % p.H), b = (int)(bh / p.H);

    const int tid = threadIdx.x;
    const int lane = __lane_id();
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 5, c = lane & 31;
    const int kw = p.k, pi = p.pi;
    // absolute positions: queries [qpos0, NQ), keys and partners below NS
    const int NQ = p.qpos0 + p.N, NS = p.nseq;
    const int t0 = p.qpos0 + qt * BM;
    const int q0 = t0 + 32 * w;   // first query of this wavefront
    const int t = q0 + c;         // this lane's query
    const bool t_ok = t < NQ;

    const int64_t sn = p.sn, ksn = p.ksn;
    // row pointers indexed by absolute position (only rows held are read)
    const __bf16 *qp = (const __bf16 *)p.q + b * p.sb + h * p.sh - (int64_t)p.qpos0 * sn;
    const int64_t kvbase = b * p.ksb + h * p.ksh - (int64_t)p.kvpos0 * ksn;
    const __bf16 *kp = (const __bf16 *)p.k_ptr + kvbase;
    const __bf16 *vp = (const __bf16 *)p.v + kvbase;

    // Window tiles: rows [kb0, kend) in 64-row steps, blocks aligned to 32.
    const int kb0 = window_lo(t0, kw) & ~31;
    const int kend = min(BIDIR ? (int)min((int64_t)t0 + BM + kw, (int64_t)NS) : min(t0 + BM, NQ), p.kvend);
    const int ntiles = (kend - kb0 + TK - 1) / TK;
    // ---- prologue: every load is issued before any is waited for ----------
    // (the query fragments, the gate logit, the partner key/value rows, then
    // the first tile), so the prologue costs one memory round trip.
    // Buffer descriptors over rows [kb0, kend) of this head's keys and values.
    const int rowb = (int)(2 * ksn);
    const u32x4 rk = raw_rsrc(kp + (int64_t)kb0 * ksn, (kend - kb0) * rowb);
    const u32x4 rv = raw_rsrc(vp + (int64_t)kb0 * ksn, (kend - kb0) * rowb);

    // Loads use a clamped, always-readable row; lanes without a query or a
    // partner zero the data afterwards.
    W ws;
    const int tq = t_ok ? t : p.qpos0;
    bf16x8 qraw[W::KS];
#pragma unroll
    for (int s = 0; s < W::KS; ++s) qraw[s] = *reinterpret_cast<const bf16x8 *>(qp + tq * sn + 16 * s + 8 * g);
    const float gl = p.gate[b * p.gsb + h * p.gsh + (tq - p.qpos0) * p.gsn];

    // Partner rows: A-operand row c of the wavefront is row q0 + c - pi, the
    // partner of query q0 + c; the accumulator seed is that row's value, of
    // which lane (c, g) holds dims 32db + 8i + 4g + [0, 4).  Both rows are
    // read in the layout of the query fragments (dims 16s + 8g + [0, 8));
    // the value row is then regrouped by an exchange between the two halves
    // of the wavefront (seed_layout).
    const int prow = t - pi;
    const bool has_p = partner_enabled(kw, pi) && prow >= 0 && t_ok;   // depends on c only
    const bool any_p = __builtin_amdgcn_ballot_w64(has_p) != 0;       // wave-uniform
    const int prc = has_p ? prow : p.kvpos0;
    bf16x8 kpf[W::KS], vpf[W::KS];
    if (any_p) {
#pragma unroll
        for (int s = 0; s < W::KS; ++s) {
            kpf[s] = *reinterpret_cast<const bf16x8 *>(kp + prc * ksn + 16 * s + 8 * g);
            vpf[s] = *reinterpret_cast<const bf16x8 *>(vp + prc * ksn + 16 * s + 8 * g);
        }
    }
    // Bidirectional: the second partner t + pi, loaded the same way.
    const bool has_f = BIDIR && t_ok && partner_fwd_of(t, kw, pi, NS) >= 0;
    const bool any_f = BIDIR && __builtin_amdgcn_ballot_w64(has_f) != 0;
    const int frc = has_f ? t + pi : p.kvpos0;
    bf16x8 kff[W::KS], vff[W::KS];
    if (any_f) {
#pragma unroll
        for (int s = 0; s < W::KS; ++s) {
            kff[s] = *reinterpret_cast<const bf16x8 *>(kp + frc * ksn + 16 * s + 8 * g);
            vff[s] = *reinterpret_cast<const bf16x8 *>(vp + frc * ksn + 16 * s + 8 * g);
        }
    }
    if (ntiles > 0) tile_fetch<D>(tA, rk, rv, rowb, 0, w, lane);
#pragma unroll
    for (int s = 0; s < W::KS; ++s) ws.qf[s] = t_ok ? qraw[s] : bf16x8{};

    const FusionBias fb = fusion_bias(gl, CLAMP);
    const float c2 = p.scale * kLog2e;
    // Partner logit (log2 units) of this lane's query from the partner rows
    // kf: lane (c, g) holds dims 16s + 8g + [0, 8) of query c and of its
    // partner row, so the score is a per-lane dot product (packed bf16
    // pairs, fp32 sums) plus the other half's.
    auto partner_logit = [&](const bf16x8 (&kf)[W::KS], bool has) {
        float part = 0.0f;
#pragma unroll
        for (int s = 0; s < W::KS; ++s) part = dot_bf16x8(ws.qf[s], has ? kf[s] : bf16x8{}, part);
        const float diag = part + other_half(part);
        float sp;
        if constexpr (CLAMP) {
            sp = fminf(fmaxf(diag * p.scale + fb.partner, -p.clamp), p.clamp) * kLog2e;
        } else {
            sp = diag * c2 + fb.partner * kLog2e;
        }
        return has ? sp : -INFINITY;
    };
    // Seed: running max = the larger partner logit, running sum and
    // accumulator = the partners' weights and weighted values.
    const float sp = any_p ? partner_logit(kpf, has_p) : -INFINITY;
    const float sf = any_f ? partner_logit(kff, has_f) : -INFINITY;
    ws.m = fmaxf(sp, sf);
    const float wp = has_p ? (BIDIR ? __builtin_amdgcn_exp2f(sp - ws.m) : 1.0f) : 0.0f;
    const float wf = has_f ? __builtin_amdgcn_exp2f(sf - ws.m) : 0.0f;
    ws.l = g == 0 ? wp + wf : 0.0f;
    ws.lb = ws.l;   // the partner weights enter the accumulator unrounded
    // Lanes without that partner contribute exactly 0 (their loads read a
    // clamped row whose data is not used, not even multiplied by 0).
    // The value row in the accumulator layout: the 8-dim group m = 4db + i,
    // of which this lane needs dims 4g..4g+3, is held whole by lane
    // (c, m & 1) in vf[m >> 1]; each lane keeps its own half of its groups
    // and takes the other half from the other half of the wavefront.
    auto seed_layout = [&](const bf16x8 (&vf)[W::KS], uint2 (&vr)[W::DB][4]) {
#pragma unroll
        for (int s2 = 0; s2 < W::KS; ++s2) {
            const uint4 own = __builtin_bit_cast(uint4, vf[s2]);
            // lane g = 0 sends dims 4..7 of its group, lane g = 1 dims 0..3
            const uint2 send = g == 0 ? make_uint2(own.z, own.w) : make_uint2(own.x, own.y);
            const uint2 recv = make_uint2(__float_as_uint(other_half(__uint_as_float(send.x))),
                                          __float_as_uint(other_half(__uint_as_float(send.y))));
            const int m0 = 2 * s2, m1 = 2 * s2 + 1;
            vr[m0 >> 2][m0 & 3] = g == 0 ? make_uint2(own.x, own.y) : recv;
            vr[m1 >> 2][m1 & 3] = g == 0 ? recv : make_uint2(own.z, own.w);
        }
    };
    auto seed = [&](uint2 (&vr)[W::DB][4], float wt, bool has, bool add) {
#pragma unroll
        for (int db = 0; db < W::DB; ++db) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                if (!has) vr[db][i] = make_uint2(0, 0);
                const float e[4] = {__uint_as_float(vr[db][i].x << 16), __uint_as_float(vr[db][i].x & 0xffff0000u),
                                    __uint_as_float(vr[db][i].y << 16), __uint_as_float(vr[db][i].y & 0xffff0000u)};
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const float x = BIDIR ? wt * e[j] : e[j];   // causal: the one partner has weight 1
                    ws.o[db][4 * i + j] = add ? ws.o[db][4 * i + j] + x : x;
                }
            }
        }
    };
    uint2 vraw[W::DB][4];
    if (any_p) {
        seed_layout(vpf, vraw);
    } else {
#pragma unroll
        for (int db = 0; db < W::DB; ++db)
#pragma unroll
            for (int i = 0; i < 4; ++i) vraw[db][i] = make_uint2(0, 0);
    }
    seed(vraw, wp, has_p, false);
    if constexpr (BIDIR) {
        uint2 vfraw[W::DB][4];
        if (any_f) {
            seed_layout(vff, vfraw);
        } else {
#pragma unroll
            for (int db = 0; db < W::DB; ++db)
#pragma unroll
                for (int i = 0; i < 4; ++i) vfraw[db][i] = make_uint2(0, 0);
        }
        seed(vfraw, wf, has_f, true);
    }

    // ---- window band -------------------------------------------------------
    // One 32-key block: rows [32 blk, 32 blk + 32) of the tile at kt / vt,
    // keys [j0, j0 + 32).
    auto block = [&](const unsigned char *kt, const unsigned char *vt, int j0, int blk) {
        // Wave-uniform: does the block meet the band, is it wholly inside it?
        const bool act = BIDIR ? j0 < kend && q0 < NQ && j0 - (q0 + 31) <= kw && j0 + 31 >= q0 - kw
                               : j0 < kend && q0 < NQ && j0 <= q0 + 31 && j0 + 31 >= q0 - kw;
        if (!act) return;
        const bool edge = BIDIR ? !(j0 + 31 - q0 <= kw && q0 + 31 - j0 <= kw) || q0 + 31 >= NQ || j0 + 31 >= NS
                                : !(j0 + 31 <= q0 && j0 >= q0 + 31 - kw) || q0 + 31 >= NQ;

        // Fragment reads: the K rows (A operand of the scores) are issued
        // together ahead of the score MFMAs; the V^T reads (A operand of
        // O^T, by transpose reads) go out behind the score MFMAs and land
        // during the softmax.
        const int krow = 32 * blk + c;
        bf16x8 kf[W::KS];
#pragma unroll
        for (int s = 0; s < W::KS; ++s)
            kf[s] = *reinterpret_cast<const bf16x8 *>(kt + krow * T::ROW_BYTES + k_swz(krow, 2 * s + g, T::CPR) * 16);
        __builtin_amdgcn_sched_barrier(0);

        f32x16 sc = {};
#pragma unroll
        for (int s = 0; s < W::KS; ++s) sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[s], ws.qf[s], sc, 0, 0, 0);
        const int G = lane >> 4, r = (lane >> 2) & 3, qd = lane & 3;
        bf16x8 vf[2][W::DB];
#pragma unroll
        for (int cc = 0; cc < 2; ++cc) {
#pragma unroll
            for (int db = 0; db < W::DB; ++db) {
#pragma unroll
                for (int hh = 0; hh < 2; ++hh) {
                    const int vrow = 32 * blk + 16 * cc + 8 * hh + 4 * g + r;
                    const int chunk = 4 * db + 2 * (G & 1) + (qd >> 1);
                    const unsigned char *src =
                        T::VPAD ? vt + vrow * T::VROW + chunk * 16 + (qd & 1) * 8
                                : vt + vrow * T::ROW_BYTES + v_swz(vrow, chunk) * 16 + (qd & 1) * 8;
                    const bf16x4 y =
                        __builtin_bit_cast(bf16x4, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)src));
                    vf[cc][db][4 * hh + 0] = y[0];
                    vf[cc][db][4 * hh + 1] = y[1];
                    vf[cc][db][4 * hh + 2] = y[2];
                    vf[cc][db][4 * hh + 3] = y[3];
                }
            }
        }
        bf16x8 pb[2];
        softmax_block<D, CLAMP, BIDIR, LSE>(ws, sc, edge, j0, t, kw, NS, t_ok, c2, p.scale, fb.local, p.clamp, g, pb);
#pragma unroll
        for (int cc = 0; cc < 2; ++cc) {
#pragma unroll
            for (int db = 0; db < W::DB; ++db)
                ws.o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[cc][db], pb[cc], ws.o[db], 0, 0, 0);
        }
    };
    // Tile m (keys kb0 + 64m ..) is in buffer m mod 2.  Before its blocks a
    // wavefront waits for its own fetches of it (the only ones in flight)
    // and the barrier makes every wavefront's share visible; then tile m + 1
    // is fetched into the other buffer, which every wavefront finished
    // reading (tile m - 1) before that barrier, and lands while tile m's two
    // blocks are computed.  The fences around the barrier are LDS-scoped: a
    // work-group fence would also wait for the fetch of the next tile.
    auto tile = [&](const TileBuf<D> &cur, TileBuf<D> &ahead, int m) {
        __builtin_amdgcn_s_waitcnt(0xF70);   // vmcnt(0): this wavefront's fetches of tile m
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
        if (m + 1 < ntiles) tile_fetch<D>(ahead, rk, rv, rowb, TK * (m + 1), w, lane);
        block(cur.k, cur.v, kb0 + TK * m, 0);
        block(cur.k, cur.v, kb0 + TK * m + 32, 1);
    };
    // unrolled by two so that every fetch and every read names its buffer
    // statically
    for (int m = 0; m < ntiles; m += 2) {
        tile(tA, tB, m);
        if (m + 1 >= ntiles) break;
        tile(tB, tA, m + 1);
    }

    // ---- normalise and store -----------------------------------------------
    const float lb_tot = ws.lb + other_half(ws.lb);
    if (t_ok) {
        const float inv = 1.0f / lb_tot;
        __bf16 *op = (__bf16 *)p.out + b * p.osb + h * p.osh + (int64_t)(t - p.qpos0) * p.osn;
#pragma unroll
        for (int db = 0; db < W::DB; ++db) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                bf16x4 o4;
#pragma unroll
                for (int j = 0; j < 4; ++j) o4[j] = (__bf16)(ws.o[db][4 * i + j] * inv);
                *reinterpret_cast<bf16x4 *>(op + 32 * db + 8 * i + 4 * g) = o4;
            }
        }
        if constexpr (LSE) {
            const float l_tot = ws.l + other_half(ws.l);
            if (g == 0) p.lse[bh * p.N + (t - p.qpos0)] = (ws.m + __log2f(l_tot)) * kLn2 + fb.lse_shift;
        }
    }
}

template <int D, bool CLAMP, bool BIDIR, bool LSE>
hipError_t launch(const FwdParams &p, hipStream_t stream) {
    const int n_qt = (p.N + BM - 1) / BM;
    const int64_t n_logical = (int64_t)p.B * p.H * n_qt;
    if (n_logical == 0) return hipSuccess;
    const int64_t grid = xcd_grid(n_logical);
    return launch_kernel(forward_bf16_kernel<D, CLAMP, BIDIR, LSE>, dim3((unsigned)grid), dim3(NT), stream, p, n_qt,
                         n_logical);
}

template <int D, bool BIDIR, bool LSE>
hipError_t launch_l(const FwdParams &p, hipStream_t stream) {
    return p.clamp > 0.0f ? launch<D, true, BIDIR, LSE>(p, stream) : launch<D, false, BIDIR, LSE>(p, stream);
}

template <int D, bool BIDIR>
hipError_t launch_d(const FwdParams &p, hipStream_t stream) {
    return p.lse ? launch_l<D, BIDIR, true>(p, stream) : launch_l<D, BIDIR, false>(p, stream);
}

}  // namespace

hipError_t launch_forward_bf16(const FwdParams &p, hipStream_t stream) {
    if (p.D == 64) return p.causal ? launch_d<64, false>(p, stream) : launch_d<64, true>(p, stream);
    return p.causal ? launch_d<128, false>(p, stream) : launch_d<128, true>(p, stream);
}

}  // namespace pi_attn
