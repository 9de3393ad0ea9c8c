// backward_bf16.hip -- MFMA query pass of the backward for bf16 inputs:
// dq and the per-query gate gradient (D = 64 or 128), fp32 accumulation.
//
// Same decomposition and operand layouts as the bf16 forward: a work-group
// of 4 wavefronts owns 128 queries of one (b, h), wavefront w the 32 queries
// q0 = t0 + 32w + [0, 32); the window keys stream through LDS in 64-row
// tiles.  Per 32-key block, on v_mfma_f32_32x32x16_bf16:
//   S^T  = K Q^T        A = K rows (LDS), B = Q^T (registers)
//   dP^T = V dO^T       A = V rows (LDS), B = dO^T (registers)
// which land in the same accumulator layout (lane l: query l%32, keys
// 8i + 4(l/32) + j at slot 4i + j).  The weights come back from the
// forward's lse, alpha^ = exp(delta - lse), and
//   dS^T = alpha^ (dP^T - r_t)     (softmax Jacobian, Sec. 3.5 eq. jac)
// with r_t = <dL/dy_t, y_t> from the forward output (two lanes per query,
// each with half the dims of dL/dy_t and y_t); dS^T, rounded to bf16, is
// the B operand of
//   dQ^T += K^T dS^T    A = K^T by LDS transpose reads of the key tile
// with the key order permuted inside each 16-key chunk exactly as the
// forward permutes V^T against P^T.  The gate gradient
// sum_j dS_tj d(log omega_tj)/dg (eqs. ddelta_da, dalpha_da) nearly cancels
// between window and partner, so it is formed at the end from the exact
// row term r* = sum_j alpha^_tj dP_tj accumulated along the way (the r_t
// used for dS comes from the bf16-rounded forward output): with
// A = sum alpha^ dP and B = sum alpha^ over the unclamped entries of each
// prior, dg = sum_prior d(log omega)/dg (A - r* B).  r* is also written out
// as the row term of the key pass.  The partner
// row (Sec. 3.4, eq. Npi) is read straight from global memory in the layout
// of the query fragments, and its score and dP are per-lane dot products
// (then the other half's), as in the forward; the bidirectional mode
// (window |j - t| <= k, band up to t0 + 127 + k) adds the second partner
// t + pi the same way.
//
// Tiles go from global memory straight into LDS (buffer loads with the LDS
// destination, range-checked so that rows past the query tile's last usable
// row read as zeros), the next tile while the two blocks of the current one
// are consumed.  The key tile is read both as rows and by transpose reads:
// its rows are padded by 64 bytes and the low two bits of a row's 16-byte
// chunk index are XORed with bits 2-3 of the row, which keeps both patterns
// free of bank conflicts; the value tile, read as rows only, has rows padded
// by 16 bytes.
#include "kernels.h"
#include "pi_common.h"

namespace pi_attn {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

constexpr int WAVES = 4;
constexpr int NT = 64 * WAVES;
constexpr int BM = 32 * WAVES;
constexpr int TK = 64;

template <int D>
struct Tile {
    static constexpr int CPR = D / 8;         // 16-byte chunks per row
    static constexpr int KROW = 2 * D + 64;   // key-tile LDS row stride (bytes)
    static constexpr int VROW = 2 * D + 16;   // value-tile LDS row stride (bytes)
    static constexpr int KS = D / 16;         // k-steps of the score products
    static constexpr int DB = D / 32;         // 32-dim output blocks
};

template <int D>
struct TileBuf {
    alignas(16) unsigned char k[TK * Tile<D>::KROW];
    alignas(16) unsigned char v[TK * Tile<D>::VROW];
};

// Key-tile chunk swizzle: chunk pc of row r sits at chunk pc ^ chunk_x(r).
__device__ inline int chunk_x(int row) { return (row >> 2) & 3; }

// Fetch tile rows [row0, row0 + TK) (counted from the window start) into
// LDS buffer tb: instruction u of a tensor fills bytes [1024u, 1024u + 1024)
// of its buffer, 16 bytes per lane, each lane's source chosen so that the
// bytes land in the tile's layout (pad chunks take an out-of-range offset
// and are written as zeros); wavefront w issues u = w, w + WAVES, ...
template <int D>
__device__ inline void tile_fetch(TileBuf<D> &tb, u32x4 rk, u32x4 rv, int rowb, int row0, int w, int lane) {
    using T = Tile<D>;
    constexpr int KU = T::KROW / 16, VU = T::VROW / 16;   // LDS chunks per row
    constexpr int KI = TK * KU / 64, VI = TK * VU / 64;   // instructions per tile
    static_assert(TK * KU % 64 == 0 && TK * VU % 64 == 0, "tile fetch shape");
#pragma unroll
    for (int u0 = 0; u0 < KI; u0 += WAVES) {
        const int u = u0 + w;
        if (u < KI) {   // wave-uniform
            const int pidx = 64 * u + lane, row = pidx / KU, pc = pidx % KU;
            const int off = pc < T::CPR ? (row0 + row) * rowb + (pc ^ chunk_x(row)) * 16 : kOutOfRange;
            lds_fetch16(rk, off, tb.k + 1024 * u);
        }
    }
#pragma unroll
    for (int u0 = 0; u0 < VI; u0 += WAVES) {
        const int u = u0 + w;
        if (u < VI) {
            const int pidx = 64 * u + lane, row = pidx / VU, pc = pidx % VU;
            const int off = pc < T::CPR ? (row0 + row) * rowb + pc * 16 : kOutOfRange;
            lds_fetch16(rv, off, tb.v + 1024 * u);
        }
    }
}

__device__ inline float other_half(float x) {
    const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(__lane_id() < 32 ? p[1] : p[0]);
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

// Row fragments (A operand, row l%32, dims 16s + 8(l/32)) of 32-row block
// `blk` of the value tile ...
template <int D>
__device__ inline void read_vrows(bf16x8 f[Tile<D>::KS], const unsigned char *tile, int blk, int c, int g) {
    const unsigned char *base = tile + (32 * blk + c) * Tile<D>::VROW + 16 * g;
#pragma unroll
    for (int s = 0; s < Tile<D>::KS; ++s) f[s] = *reinterpret_cast<const bf16x8 *>(base + 32 * s);
}

// ... and of the key tile: chunk (2s + g) ^ x = 2(s ^ (x >> 1)) + (g ^ (x & 1)),
// x = chunk_x(row), so even and odd k-steps have one base each.
template <int D>
__device__ inline void read_krows(bf16x8 f[Tile<D>::KS], const unsigned char *tile, int blk, int c, int g) {
    const int row = 32 * blk + c, x = chunk_x(row);
    const int rb = row * Tile<D>::KROW + 16 * (g ^ (x & 1));
    const int rbo[2] = {rb + 32 * (x >> 1), rb - 32 * (x >> 1)};
#pragma unroll
    for (int s = 0; s < Tile<D>::KS; ++s) f[s] = *reinterpret_cast<const bf16x8 *>(tile + rbo[s & 1] + 32 * s);
}

// Transposed fragments (A operand: dim 32db + l%32, keys 16cc + {4g..4g+3,
// 8+4g..8+4g+3}) of 32-row block `blk` of the key tile by LDS transpose
// reads: rows 32 blk + 4g + r + 8hh + 16cc, whose chunk_x is g + 2hh.
template <int D>
__device__ inline void read_cols(bf16x8 f[2][Tile<D>::DB], const unsigned char *tile, int blk, int lane) {
    const int g = lane >> 5, G = lane >> 4, r = (lane >> 2) & 3, qd = lane & 3;
    const int jq = 2 * (G & 1) + (qd >> 1);
    const int toff[2] = {(32 * blk + 4 * g + r) * Tile<D>::KROW + 16 * (jq ^ g) + (qd & 1) * 8,
                         (32 * blk + 4 * g + r + 8) * Tile<D>::KROW + 16 * (jq ^ (g + 2)) + (qd & 1) * 8};
#pragma unroll
    for (int cc = 0; cc < 2; ++cc) {
#pragma unroll
        for (int db = 0; db < Tile<D>::DB; ++db) {
#pragma unroll
            for (int hh = 0; hh < 2; ++hh) {
                const unsigned char *src = tile + toff[hh] + 16 * cc * Tile<D>::KROW + 64 * db;
                const bf16x4 y = __builtin_bit_cast(bf16x4, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)src));
                f[cc][db][4 * hh + 0] = y[0];
                f[cc][db][4 * hh + 1] = y[1];
                f[cc][db][4 * hh + 2] = y[2];
                f[cc][db][4 * hh + 3] = y[3];
            }
        }
    }
}

template <int D, bool CLAMP, bool BIDIR>
__global__ __launch_bounds__(NT, 2) void backward_q_bf16_kernel(BwdParams bp, int n_qt, int64_t n_logical) {
    using T = Tile<D>;
    constexpr int KS = T::KS, DB = T::DB;
    const FwdParams &p = bp.f;
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
    const int N = p.N, kw = p.k, pi = p.pi;
    // absolute positions: queries [qpos0, NQ), keys and partners below NS
    const int NQ = p.qpos0 + N, NS = p.nseq;
    const int t0 = p.qpos0 + qt * BM;
    const int q0 = t0 + 32 * w;
    const int t = q0 + c;
    const bool t_ok = t < NQ;
    const int tq = t_ok ? t : p.qpos0;
    const int64_t row = bh * N + (tq - p.qpos0);

    // row pointers indexed by absolute position (only rows held are read)
    const int64_t sn = p.sn, ksn = p.ksn;
    const __bf16 *qp = (const __bf16 *)p.q + b * p.sb + h * p.sh - (int64_t)p.qpos0 * sn;
    const int64_t kvbase = b * p.ksb + h * p.ksh - (int64_t)p.kvpos0 * ksn;
    const __bf16 *kp = (const __bf16 *)p.k_ptr + kvbase;
    const __bf16 *vp = (const __bf16 *)p.v + kvbase;
    const __bf16 *op = (const __bf16 *)bp.dout + b * bp.osb + h * bp.osh - (int64_t)p.qpos0 * bp.osn;

    const int kb0 = window_lo(t0, kw) & ~31;
    const int kend = min(BIDIR ? (int)min((int64_t)t0 + BM + kw, (int64_t)NS) : min(t0 + BM, NQ), p.kvend);
    const int ntiles = (kend - kb0 + TK - 1) / TK;
    const int rowb = (int)(2 * ksn);
    const u32x4 rk = raw_rsrc(kp + (int64_t)kb0 * ksn, (kend - kb0) * rowb);
    const u32x4 rv = raw_rsrc(vp + (int64_t)kb0 * ksn, (kend - kb0) * rowb);
    if (ntiles > 0) tile_fetch<D>(tA, rk, rv, rowb, 0, w, lane);

    // Query and dL/dy rows as B operands (lanes without a query hold zeros).
    bf16x8 qf[KS], of[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        const bf16x8 qv = *reinterpret_cast<const bf16x8 *>(qp + tq * sn + 16 * s + 8 * g);
        const bf16x8 ov = *reinterpret_cast<const bf16x8 *>(op + tq * bp.osn + 16 * s + 8 * g);
        qf[s] = t_ok ? qv : bf16x8{};
        of[s] = t_ok ? ov : bf16x8{};
    }
    const float gl = p.gate[b * p.gsb + h * p.gsh + (tq - p.qpos0) * p.gsn];
    const FusionBias fb = fusion_bias(gl, CLAMP);
    // r_t = <dL/dy_t, y_t>: this lane's dims 16s + 8g + [0, 8), then the pair
    const __bf16 *yp = (const __bf16 *)bp.out + b * bp.osb + h * bp.osh - (int64_t)p.qpos0 * bp.osn;
    float rpart = 0.0f;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        const bf16x8 yv = *reinterpret_cast<const bf16x8 *>(yp + tq * bp.osn + 16 * s + 8 * g);
#pragma unroll
        for (int e = 0; e < 8; ++e) rpart += (float)of[s][e] * (float)yv[e];
    }
    const float r = rpart + other_half(rpart);
    const float lse = bp.lse[row];
    // alpha^ = exp2(delta * log2e - lse2), delta with the biases of fb
    const float lse2 = (lse - fb.lse_shift) * kLog2e;
    const float c2 = p.scale * kLog2e;
    const float ga = 1.0f / (1.0f + __expf(-gl));
    const float gat = kGateEps + (1.0f - 2.0f * kGateEps) * ga;
    const float gcoef = (1.0f - 2.0f * kGateEps) * ga * (1.0f - ga);
    const float dlog_local = gcoef / gat, dlog_partner = -gcoef / (1.0f - gat);

    f32x16 dq[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) dq[db] = f32x16{};
    // exact row term and per-prior sums for the gate gradient
    float r_all = 0.0f, a_loc = 0.0f, b_loc = 0.0f, a_par = 0.0f, b_par = 0.0f;

    // ---- partners: scores and dP of the partner rows ------------------------
    // Partner row prow of this lane's query (has_p: it exists).
    auto partner = [&](int prow, bool has_p) __attribute__((always_inline)) {
        if (__builtin_amdgcn_ballot_w64(has_p) == 0) return;
        const int prc = has_p ? prow : p.kvpos0;
        bf16x8 kpf[KS], vpf[KS];
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            kpf[s] = *reinterpret_cast<const bf16x8 *>(kp + prc * ksn + 16 * s + 8 * g);
            vpf[s] = *reinterpret_cast<const bf16x8 *>(vp + prc * ksn + 16 * s + 8 * g);
        }
        // score and dP of the partner: per-lane dot products of the query and
        // dL/dy fragments with the partner rows (same layout), then the pair
        float sa = 0.0f, da = 0.0f;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            sa = dot_bf16x8(qf[s], has_p ? kpf[s] : bf16x8{}, sa);
            da = dot_bf16x8(of[s], has_p ? vpf[s] : bf16x8{}, da);
        }
        const float sd = sa + other_half(sa), dpd = da + other_half(da);
        float delta2;
        bool cut = false;
        if constexpr (CLAMP) {
            const float dl = fminf(fmaxf(sd * p.scale + fb.partner, -p.clamp), p.clamp);
            cut = fabsf(dl) >= p.clamp;
            delta2 = dl * kLog2e;
        } else {
            delta2 = sd * c2 + fb.partner * kLog2e;
        }
        const float wgt = has_p ? __builtin_amdgcn_exp2f(delta2 - lse2) : 0.0f;
        const float dd = cut ? 0.0f : wgt * (dpd - r);
        if (g == 0) {   // one lane of the pair counts the partner
            r_all += wgt * dpd;
            a_par += cut ? 0.0f : wgt * dpd;
            b_par += cut ? 0.0f : wgt;
        }
        // dq += dd * k_p over this lane's dims 32db + 8i + 4g + [0, 4): the
        // 8-dim group m = 4db + i, whose half 4g..4g+3 this lane needs, is
        // held whole by lane (c, m & 1) in kpf[m >> 1]; each lane keeps its
        // own half of its groups and takes the other half from the other
        // half of the wavefront
        const auto kh = [&](int s2) { return __builtin_bit_cast(uint4, has_p ? kpf[s2] : bf16x8{}); };
#pragma unroll
        for (int s2 = 0; s2 < KS; ++s2) {
            const uint4 own = kh(s2);
            // lane g = 0 sends dims 4..7 of its group, lane g = 1 dims 0..3
            const uint2 send = g == 0 ? make_uint2(own.z, own.w) : make_uint2(own.x, own.y);
            const uint2 recv = make_uint2(__float_as_uint(other_half(__uint_as_float(send.x))),
                                          __float_as_uint(other_half(__uint_as_float(send.y))));
            // groups 2 s2 (held by g = 0) and 2 s2 + 1 (held by g = 1)
            const uint2 lo = g == 0 ? make_uint2(own.x, own.y) : recv;   // group 2 s2, dims 4g..4g+3
            const uint2 hi = g == 0 ? recv : make_uint2(own.z, own.w);   // group 2 s2 + 1
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                const int m = 2 * s2 + half;
                const uint2 raw = half ? hi : lo;
                const int db = m >> 2, i = m & 3;
                dq[db][4 * i + 0] += dd * __uint_as_float(raw.x << 16);
                dq[db][4 * i + 1] += dd * __uint_as_float(raw.x & 0xffff0000u);
                dq[db][4 * i + 2] += dd * __uint_as_float(raw.y << 16);
                dq[db][4 * i + 3] += dd * __uint_as_float(raw.y & 0xffff0000u);
            }
        }
    };
    partner(t - pi, partner_enabled(kw, pi) && t - pi >= 0 && t_ok);
    if constexpr (BIDIR) partner(t + pi, t_ok && partner_fwd_of(t, kw, pi, NS) >= 0);

    // ---- window band ---------------------------------------------------------
    auto block = [&](const TileBuf<D> &tb, int j0, int blk) __attribute__((always_inline)) {
        const bool act = BIDIR ? j0 < kend && q0 < NQ && j0 - (q0 + 31) <= kw && j0 + 31 >= q0 - kw
                               : j0 < kend && q0 < NQ && j0 <= q0 + 31 && j0 + 31 >= q0 - kw;
        if (!act) return;
        const bool edge = BIDIR ? !(j0 + 31 - q0 <= kw && q0 + 31 - j0 <= kw) || q0 + 31 >= NQ || j0 + 31 >= NS
                                : !(j0 + 31 <= q0 && j0 >= q0 + 31 - kw) || q0 + 31 >= NQ;
        bf16x8 f[KS];
        read_krows<D>(f, tb.k, blk, c, g);
        f32x16 sc = {};
#pragma unroll
        for (int s = 0; s < KS; ++s) sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[s], qf[s], sc, 0, 0, 0);
        read_vrows<D>(f, tb.v, blk, c, g);
        f32x16 dp = {};
#pragma unroll
        for (int s = 0; s < KS; ++s) dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[s], of[s], dp, 0, 0, 0);
        bf16x8 kt[2][DB];
        float ds[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            float delta2;
            bool cut = false;
            if constexpr (CLAMP) {
                const float dl = fminf(fmaxf(sc[e] * p.scale + fb.local, -p.clamp), p.clamp);
                cut = fabsf(dl) >= p.clamp;
                delta2 = dl * kLog2e;
            } else {
                delta2 = sc[e] * c2;
            }
            if (edge) {
                const int j = j0 + 8 * (e >> 2) + 4 * g + (e & 3);
                const bool ok = BIDIR ? t_ok & (j < NS) & (j - t <= kw) & (t - j <= kw) : t_ok & (j <= t) & (j >= t - kw);
                delta2 = ok ? delta2 : -INFINITY;
            }
            const float wgt = __builtin_amdgcn_exp2f(delta2 - lse2);
            const float pd = wgt * dp[e];
            ds[e] = cut ? 0.0f : pd - wgt * r;
            r_all += pd;
            a_loc += cut ? 0.0f : pd;
            b_loc += cut ? 0.0f : wgt;
        }
        read_cols<D>(kt, tb.k, blk, lane);
        bf16x8 dsb[2];
#pragma unroll
        for (int cc = 0; cc < 2; ++cc)
#pragma unroll
            for (int e = 0; e < 8; ++e) dsb[cc][e] = (__bf16)ds[8 * cc + e];
#pragma unroll
        for (int cc = 0; cc < 2; ++cc)
#pragma unroll
            for (int db = 0; db < DB; ++db)
                dq[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kt[cc][db], dsb[cc], dq[db], 0, 0, 0);
    };
    // Tile m (keys kb0 + 64m ..) is in buffer m mod 2.  A wavefront waits
    // for its own fetches of it (the only vector-memory operations in flight
    // here), the barrier makes every wavefront's share visible, and tile
    // m + 1 then goes into the other buffer (last read for tile m - 1,
    // before that barrier).  LDS-scoped fences: a work-group fence would
    // also wait for the fetch of the next tile.
    auto tile = [&](const TileBuf<D> &cur, TileBuf<D> &ahead, int m) __attribute__((always_inline)) {
        __builtin_amdgcn_s_waitcnt(0xF70);   // vmcnt(0)
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
        if (m + 1 < ntiles) tile_fetch<D>(ahead, rk, rv, rowb, TK * (m + 1), w, lane);
        block(cur, kb0 + TK * m, 0);
        block(cur, kb0 + TK * m + 32, 1);
    };
    // unrolled by two so that every fetch and every read names its buffer
    // statically
    for (int m = 0; m < ntiles; m += 2) {
        tile(tA, tB, m);
        if (m + 1 >= ntiles) break;
        tile(tB, tA, m + 1);
    }

    // ---- store ---------------------------------------------------------------
    const float rs = r_all + other_half(r_all);
    const float al = a_loc + other_half(a_loc), bl = b_loc + other_half(b_loc);
    const float ap = a_par + other_half(a_par), bpar = b_par + other_half(b_par);
    const float dg_tot = dlog_local * (al - rs * bl) + dlog_partner * (ap - rs * bpar);
    if (t_ok) {
        float *dqp = bp.dq + row * D;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                f32x4 o;
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) o[jj] = dq[db][4 * i + jj] * p.scale;
                *reinterpret_cast<f32x4 *>(dqp + 32 * db + 8 * i + 4 * g) = o;
            }
        }
        if (g == 0) {
            bp.dgate[row] = dg_tot;
            bp.rowterm[row] = rs;
        }
    }
}

template <int D, bool CLAMP, bool BIDIR>
hipError_t launch_q(const BwdParams &p, hipStream_t stream) {
    const int n_qt = (p.f.N + BM - 1) / BM;
    const int64_t n_logical = (int64_t)p.f.B * p.f.H * n_qt;
    const int64_t grid = xcd_grid(n_logical);
    return launch_kernel(backward_q_bf16_kernel<D, CLAMP, BIDIR>, dim3((unsigned)grid), dim3(NT), stream, p, n_qt,
                         n_logical);
}

template <int D, bool BIDIR>
hipError_t launch_qc(const BwdParams &p, hipStream_t stream) {
    return p.f.clamp > 0.0f ? launch_q<D, true, BIDIR>(p, stream) : launch_q<D, false, BIDIR>(p, stream);
}

}  // namespace

hipError_t launch_backward_q_bf16(const BwdParams &p, hipStream_t stream) {
    if (p.f.D == 64) return p.f.causal ? launch_qc<64, false>(p, stream) : launch_qc<64, true>(p, stream);
    return p.f.causal ? launch_qc<128, false>(p, stream) : launch_qc<128, true>(p, stream);
}

}  // namespace pi_attn
