// backward_kv_bf16.hip -- MFMA key pass of the backward for bf16 inputs:
// dk and dv (D = 64 or 128), fp32 accumulation.
//
// A work-group of 8 wavefronts owns 128 keys [j0, j0 + 128) of one (b, h),
// as 4 pairs: pair w (wavefronts w and w + 4) the 32 keys
// kq0 = j0 + 32w + [0, 32).  The queries that hold these keys in their
// window stream through LDS in 64-row tiles of Q and dL/dy, with the
// per-query lse, row term r_t = <dL/dy_t, y_t> and prior bias: the band
// of queries [j0, j0 + 127 + k] (key j is in W_t iff j <= t <= j + k,
// Sec. 3.2 eq. Nr; bidirectionally [j0 - k, j0 + 127 + k], |t - j| <= k);
// rows outside [0, N) are zero and masked.  After the band, the queries
// whose partner is one of these keys (Sec. 3.4 eq. Npi, pi > k), the run
// [j0 + pi, j0 + pi + 128) of queries t = j + pi (bidirectionally also
// [j0 - pi, j0 - pi + 128), t = j - pi), are staged into the two tile
// buffers: each key meets exactly one query of a run, row 32w + c for key
// kq0 + c, and each lane forms that entry with per-lane dot products.
//
// The two wavefronts of a pair split each 32-query block between them, on
// v_mfma_f32_32x32x16_bf16 with lane l holding key l%32 and queries
// 8i + 4(l/32) + j at slot 4i + j:
//   value wavefront (K^T in registers, dV^T accumulator)
//     S = Q K^T (A = Q rows from LDS), alpha^ = exp(delta - lse_t),
//     alpha^ to LDS for the pair's key wavefront, then dV^T += dO^T alpha^
//   key wavefront (V^T in registers, dK^T accumulator)
//     dP = dO V^T, then with alpha^ from LDS dS = alpha^ (dP - r_t)
//     (Sec. 3.5 eq. jac; 0 where the clamp saturates), dK^T += Q^T dS
// The transposed A operands are LDS transpose reads, with the query order
// permuted inside each 16-query chunk as the forward permutes V^T against
// P^T.  dk carries the factor scale.  The alpha^ handed over is the float32
// value the value wavefront computed (sign bit set where the clamp
// saturates), so the split changes no result.  Each wavefront holds one
// accumulator (64 registers at D = 128) and one operand block, so two
// wavefronts fit each SIMD and one's exponentials and conversions run while
// the other's MFMAs do.  Every block is two phases split by a work-group
// barrier: S and dP, then dV and dK; alpha^ is double-buffered by block.
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

constexpr int PAIRS = 4;
constexpr int NT = 64 * 2 * PAIRS;
constexpr int BK = 32 * PAIRS;   // keys per work-group
constexpr int TQ = 64;           // query rows per LDS tile

template <int D>
struct Tile {
    static constexpr int CPR = D / 8;
    static constexpr int ROW = 2 * D + 64;   // LDS row stride (bytes), see chunk_x
    static constexpr int BYTES = TQ * ROW;
    static constexpr int KS = D / 16;
    static constexpr int DB = D / 32;
    static constexpr int CH = TQ * CPR / NT;  // staged chunks per thread and tensor
};

template <int D>
struct QTile {
    alignas(16) unsigned char q[Tile<D>::BYTES];
    alignas(16) unsigned char o[Tile<D>::BYTES];
    alignas(16) float lse2[TQ];   // (lse_t - lse_shift_t) * log2 e (with the clamp)
    alignas(16) float r[TQ];      // row term
    alignas(16) float bias[TQ];   // with the clamp: prior bias of this stream (natural log);
                                  // without: that bias * log2 e - lse2, the exponent offset
};

// alpha^ of one block, handed from each pair's value wavefront to its key
// wavefront: slot group i (slots 4i..4i+3) of lane l at [i][l], so each
// 16-byte access of a wavefront covers consecutive addresses.
struct PBuf {
    alignas(16) float v[2][PAIRS][4][64][4];   // [block parity][pair][i][lane]
};

template <int D>
struct Stage {
    uint4 q[Tile<D>::CH];
    uint4 o[Tile<D>::CH];
    float gl, lse, r;   // raw per-row values: gate logit, lse, row term
    bool band;          // a window-band row (else a partner-run row)
};

// LDS layout of the Q and dL/dy tiles: rows padded by 64 bytes, and the low
// two bits of a row's 16-byte chunk index XORed with bits 2-3 of the row.
// Both reads of a tile are then free of bank conflicts: the row fragments
// (16 consecutive rows, one chunk each) and the transpose reads (4
// consecutive rows, 4 consecutive chunks each); the offsets stay affine in
// the k-step (two bases, even and odd steps) and in the dimension block.
__device__ inline int chunk_x(int row) { return (row >> 2) & 3; }

// The value held by the other half of the wavefront (lane l ^ 32).
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

template <int D, bool CLAMP, bool BIDIR>
__global__ __launch_bounds__(NT) void backward_kv_bf16_kernel(BwdParams bp, int n_kt, int64_t n_logical) {
    using T = Tile<D>;
    constexpr int KS = T::KS, DB = T::DB;
    const FwdParams &p = bp.f;
    __shared__ QTile<D> tA, tB;
    __shared__ PBuf pbuf;
    const int64_t logical = xcd_remap(blockIdx.x, n_logical);
    if (logical < 0) return;
    const int kt = (int)(logical % n_kt);
    const int64_t bh = logical / n_kt;
    const int h = (int)(bh % p.H), b = (int)(bh / p.H);

    const int tid = threadIdx.x;
    const int lane = __lane_id();
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int w = wv % PAIRS;               // pair
    const bool keyw = wv >= PAIRS;          // key wavefront (else value wavefront)
    const int g = lane >> 5, c = lane & 31;
    const int N = p.N, kw = p.k, pi = p.pi;
    // absolute positions: keys [kvpos0, NK) (this pass's keys), query rows
    // held [QS, QE) (their q, dL/dy, lse, row terms and gate)
    const int NK = p.kvpos0 + N, QS = p.qpos0, QE = min(p.qend, p.nseq);
    const int j0 = p.kvpos0 + kt * BK;
    const int kq0 = j0 + 32 * w;
    const int j = kq0 + c;           // this lane's key
    const bool j_ok = j < NK;
    const int jq = j_ok ? j : p.kvpos0;

    // row pointers and per-row arrays indexed by absolute position
    const int64_t sn = p.sn, ksn = p.ksn, osn = bp.osn;
    const __bf16 *qp = (const __bf16 *)p.q + b * p.sb + h * p.sh - (int64_t)QS * sn;
    const int64_t kvbase = b * p.ksb + h * p.ksh - (int64_t)p.kvpos0 * ksn;
    const __bf16 *op = (const __bf16 *)bp.dout + b * bp.osb + h * bp.osh - (int64_t)QS * osn;
    const int64_t rbase = bh * (int64_t)(p.qend - QS) - QS;   // lse, row terms [B][H][qend - qpos0]
    const int64_t obase = bh * (int64_t)N - p.kvpos0;         // dk, dv [B][H][N]
    const bool exact = CLAMP;
    const float c2 = p.scale * kLog2e;

    // B operand of this wavefront's keys: K^T (value wavefront) or V^T (key
    // wavefront), zero past N; and its accumulator, dV^T or dK^T.
    const __bf16 *kvp = (const __bf16 *)(keyw ? p.v : p.k_ptr) + kvbase;
    bf16x8 kvf[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        const bf16x8 x = *reinterpret_cast<const bf16x8 *>(kvp + jq * ksn + 16 * s + 8 * g);
        kvf[s] = j_ok ? x : bf16x8{};
    }
    f32x16 acc[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) acc[db] = f32x16{};

    // The window band streams through LDS: query rows [band_lo, band_hi) in
    // 64-row tiles (rows outside the held [QS, QE) are zero and masked).
    // The partner runs, queries [par_lo, par_hi) whose partner t - pi is
    // one of these keys and (bidirectional) [par2_lo, par2_hi) whose
    // partner t + pi is, are handled after the band.
    const int band_lo = BIDIR ? window_lo(j0, kw) & ~31 : j0;
    const int band_hi = BIDIR ? (int)min((int64_t)j0 + BK + kw, (int64_t)QE) : min(QE, j0 + BK + kw);
    const int ntiles = band_hi > band_lo ? (band_hi - band_lo + TQ - 1) / TQ : 0;
    const bool has_par = partner_enabled(kw, pi) && (int64_t)j0 + pi < QE;
    const int par_lo = j0 + pi;
    const int par_hi = has_par ? min(QE, j0 + pi + BK) : par_lo;
    const bool has_par2 = BIDIR && partner_enabled(kw, pi) && j0 + BK > pi;
    const int par2_lo = j0 - pi;   // may be negative
    const int par2_hi = has_par2 ? min(QE, j0 + BK - pi) : par2_lo;

    // Stage 64 query rows starting at q0m (held [max(q0m, QS), lim)).
    auto load_rows = [&](Stage<D> &st, int q0m, int lim, bool band) __attribute__((always_inline)) {
        const int tfirst = min(max(q0m, QS), QE - 1);   // an always-held row
#pragma unroll
        for (int u = 0; u < T::CH; ++u) {
            const int cid = tid + NT * u;
            const int row = cid / T::CPR, pc = cid % T::CPR;
            const int t = q0m + row;
            const bool ok = t >= QS && t < lim;
            const int tc = ok ? t : tfirst;
            const uint4 qv = *reinterpret_cast<const uint4 *>(qp + tc * sn + 8 * pc);
            const uint4 ov = *reinterpret_cast<const uint4 *>(op + tc * osn + 8 * pc);
            st.q[u] = ok ? qv : make_uint4(0, 0, 0, 0);
            st.o[u] = ok ? ov : make_uint4(0, 0, 0, 0);
        }
        // Only loads here: the values derived from them are formed in store,
        // after the tile's blocks, so that no wavefront waits for this
        // tile's loads before it consumes the current one.
        if (tid < TQ) {
            const int t = q0m + tid;
            const int tc = (t >= QS && t < lim) ? t : tfirst;
            st.gl = p.gate[b * p.gsb + h * p.gsh + (tc - QS) * p.gsn];
            st.lse = bp.lse[rbase + tc];
            st.r = bp.rowterm[rbase + tc];
            st.band = band;
        }
    };
    auto load = [&](Stage<D> &st, int m) __attribute__((always_inline)) {
        load_rows(st, band_lo + TQ * m, band_hi, true);
    };
    auto store = [&](const Stage<D> &st, QTile<D> &tb) {
#pragma unroll
        for (int u = 0; u < T::CH; ++u) {
            const int cid = tid + NT * u;
            const int row = cid / T::CPR, pc = cid % T::CPR;
            *reinterpret_cast<uint4 *>(tb.q + row * T::ROW + (pc ^ chunk_x(row)) * 16) = st.q[u];
            *reinterpret_cast<uint4 *>(tb.o + row * T::ROW + (pc ^ chunk_x(row)) * 16) = st.o[u];
        }
        if (tid < TQ) {
            const FusionBias fb = fusion_bias(st.gl, exact);
            const float l2 = (st.lse - fb.lse_shift) * kLog2e;
            tb.lse2[tid] = l2;
            tb.r[tid] = st.r;
            const float bias_local = fb.local, bias_partner = fb.partner;
            const float bias = st.band ? bias_local : bias_partner;
            tb.bias[tid] = CLAMP ? bias : bias * kLog2e - l2;
        }
    };

    // Whether pair w meets the 32-query block starting at t0b, and whether
    // the block needs masking.
    auto active = [&](int t0b) {
        if constexpr (BIDIR) return t0b < band_hi && kq0 < NK && t0b - (kq0 + 31) <= kw && t0b + 31 >= kq0 - kw;
        return t0b < band_hi && kq0 < NK && t0b <= kq0 + 31 + kw && t0b + 31 >= kq0;
    };
    auto edge_block = [&](int t0b) {
        return BIDIR ? !(t0b + 31 - kq0 <= kw && kq0 + 31 - t0b <= kw) || t0b + 31 >= QE || kq0 + 31 >= NK ||
                           t0b < QS
                     : !(t0b >= kq0 + 31 && t0b + 31 <= kq0 + kw) || t0b + 31 >= QE || kq0 + 31 >= NK;
    };

    // First phase of a block (rows 32 blk.. of tile tb, first query t0b):
    // the value wavefront forms alpha^ (to pb for dV, to LDS for the pair's
    // key wavefront), the key wavefront dP (to dp).
    auto phase1 = [&](const QTile<D> &tb, int t0b, int blk, bool edge, int par, bf16x8 (&pb)[2],
                      f32x16 &dp) {
        // rows of this block (A operands: query l%32, dims 16s + 8g): chunk
        // (2s + g) ^ x = 2(s ^ (x >> 1)) + (g ^ (x & 1)), x = chunk_x(row)
        const int xr = chunk_x(32 * blk + c);
        const int rb = (32 * blk + c) * T::ROW + 16 * (g ^ (xr & 1));
        const int rbo[2] = {rb + 32 * (xr >> 1), rb - 32 * (xr >> 1)};   // even, odd k-steps
        const unsigned char *src = keyw ? tb.o : tb.q;
        bf16x8 ra[KS];
#pragma unroll
        for (int s = 0; s < KS; ++s) ra[s] = *reinterpret_cast<const bf16x8 *>(src + rbo[s & 1] + 32 * s);
        f32x16 sc = {};
#pragma unroll
        for (int s = 0; s < KS; ++s) sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ra[s], kvf[s], sc, 0, 0, 0);
        if (keyw) {
            dp = sc;
            return;
        }
        // alpha^ of this lane's queries 8i + 4g + jj, slot 4i + jj
        bool cut[16];
        float pr[16];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const f32x4 b4 = *reinterpret_cast<const f32x4 *>(tb.bias + 32 * blk + 8 * i + 4 * g);
            if constexpr (CLAMP) {
                const f32x4 l4 = *reinterpret_cast<const f32x4 *>(tb.lse2 + 32 * blk + 8 * i + 4 * g);
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                    const int e = 4 * i + jj;
                    const float dl = fminf(fmaxf(sc[e] * p.scale + b4[jj], -p.clamp), p.clamp);
                    cut[e] = fabsf(dl) >= p.clamp;
                    pr[e] = __builtin_amdgcn_exp2f(dl * kLog2e - l4[jj]);
                }
            } else {
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                    const int e = 4 * i + jj;
                    cut[e] = false;
                    pr[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[e], c2, b4[jj]));
                }
            }
        }
        // Edge blocks: the working-set entries of this lane's key j among the
        // block's queries are one run of rows, the window [j, j + k] (|t - j|
        // <= k bidirectionally), cut to the held rows [QS, QE) and to the
        // block; bit r of keep marks
        // row 4g + r of the block (this lane's rows 4g + 8i + jj at bit
        // 8i + jj), and alpha^ of the other entries is cleared.  The empty
        // asm keeps this a branch that interior blocks skip.
        if (edge) {
            asm volatile("" ::: "memory");
            const int lo = max(BIDIR ? j - kw : j, max(QS, t0b));
            const int hi = min(j + kw, min(QE - 1, t0b + 31));
            const int n = hi - lo + 1;
            uint32_t keep = !j_ok || n <= 0 ? 0u : n >= 32 ? ~0u : ((1u << n) - 1u) << (lo - t0b);
            keep >>= 4 * g;
#pragma unroll
            for (int e = 0; e < 16; ++e) {   // all bits of pr[e], or none
                const int bit = __builtin_amdgcn_sbfe((int)keep, 8 * (e >> 2) + (e & 3), 1);
                pr[e] = __int_as_float(__float_as_int(pr[e]) & bit);
            }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            f32x4 h4;
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) h4[jj] = cut[4 * i + jj] ? -pr[4 * i + jj] : pr[4 * i + jj];
            *reinterpret_cast<f32x4 *>(&pbuf.v[par][w][i][lane][0]) = h4;
        }
#pragma unroll
        for (int cc = 0; cc < 2; ++cc) {
#pragma unroll
            for (int e = 0; e < 8; ++e) pb[cc][e] = (__bf16)pr[8 * cc + e];
        }
    };

    // Second phase: dV^T += dO^T alpha^ (value wavefront) or, with alpha^
    // from LDS, dK^T += Q^T dS (key wavefront).
    auto phase2 = [&](const QTile<D> &tb, int blk, int par, const bf16x8 (&pb)[2], const f32x16 &dp) {
        bf16x8 bop[2];
        if (keyw) {
            float ds[16];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const f32x4 a4 = *reinterpret_cast<const f32x4 *>(&pbuf.v[par][w][i][lane][0]);
                const f32x4 r4 = *reinterpret_cast<const f32x4 *>(tb.r + 32 * blk + 8 * i + 4 * g);
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                    const int e = 4 * i + jj;
                    const float d = a4[jj] * (dp[e] - r4[jj]);
                    ds[e] = CLAMP && a4[jj] < 0.0f ? 0.0f : d;
                }
            }
#pragma unroll
            for (int cc = 0; cc < 2; ++cc) {
#pragma unroll
                for (int e = 0; e < 8; ++e) bop[cc][e] = (__bf16)ds[8 * cc + e];
            }
        } else {
            bop[0] = pb[0];
            bop[1] = pb[1];
        }
        // transposed tiles (A operands: dim 32db + l%32, queries permuted)
        // rows 32 blk + 4g + rr + 8hh + 16cc, chunks 4d + (j ^ (g + 2hh))
        const unsigned char *src = keyw ? tb.q : tb.o;
        const int G = lane >> 4, rr = (lane >> 2) & 3, qd = lane & 3;
        const int jq = 2 * (G & 1) + (qd >> 1);
        const int toff[2] = {(32 * blk + 4 * g + rr) * T::ROW + 16 * (jq ^ g) + (qd & 1) * 8,
                             (32 * blk + 4 * g + rr + 8) * T::ROW + 16 * (jq ^ (g + 2)) + (qd & 1) * 8};
#pragma unroll
        for (int cc = 0; cc < 2; ++cc) {
#pragma unroll
            for (int d = 0; d < DB; ++d) {
                bf16x8 at;
#pragma unroll
                for (int hh = 0; hh < 2; ++hh) {
                    const int off = toff[hh] + 16 * cc * T::ROW + 64 * d;
                    const bf16x4 y = __builtin_bit_cast(
                        bf16x4, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(src + off)));
#pragma unroll
                    for (int x = 0; x < 4; ++x) at[4 * hh + x] = y[x];
                }
                acc[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(at, bop[cc], acc[d], 0, 0, 0);
            }
        }
    };

    // One 64-row tile (cur) of the combined stream; the staged next tile goes
    // into nxt between the two blocks (nxt's last reader, the previous
    // tile's second block, finished before this tile's first barrier).
    Stage<D> st;
    auto tile = [&](const QTile<D> &cur, QTile<D> &nxt, int m) {
        const int t0 = band_lo + TQ * m;
        bf16x8 pb[2];
        f32x16 dp;
        const bool a0 = active(t0), a1 = active(t0 + 32);
        if (a0) phase1(cur, t0, 0, edge_block(t0), 0, pb, dp);
        __syncthreads();
        if (a0) phase2(cur, 0, 0, pb, dp);
        if (a1) phase1(cur, t0 + 32, 1, edge_block(t0 + 32), 1, pb, dp);
        if (m + 1 < ntiles) {
            store(st, nxt);
            if (m + 2 < ntiles) load(st, m + 2);
        }
        __syncthreads();
        if (a1) phase2(cur, 1, 1, pb, dp);
    };

    if (ntiles > 0) {
        load(st, 0);
        store(st, tA);
        if (ntiles > 1) load(st, 1);
        __syncthreads();
        for (int m = 0; m < ntiles; m += 2) {
            tile(tA, tB, m);
            if (m + 1 >= ntiles) break;
            tile(tB, tA, m + 1);
        }
    }

    // ---- partners (Sec. 3.4, eq. Npi) ---------------------------------------
    // The queries whose partner is one of this work-group's keys form one run
    // of 128 rows (t = j + pi; bidirectionally also t = j - pi), row 32w + c
    // the partner of key kq0 + c.  The run is staged into the two tile
    // buffers after the band; each lane then forms its one entry by a dot
    // product of its half of the query (dL/dy) row with its half of k_j
    // (v_j), plus the other half's: the value wavefront adds alpha^ dO_t to
    // dV and hands alpha^ over through LDS, the key wavefront adds
    // alpha^ (dP - r_t) q_t to dK.
    auto partner_run = [&](int lo, int hi) __attribute__((always_inline)) {
        __syncthreads();   // every wavefront is done with the tile buffers
        load_rows(st, lo, hi, false);
        store(st, tA);
        load_rows(st, lo + TQ, hi, false);
        store(st, tB);
        __syncthreads();
        const QTile<D> &tb = w < 2 ? tA : tB;
        const int row = 32 * (w & 1) + c, t = lo + 32 * w + c;
        const bool has = j_ok && t >= QS && t < hi;
        const int xr = chunk_x(row);
        const int rb = row * T::ROW + 16 * (g ^ (xr & 1));
        const int rbo[2] = {rb + 32 * (xr >> 1), rb - 32 * (xr >> 1)};   // even, odd k-steps
        const unsigned char *src = keyw ? tb.o : tb.q;
        float part = 0.0f;
#pragma unroll
        for (int s = 0; s < KS; ++s)
            part = dot_bf16x8(*reinterpret_cast<const bf16x8 *>(src + rbo[s & 1] + 32 * s), kvf[s], part);
        const float d = part + other_half(part);
        // the other operand row in the accumulator layout: dims 32db + 8i + 4g + [0, 4)
        auto add_row = [&](const unsigned char *rows, float wgt) __attribute__((always_inline)) {
#pragma unroll
            for (int db = 0; db < DB; ++db) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const uint2 raw = *reinterpret_cast<const uint2 *>(
                        rows + row * T::ROW + ((4 * db + i) ^ xr) * 16 + 8 * g);
                    acc[db][4 * i + 0] += wgt * __uint_as_float(raw.x << 16);
                    acc[db][4 * i + 1] += wgt * __uint_as_float(raw.x & 0xffff0000u);
                    acc[db][4 * i + 2] += wgt * __uint_as_float(raw.y << 16);
                    acc[db][4 * i + 3] += wgt * __uint_as_float(raw.y & 0xffff0000u);
                }
            }
        };
        if (!keyw) {
            float pr;
            bool cut = false;
            if constexpr (CLAMP) {
                const float dl = fminf(fmaxf(d * p.scale + tb.bias[row], -p.clamp), p.clamp);
                cut = fabsf(dl) >= p.clamp;
                pr = __builtin_amdgcn_exp2f(dl * kLog2e - tb.lse2[row]);
            } else {
                pr = __builtin_amdgcn_exp2f(__builtin_fmaf(d, c2, tb.bias[row]));
            }
            pr = has ? pr : 0.0f;
            pbuf.v[0][w][0][lane][0] = cut ? -pr : pr;
            add_row(tb.o, pr);
        }
        __syncthreads();   // alpha^ handed over
        if (keyw) {
            const float hv = pbuf.v[0][w][0][lane][0];
            const float dsv = CLAMP && hv < 0.0f ? 0.0f : hv * (d - tb.r[row]);
            add_row(tb.q, dsv);
        }
    };
    if (has_par) partner_run(par_lo, par_hi);
    if (has_par2) partner_run(par2_lo, par2_hi);

    // ---- store: lane (c, g) holds dims 32db + 8i + 4g + [0, 4) of key c ----
    // The accumulator goes out in whole rows: each wavefront writes half of
    // its 32 rows' dims to a private LDS region (the tile buffers, free once
    // every wavefront has left the loop), reads them back 16 bytes per lane
    // along the rows and stores 256 contiguous bytes per row (128 at D = 64),
    // instead of 16-byte pieces of 32 rows per instruction.
    {
        constexpr int HW = D / 2;              // dims per pass
        constexpr int P = HW * 4 + 16;         // LDS row pitch (bytes), padded against bank conflicts
        constexpr int LPR = HW / 4;            // lanes per row when reading back
        constexpr int RPI = 64 / LPR;          // rows per read instruction
        static_assert(4 * 32 * P <= (int)sizeof(QTile<D>), "store staging fits a tile buffer");
        __syncthreads();
        unsigned char *reg = reinterpret_cast<unsigned char *>(wv < PAIRS ? &tA : &tB) + (wv % PAIRS) * 32 * P;
        float *dst = keyw ? bp.dk : bp.dv;
        const float f = keyw ? p.scale : 1.0f;
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
#pragma unroll
            for (int d = 0; d < DB / 2; ++d) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    f32x4 a;
#pragma unroll
                    for (int x = 0; x < 4; ++x) a[x] = acc[hf * (DB / 2) + d][4 * i + x] * f;
                    *reinterpret_cast<f32x4 *>(reg + c * P + (32 * d + 8 * i + 4 * g) * 4) = a;
                }
            }
#pragma unroll
            for (int v = 0; v < 32 / RPI; ++v) {
                const int r = RPI * v + lane / LPR, ch = lane % LPR;
                const f32x4 a = *reinterpret_cast<const f32x4 *>(reg + r * P + ch * 16);
                if (kq0 + r < NK) *reinterpret_cast<f32x4 *>(dst + (obase + kq0 + r) * D + hf * HW + 4 * ch) = a;
            }
        }
    }
}

template <int D, bool CLAMP, bool BIDIR>
hipError_t launch_kv(const BwdParams &p, hipStream_t stream) {
    const int n_kt = (p.f.N + BK - 1) / BK;
    const int64_t n_logical = (int64_t)p.f.B * p.f.H * n_kt;
    const int64_t grid = xcd_grid(n_logical);
    return launch_kernel(backward_kv_bf16_kernel<D, CLAMP, BIDIR>, dim3((unsigned)grid), dim3(NT), stream, p, n_kt,
                         n_logical);
}

template <int D, bool BIDIR>
hipError_t launch_kvc(const BwdParams &p, hipStream_t stream) {
    return p.f.clamp > 0.0f ? launch_kv<D, true, BIDIR>(p, stream) : launch_kv<D, false, BIDIR>(p, stream);
}
}  // namespace

hipError_t launch_backward_kv_bf16(const BwdParams &p, hipStream_t stream) {
    if (p.f.D == 64) return p.f.causal ? launch_kvc<64, false>(p, stream) : launch_kvc<64, true>(p, stream);
    return p.f.causal ? launch_kvc<128, false>(p, stream) : launch_kvc<128, true>(p, stream);
}
}  // namespace pi_attn
