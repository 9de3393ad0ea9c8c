// forward_bf16.hip -- banded MFMA forward of causal pi-Attention, bf16 in,
// fp32 accumulate, for head dimension D = 64 or 128.
//
// Work decomposition.  One work-group (4 wavefronts) owns a query tile of
// BM = 128 consecutive positions [t0, t0+128) of one (b, h).  Wavefront w owns
// the 32 queries t0 + 32w + [0, 32).  The working sets of the tile are
//   window keys   [max(0, t0-k), t0+127]  -- a band, streamed in 64-key tiles
//   partner keys  [t0-pi, t0-pi+127]      -- one contiguous shifted tile
// (Sec. 3.5, eq. online_ws: the partner rows of consecutive queries are
// consecutive, so the long-range fetch is a coalesced tile, not a gather).
//
// Scores are computed transposed, S^T = K Q^T, on v_mfma_f32_32x32x16_bf16:
//   A = K tile rows (32 keys x 16 dims, from LDS),
//   B = Q^T (16 dims x 32 queries, resident in registers for the whole tile),
//   C = 32 keys x 32 queries; lane l holds query column l%32 and key rows
//       8i + 4(l/32) + j in accumulator slot 4i+j.
// A lane therefore holds one query's scores, so the softmax row reductions
// are in-lane plus one exchange with lane l^32.  The output is O^T = V^T P^T
// on the same instruction: B = P^T comes straight from the score registers
// (slots 8c..8c+7 of a 32-key block are the B operand of key chunk c, with
// the key order permuted inside the chunk), A = V^T read from a transposed
// LDS copy of the value tile with the same permutation.
//
// The partner block joins the same online softmax: it is processed first, as
// a 32x32 score block whose only valid entries are on the diagonal (query i
// of the wavefront pairs with key row i of its partner rows).
#include "kernels.h"
#include "pi_common.h"

namespace pi_attn {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int BM = 128;       // queries per work-group
constexpr int BN = 64;        // keys per LDS tile
constexpr int QW = 32;        // queries per wavefront
constexpr int NT = 256;       // threads per work-group
constexpr int KPAD = 8;       // K tile row padding (elements)
constexpr int VPAD = 4;       // V^T tile row padding (elements)

template <int D>
struct Smem {
    __bf16 k[2][BN][D + KPAD];     // key rows, row-major
    __bf16 vt[2][D][BN + VPAD];    // value tile, transposed (dim-major)
};

// Register staging of one 64-key tile: K and V rows as 16-byte chunks.
template <int D>
struct Stage {
    static constexpr int CH = BN * D / 8 / NT;   // 16-byte chunks per thread (4 or 2)
    uint4 kc[CH];
    uint4 vc[CH];
};

__device__ inline uint4 ld16(const __bf16 *p) { return *reinterpret_cast<const uint4 *>(p); }

// Issue the global loads of key/value rows [row0, row0+64); rows outside
// [0, lim) are not read and stage as zero.  For window tiles lim is the end
// of the query tile, so no row later than every query of the tile is ever
// touched (a masked weight is 0, but 0 times a non-finite value is not).
template <int D>
__device__ inline void stage_load(Stage<D> &st, const __bf16 *kb, const __bf16 *vb, int64_t sn, int row0, int lim,
                                  int tid) {
    constexpr int CPR = D / 8;   // chunks per row
#pragma unroll
    for (int c = 0; c < Stage<D>::CH; ++c) {
        // K: consecutive threads take consecutive chunks of a row.
        int cid = tid + NT * c;
        int r = cid / CPR, col = cid % CPR;
        int gr = row0 + r;
        st.kc[c] = (gr >= 0 && gr < lim) ? ld16(kb + gr * sn + col * 8) : make_uint4(0, 0, 0, 0);
        // V: thread owns CH consecutive rows of one 8-dim chunk (for the
        // transposed store); each load instruction still reads whole rows.
        int vcol = tid % CPR, vrg = tid / CPR;
        int vr = vrg * Stage<D>::CH + c;
        int gv = row0 + vr;
        st.vc[c] = (gv >= 0 && gv < lim) ? ld16(vb + gv * sn + vcol * 8) : make_uint4(0, 0, 0, 0);
    }
}

template <int D>
__device__ inline void stage_store(const Stage<D> &st, Smem<D> &sm, int buf, int tid) {
    constexpr int CPR = D / 8;
    constexpr int CH = Stage<D>::CH;
#pragma unroll
    for (int c = 0; c < CH; ++c) {
        int cid = tid + NT * c;
        int r = cid / CPR, col = cid % CPR;
        *reinterpret_cast<uint4 *>(&sm.k[buf][r][col * 8]) = st.kc[c];
    }
    int vcol = tid % CPR, vrg = tid / CPR;
    const bf16x8 *rows = reinterpret_cast<const bf16x8 *>(st.vc);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        if constexpr (CH == 4) {
            bf16x4 w = {rows[0][i], rows[1][i], rows[2][i], rows[3][i]};
            *reinterpret_cast<bf16x4 *>(&sm.vt[buf][vcol * 8 + i][vrg * 4]) = w;
        } else {
            bf16x2 w = {rows[0][i], rows[1][i]};
            *reinterpret_cast<bf16x2 *>(&sm.vt[buf][vcol * 8 + i][vrg * 2]) = w;
        }
    }
}

// Per-wavefront online-softmax state for its 32 queries (lane = query l%32).
template <int D>
struct WaveState {
    static constexpr int DB = D / 32;   // 32-dim output blocks
    static constexpr int KS = D / 16;   // 16-dim k-steps of the score MFMA
    bf16x8 qb[KS];                      // B operand: Q[t][16s + 8g .. +8]
    f32x16 o[DB];                       // O^T accumulators
    float m;                            // running max (log2 domain)
    float l;                            // this lane's partial running sum
};

// S^T block (32 keys x 32 queries) for key rows [r0, r0+32) of LDS buffer buf.
template <int D>
__device__ inline f32x16 score_block(const Smem<D> &sm, int buf, int r0, const WaveState<D> &ws, int lane) {
    f32x16 acc = {};
    const int row = r0 + (lane & 31), g = lane >> 5;
#pragma unroll
    for (int s = 0; s < WaveState<D>::KS; ++s) {
        bf16x8 a = *reinterpret_cast<const bf16x8 *>(&sm.k[buf][row][16 * s + 8 * g]);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, ws.qb[s], acc, 0, 0, 0);
    }
    return acc;
}

// O^T += V^T P^T over key rows [r0, r0+32) of buffer buf.  pb[c] is the B
// operand of key chunk c (keys 16c + {4g..4g+3, 8+4g..8+4g+3}).
template <int D>
__device__ inline void pv_block(const Smem<D> &sm, int buf, int r0, const bf16x8 pb[2], WaveState<D> &ws,
                                int lane) {
    const int dl = lane & 31, g = lane >> 5;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
        const int kc = r0 + 16 * c + 4 * g;
#pragma unroll
        for (int db = 0; db < WaveState<D>::DB; ++db) {
            const __bf16 *vrow = &sm.vt[buf][32 * db + dl][0];
            bf16x4 lo = *reinterpret_cast<const bf16x4 *>(vrow + kc);
            bf16x4 hi = *reinterpret_cast<const bf16x4 *>(vrow + kc + 8);
            bf16x8 a = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
            ws.o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[c], ws.o[db], 0, 0, 0);
        }
    }
}

__device__ inline float xor32_max(float x) { return fmaxf(x, __shfl_xor(x, 32)); }

// Fold up to two scored 32-key blocks (already in log2 units, -inf where
// invalid) into the running state and accumulate their values.
template <int D, int NBLK>
__device__ inline void softmax_pv(const Smem<D> &sm, int buf, const int r0[NBLK], const bool act[NBLK],
                                  f32x16 sc[NBLK], WaveState<D> &ws, int lane) {
    float mx = -INFINITY;
#pragma unroll
    for (int b = 0; b < NBLK; ++b)
        if (act[b]) {
#pragma unroll
            for (int e = 0; e < 16; ++e) mx = fmaxf(mx, sc[b][e]);
        }
    mx = xor32_max(mx);
    const float m_new = fmaxf(ws.m, mx);
    const float m_use = m_new == -INFINITY ? 0.0f : m_new;
    const float alpha = __builtin_amdgcn_exp2f(ws.m - m_use);
    ws.m = m_new;
    ws.l *= alpha;
#pragma unroll
    for (int db = 0; db < WaveState<D>::DB; ++db) ws.o[db] *= alpha;
#pragma unroll
    for (int b = 0; b < NBLK; ++b) {
        if (!act[b]) continue;
        bf16x8 pb[2];
#pragma unroll
        for (int c = 0; c < 2; ++c) {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                float pr = __builtin_amdgcn_exp2f(sc[b][8 * c + e] - m_use);
                ws.l += pr;
                pb[c][e] = (__bf16)pr;
            }
        }
        pv_block<D>(sm, buf, r0[b], pb, ws, lane);
    }
}

template <int D, bool CLAMP>
__global__ __launch_bounds__(NT, 2) void forward_bf16_kernel(FwdParams p, int n_qt, int64_t n_logical) {
    __shared__ Smem<D> sm;
    const int64_t logical = xcd_remap(blockIdx.x, n_logical);
    if (logical < 0) return;
    const int qt = (int)(logical % n_qt);
    const int64_t bh = logical / n_qt;
    const int h = (int)(bh % p.H), b = (int)(bh / p.H);

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int g = lane >> 5, c = lane & 31;
    const int N = p.N, kw = p.k;
    const int t0 = qt * BM;
    const int qw0 = t0 + QW * w;    // first query of this wavefront
    const int t = qw0 + c;          // this lane's query
    const bool t_ok = t < N;

    const int64_t base = b * p.sb + h * p.sh;
    const __bf16 *qp = (const __bf16 *)p.q + base;
    const __bf16 *kp = (const __bf16 *)p.k_ptr + base;
    const __bf16 *vp = (const __bf16 *)p.v + base;
    const int64_t sn = p.sn;

    WaveState<D> ws;
#pragma unroll
    for (int s = 0; s < WaveState<D>::KS; ++s) {
        if (t_ok) {
            ws.qb[s] = *reinterpret_cast<const bf16x8 *>(qp + t * sn + 16 * s + 8 * g);
        } else {
            ws.qb[s] = bf16x8{};
        }
    }
#pragma unroll
    for (int db = 0; db < WaveState<D>::DB; ++db) ws.o[db] = f32x16{};
    ws.m = -INFINITY;
    ws.l = 0.0f;

    const float gl = p.gate[b * p.gsb + h * p.gsh + (t_ok ? t : 0) * p.gsn];
    const FusionBias fb = fusion_bias(gl, CLAMP);
    const float c2 = p.scale * kLog2e;          // score -> log2 units
    const float clampv = p.clamp;

    // ---- partner tile: rows [t0 - pi, t0 - pi + 128) -------------------
    const bool has_partner = partner_enabled(kw, p.pi) && (t0 + BM - 1) >= p.pi && t0 < N;
    Stage<D> st;
    if (has_partner) {
        const int prow0 = t0 - p.pi;
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            stage_load<D>(st, kp, vp, sn, prow0 + BN * half, N, tid);
            stage_store<D>(st, sm, half, tid);
        }
    }
    // window tiles: [kstart, kend) in 64-key steps
    const int kstart = window_lo(t0, kw);
    const int kend = min(t0 + BM, N);
    const int ntiles = kend > kstart ? (kend - kstart + BN - 1) / BN : 0;
    if (ntiles > 0) stage_load<D>(st, kp, vp, sn, kstart, kend, tid);
    if (has_partner) {
        __syncthreads();
        // wavefront w's partner rows are rows 32w.. of the 128-row tile:
        // buffer w/2, block (w%2)
        if (qw0 + QW - 1 >= p.pi && qw0 < N) {
            const int buf = w >> 1, r0 = QW * (w & 1);
            f32x16 raw = score_block<D>(sm, buf, r0, ws, lane);
            f32x16 sc[1];
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int r = 8 * (e >> 2) + 4 * g + (e & 3);   // key row in block
                const bool valid = (r == c) && t_ok && t >= p.pi;
                float v;
                if constexpr (CLAMP) {
                    v = fminf(fmaxf(raw[e] * p.scale + fb.partner, -clampv), clampv) * kLog2e;
                } else {
                    v = raw[e] * c2 + fb.partner * kLog2e;
                }
                sc[0][e] = valid ? v : -INFINITY;
            }
            const int r0a[1] = {r0};
            const bool act[1] = {true};
            softmax_pv<D, 1>(sm, buf, r0a, act, sc, ws, lane);
        }
        __syncthreads();
    }
    if (ntiles > 0) {
        stage_store<D>(st, sm, 0, tid);
        __syncthreads();
    }

    // ---- window band ----------------------------------------------------
    for (int it = 0; it < ntiles; ++it) {
        const int buf = it & 1;
        const int j0 = kstart + BN * it;
        if (it + 1 < ntiles) stage_load<D>(st, kp, vp, sn, j0 + BN, kend, tid);

        // blocks of this tile that intersect the wavefront's band
        // [qw0 - k, qw0 + 31]
        bool act[2];
        int r0a[2];
        bool any = false;
#pragma unroll
        for (int bb = 0; bb < 2; ++bb) {
            const int jb = j0 + QW * bb;
            r0a[bb] = QW * bb;
            act[bb] = (jb <= qw0 + QW - 1) && (jb + QW - 1 >= qw0 - kw) && (jb < N) && (qw0 < N);
            any |= act[bb];
        }
        if (any) {
            f32x16 sc[2];
#pragma unroll
            for (int bb = 0; bb < 2; ++bb) {
                if (!act[bb]) continue;
                f32x16 raw = score_block<D>(sm, buf, r0a[bb], ws, lane);
                const int jb = j0 + QW * bb;
                // interior: every key of the block is in every query's window
                const bool interior = (jb + QW - 1 <= qw0) && (jb >= qw0 + QW - 1 - kw);
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    float v;
                    if constexpr (CLAMP) {
                        v = fminf(fmaxf(raw[e] * p.scale + fb.local, -clampv), clampv) * kLog2e;
                    } else {
                        v = raw[e] * c2;
                    }
                    if (!interior) {
                        const int j = jb + 8 * (e >> 2) + 4 * g + (e & 3);
                        v = in_window(j, t, kw) ? v : -INFINITY;
                    }
                    sc[bb][e] = v;
                }
            }
            softmax_pv<D, 2>(sm, buf, r0a, act, sc, ws, lane);
        }
        if (it + 1 < ntiles) stage_store<D>(st, sm, buf ^ 1, tid);
        __syncthreads();
    }

    // ---- normalise and store ---------------------------------------------
    const float l_tot = ws.l + __shfl_xor(ws.l, 32);
    if (t_ok) {
        const float inv = 1.0f / l_tot;
        __bf16 *op = (__bf16 *)p.out + b * p.osb + h * p.osh + t * p.osn;
#pragma unroll
        for (int db = 0; db < WaveState<D>::DB; ++db) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                bf16x4 o4;
#pragma unroll
                for (int j = 0; j < 4; ++j) o4[j] = (__bf16)(ws.o[db][4 * i + j] * inv);
                *reinterpret_cast<bf16x4 *>(op + 32 * db + 8 * i + 4 * g) = o4;
            }
        }
        if (p.lse && g == 0) {
            p.lse[bh * N + t] = (ws.m + __log2f(l_tot)) * kLn2 + fb.lse_shift;
        }
    }
}

template <int D, bool CLAMP>
hipError_t launch(const FwdParams &p, hipStream_t stream) {
    const int n_qt = (p.N + BM - 1) / BM;
    const int64_t n_logical = (int64_t)p.B * p.H * n_qt;
    if (n_logical == 0) return hipSuccess;
    const int64_t grid = xcd_grid(n_logical);
    return launch_kernel(forward_bf16_kernel<D, CLAMP>, dim3((unsigned)grid), dim3(NT), stream, p, n_qt, n_logical);
}

}  // namespace

hipError_t launch_forward_bf16(const FwdParams &p, hipStream_t stream) {
    const bool clamp = p.clamp > 0.0f;
    if (p.D == 64) return clamp ? launch<64, true>(p, stream) : launch<64, false>(p, stream);
    return clamp ? launch<128, true>(p, stream) : launch<128, false>(p, stream);
}

}  // namespace pi_attn
