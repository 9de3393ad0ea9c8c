// smallk_bf16.hip -- forward of pi-Attention for a small window radius
// (k <= 16; the paper's defaults are k = 4, pi = 16, Sec. 4 and App. B), bf16
// in, fp32 arithmetic, D = 64 or 128, causal or bidirectional, with the
// Variant-3 gate either given as logits or computed from the gate MLP's last
// layer (App. A gate module) in the same kernel.
//
// With |W_t| = k + 2 (k = 4: six keys) a query tile of the banded MFMA kernel
// would compute 128 + k scores per query to use k + 2, so this path gathers
// instead.  A work-group owns 32 consecutive tokens of one batch row and a
// group of up to 32 heads, and loops over the heads:
//   - per head, the window band of its 32 queries (rows [t0 - k, t0 + 31],
//     bidirectional up to t0 + 31 + k) is staged in LDS, the next head's band
//     loaded into registers while the current one is consumed;
//   - a query row is handled by 8 lanes holding D/8 dimensions each; a score
//     is 4 (D = 64) or 8 packed-bf16 dot products per lane
//     (v_dot2c_f32_bf16) and a 3-step DPP reduction inside the 8 lanes, which
//     leaves the same sum in each of them;
//   - the kernel is instantiated for a window bound KMAX (4, 8 or 16, the
//     smallest that holds k); the working set is unrolled to its KMAX-bound
//     size: every score first (independent chains: the partners t - pi and
//     t + pi read straight from global memory, the window from LDS), then
//     one exact maximum, the fp32 softmax and the weighted sum of V.
//     Absent entries (and slots beyond k) read a clamped row of the band and
//     get weight exactly 0.
// Gate MLP epilogue: the logits g[t, h] = <u_t, w2_h> + b2_h of the work-group's
// 32 tokens and heads are one 32x32 block of v_mfma_f32_32x32x16_bf16 products
// (A = the tokens' hidden activations u, B = the heads' rows of w2), the K
// dimension split over the 4 wavefronts and summed in LDS; they are written
// to gate_out for the backward.  u is read once per token for all heads of
// the group.
#include "smallk.h"
#include "pi_common.h"
#include "smallk_common.h"

namespace pi_attn {

namespace {

using namespace sk;

// The gate logits of tokens [t0, t0 + 32) and heads [h0, h0 + nh) (nh <= 32)
// into glds[h - h0][t - t0] (fp32, plus b2) and, when `out` is set, into
// gate_out.  `scratch` holds kGateScratch floats (per wavefront a [head]
// [token] block, rows padded to 33).  Called by all threads.
__device__ void gate_tile(const FwdParams &p, const GateMlp &m, int b, int t0, int h0, int nh, float *scratch,
                          float *glds, bool out) {
    const int tid = threadIdx.x, lane = __lane_id(), w = tid >> 6;
    const int i = lane & 31, g = lane >> 5;
    const int t = t0 + i, h = h0 + i;
    const bool t_ok = t < p.N, h_ok = i < nh;
    const __bf16 *ur = (const __bf16 *)m.u + b * m.usb + (int64_t)(t_ok ? t : 0) * m.usn;
    const __bf16 *wr = (const __bf16 *)m.w2 + (int64_t)(h_ok ? h : 0) * m.dh;
    f32x16 acc = {};
    const int nks = (m.dh + 15) / 16;
    for (int s = w; s < nks; s += 4) {
        const int col = 16 * s + 8 * g;
        const bool c_ok = col < m.dh;   // dh is a multiple of 8
        const bf16x8 a = (t_ok && c_ok) ? *reinterpret_cast<const bf16x8 *>(ur + col) : bf16x8{};
        const bf16x8 bb = (h_ok && c_ok) ? *reinterpret_cast<const bf16x8 *>(wr + col) : bf16x8{};
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bb, acc, 0, 0, 0);
    }
    // C[token r][head i]: lane (i, g) holds rows r = 8(e/4) + 4g + e%4
#pragma unroll
    for (int e = 0; e < 16; ++e) scratch[(w * 32 + i) * 33 + 8 * (e >> 2) + 4 * g + (e & 3)] = acc[e];
    __syncthreads();
    for (int x = tid; x < 32 * 32; x += NT) {
        const int hh = x >> 5, r = x & 31;   // consecutive threads: consecutive tokens of one head
        float v = scratch[(0 * 32 + hh) * 33 + r] + scratch[(1 * 32 + hh) * 33 + r] + scratch[(2 * 32 + hh) * 33 + r] +
                  scratch[(3 * 32 + hh) * 33 + r];
        if (hh < nh) {
            if (m.b2) v += m.b2[h0 + hh];
            glds[hh * TT + r] = v;
            if (out && t0 + r < p.N) m.gate_out[((int64_t)b * p.H + h0 + hh) * p.N + t0 + r] = v;
        }
    }
    __syncthreads();
}

template <int D, bool BIDIR, bool GATED, int KMAX>
__global__ __launch_bounds__(NT) void smallk_bf16_kernel(FwdParams p, GateMlp m, int n_tt, int n_hg,
                                                         int64_t n_logical) {
    using BD = Band<D, BIDIR, KMAX>;
    constexpr int E = BD::E, CPR = BD::CPR, ROWB = BD::ROWB;
    __shared__ alignas(16) unsigned char band[2][2][BD::ROWS * ROWB];   // [buffer][K, V]
    __shared__ float glds[HG * TT];
    static_assert(sizeof(band) >= kGateScratch * sizeof(float), "the gate prologue borrows the band buffers");
    const int64_t logical = xcd_remap(blockIdx.x, n_logical);
    if (logical < 0) return;
    const int hg = (int)(logical % n_hg);
    const int tt = (int)((logical / n_hg) % n_tt);
    const int b = (int)(logical / ((int64_t)n_hg * n_tt));
    const int N = p.N, kw = p.k, pi = p.pi;
    const int hpg = (p.H + n_hg - 1) / n_hg;   // heads per group
    const int h0 = hg * hpg, h1 = min(p.H, h0 + hpg);
    if (h0 >= h1) return;
    const int t0 = tt * TT;
    const int tid = threadIdx.x;
    const int qi = tid >> 3, sl = tid & 7;   // query of the tile, lane within its row
    const int t = t0 + qi;
    const bool t_ok = t < N;
    const int tq = t_ok ? t : N - 1;

    // band rows: LDS row r <-> sequence row t0 - k + r; loaded rows [lo, hi)
    const int rlo = t0 - kw;
    const int lo = max(0, rlo);
    const int hi = BIDIR ? (int)min((int64_t)t0 + TT + kw, (int64_t)N) : min(t0 + TT, N);
    const int rowb_g = (int)(2 * p.sn);
    const int nw = BIDIR ? 2 * kw + 1 : kw + 1;   // window slots
    const int jp_raw = t - pi;
    const bool has_p = t_ok && partner_enabled(kw, pi) && jp_raw >= 0;
    const bool has_f = BIDIR && t_ok && partner_fwd_of(t, kw, pi, N) >= 0;


    // staged state of one head: band chunks, the query chunk, partner chunks, gate logit
    struct Next {
        uint4 k[BD::CH], v[BD::CH];
        uint4 q[E / 8];
        uint4 kp[E / 8], vp[E / 8], kf[E / 8], vf[E / 8];
        float gl;
    };
    auto fetch = [&](Next &nx, int h) {
        const int64_t base = b * p.sb + h * p.sh;
        const __bf16 *kp = (const __bf16 *)p.k_ptr + base;
        const __bf16 *vp = (const __bf16 *)p.v + base;
        const __amdgpu_buffer_rsrc_t rk =
            __builtin_amdgcn_make_buffer_rsrc((void *)(kp + (int64_t)lo * p.sn), (short)0, (hi - lo) * rowb_g, 0x00020000);
        const __amdgpu_buffer_rsrc_t rv =
            __builtin_amdgcn_make_buffer_rsrc((void *)(vp + (int64_t)lo * p.sn), (short)0, (hi - lo) * rowb_g, 0x00020000);
#pragma unroll
        for (int u = 0; u < BD::CH; ++u) {
            const int cid = tid + NT * u;
            const int r = cid / CPR, c = cid % CPR;
            const int gr = rlo + r;
            // rows outside [lo, hi) read as zeros (offset past the range)
            const int off = (gr >= lo && gr < hi && r < BD::ROWS) ? (gr - lo) * rowb_g + 16 * c : (hi - lo) * rowb_g;
            nx.k[u] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rk, off, 0, 0));
            nx.v[u] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rv, off, 0, 0));
        }
        const __bf16 *qrow = (const __bf16 *)p.q + base + (int64_t)tq * p.sn + E * sl;
#pragma unroll
        for (int x = 0; x < E / 8; ++x) nx.q[x] = *reinterpret_cast<const uint4 *>(qrow + 8 * x);
        const int jp = has_p ? jp_raw : tq, jf = has_f ? t + pi : tq;
#pragma unroll
        for (int x = 0; x < E / 8; ++x) {
            nx.kp[x] = *reinterpret_cast<const uint4 *>(kp + (int64_t)jp * p.sn + E * sl + 8 * x);
            nx.vp[x] = *reinterpret_cast<const uint4 *>(vp + (int64_t)jp * p.sn + E * sl + 8 * x);
            if constexpr (BIDIR) {
                nx.kf[x] = *reinterpret_cast<const uint4 *>(kp + (int64_t)jf * p.sn + E * sl + 8 * x);
                nx.vf[x] = *reinterpret_cast<const uint4 *>(vp + (int64_t)jf * p.sn + E * sl + 8 * x);
            }
        }
        if constexpr (GATED) {
            if (h > h0) nx.gl = glds[(h - h0) * TT + qi];   // head h0: after the gate prologue
        } else {
            nx.gl = p.gate[b * p.gsb + h * p.gsh + tq * p.gsn];
        }
    };
    auto stage = [&](const Next &nx, int buf) {
#pragma unroll
        for (int u = 0; u < BD::CH; ++u) {
            const int cid = tid + NT * u;
            const int r = cid / CPR, c = cid % CPR;
            if (r < BD::ROWS) {
                *reinterpret_cast<uint4 *>(&band[buf][0][r * ROWB + 16 * chunk_pos<D>(r, c)]) = nx.k[u];
                *reinterpret_cast<uint4 *>(&band[buf][1][r * ROWB + 16 * chunk_pos<D>(r, c)]) = nx.v[u];
            }
        }
    };

    const bool clamp_on = p.clamp > 0.0f;
    const float c2 = p.scale * kLog2e;
    Next cur, nxt;
    fetch(cur, h0);   // head h0's loads fly during the gate prologue
    if constexpr (GATED) {
        gate_tile(p, m, b, t0, h0, h1 - h0, reinterpret_cast<float *>(&band[0][0][0]), glds, true);
        cur.gl = glds[qi];
    }
    stage(cur, 0);
    __syncthreads();
    for (int h = h0; h < h1; ++h) {
        const int buf = (h - h0) & 1;
        if (h + 1 < h1) fetch(nxt, h + 1);
        const FusionBias fb = fusion_bias(cur.gl, clamp_on);
        // logit of one entry (log2 units) from this lane's dot-product part
        auto logit = [&](float part, float bias) {
            const float dot = sum8(part);
            return clamp_on ? fminf(fmaxf(dot * p.scale + bias, -p.clamp), p.clamp) * kLog2e
                            : __builtin_fmaf(dot, c2, bias * kLog2e);
        };
        constexpr int NW = BIDIR ? 2 * KMAX + 1 : KMAX + 1;   // window slots at most
        constexpr int NP = BIDIR ? 2 : 1;                     // partner slots
        const unsigned char *kb = band[buf][0];
        const unsigned char *vb = band[buf][1];
        // ---- scores: partners, then window slot s (row t - k + s, LDS row qi + s)
        float sc[NP + NW];
        int row[NW];
        {
            float part = 0.0f;
#pragma unroll
            for (int x = 0; x < E / 8; ++x) part = dot8(cur.q[x], cur.kp[x], part);
            sc[0] = has_p ? logit(part, fb.partner) : -INFINITY;
            if constexpr (BIDIR) {
                part = 0.0f;
#pragma unroll
                for (int x = 0; x < E / 8; ++x) part = dot8(cur.q[x], cur.kf[x], part);
                sc[1] = has_f ? logit(part, fb.partner) : -INFINITY;
            }
        }
#pragma unroll
        for (int s = 0; s < NW; ++s) {
            const int j = t - kw + s;
            const bool ok = s < nw && t_ok && j >= 0 && j < N;
            row[s] = ok ? qi + s : tq - rlo;   // a clamped row of the band otherwise
            float part = 0.0f;
#pragma unroll
            for (int x = 0; x < E / 8; ++x) {
                const int c = (E / 8) * sl + x;
                const uint4 kk =
                    *reinterpret_cast<const uint4 *>(kb + row[s] * ROWB + 16 * chunk_pos<D>(row[s], c));
                part = dot8(cur.q[x], kk, part);
            }
            sc[NP + s] = ok ? logit(part, fb.local) : -INFINITY;
        }
        // ---- softmax (the 8 lanes of a row hold identical scores)
        float mx = sc[0];
#pragma unroll
        for (int e = 1; e < NP + NW; ++e) mx = fmaxf(mx, sc[e]);
        mx = t_ok ? mx : 0.0f;   // every entry absent: keep the arithmetic finite
        float l = 0.0f, acc[E];
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] = 0.0f;
        {
            const float pp = __builtin_amdgcn_exp2f(sc[0] - mx);   // 0 for an absent entry
            l += pp;
#pragma unroll
            for (int x = 0; x < E / 8; ++x) axpy8(acc + 8 * x, pp, cur.vp[x]);
            if constexpr (BIDIR) {
                const float pf = __builtin_amdgcn_exp2f(sc[1] - mx);
                l += pf;
#pragma unroll
                for (int x = 0; x < E / 8; ++x) axpy8(acc + 8 * x, pf, cur.vf[x]);
            }
        }
#pragma unroll
        for (int s = 0; s < NW; ++s) {
            const float pr = __builtin_amdgcn_exp2f(sc[NP + s] - mx);
            l += pr;
#pragma unroll
            for (int x = 0; x < E / 8; ++x) {
                const int c = (E / 8) * sl + x;
                const uint4 vv =
                    *reinterpret_cast<const uint4 *>(vb + row[s] * ROWB + 16 * chunk_pos<D>(row[s], c));
                axpy8(acc + 8 * x, pr, vv);
            }
        }
        // normalise and store
        if (t_ok) {
            const float inv = 1.0f / l;
            __bf16 *op = (__bf16 *)p.out + b * p.osb + h * p.osh + (int64_t)t * p.osn + E * sl;
#pragma unroll
            for (int x = 0; x < E / 8; ++x) {
                bf16x8 o;
#pragma unroll
                for (int e = 0; e < 8; ++e) o[e] = (__bf16)(acc[8 * x + e] * inv);
                *reinterpret_cast<bf16x8 *>(op + 8 * x) = o;
            }
            if (p.lse && sl == 0) p.lse[((int64_t)b * p.H + h) * N + t] = (mx + __log2f(l)) * kLn2 + fb.lse_shift;
        }
        if (h + 1 < h1) {
            stage(nxt, buf ^ 1);
            cur = nxt;
        }
        __syncthreads();
    }
}

// The gate logits alone (bf16 operands, MFMA), one work-group per
// (b, 32 tokens, 32 heads).
__global__ __launch_bounds__(NT) void gate_bf16_kernel(FwdParams p, GateMlp m, int n_tt, int n_hb) {
    __shared__ float scratch[kGateScratch];
    __shared__ float glds[HG * TT];
    const int hb = blockIdx.x % n_hb;
    const int tt = (blockIdx.x / n_hb) % n_tt;
    const int b = blockIdx.x / (n_hb * n_tt);
    gate_tile(p, m, b, tt * TT, hb * HG, min(HG, p.H - hb * HG), scratch, glds, true);
}

// float32 operands: one thread per (b, h, t).
__global__ __launch_bounds__(NT) void gate_f32_kernel(FwdParams p, GateMlp m) {
    const int64_t x = (int64_t)blockIdx.x * NT + threadIdx.x;
    if (x >= (int64_t)p.B * p.H * p.N) return;
    const int t = (int)(x % p.N);
    const int64_t bh = x / p.N;
    const int h = (int)(bh % p.H), b = (int)(bh / p.H);
    const float *ur = (const float *)m.u + b * m.usb + (int64_t)t * m.usn;
    const float *wr = (const float *)m.w2 + (int64_t)h * m.dh;
    float s = 0.0f;
    for (int c = 0; c < m.dh; ++c) s += ur[c] * wr[c];
    m.gate_out[x] = s + (m.b2 ? m.b2[h] : 0.0f);
}

template <int D, bool BIDIR, bool GATED, int KMAX>
hipError_t launch_sk(const FwdParams &p, const GateMlp &m, hipStream_t stream) {
    const int n_tt = (p.N + TT - 1) / TT;
    // head groups: at least ceil(H / 32); more while the grid is small
    int n_hg = (p.H + HG - 1) / HG;
    while (n_hg < p.H && (int64_t)p.B * n_tt * n_hg < 2048) ++n_hg;
    const int64_t n_logical = (int64_t)p.B * n_tt * n_hg;
    const int64_t grid = xcd_grid(n_logical);
    return launch_kernel(smallk_bf16_kernel<D, BIDIR, GATED, KMAX>, dim3((unsigned)grid), dim3(NT), stream, p, m,
                         n_tt, n_hg, n_logical);
}

template <int D, bool BIDIR, bool GATED>
hipError_t launch_skk(const FwdParams &p, const GateMlp &m, hipStream_t stream) {
    if (p.k <= 4) return launch_sk<D, BIDIR, GATED, 4>(p, m, stream);
    if (p.k <= 8) return launch_sk<D, BIDIR, GATED, 8>(p, m, stream);
    return launch_sk<D, BIDIR, GATED, kSmallK>(p, m, stream);
}

template <int D, bool BIDIR>
hipError_t launch_skg(const FwdParams &p, const GateMlp *m, hipStream_t stream) {
    if (m) return launch_skk<D, BIDIR, true>(p, *m, stream);
    return launch_skk<D, BIDIR, false>(p, GateMlp{}, stream);
}

}  // namespace

hipError_t launch_forward_smallk(const FwdParams &p, const GateMlp *mlp, hipStream_t stream) {
    if ((int64_t)p.B * p.H * p.N == 0) return hipSuccess;
    if (p.D == 64) return p.causal ? launch_skg<64, false>(p, mlp, stream) : launch_skg<64, true>(p, mlp, stream);
    return p.causal ? launch_skg<128, false>(p, mlp, stream) : launch_skg<128, true>(p, mlp, stream);
}

hipError_t launch_gate_logits(const FwdParams &p, const GateMlp &mlp, int dtype, hipStream_t stream) {
    const int64_t rows = (int64_t)p.B * p.H * p.N;
    if (rows == 0) return hipSuccess;
    if (dtype == 1) {
        const int n_tt = (p.N + TT - 1) / TT, n_hb = (p.H + HG - 1) / HG;
        return launch_kernel(gate_bf16_kernel, dim3((unsigned)((int64_t)p.B * n_tt * n_hb)), dim3(NT), stream, p, mlp,
                             n_tt, n_hb);
    }
    return launch_kernel(gate_f32_kernel, dim3((unsigned)((rows + NT - 1) / NT)), dim3(NT), stream, p, mlp);
}

}  // namespace pi_attn
