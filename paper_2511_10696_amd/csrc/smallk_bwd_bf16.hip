// smallk_bwd_bf16.hip -- backward of pi-Attention for a small window radius
// (k <= 16), bf16 inputs, fp32 arithmetic and fp32 gradients, D = 64 or
// 128, causal or bidirectional.  Same work decomposition as the
// small-window forward (smallk_bf16.hip): a work-group owns 32 rows of one
// batch row and a group of heads and loops over the heads; a row is handled
// by 8 lanes of D/8 dimensions; the working set is unrolled to the
// instantiation's window bound KMAX.
//
// Query pass (dq, gate gradient, row terms), per query t: the K and V rows of
// its window band are staged in LDS, the partners read from global memory;
// for every entry j of W_t
//   alpha^_tj = exp(delta_tj - lse_t),   dP_tj = <dL/dy_t, v_j>,
// then the exact row term r_t = sum_j alpha^_tj dP_tj (no rounding of the
// weights: nothing here goes through bf16 products), and
//   ddelta_tj = alpha^_tj (dP_tj - r_t)         (softmax Jacobian, Sec. 3.5 eq. jac)
//   dq_t = scale sum_j ddelta_tj k_j,
//   dg_t = sum_j ddelta_tj d(log omega_tj)/dg   (eqs. ddelta_da, dalpha_da),
// ddelta cut to 0 where the clamp saturates.  r_t is written as the row term.
//
// Key pass (dk, dv), per key j: the queries whose working set holds j are
// the window rows t = j .. j + k (bidirectional j - k .. j + k) -- Q and
// dL/dy rows staged in LDS with each row's lse, row term and gate biases --
// and the partner queries t = j + pi (bidirectional also j - pi), read from
// global memory:
//   dk_j = scale sum_t ddelta_tj q_t,   dv_j = sum_t alpha^_tj dL/dy_t.
#include "kernels.h"
#include "pi_common.h"
#include "smallk.h"
#include "smallk_common.h"

namespace pi_attn {

namespace {

using namespace sk;

// Prior derivatives of one gate logit: d log alpha~/dg and d log(1 - alpha~)/dg.
struct GateDeriv {
    float local, partner;
};

__device__ inline GateDeriv gate_deriv(float g) {
    const float a = 1.0f / (1.0f + __expf(-g));
    const float at = kGateEps + (1.0f - 2.0f * kGateEps) * a;
    const float c = (1.0f - 2.0f * kGateEps) * a * (1.0f - a);
    return GateDeriv{c / at, -c / (1.0f - at)};
}

// Work-group -> (b, tile, head group) with at least ceil(H / 32) groups and
// more while the grid is small (as in the forward).
struct Grid {
    int n_tt, n_hg;
    int64_t n_logical;
};

inline Grid make_grid(const FwdParams &f) {
    Grid g;
    g.n_tt = (f.N + TT - 1) / TT;
    g.n_hg = (f.H + HG - 1) / HG;
    while (g.n_hg < f.H && (int64_t)f.B * g.n_tt * g.n_hg < 2048) ++g.n_hg;
    g.n_logical = (int64_t)f.B * g.n_tt * g.n_hg;
    return g;
}

// Fused logit in log2 units of one entry from its dot product: clamped with
// the exact prior, or shifted (see fusion_bias); `cut` when it saturates.
__device__ inline float logit2(float dot, float bias, const FwdParams &f, bool clamp_on, bool &cut) {
    if (clamp_on) {
        const float dl = fminf(fmaxf(dot * f.scale + bias, -f.clamp), f.clamp);
        cut = fabsf(dl) >= f.clamp;
        return dl * kLog2e;
    }
    cut = false;
    return __builtin_fmaf(dot, f.scale * kLog2e, bias * kLog2e);
}

// ---------------------------------------------------------------------------
// query pass
// ---------------------------------------------------------------------------
template <int D, bool BIDIR, int KMAX>
__global__ __launch_bounds__(NT) void smallk_bwd_q_kernel(BwdParams bp, Grid gd) {
    using BD = Band<D, BIDIR, KMAX>;
    constexpr int E = BD::E, CPR = BD::CPR, ROWB = BD::ROWB;
    const FwdParams &p = bp.f;
    __shared__ alignas(16) unsigned char band[2][2][BD::ROWS * ROWB];   // [buffer][K, V]
    const int64_t logical = xcd_remap(blockIdx.x, gd.n_logical);
    if (logical < 0) return;
    const int hg = (int)(logical % gd.n_hg);
    const int tt = (int)((logical / gd.n_hg) % gd.n_tt);
    const int b = (int)(logical / ((int64_t)gd.n_hg * gd.n_tt));
    const int N = p.N, kw = p.k, pi = p.pi;
    const int hpg = (p.H + gd.n_hg - 1) / gd.n_hg;
    const int h0 = hg * hpg, h1 = min(p.H, h0 + hpg);
    if (h0 >= h1) return;
    const int t0 = tt * TT;
    const int tid = threadIdx.x;
    const int qi = tid >> 3, sl = tid & 7;
    const int t = t0 + qi;
    const bool t_ok = t < N;
    const int tq = t_ok ? t : N - 1;
    const int rlo = t0 - kw;
    const int lo = max(0, rlo);
    const int hi = BIDIR ? (int)min((int64_t)t0 + TT + kw, (int64_t)N) : min(t0 + TT, N);
    const int rowb_g = (int)(2 * p.sn);
    const int nw = BIDIR ? 2 * kw + 1 : kw + 1;
    const bool has_p = t_ok && partner_enabled(kw, pi) && t - pi >= 0;
    const bool has_f = BIDIR && t_ok && partner_fwd_of(t, kw, pi, N) >= 0;
    const bool clamp_on = p.clamp > 0.0f;

    struct Next {
        uint4 k[BD::CH], v[BD::CH];
        uint4 q[E / 8], o[E / 8];
        uint4 kp[E / 8], vp[E / 8], kf[E / 8], vf[E / 8];
        float gl, lse;
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
            const int off = (gr >= lo && gr < hi && r < BD::ROWS) ? (gr - lo) * rowb_g + 16 * c : (hi - lo) * rowb_g;
            nx.k[u] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rk, off, 0, 0));
            nx.v[u] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rv, off, 0, 0));
        }
        const __bf16 *qrow = (const __bf16 *)p.q + base + (int64_t)tq * p.sn + E * sl;
        const __bf16 *orow = (const __bf16 *)bp.dout + b * bp.osb + h * bp.osh + (int64_t)tq * bp.osn + E * sl;
        const int jp = has_p ? t - pi : tq, jf = has_f ? t + pi : tq;
#pragma unroll
        for (int x = 0; x < E / 8; ++x) {
            nx.q[x] = *reinterpret_cast<const uint4 *>(qrow + 8 * x);
            nx.o[x] = *reinterpret_cast<const uint4 *>(orow + 8 * x);
            nx.kp[x] = *reinterpret_cast<const uint4 *>(kp + (int64_t)jp * p.sn + E * sl + 8 * x);
            nx.vp[x] = *reinterpret_cast<const uint4 *>(vp + (int64_t)jp * p.sn + E * sl + 8 * x);
            if constexpr (BIDIR) {
                nx.kf[x] = *reinterpret_cast<const uint4 *>(kp + (int64_t)jf * p.sn + E * sl + 8 * x);
                nx.vf[x] = *reinterpret_cast<const uint4 *>(vp + (int64_t)jf * p.sn + E * sl + 8 * x);
            }
        }
        nx.gl = p.gate[b * p.gsb + h * p.gsh + tq * p.gsn];
        nx.lse = bp.lse[((int64_t)b * p.H + h) * N + tq];
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
    // this lane's part of a row held in the band (LDS row r)
    auto band_chunk = [&](int buf, int which, int r, int x) {
        const int c = (E / 8) * sl + x;
        return *reinterpret_cast<const uint4 *>(&band[buf][which][r * ROWB + 16 * chunk_pos<D>(r, c)]);
    };

    Next cur, nxt;
    fetch(cur, h0);
    stage(cur, 0);
    __syncthreads();
    for (int h = h0; h < h1; ++h) {
        const int buf = (h - h0) & 1;
        if (h + 1 < h1) fetch(nxt, h + 1);
        const FusionBias fb = fusion_bias(cur.gl, clamp_on);
        const GateDeriv gdv = gate_deriv(cur.gl);
        const float lse2 = (cur.lse - fb.lse_shift) * kLog2e;
        // ---- one pass over W_t.  With w_j = alpha^_j, or 0 where the clamp
        // saturates: dq = sum w dP k - r sum w k, dg = sum w dP dlog - r sum w dlog,
        // so that r is not needed before the pass.
        float X[E], Y[E], r = 0.0f, ga = 0.0f, gb = 0.0f;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            X[e] = 0.0f;
            Y[e] = 0.0f;
        }
        auto entry = [&](bool ok, const uint4 *kc, const uint4 *vc, float bias, float dlog) {
            float pk = 0.0f, pv = 0.0f;
#pragma unroll
            for (int x = 0; x < E / 8; ++x) {
                pk = dot8(cur.q[x], kc[x], pk);
                pv = dot8(cur.o[x], vc[x], pv);
            }
            bool cut;
            const float s2 = logit2(sum8(pk), bias, p, clamp_on, cut);
            const float a = ok ? __builtin_amdgcn_exp2f(s2 - lse2) : 0.0f;
            const float dp = sum8(pv);
            r += a * dp;
            const float w = cut ? 0.0f : a;
            const float wd = w * dp;
            ga += wd * dlog;
            gb += w * dlog;
#pragma unroll
            for (int x = 0; x < E / 8; ++x) {
                axpy8(X + 8 * x, wd, kc[x]);
                axpy8(Y + 8 * x, w, kc[x]);
            }
        };
        entry(has_p, cur.kp, cur.vp, fb.partner, gdv.partner);
        if constexpr (BIDIR) entry(has_f, cur.kf, cur.vf, fb.partner, gdv.partner);
#pragma unroll 2
        for (int s = 0; s < nw; ++s) {
            const int j = t - kw + s;
            const bool ok = t_ok && j >= 0 && j < N;
            const int rw = ok ? qi + s : tq - rlo;
            uint4 kc[E / 8], vc[E / 8];
#pragma unroll
            for (int x = 0; x < E / 8; ++x) {
                kc[x] = band_chunk(buf, 0, rw, x);
                vc[x] = band_chunk(buf, 1, rw, x);
            }
            entry(ok, kc, vc, fb.local, gdv.local);
        }
        float dq[E];
#pragma unroll
        for (int e = 0; e < E; ++e) dq[e] = X[e] - r * Y[e];
        const float dg = ga - r * gb;
        if (t_ok) {
            const int64_t grow = ((int64_t)b * p.H + h) * N + t;
            float *dqp = bp.dq + grow * D + E * sl;
#pragma unroll
            for (int x = 0; x < E / 4; ++x)
                *reinterpret_cast<float4 *>(dqp + 4 * x) =
                    make_float4(dq[4 * x] * p.scale, dq[4 * x + 1] * p.scale, dq[4 * x + 2] * p.scale,
                                dq[4 * x + 3] * p.scale);
            if (sl == 0) {
                bp.dgate[grow] = dg;
                bp.rowterm[grow] = r;
            }
        }
        if (h + 1 < h1) {
            stage(nxt, buf ^ 1);
            cur = nxt;
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// key pass
// ---------------------------------------------------------------------------
template <int D, bool BIDIR, int KMAX>
__global__ __launch_bounds__(NT) void smallk_bwd_kv_kernel(BwdParams bp, Grid gd) {
    using BD = Band<D, BIDIR, KMAX>;
    constexpr int E = BD::E, CPR = BD::CPR, ROWB = BD::ROWB;
    const FwdParams &p = bp.f;
    __shared__ alignas(16) unsigned char band[2][2][BD::ROWS * ROWB];   // [buffer][Q, dL/dy]
    __shared__ float rowf[2][4][BD::ROWS];   // [buffer][lse2, r, local bias2, partner bias2]
    const int64_t logical = xcd_remap(blockIdx.x, gd.n_logical);
    if (logical < 0) return;
    const int hg = (int)(logical % gd.n_hg);
    const int tt = (int)((logical / gd.n_hg) % gd.n_tt);
    const int b = (int)(logical / ((int64_t)gd.n_hg * gd.n_tt));
    const int N = p.N, kw = p.k, pi = p.pi;
    const int hpg = (p.H + gd.n_hg - 1) / gd.n_hg;
    const int h0 = hg * hpg, h1 = min(p.H, h0 + hpg);
    if (h0 >= h1) return;
    const int j0 = tt * TT;
    const int tid = threadIdx.x;
    const int ki = tid >> 3, sl = tid & 7;   // key of the tile, lane within its row
    const int j = j0 + ki;
    const bool j_ok = j < N;
    const int jq = j_ok ? j : N - 1;
    // query band: LDS row r <-> query row qlo + r; loaded rows [lo, hi)
    const int qlo = BIDIR ? j0 - kw : j0;
    const int lo = max(0, qlo);
    const int hi = (int)min((int64_t)j0 + TT + kw, (int64_t)N);
    const int rowq_g = (int)(2 * p.sn), rowo_g = (int)(2 * bp.osn);
    const int nw = BIDIR ? 2 * kw + 1 : kw + 1;
    // partner queries: j is the partner t - pi of t = j + pi, and (bidirectional)
    // the partner t + pi of t = j - pi
    const bool has_p = j_ok && partner_fwd_of(j, kw, pi, N) >= 0;
    const bool has_f = BIDIR && j_ok && partner_of(j, kw, pi) >= 0;
    const int tp = has_p ? j + pi : jq, tf = has_f ? j - pi : jq;
    const bool clamp_on = p.clamp > 0.0f;

    struct Next {
        uint4 q[BD::CH], o[BD::CH];
        uint4 kj[E / 8], vj[E / 8];
        uint4 qp[E / 8], op[E / 8], qf[E / 8], of[E / 8];
        float rg, rl, rr;        // this thread's staged row: gate, lse, row term
        float pg, pl, pr;        // partner query t = j + pi
        float fg, fl, fr;        // partner query t = j - pi
    };
    auto fetch = [&](Next &nx, int h) {
        const int64_t base = b * p.sb + h * p.sh;
        const int64_t obase = b * bp.osb + h * bp.osh;
        const int64_t rbase = ((int64_t)b * p.H + h) * N;
        const __bf16 *qp = (const __bf16 *)p.q + base;
        const __bf16 *op = (const __bf16 *)bp.dout + obase;
        const __amdgpu_buffer_rsrc_t rq =
            __builtin_amdgcn_make_buffer_rsrc((void *)(qp + (int64_t)lo * p.sn), (short)0, (hi - lo) * rowq_g, 0x00020000);
        const __amdgpu_buffer_rsrc_t ro = __builtin_amdgcn_make_buffer_rsrc(
            (void *)(op + (int64_t)lo * bp.osn), (short)0, (hi - lo) * rowo_g, 0x00020000);
#pragma unroll
        for (int u = 0; u < BD::CH; ++u) {
            const int cid = tid + NT * u;
            const int r = cid / CPR, c = cid % CPR;
            const int gr = qlo + r;
            const bool in = gr >= lo && gr < hi && r < BD::ROWS;
            const int offq = in ? (gr - lo) * rowq_g + 16 * c : (hi - lo) * rowq_g;
            const int offo = in ? (gr - lo) * rowo_g + 16 * c : (hi - lo) * rowo_g;
            nx.q[u] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rq, offq, 0, 0));
            nx.o[u] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(ro, offo, 0, 0));
        }
        {   // per-row scalars of staged row tid (rows outside [lo, hi) read row lo)
            const int gr = qlo + tid;
            const int rc = (gr >= lo && gr < hi) ? gr : lo;
            nx.rg = p.gate[b * p.gsb + h * p.gsh + rc * p.gsn];
            nx.rl = bp.lse[rbase + rc];
            nx.rr = bp.rowterm[rbase + rc];
        }
        const __bf16 *kp = (const __bf16 *)p.k_ptr + base;
        const __bf16 *vp = (const __bf16 *)p.v + base;
#pragma unroll
        for (int x = 0; x < E / 8; ++x) {
            nx.kj[x] = *reinterpret_cast<const uint4 *>(kp + (int64_t)jq * p.sn + E * sl + 8 * x);
            nx.vj[x] = *reinterpret_cast<const uint4 *>(vp + (int64_t)jq * p.sn + E * sl + 8 * x);
            nx.qp[x] = *reinterpret_cast<const uint4 *>(qp + (int64_t)tp * p.sn + E * sl + 8 * x);
            nx.op[x] = *reinterpret_cast<const uint4 *>(op + (int64_t)tp * bp.osn + E * sl + 8 * x);
            if constexpr (BIDIR) {
                nx.qf[x] = *reinterpret_cast<const uint4 *>(qp + (int64_t)tf * p.sn + E * sl + 8 * x);
                nx.of[x] = *reinterpret_cast<const uint4 *>(op + (int64_t)tf * bp.osn + E * sl + 8 * x);
            }
        }
        nx.pg = p.gate[b * p.gsb + h * p.gsh + tp * p.gsn];
        nx.pl = bp.lse[rbase + tp];
        nx.pr = bp.rowterm[rbase + tp];
        if constexpr (BIDIR) {
            nx.fg = p.gate[b * p.gsb + h * p.gsh + tf * p.gsn];
            nx.fl = bp.lse[rbase + tf];
            nx.fr = bp.rowterm[rbase + tf];
        }
    };
    auto stage = [&](const Next &nx, int buf) {
#pragma unroll
        for (int u = 0; u < BD::CH; ++u) {
            const int cid = tid + NT * u;
            const int r = cid / CPR, c = cid % CPR;
            if (r < BD::ROWS) {
                *reinterpret_cast<uint4 *>(&band[buf][0][r * ROWB + 16 * chunk_pos<D>(r, c)]) = nx.q[u];
                *reinterpret_cast<uint4 *>(&band[buf][1][r * ROWB + 16 * chunk_pos<D>(r, c)]) = nx.o[u];
            }
        }
        if (tid < BD::ROWS) {
            const FusionBias fb = fusion_bias(nx.rg, clamp_on);
            rowf[buf][0][tid] = (nx.rl - fb.lse_shift) * kLog2e;
            rowf[buf][1][tid] = nx.rr;
            rowf[buf][2][tid] = fb.local;
            rowf[buf][3][tid] = fb.partner;
        }
    };
    auto band_chunk = [&](int buf, int which, int r, int x) {
        const int c = (E / 8) * sl + x;
        return *reinterpret_cast<const uint4 *>(&band[buf][which][r * ROWB + 16 * chunk_pos<D>(r, c)]);
    };

    Next cur, nxt;
    fetch(cur, h0);
    stage(cur, 0);
    __syncthreads();
    for (int h = h0; h < h1; ++h) {
        const int buf = (h - h0) & 1;
        if (h + 1 < h1) fetch(nxt, h + 1);
        float dk[E], dv[E];
#pragma unroll
        for (int e = 0; e < E; ++e) {
            dk[e] = 0.0f;
            dv[e] = 0.0f;
        }
        // one query t of key j: its q and dL/dy chunks, lse2, row term and prior bias
        auto visit = [&](bool ok, const uint4 *qc, const uint4 *oc, float lse2, float rt, float bias) {
            float pk = 0.0f, pv = 0.0f;
#pragma unroll
            for (int x = 0; x < E / 8; ++x) {
                pk = dot8(qc[x], cur.kj[x], pk);
                pv = dot8(oc[x], cur.vj[x], pv);
            }
            bool cut;
            const float s2 = logit2(sum8(pk), bias, p, clamp_on, cut);
            const float a = ok ? __builtin_amdgcn_exp2f(s2 - lse2) : 0.0f;
            const float dd = cut ? 0.0f : a * (sum8(pv) - rt);
#pragma unroll
            for (int x = 0; x < E / 8; ++x) {
                axpy8(dk + 8 * x, dd, qc[x]);
                axpy8(dv + 8 * x, a, oc[x]);
            }
        };
        {   // partner queries
            const FusionBias fp = fusion_bias(cur.pg, clamp_on);
            visit(has_p, cur.qp, cur.op, (cur.pl - fp.lse_shift) * kLog2e, cur.pr, fp.partner);
            if constexpr (BIDIR) {
                const FusionBias ff = fusion_bias(cur.fg, clamp_on);
                visit(has_f, cur.qf, cur.of, (cur.fl - ff.lse_shift) * kLog2e, cur.fr, ff.partner);
            }
        }
        // window queries: slot s holds query qlo + ki + s (causal: j + s)
#pragma unroll 2
        for (int s = 0; s < nw; ++s) {
            const int tw = j - (BIDIR ? kw : 0) + s;
            const bool ok = j_ok && tw >= 0 && tw < N;
            const int r = ok ? ki + s : jq - qlo;   // a loaded row otherwise
            uint4 qc[E / 8], oc[E / 8];
#pragma unroll
            for (int x = 0; x < E / 8; ++x) {
                qc[x] = band_chunk(buf, 0, r, x);
                oc[x] = band_chunk(buf, 1, r, x);
            }
            visit(ok, qc, oc, rowf[buf][0][r], rowf[buf][1][r], rowf[buf][2][r]);
        }
        if (j_ok) {
            const int64_t grow = ((int64_t)b * p.H + h) * N + j;
            float *dkp = bp.dk + grow * D + E * sl;
            float *dvp = bp.dv + grow * D + E * sl;
#pragma unroll
            for (int x = 0; x < E / 4; ++x) {
                *reinterpret_cast<float4 *>(dkp + 4 * x) =
                    make_float4(dk[4 * x] * p.scale, dk[4 * x + 1] * p.scale, dk[4 * x + 2] * p.scale,
                                dk[4 * x + 3] * p.scale);
                *reinterpret_cast<float4 *>(dvp + 4 * x) = make_float4(dv[4 * x], dv[4 * x + 1], dv[4 * x + 2], dv[4 * x + 3]);
            }
        }
        if (h + 1 < h1) {
            stage(nxt, buf ^ 1);
            cur = nxt;
        }
        __syncthreads();
    }
}

template <int D, bool BIDIR, int KMAX>
hipError_t launch_kmax(const BwdParams &p, hipStream_t stream) {
    const Grid gd = make_grid(p.f);
    const int64_t grid = xcd_grid(gd.n_logical);
    hipError_t e =
        launch_kernel(smallk_bwd_q_kernel<D, BIDIR, KMAX>, dim3((unsigned)grid), dim3(NT), stream, p, gd);
    if (e != hipSuccess) return e;
    return launch_kernel(smallk_bwd_kv_kernel<D, BIDIR, KMAX>, dim3((unsigned)grid), dim3(NT), stream, p, gd);
}

template <int D, bool BIDIR>
hipError_t launch_mode(const BwdParams &p, hipStream_t stream) {
    if (p.f.k <= 4) return launch_kmax<D, BIDIR, 4>(p, stream);
    if (p.f.k <= 8) return launch_kmax<D, BIDIR, 8>(p, stream);
    return launch_kmax<D, BIDIR, kSmallK>(p, stream);
}

}  // namespace

hipError_t launch_backward_smallk(const BwdParams &p, hipStream_t stream) {
    if ((int64_t)p.f.B * p.f.H * p.f.N == 0) return hipSuccess;
    if (p.f.D == 64) return p.f.causal ? launch_mode<64, false>(p, stream) : launch_mode<64, true>(p, stream);
    return p.f.causal ? launch_mode<128, false>(p, stream) : launch_mode<128, true>(p, stream);
}

}  // namespace pi_attn
