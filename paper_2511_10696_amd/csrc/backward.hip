// backward.hip -- gradients of the full-sequence operator: one wavefront per
// row, fp32 arithmetic for float32 and bf16 inputs.
//
// For a loss L with dL/dy given, the weights are recomputed from the
// forward's lse as alpha^_tj = exp(delta_tj - lse_t), and
//   dp_tj    = <dL/dy_t, v_j>                    (eq. attn_adapt)
//   r_t      = sum_j alpha^_tj dp_tj = <dL/dy_t, y_t>
//   ddelta_tj = alpha^_tj (dp_tj - r_t)          (softmax Jacobian, eq. jac)
// with ddelta cut to 0 where the optional clamp saturates.  Then
//   dq_t = scale sum_j ddelta_tj k_j,  dk_j = scale sum_t ddelta_tj q_t,
//   dv_j = sum_t alpha^_tj dL/dy_t,
//   dg_t = sum_j ddelta_tj d(log omega_tj)/dg    (eqs. ddelta_da, dalpha_da)
// where d log alpha~/dg = (1 - 2 eps) a (1 - a) / alpha~ on the window and
// d log(1 - alpha~)/dg = -(1 - 2 eps) a (1 - a) / (1 - alpha~) on the partner,
// a = sigmoid(g).
//
// Row terms (float32): r_t from the forward output y (a wavefront per row).  Query
// pass: wavefront per (b, h, t), lane l holding elements l, l+64, ..., one
// sweep over W_t.  Key pass: wavefront per (b, h, j) over the queries whose
// working set holds j: t in [j, j + k] and, when pi > k, t = j + pi (causal);
// t in [j - k, j + k] and t = j -/+ pi (bidirectional).  These
// are the float32 kernels (every dot product a wavefront reduction); bf16
// inputs run the MFMA passes of backward_bf16.hip and backward_kv_bf16.hip.
#include "kernels.h"
#include "pi_common.h"
#include "smallk.h"

namespace pi_attn {

namespace {

__device__ inline float wave_sum(float x) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
    return x;
}

template <typename T>
__device__ inline float ld(const void *p, int64_t i) {
    if constexpr (sizeof(T) == 4) {
        return reinterpret_cast<const float *>(p)[i];
    } else {
        return (float)reinterpret_cast<const __bf16 *>(p)[i];
    }
}

// Prior derivatives of one gate logit (natural-log units).
struct GateGrad {
    float local, partner;
};

__device__ inline GateGrad gate_grad(float g) {
    const float a = 1.0f / (1.0f + __expf(-g));
    const float at = kGateEps + (1.0f - 2.0f * kGateEps) * a;
    const float c = (1.0f - 2.0f * kGateEps) * a * (1.0f - a);
    return GateGrad{c / at, -c / (1.0f - at)};
}

// Fused logit of one (t, j) pair from its partial dot product; `bias` and
// the clamp as in the forward.  Returns delta and sets `cut` when the clamp
// saturates.
__device__ inline float fused_logit(float dot, float scale, float bias, float clamp, bool &cut) {
    float d = dot * scale + bias;
    cut = false;
    if (clamp > 0.0f) {
        const float c = fminf(fmaxf(d, -clamp), clamp);
        cut = fabsf(c) >= clamp;
        d = c;
    }
    return d;
}

template <int D, typename T>
__global__ __launch_bounds__(256) void rowterm_kernel(BwdParams p) {
    const FwdParams &f = p.f;
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= (int64_t)f.B * f.H * f.N) return;
    const int t = (int)(row % f.N);
    const int64_t bh = row / f.N;
    const int h = (int)(bh % f.H), b = (int)(bh / f.H);
    const int64_t ob = b * p.osb + h * p.osh + t * p.osn;
    float part = 0.0f;
#pragma unroll
    for (int e = 0; e < D / 64; ++e) part += ld<T>(p.dout, ob + lane + 64 * e) * ld<T>(p.out, ob + lane + 64 * e);
    part = wave_sum(part);
    if (lane == 0) p.rowterm[row] = part;
}

template <int D, typename T>
__global__ __launch_bounds__(256) void backward_q_kernel(BwdParams p) {
    constexpr int E = D / 64;
    const FwdParams &f = p.f;
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= (int64_t)f.B * f.H * f.N) return;
    const int t = (int)(row % f.N);
    const int64_t bh = row / f.N;
    const int h = (int)(bh % f.H), b = (int)(bh / f.H);
    const int64_t base = b * f.sb + h * f.sh;
    const int64_t obase = b * p.osb + h * p.osh + t * p.osn;

    float q[E], go[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        q[e] = ld<T>(f.q, base + t * f.sn + lane + 64 * e);
        go[e] = ld<T>(p.dout, obase + lane + 64 * e);
    }
    const bool exact = f.clamp > 0.0f;
    const float g = f.gate[b * f.gsb + h * f.gsh + t * f.gsn];
    const FusionBias fb = fusion_bias(g, exact);
    const GateGrad gg = gate_grad(g);
    const float shift = fb.lse_shift - p.lse[row];   // alpha^ = exp(delta + shift)
    const int jp = partner_of(t, f.k, f.pi);
    const int jf = f.causal ? -1 : partner_fwd_of(t, f.k, f.pi, f.N);
    const int lo = window_lo(t, f.k), hi = window_hi(t, f.k, f.N, f.causal);

    // (weight, dp) of one working-set entry
    auto entry = [&](int j, float bias, float &w, float &dp, bool &cut) {
        float pk = 0.0f, pv = 0.0f;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            pk += q[e] * ld<T>(f.k_ptr, base + j * f.sn + lane + 64 * e);
            pv += go[e] * ld<T>(f.v, base + j * f.sn + lane + 64 * e);
        }
        const float delta = fused_logit(wave_sum(pk), f.scale, bias, f.clamp, cut);
        w = __expf(delta + shift);
        dp = wave_sum(pv);
    };

    const float r = p.rowterm[row];
    bool cut;
    float w, dp;

    float dq[E] = {};
    float dg = 0.0f;
    auto grad = [&](int j, float bias, float dlogw) {
        entry(j, bias, w, dp, cut);
        const float dd = cut ? 0.0f : w * (dp - r);
#pragma unroll
        for (int e = 0; e < E; ++e) dq[e] += dd * ld<T>(f.k_ptr, base + j * f.sn + lane + 64 * e);
        dg += dd * dlogw;
    };
    if (jp >= 0) grad(jp, fb.partner, gg.partner);
    if (jf >= 0) grad(jf, fb.partner, gg.partner);
    for (int j = lo; j <= hi; ++j) grad(j, fb.local, gg.local);

#pragma unroll
    for (int e = 0; e < E; ++e) p.dq[row * D + lane + 64 * e] = dq[e] * f.scale;
    if (lane == 0) p.dgate[row] = dg;
}

template <int D, typename T>
__global__ __launch_bounds__(256) void backward_kv_kernel(BwdParams p) {
    constexpr int E = D / 64;
    const FwdParams &f = p.f;
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= (int64_t)f.B * f.H * f.N) return;
    const int j = (int)(row % f.N);
    const int64_t bh = row / f.N;
    const int h = (int)(bh % f.H), b = (int)(bh / f.H);
    const int64_t base = b * f.sb + h * f.sh;
    const int64_t rbase = bh * f.N;   // row index of (b, h, 0)

    float kj[E], vj[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        kj[e] = ld<T>(f.k_ptr, base + j * f.sn + lane + 64 * e);
        vj[e] = ld<T>(f.v, base + j * f.sn + lane + 64 * e);
    }
    const bool exact = f.clamp > 0.0f;
    float dk[E] = {}, dv[E] = {};

    // Query t sees key j as a window entry (partner == false) or as its partner.
    auto visit = [&](int t, bool partner) {
        const FusionBias fb = fusion_bias(f.gate[b * f.gsb + h * f.gsh + t * f.gsn], exact);
        const int64_t ob = b * p.osb + h * p.osh + t * p.osn;
        float q[E], go[E], pk = 0.0f, pv = 0.0f;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            q[e] = ld<T>(f.q, base + t * f.sn + lane + 64 * e);
            go[e] = ld<T>(p.dout, ob + lane + 64 * e);
            pk += q[e] * kj[e];
            pv += go[e] * vj[e];
        }
        bool cut;
        const float delta = fused_logit(wave_sum(pk), f.scale, partner ? fb.partner : fb.local, f.clamp, cut);
        const float w = __expf(delta + fb.lse_shift - p.lse[rbase + t]);
        const float dp = wave_sum(pv);
        const float dd = cut ? 0.0f : w * (dp - p.rowterm[rbase + t]);
#pragma unroll
        for (int e = 0; e < E; ++e) {
            dk[e] += dd * q[e];
            dv[e] += w * go[e];
        }
    };
    // The windows holding j are symmetric to j's own: causal t in [j, j + k],
    // bidirectional t in [j - k, j + k].
    const int t_lo = f.causal ? j : window_lo(j, f.k);
    const int t_hi = window_hi(j, f.k, f.N, false);
    for (int t = t_lo; t <= t_hi; ++t) visit(t, false);
    // j is the partner t - pi of t = j + pi and, bidirectional, t + pi of t = j - pi.
    const int tp = partner_fwd_of(j, f.k, f.pi, f.N);
    if (tp >= 0) visit(tp, true);
    const int tm = f.causal ? -1 : partner_of(j, f.k, f.pi);
    if (tm >= 0) visit(tm, true);

#pragma unroll
    for (int e = 0; e < E; ++e) {
        p.dk[row * D + lane + 64 * e] = dk[e] * f.scale;
        p.dv[row * D + lane + 64 * e] = dv[e];
    }
}

template <int D, typename T>
hipError_t launch(const BwdParams &p, hipStream_t stream) {
    const int64_t rows = (int64_t)p.f.B * p.f.H * p.f.N;
    const dim3 grid((unsigned)((rows + 3) / 4)), block(256);
    hipError_t e;
    if constexpr (sizeof(T) == 2) {
        // the MFMA query pass computes its row terms and writes the exact ones
        e = launch_backward_q_bf16(p, stream);
        if (e != hipSuccess) return e;
        return launch_backward_kv_bf16(p, stream);
    }
    e = launch_kernel(rowterm_kernel<D, T>, grid, block, stream, p);
    if (e != hipSuccess) return e;
    e = launch_kernel(backward_q_kernel<D, T>, grid, block, stream, p);
    if (e != hipSuccess) return e;
    return launch_kernel(backward_kv_kernel<D, T>, grid, block, stream, p);
}

}  // namespace

namespace {

// One work-group per head: thread i sums entries t = i, i + 1024, ... of
// every batch row of the head into four fp64 partial sums (a fixed order,
// independent additions in flight), then a fixed-shape tree in LDS.
constexpr int kGateRedThreads = 1024;

__global__ __launch_bounds__(kGateRedThreads) void gate_grad_per_head_kernel(int B, int H, int N,
                                                                              const float *dgate, float *out) {
    __shared__ double part[kGateRedThreads];
    const int h = blockIdx.x;
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
    for (int b = 0; b < B; ++b) {
        const float *row = dgate + ((int64_t)b * H + h) * N;
        int64_t t = threadIdx.x;
        for (; t + 3 * kGateRedThreads < N; t += 4 * kGateRedThreads) {
#pragma unroll
            for (int u = 0; u < 4; ++u) acc[u] += (double)row[t + u * kGateRedThreads];
        }
        // at most three entries remain for this thread
#pragma unroll
        for (int u = 0; u < 3; ++u)
            if (t + u * kGateRedThreads < N) acc[u] += (double)row[t + u * kGateRedThreads];
    }
    part[threadIdx.x] = (acc[0] + acc[1]) + (acc[2] + acc[3]);
    __syncthreads();
    for (int w = kGateRedThreads / 2; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) out[h] = (float)part[0];
}

}  // namespace

hipError_t launch_gate_grad_per_head(int B, int H, int N, const float *dgate, float *out, hipStream_t stream) {
    if (H == 0) return hipSuccess;
    return launch_kernel(gate_grad_per_head_kernel, dim3((unsigned)H), dim3(kGateRedThreads), stream, B, H, N,
                         dgate, out);
}

hipError_t launch_backward(const BwdParams &p, hipStream_t stream) {
    if ((int64_t)p.f.B * p.f.H * p.f.N == 0) return hipSuccess;
    if (p.dtype == 1 && p.f.k <= kSmallK) return launch_backward_smallk(p, stream);
    if (p.dtype == 1) return p.f.D == 64 ? launch<64, __bf16>(p, stream) : launch<128, __bf16>(p, stream);
    return p.f.D == 64 ? launch<64, float>(p, stream) : launch<128, float>(p, stream);
}

}  // namespace pi_attn
