// attn_f32.hip -- float32 forward and decode: one wavefront per query.
//
// Lane l holds elements l, l+64, ... of the D-vector.  The working set is
// visited entry by entry (partners first, then the window oldest to newest);
// each score is a wavefront-wide dot product, folded into a running max /
// running sum (online softmax) in the log2 domain.  This is the plain,
// correctness-first GPU path; the bf16 kernels are the fast ones.
#include "kernels.h"
#include "pi_common.h"

namespace pi_attn {

namespace {

__device__ inline float wave_sum(float x) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
    return x;
}

template <int D>
struct OnlineRow {
    static constexpr int E = D / 64;
    float q[E];
    float acc[E];
    float m = -INFINITY;   // running max, log2 domain
    float l = 0.0f;        // running sum of exp2(s - m)

    // One working-set entry: key row kj, value row vj, fused bias (natural log).
    __device__ inline void visit(const float *kj, const float *vj, float bias, float scale, float clamp, int lane) {
        float part = 0.0f;
#pragma unroll
        for (int e = 0; e < E; ++e) part += q[e] * kj[lane + 64 * e];
        float delta = wave_sum(part) * scale + bias;
        if (clamp > 0.0f) delta = fminf(fmaxf(delta, -clamp), clamp);
        float s = delta * kLog2e;
        float mn = fmaxf(m, s);
        float c = __builtin_amdgcn_exp2f(m - mn);   // m = -inf -> 0
        float pr = __builtin_amdgcn_exp2f(s - mn);
        l = l * c + pr;
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] = acc[e] * c + pr * vj[lane + 64 * e];
        m = mn;
    }
};

template <int D>
__global__ __launch_bounds__(256) void forward_f32_kernel(FwdParams p) {
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int64_t rows = (int64_t)p.B * p.H * p.N;
    if (row >= rows) return;
    const int t = (int)(row % p.N);
    const int64_t bh = row / p.N;
    const int h = (int)(bh % p.H), b = (int)(bh / p.H);
    const float *q = (const float *)p.q, *kk = (const float *)p.k_ptr, *v = (const float *)p.v;
    const int64_t base = b * p.sb + h * p.sh;

    OnlineRow<D> st;
#pragma unroll
    for (int e = 0; e < OnlineRow<D>::E; ++e) {
        st.q[e] = q[base + t * p.sn + lane + 64 * e];
        st.acc[e] = 0.0f;
    }
    const bool exact = p.clamp > 0.0f;
    const FusionBias fb = fusion_bias(p.gate[b * p.gsb + h * p.gsh + t * p.gsn], exact);

    const int jp = partner_of(t, p.k, p.pi);
    if (jp >= 0) st.visit(kk + base + jp * p.sn, v + base + jp * p.sn, fb.partner, p.scale, p.clamp, lane);
    const int jf = p.causal ? -1 : partner_fwd_of(t, p.k, p.pi, p.N);
    if (jf >= 0) st.visit(kk + base + jf * p.sn, v + base + jf * p.sn, fb.partner, p.scale, p.clamp, lane);
    const int hi = window_hi(t, p.k, p.N, p.causal);
    for (int j = window_lo(t, p.k); j <= hi; ++j)
        st.visit(kk + base + j * p.sn, v + base + j * p.sn, fb.local, p.scale, p.clamp, lane);

    float *out = (float *)p.out;
    const int64_t ob = b * p.osb + h * p.osh + t * p.osn;
    const float inv = 1.0f / st.l;
#pragma unroll
    for (int e = 0; e < OnlineRow<D>::E; ++e) out[ob + lane + 64 * e] = st.acc[e] * inv;
    if (p.lse && lane == 0) p.lse[row] = (st.m + __log2f(st.l)) * kLn2 + fb.lse_shift;
}

template <int D>
__global__ __launch_bounds__(256) void decode_f32_kernel(DecodeParams p) {
    const int lane = threadIdx.x & 63;
    const int64_t sh = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (sh >= (int64_t)p.S * p.H) return;
    const int s = (int)(sh / p.H), h = (int)(sh % p.H);
    const int t = p.len_in[s];
    float *out = (float *)p.out;
    if (t < 0 || t >= p.cap) {
        for (int e = lane; e < D; e += 64) out[sh * D + e] = NAN;
        if (lane == 0) {
            if (p.lse) p.lse[sh] = NAN;
            if (p.len_out && h == 0) p.len_out[s] = t;
        }
        return;
    }
    const float *qn = (const float *)p.q_new + sh * D;
    const float *kn = (const float *)p.k_new + sh * D;
    const float *vn = (const float *)p.v_new + sh * D;
    float *kc = (float *)p.k_cache + sh * (int64_t)p.cap * D;
    float *vc = (float *)p.v_cache + sh * (int64_t)p.cap * D;

    OnlineRow<D> st;
#pragma unroll
    for (int e = 0; e < OnlineRow<D>::E; ++e) {
        st.q[e] = qn[lane + 64 * e];
        st.acc[e] = 0.0f;
    }
    const bool exact = p.clamp > 0.0f;
    const FusionBias fb = fusion_bias(p.gate[s * p.gss + h * p.gsh], exact);

    const int jp = partner_of(t, p.k, p.pi);
    if (jp >= 0) st.visit(kc + (int64_t)jp * D, vc + (int64_t)jp * D, fb.partner, p.scale, p.clamp, lane);
    for (int j = window_lo(t, p.k); j < t; ++j)
        st.visit(kc + (int64_t)j * D, vc + (int64_t)j * D, fb.local, p.scale, p.clamp, lane);
    st.visit(kn, vn, fb.local, p.scale, p.clamp, lane);   // self: the new row t

    // Append the new key/value as cache row t (rows read above are all < t).
#pragma unroll
    for (int e = 0; e < OnlineRow<D>::E; ++e) {
        kc[(int64_t)t * D + lane + 64 * e] = kn[lane + 64 * e];
        vc[(int64_t)t * D + lane + 64 * e] = vn[lane + 64 * e];
    }
    const float inv = 1.0f / st.l;
#pragma unroll
    for (int e = 0; e < OnlineRow<D>::E; ++e) out[sh * D + lane + 64 * e] = st.acc[e] * inv;
    if (lane == 0) {
        if (p.lse) p.lse[sh] = (st.m + __log2f(st.l)) * kLn2 + fb.lse_shift;
        if (p.len_out && h == 0) p.len_out[s] = t + 1;
    }
}

}  // namespace

hipError_t launch_forward_f32(const FwdParams &p, hipStream_t stream) {
    int64_t rows = (int64_t)p.B * p.H * p.N;
    if (rows == 0) return hipSuccess;
    dim3 grid((unsigned)((rows + 3) / 4)), block(256);
    if (p.D == 64) return launch_kernel(forward_f32_kernel<64>, grid, block, stream, p);
    return launch_kernel(forward_f32_kernel<128>, grid, block, stream, p);
}

hipError_t launch_decode_f32(const DecodeParams &p, hipStream_t stream) {
    int64_t n = (int64_t)p.S * p.H;
    if (n == 0) return hipSuccess;
    dim3 grid((unsigned)((n + 3) / 4)), block(256);
    if (p.D == 64) return launch_kernel(decode_f32_kernel<64>, grid, block, stream, p);
    return launch_kernel(decode_f32_kernel<128>, grid, block, stream, p);
}

}  // namespace pi_attn
