// decode_bf16.hip -- one KV-cached decode step of causal pi-Attention,
// bf16 caches, fp32 arithmetic, D = 64 or 128.
//
// One work-group per (sequence s, head h); t = len_in[s].  The working set
// W_t (Sec. 3.5, eq. online_ws) is the cache window rows max(0,t-k)..t-1,
// the partner row t-pi (when pi > k and t >= pi) and the new row t itself,
// which is taken from k_new/v_new and also appended to the caches.
//
// The rows are split across the work-group's wavefronts in chunks.  Inside a
// wavefront, D/8 lanes cover one row with 16-byte loads, so one load
// instruction reads 64/(D/8) whole rows (coalesced).  Each lane keeps an
// 8-wide slice of q and of the output accumulator; a row's score is the sum
// of its D/8 lanes' partial dot products.  Every chunk issues all of its key
// and value loads before using any, to keep many bytes in flight.  Each
// wavefront runs its own online softmax; the wavefronts are merged in LDS
// at the end (max, rescaled sums).
#include "kernels.h"
#include "pi_common.h"

namespace pi_attn {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int WAVES = 4;
constexpr int NT = WAVES * 64;
constexpr int CH = 8;   // load instructions per chunk

__device__ inline uint4 ld16(const __bf16 *p) { return *reinterpret_cast<const uint4 *>(p); }

__device__ inline void to_f32(uint4 u, float f[8]) {
    const bf16x8 b = __builtin_bit_cast(bf16x8, u);
#pragma unroll
    for (int i = 0; i < 8; ++i) f[i] = (float)b[i];
}

template <int D, bool CLAMP>
__global__ __launch_bounds__(NT) void decode_bf16_kernel(DecodeParams p) {
    constexpr int LPR = D / 8;       // lanes per row
    constexpr int RPI = 64 / LPR;    // rows per load instruction
    constexpr int RPC = RPI * CH;    // rows per chunk

    __shared__ float s_m[WAVES], s_l[WAVES];
    __shared__ float s_acc[WAVES][D];

    const int64_t sh = blockIdx.x;
    const int s = (int)(sh / p.H), h = (int)(sh % p.H);
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int sub = lane % LPR, rg = lane / LPR;
    const int t = p.len_in[s];
    __bf16 *out = (__bf16 *)p.out + sh * D;

    if (t < 0 || t >= p.cap) {
        if (tid < D) out[tid] = (__bf16)NAN;
        if (tid == 0) {
            if (p.lse) p.lse[sh] = NAN;
            if (p.len_out && h == 0) p.len_out[s] = t;
        }
        return;
    }

    const __bf16 *kc = (const __bf16 *)p.k_cache + sh * (int64_t)p.cap * D;
    const __bf16 *vc = (const __bf16 *)p.v_cache + sh * (int64_t)p.cap * D;
    const __bf16 *kn = (const __bf16 *)p.k_new + sh * D;
    const __bf16 *vn = (const __bf16 *)p.v_new + sh * D;

    float qf[8];
    to_f32(ld16((const __bf16 *)p.q_new + sh * D + sub * 8), qf);

    const FusionBias fb = fusion_bias(p.gate[s * p.gss + h * p.gsh], CLAMP);
    const float c2 = p.scale * kLog2e;

    // Row list: i in [0, nwin) -> cache row lo + i; i == nwin -> partner
    // (if any); last -> the new row.
    const int lo = window_lo(t, p.k);
    const int nwin = t - lo;
    const int jp = partner_of(t, p.k, p.pi);
    const int nrows = nwin + (jp >= 0 ? 1 : 0) + 1;
    const int nchunks = (nrows + RPC - 1) / RPC;

    float m = -INFINITY, l = 0.0f;
    float acc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = 0.0f;

    for (int ch = w; ch < nchunks; ch += WAVES) {
        uint4 kr[CH], vr[CH];
        int ri[CH];
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const int i = ch * RPC + c * RPI + rg;
            ri[c] = i;
            const __bf16 *krow, *vrow;
            if (i < nwin) {
                krow = kc + (int64_t)(lo + i) * D;
                vrow = vc + (int64_t)(lo + i) * D;
            } else if (i == nwin && jp >= 0) {
                krow = kc + (int64_t)jp * D;
                vrow = vc + (int64_t)jp * D;
            } else {
                krow = kn;
                vrow = vn;
            }
            if (i < nrows) {
                kr[c] = ld16(krow + sub * 8);
                vr[c] = ld16(vrow + sub * 8);
            } else {
                kr[c] = make_uint4(0, 0, 0, 0);
                vr[c] = make_uint4(0, 0, 0, 0);
            }
        }
        float sc[CH];
        float cmax = -INFINITY;
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            float kf[8];
            to_f32(kr[c], kf);
            float part = 0.0f;
#pragma unroll
            for (int e = 0; e < 8; ++e) part += qf[e] * kf[e];
#pragma unroll
            for (int o = 1; o < LPR; o <<= 1) part += __shfl_xor(part, o);
            const int i = ri[c];
            const bool is_partner = (i == nwin) && jp >= 0;
            float v;
            if constexpr (CLAMP) {
                v = fminf(fmaxf(part * p.scale + (is_partner ? fb.partner : fb.local), -p.clamp), p.clamp) * kLog2e;
            } else {
                v = part * c2 + (is_partner ? fb.partner * kLog2e : 0.0f);
            }
            sc[c] = i < nrows ? v : -INFINITY;
            cmax = fmaxf(cmax, sc[c]);
        }
#pragma unroll
        for (int o = LPR; o < 64; o <<= 1) cmax = fmaxf(cmax, __shfl_xor(cmax, o));
        const float m_new = fmaxf(m, cmax);
        const float m_use = m_new == -INFINITY ? 0.0f : m_new;
        const float alpha = __builtin_amdgcn_exp2f(m - m_use);
        m = m_new;
        l *= alpha;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] *= alpha;
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const float pr = __builtin_amdgcn_exp2f(sc[c] - m_use);
            l += pr;
            float vf[8];
            to_f32(vr[c], vf);
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[e] += pr * vf[e];
        }
    }

    // Merge the row groups of the wavefront (lanes with the same sub).
#pragma unroll
    for (int o = LPR; o < 64; o <<= 1) {
        l += __shfl_xor(l, o);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] += __shfl_xor(acc[e], o);
    }
    if (rg == 0) {
#pragma unroll
        for (int e = 0; e < 8; ++e) s_acc[w][sub * 8 + e] = acc[e];
        if (sub == 0) {
            s_m[w] = m;
            s_l[w] = l;
        }
    }
    // Append the new key/value as cache row t (no row read above is row t).
    if (w == WAVES - 1 && lane < 2 * LPR) {
        const int which = lane / LPR, part = lane % LPR;
        const __bf16 *src = which ? vn : kn;
        __bf16 *dst = (__bf16 *)(which ? p.v_cache : p.k_cache) + (sh * (int64_t)p.cap + t) * D;
        *reinterpret_cast<uint4 *>(dst + part * 8) = ld16(src + part * 8);
    }
    __syncthreads();

    if (tid < D) {
        float M = -INFINITY;
#pragma unroll
        for (int i = 0; i < WAVES; ++i) M = fmaxf(M, s_m[i]);
        float L = 0.0f, o = 0.0f;
#pragma unroll
        for (int i = 0; i < WAVES; ++i) {
            const float f = s_m[i] == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(s_m[i] - M);
            L += s_l[i] * f;
            o += s_acc[i][tid] * f;
        }
        out[tid] = (__bf16)(o / L);
        if (tid == 0) {
            if (p.lse) p.lse[sh] = (M + __log2f(L)) * kLn2 + fb.lse_shift;
            if (p.len_out && h == 0) p.len_out[s] = t + 1;
        }
    }
}

template <int D, bool CLAMP>
hipError_t launch(const DecodeParams &p, hipStream_t stream) {
    const int64_t n = (int64_t)p.S * p.H;
    if (n == 0) return hipSuccess;
    return launch_kernel(decode_bf16_kernel<D, CLAMP>, dim3((unsigned)n), dim3(NT), stream, p);
}

}  // namespace

hipError_t launch_decode_bf16(const DecodeParams &p, hipStream_t stream) {
    const bool clamp = p.clamp > 0.0f;
    if (p.D == 64) return clamp ? launch<64, true>(p, stream) : launch<64, false>(p, stream);
    return clamp ? launch<128, true>(p, stream) : launch<128, false>(p, stream);
}

}  // namespace pi_attn
