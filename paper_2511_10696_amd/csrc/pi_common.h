// pi_common.h -- working-set enumeration and fusion prior shared by every
// kernel of the library and by pi_attn_index_set, so that the exported index
// set is the one the attention kernels use; the XCD-aware work-group order and
// the direct global-to-LDS fetch the MFMA kernels share.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pi_attn {

// Gate clip of Variant 3 (Sec. 3.5): alpha~ = eps + (1 - 2 eps) sigmoid(g).
constexpr float kGateEps = 1e-4f;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Window N_r(t) (Sec. 3.2, eq. Nr): j in [window_lo, window_hi], where the
// causal window ends at t and the bidirectional one at min(t + k, n - 1).
__host__ __device__ inline int window_lo(int t, int k) { return t - k > 0 ? t - k : 0; }

__host__ __device__ inline int window_hi(int t, int k, int n, bool causal) {
    if (causal) return t;
    return k >= n - 1 - t ? n - 1 : t + k;
}

// Partner slots exist only when t -/+ pi can lie outside the window.
__host__ __device__ inline bool partner_enabled(int k, int pi) { return pi > k; }

// Partner N_pi(t) = {t - pi} (Sec. 3.4, eq. Npi); -1 when absent.
__host__ __device__ inline int partner_of(int t, int k, int pi) {
    return (partner_enabled(k, pi) && t >= pi) ? t - pi : -1;
}

// The second partner t + pi of the bidirectional mode (App. B,
// hyper-parameter table); -1 when absent.
__host__ __device__ inline int partner_fwd_of(int t, int k, int pi, int n) {
    return (partner_enabled(k, pi) && pi < n - t) ? t + pi : -1;
}

// Window slots per query: offsets -k..0 (causal) or -k..k (bidirectional).
__host__ __device__ inline int64_t window_slots(int k, bool causal) {
    return causal ? (int64_t)k + 1 : 2 * (int64_t)k + 1;
}

// Slots per query: the window slots, then t - pi, then (bidirectional) t + pi.
__host__ __device__ inline int64_t ws_width(int k, int pi, bool causal) {
    return window_slots(k, causal) + (partner_enabled(k, pi) ? (causal ? 1 : 2) : 0);
}

// Slot s of W_t (sequence length n) in the exported layout; -1 for an
// absent entry.  Requires ws_width(k, pi, causal) to fit in int.
__host__ __device__ inline int ws_slot(int t, int s, int k, int pi, int n, bool causal) {
    const int nw = (int)window_slots(k, causal);
    if (s < nw) {
        const int j = t - k + s;
        return (j >= 0 && j < n) ? j : -1;
    }
    if (s == nw) return partner_of(t, k, pi);
    return partner_fwd_of(t, k, pi, n);
}

// Per-query fusion biases, natural-log units.
//   exact:    local = log alpha~, partner = log(1 - alpha~)
//   shifted:  local = 0,          partner = log(1 - alpha~) - log alpha~
// The shifted form differs from the exact one by the common log alpha~ on
// every entry of W_t, which the softmax removes; lse adds it back.
struct FusionBias {
    float local;
    float partner;
    float lse_shift;
};

__device__ inline FusionBias fusion_bias(float g, bool exact) {
    float a = 1.0f / (1.0f + __expf(-g));
    float at = kGateEps + (1.0f - 2.0f * kGateEps) * a;
    float ll = __logf(at);
    float lp = __logf(1.0f - at);
    FusionBias fb;
    if (exact) {
        fb.local = ll;
        fb.partner = lp;
        fb.lse_shift = 0.0f;
    } else {
        fb.local = 0.0f;
        fb.partner = lp - ll;
        fb.lse_shift = ll;
    }
    return fb;
}

// XCD-aware work-group order.  Consecutive work-group ids are dispatched
// round-robin over the 8 XCDs; this remaps them so that each XCD receives a
// contiguous range of logical tiles (neighbouring query tiles share most of
// their keys, which then stay in that XCD's L2).  The grid is padded to a
// multiple of 8; ids mapping past n_logical return -1.
constexpr int kNumXcd = 8;

__device__ inline int64_t xcd_remap(int64_t bid, int64_t n_logical) {
    int64_t per = (n_logical + kNumXcd - 1) / kNumXcd;
    int64_t logical = (bid % kNumXcd) * per + bid / kNumXcd;
    return logical < n_logical ? logical : -1;
}

inline int64_t xcd_grid(int64_t n_logical) {
    int64_t per = (n_logical + kNumXcd - 1) / kNumXcd;
    return per * kNumXcd;
}

// ---- direct global-to-LDS tile fetch ---------------------------------------
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

constexpr int kOutOfRange = 1 << 30;   // past any tile range the descriptors describe

// Raw buffer descriptor over nbytes from base (stride 0; word 3 is the gfx9
// raw-buffer format: 32-bit data, range checked).
__device__ inline u32x4 raw_rsrc(const void *base, int nbytes) {
    const unsigned long long a = (unsigned long long)base;
    u32x4 r;
    r.x = __builtin_amdgcn_readfirstlane((unsigned)a);
    r.y = __builtin_amdgcn_readfirstlane((unsigned)(a >> 32) & 0xffffu);
    r.z = __builtin_amdgcn_readfirstlane((unsigned)nbytes);
    r.w = 0x00020000u;
    return r;
}

// One 16-byte-per-lane buffer load into LDS at lds + 16 * lane.  Issued as
// inline asm: the compiler then keeps no count of it (its own waits for
// LDS reads after such a load would wait for every fetch in flight); the
// kernel waits for it with an explicit counter before the barrier that
// publishes the tile, and reads the buffer only after that barrier and an
// LDS acquire fence.  No memory clobber: the volatile asm stays after the
// barrier that frees its buffer (both have side effects), and a clobber
// would force every object whose address the kernel takes into private
// memory.
__device__ inline void lds_fetch16(u32x4 rsrc, int voff, void *lds) {
    const unsigned m0 = __builtin_amdgcn_readfirstlane(
        (unsigned)(uintptr_t)(__attribute__((address_space(3))) void *)lds);
    asm volatile("buffer_load_dwordx4 %0, %1, 0 offen lds" ::"v"(voff), "s"(rsrc), "{m0}"(m0));
}

}  // namespace pi_attn
