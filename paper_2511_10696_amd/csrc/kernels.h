// kernels.h -- launch parameters and host launchers of the HIP kernels.
// The C ABI (api.hip) validates arguments and calls these; they only launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace pi_attn {

// Launch through hipLaunchKernel so the launch status is returned directly
// (no reliance on the per-thread last-error state).  Arguments convert to the
// kernel's parameter types.
template <typename... KArgs>
inline hipError_t launch_kernel(void (*kernel)(KArgs...), dim3 grid, dim3 block, hipStream_t stream,
                                typename std::common_type<KArgs>::type... args) {
    void *argv[] = {static_cast<void *>(&args)...};
    return hipLaunchKernel(reinterpret_cast<const void *>(kernel), grid, block, argv, 0, stream);
}

struct FwdParams {
    int B, H, N, D, k, pi;
    int causal;                     // 1: causal window and t - pi; 0: bidirectional, t -/+ pi
    const void *q, *k_ptr, *v;
    int64_t sb, sh, sn;             // element strides shared by q, k, v
    const float *gate;
    int64_t gsb, gsh, gsn;          // element strides of the gate logits
    float scale, clamp;             // clamp <= 0: off
    void *out;
    int64_t osb, osh, osn;
    float *lse;                     // [B][H][N] or nullptr
    // Sequence shard (the banded bf16 forward only): q/out/lse/gate row i is
    // absolute position qpos0 + i, k/v row i is kvpos0 + i, k/v rows end at
    // kvend, the sequence has nseq positions.  A whole sequence: 0, 0, N, N.
    int qpos0, kvpos0, kvend, nseq;
    int qend;                       // backward key pass: query rows held end at qend (a whole sequence: N)
    int64_t ksb, ksh, ksn;          // element strides of k and v (a whole sequence: sb, sh, sn)
};

struct DecodeParams {
    int S, H, D, cap, k, pi;
    const int32_t *len_in;
    int32_t *len_out;               // nullptr: not written
    const void *q_new, *k_new, *v_new;   // [S][H][D]
    void *k_cache, *v_cache;        // [S][H][cap][D]
    const float *gate;
    int64_t gss, gsh;
    float scale, clamp;
    void *out;                      // [S][H][D]
    float *lse;                     // [S][H] or nullptr
};

struct BwdParams {
    FwdParams f;                    // inputs as for the forward (out/lse unused)
    int dtype;                      // 0 = float32, 1 = bf16 (q, k, v, dout)
    const float *lse;               // [B][H][N]
    const void *out, *dout;         // forward output and dL/dy
    int64_t osb, osh, osn;          // element strides of out and dout
    float *dq, *dk, *dv;            // [B][H][N][D] contiguous
    float *dgate, *rowterm;         // [B][H][N] contiguous
};

hipError_t launch_index_set(int n, int k, int pi, bool causal, int32_t *idx, hipStream_t stream);

// Reference-style fp32 kernels: one wavefront per query, W_t visited entry by
// entry with an online softmax.  Correctness path for float32 data.
hipError_t launch_forward_f32(const FwdParams &p, hipStream_t stream);
hipError_t launch_decode_f32(const DecodeParams &p, hipStream_t stream);

// bf16 banded MFMA forward (D = 64 or 128).
hipError_t launch_forward_bf16(const FwdParams &p, hipStream_t stream);

// bf16 decode step, working set split across wavefronts (D = 64 or 128).
hipError_t launch_decode_bf16(const DecodeParams &p, hipStream_t stream);

// Backward: the row terms <dL/dy_t, y_t>, a query pass (dq, dgate) and a
// key pass (dk, dv).
hipError_t launch_backward(const BwdParams &p, hipStream_t stream);

// out[h] = sum over b and t of dgate[b][h][t] (fixed order, fp64 sums).
hipError_t launch_gate_grad_per_head(int B, int H, int N, const float *dgate, float *out, hipStream_t stream);

// MFMA query pass (dq, dgate) for bf16 inputs; needs the row terms.
hipError_t launch_backward_q_bf16(const BwdParams &p, hipStream_t stream);

// MFMA key pass (dk, dv) for bf16 inputs; needs the row terms.
hipError_t launch_backward_kv_bf16(const BwdParams &p, hipStream_t stream);

}  // namespace pi_attn
