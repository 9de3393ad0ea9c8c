/*
 * pi_attn.h -- C ABI of the MI355X (gfx950) pi-Attention operator.
 *
 * pi-Attention (arXiv 2511.10696) evaluates attention of query t on the
 * online working set W_t = N_r(t) u N_pi(t) (Sec. 3.5, eq. online_ws).
 * Causal mode (causal != 0):
 *   - the local window N_r(t) = { j : max(0, t-k) <= j <= t }, radius k,
 *     self included (Sec. 3.2, eq. Nr, causal case);
 *   - the long-range partner N_pi(t) = { t - pi } (Sec. 3.4, eq. Npi), kept
 *     only when it lies in [0, t] and outside the window (pi > k; a partner
 *     inside the window is not counted twice, App. A offset list).
 * Bidirectional mode (causal == 0; App. B hyper-parameter table):
 *   - the window N_r(t) = { j : |j - t| <= k } (eq. Nr, bidirectional case);
 *   - the partners t - pi and t + pi, each kept when it lies in [0, N) and
 *     pi > k, both priced as partners.
 * Adaptive fusion (Sec. 3.5 Variant 3, eqs. gate..attn_adapt; App. A eqs.
 * app_gate..app_out): with gate logit g (pre-sigmoid),
 *   alpha~ = eps + (1 - 2 eps) * sigmoid(g),  eps = 1e-4,
 *   delta_tj = scale * <q_t, k_j> + log(alpha~)      for j in the window,
 *   delta_tj = scale * <q_t, k_j> + log(1 - alpha~)  for a partner,
 *   y_t = sum_j softmax_j(delta_t) v_j                 (one shared softmax).
 * scale is 1/sqrt(D) in the paper (Sec. 3.2, eq. z); it is an argument here.
 *
 * Conventions for every entry point
 *   - Device pointers are HIP device (or managed) memory owned by the caller;
 *     the library allocates nothing and keeps no state between calls.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = the default stream)
 *     and is asynchronous: argument errors are returned before anything is
 *     enqueued, execution errors surface at the caller's next synchronise.
 *   - Return value: PI_ATTN_OK (0) or a negative status (pi_attn_strerror).
 *   - Element types: PI_ATTN_F32 (float32) or PI_ATTN_BF16 (bfloat16); the
 *     arithmetic is fp32 in both (bf16 operands are multiplied on MFMA with
 *     fp32 accumulation; softmax weights enter the value product as bf16).
 *   - Supported head dimensions D: 64 and 128.
 *   - Rows of q/k/v/out (the D elements of one position) are contiguous and
 *     start 16-byte aligned: base pointers 16-byte aligned and every stride a
 *     multiple of 16 bytes.
 *   - Zero-sized problems (N == 0, B == 0, ...) are valid no-ops.
 *   - Calls on different streams may run concurrently; calls that write the
 *     same buffers must be ordered by the caller.
 */
#ifndef PI_ATTN_H
#define PI_ATTN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { PI_ATTN_F32 = 0, PI_ATTN_BF16 = 1 } pi_attn_dtype;

enum {
    PI_ATTN_OK = 0,
    PI_ATTN_EINVAL = -1,       /* null pointer, negative size, bad stride or alignment */
    PI_ATTN_EUNSUPPORTED = -2, /* valid request outside what is built (D, dtype)       */
    PI_ATTN_EHIP = -3,         /* the HIP runtime refused a launch                      */
    PI_ATTN_ESCRATCH = -4      /* too large for pi_attn_backward_noalloc's fixed array  */
};

/* Human-readable text for a status code (static storage, never NULL). */
const char *pi_attn_strerror(int status);

/* Slots per query in the index-set layout, the largest |W_t| (Sec. 3.5, eq.
 * online_ws: the window of eq. Nr, radius k with self, plus the partners of
 * eq. Npi, not counted twice when they lie in the window, App. A offset
 * list): causal, k+1 window slots plus one partner slot iff pi > k;
 * bidirectional, 2k+1 window slots plus two partner slots iff pi > k.
 * Returns -1 for k < 0, pi < 0 or a width beyond int32. */
int32_t pi_attn_ws_width(int32_t k, int32_t pi, int32_t causal);

/* The paper's score scale 1/sqrt(D) (Sec. 3.2, eq. z), the value to pass as
 * `scale` for the paper's operator; 0 for D < 1. */
float pi_attn_default_scale(int32_t D);

/*
 * pi_attn_index_set -- the working sets W_t of a length-n sequence
 * (Sec. 3.2 eq. Nr; Sec. 3.4 eqs. U, Npi; App. A offset list).
 *   causal  non-zero: causal mode; zero: bidirectional mode.
 *   idx     device int32 [n][m], m = pi_attn_ws_width(k, pi, causal),
 *           written fully, with w = k+1 (causal) or 2k+1 (bidirectional):
 *           idx[t*m + s] = t - k + s for s in [0, w) (window offsets from -k),
 *           idx[t*m + w] = t - pi and, bidirectional, idx[t*m + w + 1] = t + pi
 *           (only when pi > k), and -1 wherever that position is outside
 *           [0, n).
 *   Errors: EINVAL for n < 0, k < 0, pi < 0, idx == NULL with n > 0, or
 *   n*m beyond 2^31 entries.
 */
int pi_attn_index_set(int32_t n, int32_t k, int32_t pi, int32_t causal, int32_t *idx, void *stream);

/*
 * pi_attn_forward -- full-sequence pi-Attention with adaptive fusion
 * (Sec. 3.5 Variant 3; App. A eqs. app_gate..app_out).
 *   dtype        PI_ATTN_F32 or PI_ATTN_BF16: element type of q, k, v and out.
 *   B, H, N, D   batch, heads, sequence length, head dimension.
 *   k, pi        window radius (k >= 0) and partner period (pi >= 0; pi <= k
 *                means no separate partner, i.e. sliding-window attention;
 *                k >= N-1 is dense attention).
 *   causal       non-zero: causal mode; zero: bidirectional mode.
 *   q, kk, v     device [B][H][N][D] through element strides (sb, sh, sn)
 *                shared by the three tensors; the D elements are contiguous.
 *   gate         device float32 pre-sigmoid gate logits g, read at
 *                gate[b*gsb + h*gsh + t*gsn] (element strides): per-head
 *                gates [H] use (0, 1, 0), per-query gates [B][H][N] use
 *                (H*N, N, 1).
 *   scale        score scale (1/sqrt(D) in the paper).
 *   logit_clamp  > 0: clamp every fused logit delta to [-clamp, clamp]
 *                (hyper-parameter L_c of App. B; off when <= 0).
 *   out          device [B][H][N][D] through (osb, osh, osn), same dtype.
 *   lse          optional device float32 [B][H][N] contiguous: natural-log
 *                sum over W_t of exp(delta), or NULL.
 * bf16 with k <= 16 runs a gather kernel (the window band staged in LDS per
 * head); larger windows the banded MFMA kernel.
 * Errors: EINVAL (null pointer with non-empty problem, negative size or
 * stride, misalignment), EUNSUPPORTED (D not 64/128, unknown dtype; for
 * bf16, (c * min(k, N) + 256) * sn * 2 bytes >= 2 GiB, c = 1 causal and 2
 * bidirectional), EHIP (launch refused).
 */
int pi_attn_forward(int32_t dtype, int32_t B, int32_t H, int32_t N, int32_t D,
                    int32_t k, int32_t pi, int32_t causal,
                    const void *q, const void *kk, const void *v,
                    int64_t sb, int64_t sh, int64_t sn,
                    const float *gate, int64_t gsb, int64_t gsh, int64_t gsn,
                    float scale, float logit_clamp,
                    void *out, int64_t osb, int64_t osh, int64_t osn,
                    float *lse, void *stream);

/*
 * pi_attn_forward_gated -- pi_attn_forward with the Variant-3 gate logits
 * computed from the gate MLP (App. A gate module: Linear(d, d/2), GELU,
 * Linear(d/2, h), Sigmoid; Sec. 3.5 eq. gate): the caller passes the GELU
 * output u and the last Linear layer, and the operator forms
 *   g[b, h, t] = sum_c u[b, t, c] * w2[h, c] + b2[h]
 * (fp32 accumulation) before the sigmoid, the eps clip and the fusion.
 *   dtype ... k, pi, causal, q, kk, v, strides, scale, logit_clamp, out,
 *                lse  as in pi_attn_forward.
 *   u            device [B][N][dh] in dtype through element strides (usb,
 *                usn), the dh elements contiguous, rows 16-byte aligned.
 *   dh           hidden width (the paper uses d/2); dh * sizeof(dtype) must
 *                be a multiple of 16.
 *   w2           device [H][dh] in dtype, contiguous (the Linear weight as
 *                stored, output-major), 16-byte aligned.
 *   b2           device float32 [H], or NULL for no bias.
 *   gate_out     device float32 [B][H][N] contiguous, overwritten with g (the
 *                gate argument that pi_attn_backward takes, strides
 *                (H*N, N, 1); dL/dg from there flows back into u, w2, b2).
 * For bf16 with k <= 16 the logits are computed inside the attention kernel
 * (u read once per token for a group of up to 32 heads); otherwise a gate
 * kernel writes gate_out first and the forward reads it.
 * Errors: as pi_attn_forward, plus EINVAL for a null u, w2 or gate_out, a
 * misaligned u, w2, b2 or gate_out, dh < 1 or dh not a multiple of
 * 16 bytes.
 */
int pi_attn_forward_gated(int32_t dtype, int32_t B, int32_t H, int32_t N, int32_t D,
                          int32_t k, int32_t pi, int32_t causal,
                          const void *q, const void *kk, const void *v,
                          int64_t sb, int64_t sh, int64_t sn,
                          const void *u, int64_t usb, int64_t usn, int32_t dh,
                          const void *w2, const float *b2,
                          float scale, float logit_clamp,
                          void *out, int64_t osb, int64_t osh, int64_t osn,
                          float *lse, float *gate_out, void *stream);

/*
 * pi_attn_decode_step -- one KV-cached decode step of the online operator
 * (causal mode; Sec. 3.5, eq. online_ws): for each sequence s and head h, with
 * t = len_in[s], first store the new key/value as cache row t, then attend
 * the new query over W_t (window rows max(0,t-k)..t, partner row t-pi when
 * pi > k and t >= pi).
 *   dtype        PI_ATTN_BF16 or PI_ATTN_F32 (q/k/v/out/caches).
 *   S, H, D      sequences, heads, head dimension; cap = cache rows.
 *   len_in       device int32 [S]: current lengths (0 <= len_in[s] < cap).
 *   len_out      optional device int32 [S] (NULL to skip): receives
 *                len_in[s] + 1.  Must not overlap len_in (other work-groups
 *                of the same step still read it): EINVAL if the two
 *                S-element ranges share a byte.
 *   q_new, k_new, v_new   device [S][H][D] contiguous.
 *   k_cache, v_cache      device [S][H][cap][D] contiguous; row len_in[s]
 *                of every head is overwritten, nothing else is written.
 *   gate         device float32 gate logits gate[s*gss + h*gsh].
 *   out          device [S][H][D] contiguous; lse optional float32 [S][H].
 * A length outside [0, cap) cannot be checked on the host (it lives in
 * device memory): the step then writes NaN to that sequence's outputs (and
 * lse), leaves its caches untouched and stores len_out[s] = len_in[s].
 * Errors: as pi_attn_forward, plus EINVAL for cap < 1.
 */
int pi_attn_decode_step(int32_t dtype, int32_t S, int32_t H, int32_t D, int32_t cap,
                        int32_t k, int32_t pi,
                        const int32_t *len_in, int32_t *len_out,
                        const void *q_new, const void *k_new, const void *v_new,
                        void *k_cache, void *v_cache,
                        const float *gate, int64_t gss, int64_t gsh,
                        float scale, float logit_clamp,
                        void *out, float *lse, void *stream);

/*
 * pi_attn_backward -- gradients of the full-sequence operator for a loss L
 * given dL/dy (the softmax Jacobian on the fused logits, Sec. 3.5 eq. jac;
 * the prior derivatives for the clipped gate, eqs. ddelta_da and dalpha_da;
 * the same W_t, scale, gate and clamp as pi_attn_forward).
 *   dtype ... logit_clamp   exactly as passed to pi_attn_forward (causal
 *                included).
 *   lse          device float32 [B][H][N] contiguous: the lse that
 *                pi_attn_forward wrote for these inputs (the weights are
 *                recomputed as exp(delta - lse)).
 *   out          device y [B][H][N][D] in dtype: the output that
 *                pi_attn_forward wrote for these inputs, through the same
 *                strides as dout.
 *   dout         device dL/dy [B][H][N][D] in dtype through (osb, osh, osn).
 *   dq, dk, dv   device float32 [B][H][N][D] contiguous, overwritten.
 *   dgate        device float32 [B][H][N] contiguous, overwritten: dL/dg of
 *                the gate logit as seen by query t (a per-head gate's
 *                gradient is the sum of its entries over b and t).
 *   rowterm      device float32 [B][H][N] contiguous scratch owned by the
 *                caller: receives the row terms
 *                r_t = sum_j alpha^_tj dL/dalpha^_tj = <dL/dy_t, y_t>
 *                (float32: from out; bf16: as recomputed by the query pass).
 * Kernels on the stream, in order: (float32) the row terms, then a query
 * pass (dq, dgate; for bf16 it also writes the row terms) and a key pass
 * (dk, dv).  bf16 with k <= 16 takes gather-style passes whose weights and
 * products stay in float32 throughout (the row terms exact); larger windows
 * take the banded MFMA passes, whose softmax gradients enter the products
 * rounded to bf16.  Nothing is allocated; buffers must not overlap.
 * Errors: as pi_attn_forward, plus EINVAL for a null or misaligned lse,
 * out, dout, dq, dk, dv, dgate or rowterm.
 */
int pi_attn_backward(int32_t dtype, int32_t B, int32_t H, int32_t N, int32_t D,
                     int32_t k, int32_t pi, int32_t causal,
                     const void *q, const void *kk, const void *v,
                     int64_t sb, int64_t sh, int64_t sn,
                     const float *gate, int64_t gsb, int64_t gsh, int64_t gsn,
                     float scale, float logit_clamp, const float *lse, const void *out,
                     const void *dout, int64_t osb, int64_t osh, int64_t osn,
                     float *dq, float *dk, float *dv, float *dgate, float *rowterm,
                     void *stream);

/*
 * pi_attn_backward_noalloc -- pi_attn_backward for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving or
 * training loops, harnesses that forbid hipMalloc): the same arguments,
 * kernels and results without the rowterm workspace.  The row terms go to
 * a fixed array of 4194304 float32 (16 MiB) that the library holds on every
 * device it runs on until the process ends; the call uses the current
 * device's array (hipGetDevice), so the buffers and the stream must be on
 * that device.  It calls no allocating routine.
 *   Arguments    as pi_attn_backward, without rowterm.
 *   Results      bit-identical to pi_attn_backward's on the same inputs.
 *   Sharing      every call on one device uses that device's array: calls
 *                that overlap in time on one device (different streams,
 *                threads without ordering) race on it and must be ordered by
 *                the caller; calls in order on one stream are safe.  Each call
 *                writes every row term it reads, so stale contents from an
 *                earlier call never matter.
 * Errors: as pi_attn_backward; ESCRATCH when B*H*N > 4194304 (nothing is
 * enqueued); EHIP if the array's address cannot be obtained.
 */
int pi_attn_backward_noalloc(int32_t dtype, int32_t B, int32_t H, int32_t N, int32_t D,
                             int32_t k, int32_t pi, int32_t causal,
                             const void *q, const void *kk, const void *v,
                             int64_t sb, int64_t sh, int64_t sn,
                             const float *gate, int64_t gsb, int64_t gsh, int64_t gsn,
                             float scale, float logit_clamp, const float *lse, const void *out,
                             const void *dout, int64_t osb, int64_t osh, int64_t osn,
                             float *dq, float *dk, float *dv, float *dgate, void *stream);

/*
 * pi_attn_forward_shard -- pi_attn_forward over one shard of a sequence:
 * the queries at absolute positions [qpos0, qpos0 + nq) of a sequence of
 * nseq positions, with the k/v rows held from absolute position kvpos0 on
 * (the shard's own rows plus the halo before it, and for the bidirectional
 * mode after it).  The working set of a query is that of the whole sequence
 * (Sec. 3.2 eq. Nr, Sec. 3.4 eq. Npi: window and partners by absolute
 * position), so the outputs equal the corresponding rows of pi_attn_forward
 * over the whole sequence; this is the part of a sequence-sharded run that
 * one GPU executes once its halo has arrived (the network term of the cost
 * model, Sec. 3.5 eq. online_cost).  bf16 only.
 *   dtype, B, H, D, k, pi, causal, scale, logit_clamp   as pi_attn_forward.
 *   nseq, qpos0, nq   sequence length and the shard's queries; 0 <= qpos0,
 *                qpos0 + nq <= nseq.
 *   kvpos0, nkv  absolute position of k/v row 0 and the rows held:
 *                kvpos0 <= min(window start of qpos0 rounded down to a
 *                multiple of 32, max(0, qpos0 - pi) when pi > k), and
 *                kvpos0 + nkv >= qpos0 + nq (causal) or
 *                min(nseq, qpos0 + nq + max(k, pi)) (bidirectional; k when
 *                pi <= k); kvpos0 + nkv <= nseq.
 *   q            device [B][H][nq][D] through (sb, sh, sn).
 *   kk, v        device [B][H][nkv][D] through (ksb, ksh, ksn).
 *   gate         per head [H] or per query [B][H][nq] (query rows of the
 *                shard) through (gsb, gsh, gsn).
 *   out, lse     [B][H][nq][D] through (osb, osh, osn) and [B][H][nq].
 * Results: rows equal to pi_attn_forward's for the same absolute positions
 * up to rounding, and bit-identical when qpos0 is a multiple of 128 and
 * kvpos0 a multiple of 32 (the same tiles in the same order).
 * Errors: as pi_attn_forward; EUNSUPPORTED for float32; EINVAL for
 * positions or k/v rows that do not satisfy the conditions above.
 */
int pi_attn_forward_shard(int32_t dtype, int32_t B, int32_t H, int32_t D, int32_t k, int32_t pi, int32_t causal,
                          int32_t nseq, int32_t qpos0, int32_t nq, int32_t kvpos0, int32_t nkv, const void *q,
                          int64_t sb, int64_t sh, int64_t sn, const void *kk, const void *v, int64_t ksb, int64_t ksh,
                          int64_t ksn, const float *gate, int64_t gsb, int64_t gsh, int64_t gsn, float scale,
                          float logit_clamp, void *out, int64_t osb, int64_t osh, int64_t osn, float *lse,
                          void *stream);

/*
 * pi_attn_backward_shard_q, pi_attn_backward_shard_kv -- pi_attn_backward
 * split into its two passes over one shard of a sequence of nseq positions
 * (the gradients of Sec. 3.5 eq. jac and eqs. ddelta_da, dalpha_da, every
 * working set taken by absolute position as in pi_attn_forward_shard).  A
 * sequence-sharded run calls the query pass on its queries, exchanges the
 * halo of query rows the key pass needs (q, dL/dy, lse, the row terms the
 * neighbour's query pass wrote, and per-query gates), then calls the key
 * pass on its keys.  bf16 only; the banded passes for every k.
 *
 * pi_attn_backward_shard_q: queries [qpos0, qpos0 + nq) with the k/v rows
 * held from kvpos0 (nkv rows; the coverage pi_attn_forward_shard requires).
 *   q [B][H][nq][D] (sb, sh, sn); kk, v [B][H][nkv][D] (ksb, ksh, ksn);
 *   gate [H] or [B][H][nq]; lse [B][H][nq] (the forward's); out and dout
 *   [B][H][nq][D] (osb, osh, osn); writes dq [B][H][nq][D], dgate and the
 *   row terms [B][H][nq], all contiguous float32.
 *
 * pi_attn_backward_shard_kv: keys [kpos0, kpos0 + nk) (kk, v hold exactly
 * these rows, [B][H][nk][D] through ksb, ksh, ksn) with the query rows held
 * from qpos0 (nqh rows): q and dout [B][H][nqh][D] through (sb, sh, sn) and
 * (osb, osh, osn), gate [H] or [B][H][nqh], lse and row terms [B][H][nqh]
 * contiguous.  The query rows must cover every query whose working set
 * holds one of the keys: qpos0 <= kpos0 (causal) or
 * max(0, kpos0 - max(k, pi)) (bidirectional; k when pi <= k), and
 * qpos0 + nqh >= min(nseq, kpos0 + nk + max(k, pi)) (k when pi <= k).
 * Writes dk, dv [B][H][nk][D] contiguous float32.
 *
 * Results: the rows of pi_attn_backward's gradients (with k > 16, whose
 * whole-sequence call also takes the banded passes) for the same absolute
 * positions, bit-identical when qpos0 and kpos0 are multiples of 128.
 * Errors: as pi_attn_backward; EUNSUPPORTED for float32; EINVAL for
 * positions or rows held that do not satisfy the conditions above.
 */
int pi_attn_backward_shard_q(int32_t dtype, int32_t B, int32_t H, int32_t D, int32_t k, int32_t pi,
                             int32_t causal, int32_t nseq, int32_t qpos0, int32_t nq, int32_t kvpos0, int32_t nkv,
                             const void *q, int64_t sb, int64_t sh, int64_t sn, const void *kk, const void *v,
                             int64_t ksb, int64_t ksh, int64_t ksn, const float *gate, int64_t gsb, int64_t gsh,
                             int64_t gsn, float scale, float logit_clamp, const float *lse, const void *out,
                             const void *dout, int64_t osb, int64_t osh, int64_t osn, float *dq, float *dgate,
                             float *rowterm, void *stream);
int pi_attn_backward_shard_kv(int32_t dtype, int32_t B, int32_t H, int32_t D, int32_t k, int32_t pi,
                              int32_t causal, int32_t nseq, int32_t kpos0, int32_t nk, int32_t qpos0, int32_t nqh,
                              const void *q, int64_t sb, int64_t sh, int64_t sn, const void *kk, const void *v,
                              int64_t ksb, int64_t ksh, int64_t ksn, const float *gate, int64_t gsb, int64_t gsh,
                              int64_t gsn, float scale, float logit_clamp, const float *lse, const float *rowterm,
                              const void *dout, int64_t osb, int64_t osh, int64_t osn, float *dk, float *dv,
                              void *stream);

/*
 * pi_attn_gate_grad_per_head -- the gradient of a per-head gate logit g_h
 * shared by every b and t: out[h] = sum over b, t of dgate[b][h][t], the
 * per-query gradients pi_attn_backward writes (the gate enters each query's
 * prior separately, Sec. 3.5 eqs. ddelta_da and dalpha_da, so its gradient
 * is the sum of the per-query ones).
 *   B, H, N      sizes, >= 0; B*H*N below 2^31.
 *   dgate        device float32 [B][H][N] contiguous (may be null when
 *                B*N == 0).
 *   out          device float32 [H], overwritten (zeros when B*N == 0).
 * The sums are taken in fp64 in a fixed order: results are deterministic.
 * One kernel on the stream; nothing is allocated.
 * Errors: EINVAL for negative sizes, B*H*N too large, a null or misaligned
 * out (H > 0) or dgate (B*N > 0).
 */
int pi_attn_gate_grad_per_head(int32_t B, int32_t H, int32_t N, const float *dgate, float *out, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* PI_ATTN_H */
