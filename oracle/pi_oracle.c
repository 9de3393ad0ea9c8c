/*
 * pi_oracle.c -- fp64 CPU oracle for pi-Attention (Variant 3, adaptive
 * fusion), causal and bidirectional.  TEST INFRASTRUCTURE ONLY: the product path never links,
 * loads or calls this file.  It shares no code with the HIP library.
 *
 * Plain, slow, obviously correct.  For every (b, h, t) it enumerates the
 * working set W_t explicitly, forms the fused logits in fp64 and runs a naive
 * (two-pass, non-online) softmax followed by the weighted sum of V.
 *
 * Definitions followed (pi-Attention, arXiv 2511.10696):
 *   - score z_tj = <q_t, k_j> * scale, scale = 1/sqrt(d_h)         (Sec. 3.2, eq. z)
 *   - local window N_r(t) = { j : max(0, t-k) <= j <= t }, causal,
 *     self included, so k+1 entries once t >= k;
 *     N_r(t) = { j : |j - t| <= k }, bidirectional                   (Sec. 3.2, eq. Nr)
 *   - long-range partner N_pi(t) = { t - pi } causal; bidirectional
 *     tasks add t + pi, both priced as partners                      (Sec. 3.4, eq. Npi; App. B,
 *                                                                      hyper-parameter table)
 *   - union U(t) = N_r(t) u N_pi(t); positions outside [0, T) are
 *     dropped (the appendix masks them to -inf)                      (eq. U; App. A, eqs. app_delta..app_out)
 *   - a partner that already lies in the window is not added twice
 *     (the appendix offset list appends -pi, and +pi when
 *     bidirectional, only if absent), so for pi <= k the set is the
 *     window alone                                                    (App. A, Fig. code)
 *   - gate: alpha = sigmoid(g), clipped alpha~ = eps + (1-2 eps) alpha,
 *     eps = 1e-4; g is the pre-sigmoid gate logit                    (Sec. 3.5 Variant 3; eq. app_gate)
 *   - prior omega = alpha~ on local keys, 1 - alpha~ on a partner     (eqs. omega, app_omega)
 *   - fused logit delta = z + log omega                              (eqs. delta_adapt, app_delta)
 *   - optional clamp of delta to [-Lc, Lc] (hyper-parameter table,
 *     App. B; not in the equations, off unless clamp > 0)
 *   - alpha^ = softmax(delta over U(t)), y_t = sum_j alpha^_j v_j    (eqs. alphahat_adapt, attn_adapt)
 *   - lse_t = log sum_j exp(delta_j)  (natural log, fused logits)
 * Backward (gradient of a loss L with dL/dy given), from the same forward:
 *   - dL/dalpha^_tj = <dL/dy_t, v_j>                                  (eq. attn_adapt)
 *   - softmax Jacobian on the fused logits:
 *       dL/ddelta_tj = alpha^_tj (dL/dalpha^_tj - sum_i alpha^_ti dL/dalpha^_ti)   (eq. jac)
 *   - dL/dz_tj = dL/ddelta_tj where delta is not clamped, else 0; dz/dq and
 *     dz/dk carry the factor scale                                    (eqs. z, delta_adapt)
 *   - dL/dv_j = sum_t alpha^_tj dL/dy_t                               (eq. attn_adapt)
 *   - gate: ddelta/dalpha~ = 1/alpha~ on local keys, -1/(1-alpha~) on
 *     the partner (eq. ddelta_da, written for the clipped gate the forward
 *     uses), dalpha~/dalpha = 1 - 2 eps, dalpha/dg = alpha (1 - alpha); the
 *     clamp cuts these paths too                                      (eqs. ddelta_da, dalpha_da; Sec. 3.5)
 * Decode step (causal; Sec. 3.5, online working set eq. online_ws): query at
 * position t = len[s] attends to cache rows W_t, where row t is the new
 * key/value, which the step first writes into the cache.
 *
 * Inputs are float32 (bf16 data is widened exactly by the caller) except the
 * gate logits, which are double (so logits computed in fp64 from the gate
 * MLP's last layer enter unrounded); every arithmetic operation is double
 * precision.  Layouts are dense row-major:
 * q, k, v [B][H][N][D]; gate logits addressed as g[b*gsb + h*gsh + t*gsn]
 * (element strides; zeros broadcast a per-head gate).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>

#define ORACLE_EPS 1e-4

/* Window slots per query: offsets -k..0 (causal) or -k..k (bidirectional). */
static int window_slots(int k, int causal) { return causal ? k + 1 : 2 * k + 1; }

/* Number of index slots per query: the window slots, then one partner slot
 * per partner (t-pi; t+pi too when bidirectional) when partners can lie
 * outside the window (pi > k). */
int oracle_ws_width(int k, int pi, int causal)
{
    return window_slots(k, causal) + (pi > k ? (causal ? 1 : 2) : 0);
}

/* Working set of query t as an explicit list.  Slot s of the window holds
 * position t-k+s (window ordered by offset, -k first, as in the appendix
 * offset list); slot nw (present iff pi > k) holds t-pi and, bidirectional,
 * slot nw+1 holds t+pi.  Absent entries are -1.  Returns the number of valid
 * entries. */
static int working_set(int t, int n, int k, int pi, int causal, int32_t *slot)
{
    int m = oracle_ws_width(k, pi, causal), nw = window_slots(k, causal), cnt = 0;
    for (int s = 0; s < m; ++s) slot[s] = -1;
    int lo = t - k > 0 ? t - k : 0;
    int hi = causal ? t : (t + k < n - 1 ? t + k : n - 1);
    for (int j = lo; j <= hi; ++j) {
        if (j < n) { slot[j - (t - k)] = j; ++cnt; }
    }
    if (pi > k && t - pi >= 0) { slot[nw] = t - pi; ++cnt; }
    if (!causal && pi > k && t + pi < n) { slot[nw + 1] = t + pi; ++cnt; }
    return cnt;
}

void oracle_index_set(int n, int k, int pi, int causal, int32_t *idx)
{
    int m = oracle_ws_width(k, pi, causal);
    for (int t = 0; t < n; ++t) working_set(t, n, k, pi, causal, idx + (int64_t)t * m);
}

/* alpha~ = eps + (1 - 2 eps) * sigmoid(g) */
static double clipped_gate(double g)
{
    double a = 1.0 / (1.0 + exp(-g));
    return ORACLE_EPS + (1.0 - 2.0 * ORACLE_EPS) * a;
}

/* One query against an explicit working set.  Key/value row j lives at
 * krows + j*D / vrows + j*D; slots below nw are window slots, the rest
 * partners.  delta[m] is scratch.  Writes y[D], returns lse; fills p[m]
 * (softmax weight per slot) if p is non-null. */
static double attend(int D, const float *q, const float *krows, const float *vrows,
                     const int32_t *slot, int m, int nw, double gate_logit,
                     double scale, double clamp, double *delta, double *y, double *p)
{
    double at = clipped_gate(gate_logit);
    double log_local = log(at), log_skip = log1p(-at);
    double mu = -INFINITY;
    for (int s = 0; s < m; ++s) {
        if (slot[s] < 0) { delta[s] = -INFINITY; continue; }
        const float *kj = krows + (int64_t)slot[s] * D;
        double z = 0.0;
        for (int d = 0; d < D; ++d) z += (double)q[d] * (double)kj[d];
        z *= scale;
        double dl = z + (s < nw ? log_local : log_skip);
        if (clamp > 0.0) dl = dl < -clamp ? -clamp : (dl > clamp ? clamp : dl);
        delta[s] = dl;
        if (dl > mu) mu = dl;
    }
    double Z = 0.0;
    for (int s = 0; s < m; ++s)
        if (slot[s] >= 0) Z += exp(delta[s] - mu);
    for (int d = 0; d < D; ++d) y[d] = 0.0;
    for (int s = 0; s < m; ++s) {
        double ps = slot[s] >= 0 ? exp(delta[s] - mu) / Z : 0.0;
        if (p) p[s] = ps;
        if (slot[s] < 0) continue;
        const float *vj = vrows + (int64_t)slot[s] * D;
        for (int d = 0; d < D; ++d) y[d] += ps * (double)vj[d];
    }
    return mu + log(Z);
}

/* Full-sequence forward, evaluated on a list of query rows.  A row is the
 * flat index r = (b*H + h)*N + t.  rows == NULL means every row, in order.
 * out [nrows][D]; lse [nrows] and probs [nrows][m] (softmax weight per slot,
 * 0 for absent slots) are optional (NULL). */
void oracle_forward_rows(int B, int H, int N, int D, int k, int pi, int causal,
                         const float *q, const float *kk, const float *v,
                         const double *gate, int64_t gsb, int64_t gsh, int64_t gsn,
                         double scale, double clamp,
                         const int64_t *rows, int64_t nrows,
                         double *out, double *lse, double *probs)
{
    int m = oracle_ws_width(k, pi, causal), nw = window_slots(k, causal);
    if (!rows) nrows = (int64_t)B * H * N;
#pragma omp parallel
    {
        int32_t *slot = (int32_t *)malloc(sizeof(int32_t) * (size_t)m);
        double *delta = (double *)malloc(sizeof(double) * (size_t)m);
#pragma omp for schedule(dynamic, 64)
        for (int64_t i = 0; i < nrows; ++i) {
            int64_t r = rows ? rows[i] : i;
            int t = (int)(r % N);
            int64_t bh = r / N;
            int h = (int)(bh % H), b = (int)(bh / H);
            working_set(t, N, k, pi, causal, slot);
            const float *kbase = kk + bh * (int64_t)N * D;
            const float *vbase = v + bh * (int64_t)N * D;
            double g = gate[b * gsb + h * gsh + (int64_t)t * gsn];
            double l = attend(D, q + r * D, kbase, vbase, slot, m, nw, g, scale, clamp,
                              delta, out + i * D, probs ? probs + i * m : NULL);
            if (lse) lse[i] = l;
        }
        free(slot);
        free(delta);
    }
}

/* Backward over whole heads.  dout [B][H][N][D] is dL/dy.  Writes dq, dk,
 * dv [B][H][N][D] and dgate [B][H][N] (dL/dg for the gate logit as seen by
 * query t; a per-head gate's gradient is the sum over its queries).
 * Every (b, h) is independent; within one, queries are visited in order. */
void oracle_backward(int B, int H, int N, int D, int k, int pi, int causal,
                     const float *q, const float *kk, const float *v,
                     const double *gate, int64_t gsb, int64_t gsh, int64_t gsn,
                     double scale, double clamp, const float *dout,
                     double *dq, double *dk, double *dv, double *dgate)
{
    int m = oracle_ws_width(k, pi, causal), nw = window_slots(k, causal);
#pragma omp parallel
    {
        int32_t *slot = (int32_t *)malloc(sizeof(int32_t) * (size_t)m);
        double *delta = (double *)malloc(sizeof(double) * (size_t)m);
        double *p = (double *)malloc(sizeof(double) * (size_t)m);
        double *dp = (double *)malloc(sizeof(double) * (size_t)m);
        double *y = (double *)malloc(sizeof(double) * (size_t)D);
#pragma omp for schedule(dynamic, 1)
        for (int64_t bh = 0; bh < (int64_t)B * H; ++bh) {
            int h = (int)(bh % H), b = (int)(bh / H);
            const float *qb = q + bh * (int64_t)N * D, *kb = kk + bh * (int64_t)N * D;
            const float *vb = v + bh * (int64_t)N * D, *ob = dout + bh * (int64_t)N * D;
            double *dqb = dq + bh * (int64_t)N * D, *dkb = dk + bh * (int64_t)N * D;
            double *dvb = dv + bh * (int64_t)N * D;
            for (int64_t i = 0; i < (int64_t)N * D; ++i) dqb[i] = dkb[i] = dvb[i] = 0.0;
            for (int t = 0; t < N; ++t) {
                const float *qt = qb + (int64_t)t * D, *gt = ob + (int64_t)t * D;
                working_set(t, N, k, pi, causal, slot);
                double g = gate[b * gsb + h * gsh + (int64_t)t * gsn];
                attend(D, qt, kb, vb, slot, m, nw, g, scale, clamp, delta, y, p);
                /* dL/dalpha^ per slot and its weighted mean */
                double mean = 0.0;
                for (int s = 0; s < m; ++s) {
                    dp[s] = 0.0;
                    if (slot[s] < 0) continue;
                    const float *vj = vb + (int64_t)slot[s] * D;
                    for (int d = 0; d < D; ++d) dp[s] += (double)gt[d] * (double)vj[d];
                    mean += p[s] * dp[s];
                }
                double a = 1.0 / (1.0 + exp(-g)), at = clipped_gate(g);
                double dg_local = (1.0 - 2.0 * ORACLE_EPS) * a * (1.0 - a) / at;
                double dg_skip = -(1.0 - 2.0 * ORACLE_EPS) * a * (1.0 - a) / (1.0 - at);
                double dgt = 0.0;
                for (int s = 0; s < m; ++s) {
                    if (slot[s] < 0) continue;
                    int j = slot[s];
                    double dd = p[s] * (dp[s] - mean); /* dL/ddelta (eq. jac) */
                    if (clamp > 0.0 && fabs(delta[s]) >= clamp) dd = 0.0;
                    const float *kj = kb + (int64_t)j * D;
                    for (int d = 0; d < D; ++d) {
                        dqb[(int64_t)t * D + d] += scale * dd * (double)kj[d];
                        dkb[(int64_t)j * D + d] += scale * dd * (double)qt[d];
                        dvb[(int64_t)j * D + d] += p[s] * (double)gt[d];
                    }
                    dgt += dd * (s < nw ? dg_local : dg_skip);
                }
                dgate[bh * (int64_t)N + t] = dgt;
            }
        }
        free(slot);
        free(delta);
        free(p);
        free(dp);
        free(y);
    }
}

/* KV-cached decode step.  For each (s, h): t = len_in[s]; rows t of k_cache /
 * v_cache [S][H][cap][D] are overwritten by k_new / v_new [S][H][D]; the query
 * q_new[s][h] then attends to W_t over the cache.  Requires t < cap.
 * out [S][H][D]; lse [S][H] optional.  Returns 0, or -1 if some t >= cap or t < 0. */
int oracle_decode_step(int S, int H, int D, int cap, int k, int pi,
                       const int32_t *len_in,
                       const float *q_new, const float *k_new, const float *v_new,
                       float *k_cache, float *v_cache,
                       const double *gate, int64_t gss, int64_t gsh,
                       double scale, double clamp, double *out, double *lse)
{
    for (int s = 0; s < S; ++s)
        if (len_in[s] < 0 || len_in[s] >= cap) return -1;
    int m = oracle_ws_width(k, pi, 1);
#pragma omp parallel
    {
        int32_t *slot = (int32_t *)malloc(sizeof(int32_t) * (size_t)m);
        double *delta = (double *)malloc(sizeof(double) * (size_t)m);
#pragma omp for schedule(dynamic, 1)
        for (int64_t r = 0; r < (int64_t)S * H; ++r) {
            int s = (int)(r / H), h = (int)(r % H);
            int t = len_in[s];
            float *kc = k_cache + r * (int64_t)cap * D;
            float *vc = v_cache + r * (int64_t)cap * D;
            for (int d = 0; d < D; ++d) {
                kc[(int64_t)t * D + d] = k_new[r * D + d];
                vc[(int64_t)t * D + d] = v_new[r * D + d];
            }
            working_set(t, t + 1, k, pi, 1, slot);
            double g = gate[s * gss + h * gsh];
            double l = attend(D, q_new + r * D, kc, vc, slot, m, k + 1, g, scale, clamp,
                              delta, out + r * D, NULL);
            if (lse) lse[r] = l;
        }
        free(slot);
        free(delta);
    }
    return 0;
}
