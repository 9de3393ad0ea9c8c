// smallk.h -- launchers of the small-window forward and of the gate MLP's
// last layer (the Variant-3 gate logits computed inside the library).
#pragma once

#include "kernels.h"

namespace pi_attn {

// Largest window radius the small-window forward takes.
constexpr int kSmallK = 16;

// Operands of the gate MLP's last layer (App. A gate module: Linear(d, d/2),
// GELU, Linear(d/2, h), Sigmoid): g[b, h, t] = sum_c u[b, t, c] w2[h, c] + b2[h].
struct GateMlp {
    const void *u;        // [B][N][dh], element strides (usb, usn), dh contiguous; dtype of q
    int64_t usb, usn;
    int dh;               // hidden width (multiple of 8)
    const void *w2;       // [H][dh] contiguous (the Linear weight as stored); dtype of q
    const float *b2;      // [H] or nullptr (no bias)
    float *gate_out;      // [B][H][N] contiguous: the logits g, written
};

// Small-window forward (k <= kSmallK), bf16, D = 64 or 128: one work-group
// per (b, 32 tokens, group of up to 32 heads), the window band staged in LDS
// per head.  With mlp != nullptr the gate logits come from the gate MLP's
// last layer, computed in the same kernel (and written to mlp->gate_out);
// otherwise from p.gate.
hipError_t launch_forward_smallk(const FwdParams &p, const GateMlp *mlp, hipStream_t stream);

// The gate logits alone, into mlp.gate_out (bf16 on MFMA, float32 on VALU).
hipError_t launch_gate_logits(const FwdParams &p, const GateMlp &mlp, int dtype, hipStream_t stream);

// Small-window backward (k <= kSmallK), bf16, D = 64 or 128: a query pass
// (dq, gate gradient, exact row terms) and a key pass (dk, dv), both in the
// forward's work decomposition.  Needs the forward's lse.
hipError_t launch_backward_smallk(const BwdParams &p, hipStream_t stream);

}  // namespace pi_attn
