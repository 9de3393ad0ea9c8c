// index_set.hip -- writes W_t for every t with the enumerator the attention
// kernels use (pi_common.h): window offsets -k..0 (causal) or -k..k
// (bidirectional), then the partner t - pi and, bidirectional, t + pi.
#include "kernels.h"
#include "pi_common.h"

namespace pi_attn {

__global__ __launch_bounds__(256) void index_set_kernel(int n, int k, int pi, int causal, int m, int32_t *idx) {
    int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t total = (int64_t)n * m;
    if (e >= total) return;
    int t = (int)(e / m), s = (int)(e % m);
    idx[e] = ws_slot(t, s, k, pi, n, causal != 0);
}

hipError_t launch_index_set(int n, int k, int pi, bool causal, int32_t *idx, hipStream_t stream) {
    const int m = (int)ws_width(k, pi, causal);
    int64_t total = (int64_t)n * m;
    if (total == 0) return hipSuccess;
    int64_t blocks = (total + 255) / 256;
    return launch_kernel(index_set_kernel, dim3((unsigned)blocks), dim3(256), stream, n, k, pi, (int)causal, m, idx);
}

}  // namespace pi_attn
