// smallk_common.h -- lane layout and helpers shared by the small-window
// kernels (forward and backward): 32 rows per work-group of 256 threads, a
// row handled by 8 lanes of D/8 dimensions each.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "smallk.h"

namespace pi_attn {
namespace sk {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int NT = 256;    // threads per work-group
constexpr int TT = 32;     // tokens per work-group
constexpr int HG = 32;     // heads per work-group at most
constexpr int kGateScratch = 4 * 32 * 33;

template <int D, bool BIDIR, int KMAX>
struct Band {
    static constexpr int ROWS = TT + (BIDIR ? 2 : 1) * KMAX;      // staged rows at most
    static constexpr int ROWB = 2 * D;                            // LDS bytes per row
    static constexpr int CPR = D / 8;                             // 16-byte chunks per row
    static constexpr int CH = (ROWS * CPR + NT - 1) / NT;         // staged chunks per thread and tensor
    static constexpr int E = D / 8;                               // dimensions per lane
};

// LDS position of 16-byte chunk c of band row r.  D = 128: the two halves of
// a row swap on odd rows, so the 8 lanes of neighbouring queries (adjacent
// rows) read disjoint banks.
template <int D>
__device__ inline int chunk_pos(int r, int c) {
    if constexpr (D == 128) {
        return c ^ ((r & 1) << 3);
    } else {
        return c;
    }
}

// Sum over the 8 lanes of a query row (xor 1, xor 2 within quads, then the
// mirrored quad of the half-row): every lane ends with the same value.
__device__ inline float sum8(float x) {
    x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0xB1, 0xF, 0xF, false));
    x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x4E, 0xF, 0xF, false));
    x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x141, 0xF, 0xF, false));
    return x;
}

__device__ inline float dot8(const uint4 &a, const uint4 &b, float s) {
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a.x), __builtin_bit_cast(bf16x2, b.x), s, false);
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a.y), __builtin_bit_cast(bf16x2, b.y), s, false);
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a.z), __builtin_bit_cast(bf16x2, b.z), s, false);
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a.w), __builtin_bit_cast(bf16x2, b.w), s, false);
    return s;
}

// acc[0..8) += p * (8 bf16 values of v)
__device__ inline void axpy8(float *acc, float p, const uint4 &v) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        acc[2 * i + 0] += p * __uint_as_float(w[i] << 16);
        acc[2 * i + 1] += p * __uint_as_float(w[i] & 0xffff0000u);
    }
}

}  // namespace sk
}  // namespace pi_attn
