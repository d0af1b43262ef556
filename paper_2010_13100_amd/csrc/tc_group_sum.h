// Lane-group walk shared by the forward and the backward gather-reduce.
#pragma once

#include "tc_internal.h"

namespace tc {

constexpr int kUnroll = 8;

__device__ __forceinline__ float4 f4_add(float4 a, float4 b) {
    return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
}

// Ordered sum of the rows ids[beg..end) of `src` (plus `base`) into acc, for
// one lane group of LANES lanes: LANES indices are fetched at once (one per
// lane) and broadcast with __shfl; kUnroll row loads are issued before the
// adds that consume them. All lanes of a group must call this together.
template <int LANES, int CHUNKS>
__device__ __forceinline__ void group_range_sum(const float *__restrict__ src, int32_t dim,
                                                const int32_t *__restrict__ ids, int64_t base,
                                                int32_t beg, int32_t end, int sub,
                                                float4 (&acc)[CHUNKS]) {
    const int d4 = dim >> 2;
    for (int32_t j0 = beg; j0 < end; j0 += LANES) {
        const int cnt = min(LANES, end - j0);
        const int32_t my_id = (sub < cnt) ? ids[j0 + sub] : 0;
        for (int k = 0; k < cnt; k += kUnroll) {
            float4 v[kUnroll][CHUNKS];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const int kk = k + u;
                const int32_t id = __shfl(my_id, kk & (LANES - 1), LANES);
                const float *row = src + (base + id) * int64_t(dim);
#pragma unroll
                for (int c = 0; c < CHUNKS; ++c) {
                    const int col4 = sub + c * LANES;
                    v[u][c] = (kk < cnt && col4 < d4)
                                  ? *reinterpret_cast<const float4 *>(row + 4 * col4)
                                  : make_float4(0.f, 0.f, 0.f, 0.f);
                }
            }
            // Adding +0 for the slots past the end leaves acc unchanged bit
            // for bit (acc is never -0 when it starts at +0).
#pragma unroll
            for (int u = 0; u < kUnroll; ++u)
#pragma unroll
                for (int c = 0; c < CHUNKS; ++c) acc[c] = f4_add(acc[c], v[u][c]);
        }
    }
}

template <int LANES, int CHUNKS>
__device__ __forceinline__ void group_store(float *__restrict__ orow, int32_t dim, int sub,
                                            const float4 (&acc)[CHUNKS]) {
    const int d4 = dim >> 2;
#pragma unroll
    for (int c = 0; c < CHUNKS; ++c) {
        const int col4 = sub + c * LANES;
        if (col4 < d4) *reinterpret_cast<float4 *>(orow + 4 * col4) = acc[c];
    }
}

}  // namespace tc
