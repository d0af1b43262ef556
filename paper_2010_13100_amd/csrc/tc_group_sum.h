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

// The forward gather-reduce of bags [bag_lo, bag_hi) (Sec. II-B): out[g] =
// sum over the bag's pairs j, in order, of W[table_row_offset[g / B] +
// ids[j]], from +0. Run by k_forward, and by workgroups of the cast's
// kernels in tc_embed_forward_cast.
struct FwdSlice {
    const float *W;
    const int32_t *ids;
    const int32_t *offsets;
    const int64_t *table_row_offset;
    float *out;
    int64_t bag_lo, bag_hi;
    int32_t dim, bags_per_table;
};

// Wavefront `wave` of `nwave` takes kWave/LANES bags at a time (one per lane
// group), grid-stride over the slice. Every lane of the wavefront calls this.
template <int LANES, int CHUNKS>
__device__ __forceinline__ void forward_bags(const FwdSlice &f, int64_t wave, int64_t nwave) {
    constexpr int kGroups = kWave / LANES;  // bags per wavefront
    const int lane = threadIdx.x & (kWave - 1);
    const int sub = lane & (LANES - 1);
    const int grp = lane / LANES;
    for (int64_t o0 = f.bag_lo + wave * kGroups; o0 < f.bag_hi; o0 += nwave * kGroups) {
        const int64_t o = o0 + grp;
        const bool live = o < f.bag_hi;
        int32_t beg = 0, end = 0;
        int64_t base = 0;
        if (live) {
            beg = f.offsets[o];
            end = f.offsets[o + 1];
            base = f.table_row_offset[o / f.bags_per_table];
        }
        float4 acc[CHUNKS];
#pragma unroll
        for (int c = 0; c < CHUNKS; ++c) acc[c] = make_float4(0.f, 0.f, 0.f, 0.f);
        group_range_sum<LANES, CHUNKS>(f.W, f.dim, f.ids, base, beg, end, sub, acc);
        if (live) group_store<LANES, CHUNKS>(f.out + o * int64_t(f.dim), f.dim, sub, acc);
    }
}

// Lanes per bag of a forward run inside the cast's kernels: the lane groups
// of one float4 chunk per lane and at least 16 lanes (dim 36..256); 0 for
// other row shapes (the forward then runs as its own kernel).
inline int ride_along_lanes(int32_t dim) {
    const RowShape s = row_shape(dim);
    return s.chunks == 1 && s.lanes >= 16 ? s.lanes : 0;
}

// The forward over all num_bags bags as its own kernel (tc_gather_reduce.hip).
tc_status launch_forward(const float *W, int32_t dim, const int32_t *ids, const int32_t *offsets,
                         const int64_t *table_row_offset, int32_t bags_per_table,
                         int64_t num_bags, float *out, hipStream_t stream);

}  // namespace tc
