// Gather-reduce on CDNA4: the forward embedding pass (Sec. II-B) and the
// casted gradient gather-reduce (Algorithm 3) are the same operation -- an
// output row is the ordered sum of source rows named by an index range -- so
// one kernel serves both, as the paper unifies them under one operator.
//
// Mapping: a group of LANES lanes (a power of two <= 64) owns one output
// row; each lane holds CHUNKS float4 column chunks (dwordx4 loads), so one
// row of 4*dim bytes is read by one vector instruction per chunk. The group
// walks its index range in order: LANES indices are fetched at once, one per
// lane, then broadcast lane by lane (ds_bpermute) while UNROLL row loads are
// issued before the adds that consume them, so up to UNROLL rows per group
// are in flight. The adds themselves stay in index order from +0, which
// keeps the result independent of the launch shape and bitwise equal to the
// sequential definition. No atomics: every output row has one owner.
#include "tc_internal.h"

namespace tc {
namespace {

constexpr int kUnroll = 8;

__device__ __forceinline__ float4 f4_add(float4 a, float4 b) {
    return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
}

// FWD: rows come from the table, src row = table_row_offset[bag / B] + ids[j],
//      number of outputs known on the host (num_out_cap).
// !FWD: rows come from grad_out, src row = ids[j] (casted src),
//      number of outputs read from the device (min(*num_out_dev, cap)).
template <int LANES, int CHUNKS, bool FWD>
__global__ __launch_bounds__(kBlock) void k_gather_reduce(
    const float *__restrict__ src, int32_t dim, const int32_t *__restrict__ ids,
    const int32_t *__restrict__ offsets, const int64_t *__restrict__ table_row_offset,
    int32_t bags_per_table, const int32_t *__restrict__ num_out_dev, int64_t num_out_cap,
    float *__restrict__ out) {
    constexpr int kGroups = kWave / LANES;  // output rows per wavefront
    const int lane = threadIdx.x & (kWave - 1);
    const int sub = lane & (LANES - 1);
    const int grp = lane / LANES;
    int64_t num_out = num_out_cap;
    if (!FWD) {
        const int64_t u = *num_out_dev;
        num_out = u < num_out_cap ? u : num_out_cap;
    }
    const int64_t wave = (int64_t(blockIdx.x) * blockDim.x + threadIdx.x) / kWave;
    const int64_t nwave = (int64_t(gridDim.x) * blockDim.x) / kWave;
    const int d4 = dim >> 2;

    for (int64_t o0 = wave * kGroups; o0 < num_out; o0 += nwave * kGroups) {
        const int64_t o = o0 + grp;
        const bool live = o < num_out;
        int32_t beg = 0, end = 0;
        int64_t base = 0;
        if (live) {
            beg = offsets[o];
            end = offsets[o + 1];
            if (FWD) base = table_row_offset[o / bags_per_table];
        }
        float4 acc[CHUNKS];
#pragma unroll
        for (int c = 0; c < CHUNKS; ++c) acc[c] = make_float4(0.f, 0.f, 0.f, 0.f);

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
                // Adding +0 for the slots past the end leaves acc unchanged
                // bit for bit (acc is never -0 when it starts at +0).
#pragma unroll
                for (int u = 0; u < kUnroll; ++u)
#pragma unroll
                    for (int c = 0; c < CHUNKS; ++c) acc[c] = f4_add(acc[c], v[u][c]);
            }
        }
        if (live) {
            float *orow = out + o * int64_t(dim);
#pragma unroll
            for (int c = 0; c < CHUNKS; ++c) {
                const int col4 = sub + c * LANES;
                if (col4 < d4) *reinterpret_cast<float4 *>(orow + 4 * col4) = acc[c];
            }
        }
    }
}

template <bool FWD>
tc_status launch_gather_reduce(const float *src, int32_t dim, const int32_t *ids,
                               const int32_t *offsets, const int64_t *table_row_offset,
                               int32_t bags_per_table, const int32_t *num_out_dev,
                               int64_t num_out_cap, float *out, hipStream_t stream) {
    const RowShape s = row_shape(dim);
    const int64_t rows_per_block = (kBlock / kWave) * (kWave / s.lanes);
    const unsigned grid = grid_for(num_out_cap, rows_per_block, int64_t(kNumCUs) * 8);
#define TC_GR_CASE(L, C)                                                                      \
    if (s.lanes == L && s.chunks == C) {                                                      \
        k_gather_reduce<L, C, FWD><<<grid, kBlock, 0, stream>>>(                               \
            src, dim, ids, offsets, table_row_offset, bags_per_table, num_out_dev, num_out_cap, \
            out);                                                                             \
        return check_launch(FWD ? "k_gather_reduce(forward)" : "k_gather_reduce(backward)"); \
    }
    TC_GR_CASE(1, 1)
    TC_GR_CASE(2, 1)
    TC_GR_CASE(4, 1)
    TC_GR_CASE(8, 1)
    TC_GR_CASE(16, 1)
    TC_GR_CASE(32, 1)
    TC_GR_CASE(64, 1)
    TC_GR_CASE(64, 2)
    TC_GR_CASE(64, 3)
    TC_GR_CASE(64, 4)
#undef TC_GR_CASE
    set_error("no gather-reduce kernel for dim %d", dim);
    return TC_ERR_UNSUPPORTED;
}

}  // namespace
}  // namespace tc

using namespace tc;

extern "C" tc_status tc_embed_forward(const float *W, int64_t total_rows, int32_t dim,
                                      const int64_t *table_row_offset, int32_t num_tables,
                                      int32_t bags_per_table, const int32_t *indices,
                                      const int32_t *bag_offsets, float *out,
                                      hipStream_t stream) {
    clear_error();
    TC_REQUIRE(num_tables >= 0 && bags_per_table >= 0 && total_rows >= 0, TC_ERR_INVALID_ARG,
               "tc_embed_forward: negative size");
    TC_REQUIRE(total_rows < (int64_t(1) << 31), TC_ERR_INVALID_ARG,
               "tc_embed_forward: total_rows must be below 2^31");
    const int64_t num_bags = int64_t(num_tables) * bags_per_table;
    TC_REQUIRE(num_bags < (int64_t(1) << 31), TC_ERR_INVALID_ARG,
               "tc_embed_forward: more than 2^31-1 bags");
    TC_REQUIRE(dim > 0 && dim % 4 == 0 && dim <= kMaxDim, TC_ERR_UNSUPPORTED,
               "tc_embed_forward: dim %d must be a multiple of 4 in [4, %d]", dim, kMaxDim);
    if (num_bags == 0) return TC_OK;
    // indices is only read for bags that have pairs, so it may be NULL for an
    // empty index array
    TC_REQUIRE(W && table_row_offset && bag_offsets && out, TC_ERR_INVALID_ARG,
               "tc_embed_forward: null pointer");
    TC_REQUIRE(aligned16(W) && aligned16(out), TC_ERR_UNSUPPORTED,
               "tc_embed_forward: W and out must be 16-byte aligned");
    return launch_gather_reduce<true>(W, dim, indices, bag_offsets, table_row_offset,
                                      bags_per_table, nullptr, num_bags, out, stream);
}

extern "C" tc_status tc_embed_backward(const float *grad_out, int32_t num_bags, int32_t dim,
                                       const int32_t *seg_offsets, const int32_t *casted_src,
                                       const int32_t *num_unique, int64_t max_unique,
                                       float *coal_grad, hipStream_t stream) {
    clear_error();
    TC_REQUIRE(num_bags >= 0 && max_unique >= 0, TC_ERR_INVALID_ARG,
               "tc_embed_backward: negative size");
    TC_REQUIRE(max_unique < (int64_t(1) << 31), TC_ERR_INVALID_ARG,
               "tc_embed_backward: max_unique must be below 2^31");
    TC_REQUIRE(dim > 0 && dim % 4 == 0 && dim <= kMaxDim, TC_ERR_UNSUPPORTED,
               "tc_embed_backward: dim %d must be a multiple of 4 in [4, %d]", dim, kMaxDim);
    if (max_unique == 0) return TC_OK;
    TC_REQUIRE(grad_out && seg_offsets && casted_src && num_unique && coal_grad,
               TC_ERR_INVALID_ARG, "tc_embed_backward: null pointer");
    TC_REQUIRE(aligned16(grad_out) && aligned16(coal_grad), TC_ERR_UNSUPPORTED,
               "tc_embed_backward: grad_out and coal_grad must be 16-byte aligned");
    return launch_gather_reduce<false>(grad_out, dim, casted_src, seg_offsets, nullptr, 1,
                                       num_unique, max_unique, coal_grad, stream);
}
