// Gather-reduce on CDNA4: the forward embedding pass (Sec. II-B) and the
// casted gradient gather-reduce (Algorithm 3) are the same operation -- an
// output row is the ordered sum of source rows named by an index range -- and
// share the same lane-group walk, as the paper unifies them under one
// operator.
//
// Mapping: a group of LANES lanes (a power of two <= 64) owns one output
// row; each lane holds CHUNKS float4 column chunks (dwordx4 loads), so one
// row of 4*dim bytes is read by one vector instruction per chunk. The group
// walks its index range in order: LANES indices are fetched at once, one per
// lane, then broadcast lane by lane (ds_bpermute) while kUnroll row loads are
// issued before the adds that consume them. The adds themselves stay in index
// order from +0, which keeps the result independent of the launch shape and
// bitwise equal to the sequential definition. No atomics: every output row
// has one owner.
//
// This file holds the forward; the backward (with its long-segment path) is
// in tc_backward.hip.
#include "tc_group_sum.h"

namespace tc {
namespace {

// Forward: one output row per bag, source row = table_row_offset[bag / B] + ids[j].
template <int LANES, int CHUNKS>
__global__ __launch_bounds__(kBlock) void k_forward(FwdSlice f) {
    const int64_t wave = (int64_t(blockIdx.x) * blockDim.x + threadIdx.x) / kWave;
    const int64_t nwave = (int64_t(gridDim.x) * blockDim.x) / kWave;
    forward_bags<LANES, CHUNKS>(f, wave, nwave);
}

}  // namespace

tc_status launch_forward(const float *W, int32_t dim, const int32_t *ids, const int32_t *offsets,
                         const int64_t *table_row_offset, int32_t bags_per_table,
                         int64_t num_bags, float *out, hipStream_t stream) {
    const RowShape s = row_shape(dim);
    const int64_t rows_per_block = (kBlock / kWave) * (kWave / s.lanes);
    // up to 32 workgroups per CU in the grid (8 are resident at a time): on
    // 33 GB tables the random row reads finish about 3% sooner than with 8
    const unsigned grid = grid_for(num_bags, rows_per_block, int64_t(device_cus()) * 32);
    const FwdSlice f{W, ids, offsets, table_row_offset, out, 0, num_bags, dim, bags_per_table};
#define TC_FWD_CASE(L, C)                                                                      \
    if (s.lanes == L && s.chunks == C) {                                                       \
        k_forward<L, C><<<grid, kBlock, 0, stream>>>(f);                                       \
        return check_launch("k_forward");                                                      \
    }
    TC_FWD_CASE(1, 1)
    TC_FWD_CASE(2, 1)
    TC_FWD_CASE(4, 1)
    TC_FWD_CASE(8, 1)
    TC_FWD_CASE(16, 1)
    TC_FWD_CASE(32, 1)
    TC_FWD_CASE(64, 1)
    TC_FWD_CASE(64, 2)
    TC_FWD_CASE(64, 3)
    TC_FWD_CASE(64, 4)
#undef TC_FWD_CASE
    set_error("no forward kernel for dim %d", dim);
    return TC_ERR_UNSUPPORTED;
}

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
    return launch_forward(W, dim, indices, bag_offsets, table_row_offset, bags_per_table,
                          num_bags, out, stream);
}

