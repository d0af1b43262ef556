// Backward: the casted gradient gather-reduce (Algorithm 3) on CDNA4.
//
// coal_grad[u] is the ordered sum of grad_out rows casted_src[j] over the
// segment j in [seg_offsets[u], seg_offsets[u+1]). Segment lengths follow the
// index skew: under Zipf lookups a few table rows own tens of thousands of
// pairs, and each such sum is a dependency chain that must stay in order to
// keep the result bitwise equal to the sequential definition. Two kernels
// split the work by segment length:
//
//  k_backward_long   segments of at least kLongSegment pairs. One wavefront
//                    per (segment, 16-column part); each load instruction
//                    brings 4 rows of the part into neighbouring lanes, a
//                    register ring keeps 64 loads (256 rows) in flight, and
//                    the ordered adds take the rows through DPP row shifts
//                    (column_chain).
//  k_backward_short  the other segments: lane groups exactly as the forward.
//
// The long kernel is launched first; both only read their inputs and write
// disjoint rows of coal_grad. No atomics anywhere.
#include <type_traits>

#include "tc_group_sum.h"

namespace tc {
namespace {

// Segments at least this long go to k_backward_long.
constexpr int kLongSegment = 128;
// Columns per long-chain wavefront, and rows per load instruction: a
// wavefront issues about one load instruction per 32 cycles, so each load
// brings 4 rows (of 64 bytes; narrower pieces cost more memory requests).
constexpr int kChainCols = 16;
constexpr int kRowsPerLoad = kWave / kChainCols;  // 4
constexpr int kGroupsPerIdVector = kWave / kRowsPerLoad;  // 16 groups = 64 rows
// Groups (one load each) a chain keeps in flight: four id blocks.
constexpr int kRing = 4 * kGroupsPerIdVector;  // 64 loads, 256 rows
// Blocks of the long kernel; each scans its own range of segments and has up
// to kMaxLongWaves wavefronts.
constexpr int kLongBlocks = 1024;
constexpr int kMaxLongWaves = 8;
// Buffer resource word 3 for gfx9-family buffers; out-of-range reads give 0.
constexpr int32_t kBufferWord3 = 0x00020000;

// Per-wavefront LDS table of the byte offsets of the rows of one block.
struct ChainLds {
    int32_t offs[kWave];
};

// v of the lane K places up within each row of 16 lanes (DPP row_shl:K).
// All 64 lanes are active wherever this is used, and the lanes that keep the
// result read within their row, so the bound_ctrl setting (which lets the
// compiler fold the move into the add) never changes a kept value.
template <int K>
__device__ __forceinline__ float lane_up(float v) {
    return __builtin_bit_cast(
        float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x100 + K, 0xf, 0xf, true));
}

// acc + the lane's group of kRowsPerLoad rows (its own value, then those of
// the next lanes), in order.
__device__ __forceinline__ float add_group(float acc, float x) {
    acc = acc + x;
    acc = acc + lane_up<1>(x);
    acc = acc + lane_up<2>(x);
    acc = acc + lane_up<3>(x);
    return acc;
}
// The same for only the first n rows of the group.
__device__ __forceinline__ float add_group_partial(float acc, float x, int32_t n) {
    if (n > 0) acc = acc + x;
    if (n > 1) acc = acc + lane_up<1>(x);
    if (n > 2) acc = acc + lane_up<2>(x);
    if (n > 3) acc = acc + lane_up<3>(x);
    return acc;
}
static_assert(kRowsPerLoad == 4, "add_group adds four rows");

// One wavefront sums rows ids[beg..end) of grad for the kChainCols columns
// [q0, q0+16) in order. Lane l reads column q0 + l/4 of row 4g + l%4 of
// group g, so one dword load brings 4 rows (64 bytes each) and the four rows
// of a column sit in four neighbouring lanes; lane 4c adds them in order
// through DPP row shifts, which need no LDS and fold into the adds.
// Loads are buffer loads (row byte offset + lane column offset) against a
// resource spanning the segment's rows, whose ids are sorted; ids are read
// 64 at a time (one per lane, positions clamped into the segment) eight id
// blocks ahead of use, so waiting for them never drains the ring, and a
// block's row offsets pass through a small LDS table. The ring holds kRing
// loads (256 rows); the slot of group g is g % kRing, refilled with group
// g + kRing right after it is consumed. Scheduling barriers every 4 groups
// keep loads and adds from being regrouped. Rows past the end are skipped.
__device__ void column_chain(ChainLds &lds, const float *__restrict__ grad, int32_t dim,
                              const int32_t *__restrict__ ids, int32_t beg, int32_t end,
                              int32_t q0, float *__restrict__ out_row) {
    const int lane = threadIdx.x & (kWave - 1);
    const int row_sel = lane & (kRowsPerLoad - 1);
    const int32_t col = q0 + lane / kRowsPerLoad;
    const int32_t rcol = col < dim ? col : dim - 1;  // column this lane reads
    const int32_t len = end - beg;
    const int32_t *sid = ids + beg;
    const int32_t first = __builtin_amdgcn_readfirstlane(sid[0]);
    const int32_t last = __builtin_amdgcn_readfirstlane(sid[len - 1]);
    const int32_t row_bytes = dim * 4;
    const uint64_t span = uint64_t(last - first + 1) * uint64_t(row_bytes);
    const bool writer = row_sel == 0 && col < dim;
    if (span >= (uint64_t(1) << 31)) {
        // rows spread over 2 GiB or more: plain 64-bit addressed loads
        float acc = 0.f;
        const float *colp = grad + rcol;
        for (int32_t k = 0; k < len; ++k) acc = acc + colp[int64_t(sid[k]) * dim];
        if (writer) out_row[col] = acc;
        return;
    }
    const auto rsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float *>(grad + int64_t(first) * dim), 0, int32_t(span), kBufferWord3);
    const int32_t lane_bytes = rcol * 4;
    // ids of block k (rows 64k..64k+63), one per lane; positions clamped into
    // the segment
    auto load_ids = [&](int32_t k) -> int32_t { return sid[min(k * kWave + lane, len - 1)]; };
    auto set_offsets = [&](int32_t idv) { lds.offs[lane] = (idv - first) * row_bytes; };
    auto group_offset = [&](int gi) -> int32_t { return lds.offs[gi * kRowsPerLoad + row_sel]; };
    auto load_group = [&](int32_t off) -> float {
        return __builtin_bit_cast(
            float, __builtin_amdgcn_raw_buffer_load_b32(rsrc, off + lane_bytes, 0, 0));
    };

    // Block B's ids live in iv[B % 8] from 8 blocks before the block that
    // uses them (block B-4 refills the ring with block B). Issue every id load
    // of blocks 0..11 before the first row load.
    int32_t iv[8];
    const int32_t p0 = load_ids(0), p1 = load_ids(1), p2 = load_ids(2), p3 = load_ids(3);
#pragma unroll
    for (int k = 0; k < 8; ++k) iv[k] = load_ids(k < 4 ? k + 8 : k);
    float ring[kRing];
    {
        const int32_t pk[4] = {p0, p1, p2, p3};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            set_offsets(pk[k]);
#pragma unroll
            for (int gi = 0; gi < kGroupsPerIdVector; ++gi)
                ring[k * kGroupsPerIdVector + gi] = load_group(group_offset(gi));
        }
    }

    float acc = 0.f;
    // A full block blk (64 rows; B = blk % 8 at compile time): consume its
    // ring slots (those of blk % 4) and refill them with block blk + 4.
    auto full_block = [&](auto bconst, int32_t blk) {
        constexpr int B = decltype(bconst)::value;
        set_offsets(iv[(B + 4) % 8]);
        int32_t offs[kGroupsPerIdVector];
#pragma unroll
        for (int gi = 0; gi < kGroupsPerIdVector; ++gi) offs[gi] = group_offset(gi);
#pragma unroll
        for (int gi = 0; gi < kGroupsPerIdVector; ++gi) {
            const int slot = (B % 4) * kGroupsPerIdVector + gi;
            acc = add_group(acc, ring[slot]);
            ring[slot] = load_group(offs[gi]);
            if (gi % 4 == 3) __builtin_amdgcn_sched_barrier(0);
        }
        iv[(B + 4) % 8] = load_ids(blk + 12);
    };
    // The partial last block (fewer than 64 rows left; Q = blk % 4).
    auto last_block = [&](auto qconst, int32_t rows_left) {
        constexpr int Q = decltype(qconst)::value;
#pragma unroll
        for (int gi = 0; gi < kGroupsPerIdVector; ++gi) {
            acc = add_group_partial(acc, ring[Q * kGroupsPerIdVector + gi],
                                    rows_left - gi * kRowsPerLoad);
        }
    };
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2>;
    using I3 = std::integral_constant<int, 3>;
    using I4 = std::integral_constant<int, 4>;
    using I5 = std::integral_constant<int, 5>;
    using I6 = std::integral_constant<int, 6>;
    using I7 = std::integral_constant<int, 7>;
    // Only full blocks run in the loop, and it is left by early exits, so
    // no partial path joins the steady state (which would make the compiler
    // wait for every outstanding load).
    int32_t blk = 0;
    for (;;) {
        if (len - blk * kWave < kWave) break;
        full_block(I0{}, blk++);
        if (len - blk * kWave < kWave) break;
        full_block(I1{}, blk++);
        if (len - blk * kWave < kWave) break;
        full_block(I2{}, blk++);
        if (len - blk * kWave < kWave) break;
        full_block(I3{}, blk++);
        if (len - blk * kWave < kWave) break;
        full_block(I4{}, blk++);
        if (len - blk * kWave < kWave) break;
        full_block(I5{}, blk++);
        if (len - blk * kWave < kWave) break;
        full_block(I6{}, blk++);
        if (len - blk * kWave < kWave) break;
        full_block(I7{}, blk++);
    }
    const int32_t rows_left = len - blk * kWave;
    if (rows_left > 0) {
        switch (blk % 4) {
            case 0: last_block(I0{}, rows_left); break;
            case 1: last_block(I1{}, rows_left); break;
            case 2: last_block(I2{}, rows_left); break;
            default: last_block(I3{}, rows_left); break;
        }
    }
    if (writer) out_row[col] = acc;
}

// Each block scans a contiguous range of segments; its wavefronts split the
// 16-column parts of every long segment found. A first pass reads every
// 64th offset: a batch of 64 segments spanning fewer than kLongSegment pairs
// cannot hold a long one and is skipped without reading its offsets.
__global__ __launch_bounds__(512) void k_backward_long(
    const float *__restrict__ grad, int32_t dim, const int32_t *__restrict__ ids,
    const int32_t *__restrict__ offsets, const int32_t *__restrict__ num_out_dev,
    int64_t num_out_cap, float *__restrict__ out) {
    __shared__ ChainLds chain_lds[kMaxLongWaves];
    const int lane = threadIdx.x & (kWave - 1);
    const int w = threadIdx.x / kWave;
    const int nw = blockDim.x / kWave;
    const int32_t parts = (dim + kChainCols - 1) / kChainCols;
    const int64_t u_dev = *num_out_dev;
    const int64_t num = u_dev < num_out_cap ? u_dev : num_out_cap;
    const int64_t per = (num + gridDim.x - 1) / gridDim.x;
    const int64_t r0 = int64_t(blockIdx.x) * per;
    const int64_t r1 = r0 + per < num ? r0 + per : num;
    for (int64_t c0 = r0; c0 < r1; c0 += int64_t(kWave) * kWave) {
        const int64_t s0 = c0 + int64_t(kWave) * lane;  // this lane's batch
        const int32_t os = offsets[s0 < r1 ? s0 : r1];
        const int64_t s1 = s0 + kWave < r1 ? s0 + kWave : r1;
        const int32_t oe = offsets[s1];
        uint64_t batches = __ballot(s0 < r1 && oe - os >= kLongSegment);
        while (batches) {
            const int i = __builtin_ctzll(batches);
            batches &= batches - 1;
            const int64_t u = c0 + int64_t(kWave) * i + lane;
            int32_t o0 = 0, o1 = 0;
            if (u < r1) {
                o0 = offsets[u];
                o1 = offsets[u + 1];
            }
            uint64_t longs = __ballot(u < r1 && o1 - o0 >= kLongSegment);
            while (longs) {
                const int j = __builtin_ctzll(longs);
                longs &= longs - 1;
                const int32_t b = __builtin_amdgcn_readlane(o0, j);
                const int32_t e = __builtin_amdgcn_readlane(o1, j);
                const int64_t seg = c0 + int64_t(kWave) * i + j;
                for (int32_t q = w; q < parts; q += nw)
                    column_chain(chain_lds[w], grad, dim, ids, b, e, q * kChainCols,
                                 out + seg * int64_t(dim));
            }
        }
    }
}

// Short segments: one lane group per segment, as the forward; long ones are
// left to k_backward_long.
template <int LANES, int CHUNKS>
__global__ __launch_bounds__(kBlock) void k_backward_short(
    const float *__restrict__ grad, int32_t dim, const int32_t *__restrict__ ids,
    const int32_t *__restrict__ offsets, const int32_t *__restrict__ num_out_dev,
    int64_t num_out_cap, float *__restrict__ out) {
    constexpr int kGroups = kWave / LANES;
    const int lane = threadIdx.x & (kWave - 1);
    const int sub = lane & (LANES - 1);
    const int grp = lane / LANES;
    const int64_t u_dev = *num_out_dev;
    const int64_t num = u_dev < num_out_cap ? u_dev : num_out_cap;
    const int64_t wave = (int64_t(blockIdx.x) * blockDim.x + threadIdx.x) / kWave;
    const int64_t nwave = (int64_t(gridDim.x) * blockDim.x) / kWave;
    for (int64_t o0 = wave * kGroups; o0 < num; o0 += nwave * kGroups) {
        const int64_t o = o0 + grp;
        int32_t beg = 0, end = 0;
        bool mine = false;
        if (o < num) {
            beg = offsets[o];
            end = offsets[o + 1];
            mine = end - beg < kLongSegment;
            if (!mine) end = beg;
        }
        float4 acc[CHUNKS];
#pragma unroll
        for (int c = 0; c < CHUNKS; ++c) acc[c] = make_float4(0.f, 0.f, 0.f, 0.f);
        group_range_sum<LANES, CHUNKS>(grad, dim, ids, 0, beg, end, sub, acc);
        if (mine) group_store<LANES, CHUNKS>(out + o * int64_t(dim), dim, sub, acc);
    }
}

tc_status launch_backward(const float *grad, int32_t dim, const int32_t *ids,
                          const int32_t *offsets, const int32_t *num_out_dev, int64_t cap,
                          float *out, hipStream_t stream) {
    const int parts = (dim + kChainCols - 1) / kChainCols;
    const int long_waves = parts < kMaxLongWaves ? parts : kMaxLongWaves;
    k_backward_long<<<kLongBlocks, long_waves * kWave, 0, stream>>>(grad, dim, ids, offsets,
                                                                     num_out_dev, cap, out);
    tc_status st = check_launch("k_backward_long");
    if (st != TC_OK) return st;
    const RowShape s = row_shape(dim);
    const int64_t rows_per_block = (kBlock / kWave) * (kWave / s.lanes);
    const unsigned grid = grid_for(cap, rows_per_block, int64_t(kNumCUs) * 8);
#define TC_BWD_CASE(L, C)                                                                    \
    if (s.lanes == L && s.chunks == C) {                                                     \
        k_backward_short<L, C><<<grid, kBlock, 0, stream>>>(grad, dim, ids, offsets,          \
                                                            num_out_dev, cap, out);          \
        return check_launch("k_backward_short");                                             \
    }
    TC_BWD_CASE(1, 1)
    TC_BWD_CASE(2, 1)
    TC_BWD_CASE(4, 1)
    TC_BWD_CASE(8, 1)
    TC_BWD_CASE(16, 1)
    TC_BWD_CASE(32, 1)
    TC_BWD_CASE(64, 1)
    TC_BWD_CASE(64, 2)
    TC_BWD_CASE(64, 3)
    TC_BWD_CASE(64, 4)
#undef TC_BWD_CASE
    set_error("no backward kernel for dim %d", dim);
    return TC_ERR_UNSUPPORTED;
}

}  // namespace
}  // namespace tc

using namespace tc;

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
    return launch_backward(grad_out, dim, casted_src, seg_offsets, num_unique, max_unique,
                           coal_grad, stream);
}
