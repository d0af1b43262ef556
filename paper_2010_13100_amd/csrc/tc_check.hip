// Device-side check of the bag-major CSR index (the (src, dst) pairs of
// Sec. II-B) against the layout the other entry points assume without
// checking it: table and bag offsets that start at 0, never decrease and end
// at the row and pair counts, and every index inside its table (and under the
// caller's table-size bound). An index outside its table would make the
// forward pass read, and the update write, outside the embedding table.
//
// Three launches: the report word is set to "no problem", one grid-stride
// kernel folds every violation it finds into that word with an atomic
// minimum (one per wavefront that found any), and a one-thread kernel
// decodes it. The minimum of (kind << 56 | position) is the lowest kind,
// then the lowest position, whatever the scheduling order.
#include "tc_internal.h"

namespace tc {
namespace {

constexpr uint64_t kNoProblem = ~uint64_t(0);
constexpr int kKindShift = 56;
constexpr int kStagedTables = 1024;  // table pair starts kept in LDS up to this many tables

__device__ __forceinline__ uint64_t problem(int kind, int64_t pos) {
    return (uint64_t(kind) << kKindShift) | uint64_t(pos);
}

// Wave-wide minimum of v into *slot. Called by every lane of the wavefront.
__device__ __forceinline__ void fold_min(uint64_t v, unsigned long long *slot) {
    if (!__any(v != kNoProblem)) return;
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
        const uint32_t lo = __shfl_xor(uint32_t(v), off, kWave);
        const uint32_t hi = __shfl_xor(uint32_t(v >> 32), off, kWave);
        const uint64_t o = (uint64_t(hi) << 32) | lo;
        v = o < v ? o : v;
    }
    if ((threadIdx.x & (kWave - 1)) == 0) atomicMin(slot, static_cast<unsigned long long>(v));
}

__global__ void k_check_init(int64_t *report) {
    report[0] = TC_INDEX_OK;
    report[1] = int64_t(kNoProblem);
}

__global__ __launch_bounds__(kBlock) void k_check_index(
    const int64_t *__restrict__ table_row_offset, int32_t num_tables, int32_t bags_per_table,
    int64_t total_rows, int64_t max_table_rows, const int32_t *__restrict__ indices,
    const int32_t *__restrict__ bag_offsets, int64_t num_pairs, int64_t *report) {
    auto *slot = reinterpret_cast<unsigned long long *>(report + 1);
    const int64_t num_bags = int64_t(num_tables) * bags_per_table;
    const int64_t stride = int64_t(gridDim.x) * blockDim.x;
    const int64_t first = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    // loop bounds rounded up to a multiple of the stride, so that every
    // thread makes the same number of trips and whole wavefronts call
    // fold_min (which shuffles across the wavefront) together
    auto rounded = [stride](int64_t n) { return (n + stride - 1) / stride * stride; };
    const int64_t end_t = rounded(int64_t(num_tables) + 1), end_g = rounded(num_bags + 1),
                  end_j = rounded(num_pairs);

    // kind 1: table_row_offset, entries 0..T
    for (int64_t t = first; t < end_t; t += stride) {
        uint64_t v = kNoProblem;
        if (t <= num_tables) {
            const int64_t o = table_row_offset[t];
            const bool bad = (t == 0 && o != 0) || (t > 0 && o < table_row_offset[t - 1]) ||
                             (t == num_tables && o != total_rows);
            if (bad) v = problem(TC_INDEX_BAD_TABLE_OFFSETS, t);
        }
        fold_min(v, slot);
    }
    // kind 2: bag_offsets, entries 0..T*B
    for (int64_t g = first; g < end_g; g += stride) {
        uint64_t v = kNoProblem;
        if (g <= num_bags) {
            const int32_t o = bag_offsets[g];
            const bool bad = (g == 0 && o != 0) || (g > 0 && o < bag_offsets[g - 1]) ||
                             (g == num_bags && o != num_pairs);
            if (bad) v = problem(TC_INDEX_BAD_BAG_OFFSETS, g);
        }
        fold_min(v, slot);
    }
    if (num_tables == 0) return;  // uniform: no table to hold any pair

    // kind 3: the table of pair j is the last t whose first pair
    // bag_offsets[t*B] is at most j (tables without pairs are passed over).
    // With malformed offsets the search still ends inside [0, T).
    __shared__ int32_t tstart[kStagedTables];
    const bool staged = num_tables <= kStagedTables;
    if (staged) {
        for (int t = threadIdx.x; t < num_tables; t += blockDim.x)
            tstart[t] = bag_offsets[int64_t(t) * bags_per_table];
        __syncthreads();
    }
    for (int64_t j = first; j < end_j; j += stride) {
        uint64_t v = kNoProblem;
        if (j < num_pairs) {
            int32_t lo = 0, hi = num_tables - 1;
            while (lo < hi) {
                const int32_t mid = lo + (hi - lo + 1) / 2;
                const int32_t s = staged ? tstart[mid] : bag_offsets[int64_t(mid) * bags_per_table];
                if (s <= j) lo = mid; else hi = mid - 1;
            }
            const int64_t rows = table_row_offset[lo + 1] - table_row_offset[lo];
            const int64_t idx = indices[j];
            if (idx < 0 || idx >= rows || (max_table_rows > 0 && idx >= max_table_rows))
                v = problem(TC_INDEX_OUT_OF_RANGE, j);
        }
        fold_min(v, slot);
    }
}

__global__ void k_check_finish(int64_t *report) {
    const uint64_t v = uint64_t(report[1]);
    if (v == kNoProblem) {
        report[0] = TC_INDEX_OK;
        report[1] = -1;
    } else {
        report[0] = int64_t(v >> kKindShift);
        report[1] = int64_t(v & ((uint64_t(1) << kKindShift) - 1));
    }
}

}  // namespace
}  // namespace tc

using namespace tc;

extern "C" tc_status tc_check_index(const int64_t *table_row_offset, int32_t num_tables,
                                    int32_t bags_per_table, int64_t total_rows,
                                    int64_t max_table_rows, const int32_t *indices,
                                    const int32_t *bag_offsets, int64_t num_pairs,
                                    int64_t *report, hipStream_t stream) {
    clear_error();
    TC_REQUIRE(num_tables >= 0 && bags_per_table >= 0 && total_rows >= 0 && num_pairs >= 0 &&
                   max_table_rows >= 0,
               TC_ERR_INVALID_ARG, "tc_check_index: negative size");
    TC_REQUIRE(total_rows < (int64_t(1) << 31) && num_pairs < (int64_t(1) << 31),
               TC_ERR_INVALID_ARG, "tc_check_index: total_rows and num_pairs must be below 2^31");
    const int64_t num_bags = int64_t(num_tables) * bags_per_table;
    TC_REQUIRE(num_bags < (int64_t(1) << 31), TC_ERR_INVALID_ARG,
               "tc_check_index: more than 2^31-1 bags");
    TC_REQUIRE(table_row_offset && bag_offsets && report && (indices || num_pairs == 0),
               TC_ERR_INVALID_ARG, "tc_check_index: null pointer");
    TC_REQUIRE((reinterpret_cast<uintptr_t>(report) & 7u) == 0, TC_ERR_INVALID_ARG,
               "tc_check_index: report must be 8-byte aligned");
    k_check_init<<<1, 1, 0, stream>>>(report);
    if (tc_status s = check_launch("tc_check_index"); s != TC_OK) return s;
    int64_t items = num_pairs;
    if (num_bags + 1 > items) items = num_bags + 1;
    if (int64_t(num_tables) + 1 > items) items = int64_t(num_tables) + 1;
    const unsigned grid = grid_for(items, int64_t(kBlock) * 4, int64_t(device_cus()) * 8);
    k_check_index<<<grid, kBlock, 0, stream>>>(table_row_offset, num_tables, bags_per_table,
                                               total_rows, max_table_rows, indices, bag_offsets,
                                               num_pairs, report);
    if (tc_status s = check_launch("tc_check_index"); s != TC_OK) return s;
    k_check_finish<<<1, 1, 0, stream>>>(report);
    return check_launch("tc_check_index");
}
