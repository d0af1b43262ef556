// Tensor Casting (Algorithm 2) on CDNA4.
//
//  1. k_build_keys   -- (src, dst) pairs from the bag-major CSR index:
//                       key = global row, value = bag id.
//  2. LSD radix sort by key, stable, kRadixBits bits per pass over the
//     ceil(log2(total_rows)) bits that can be set. Each pass is
//       k_radix_hist    per-tile digit counts (LDS histograms, one per wave)
//       k_radix_scan    per-digit exclusive scan over tiles (one block/digit)
//       k_radix_scatter stable scatter: a wave ranks equal digits among its
//                       64 lanes with kRadixBits ballots + popcount, keeps a
//                       running per-digit count per wave in LDS, and waves
//                       are combined in tile order; the tile is laid out in
//                       sorted order in LDS and stored in that order.
//     A pass reads and writes 8 bytes per pair plus a 4-byte read for the
//     histogram. The last pass writes the values straight into casted_src.
//  3. Segment build (the scan and cumulative sum of Algorithm 2):
//       k_seg_count  heads (key differs from its predecessor) per tile
//       k_seg_scan   exclusive scan of tile head counts -> *num_unique
//       k_seg_write  casted_dst, unique_rows, seg_offsets
//
// Tiles are kTile consecutive sorted positions; wave w of a block owns
// positions [w*kWaveSpan, (w+1)*kWaveSpan) of its tile and walks them 64 at a
// time, lane l taking position base + 64*i + l, so tile order = (wave,
// iteration, lane) order and every pass is stable. No atomics on global
// memory; nothing here depends on scheduling order.
#include "tc_internal.h"

namespace tc {
namespace {

constexpr int kRadixBits = 8;
constexpr int kRadix = 1 << kRadixBits;
constexpr int kSortWaves = kBlock / kWave;        // 4
constexpr int kItems = 8;                         // positions per lane per tile
constexpr int kWaveSpan = kWave * kItems;         // 512
constexpr int kTile = kSortWaves * kWaveSpan;     // 2048
static_assert(kRadix == kBlock, "one thread per digit in the per-digit loops");

__device__ __forceinline__ uint64_t lanemask_lt(int lane) { return (uint64_t(1) << lane) - 1; }

// ---------------------------------------------------------------------------
// 1. key build: one group of 16 lanes per bag writes that bag's pairs.
__global__ __launch_bounds__(kBlock) void k_build_keys(
    const int32_t *__restrict__ indices, const int32_t *__restrict__ bag_offsets,
    const int64_t *__restrict__ table_row_offset, int64_t num_bags, int32_t bags_per_table,
    int32_t *__restrict__ keys, int32_t *__restrict__ vals) {
    constexpr int kLanes = 16;
    const int64_t group = (int64_t(blockIdx.x) * blockDim.x + threadIdx.x) / kLanes;
    const int64_t ngroups = (int64_t(gridDim.x) * blockDim.x) / kLanes;
    const int sub = threadIdx.x & (kLanes - 1);
    for (int64_t g = group; g < num_bags; g += ngroups) {
        const int32_t beg = bag_offsets[g], end = bag_offsets[g + 1];
        const int64_t base = table_row_offset[g / bags_per_table];
        for (int32_t j = beg + sub; j < end; j += kLanes) {
            keys[j] = int32_t(base + indices[j]);
            vals[j] = int32_t(g);
        }
    }
}

// ---------------------------------------------------------------------------
// Lanes of a wavefront whose digit equals this lane's (BITS ballots), among
// the lanes where ok holds.
template <int BITS>
__device__ __forceinline__ uint64_t match_digit(uint32_t d, bool ok) {
    uint64_t peers = __ballot(ok);
#pragma unroll
    for (int b = 0; b < BITS; ++b) {
        const bool bit = (d >> b) & 1u;
        const uint64_t m = __ballot(bit);
        peers &= bit ? m : ~m;
    }
    return peers;
}

// 2a. per-tile digit histogram -> counts[digit * num_tiles + tile]. Equal
// digits within a wavefront are counted by one lane (no LDS atomic
// conflicts under skewed keys).
template <int BITS>
__global__ __launch_bounds__(kBlock) void k_radix_hist(const int32_t *__restrict__ keys,
                                                       int64_t n, int shift,
                                                       int32_t *__restrict__ counts,
                                                       int32_t num_tiles) {
    __shared__ int32_t hist[kSortWaves][kRadix];
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    constexpr uint32_t mask = (1u << BITS) - 1u;
    const int64_t base = int64_t(blockIdx.x) * kTile + int64_t(w) * kWaveSpan;
    int32_t key[kItems];
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
        const int64_t j = base + i * kWave + lane;
        key[i] = j < n ? keys[j] : 0;
    }
    for (int i = tid; i < kSortWaves * kRadix; i += kBlock) (&hist[0][0])[i] = 0;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
        const bool ok = base + i * kWave + lane < n;
        const uint32_t d = (uint32_t(key[i]) >> shift) & mask;
        const uint64_t peers = match_digit<BITS>(d, ok);
        if (ok && (peers & lanemask_lt(lane)) == 0) atomicAdd(&hist[w][d], __popcll(peers));
    }
    __syncthreads();
    const int d = tid;
    int32_t s = 0;
#pragma unroll
    for (int ww = 0; ww < kSortWaves; ++ww) s += hist[ww][d];
    counts[int64_t(d) * num_tiles + blockIdx.x] = s;
}

// Block-wide exclusive scan of one value per thread; returns the prefix and
// writes the block total to *total.
__device__ __forceinline__ int32_t block_exclusive_scan(int32_t v, int32_t *total) {
    __shared__ int32_t wsum[kSortWaves];
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    int32_t incl = v;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const int32_t o = __shfl_up(incl, off, kWave);
        if (lane >= off) incl += o;
    }
    if (lane == kWave - 1) wsum[w] = incl;
    __syncthreads();
    int32_t wbase = 0, tot = 0;
#pragma unroll
    for (int ww = 0; ww < kSortWaves; ++ww) {
        const int32_t s = wsum[ww];
        if (ww < w) wbase += s;
        tot += s;
    }
    __syncthreads();  // wsum may be reused by the next call
    *total = tot;
    return wbase + incl - v;
}

// 2b. counts[d][*] -> exclusive prefix over tiles (in place); totals[d].
__global__ __launch_bounds__(kBlock) void k_radix_scan(int32_t *__restrict__ counts,
                                                       int32_t num_tiles,
                                                       int32_t *__restrict__ totals) {
    constexpr int kPer = 4;
    int32_t *row = counts + int64_t(blockIdx.x) * num_tiles;
    int32_t carry = 0;
    for (int32_t base = 0; base < num_tiles; base += kBlock * kPer) {
        int32_t v[kPer], s = 0;
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const int32_t i = base + threadIdx.x * kPer + k;
            v[k] = i < num_tiles ? row[i] : 0;
            s += v[k];
        }
        int32_t tot;
        int32_t p = block_exclusive_scan(s, &tot) + carry;
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const int32_t i = base + threadIdx.x * kPer + k;
            if (i < num_tiles) row[i] = p;
            p += v[k];
        }
        carry += tot;
    }
    if (threadIdx.x == 0) totals[blockIdx.x] = carry;
}

// 2c. stable scatter of one tile. Ranks are computed as described at the
// top: within a wavefront the lanes holding equal digits are found with
// ballots, the lowest of them adds their number to the wave's running count
// of that digit with one LDS atomic (the returned old value is the count of
// that digit in earlier items, since a wave's LDS operations complete in
// order) and the others take it from that lane. The tile is then laid out in
// sorted order in LDS and written back thread by thread in that order, so
// neighbouring threads write neighbouring addresses of the same digit run
// (coalesced stores instead of one scattered store per pair).
template <int BITS>
__global__ __launch_bounds__(kBlock) void k_radix_scatter(
    const int32_t *__restrict__ keys_in, const int32_t *__restrict__ vals_in,
    int32_t *__restrict__ keys_out, int32_t *__restrict__ vals_out, int64_t n, int shift,
    const int32_t *__restrict__ counts, const int32_t *__restrict__ totals,
    int32_t num_tiles) {
    __shared__ int32_t wcount[kSortWaves][kRadix];  // running, then exclusive over waves
    __shared__ int32_t run_start[kSortWaves][kRadix];  // local start of wave w's digit d
    __shared__ int32_t run_shift[kRadix];            // global position - local position
    __shared__ int32_t stage_key[kTile];
    __shared__ int32_t stage_val[kTile];
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    constexpr uint32_t mask = (1u << BITS) - 1u;

    const int64_t base = int64_t(blockIdx.x) * kTile + int64_t(w) * kWaveSpan;
    int32_t key[kItems], val[kItems], rank[kItems];
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
        const int64_t j = base + i * kWave + lane;
        const bool ok = j < n;
        key[i] = ok ? keys_in[j] : 0;
        val[i] = ok ? vals_in[j] : 0;
    }
    const int32_t total_d = totals[tid];
    const int32_t count_d = counts[int64_t(tid) * num_tiles + blockIdx.x];
    for (int i = tid; i < kSortWaves * kRadix; i += kBlock) (&wcount[0][0])[i] = 0;
    int32_t tile_base;  // global start of this tile's run of digit `tid`
    {
        int32_t tot;
        tile_base = block_exclusive_scan(total_d, &tot) + count_d;
    }
    __syncthreads();

    // all atomics first, then the broadcasts, so no item waits for the LDS
    // round trip of the one before it
    int32_t lower_n[kItems], leader[kItems], old[kItems];
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
        const bool ok = base + i * kWave + lane < n;
        const uint32_t d = (uint32_t(key[i]) >> shift) & mask;
        const uint64_t peers = match_digit<BITS>(d, ok);
        const uint64_t lower = peers & lanemask_lt(lane);
        lower_n[i] = __popcll(lower);
        leader[i] = peers ? __builtin_ctzll(peers) : lane;
        old[i] = 0;
        if (ok && lower == 0) old[i] = atomicAdd(&wcount[w][d], __popcll(peers));
    }
    // the leader (lowest peer) holds the count of the digit before this item
#pragma unroll
    for (int i = 0; i < kItems; ++i) rank[i] = __shfl(old[i], leader[i], kWave) + lower_n[i];
    __syncthreads();
    {
        // per digit: exclusive prefix over waves, then over digits
        int32_t s = 0, c[kSortWaves];
#pragma unroll
        for (int ww = 0; ww < kSortWaves; ++ww) c[ww] = wcount[ww][tid];
#pragma unroll
        for (int ww = 0; ww < kSortWaves; ++ww) s += c[ww];
        int32_t tot;
        const int32_t start = block_exclusive_scan(s, &tot);
        int32_t r = start;
#pragma unroll
        for (int ww = 0; ww < kSortWaves; ++ww) {
            run_start[ww][tid] = r;
            r += c[ww];
        }
        run_shift[tid] = tile_base - start;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
        const int64_t j = base + i * kWave + lane;
        if (j < n) {
            const uint32_t d = (uint32_t(key[i]) >> shift) & mask;
            const int32_t lp = run_start[w][d] + rank[i];
            stage_key[lp] = key[i];
            stage_val[lp] = val[i];
        }
    }
    __syncthreads();
    const int64_t tile0 = int64_t(blockIdx.x) * kTile;
    const int32_t in_tile = int32_t(n - tile0 < kTile ? n - tile0 : kTile);
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
        const int32_t lp = i * kBlock + tid;
        if (lp < in_tile) {
            const int32_t k = stage_key[lp];
            const uint32_t d = (uint32_t(k) >> shift) & mask;
            const int32_t pos = run_shift[d] + lp;
            keys_out[pos] = k;
            vals_out[pos] = stage_val[lp];
        }
    }
}

// ---------------------------------------------------------------------------
// 3a. number of segment heads per tile of the sorted keys.
__global__ __launch_bounds__(kBlock) void k_seg_count(const int32_t *__restrict__ keys,
                                                      int64_t n,
                                                      int32_t *__restrict__ tile_heads) {
    __shared__ int32_t wsum[kSortWaves];
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    const int64_t base = int64_t(blockIdx.x) * kTile + int64_t(w) * kWaveSpan;
    int32_t c = 0;
#pragma unroll 4
    for (int i = 0; i < kItems; ++i) {
        const int64_t j = base + i * kWave + lane;
        const bool head = j < n && (j == 0 || keys[j] != keys[j - 1]);
        c += __popcll(__ballot(head));
    }
    if (lane == 0) wsum[w] = c;
    __syncthreads();
    if (tid == 0) {
        int32_t s = 0;
        for (int ww = 0; ww < kSortWaves; ++ww) s += wsum[ww];
        tile_heads[blockIdx.x] = s;
    }
}

// 3b. exclusive scan of the tile head counts (one block); total -> *num_unique.
__global__ __launch_bounds__(kBlock) void k_seg_scan(int32_t *__restrict__ tile_heads,
                                                     int32_t num_tiles,
                                                     int32_t *__restrict__ num_unique) {
    constexpr int kPer = 4;
    int32_t carry = 0;
    for (int32_t base = 0; base < num_tiles; base += kBlock * kPer) {
        int32_t v[kPer], s = 0;
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const int32_t i = base + threadIdx.x * kPer + k;
            v[k] = i < num_tiles ? tile_heads[i] : 0;
            s += v[k];
        }
        int32_t tot;
        int32_t p = block_exclusive_scan(s, &tot) + carry;
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const int32_t i = base + threadIdx.x * kPer + k;
            if (i < num_tiles) tile_heads[i] = p;
            p += v[k];
        }
        carry += tot;
    }
    if (threadIdx.x == 0) *num_unique = carry;
}

// 3c. casted_dst (inclusive head count - 1), unique_rows and seg_offsets.
__global__ __launch_bounds__(kBlock) void k_seg_write(
    const int32_t *__restrict__ keys, int64_t n, const int32_t *__restrict__ tile_heads,
    int32_t *__restrict__ unique_rows, int32_t *__restrict__ seg_offsets,
    int32_t *__restrict__ casted_dst) {
    __shared__ int32_t wsum[kSortWaves];
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    const int64_t base = int64_t(blockIdx.x) * kTile + int64_t(w) * kWaveSpan;
    int32_t key[kItems];
    uint64_t heads[kItems];
    int32_t c = 0;
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
        const int64_t j = base + i * kWave + lane;
        key[i] = j < n ? keys[j] : 0;
        const bool head = j < n && (j == 0 || key[i] != keys[j - 1]);
        heads[i] = __ballot(head);
        c += __popcll(heads[i]);
    }
    if (lane == 0) wsum[w] = c;
    __syncthreads();
    int32_t run = tile_heads[blockIdx.x];
    for (int ww = 0; ww < w; ++ww) run += wsum[ww];
    const uint64_t le = lanemask_lt(lane) | (uint64_t(1) << lane);
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
        const int64_t j = base + i * kWave + lane;
        const int32_t incl = run + __popcll(heads[i] & le);
        if (j < n) {
            if (casted_dst) casted_dst[j] = incl - 1;
            if ((heads[i] >> lane) & 1u) {
                unique_rows[incl - 1] = key[i];
                seg_offsets[incl - 1] = int32_t(j);
            }
            if (j == n - 1) seg_offsets[incl] = int32_t(n);
        }
        run += __popcll(heads[i]);
    }
}

// No pairs: zero segments, seg_offsets[0] = 0.
__global__ void k_cast_empty(int32_t *seg_offsets, int32_t *num_unique) {
    if (threadIdx.x == 0) {
        seg_offsets[0] = 0;
        *num_unique = 0;
    }
}

// One LSD pass over `bits` (1..kRadixBits) digit bits starting at `shift`.
tc_status launch_radix_pass(int bits, const int32_t *kin, const int32_t *vin, int32_t *kout,
                            int32_t *vout, int64_t n, int shift, int32_t *counts,
                            int32_t *totals, int32_t tiles, hipStream_t stream) {
#define TC_PASS_CASE(B)                                                                      \
    case B:                                                                                  \
        k_radix_hist<B><<<tiles, kBlock, 0, stream>>>(kin, n, shift, counts, tiles);         \
        if (check_launch("k_radix_hist") != TC_OK) return TC_ERR_HIP;                        \
        k_radix_scan<<<kRadix, kBlock, 0, stream>>>(counts, tiles, totals);                  \
        if (check_launch("k_radix_scan") != TC_OK) return TC_ERR_HIP;                        \
        k_radix_scatter<B><<<tiles, kBlock, 0, stream>>>(kin, vin, kout, vout, n, shift,     \
                                                         counts, totals, tiles);             \
        return check_launch("k_radix_scatter");
    switch (bits) {
        TC_PASS_CASE(1)
        TC_PASS_CASE(2)
        TC_PASS_CASE(3)
        TC_PASS_CASE(4)
        TC_PASS_CASE(5)
        TC_PASS_CASE(6)
        TC_PASS_CASE(7)
        TC_PASS_CASE(8)
        default:
            break;
    }
#undef TC_PASS_CASE
    set_error("no radix pass for %d bits", bits);
    return TC_ERR_UNSUPPORTED;
}
static_assert(kRadixBits == 8, "launch_radix_pass instantiates 1..8 bits");

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct CastPlan {
    int64_t num_tiles;
    size_t off_ka, off_va, off_kb, off_vb, off_counts, off_totals, off_heads, bytes;
};

inline CastPlan cast_plan(int64_t n) {
    CastPlan p{};
    p.num_tiles = (n + kTile - 1) / kTile;
    const size_t arr = align_up(size_t(n) * 4);
    size_t o = 0;
    p.off_ka = o; o += arr;
    p.off_va = o; o += arr;
    p.off_kb = o; o += arr;
    p.off_vb = o; o += arr;
    p.off_counts = o; o += align_up(size_t(kRadix) * size_t(p.num_tiles) * 4);
    p.off_totals = o; o += align_up(size_t(kRadix) * 4);
    p.off_heads = o; o += align_up(size_t(p.num_tiles) * 4);
    p.bytes = o;
    return p;
}

inline int key_bits(int64_t total_rows) {
    int b = 0;
    while (b < 31 && (int64_t(1) << b) < total_rows) ++b;
    return b < 1 ? 1 : b;  // at least one pass, so the values are always moved
}

}  // namespace
}  // namespace tc

using namespace tc;

extern "C" size_t tc_cast_workspace_bytes(int64_t num_pairs, int64_t total_rows) {
    (void)total_rows;
    if (num_pairs < 0) return 0;
    return cast_plan(num_pairs).bytes;
}

extern "C" tc_status tc_cast_index(const int64_t *table_row_offset, int32_t num_tables,
                                   int32_t bags_per_table, int64_t total_rows,
                                   const int32_t *indices, const int32_t *bag_offsets,
                                   int64_t num_pairs, int32_t *unique_rows, int32_t *seg_offsets,
                                   int32_t *casted_src, int32_t *casted_dst, int32_t *num_unique,
                                   void *workspace, size_t workspace_bytes, hipStream_t stream) {
    clear_error();
    TC_REQUIRE(num_tables >= 0 && bags_per_table >= 0 && total_rows >= 0 && num_pairs >= 0,
               TC_ERR_INVALID_ARG, "tc_cast_index: negative size");
    TC_REQUIRE(total_rows < (int64_t(1) << 31) && num_pairs < (int64_t(1) << 31),
               TC_ERR_INVALID_ARG, "tc_cast_index: total_rows and num_pairs must be below 2^31");
    const int64_t num_bags = int64_t(num_tables) * bags_per_table;
    TC_REQUIRE(num_bags < (int64_t(1) << 31), TC_ERR_INVALID_ARG,
               "tc_cast_index: more than 2^31-1 bags");
    TC_REQUIRE(seg_offsets && num_unique, TC_ERR_INVALID_ARG, "tc_cast_index: null pointer");
    if (num_pairs == 0) {
        k_cast_empty<<<1, kWave, 0, stream>>>(seg_offsets, num_unique);
        return check_launch("k_cast_empty");
    }
    TC_REQUIRE(num_bags > 0 && total_rows > 0, TC_ERR_INVALID_ARG,
               "tc_cast_index: pairs without bags or rows");
    TC_REQUIRE(table_row_offset && indices && bag_offsets && unique_rows && casted_src,
               TC_ERR_INVALID_ARG, "tc_cast_index: null pointer");
    const CastPlan plan = cast_plan(num_pairs);
    TC_REQUIRE(workspace && workspace_bytes >= plan.bytes, TC_ERR_WORKSPACE,
               "tc_cast_index: workspace of %zu bytes, %zu needed", workspace_bytes, plan.bytes);
    TC_REQUIRE((reinterpret_cast<uintptr_t>(workspace) & (kAlign - 1)) == 0, TC_ERR_WORKSPACE,
               "tc_cast_index: workspace must be 256-byte aligned");
    TC_REQUIRE(plan.num_tiles < (int64_t(1) << 31) / kRadix, TC_ERR_INVALID_ARG,
               "tc_cast_index: too many pairs");

    char *ws = static_cast<char *>(workspace);
    int32_t *ka = reinterpret_cast<int32_t *>(ws + plan.off_ka);
    int32_t *va = reinterpret_cast<int32_t *>(ws + plan.off_va);
    int32_t *kb = reinterpret_cast<int32_t *>(ws + plan.off_kb);
    int32_t *vb = reinterpret_cast<int32_t *>(ws + plan.off_vb);
    int32_t *counts = reinterpret_cast<int32_t *>(ws + plan.off_counts);
    int32_t *totals = reinterpret_cast<int32_t *>(ws + plan.off_totals);
    int32_t *heads = reinterpret_cast<int32_t *>(ws + plan.off_heads);
    const int32_t tiles = int32_t(plan.num_tiles);

    {
        const unsigned grid = grid_for(num_bags, kBlock / 16, int64_t(kNumCUs) * 8);
        k_build_keys<<<grid, kBlock, 0, stream>>>(indices, bag_offsets, table_row_offset,
                                                  num_bags, bags_per_table, ka, va);
        tc_status st = check_launch("k_build_keys");
        if (st != TC_OK) return st;
    }

    const int bits = key_bits(total_rows);
    const int passes = (bits + kRadixBits - 1) / kRadixBits;
    const int per_pass = (bits + passes - 1) / passes;
    int32_t *kin = ka, *vin = va, *kout = kb, *vout = vb;
    for (int p = 0; p < passes; ++p) {
        const int shift = p * per_pass;
        const int pb = (shift + per_pass <= bits) ? per_pass : bits - shift;
        const bool last = p == passes - 1;
        int32_t *vdst = last ? casted_src : vout;
        tc_status st = launch_radix_pass(pb, kin, vin, kout, vdst, num_pairs, shift, counts,
                                         totals, tiles, stream);
        if (st != TC_OK) return st;
        // next pass reads what this one wrote
        int32_t *tk = kin, *tv = vin;
        kin = kout;
        vin = vout;
        kout = tk;
        vout = tv;
    }
    const int32_t *sorted_keys = kin;

    k_seg_count<<<tiles, kBlock, 0, stream>>>(sorted_keys, num_pairs, heads);
    tc_status st = check_launch("k_seg_count");
    if (st != TC_OK) return st;
    k_seg_scan<<<1, kBlock, 0, stream>>>(heads, tiles, num_unique);
    st = check_launch("k_seg_scan");
    if (st != TC_OK) return st;
    k_seg_write<<<tiles, kBlock, 0, stream>>>(sorted_keys, num_pairs, heads, unique_rows,
                                              seg_offsets, casted_dst);
    return check_launch("k_seg_write");
}
