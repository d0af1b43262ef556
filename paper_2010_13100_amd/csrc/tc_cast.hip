// Tensor Casting (Algorithm 2) on CDNA4.
//
//  1. k_build_keys   -- (src, dst) pairs from the bag-major CSR index:
//                       key = row, value = bag id. Block 0 also writes the
//                       tile records of the sort segments (below).
//  2. LSD radix sort by key, stable, at most kMaxRadixBits bits per pass over
//     the key bits that can be set. Each pass is
//       k_radix_hist    per-tile digit counts (LDS histograms, one per wave)
//       k_radix_scan    per-digit exclusive scan over tiles (one block/digit)
//       k_radix_scatter stable scatter: a wave finds the lanes holding equal
//                       digits with ballots, counts them into its running
//                       per-digit count in LDS, waves are combined in tile
//                       order, and the tile is laid out in sorted order in
//                       LDS and stored in that order.
//     A pass reads and writes 8 bytes per pair plus a 4-byte read for the
//     histogram. The last pass writes the values straight into casted_src.
//  3. Segment build (the scan and cumulative sum of Algorithm 2):
//       k_seg_count  heads (key differs from its predecessor) per tile
//       k_seg_write  casted_dst, unique_rows, seg_offsets, *num_unique (each
//                    block sums the head counts of the tiles before it)
//
// Sort segments. The pairs of table t are contiguous in the input
// (bag-major CSR, tables in order) and so are their rows in the output. When
// the caller bounds the table sizes, each table is sorted on its
// table-local row, which needs fewer key bits than the global row (32 tables
// of 2^20 rows: 20 bits, three passes, instead of 25 bits and four), and the
// last pass adds the table's row offset back. A segment is cut into tiles of
// kTile pairs (its last tile may be short), tiles of all segments are
// numbered in segment order, and a digit's position inside its segment comes
// from the per-digit scan over all tiles minus that scan at the segment's
// first tile. k_build_keys writes one record per tile (its pair range and its
// segment's), so a pass kernel finds its tile with a single load. Without a
// bound there is one segment, all pairs on global rows, and tiles are plain
// slices of kTile pairs.
//
// Within a tile, wave w owns positions [w*kWaveSpan, (w+1)*kWaveSpan) and
// walks them 64 at a time, lane l taking position base + 64*i + l, so tile
// order = (wave, iteration, lane) order and every pass is stable. No atomics
// on global memory; nothing here depends on scheduling order.
//
// tc_embed_forward_cast runs the forward gather-reduce in the cast's
// launches: k_forward_build (pairs and first-pass digit counts built per
// tile, then workgroups of the forward; the first pass needs no
// k_radix_hist) or, for a small batch, beside the one k_cast_small
// workgroup.
#include "tc_group_sum.h"

namespace tc {
namespace {

// Digits of at most 8 bits: with 2048-pair tiles, wider digits cost more
// per-tile digit bookkeeping (counts written, scanned and read back for every
// digit of every tile) than the pass they save, at these sizes.
constexpr int kMaxRadixBits = 8;
constexpr int kMaxRadix = 1 << kMaxRadixBits;
constexpr int kSortWaves = kBlock / kWave;        // 4
constexpr int kItems = 8;                         // positions per lane per tile
constexpr int kWaveSpan = kWave * kItems;         // 512
constexpr int kTile = kSortWaves * kWaveSpan;     // 2048
// Table-local sorting for at most this many tables (one thread per table
// lays the segments out).
constexpr int kMaxSegTables = kBlock;

__device__ __forceinline__ uint64_t lanemask_lt(int lane) { return (uint64_t(1) << lane) - 1; }

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

// One tile of a radix pass: pairs [p0, p1) of segment s, whose tiles are
// [first, next), whose pairs start at pstart, and whose keys get rowoff added
// by the last pass. Tiles past the last one have p0 = p1 = 0 and s = -1.
struct alignas(16) TileRec {
    int32_t p0, p1, first, next, pstart, rowoff, s, pad;
};
// ---------------------------------------------------------------------------
// 1. key build. The segments of the table-local sort, in LDS: segment s has
// tiles [tstart[s], tstart[s+1]) and pairs [pstart[s], pstart[s+1]), and
// rowoff[s] is its table's first row. seg_layout fills it (whole workgroup)
// and returns the number of tiles; tile_record reads tile b's record off it.
struct SegLayout {
    int32_t tstart[kMaxSegTables + 1], pstart[kMaxSegTables + 1], rowoff[kMaxSegTables];
};

__device__ int32_t seg_layout(SegLayout &L, const int32_t *__restrict__ bag_offsets,
                              const int64_t *__restrict__ table_row_offset, int64_t num_bags,
                              int32_t bags_per_table, int32_t num_tables) {
    const int t = threadIdx.x;
    int32_t p0 = 0, n_t = 0;
    if (t < num_tables) {
        p0 = bag_offsets[int64_t(t) * bags_per_table];
        n_t = bag_offsets[int64_t(t + 1) * bags_per_table] - p0;
        L.rowoff[t] = int32_t(table_row_offset[t]);
    }
    int32_t total;
    const int32_t ts = block_exclusive_scan((n_t + kTile - 1) / kTile, &total);
    if (t < num_tables) {
        L.tstart[t] = ts;
        L.pstart[t] = p0;
    }
    if (t == 0) {
        L.tstart[num_tables] = total;
        L.pstart[num_tables] = bag_offsets[num_bags];
    }
    __syncthreads();
    return total;
}

__device__ TileRec tile_record(const SegLayout &L, int32_t num_tables, int32_t total, int32_t b) {
    TileRec r{0, 0, 0, 0, 0, 0, -1, 0};
    if (b < total) {
        // the segment holding tile b: last s with tstart[s] <= b (segments
        // without pairs have no tiles and are passed over)
        int32_t lo = 0, hi = num_tables - 1;
        while (lo < hi) {
            const int32_t mid = (lo + hi + 1) / 2;
            if (L.tstart[mid] <= b) lo = mid; else hi = mid - 1;
        }
        const int32_t sg = lo;
        r.s = sg;
        r.first = L.tstart[sg];
        r.next = L.tstart[sg + 1];
        r.pstart = L.pstart[sg];
        r.rowoff = L.rowoff[sg];
        r.p0 = L.pstart[sg] + (b - r.first) * kTile;
        const int32_t end = L.pstart[sg + 1];
        r.p1 = r.p0 + kTile < end ? r.p0 + kTile : end;
    }
    return r;
}

// Bag offsets staged per tile by build_tile (a 2048-pair tile spans at most
// 2048 bags with pairs; more only with bags without pairs between them).
constexpr int kStageBags = 2048;

// One sort tile's (src, dst) pairs, with the tile's digit counts for the
// first radix pass (digits key & mask0, counts[digit * tiles + b], as
// k_radix_hist writes them): keys are table-local rows when `local`, else
// global rows; values are bag ids (dst), or pair positions when `positions`
// (an argsort). Pair j's bag comes from a search: the bag holding the tile's
// first pair by a 64-way search of the segment's bag offsets, then each
// pair's by binary search of the tile's bag offsets staged in LDS. Tile b
// has its record from the segment layout (local; workgroup 0 also writes
// every tile's record) or is pairs [b*kTile, (b+1)*kTile) of one segment.
__device__ void build_tile(int32_t b, const int32_t *__restrict__ indices,
                           const int32_t *__restrict__ bag_offsets,
                           const int64_t *__restrict__ table_row_offset, int64_t num_bags,
                           int32_t bags_per_table, int32_t num_tables, int32_t n, bool local,
                           bool positions, TileRec *__restrict__ recs, int32_t tiles,
                           int32_t *__restrict__ keys, int32_t *__restrict__ vals,
                           int32_t *__restrict__ counts, uint32_t mask0) {
    __shared__ SegLayout L;
    __shared__ int32_t sbo[kStageBags + 1];
    __shared__ int32_t hist[kSortWaves][kMaxRadix];
    __shared__ int32_t s_g0;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    TileRec tr{0, 0, 0, 0, 0, 0, -1, 0};
    int64_t glo = 0, ghi = num_bags;  // the bags of the tile's segment
    if (local) {
        const int32_t total = seg_layout(L, bag_offsets, table_row_offset, num_bags,
                                         bags_per_table, num_tables);
        if (b == 0)
            for (int32_t bb = tid; bb < tiles; bb += kBlock)
                recs[bb] = tile_record(L, num_tables, total, bb);
        tr = tile_record(L, num_tables, total, b);
        glo = int64_t(tr.s) * bags_per_table;
        ghi = glo + bags_per_table;
    } else if (int64_t(b) * kTile < n) {
        tr.s = 0;
        tr.p0 = b * kTile;
        tr.p1 = tr.p0 + kTile < n ? tr.p0 + kTile : n;
    }
    for (int i = tid; i < kSortWaves * kMaxRadix; i += kBlock) (&hist[0][0])[i] = 0;
    if (tr.s >= 0) {  // uniform
        const int32_t p0 = tr.p0, p1 = tr.p1;
        if (w == 0) {
            // the last bag g in [glo, ghi) with bag_offsets[g] <= p0, the
            // range narrowed 64-fold per step
            int64_t lo = glo, hi = ghi;
            while (hi - lo > 1) {
                const int64_t step = (hi - lo + kWave - 1) / kWave;
                const int64_t g = lo + lane * step;
                const bool le = g < hi && bag_offsets[g] <= p0;
                const uint64_t m = __ballot(le);
                const int l = m ? 63 - __builtin_clzll(m) : 0;
                lo = lo + l * step;
                hi = lo + step < hi ? lo + step : hi;
            }
            if (lane == 0) s_g0 = int32_t(lo);
        }
        __syncthreads();
        const int64_t g0 = s_g0;
        const int32_t nst = int32_t(ghi - g0 < kStageBags ? ghi - g0 : kStageBags);
        for (int32_t i = tid; i <= nst; i += kBlock) sbo[i] = bag_offsets[g0 + i];
        __syncthreads();
        // whether the staged offsets hold the bag of every pair of the tile
        const bool staged = g0 + nst == ghi || sbo[nst] >= p1;
#pragma unroll
        for (int i = 0; i < kItems; ++i) {
            const int32_t j = p0 + i * kBlock + tid;
            if (j < p1) {
                int64_t g;
                if (staged) {
                    int32_t lo = 0, hi = nst - 1;
                    while (lo < hi) {
                        const int32_t mid = (lo + hi + 1) / 2;
                        if (sbo[mid] <= j) lo = mid; else hi = mid - 1;
                    }
                    g = g0 + lo;
                } else {
                    int64_t lo = g0, hi = ghi - 1;
                    while (lo < hi) {
                        const int64_t mid = (lo + hi + 1) / 2;
                        if (bag_offsets[mid] <= j) lo = mid; else hi = mid - 1;
                    }
                    g = lo;
                }
                const int32_t idx = indices[j];
                const int32_t key =
                    local ? idx : int32_t(table_row_offset[g / bags_per_table] + idx);
                keys[j] = key;
                vals[j] = positions ? j : int32_t(g);
                atomicAdd(&hist[w][uint32_t(key) & mask0], 1);
            }
        }
    }
    __syncthreads();
    for (uint32_t d = tid; d <= mask0; d += kBlock) {
        int32_t c = 0;
#pragma unroll
        for (int ww = 0; ww < kSortWaves; ++ww) c += hist[ww][d];
        counts[int64_t(d) * tiles + b] = c;
    }
}

// The records of all num_tile_slots tile slots, written by one workgroup.
__device__ void write_tile_records(const int32_t *__restrict__ bag_offsets,
                                   const int64_t *__restrict__ table_row_offset,
                                   int64_t num_bags, int32_t bags_per_table, int32_t num_tables,
                                   TileRec *__restrict__ tiles, int32_t num_tile_slots) {
    __shared__ SegLayout L;
    const int32_t total = seg_layout(L, bag_offsets, table_row_offset, num_bags, bags_per_table,
                                     num_tables);
    for (int32_t b = threadIdx.x; b < num_tile_slots; b += kBlock)
        tiles[b] = tile_record(L, num_tables, total, b);
}

// (src, dst) pairs by a walk over the bags (tc_cast_index, tc_argsort_rows):
// one group of 16 lanes per bag writes that bag's pairs; keys and values as
// in build_tile. With `local`, block 0 also writes the tile records. The
// first pass then counts its digits with k_radix_hist: on its own, this walk
// and that count take less time than build_tile's searches.
__global__ __launch_bounds__(kBlock) void k_build_keys(
    const int32_t *__restrict__ indices, const int32_t *__restrict__ bag_offsets,
    const int64_t *__restrict__ table_row_offset, int64_t num_bags, int32_t bags_per_table,
    int32_t num_tables, bool local, bool positions, TileRec *__restrict__ tiles,
    int32_t num_tile_slots, int32_t *__restrict__ keys, int32_t *__restrict__ vals) {
    if (local && blockIdx.x == 0)
        write_tile_records(bag_offsets, table_row_offset, num_bags, bags_per_table, num_tables,
                           tiles, num_tile_slots);
    constexpr int kLanes = 16;
    const int64_t group = (int64_t(blockIdx.x) * blockDim.x + threadIdx.x) / kLanes;
    const int64_t ngroups = (int64_t(gridDim.x) * blockDim.x) / kLanes;
    const int sub = threadIdx.x & (kLanes - 1);
    for (int64_t g = group; g < num_bags; g += ngroups) {
        const int32_t beg = bag_offsets[g], end = bag_offsets[g + 1];
        const int64_t base = local ? 0 : table_row_offset[g / bags_per_table];
        for (int32_t j = beg + sub; j < end; j += kLanes) {
            keys[j] = int32_t(base + indices[j]);
            vals[j] = positions ? j : int32_t(g);
        }
    }
}

// The pair build and the first pass's digit counts (build_tile, one sort
// tile per workgroup) with the forward gather-reduce in one launch
// (tc_embed_forward_cast): the first `tiles` workgroups build the tiles,
// the others run the forward (FL lanes per bag, as k_forward). Both
// read the index array; the tile workgroups' searches and stores stay out of
// the forward's chains of dependent loads, and their latency hides behind
// the forward's.
template <int FL>
__global__ __launch_bounds__(kBlock) void k_forward_build(
    FwdSlice f, int32_t num_tables, int32_t n, bool local, TileRec *__restrict__ recs,
    int32_t tiles, int32_t *__restrict__ keys, int32_t *__restrict__ vals,
    int32_t *__restrict__ counts, uint32_t mask0) {
    if (int32_t(blockIdx.x) < tiles) {  // uniform
        build_tile(blockIdx.x, f.ids, f.offsets, f.table_row_offset, f.bag_hi, f.bags_per_table,
                   num_tables, n, local, false, recs, tiles, keys, vals, counts, mask0);
        return;
    }
    constexpr int64_t kWaves = kBlock / kWave;
    forward_bags<FL, 1>(f, (int64_t(blockIdx.x) - tiles) * kWaves + threadIdx.x / kWave,
                        (int64_t(gridDim.x) - tiles) * kWaves);
}

// This block's tile: its record (table-local sort) or a plain slice of the
// n pairs (global sort: one segment, tiles 0 .. ceil(n/kTile)-1).
__device__ __forceinline__ TileRec tile_of(const TileRec *__restrict__ tiles, int32_t n) {
    if (tiles) return tiles[blockIdx.x];
    const int32_t used = (n + kTile - 1) / kTile;
    const int32_t p0 = int32_t(blockIdx.x) * kTile;
    TileRec r{0, 0, 0, used, 0, 0, -1, 0};
    if (p0 < n) {
        r.s = 0;
        r.p0 = p0;
        r.p1 = p0 + kTile < n ? p0 + kTile : n;
    }
    return r;
}

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

// The same with the digit width known only at run time (uniform branches).
template <int MAXB = kMaxRadixBits>
__device__ __forceinline__ uint64_t match_digit_n(uint32_t d, bool ok, int bits) {
    uint64_t peers = __ballot(ok);
#pragma unroll
    for (int b = 0; b < MAXB; ++b) {
        if (b < bits) {
            const bool bit = (d >> b) & 1u;
            const uint64_t m = __ballot(bit);
            peers &= bit ? m : ~m;
        }
    }
    return peers;
}

// Whether every item of the wavefront where ok holds has the same digit (a
// run of one hot row, common in the later passes under skewed keys); *act
// gets those lanes. Two ballots, against one per digit bit for a match.
__device__ __forceinline__ bool all_same_digit(uint32_t d, bool ok, uint64_t *act) {
    const uint32_t d0 = __builtin_amdgcn_readfirstlane(d);
    *act = __ballot(ok);
    return __ballot(ok && d == d0) == *act;
}

// ---------------------------------------------------------------------------
// 2a. per-tile digit histogram -> counts[digit * tiles + tile]. Every item
// adds one to its wave's count of its digit (an LDS atomic; the order of
// the adds does not matter here), except that a wavefront whose items share
// one digit adds them all at once. Blocks past the last tile write zeros.
template <int BITS>
__global__ __launch_bounds__(kBlock) void k_radix_hist(const int32_t *__restrict__ keys,
                                                       int32_t n, int shift,
                                                       const TileRec *__restrict__ recs,
                                                       int32_t *__restrict__ counts,
                                                       int32_t tiles) {
    constexpr int R = 1 << BITS;
    __shared__ int32_t hist[kSortWaves][R];
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    constexpr uint32_t mask = R - 1u;
    const TileRec tr = tile_of(recs, n);
    const int32_t base = tr.p0 + w * kWaveSpan;
    int32_t key[kItems];
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
        const int32_t j = base + i * kWave + lane;
        key[i] = j < tr.p1 ? keys[j] : 0;
    }
    for (int i = tid; i < kSortWaves * R; i += kBlock) (&hist[0][0])[i] = 0;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
        const bool ok = base + i * kWave + lane < tr.p1;
        const uint32_t d = (uint32_t(key[i]) >> shift) & mask;
        uint64_t act;
        if (all_same_digit(d, ok, &act)) {
            if (lane == 0 && act) atomicAdd(&hist[w][d], __popcll(act));
        } else if (ok) {
            atomicAdd(&hist[w][d], 1);
        }
    }
    __syncthreads();
    for (int d = tid; d < R; d += kBlock) {
        int32_t s = 0;
#pragma unroll
        for (int ww = 0; ww < kSortWaves; ++ww) s += hist[ww][d];
        counts[int64_t(d) * tiles + blockIdx.x] = s;
    }
}

// 2b. counts[d][*] -> exclusive prefix over tiles (in place); totals[d].
__global__ __launch_bounds__(kBlock) void k_radix_scan(int32_t *__restrict__ counts,
                                                       int32_t tiles,
                                                       int32_t *__restrict__ totals) {
    constexpr int kPer = 4;
    int32_t *row = counts + int64_t(blockIdx.x) * tiles;
    int32_t carry = 0;
    for (int32_t base = 0; base < tiles; base += kBlock * kPer) {
        int32_t v[kPer], s = 0;
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const int32_t i = base + threadIdx.x * kPer + k;
            v[k] = i < tiles ? row[i] : 0;
            s += v[k];
        }
        int32_t tot;
        int32_t p = block_exclusive_scan(s, &tot) + carry;
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const int32_t i = base + threadIdx.x * kPer + k;
            if (i < tiles) row[i] = p;
            p += v[k];
        }
        carry += tot;
    }
    if (threadIdx.x == 0) totals[blockIdx.x] = carry;
}

// 2c. stable scatter of one tile. Within a wavefront the lanes holding equal
// digits are found with ballots (two if they all share one digit); the lowest of them adds their number to the
// wave's running count of that digit with one LDS atomic (the returned old
// value is the count of that digit in earlier items, since a wave's LDS
// operations complete in order) and the others take it from that lane. The
// tile is then laid out in sorted order in LDS and written back thread by
// thread in that order, so neighbouring threads write neighbouring addresses
// of the same digit run (coalesced stores instead of one scattered store per
// pair). With add_rowoff the keys leave with the segment's row offset added.
template <int BITS>
__global__ __launch_bounds__(kBlock) void k_radix_scatter(
    const int32_t *__restrict__ keys_in, const int32_t *__restrict__ vals_in,
    int32_t *__restrict__ keys_out, int32_t *__restrict__ vals_out, int32_t n, int shift,
    const TileRec *__restrict__ recs, const int32_t *__restrict__ counts,
    const int32_t *__restrict__ totals, int32_t tiles, bool add_rowoff) {
    constexpr int R = 1 << BITS;
    constexpr int DPT = R > kBlock ? R / kBlock : 1;  // digits per thread
    constexpr uint32_t mask = R - 1u;
    // wave w's running count of digit d, then the tile-local start of its run
    __shared__ int32_t wcount[kSortWaves][R];
    __shared__ int32_t run_shift[R];  // global position - tile-local position
    __shared__ int32_t stage_key[kTile];
    __shared__ int32_t stage_val[kTile];
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    const TileRec tr = tile_of(recs, n);
    if (tr.s < 0) return;  // uniform: past the last tile

    const int32_t base = tr.p0 + w * kWaveSpan;
    int32_t key[kItems], val[kItems], rank[kItems];
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
        const int32_t j = base + i * kWave + lane;
        const bool ok = j < tr.p1;
        key[i] = ok ? keys_in[j] : 0;
        val[i] = ok ? vals_in[j] : 0;
    }
    // Thread tid handles digits tid*DPT .. tid*DPT+DPT-1 (digit order): where
    // this tile's run of each digit starts in the output.
    const int32_t first = tr.first, next = tr.next;
    int32_t tile_off[DPT], seg_tot[DPT], my = 0;
#pragma unroll
    for (int k = 0; k < DPT; ++k) {
        const int32_t d = tid * DPT + k;
        tile_off[k] = seg_tot[k] = 0;
        if (d < R) {
            const int64_t row = int64_t(d) * tiles;
            const int32_t at_first = counts[row + first];
            tile_off[k] = counts[row + blockIdx.x] - at_first;
            seg_tot[k] = (next < tiles ? counts[row + next] : totals[d]) - at_first;
        }
        my += seg_tot[k];
    }
    for (int i = tid; i < kSortWaves * R; i += kBlock) (&wcount[0][0])[i] = 0;
    int32_t digit_base[DPT];
    {
        int32_t tot;
        int32_t p = block_exclusive_scan(my, &tot) + tr.pstart;
#pragma unroll
        for (int k = 0; k < DPT; ++k) {
            digit_base[k] = p + tile_off[k];
            p += seg_tot[k];
        }
    }
    __syncthreads();

    // all atomics first, then the broadcasts, so no item waits for the LDS
    // round trip of the one before it
    int32_t lower_n[kItems], leader[kItems], old[kItems];
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
        const bool ok = base + i * kWave + lane < tr.p1;
        const uint32_t d = (uint32_t(key[i]) >> shift) & mask;
        uint64_t act;
        const uint64_t peers = all_same_digit(d, ok, &act) ? act : match_digit<BITS>(d, ok);
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
        // per digit: tile-local start of each wave's run (digit order, then
        // wave order) and the shift from tile-local to global positions
        int32_t c[DPT][kSortWaves], my_n = 0;
#pragma unroll
        for (int k = 0; k < DPT; ++k) {
            const int32_t d = tid * DPT + k;
#pragma unroll
            for (int ww = 0; ww < kSortWaves; ++ww) {
                c[k][ww] = d < R ? wcount[ww][d] : 0;
                my_n += c[k][ww];
            }
        }
        int32_t tot;
        int32_t start = block_exclusive_scan(my_n, &tot);
#pragma unroll
        for (int k = 0; k < DPT; ++k) {
            const int32_t d = tid * DPT + k;
            if (d < R) {
                run_shift[d] = digit_base[k] - start;
                int32_t r = start;
#pragma unroll
                for (int ww = 0; ww < kSortWaves; ++ww) {
                    wcount[ww][d] = r;
                    r += c[k][ww];
                }
                start = r;
            }
        }
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
        if (base + i * kWave + lane < tr.p1) {
            const uint32_t d = (uint32_t(key[i]) >> shift) & mask;
            const int32_t lp = wcount[w][d] + rank[i];
            stage_key[lp] = key[i];
            stage_val[lp] = val[i];
        }
    }
    __syncthreads();
    const int32_t in_tile = tr.p1 - tr.p0;
    const int32_t koff = add_rowoff ? tr.rowoff : 0;
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
        const int32_t lp = i * kBlock + tid;
        if (lp < in_tile) {
            const int32_t k = stage_key[lp];
            const uint32_t d = (uint32_t(k) >> shift) & mask;
            const int32_t pos = run_shift[d] + lp;
            keys_out[pos] = k + koff;
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

// 3b. casted_dst (inclusive head count - 1), unique_rows and seg_offsets.
// Each block adds up the head counts of the tiles before it (a few loads per
// thread even for thousands of tiles, so no separate scan kernel); the last
// block writes *num_unique.
__global__ __launch_bounds__(kBlock) void k_seg_write(
    const int32_t *__restrict__ keys, int64_t n, const int32_t *__restrict__ tile_heads,
    int32_t *__restrict__ unique_rows, int32_t *__restrict__ seg_offsets,
    int32_t *__restrict__ casted_dst, int32_t *__restrict__ num_unique) {
    __shared__ int32_t wsum[kSortWaves];
    __shared__ int32_t before;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
    const int64_t base = int64_t(blockIdx.x) * kTile + int64_t(w) * kWaveSpan;
    {
        int32_t part = 0;
        for (int32_t t = tid; t < int32_t(blockIdx.x); t += kBlock) part += tile_heads[t];
        int32_t tot;
        block_exclusive_scan(part, &tot);
        if (tid == 0) before = tot;
    }
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
    int32_t run = before;
    for (int ww = 0; ww < w; ++ww) run += wsum[ww];
    if (blockIdx.x == gridDim.x - 1 && tid == 0) {
        int32_t total = before;
        for (int ww = 0; ww < kSortWaves; ++ww) total += wsum[ww];
        *num_unique = total;
    }
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

// ---------------------------------------------------------------------------
// Small batches (at most kSmallPairs pairs): the whole cast in one workgroup
// of kSmallThreads threads, keys and values in LDS. Same stable LSD passes
// (the pairs are spread evenly over the wavefronts in whole trips of 64:
// wave w owns positions [w*span, (w+1)*span), walked 64 at a time; equal
// digits ranked with ballots and one LDS atomic per digit group)
// and the same segment build, without the kernel chain: for a few thousand
// pairs the multi-kernel cast is all launch and memory latency.
constexpr int kSmallThreads = 1024;
constexpr int kSmallWaves = kSmallThreads / kWave;  // 16
constexpr int kSmallItems = 8;
constexpr int kSmallSpan = kWave * kSmallItems;     // 512
constexpr int kSmallPairs = kSmallWaves * kSmallSpan;  // 8192
// Digits of up to 9 bits in the one-workgroup cast: its per-wave digit
// counts stay in LDS (16 x 512), and 17- or 18-bit keys take two passes
// instead of three.
constexpr int kSmallRadixBits = 9;
constexpr int kSmallRadix = 1 << kSmallRadixBits;
static_assert(kSmallRadix <= kSmallThreads, "one digit per thread in the digit scan");
static_assert(kSmallPairs == kSmallItems * kSmallThreads, "k_cast_small stages one item per trip");

// Block-wide exclusive scan over the kSmallThreads threads.
__device__ __forceinline__ int32_t small_block_scan(int32_t v, int32_t *total) {
    __shared__ int32_t wsum[kSmallWaves];
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
    for (int ww = 0; ww < kSmallWaves; ++ww) {
        const int32_t s = wsum[ww];
        if (ww < w) wbase += s;
        tot += s;
    }
    __syncthreads();
    *total = tot;
    return wbase + incl - v;
}

//
// With FL > 0 (tc_embed_forward_cast) the workgroups after the first run the
// forward gather-reduce beside it, FL lanes per bag: a small cast keeps one
// CU busy and leaves the others to the forward.
template <int FL>
__global__ __launch_bounds__(kSmallThreads) void k_cast_small(
    const int32_t *__restrict__ indices, const int32_t *__restrict__ bag_offsets,
    const int64_t *__restrict__ table_row_offset, int32_t num_tables, int32_t num_bags,
    int32_t bags_per_table, int32_t n, int bits, bool positions, int32_t *__restrict__ unique_rows,
    int32_t *__restrict__ seg_offsets, int32_t *__restrict__ casted_src,
    int32_t *__restrict__ casted_dst, int32_t *__restrict__ num_unique, FwdSlice fs) {
    // keys ping-pong between two buffers; values have one: every item of a
    // pass is in registers before the pass writes any (barriers between)
    __shared__ int32_t keys[2][kSmallPairs];
    __shared__ int32_t vals[kSmallPairs];
    __shared__ int32_t wcount[kSmallWaves][kSmallRadix];
    if constexpr (FL > 0) {
        if (blockIdx.x > 0) {  // uniform: a forward workgroup
            constexpr int64_t kWaves = kSmallThreads / kWave;
            forward_bags<FL, 1>(fs, (int64_t(blockIdx.x) - 1) * kWaves + threadIdx.x / kWave,
                                (int64_t(gridDim.x) - 1) * kWaves);
            return;
        }
    }
    const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;

    // (src, dst) pairs from the bag-major CSR index: 16 lanes per bag. The
    // index, the bag offsets and the table offsets are first staged in LDS
    // (in the value buffer, the second key buffer and the digit counters)
    // with independent loads, so the walk over bags waits for memory once.
    // The index shares the value buffer: position j's index is read and its
    // value then written by the same thread, and no other.
    {
        constexpr int kLanes = 16;
        const int sub = tid & (kLanes - 1);
        const bool staged = num_bags < kSmallPairs && num_tables <= kSmallWaves * kSmallRadix;
        int32_t *s_idx = vals, *s_bo = keys[1], *s_off = &wcount[0][0];
        if (staged) {
            // every load issued before the first LDS store (n and num_bags
            // + 1 are at most kSmallPairs = kSmallItems * kSmallThreads), so
            // the staging waits for memory once, not once per trip
            int32_t vi[kSmallItems], vb[kSmallItems];
#pragma unroll
            for (int i = 0; i < kSmallItems; ++i) {
                const int32_t j = tid + i * kSmallThreads;
                vi[i] = j < n ? indices[j] : 0;
                vb[i] = j <= num_bags ? bag_offsets[j] : 0;
            }
            for (int32_t t = tid; t < num_tables; t += kSmallThreads)
                s_off[t] = int32_t(table_row_offset[t]);
#pragma unroll
            for (int i = 0; i < kSmallItems; ++i) {
                const int32_t j = tid + i * kSmallThreads;
                if (j < n) s_idx[j] = vi[i];
                if (j <= num_bags) s_bo[j] = vb[i];
            }
            __syncthreads();
        }
        for (int32_t g = tid / kLanes; g < num_bags; g += kSmallThreads / kLanes) {
            const int32_t beg = staged ? s_bo[g] : bag_offsets[g];
            const int32_t end = staged ? s_bo[g + 1] : bag_offsets[g + 1];
            const int32_t t = g / bags_per_table;
            const int32_t base = staged ? s_off[t] : int32_t(table_row_offset[t]);
            for (int32_t j = beg + sub; j < end; j += kLanes) {
                keys[0][j] = base + (staged ? s_idx[j] : indices[j]);
                vals[j] = positions ? j : g;
            }
        }
    }
    __syncthreads();

    const int passes = (bits + kSmallRadixBits - 1) / kSmallRadixBits;
    const int per_pass = (bits + passes - 1) / passes;
    // trips of 64 positions per wavefront (at most kSmallItems), so that
    // every wavefront holds a share of the pairs
    const int trips = (n + kSmallThreads - 1) / kSmallThreads;
    const int32_t base = w * trips * kWave;
    int cur = 0;
    for (int p = 0; p < passes; ++p) {
        const int shift = p * per_pass;
        const int pbits = shift + per_pass <= bits ? per_pass : bits - shift;
        const uint32_t mask = (1u << pbits) - 1u;
        for (int i = tid; i < kSmallWaves * kSmallRadix; i += kSmallThreads)
            (&wcount[0][0])[i] = 0;
        __syncthreads();
        int32_t key[kSmallItems], val[kSmallItems], lower_n[kSmallItems], leader[kSmallItems],
            old[kSmallItems];
#pragma unroll
        for (int i = 0; i < kSmallItems; ++i) {
            old[i] = lower_n[i] = 0;
            leader[i] = lane;
            key[i] = val[i] = 0;
            if (i >= trips) continue;  // uniform
            const int32_t j = base + i * kWave + lane;
            const bool ok = j < n;
            key[i] = ok ? keys[cur][j] : 0;
            val[i] = ok ? vals[j] : 0;
            const uint32_t d = (uint32_t(key[i]) >> shift) & mask;
            uint64_t act;
            const uint64_t peers =
                all_same_digit(d, ok, &act) ? act : match_digit_n<kSmallRadixBits>(d, ok, pbits);
            const uint64_t lower = peers & lanemask_lt(lane);
            lower_n[i] = __popcll(lower);
            leader[i] = peers ? __builtin_ctzll(peers) : lane;
            old[i] = 0;
            if (ok && lower == 0) old[i] = atomicAdd(&wcount[w][d], __popcll(peers));
        }
        int32_t rank[kSmallItems];
#pragma unroll
        for (int i = 0; i < kSmallItems; ++i)
            rank[i] = i < trips ? __shfl(old[i], leader[i], kWave) + lower_n[i] : 0;
        __syncthreads();
        {
            // digit d = tid (threads past the radix hold zeros): start of each
            // wave's run, in digit order then wave order
            int32_t c[kSmallWaves], my = 0;
#pragma unroll
            for (int ww = 0; ww < kSmallWaves; ++ww) {
                c[ww] = tid < kSmallRadix ? wcount[ww][tid] : 0;
                my += c[ww];
            }
            int32_t tot;
            int32_t r = small_block_scan(my, &tot);
            if (tid < kSmallRadix) {
#pragma unroll
                for (int ww = 0; ww < kSmallWaves; ++ww) {
                    wcount[ww][tid] = r;
                    r += c[ww];
                }
            }
        }
        __syncthreads();
#pragma unroll
        for (int i = 0; i < kSmallItems; ++i) {
            if (i < trips && base + i * kWave + lane < n) {
                const uint32_t d = (uint32_t(key[i]) >> shift) & mask;
                const int32_t lp = wcount[w][d] + rank[i];
                keys[cur ^ 1][lp] = key[i];
                vals[lp] = val[i];
            }
        }
        __syncthreads();
        cur ^= 1;
    }

    // segment build: thread tid owns sorted positions tid*trips .. tid*trips +
    // trips - 1
    int32_t head[kSmallItems], c = 0;
#pragma unroll
    for (int i = 0; i < kSmallItems; ++i) {
        const int32_t j = tid * trips + i;
        head[i] = i < trips && j < n && (j == 0 || keys[cur][j] != keys[cur][j - 1]);
        c += head[i];
    }
    int32_t total;
    int32_t run = small_block_scan(c, &total);
#pragma unroll
    for (int i = 0; i < kSmallItems; ++i) {
        const int32_t j = tid * trips + i;
        if (i < trips && j < n) {
            run += head[i];
            casted_src[j] = vals[j];
            if (casted_dst) casted_dst[j] = run - 1;
            if (head[i]) {
                unique_rows[run - 1] = keys[cur][j];
                seg_offsets[run - 1] = j;
            }
        }
    }
    if (tid == 0) {
        seg_offsets[total] = n;
        *num_unique = total;
    }
}

// No pairs: zero segments, seg_offsets[0] = 0.
__global__ void k_cast_empty(int32_t *seg_offsets, int32_t *num_unique) {
    if (threadIdx.x == 0) {
        seg_offsets[0] = 0;
        *num_unique = 0;
    }
}

// One LSD pass over `bits` (1..kMaxRadixBits) digit bits starting at `shift`.
// One radix pass; hist_done: the digit counts are already in `counts` (the
// first pass, counted by the pair build).
tc_status launch_radix_pass(int bits, const int32_t *kin, const int32_t *vin, int32_t *kout,
                            int32_t *vout, int32_t n, int shift, const TileRec *recs,
                            int32_t *counts, int32_t *totals, int32_t tiles, bool last,
                            bool hist_done, hipStream_t stream) {
#define TC_PASS_CASE(B)                                                                      \
    case B:                                                                                  \
        if (!hist_done) {                                                                    \
            k_radix_hist<B><<<tiles, kBlock, 0, stream>>>(kin, n, shift, recs, counts, tiles); \
            if (check_launch("k_radix_hist") != TC_OK) return TC_ERR_HIP;                    \
        }                                                                                    \
        k_radix_scan<<<1 << B, kBlock, 0, stream>>>(counts, tiles, totals);                  \
        if (check_launch("k_radix_scan") != TC_OK) return TC_ERR_HIP;                        \
        k_radix_scatter<B><<<tiles, kBlock, 0, stream>>>(kin, vin, kout, vout, n, shift,     \
                                                         recs, counts, totals, tiles, last); \
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
static_assert(kMaxRadixBits == 8, "launch_radix_pass instantiates 1..8 bits");

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Sort segments available to a call with num_tables tables.
inline int32_t seg_capacity(int32_t num_tables) {
    return num_tables >= 1 && num_tables <= kMaxSegTables ? num_tables : 1;
}

struct CastPlan {
    int64_t sort_tiles;  // tile slots of a radix pass (all segments)
    int64_t seg_tiles;   // tiles of the segment build (plain tiles of kTile)
    size_t off_ka, off_va, off_kb, off_vb, off_counts, off_totals, off_heads, off_recs, bytes;
};

inline CastPlan cast_plan(int64_t n, int32_t num_tables) {
    CastPlan p{};
    const int32_t nseg = seg_capacity(num_tables);
    p.seg_tiles = (n + kTile - 1) / kTile;
    p.sort_tiles = p.seg_tiles + nseg;  // each segment adds at most one short tile
    const size_t arr = align_up(size_t(n) * 4);
    size_t o = 0;
    p.off_ka = o; o += arr;
    p.off_va = o; o += arr;
    p.off_kb = o; o += arr;
    p.off_vb = o; o += arr;
    p.off_counts = o; o += align_up(size_t(kMaxRadix) * size_t(p.sort_tiles) * 4);
    p.off_totals = o; o += align_up(size_t(kMaxRadix) * 4);
    p.off_heads = o; o += align_up(size_t(p.seg_tiles) * 4);
    p.off_recs = o; o += align_up(size_t(p.sort_tiles) * sizeof(TileRec));
    p.bytes = o;
    return p;
}

// bits needed for keys in [0, rows)
inline int key_bits(int64_t rows) {
    int b = 0;
    while (b < 31 && (int64_t(1) << b) < rows) ++b;
    return b < 1 ? 1 : b;  // at least one pass, so the values are always moved
}

}  // namespace
}  // namespace tc

using namespace tc;

extern "C" size_t tc_cast_workspace_bytes(int64_t num_pairs, int64_t total_rows,
                                          int32_t num_tables) {
    (void)total_rows;
    if (num_pairs < 0) return 0;
    return cast_plan(num_pairs, num_tables).bytes;
}

namespace {
// The forward over all bags of fwd as its own kernel.
tc_status forward_alone(const FwdSlice &fwd, hipStream_t stream) {
    return launch_forward(fwd.W, fwd.dim, fwd.ids, fwd.offsets, fwd.table_row_offset,
                          fwd.bags_per_table, fwd.bag_hi, fwd.out, stream);
}

// The sort and segment build behind tc_cast_index (values = bag ids) and
// tc_argsort_rows (values = pair positions). `what` names the entry point in
// error messages. With fwd (tc_embed_forward_cast; values = bag ids), the
// forward gather-reduce of all fwd->bag_hi bags runs too: beside the
// single-workgroup cast, or as the key-building kernel of the radix sort,
// or, for row shapes without such kernels, as its own kernel first.
tc_status cast_impl(const char *what, bool positions, const int64_t *table_row_offset,
                    int32_t num_tables, int32_t bags_per_table, int64_t total_rows,
                    int64_t max_table_rows, const int32_t *indices, const int32_t *bag_offsets,
                    int64_t num_pairs, int32_t *unique_rows, int32_t *seg_offsets,
                    int32_t *casted_src, int32_t *casted_dst, int32_t *num_unique,
                    void *workspace, size_t workspace_bytes, hipStream_t stream,
                    const FwdSlice *fwd = nullptr) {
    TC_REQUIRE(num_tables >= 0 && bags_per_table >= 0 && total_rows >= 0 && num_pairs >= 0 &&
                   max_table_rows >= 0,
               TC_ERR_INVALID_ARG, "%s: negative size", what);
    TC_REQUIRE(total_rows < (int64_t(1) << 31) && num_pairs < (int64_t(1) << 31),
               TC_ERR_INVALID_ARG, "%s: total_rows and num_pairs must be below 2^31", what);
    const int64_t num_bags = int64_t(num_tables) * bags_per_table;
    TC_REQUIRE(num_bags < (int64_t(1) << 31), TC_ERR_INVALID_ARG,
               "%s: more than 2^31-1 bags", what);
    TC_REQUIRE(seg_offsets && num_unique, TC_ERR_INVALID_ARG, "%s: null pointer", what);
    if (num_pairs == 0) {
        if (fwd) {
            const tc_status st = forward_alone(*fwd, stream);
            if (st != TC_OK) return st;
        }
        k_cast_empty<<<1, kWave, 0, stream>>>(seg_offsets, num_unique);
        return check_launch("k_cast_empty");
    }
    TC_REQUIRE(num_bags > 0 && total_rows > 0, TC_ERR_INVALID_ARG,
               "%s: pairs without bags or rows", what);
    TC_REQUIRE(table_row_offset && indices && bag_offsets && unique_rows && casted_src,
               TC_ERR_INVALID_ARG, "%s: null pointer", what);
    const CastPlan plan = cast_plan(num_pairs, num_tables);
    TC_REQUIRE(workspace && workspace_bytes >= plan.bytes, TC_ERR_WORKSPACE,
               "%s: workspace of %zu bytes, %zu needed", what, workspace_bytes, plan.bytes);
    TC_REQUIRE((reinterpret_cast<uintptr_t>(workspace) & (kAlign - 1)) == 0, TC_ERR_WORKSPACE,
               "%s: workspace must be 256-byte aligned", what);
    TC_REQUIRE(plan.sort_tiles < (int64_t(1) << 31) / kMaxRadix, TC_ERR_INVALID_ARG,
               "%s: too many pairs", what);

    const int fl = fwd ? ride_along_lanes(fwd->dim) : 0;
    if (fwd && fl == 0) {
        const tc_status st = forward_alone(*fwd, stream);
        if (st != TC_OK) return st;
    }
    if (num_pairs <= kSmallPairs) {
        // one workgroup in LDS (the workspace is not touched); the forward's
        // workgroups, if any, run beside it (one per CU at most: each holds
        // the kernel's LDS), one bag per lane group
        unsigned fb = 0;
        if (fl) {
            const int64_t per_block = int64_t(kSmallThreads / kWave) * (kWave / fl);
            fb = grid_for(num_bags, per_block, device_cus() > 1 ? device_cus() - 1 : 1);
        }
        const FwdSlice fs = fl ? *fwd : FwdSlice{};
#define TC_SMALL(FL)                                                                         \
    k_cast_small<FL><<<1 + fb, kSmallThreads, 0, stream>>>(                                  \
        indices, bag_offsets, table_row_offset, num_tables, int32_t(num_bags), bags_per_table, \
        int32_t(num_pairs), key_bits(total_rows), positions, unique_rows, seg_offsets,        \
        casted_src, casted_dst, num_unique, fs)
        if (fl == 16) TC_SMALL(16);
        else if (fl == 32) TC_SMALL(32);
        else if (fl == 64) TC_SMALL(64);
        else TC_SMALL(0);
#undef TC_SMALL
        return check_launch("k_cast_small");
    }
    // Table-local keys when the tables are known to be small enough to save
    // key bits; otherwise one segment of global rows.
    const int global_bits = key_bits(total_rows);
    const bool local = max_table_rows > 0 && num_tables <= kMaxSegTables &&
                       key_bits(max_table_rows) < global_bits;
    const int bits = local ? key_bits(max_table_rows) : global_bits;

    char *ws = static_cast<char *>(workspace);
    int32_t *ka = reinterpret_cast<int32_t *>(ws + plan.off_ka);
    int32_t *va = reinterpret_cast<int32_t *>(ws + plan.off_va);
    int32_t *kb = reinterpret_cast<int32_t *>(ws + plan.off_kb);
    int32_t *vb = reinterpret_cast<int32_t *>(ws + plan.off_vb);
    int32_t *counts = reinterpret_cast<int32_t *>(ws + plan.off_counts);
    int32_t *totals = reinterpret_cast<int32_t *>(ws + plan.off_totals);
    int32_t *heads = reinterpret_cast<int32_t *>(ws + plan.off_heads);
    TileRec *recs = local ? reinterpret_cast<TileRec *>(ws + plan.off_recs) : nullptr;
    const int32_t sort_tiles = int32_t(plan.sort_tiles);
    const int32_t seg_tiles = int32_t(plan.seg_tiles);

    const int passes = (bits + kMaxRadixBits - 1) / kMaxRadixBits;
    const int per_pass = (bits + passes - 1) / passes;
    const uint32_t mask0 = (1u << per_pass) - 1u;  // the first pass's digits
    if (fl) {
        // the tiles' pair builds, then the forward's workgroups, in one launch
        const int64_t per_block = int64_t(kBlock / kWave) * (kWave / fl);
        const unsigned grid =
            unsigned(sort_tiles) + grid_for(num_bags, per_block, int64_t(device_cus()) * 32);
#define TC_FWD_BUILD(FL)                                                                     \
    k_forward_build<FL><<<grid, kBlock, 0, stream>>>(*fwd, num_tables, int32_t(num_pairs),    \
                                                     local, recs, sort_tiles, ka, va, counts,  \
                                                     mask0)
        if (fl == 16) TC_FWD_BUILD(16);
        else if (fl == 32) TC_FWD_BUILD(32);
        else TC_FWD_BUILD(64);
#undef TC_FWD_BUILD
        tc_status st = check_launch("k_forward_build");
        if (st != TC_OK) return st;
    } else {
        const unsigned grid = grid_for(num_bags, kBlock / 16, int64_t(device_cus()) * 8);
        k_build_keys<<<grid, kBlock, 0, stream>>>(indices, bag_offsets, table_row_offset,
                                                  num_bags, bags_per_table, num_tables, local,
                                                  positions, recs, sort_tiles, ka, va);
        tc_status st = check_launch("k_build_keys");
        if (st != TC_OK) return st;
    }
    int32_t *kin = ka, *vin = va, *kout = kb, *vout = vb;
    for (int p = 0; p < passes; ++p) {
        const int shift = p * per_pass;
        const int pb = (shift + per_pass <= bits) ? per_pass : bits - shift;
        const bool last = p == passes - 1;
        int32_t *vdst = last ? casted_src : vout;
        tc_status st = launch_radix_pass(pb, kin, vin, kout, vdst, int32_t(num_pairs), shift,
                                         recs, counts, totals, sort_tiles, last,
                                         p == 0 && fl != 0, stream);
        if (st != TC_OK) return st;
        // next pass reads what this one wrote
        int32_t *tk = kin, *tv = vin;
        kin = kout;
        vin = vout;
        kout = tk;
        vout = tv;
    }
    const int32_t *sorted_keys = kin;

    k_seg_count<<<seg_tiles, kBlock, 0, stream>>>(sorted_keys, num_pairs, heads);
    tc_status st = check_launch("k_seg_count");
    if (st != TC_OK) return st;
    k_seg_write<<<seg_tiles, kBlock, 0, stream>>>(sorted_keys, num_pairs, heads, unique_rows,
                                                  seg_offsets, casted_dst, num_unique);
    return check_launch("k_seg_write");
}
}  // namespace

extern "C" tc_status tc_cast_index(const int64_t *table_row_offset, int32_t num_tables,
                                   int32_t bags_per_table, int64_t total_rows,
                                   int64_t max_table_rows, const int32_t *indices,
                                   const int32_t *bag_offsets, int64_t num_pairs,
                                   int32_t *unique_rows, int32_t *seg_offsets,
                                   int32_t *casted_src, int32_t *casted_dst, int32_t *num_unique,
                                   void *workspace, size_t workspace_bytes, hipStream_t stream) {
    clear_error();
    return cast_impl("tc_cast_index", false, table_row_offset, num_tables, bags_per_table,
                     total_rows, max_table_rows, indices, bag_offsets, num_pairs, unique_rows,
                     seg_offsets, casted_src, casted_dst, num_unique, workspace,
                     workspace_bytes, stream);
}

extern "C" tc_status tc_embed_forward_cast(
    const float *W, int64_t total_rows, int32_t dim, const int64_t *table_row_offset,
    int32_t num_tables, int32_t bags_per_table, int64_t max_table_rows, const int32_t *indices,
    const int32_t *bag_offsets, int64_t num_pairs, float *out, int32_t *unique_rows,
    int32_t *seg_offsets, int32_t *casted_src, int32_t *casted_dst, int32_t *num_unique,
    void *workspace, size_t workspace_bytes, hipStream_t stream) {
    clear_error();
    const char *what = "tc_embed_forward_cast";
    TC_REQUIRE(num_tables >= 0 && bags_per_table >= 0, TC_ERR_INVALID_ARG, "%s: negative size",
               what);
    TC_REQUIRE(dim > 0 && dim % 4 == 0 && dim <= kMaxDim, TC_ERR_UNSUPPORTED,
               "%s: dim %d must be a multiple of 4 in [4, %d]", what, dim, kMaxDim);
    const int64_t num_bags = int64_t(num_tables) * bags_per_table;
    if (num_bags > 0) {
        TC_REQUIRE(W && out && table_row_offset && bag_offsets, TC_ERR_INVALID_ARG,
                   "%s: null pointer", what);
        TC_REQUIRE(aligned16(W) && aligned16(out), TC_ERR_UNSUPPORTED,
                   "%s: W and out must be 16-byte aligned", what);
    }
    // the cast checks the rest before anything is launched
    const FwdSlice f{W, indices, bag_offsets, table_row_offset, out, 0, num_bags, dim,
                     bags_per_table};
    return cast_impl(what, false, table_row_offset, num_tables, bags_per_table, total_rows,
                     max_table_rows, indices, bag_offsets, num_pairs, unique_rows, seg_offsets,
                     casted_src, casted_dst, num_unique, workspace, workspace_bytes, stream,
                     num_bags > 0 ? &f : nullptr);
}

extern "C" tc_status tc_argsort_rows(const int64_t *table_row_offset, int32_t num_tables,
                                     int32_t bags_per_table, int64_t total_rows,
                                     int64_t max_table_rows, const int32_t *indices,
                                     const int32_t *bag_offsets, int64_t num_pairs,
                                     int32_t *unique_rows, int32_t *seg_offsets,
                                     int32_t *sorted_pos, int32_t *num_unique, void *workspace,
                                     size_t workspace_bytes, hipStream_t stream) {
    clear_error();
    return cast_impl("tc_argsort_rows", true, table_row_offset, num_tables, bags_per_table,
                     total_rows, max_table_rows, indices, bag_offsets, num_pairs, unique_rows,
                     seg_offsets, sorted_pos, nullptr, num_unique, workspace, workspace_bytes,
                     stream);
}
