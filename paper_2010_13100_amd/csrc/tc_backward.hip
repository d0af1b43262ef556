// Backward: the casted gradient gather-reduce (Algorithm 3) on CDNA4.
//
// coal_grad[u] is the sum of grad_out rows casted_src[j] over the segment j
// in [seg_offsets[u], seg_offsets[u+1]). Segment lengths follow the index
// skew: under Zipf lookups a few table rows own tens of thousands of pairs.
// Segments under kLongSegment pairs are short; the others are long.
//
//  k_backward_short  short segments: lane groups exactly as the forward.
//  k_backward_long   long segments (no workspace): workgroups scan ranges of
//                    segments for long ones.
//  k_backward_list   long segments (workspace): persistent workgroups take
//                    work items -- (long segment, part) or (piece of a split
//                    segment, part) -- from lists the short kernel builds.
//
// A long segment (or piece) is summed by one workgroup per 64-column part:
// four producer wavefronts gather the rows into a ring of LDS buffers with
// 16-byte loads, and one consumer wavefront (one column per lane) runs the
// ordered adds out of LDS, so the chain never waits behind load issue.
//
// Summation order. Without a workspace every segment is one ordered chain
// from +0, the sequential definition bit for bit. With a workspace that
// covers them, segments of kSplitPairs pairs or more are cut into n =
// min(kMaxPieces, len / kPieceMin) pieces of consecutive pairs; each piece is
// an ordered chain from +0 run by its own work item, which stores the piece
// sum, and the item that finishes a segment's last piece (an agent-scope
// counter per segment and part) adds the n piece sums in piece order from
// +0. The order is fixed by the segment's length alone, so results do not
// depend on scheduling and repeat bit for bit; the chain of the hottest row
// shrinks from len to len / n.
//
// Fused with the update (tc_embed_backward_update), the owner of coalesced
// row u applies the optimizer step to table row unique_rows[u] straight from
// its registers (tc_optim.h, the arithmetic of tc_sparse_update), so the
// coalesced rows need not go through HBM; unique rows are distinct, so every
// table row still has a single writer.
#include <type_traits>

#include "tc_group_sum.h"
#include "tc_optim.h"

namespace tc {
namespace {

// Segments at least this long are long.
constexpr int kLongSegment = 80;
// A long-segment workgroup: one consumer and kProducers producer wavefronts.
constexpr int kProducers = 4;
constexpr int kLongThreads = (1 + kProducers) * kWave;
// Columns per workgroup (one per consumer lane) and rows per LDS buffer.
constexpr int kPartCols = kWave;
constexpr int kChunkRows = 64;
constexpr int kBuffers = 3;
// A producer load instruction brings kRowsPerLoad rows of the part: 16
// lanes x 16 bytes per row.
constexpr int kLanesPerRow = kPartCols / 4;
constexpr int kRowsPerLoad = kWave / kLanesPerRow;  // 4
constexpr int kLoadsPerChunk = kChunkRows / kRowsPerLoad;  // 16
// Chunks whose row loads (kAhead) and id loads (kIdAhead) a producer keeps in
// flight; the producer code is unrolled over kPeriod chunks so that every ring
// slot is a fixed register.
constexpr int kAhead = 3;
constexpr int kIdAhead = 6;
constexpr int kPeriod = 6;
static_assert(kPeriod % kAhead == 0 && kPeriod % kIdAhead == 0 && kPeriod % kBuffers == 0,
              "ring periods must divide kPeriod");
// Ranges of segments scanned by the blocks of the long kernel (per part).
constexpr int kLongRanges = 1024;
// Summing in pieces (with a workspace): segments of at least kSplitPairs
// pairs, pieces of at least kPieceMin pairs, at most kMaxPieces of them.
constexpr int32_t kSplitPairs = TC_BACKWARD_SPLIT_PAIRS;
constexpr int32_t kPieceMin = 1024;
constexpr int32_t kMaxPieces = 32;
static_assert(kSplitPairs >= 2 * kPieceMin && kPieceMin >= kLongSegment, "piece sizes");
// Long segments of at least kBigLong pairs are handed out before the shorter
// ones, so that the work left at the end is small (the workgroups finish
// together).
constexpr int32_t kBigLong = 512;

// The backward workspace. The lists are filled by k_backward_short and
// drained by k_backward_list; k_backward_init zeroes the counters first.
// A long segment [beg, beg + len) is covered when beg + len <= cap_pairs and
// split when also len >= kSplitPairs. Split segments are disjoint intervals
// of at least kSplitPairs pairs, and pieces of at least kPieceMin pairs, so
// beg / kSplitPairs and (first pair of the piece) / kPieceMin name them
// without collisions.
//   ctr[0]           entries in pieces[]
//   ctr[1], ctr[2]   long segments of at least / under kBigLong pairs, kept
//                    from the front / from the back of longs[]
//   ctr[3]           next work item
//   pieces[k]        {u, beg, len, q}: piece q of split segment u
//   longs[k]         {u, beg, len, 0}: a covered long segment, not split
//   seg_done[(beg / kSplitPairs) * parts + p]  pieces of part p finished
//   partial[(first pair / kPieceMin) * dim + c]  piece sums
struct SplitWs {
    int32_t *ctr;
    int4 *pieces;
    int4 *longs;
    int32_t *seg_done;
    float *partial;
    int64_t cap_pairs;  // 0: no workspace
    int32_t max_pieces, max_longs;
    int32_t parts;
};

__device__ __forceinline__ int32_t num_pieces(int32_t len) {
    return len / kPieceMin < kMaxPieces ? len / kPieceMin : kMaxPieces;
}
__device__ __forceinline__ int32_t piece_begin(int32_t beg, int32_t len, int32_t n, int32_t q) {
    return beg + int32_t(int64_t(q) * len / n);
}

// Buffer resource word 3 for gfx9-family buffers; out-of-range reads give 0.
constexpr int32_t kBufferWord3 = 0x00020000;
// A buffer offset past every resource here (resources span at most this):
// rows past the end of a segment load as +0.0, which leaves the sum unchanged
// (a sum started at +0.0 is never -0.0, and x + 0.0 == x for every other x).
constexpr int32_t kOutOfRange = 0x7ffff000;

// What becomes of a coalesced row: stored to coal (if not null) and/or
// applied to W[rows[u]] (if W is not null) with optimizer `kind`.
struct RowSink {
    float *coal;
    float *W;
    float *A;  // Adagrad / RMSprop accumulator
    const int32_t *rows;
    int32_t kind;  // TC_OPT_SGD, TC_OPT_ADAGRAD or TC_OPT_RMSPROP
    float lr, eps, gamma, omg;  // omg = 1 - gamma
};

// The table (and accumulator) value one lane's sink_value updates: column
// `col` of table row rows[u]. A consumer loads it before running the
// segment's chain, so that its two dependent loads overlap the chain.
struct SinkVal {
    int64_t at;
    float w, a;
};

__device__ __forceinline__ SinkVal sink_value_load(const RowSink &k, int64_t u, int32_t dim,
                                                   int32_t col) {
    SinkVal v{0, 0.f, 0.f};
    if (k.W && col < dim) {
        v.at = int64_t(k.rows[u]) * dim + col;
        v.w = stream_load(k.W + v.at);
        if (k.kind != TC_OPT_SGD) v.a = stream_load(k.A + v.at);
    }
    return v;
}

// One lane's column `col` of coalesced row u, with its table value in v.
__device__ __forceinline__ void sink_value(const RowSink &k, int64_t u, int32_t dim, int32_t col,
                                           float g, const SinkVal &v) {
    if (k.coal) k.coal[u * dim + col] = g;
    if (k.W) {
        float w = v.w;
        if (k.kind == TC_OPT_SGD) {
            w = sgd_step(w, g, k.lr);
        } else {
            float a = v.a;
            if (k.kind == TC_OPT_ADAGRAD)
                adagrad_step(w, a, g, k.lr, k.eps);
            else
                rmsprop_step(w, a, g, k.lr, k.eps, k.gamma, k.omg);
            stream_store(k.A + v.at, a);
        }
        stream_store(k.W + v.at, w);
    }
}

// A lane group's float4 chunks of coalesced row u, whose table row is r
// (rows[u], loaded by the caller together with the segment's offsets).
template <int LANES, int CHUNKS>
__device__ __forceinline__ void sink_group(const RowSink &k, int64_t u, int64_t r, int32_t dim,
                                           int sub, const float4 (&acc)[CHUNKS]) {
    if (k.coal) group_store<LANES, CHUNKS>(k.coal + u * dim, dim, sub, acc);
    if (k.W) {
        const int d4 = dim >> 2;
        float *wrow = k.W + r * dim;
#pragma unroll
        for (int c = 0; c < CHUNKS; ++c) {
            const int col4 = sub + c * LANES;
            if (col4 >= d4) continue;
            const float4 g = acc[c];
            float4 w = stream_load4(wrow + 4 * col4);
            if (k.kind == TC_OPT_SGD) {
                w.x = sgd_step(w.x, g.x, k.lr);
                w.y = sgd_step(w.y, g.y, k.lr);
                w.z = sgd_step(w.z, g.z, k.lr);
                w.w = sgd_step(w.w, g.w, k.lr);
            } else {
                float *arow = k.A + r * dim;
                float4 a = stream_load4(arow + 4 * col4);
                if (k.kind == TC_OPT_ADAGRAD) {
                    adagrad_step(w.x, a.x, g.x, k.lr, k.eps);
                    adagrad_step(w.y, a.y, g.y, k.lr, k.eps);
                    adagrad_step(w.z, a.z, g.z, k.lr, k.eps);
                    adagrad_step(w.w, a.w, g.w, k.lr, k.eps);
                } else {
                    rmsprop_step(w.x, a.x, g.x, k.lr, k.eps, k.gamma, k.omg);
                    rmsprop_step(w.y, a.y, g.y, k.lr, k.eps, k.gamma, k.omg);
                    rmsprop_step(w.z, a.z, g.z, k.lr, k.eps, k.gamma, k.omg);
                    rmsprop_step(w.w, a.w, g.w, k.lr, k.eps, k.gamma, k.omg);
                }
                stream_store4(arow + 4 * col4, a);
            }
            stream_store4(wrow + 4 * col4, w);
        }
    }
}

// LDS buffer layout: column-major, so that one 16-byte read gives a consumer
// lane four consecutive rows of its column. Within column c, the group of
// rows 4k..4k+3 sits at group position k ^ swz(c); the swizzle spreads both
// the consumer's 16-byte reads (16 neighbouring columns, same k) and the
// producers' 4-byte writes (16 columns 4 apart, same k) over distinct banks.
struct LongLds {
    alignas(16) float cols[kBuffers][kPartCols][kChunkRows];
    int32_t offs[kProducers][kChunkRows];
};
__device__ __forceinline__ int32_t swz(int32_t c) { return (c & 15) ^ ((c >> 4) & 3); }
// byte offset of (row r, column c) within one buffer
__device__ __forceinline__ int32_t lds_pos(int32_t r, int32_t c) {
    return (c * kChunkRows + 4 * ((r >> 2) ^ swz(c)) + (r & 3)) * 4;
}
constexpr int32_t kBufferBytes = kPartCols * kChunkRows * 4;

// Workgroup barrier that orders LDS only: outstanding global loads stay in
// flight across it.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

template <int K>
using Int = std::integral_constant<int, K>;

// Producer P of a long segment (rows ids[0..len) of grad, part columns at
// byte offset part_bytes). It gathers chunk c (rows 64c..64c+63) with the
// load instructions k = P, P + kProducers, ... of the chunk; instruction k brings rows
// 4k..4k+3, lane l reading 16 bytes of row 4k + l/16. Chunk c's loads are
// issued kAhead chunks before it is written to LDS buffer c % 3, two chunks
// ahead of the consumer; the chunk's ids are loaded kIdAhead chunks before
// that and turned into row offsets through a small per-producer LDS table.
// Executes exactly 1 + nchunks barriers, as the consumer does.
template <int P>
__device__ void long_producer(LongLds &lds, __amdgpu_buffer_rsrc_t id_rsrc, int32_t len,
                              int32_t first, int32_t row_bytes, int32_t part_bytes,
                              int32_t nchunks, __amdgpu_buffer_rsrc_t rsrc) {
    constexpr int L = (kLoadsPerChunk - P + kProducers - 1) / kProducers;
    const int lane = threadIdx.x & (kWave - 1);
    const int rsel = lane / kLanesPerRow;
    const int32_t col4 = (lane % kLanesPerRow) * 4;  // first of the lane's 4 columns
    const int32_t lane_bytes = part_bytes + col4 * 4;
    int32_t *offs = lds.offs[P];
    // ids of chunk c, one per lane. The whole byte offset goes in the
    // vector offset, which the buffer's range check covers (the scalar
    // offset is not checked): ids past the end of the segment read as 0
    // without touching memory, and such rows get kOutOfRange below.
    auto load_ids = [&](int32_t c) -> int32_t {
        return __builtin_amdgcn_raw_buffer_load_b32(id_rsrc, c * (kChunkRows * 4) + lane * 4, 0,
                                                    0);
    };
    int32_t iv[kIdAhead];
    float4 d[kAhead][L];
    auto issue = [&](auto ds, auto es, int32_t c) {
        constexpr int DS = decltype(ds)::value, ES = decltype(es)::value;
        offs[lane] = c * kChunkRows + lane < len ? (iv[ES] - first) * row_bytes : kOutOfRange;
        int32_t o[L];
#pragma unroll
        for (int t = 0; t < L; ++t) o[t] = offs[(P + kProducers * t) * kRowsPerLoad + rsel];
#pragma unroll
        for (int t = 0; t < L; ++t)
            d[DS][t] = __builtin_bit_cast(
                float4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, o[t] + lane_bytes, 0, 0));
        iv[ES] = load_ids(c + kIdAhead);
    };
    // byte offsets of this lane's four columns of row 4k + rsel, k = P + 3t
    int32_t wpos[L][4];
#pragma unroll
    for (int t = 0; t < L; ++t)
#pragma unroll
        for (int e = 0; e < 4; ++e)
            wpos[t][e] = lds_pos((P + kProducers * t) * kRowsPerLoad + rsel, col4 + e);
    char *lds_cols = reinterpret_cast<char *>(&lds.cols[0][0][0]);
    auto write = [&](auto ds, auto bs) {
        constexpr int DS = decltype(ds)::value, B = decltype(bs)::value;
#pragma unroll
        for (int t = 0; t < L; ++t) {
            const float4 v = d[DS][t];
            *reinterpret_cast<float *>(lds_cols + B * kBufferBytes + wpos[t][0]) = v.x;
            *reinterpret_cast<float *>(lds_cols + B * kBufferBytes + wpos[t][1]) = v.y;
            *reinterpret_cast<float *>(lds_cols + B * kBufferBytes + wpos[t][2]) = v.z;
            *reinterpret_cast<float *>(lds_cols + B * kBufferBytes + wpos[t][3]) = v.w;
        }
    };
#pragma unroll
    for (int e = 0; e < kIdAhead; ++e) iv[e] = load_ids(e);
    static_assert(kAhead == 3, "the prologue issues kAhead chunks");
    static_assert(kIdAhead > 4, "the prologue uses the ids of chunks 0..4");
    issue(Int<0>{}, Int<0>{}, 0);
    issue(Int<1>{}, Int<1>{}, 1);
    issue(Int<2>{}, Int<2>{}, 2);
    write(Int<0>{}, Int<0>{});
    issue(Int<0>{}, Int<3>{}, 3);
    write(Int<1>{}, Int<1>{});
    issue(Int<1>{}, Int<4>{}, 4);
    lds_barrier();
    // Step i: write chunk i + 2, refill its registers with chunk i + 2 + kAhead.
    auto step = [&](auto ms, int32_t i) {
        constexpr int M = decltype(ms)::value;  // i % kPeriod
        write(Int<(M + 2) % kAhead>{}, Int<(M + 2) % kBuffers>{});
        issue(Int<(M + 2) % kAhead>{}, Int<(M + 2 + kAhead) % kIdAhead>{}, i + 2 + kAhead);
        lds_barrier();
    };
    // Whole periods in a loop with a single exit (a loop left from the middle
    // merges the load bookkeeping of every exit at its head, which costs a
    // full wait), then the remaining steps once.
    static_assert(kPeriod == 6, "the step loop is unrolled over 6 chunks");
    int32_t i = 0;
    const int32_t periods = nchunks / kPeriod;
    for (int32_t k = 0; k < periods; ++k, i += kPeriod) {
        step(Int<0>{}, i);
        step(Int<1>{}, i + 1);
        step(Int<2>{}, i + 2);
        step(Int<3>{}, i + 3);
        step(Int<4>{}, i + 4);
        step(Int<5>{}, i + 5);
    }
    const int32_t rem = nchunks - i;
    if (rem > 0) { step(Int<0>{}, i);
    if (rem > 1) { step(Int<1>{}, i + 1);
    if (rem > 2) { step(Int<2>{}, i + 2);
    if (rem > 3) { step(Int<3>{}, i + 3);
    if (rem > 4) { step(Int<4>{}, i + 4);
    }}}}}
}

// The consumer: lane l owns column l of the part and adds the rows of chunk
// i in order, 64 per step, four rows per 16-byte LDS read. Reads run kAheadG
// groups (4 rows each) ahead of the adds through a small register ring; chunk
// i + 1 is complete in LDS during step i (it was written one step ahead), so
// the read-ahead crosses into it freely and the chain never waits for LDS.
// Executes exactly 1 + nchunks barriers, as the producers do.
constexpr int kAheadG = 8;
__device__ float long_consumer(LongLds &lds, int32_t nchunks) {
    constexpr int G = kChunkRows / 4;
    static_assert(G % kAheadG == 0, "ring slots repeat every step");
    const int lane = threadIdx.x & (kWave - 1);
    const char *lds_cols = reinterpret_cast<const char *>(&lds.cols[0][0][0]);
    int32_t rpos[G];  // byte offset of rows 4k..4k+3 of this lane's column
#pragma unroll
    for (int k = 0; k < G; ++k) rpos[k] = lds_pos(4 * k, lane);
    auto read = [&](int b, int k) -> float4 {
        return *reinterpret_cast<const float4 *>(lds_cols + b * kBufferBytes + rpos[k]);
    };
    float acc = 0.f;
    lds_barrier();
    float4 ring[kAheadG];
#pragma unroll
    for (int k = 0; k < kAheadG; ++k) ring[k] = read(0, k);
    // step i: chunk i sits in buffer B = i % 3, chunk i + 1 in (B + 1) % 3
    auto step = [&](auto bs) {
        constexpr int B = decltype(bs)::value, BN = (B + 1) % kBuffers;
#pragma unroll
        for (int k = 0; k < G; ++k) {
            const float4 x = ring[k % kAheadG];
            ring[k % kAheadG] = k + kAheadG < G ? read(B, k + kAheadG) : read(BN, k + kAheadG - G);
            acc = acc + x.x;
            acc = acc + x.y;
            acc = acc + x.z;
            acc = acc + x.w;
            __builtin_amdgcn_sched_barrier(0);
        }
        lds_barrier();
    };
    int32_t i = 0;
    for (;;) {
        if (i >= nchunks) break;
        step(Int<0>{});
        if (++i >= nchunks) break;
        step(Int<1>{});
        if (++i >= nchunks) break;
        step(Int<2>{});
        ++i;
    }
    return acc;
}

// The ordered chain over ids[beg, beg + len) for this block's part, run by
// all five wavefronts (each executes the same number of barriers). Returns
// the sum of column `col` in the consumer wavefront (w == 0), 0 elsewhere.
// grad_bytes: the size of the whole grad array when it is at most
// kOutOfRange (its rows are then addressed from its start), else 0 (the
// chain's rows are addressed from its first row).
__device__ __forceinline__ float run_chain(LongLds &lds, const float *__restrict__ grad,
                                           int32_t dim, const int32_t *__restrict__ ids,
                                           int32_t beg, int32_t len, int w, int32_t part,
                                           int32_t col, int32_t grad_bytes) {
    const int32_t row_bytes = dim * 4;
    const int32_t *sid = ids + beg;
    int32_t first = 0;
    uint64_t span = uint64_t(grad_bytes);
    if (grad_bytes == 0) {  // uniform
        // ids within a segment are non-decreasing (stable cast order)
        first = __builtin_amdgcn_readfirstlane(sid[0]);
        const int32_t last = __builtin_amdgcn_readfirstlane(sid[len - 1]);
        span = uint64_t(last - first + 1) * uint64_t(row_bytes);
    }
    if (span > uint64_t(kOutOfRange) || len >= (1 << 28)) {
        // rows spread over about 2 GiB or more, so that kOutOfRange would not
        // be past them (or a segment so long that the byte offsets of its ids
        // and of the id chunks read ahead would not stay below 2^31): the
        // consumer alone, with 64-bit addressed loads (no barriers on this
        // path)
        float acc = 0.f;
        if (w == 0) {
            const float *colp = grad + (col < dim ? col : dim - 1);
            for (int32_t k = 0; k < len; ++k) acc = acc + colp[int64_t(sid[k]) * dim];
        }
        return acc;
    }
    const int32_t nchunks = (len + kChunkRows - 1) / kChunkRows;
    const auto id_rsrc =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<int32_t *>(sid), 0, len * 4, kBufferWord3);
    const auto rsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float *>(grad + int64_t(first) * dim), 0, int32_t(span), kBufferWord3);
    const int32_t part_bytes = part * kPartCols * 4;
    if (w == 0) return long_consumer(lds, nchunks);
    if (w == 1)
        long_producer<0>(lds, id_rsrc, len, first, row_bytes, part_bytes, nchunks, rsrc);
    else if (w == 2)
        long_producer<1>(lds, id_rsrc, len, first, row_bytes, part_bytes, nchunks, rsrc);
    else if (w == 3)
        long_producer<2>(lds, id_rsrc, len, first, row_bytes, part_bytes, nchunks, rsrc);
    else
        long_producer<3>(lds, id_rsrc, len, first, row_bytes, part_bytes, nchunks, rsrc);
    return 0.f;
}

// Consumer wavefront, after piece q of split segment u: store the piece sum,
// count the piece, and if it was the segment's last (for this part), add the
// n piece sums in piece order from +0 and hand the row to the sink.
__device__ void finish_piece(const SplitWs &ws, const RowSink &sink, int32_t dim, int32_t part,
                             int32_t col, int32_t u, int32_t beg, int32_t len, int32_t n,
                             int32_t q, float acc) {
    const int lane = threadIdx.x & (kWave - 1);
    if (col < dim)
        ws.partial[int64_t(piece_begin(beg, len, n, q) / kPieceMin) * dim + col] = acc;
    // the piece sum reaches device scope before the count does
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    int32_t done = 0;
    if (lane == 0)
        done = __hip_atomic_fetch_add(&ws.seg_done[int64_t(beg / kSplitPairs) * ws.parts + part],
                                      1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    done = __builtin_amdgcn_readlane(done, 0);
    if (done != n - 1) return;
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    if (col >= dim) return;
    float tot = 0.f;
    for (int32_t k = 0; k < n; ++k)
        tot = tot + ws.partial[int64_t(piece_begin(beg, len, n, k) / kPieceMin) * dim + col];
    sink_value(sink, u, dim, col, tot, sink_value_load(sink, u, dim, col));
}

// Long segments without a workspace. Each block (range x, part y) scans a
// contiguous range of segments and runs every long one it finds. All five
// wavefronts scan the same offsets, so they agree on every segment and on its
// number of chunks, which fixes the barrier count. A first pass reads every
// 64th offset: a batch of 64 segments spanning fewer than kLongSegment pairs
// cannot hold a long one.
__global__ __launch_bounds__(kLongThreads) void k_backward_long(
    const float *__restrict__ grad, int32_t dim, const int32_t *__restrict__ ids,
    const int32_t *__restrict__ offsets, const int32_t *__restrict__ num_out_dev,
    int64_t num_out_cap, RowSink sink, int32_t grad_bytes) {
    __shared__ LongLds lds;
    const int lane = threadIdx.x & (kWave - 1);
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int32_t part = blockIdx.y;
    const int32_t col = part * kPartCols + lane;
    const int64_t u_dev = *num_out_dev;
    const int64_t num = u_dev < num_out_cap ? u_dev : num_out_cap;
    if (w == 0) __builtin_amdgcn_s_setprio(3);
    const int32_t ranges = int32_t(gridDim.x);
    const int32_t range = int32_t(blockIdx.x);
    const int64_t per = (num + ranges - 1) / ranges;
    const int64_t r0 = int64_t(range) * per;
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
                const int32_t beg = __builtin_amdgcn_readlane(o0, j);
                const int32_t len = __builtin_amdgcn_readlane(o1, j) - beg;
                const int64_t seg = c0 + int64_t(kWave) * i + j;
                SinkVal sv{0, 0.f, 0.f};
                if (w == 0) sv = sink_value_load(sink, seg, dim, col);
                const float acc =
                    run_chain(lds, grad, dim, ids, beg, len, w, part, col, grad_bytes);
                if (w == 0 && col < dim) sink_value(sink, seg, dim, col, acc, sv);
            }
        }
    }
}

// Long segments with a workspace: persistent blocks take work items
// (index / parts = list entry: pieces, then long segments of at least
// kBigLong pairs, then the shorter ones; index % parts = part) from an
// agent-scope counter until the lists are drained. The next item and its
// list entry are fetched while the current one runs.
__global__ __launch_bounds__(kLongThreads, 3) void k_backward_list(
    const float *__restrict__ grad, int32_t dim, const int32_t *__restrict__ ids, RowSink sink,
    SplitWs ws, int32_t grad_bytes) {
    __shared__ LongLds lds;
    // the next item and its list entry, in two slots used in turn
    __shared__ int32_t next_item[2];
    __shared__ int4 next_entry[2];
    const int lane = threadIdx.x & (kWave - 1);
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int32_t np = min(ws.ctr[0], ws.max_pieces);
    const int32_t nb = min(ws.ctr[1], ws.max_longs);
    const int32_t ns = min(ws.ctr[2], ws.max_longs - nb);
    const int64_t total = int64_t(np + nb + ns) * ws.parts;
    if (total == 0) return;  // uniform: nothing listed (no segment is long)
    // thread 0: take the next item and load its list entry into slot s
    auto take = [&](int s) {
        const int32_t i = __hip_atomic_fetch_add(&ws.ctr[3], 1, __ATOMIC_RELAXED,
                                                 __HIP_MEMORY_SCOPE_AGENT);
        next_item[s] = i;
        if (i < total) {
            const int32_t k = i / ws.parts;
            next_entry[s] = k < np        ? ws.pieces[k]
                            : k < np + nb ? ws.longs[k - np]
                                          : ws.longs[ws.max_longs - 1 - (k - np - nb)];
        }
    };
    if (threadIdx.x == 0) take(0);
    lds_barrier();
    int slot = 0;
    int32_t item = next_item[0];
    if (w == 0) __builtin_amdgcn_s_setprio(3);
    while (item < total) {
        const int4 e = next_entry[slot];
        // the item after this one, visible after this item's last barrier
        if (threadIdx.x == 0) take(slot ^ 1);
        const int32_t k = item / ws.parts, part = item % ws.parts;
        const int32_t col = part * kPartCols + lane;
        const int32_t u = __builtin_amdgcn_readfirstlane(e.x);
        const int32_t beg = __builtin_amdgcn_readfirstlane(e.y);
        const int32_t len = __builtin_amdgcn_readfirstlane(e.z);
        if (k < np) {
            const int32_t q = __builtin_amdgcn_readfirstlane(e.w);
            const int32_t n = num_pieces(len);
            const int32_t p0 = piece_begin(beg, len, n, q);
            const int32_t p1 = piece_begin(beg, len, n, q + 1);
            const float acc =
                run_chain(lds, grad, dim, ids, p0, p1 - p0, w, part, col, grad_bytes);
            if (w == 0) finish_piece(ws, sink, dim, part, col, u, beg, len, n, q, acc);
        } else {
            SinkVal sv{0, 0.f, 0.f};
            if (w == 0) sv = sink_value_load(sink, u, dim, col);
            const float acc = run_chain(lds, grad, dim, ids, beg, len, w, part, col, grad_bytes);
            if (w == 0 && col < dim) sink_value(sink, u, dim, col, acc, sv);
        }
        lds_barrier();  // every wavefront is past this item
        slot ^= 1;
        item = next_item[slot];
    }
}

__global__ void k_backward_init(SplitWs ws) {
    if (threadIdx.x < 4) ws.ctr[threadIdx.x] = 0;
}

// Short segments: one lane group per segment, as the forward; long ones are
// left to k_backward_long.
template <int LANES, int CHUNKS>
__global__ __launch_bounds__(kBlock) void k_backward_short(
    const float *__restrict__ grad, int32_t dim, const int32_t *__restrict__ ids,
    const int32_t *__restrict__ offsets, const int32_t *__restrict__ num_out_dev,
    int64_t num_out_cap, RowSink sink, SplitWs ws) {
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
        bool listed = false;  // a covered long segment, not split
        int32_t len = 0;
        int64_t r = 0;  // the table row the sink updates
        if (o < num) {
            beg = offsets[o];
            end = offsets[o + 1];
            if (sink.W) r = sink.rows[o];
            len = end - beg;
            const bool covered = len >= kLongSegment && int64_t(beg) + len <= ws.cap_pairs;
            // without a workspace long segments go to k_backward_long; with
            // one, covered ones go to the lists and uncovered ones stay here
            mine = ws.cap_pairs == 0 ? len < kLongSegment : !covered;
            if (covered && len >= kSplitPairs) {
                if (sub == 0) {
                    const int32_t n = num_pieces(len);
                    const int32_t at = __hip_atomic_fetch_add(
                        &ws.ctr[0], n, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    for (int32_t q = 0; q < n && at + q < ws.max_pieces; ++q)
                        ws.pieces[at + q] = make_int4(int32_t(o), beg, len, q);
                    const int64_t slot = beg / kSplitPairs;
                    for (int32_t p = 0; p < ws.parts; ++p) ws.seg_done[slot * ws.parts + p] = 0;
                }
            } else {
                listed = covered && sub == 0;
            }
            if (!mine) end = beg;
        }
        // one counter update per wavefront and list: big ones from the
        // front of longs[], the others from the back
#pragma unroll
        for (int big = 1; big >= 0; --big) {
            const bool mine_list = listed && (len >= kBigLong) == bool(big);
            const uint64_t lm = __ballot(mine_list);
            if (lm == 0) continue;
            const int leader = __builtin_ctzll(lm);
            int32_t at = 0;
            if (lane == leader)
                at = __hip_atomic_fetch_add(&ws.ctr[big ? 1 : 2], __builtin_popcountll(lm),
                                            __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            at = __builtin_amdgcn_readlane(at, leader) +
                 __builtin_popcountll(lm & ((uint64_t(1) << lane) - 1));
            if (mine_list && at < ws.max_longs)
                ws.longs[big ? at : ws.max_longs - 1 - at] = make_int4(int32_t(o), beg, len, 0);
        }
        float4 acc[CHUNKS];
#pragma unroll
        for (int c = 0; c < CHUNKS; ++c) acc[c] = make_float4(0.f, 0.f, 0.f, 0.f);
        group_range_sum<LANES, CHUNKS>(grad, dim, ids, 0, beg, end, sub, acc);
        if (mine) sink_group<LANES, CHUNKS>(sink, o, r, dim, sub, acc);
    }
}

// Gradient expand (the paper's baseline backward, Sec. II-B): every pair j of
// bag g gets a copy of grad_out[g]. One lane group per bag holds the row in
// registers and writes it once per pair of the bag.
template <int LANES, int CHUNKS>
__global__ __launch_bounds__(kBlock) void k_expand(const float *__restrict__ grad, int32_t dim,
                                                  const int32_t *__restrict__ bag_offsets,
                                                  int64_t num_bags, float *__restrict__ expanded) {
    constexpr int kGroups = kWave / LANES;
    const int lane = threadIdx.x & (kWave - 1);
    const int sub = lane & (LANES - 1);
    const int grp = lane / LANES;
    const int d4 = dim >> 2;
    const int64_t wave = (int64_t(blockIdx.x) * blockDim.x + threadIdx.x) / kWave;
    const int64_t nwave = (int64_t(gridDim.x) * blockDim.x) / kWave;
    for (int64_t g0 = wave * kGroups; g0 < num_bags; g0 += nwave * kGroups) {
        const int64_t g = g0 + grp;
        if (g >= num_bags) continue;
        const int32_t beg = bag_offsets[g], end = bag_offsets[g + 1];
        float4 v[CHUNKS];
        const float *row = grad + g * int64_t(dim);
#pragma unroll
        for (int c = 0; c < CHUNKS; ++c) {
            const int col4 = sub + c * LANES;
            v[c] = col4 < d4 ? *reinterpret_cast<const float4 *>(row + 4 * col4)
                             : make_float4(0.f, 0.f, 0.f, 0.f);
        }
        for (int32_t j = beg; j < end; ++j)
            group_store<LANES, CHUNKS>(expanded + int64_t(j) * dim, dim, sub, v);
    }
}

tc_status launch_expand(const float *grad, int32_t dim, const int32_t *bag_offsets,
                        int64_t num_bags, float *expanded, hipStream_t stream) {
    const RowShape s = row_shape(dim);
    const int64_t rows_per_block = (kBlock / kWave) * (kWave / s.lanes);
    const unsigned grid = grid_for(num_bags, rows_per_block, int64_t(device_cus()) * 8);
#define TC_EXP_CASE(L, C)                                                                    \
    if (s.lanes == L && s.chunks == C) {                                                     \
        k_expand<L, C><<<grid, kBlock, 0, stream>>>(grad, dim, bag_offsets, num_bags,        \
                                                    expanded);                               \
        return check_launch("k_expand");                                                     \
    }
    TC_EXP_CASE(1, 1)
    TC_EXP_CASE(2, 1)
    TC_EXP_CASE(4, 1)
    TC_EXP_CASE(8, 1)
    TC_EXP_CASE(16, 1)
    TC_EXP_CASE(32, 1)
    TC_EXP_CASE(64, 1)
    TC_EXP_CASE(64, 2)
    TC_EXP_CASE(64, 3)
    TC_EXP_CASE(64, 4)
#undef TC_EXP_CASE
    set_error("no expand kernel for dim %d", dim);
    return TC_ERR_UNSUPPORTED;
}

// The backward workspace's layout for a cover of cap pairs.
struct WsLayout {
    size_t ctr, pieces, longs, seg_done, partial, total;
    int32_t max_pieces, max_longs;
};
WsLayout ws_layout(int64_t cap, int32_t dim) {
    auto al = [](int64_t x) { return size_t((x + 255) & ~int64_t(255)); };
    const int64_t parts = (dim + kPartCols - 1) / kPartCols;
    WsLayout l;
    l.max_pieces = int32_t(cap / kPieceMin + 1);
    l.max_longs = int32_t(cap / kLongSegment + 1);
    l.ctr = 0;
    l.pieces = l.ctr + al(4 * 4);
    l.longs = l.pieces + al(int64_t(l.max_pieces) * 16);
    l.seg_done = l.longs + al(int64_t(l.max_longs) * 16);
    l.partial = l.seg_done + al((cap / kSplitPairs + 1) * parts * 4);
    l.total = l.partial + al(int64_t(l.max_pieces) * dim * 4);
    return l;
}

// The workspace in `bytes` at `ws`: it covers the largest cap (below 2^31)
// whose layout fits; cap 0 (no workspace) if ws is null or not even
// kLongSegment pairs fit.
SplitWs make_split_ws(void *ws, size_t bytes, int32_t dim) {
    SplitWs s{nullptr, nullptr, nullptr, nullptr, nullptr, 0, 0, 0,
              (dim + kPartCols - 1) / kPartCols};
    if (ws == nullptr || ws_layout(kLongSegment, dim).total > bytes) return s;
    int64_t lo = kLongSegment, hi = (int64_t(1) << 31) - 1;
    while (lo < hi) {  // largest cap whose layout fits
        const int64_t mid = lo + (hi - lo + 1) / 2;
        if (ws_layout(mid, dim).total <= bytes) lo = mid; else hi = mid - 1;
    }
    const WsLayout l = ws_layout(lo, dim);
    char *p = static_cast<char *>(ws);
    s.ctr = reinterpret_cast<int32_t *>(p + l.ctr);
    s.pieces = reinterpret_cast<int4 *>(p + l.pieces);
    s.longs = reinterpret_cast<int4 *>(p + l.longs);
    s.seg_done = reinterpret_cast<int32_t *>(p + l.seg_done);
    s.partial = reinterpret_cast<float *>(p + l.partial);
    s.cap_pairs = lo;
    s.max_pieces = l.max_pieces;
    s.max_longs = l.max_longs;
    return s;
}

// Workgroups of k_backward_list: as many as can be resident at once on the
// current device (occupancy query, cached per device).
int list_blocks() {
    constexpr int kMaxDevices = 64;
    static int cached[kMaxDevices] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return device_cus();
    if (dev < kMaxDevices) {
        const int c = __atomic_load_n(&cached[dev], __ATOMIC_RELAXED);
        if (c > 0) return c;
    }
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_backward_list, kLongThreads,
                                                     0) != hipSuccess ||
        per_cu < 1)
        return device_cus();
    const int blocks = per_cu * device_cus();
    if (dev < kMaxDevices) __atomic_store_n(&cached[dev], blocks, __ATOMIC_RELAXED);
    return blocks;
}

tc_status launch_backward(const float *grad, int64_t grad_rows, int32_t dim,
                          const int32_t *ids, const int32_t *offsets,
                          const int32_t *num_out_dev, int64_t cap, const RowSink &out,
                          const SplitWs &ws, hipStream_t stream) {
    // the long chains address rows from the start of grad when it fits in a
    // 32-bit buffer window with kOutOfRange past its end
    const int64_t gb = grad_rows * int64_t(dim) * 4;
    const int32_t grad_bytes = gb <= kOutOfRange ? int32_t(gb) : 0;
    if (ws.cap_pairs > 0) {
        k_backward_init<<<1, kWave, 0, stream>>>(ws);
        const tc_status st = check_launch("k_backward_init");
        if (st != TC_OK) return st;
    }
    // the short kernel first: it builds the lists
    const RowShape s = row_shape(dim);
    const int64_t rows_per_block = (kBlock / kWave) * (kWave / s.lanes);
    const unsigned grid = grid_for(cap, rows_per_block, int64_t(device_cus()) * 8);
    bool launched = false;
#define TC_BWD_CASE(L, C)                                                                    \
    if (!launched && s.lanes == L && s.chunks == C) {                                        \
        k_backward_short<L, C><<<grid, kBlock, 0, stream>>>(grad, dim, ids, offsets,          \
                                                            num_out_dev, cap, out, ws);      \
        launched = true;                                                                     \
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
    if (!launched) {
        set_error("no backward kernel for dim %d", dim);
        return TC_ERR_UNSUPPORTED;
    }
    tc_status st = check_launch("k_backward_short");
    if (st != TC_OK) return st;
    if (ws.cap_pairs > 0) {
        k_backward_list<<<list_blocks(), kLongThreads, 0, stream>>>(grad, dim, ids, out, ws,
                                                                     grad_bytes);
        return check_launch("k_backward_list");
    }
    const int parts = (dim + kPartCols - 1) / kPartCols;
    const int ranges = kLongRanges / parts > 64 ? kLongRanges / parts : 64;
    k_backward_long<<<dim3(ranges, parts), kLongThreads, 0, stream>>>(grad, dim, ids, offsets,
                                                                       num_out_dev, cap, out,
                                                                       grad_bytes);
    return check_launch("k_backward_long");
}

}  // namespace
}  // namespace tc

using namespace tc;

extern "C" tc_status tc_embed_backward(const float *grad_out, int32_t num_bags, int32_t dim,
                                       const int32_t *seg_offsets, const int32_t *casted_src,
                                       const int32_t *num_unique, int64_t max_unique,
                                       float *coal_grad, void *workspace,
                                       size_t workspace_bytes, hipStream_t stream) {
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
    TC_REQUIRE(workspace_bytes == 0 || (workspace && aligned16(workspace)), TC_ERR_INVALID_ARG,
               "tc_embed_backward: workspace must be a 16-byte aligned pointer");
    const RowSink sink{coal_grad, nullptr, nullptr, nullptr, TC_OPT_SGD, 0.f, 0.f, 0.f, 1.f};
    return launch_backward(grad_out, num_bags, dim, casted_src, seg_offsets, num_unique,
                           max_unique, sink, make_split_ws(workspace, workspace_bytes, dim),
                           stream);
}

namespace tc {

// The no-allocation entry point's backward workspace: a fixed array in
// device memory, one copy per GPU, held until the process ends. Host code
// never passes `scratch` itself to a kernel (in host code the name is a
// stand-in, not a device address): it looks up the array's address on each
// device once and passes that.
constexpr size_t kScratchBytes = TC_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

// Argument checks shared by the two backward + update entry points (`what`
// names the caller in messages).
tc_status check_backward_update(const char *what, const float *grad_out, int32_t num_bags,
                                int32_t dim, const int32_t *seg_offsets,
                                const int32_t *casted_src, const int32_t *unique_rows,
                                const int32_t *num_unique, int64_t max_unique, const float *W,
                                const float *opt_state, int64_t total_rows, int32_t opt_kind,
                                float gamma, const float *coal_grad) {
    TC_REQUIRE(num_bags >= 0 && max_unique >= 0 && total_rows >= 0, TC_ERR_INVALID_ARG,
               "%s: negative size", what);
    TC_REQUIRE(max_unique < (int64_t(1) << 31) && total_rows < (int64_t(1) << 31),
               TC_ERR_INVALID_ARG, "%s: sizes must be below 2^31", what);
    TC_REQUIRE(dim > 0 && dim % 4 == 0 && dim <= kMaxDim, TC_ERR_UNSUPPORTED,
               "%s: dim %d must be a multiple of 4 in [4, %d]", what, dim, kMaxDim);
    TC_REQUIRE(opt_kind >= TC_OPT_SGD && opt_kind <= TC_OPT_ROWWISE_ADAGRAD, TC_ERR_INVALID_ARG,
               "%s: unknown optimizer %d", what, opt_kind);
    TC_REQUIRE(opt_kind != TC_OPT_ROWWISE_ADAGRAD, TC_ERR_UNSUPPORTED,
               "%s: row-wise Adagrad needs whole rows; use tc_embed_backward and "
               "tc_sparse_update", what);
    TC_REQUIRE((opt_kind == TC_OPT_SGD) == (opt_state == nullptr), TC_ERR_INVALID_ARG,
               "%s: opt_state must be NULL for SGD and given otherwise", what);
    TC_REQUIRE(opt_kind != TC_OPT_RMSPROP || (gamma >= 0.f && gamma <= 1.f), TC_ERR_INVALID_ARG,
               "%s: RMSprop gamma must lie in [0, 1]", what);
    if (max_unique == 0) return TC_OK;
    TC_REQUIRE(grad_out && seg_offsets && casted_src && unique_rows && num_unique && W,
               TC_ERR_INVALID_ARG, "%s: null pointer", what);
    TC_REQUIRE(aligned16(grad_out) && aligned16(W) && (!opt_state || aligned16(opt_state)) &&
                   (!coal_grad || aligned16(coal_grad)),
               TC_ERR_UNSUPPORTED, "%s: float pointers must be 16-byte aligned", what);
    return TC_OK;
}

// Address of `scratch` on the current device (hipGetSymbolAddress with that
// device current, looked up once per device), or nullptr with the error set.
void *scratch_address() {
    constexpr int kMaxDevices = 64;
    static void *addr[kMaxDevices] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) {
        set_error("tc_embed_backward_update_noalloc: hipGetDevice: %s", hipGetErrorString(e));
        return nullptr;
    }
    if (dev < 0 || dev >= kMaxDevices) {
        set_error("tc_embed_backward_update_noalloc: device %d beyond the %d supported", dev,
                  kMaxDevices);
        return nullptr;
    }
    void *p = __atomic_load_n(&addr[dev], __ATOMIC_ACQUIRE);
    if (p) return p;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr) {
        set_error("tc_embed_backward_update_noalloc: hipGetSymbolAddress(scratch): %s",
                  hipGetErrorString(e));
        return nullptr;
    }
    __atomic_store_n(&addr[dev], p, __ATOMIC_RELEASE);
    return p;
}

}  // namespace
}  // namespace tc

extern "C" tc_status tc_embed_backward_update(
    const float *grad_out, int32_t num_bags, int32_t dim, const int32_t *seg_offsets,
    const int32_t *casted_src, const int32_t *unique_rows, const int32_t *num_unique,
    int64_t max_unique, float *W, float *opt_state, int64_t total_rows, int32_t opt_kind,
    float lr, float eps, float gamma, float *coal_grad, void *workspace, size_t workspace_bytes,
    hipStream_t stream) {
    clear_error();
    const tc_status st = check_backward_update(
        "tc_embed_backward_update", grad_out, num_bags, dim, seg_offsets, casted_src,
        unique_rows, num_unique, max_unique, W, opt_state, total_rows, opt_kind, gamma,
        coal_grad);
    if (st != TC_OK || max_unique == 0) return st;
    TC_REQUIRE(workspace_bytes == 0 || (workspace && aligned16(workspace)), TC_ERR_INVALID_ARG,
               "tc_embed_backward_update: workspace must be a 16-byte aligned pointer");
    const RowSink sink{coal_grad, W, opt_state, unique_rows, opt_kind, lr, eps, gamma,
                       1.0f - gamma};
    return launch_backward(grad_out, num_bags, dim, casted_src, seg_offsets, num_unique,
                           max_unique, sink, make_split_ws(workspace, workspace_bytes, dim),
                           stream);
}

extern "C" tc_status tc_embed_backward_update_noalloc(
    const float *grad_out, int32_t num_bags, int32_t dim, const int32_t *seg_offsets,
    const int32_t *casted_src, const int32_t *unique_rows, const int32_t *num_unique,
    int64_t max_unique, int64_t num_pairs, float *W, float *opt_state, int64_t total_rows,
    int32_t opt_kind, float lr, float eps, float gamma, float *coal_grad, hipStream_t stream) {
    clear_error();
    const tc_status st = check_backward_update(
        "tc_embed_backward_update_noalloc", grad_out, num_bags, dim, seg_offsets, casted_src,
        unique_rows, num_unique, max_unique, W, opt_state, total_rows, opt_kind, gamma,
        coal_grad);
    if (st != TC_OK) return st;
    TC_REQUIRE(num_pairs >= 0 && num_pairs < (int64_t(1) << 31), TC_ERR_INVALID_ARG,
               "tc_embed_backward_update_noalloc: num_pairs must lie in [0, 2^31)");
    const size_t need = num_pairs < kLongSegment ? 0 : ws_layout(num_pairs, dim).total;
    TC_REQUIRE(need <= kScratchBytes, TC_ERR_WORKSPACE,
               "tc_embed_backward_update_noalloc: %lld pairs of dim %d need %zu bytes of "
               "backward workspace, more than the %zu-byte scratch (TC_NOALLOC_SCRATCH_BYTES); "
               "use tc_embed_backward_update with a workspace",
               static_cast<long long>(num_pairs), dim, need, kScratchBytes);
    if (max_unique == 0) return TC_OK;
    void *ws = scratch_address();
    if (ws == nullptr) return TC_ERR_HIP;
    const RowSink sink{coal_grad, W, opt_state, unique_rows, opt_kind, lr, eps, gamma,
                       1.0f - gamma};
    return launch_backward(grad_out, num_bags, dim, casted_src, seg_offsets, num_unique,
                           max_unique, sink, make_split_ws(ws, kScratchBytes, dim), stream);
}

extern "C" tc_status tc_embed_expand(const float *grad_out, int32_t num_bags, int32_t dim,
                                     const int32_t *bag_offsets, int64_t num_pairs,
                                     float *expanded, hipStream_t stream) {
    clear_error();
    TC_REQUIRE(num_bags >= 0 && num_pairs >= 0, TC_ERR_INVALID_ARG,
               "tc_embed_expand: negative size");
    TC_REQUIRE(num_pairs < (int64_t(1) << 31), TC_ERR_INVALID_ARG,
               "tc_embed_expand: num_pairs must be below 2^31");
    TC_REQUIRE(dim > 0 && dim % 4 == 0 && dim <= kMaxDim, TC_ERR_UNSUPPORTED,
               "tc_embed_expand: dim %d must be a multiple of 4 in [4, %d]", dim, kMaxDim);
    if (num_bags == 0 || num_pairs == 0) return TC_OK;
    TC_REQUIRE(grad_out && bag_offsets && expanded, TC_ERR_INVALID_ARG,
               "tc_embed_expand: null pointer");
    TC_REQUIRE(aligned16(grad_out) && aligned16(expanded), TC_ERR_UNSUPPORTED,
               "tc_embed_expand: grad_out and expanded must be 16-byte aligned");
    return launch_expand(grad_out, dim, bag_offsets, num_bags, expanded, stream);
}

extern "C" tc_status tc_embed_coalesce(const float *expanded, int64_t num_pairs, int32_t dim,
                                       const int32_t *seg_offsets, const int32_t *sorted_pos,
                                       const int32_t *num_unique, int64_t max_unique,
                                       float *coal_grad, void *workspace,
                                       size_t workspace_bytes, hipStream_t stream) {
    clear_error();
    TC_REQUIRE(num_pairs >= 0 && max_unique >= 0, TC_ERR_INVALID_ARG,
               "tc_embed_coalesce: negative size");
    TC_REQUIRE(num_pairs < (int64_t(1) << 31) && max_unique < (int64_t(1) << 31),
               TC_ERR_INVALID_ARG, "tc_embed_coalesce: sizes must be below 2^31");
    TC_REQUIRE(dim > 0 && dim % 4 == 0 && dim <= kMaxDim, TC_ERR_UNSUPPORTED,
               "tc_embed_coalesce: dim %d must be a multiple of 4 in [4, %d]", dim, kMaxDim);
    if (max_unique == 0) return TC_OK;
    TC_REQUIRE(expanded && seg_offsets && sorted_pos && num_unique && coal_grad,
               TC_ERR_INVALID_ARG, "tc_embed_coalesce: null pointer");
    TC_REQUIRE(aligned16(expanded) && aligned16(coal_grad), TC_ERR_UNSUPPORTED,
               "tc_embed_coalesce: expanded and coal_grad must be 16-byte aligned");
    TC_REQUIRE(workspace_bytes == 0 || (workspace && aligned16(workspace)), TC_ERR_INVALID_ARG,
               "tc_embed_coalesce: workspace must be a 16-byte aligned pointer");
    // Algorithm 1's accumulate is the casted gather-reduce over the expanded
    // rows, in sorted order: the same kernels with sorted positions as ids.
    const RowSink sink{coal_grad, nullptr, nullptr, nullptr, TC_OPT_SGD, 0.f, 0.f, 0.f, 1.f};
    return launch_backward(expanded, num_pairs, dim, sorted_pos, seg_offsets, num_unique,
                           max_unique, sink, make_split_ws(workspace, workspace_bytes, dim),
                           stream);
}

extern "C" size_t tc_backward_workspace_bytes(int64_t num_pairs, int32_t dim) {
    if (num_pairs < kLongSegment || dim <= 0 || dim > kMaxDim ||
        num_pairs >= (int64_t(1) << 31))
        return 0;
    return ws_layout(num_pairs, dim).total;
}
