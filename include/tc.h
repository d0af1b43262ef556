/*
 * tc.h -- C-ABI of the Tensor Casting sparse-embedding training library for
 * AMD Instinct MI355X (gfx950).
 *
 * One training step of sparse embedding layers is four calls, in stream
 * order (Kwon, Lee, Rhu, "Tensor Casting: Co-Designing Algorithm-Architecture
 * for Personalized Recommendation Training", arXiv 2010.13100):
 *
 *   tc_embed_forward   embedding gather-reduce (Sec. II-B): pooled row sums
 *   tc_cast_index      Tensor Casting (Algorithm 2, Sec. IV-A)
 *                      (tc_embed_forward_cast does these two in one call,
 *                      overlapped, as the paper's runtime does, Sec. IV-B)
 *   tc_embed_backward  casted gradient gather-reduce (Algorithm 3)
 *   tc_sparse_update   gradient scatter with SGD, Adagrad (Eq. 2) or RMSprop
 *                      (Eq. 1), Sec. II-B
 *
 * tc_embed_backward_update does the last two in one pass (same results bit
 * for bit) without storing the coalesced gradient in device memory.
 *
 * The paper's baseline backward (gradient expand-coalesce, Sec. II-B and
 * Algorithm 1), for comparing against the casted one on the same GPU:
 *   tc_embed_expand    one copy of the output gradient per pair
 *   tc_argsort_rows    stable argsort of the pairs by row (Algorithm 1's ArgSort)
 *   tc_embed_coalesce  Algorithm 1's ordered accumulate of the expanded rows
 *
 * tc_check_index checks an index array on the device before it is trusted.
 *
 * Conventions shared by every call
 * --------------------------------
 * Pointers are DEVICE pointers owned by the caller unless a comment says
 * "host". The library never allocates or frees device memory, never
 * synchronises the stream and never copies to the host; scratch memory comes
 * from the caller's workspaces (tc_cast_workspace_bytes,
 * tc_backward_workspace_bytes), or, for tc_embed_backward_update_noalloc,
 * from a fixed array the library holds in device memory. Buffers must stay
 * alive until the stream has finished the call.
 *
 * Every call is asynchronous on `stream` (a hipStream_t; NULL is the legacy
 * default stream) and returns a tc_status. Host-side argument checks run
 * before anything is launched; on such an error nothing is launched and no
 * output is touched. A failed launch returns TC_ERR_HIP. tc_last_error()
 * then gives a message for the calling thread.
 *
 * Layout
 *  - Tables: T tables of the same width `dim` (fp32) are stored as one
 *    row-major array of `total_rows` x `dim` floats. Table t owns global rows
 *    [table_row_offset[t], table_row_offset[t+1]); `table_row_offset` is a
 *    device int64 array of T+1 entries with table_row_offset[T] = total_rows.
 *  - The index array of (src, dst) pairs (Sec. II-B) is bag-major CSR:
 *    bag g = t * bags_per_table + b holds pairs bag_offsets[g] ..
 *    bag_offsets[g+1]-1 (device int32, T*B+1 entries, non-decreasing,
 *    bag_offsets[0] = 0, bag_offsets[T*B] = num_pairs); `indices[j]` is the
 *    table-local row of pair j. src of pair j is table_row_offset[t] +
 *    indices[j], dst is g.
 *  - `dim` must be a multiple of 4 in [4, 1024], and every float pointer must
 *    be 16-byte aligned (TC_ERR_UNSUPPORTED otherwise); num_pairs and
 *    total_rows must be below 2^31.
 *  - Out-of-range indices or malformed offsets are not detected by the
 *    training calls and give undefined results (reads and writes outside
 *    the table included); tc_check_index checks an index array on the
 *    device without copying anything to the host.
 *
 * Arithmetic: fp32 values, fp32 accumulation. Sums are taken one term after
 * another, from +0, in the order of the index array (forward) or of the
 * casted index (backward). The one exception is opt-in: given a backward
 * workspace, the backward sums a segment of TC_BACKWARD_SPLIT_PAIRS pairs or
 * more in pieces (see tc_embed_backward). Either way results do not depend
 * on the launch configuration and repeat bit for bit.
 *
 * Thread safety: no global state besides the per-thread error message;
 * concurrent calls on different streams with different buffers are safe.
 */
#ifndef TC_H
#define TC_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TC_ABI_VERSION 7

/* Segments at least this long are summed in pieces when a backward
 * workspace covers them (tc_embed_backward). */
#define TC_BACKWARD_SPLIT_PAIRS 2048

typedef enum tc_status {
    TC_OK = 0,
    TC_ERR_INVALID_ARG = 1,  /* null pointer with a non-zero size, negative size, ... */
    TC_ERR_UNSUPPORTED = 2,  /* dim or alignment outside what the kernels handle */
    TC_ERR_WORKSPACE = 3,    /* workspace missing or smaller than tc_cast_workspace_bytes */
    TC_ERR_HIP = 4           /* a HIP launch failed; see tc_last_error() */
} tc_status;

typedef enum tc_opt_kind {
    TC_OPT_SGD = 0,             /* W <- W - lr*G */
    TC_OPT_ADAGRAD = 1,         /* Eq. (2): A <- A + G*G; W <- W - lr*G/sqrt(eps + A) */
    TC_OPT_RMSPROP = 2,         /* Eq. (1): A <- gamma*A + (1-gamma)*G*G; same W step */
    TC_OPT_ROWWISE_ADAGRAD = 3  /* Eq. (2) with one A per row, grown by mean(G*G) */
} tc_opt_kind;

/*
 * Forward embedding gather-reduce (Sec. II-B, forward propagation).
 * For every bag g: out[g, :] = sum over its pairs j, in order, of
 * W[table_row_offset[g / bags_per_table] + indices[j], :], starting from +0.
 * An empty bag gives a row of zeros.
 *   W        [total_rows x dim] fp32 table (read only)
 *   indices  may be NULL when every bag is empty
 *   out      [num_tables*bags_per_table x dim] fp32 (written)
 */
tc_status tc_embed_forward(const float *W, int64_t total_rows, int32_t dim,
                           const int64_t *table_row_offset, int32_t num_tables,
                           int32_t bags_per_table, const int32_t *indices,
                           const int32_t *bag_offsets, float *out, hipStream_t stream);

/*
 * Workspace bytes tc_cast_index needs for `num_pairs` pairs over
 * `total_rows` global rows in `num_tables` tables (host function; launches
 * nothing).
 */
size_t tc_cast_workspace_bytes(int64_t num_pairs, int64_t total_rows, int32_t num_tables);

/*
 * Tensor Casting (Algorithm 2). The (src, dst) pairs are sorted by src with
 * a stable sort (equal src keep their input order, so with bag-major input
 * the result is the (row, bag) lexicographic order). Then
 *   casted_src[i] = dst of the i-th sorted pair (its bag id)
 *   casted_dst[i] = (number of distinct src among sorted pairs 0..i) - 1
 * and, per coalesced row u < U (U = number of distinct src):
 *   unique_rows[u] = its global row (strictly increasing in u)
 *   seg_offsets[u] = first sorted position of that row; seg_offsets[U] = num_pairs
 *   *num_unique    = U (device int32; never copied to the host)
 * Capacities: casted_src and casted_dst hold num_pairs entries; unique_rows
 * holds min(num_pairs, total_rows) and seg_offsets one more. casted_dst may
 * be NULL (the backward pass does not need it). All outputs are int32 and
 * exact. `workspace` is device memory of at least
 * tc_cast_workspace_bytes(num_pairs, total_rows, num_tables) bytes, 256-byte
 * aligned.
 * max_table_rows (host) is an upper bound on the rows of every table, hence
 * on every index, or 0 if unknown. It only selects the sort: with a bound
 * much smaller than total_rows (and at most 256 tables) each table is sorted
 * on its table-local row, which takes fewer radix passes; the results are
 * the same either way. An index at or above a non-zero bound gives undefined
 * results, as any out-of-range index does.
 */
tc_status tc_cast_index(const int64_t *table_row_offset, int32_t num_tables,
                        int32_t bags_per_table, int64_t total_rows, int64_t max_table_rows,
                        const int32_t *indices,
                        const int32_t *bag_offsets, int64_t num_pairs, int32_t *unique_rows,
                        int32_t *seg_offsets, int32_t *casted_src, int32_t *casted_dst,
                        int32_t *num_unique, void *workspace, size_t workspace_bytes,
                        hipStream_t stream);

/*
 * tc_embed_forward followed by tc_cast_index in one call, with the same
 * results bit for bit, the forward overlapped with the cast: casting needs
 * only the index array, so it can run while the forward gather-reduce reads
 * the table (the paper's runtime hides the casting latency inside forward
 * propagation, Sec. IV-B). For dim in [36, 256] the forward runs in the
 * cast's own launches: beside the single-workgroup cast of a small batch
 * (up to 8192 pairs), else in the launch that builds the cast's (row, bag)
 * pairs from the same index array; for other dims the forward runs first,
 * then the cast. Arguments are those of the two calls (max_table_rows
 * and the workspace as for tc_cast_index, W and out as for
 * tc_embed_forward); out must not overlap the cast's outputs or workspace.
 * Every argument is checked before anything is launched.
 */
tc_status tc_embed_forward_cast(const float *W, int64_t total_rows, int32_t dim,
                                const int64_t *table_row_offset, int32_t num_tables,
                                int32_t bags_per_table, int64_t max_table_rows,
                                const int32_t *indices, const int32_t *bag_offsets,
                                int64_t num_pairs, float *out, int32_t *unique_rows,
                                int32_t *seg_offsets, int32_t *casted_src, int32_t *casted_dst,
                                int32_t *num_unique, void *workspace, size_t workspace_bytes,
                                hipStream_t stream);

/*
 * Stable argsort of the pairs by row (Algorithm 1's ArgSort, Sec. II-B):
 * sorted_pos[i] = position j of the i-th pair in row order (equal rows keep
 * their input order), with unique_rows, seg_offsets and *num_unique as in
 * tc_cast_index. Arguments, capacities and workspace are those of
 * tc_cast_index; sorted_pos holds num_pairs entries.
 */
tc_status tc_argsort_rows(const int64_t *table_row_offset, int32_t num_tables,
                          int32_t bags_per_table, int64_t total_rows, int64_t max_table_rows,
                          const int32_t *indices, const int32_t *bag_offsets, int64_t num_pairs,
                          int32_t *unique_rows, int32_t *seg_offsets, int32_t *sorted_pos,
                          int32_t *num_unique, void *workspace, size_t workspace_bytes,
                          hipStream_t stream);

/*
 * Gradient expand (Sec. II-B, the baseline backward): for every pair j of
 * bag g, expanded[j, :] = grad_out[g, :].
 *   grad_out  [num_bags x dim] fp32; bag_offsets as for tc_cast_index
 *   expanded  [num_pairs x dim] fp32 (written)
 */
tc_status tc_embed_expand(const float *grad_out, int32_t num_bags, int32_t dim,
                          const int32_t *bag_offsets, int64_t num_pairs, float *expanded,
                          hipStream_t stream);

/*
 * Gradient coalescing, Algorithm 1's accumulate: for every u < *num_unique,
 *   coal_grad[u, :] = sum over i in [seg_offsets[u], seg_offsets[u+1]), in
 *                     order, of expanded[sorted_pos[i], :], starting from +0,
 * with seg_offsets and sorted_pos from tc_argsort_rows. Equals
 * tc_embed_backward's coal_grad bit for bit (same rows, same order), also
 * with a workspace: workspace and workspace_bytes work as there.
 */
tc_status tc_embed_coalesce(const float *expanded, int64_t num_pairs, int32_t dim,
                            const int32_t *seg_offsets, const int32_t *sorted_pos,
                            const int32_t *num_unique, int64_t max_unique, float *coal_grad,
                            void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Bytes of a backward workspace that covers a step of up to num_pairs pairs
 * with rows of `dim` floats, for tc_embed_backward, tc_embed_backward_update
 * and tc_embed_coalesce; 0 if no segment can be long (num_pairs < 80) or
 * the arguments are out of range. About num_pairs * (dim / 256 + 0.25)
 * bytes.
 */
size_t tc_backward_workspace_bytes(int64_t num_pairs, int32_t dim);

/*
 * Casted gradient gather-reduce (Algorithm 3): for every u < *num_unique,
 *   coal_grad[u, :] = sum over i in [seg_offsets[u], seg_offsets[u+1]), in
 *                     order, of grad_out[casted_src[i], :], starting from +0.
 * This is the coalesced gradient of table row unique_rows[u]; the expanded
 * per-pair gradient is never formed.
 *   grad_out   [num_bags x dim] fp32, one gradient per pooled output
 *   max_unique capacity of coal_grad in rows (>= *num_unique), normally
 *              min(num_pairs, total_rows)
 *   coal_grad  [max_unique x dim] fp32; rows >= *num_unique are not written
 *   workspace, workspace_bytes
 *              optional (NULL, 0: none), sized with
 *              tc_backward_workspace_bytes for the step's pairs. With it,
 *              long segments are scheduled over persistent workgroups, and a
 *              segment [b, b + len) with len >= TC_BACKWARD_SPLIT_PAIRS that
 *              the workspace covers (b + len <= the num_pairs it was sized
 *              for) is summed in pieces instead of one chain: n =
 *              min(32, len / 1024) pieces, piece q being pairs
 *              [b + floor(q*len/n), b + floor((q+1)*len/n)), each summed in
 *              order from +0, and the n piece sums added in piece order from
 *              +0. Other segments are summed as above. The order depends on
 *              the segment's length only, so results still repeat bit for
 *              bit. Device memory, 16-byte aligned (TC_ERR_INVALID_ARG
 *              otherwise), read and written by the call; no initial contents
 *              are needed and calls that share one workspace must not
 *              overlap. Segments past the cover are still summed correctly,
 *              as one chain, but slowly.
 */
tc_status tc_embed_backward(const float *grad_out, int32_t num_bags, int32_t dim,
                            const int32_t *seg_offsets, const int32_t *casted_src,
                            const int32_t *num_unique, int64_t max_unique, float *coal_grad,
                            void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Gradient scatter + optimizer (Sec. II-B; RMSprop is Eq. 1, Adagrad Eq. 2).
 * For every u < *num_unique, with r = unique_rows[u] and G = coal_grad[u, :]:
 *   TC_OPT_SGD:     elementwise t = lr*G;  W[r] = W[r] - t
 *   TC_OPT_ADAGRAD: elementwise A[r] = A[r] + G*G;  s = sqrt(eps + A[r]);
 *                   q = G/s;  W[r] = W[r] - lr*q
 *   TC_OPT_RMSPROP: elementwise t = gamma*A[r];  c = 1 - gamma;
 *                   A[r] = t + c*(G*G);  s = sqrt(eps + A[r]);  q = G/s;
 *                   W[r] = W[r] - lr*q
 *   TC_OPT_ROWWISE_ADAGRAD: one accumulator per row (a variant of Eq. 2
 *                   that the paper does not define):
 *                   m = (G_0^2 + ... + G_{dim-1}^2) / dim, summed in column
 *                   order from +0;  A[r] = A[r] + m;  s = sqrt(eps + A[r]);
 *                   then elementwise q = G/s;  W[r] = W[r] - lr*q
 * each a separately rounded fp32 operation (no fused multiply-add; division
 * and square root correctly rounded). Rows not in unique_rows are untouched:
 * the update is lazy, which for SGD and both Adagrads equals a dense update
 * with zero gradient; for RMSprop the accumulator of an untouched row is not
 * decayed.
 *   W          [total_rows x dim] fp32 table (read-modify-write)
 *   opt_state  the accumulator A (read-modify-write): [total_rows x dim] for
 *              Adagrad and RMSprop, [total_rows] for row-wise Adagrad; must
 *              be NULL for SGD
 *   gamma      RMSprop's decay, in [0, 1] (TC_ERR_INVALID_ARG otherwise);
 *              ignored by the other optimizers
 *   unique_rows must be distinct (as tc_cast_index produces them).
 */
tc_status tc_sparse_update(float *W, float *opt_state, int64_t total_rows, int32_t dim,
                           const int32_t *unique_rows, const float *coal_grad,
                           const int32_t *num_unique, int64_t max_unique, int32_t opt_kind,
                           float lr, float eps, float gamma, hipStream_t stream);

/*
 * Casted gradient gather-reduce (Algorithm 3) fused with the gradient
 * scatter + optimizer (Sec. II-B, Eqs. 1 and 2): for every u < *num_unique,
 * the coalesced row G of tc_embed_backward is formed in registers and
 * applied to W[unique_rows[u]] (and the accumulator) exactly as
 * tc_sparse_update applies it. The results equal those two calls bit for
 * bit; the coalesced gradient is stored to coal_grad only if that is not
 * NULL. Arguments are those of the two calls (coal_grad optional, the
 * workspace as for tc_embed_backward); W,
 * opt_state and grad_out must not overlap. Supports TC_OPT_SGD,
 * TC_OPT_ADAGRAD and TC_OPT_RMSPROP; TC_OPT_ROWWISE_ADAGRAD returns
 * TC_ERR_UNSUPPORTED (a row's columns are reduced by different workgroups,
 * so no one of them sees the whole row): use tc_embed_backward followed by
 * tc_sparse_update for it.
 */
tc_status tc_embed_backward_update(const float *grad_out, int32_t num_bags, int32_t dim,
                                   const int32_t *seg_offsets, const int32_t *casted_src,
                                   const int32_t *unique_rows, const int32_t *num_unique,
                                   int64_t max_unique, float *W, float *opt_state,
                                   int64_t total_rows, int32_t opt_kind, float lr, float eps,
                                   float gamma, float *coal_grad, void *workspace,
                                   size_t workspace_bytes, hipStream_t stream);

/* Bytes of the fixed device scratch of tc_embed_backward_update_noalloc
 * (one copy per GPU the library runs that call on). */
#define TC_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)

/*
 * tc_embed_backward_update for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same computation, kernels and results bit for bit as
 * tc_embed_backward_update given a workspace that covers the step, but the
 * backward workspace is a fixed array of TC_NOALLOC_SCRATCH_BYTES in device
 * memory that the library holds, one per GPU, from the first use on that
 * GPU until the process ends. The call allocates and frees nothing.
 *   num_pairs  pairs of the step (seg_offsets[*num_unique]). The call
 *              returns TC_ERR_WORKSPACE, launching nothing, when
 *              tc_backward_workspace_bytes(num_pairs, dim) exceeds
 *              TC_NOALLOC_SCRATCH_BYTES (it covers up to 35.8M pairs at
 *              dim 64, 13.7M at dim 256, 3.9M at dim 1024).
 * Other arguments and checks are those of tc_embed_backward_update.
 * Every call on one GPU uses that GPU's one scratch array, which keeps the
 * last call's contents (the call itself clears what must start at zero):
 * calls that overlap on one GPU (different streams, or different threads
 * without ordering) race and give undefined results; calls in stream order
 * on one stream are safe. The first call on a GPU looks the array's address
 * up (hipGetSymbolAddress) and may return TC_ERR_HIP if that fails.
 */
tc_status tc_embed_backward_update_noalloc(const float *grad_out, int32_t num_bags, int32_t dim,
                                           const int32_t *seg_offsets,
                                           const int32_t *casted_src,
                                           const int32_t *unique_rows,
                                           const int32_t *num_unique, int64_t max_unique,
                                           int64_t num_pairs, float *W, float *opt_state,
                                           int64_t total_rows, int32_t opt_kind, float lr,
                                           float eps, float gamma, float *coal_grad,
                                           hipStream_t stream);

/* What tc_check_index found (report[0]). */
typedef enum tc_index_problem {
    TC_INDEX_OK = 0,
    TC_INDEX_BAD_TABLE_OFFSETS = 1,  /* table_row_offset[0] != 0, a decrease, or [T] != total_rows */
    TC_INDEX_BAD_BAG_OFFSETS = 2,    /* bag_offsets[0] != 0, a decrease, or [T*B] != num_pairs */
    TC_INDEX_OUT_OF_RANGE = 3        /* an index < 0, >= its table's rows, or >= max_table_rows */
} tc_index_problem;

/*
 * Checks the index array of a step (the (src, dst) pairs of Sec. II-B in the
 * layout above) on the device, for callers whose indices are not trusted:
 *   table_row_offset [T+1]: starts at 0, never decreases, ends at total_rows
 *   bag_offsets      [T*B+1]: starts at 0, never decreases, ends at num_pairs
 *   indices          [num_pairs]: pair j of table t (the table whose bags
 *                    hold position j) satisfies 0 <= indices[j] <
 *                    table_row_offset[t+1] - table_row_offset[t], and
 *                    indices[j] < max_table_rows when max_table_rows > 0
 *                    (the bound tc_cast_index takes)
 *   report           device int64[2], written: report[0] is a
 *                    tc_index_problem, report[1] the lowest entry t
 *                    (table_row_offset), bag g (bag_offsets) or pair j
 *                    (indices) where it holds, or -1 if there is none. Of
 *                    several problems the lowest kind is reported, then the
 *                    lowest position; the result does not depend on the
 *                    launch configuration. 8-byte aligned.
 * Arguments are those of tc_cast_index; the library does not read report
 * back: the caller copies it after the stream reaches it. Never reads
 * outside the arrays' stated sizes, whatever their contents.
 */
tc_status tc_check_index(const int64_t *table_row_offset, int32_t num_tables,
                         int32_t bags_per_table, int64_t total_rows, int64_t max_table_rows,
                         const int32_t *indices, const int32_t *bag_offsets, int64_t num_pairs,
                         int64_t *report, hipStream_t stream);

/* Static text for a status code. */
const char *tc_status_string(tc_status status);

/* Message of the calling thread's last failed call ("" if none). */
const char *tc_last_error(void);

/* TC_ABI_VERSION of the loaded library. */
int32_t tc_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* TC_H */
