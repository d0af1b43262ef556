/*
 * Tensor Casting CPU oracle -- TEST INFRASTRUCTURE, not part of the product.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * may load this library. It shares no source with the HIP library: no
 * headers, helpers, tables or generators.
 *
 * What it is: a plain, single-threaded, unoptimised implementation of one
 * training step of sparse embedding layers, written from the paper
 * (Kwon, Lee, Rhu, "Tensor Casting: Co-Designing Algorithm-Architecture for
 * Personalized Recommendation Training", arXiv 2010.13100):
 *
 *   oracle_pairs_from_csr          the (src, dst) index array, Sec. II-B
 *   oracle_forward                 embedding gather-reduce, Sec. II-B
 *   oracle_expand                  gradient expand, Sec. II-B
 *   oracle_coalesce                gradient coalescing, Algorithm 1
 *   oracle_tensor_casting          Tensor Casting, Algorithm 2 (Sec. IV-A)
 *   oracle_casted_gather_reduce    casted gradient gather-reduce, Algorithm 3
 *   oracle_scatter_sgd             gradient scatter with plain SGD, Sec. II-B
 *   oracle_scatter_adagrad         gradient scatter with Adagrad, Eq. (2)
 *   oracle_scatter_rmsprop         gradient scatter with RMSprop, Eq. (1)
 *   oracle_scatter_rowwise_adagrad gradient scatter with row-wise Adagrad, a
 *                                  variant of Eq. (2) that the paper does
 *                                  not define (one accumulator per row)
 *
 * The arithmetic type is fixed at build time: -DOREAL=double gives the
 * reference used to pin the method against closed forms, -DOREAL=float
 * gives the same steps in the fp32 arithmetic the workloads specify. Every
 * floating-point operation is a separately rounded IEEE operation: the
 * library is built with -ffp-contract=off and without -ffast-math.
 *
 * Readings of the paper where it is silent or ambiguous:
 *  - loop bounds "0 to n" mean 0..n-1, and Algorithm 2's "1 to n" means
 *    1..n-1;
 *  - Algorithm 1 carries the previous key forward (prev <- curr) after every
 *    step; without it no two gradients would ever be coalesced;
 *  - ArgSort and SortByKey are stable: equal keys keep their input order;
 *  - the reduction is a sum; sums run sequentially in index order;
 *  - Algorithm 3's coalesced-gradient array starts at zero;
 *  - Adagrad's accumulator starts at zero and epsilon sits inside the square
 *    root, as Eq. (2) writes it;
 *  - RMSprop's decay gamma is a parameter (the paper gives no value), and
 *    its update is lazy like the others: rows without a gradient in the
 *    step keep W and A, their A is not decayed;
 *  - row-wise Adagrad adds the mean of the row's squared gradient to the
 *    row's accumulator and divides every element by the one square root.
 *
 * Tables are passed as a row set: `ids` is either NULL (dense table, row r
 * stored at r*dim) or a strictly increasing list of the global row ids that
 * are stored, so a test can hand over only the rows a step touches.
 *
 * Return values: 0 (or a count >= 0) on success, a negative code on error:
 * -1 bad argument, -2 a row not present in the row set, -3 out of memory.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifndef OREAL
#define OREAL double
#endif
typedef OREAL real;

#define ORACLE_ERR_ARG (-1)
#define ORACLE_ERR_ROW (-2)
#define ORACLE_ERR_OOM (-3)

/* Square root in the arithmetic type (correctly rounded in both types). */
static real real_sqrt(real x)
{
    if (sizeof(real) == sizeof(float))
        return (real)sqrtf((float)x);
    return (real)sqrt((double)x);
}

int oracle_real_bytes(void) { return (int)sizeof(real); }

/* Storage of global row `r` in a row set (see the header comment). */
static real *row_at(real *vals, const int64_t *ids, int64_t n, int32_t dim, int64_t r)
{
    if (ids == NULL) {
        if (r < 0 || r >= n)
            return NULL;
        return vals + r * (int64_t)dim;
    }
    int64_t lo = 0, hi = n; /* search [lo, hi) */
    while (lo < hi) {
        int64_t mid = lo + (hi - lo) / 2;
        if (ids[mid] < r)
            lo = mid + 1;
        else
            hi = mid;
    }
    if (lo < n && ids[lo] == r)
        return vals + lo * (int64_t)dim;
    return NULL;
}

/*
 * The paper's index array of (src, dst) pairs (Sec. II-B): src names the
 * table row to gather, dst the reduced output (bag) it is added into. The
 * bag-major CSR form keeps dst implicit; this writes it out. Bag g belongs
 * to table g / bags_per_table, whose rows start at global row
 * table_row_offset[table].
 */
int oracle_pairs_from_csr(int32_t num_tables, int32_t bags_per_table,
                          const int64_t *table_row_offset, const int32_t *indices,
                          const int32_t *bag_offsets, int64_t *src, int32_t *dst)
{
    if (num_tables < 0 || bags_per_table < 0)
        return ORACLE_ERR_ARG;
    int64_t num_bags = (int64_t)num_tables * bags_per_table;
    for (int64_t g = 0; g < num_bags; ++g) {
        int64_t t = g / bags_per_table;
        for (int64_t j = bag_offsets[g]; j < bag_offsets[g + 1]; ++j) {
            src[j] = table_row_offset[t] + indices[j];
            dst[j] = (int32_t)g;
        }
    }
    return 0;
}

/*
 * Embedding gather-reduce (Sec. II-B, forward propagation): every output
 * row dst starts at zero and receives the table rows src of its pairs, added
 * one after another in pair order.
 */
int oracle_forward(int32_t dim, int64_t num_pairs, const int64_t *src, const int32_t *dst,
                   int64_t num_bags, const int64_t *tbl_ids, int64_t tbl_rows,
                   const real *tbl, real *out)
{
    if (dim <= 0 || num_pairs < 0 || num_bags < 0)
        return ORACLE_ERR_ARG;
    for (int64_t i = 0; i < num_bags * dim; ++i)
        out[i] = (real)0;
    for (int64_t j = 0; j < num_pairs; ++j) {
        const real *w = row_at((real *)tbl, tbl_ids, tbl_rows, dim, src[j]);
        if (w == NULL)
            return ORACLE_ERR_ROW;
        if (dst[j] < 0 || dst[j] >= num_bags)
            return ORACLE_ERR_ARG;
        real *o = out + (int64_t)dst[j] * dim;
        for (int32_t d = 0; d < dim; ++d)
            o[d] = o[d] + w[d];
    }
    return 0;
}

/*
 * Gradient expand (Sec. II-B, backpropagation): the gradient of each
 * reduced output is copied once per gather that fed it, giving one
 * gradient row per pair.
 */
int oracle_expand(int32_t dim, int64_t num_pairs, const int32_t *dst, const real *grad_out,
                  real *expanded)
{
    if (dim <= 0 || num_pairs < 0)
        return ORACLE_ERR_ARG;
    for (int64_t j = 0; j < num_pairs; ++j)
        memcpy(expanded + j * dim, grad_out + (int64_t)dst[j] * dim, sizeof(real) * (size_t)dim);
    return 0;
}

/* A key and the position it came from; ordering by (key, pos) is a stable
 * sort by key. */
typedef struct {
    int64_t key;
    int64_t pos;
} keyed_pos;

static int cmp_keyed_pos(const void *a, const void *b)
{
    const keyed_pos *x = (const keyed_pos *)a, *y = (const keyed_pos *)b;
    if (x->key != y->key)
        return x->key < y->key ? -1 : 1;
    if (x->pos != y->pos)
        return x->pos < y->pos ? -1 : 1;
    return 0;
}

/* Stable argsort of `keys`: sorted_pos[k] is the input position of the k-th
 * smallest key, ties in input order. */
static int stable_argsort(int64_t n, const int64_t *keys, int64_t *sorted_pos)
{
    keyed_pos *kp = (keyed_pos *)malloc(sizeof(keyed_pos) * (size_t)(n > 0 ? n : 1));
    if (kp == NULL)
        return ORACLE_ERR_OOM;
    for (int64_t i = 0; i < n; ++i) {
        kp[i].key = keys[i];
        kp[i].pos = i;
    }
    qsort(kp, (size_t)n, sizeof(keyed_pos), cmp_keyed_pos);
    for (int64_t i = 0; i < n; ++i)
        sorted_pos[i] = kp[i].pos;
    free(kp);
    return 0;
}

/*
 * Gradient coalescing, Algorithm 1. Step A sorts the src ids (ArgSort and
 * Sort) so that gradients of the same table row become neighbours. Step B
 * walks the sorted order: a new src id opens a new coalesced gradient that
 * starts as a copy of its first expanded gradient; a repeated id adds its
 * expanded gradient to the open one.
 *
 * Writes coal[U x dim] and coal_rows[U] (the src id of each coalesced row,
 * which the scatter needs); returns U.
 */
int64_t oracle_coalesce(int32_t dim, int64_t num_pairs, const int64_t *src,
                        const real *expanded, real *coal, int64_t *coal_rows)
{
    if (dim <= 0 || num_pairs < 0)
        return ORACLE_ERR_ARG;
    int64_t *sorted_pos = (int64_t *)malloc(sizeof(int64_t) * (size_t)(num_pairs > 0 ? num_pairs : 1));
    if (sorted_pos == NULL)
        return ORACLE_ERR_OOM;
    int rc = stable_argsort(num_pairs, src, sorted_pos);
    if (rc != 0) {
        free(sorted_pos);
        return rc;
    }
    int64_t i = -1, prev = -1;
    for (int64_t j = 0; j < num_pairs; ++j) {
        int64_t pos = sorted_pos[j];
        int64_t curr = src[pos]; /* sorted_src[j] */
        const real *e = expanded + pos * dim;
        if (curr != prev) {
            i = i + 1;
            memcpy(coal + i * dim, e, sizeof(real) * (size_t)dim);
            coal_rows[i] = curr;
        } else {
            real *c = coal + i * dim;
            for (int32_t d = 0; d < dim; ++d)
                c[d] = c[d] + e[d];
        }
        prev = curr;
    }
    free(sorted_pos);
    return i + 1;
}

/*
 * Tensor Casting, Algorithm 2: sort the (src, dst) pairs by src (stable),
 * take the sorted dst ids as the casted src ids, flag every position whose
 * src differs from its predecessor (position 0 always flagged) and take the
 * running count of flags minus one as the casted dst ids.
 *
 * Besides the two casted arrays the scatter needs, per coalesced row u, the
 * table row it belongs to (unique_rows[u], the sorted src at the flag) and
 * where its pairs start (seg_offsets[u]); seg_offsets[U] = n. Returns U.
 * casted_dst, unique_rows and seg_offsets may each be NULL.
 */
int64_t oracle_tensor_casting(int64_t num_pairs, const int64_t *src, const int32_t *dst,
                              int32_t *casted_src, int32_t *casted_dst,
                              int64_t *unique_rows, int64_t *seg_offsets)
{
    if (num_pairs < 0)
        return ORACLE_ERR_ARG;
    int64_t n = num_pairs;
    int64_t *sorted_pos = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    int64_t *sorted_src = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    int64_t *scan = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    if (!sorted_pos || !sorted_src || !scan) {
        free(sorted_pos);
        free(sorted_src);
        free(scan);
        return ORACLE_ERR_OOM;
    }
    int rc = stable_argsort(n, src, sorted_pos); /* SortByKey(src, dst) */
    if (rc != 0) {
        free(sorted_pos);
        free(sorted_src);
        free(scan);
        return rc;
    }
    for (int64_t i = 0; i < n; ++i) {
        sorted_src[i] = src[sorted_pos[i]];
        casted_src[i] = dst[sorted_pos[i]]; /* casted_src <- sorted_dst */
    }
    for (int64_t i = 1; i < n; ++i)
        scan[i] = (sorted_src[i] != sorted_src[i - 1]) ? 1 : 0;
    if (n > 0)
        scan[0] = 1;
    int64_t running = 0; /* CumulativeSum(scan) - 1 */
    for (int64_t i = 0; i < n; ++i) {
        running += scan[i];
        int64_t cd = running - 1;
        if (casted_dst)
            casted_dst[i] = (int32_t)cd;
        if (scan[i]) {
            if (unique_rows)
                unique_rows[cd] = sorted_src[i];
            if (seg_offsets)
                seg_offsets[cd] = i;
        }
    }
    if (seg_offsets)
        seg_offsets[running] = n;
    free(sorted_pos);
    free(sorted_src);
    free(scan);
    return running;
}

/*
 * Casted gradient gather-reduce, Algorithm 3 (GatherReduce): the coalesced
 * gradients start at zero and, in pair order, each casted pair adds output
 * gradient row casted_src[i] into coalesced row casted_dst[i].
 */
int oracle_casted_gather_reduce(int32_t dim, int64_t num_pairs, const int32_t *casted_src,
                                const int32_t *casted_dst, const real *grad_out,
                                int64_t num_bags, int64_t num_unique, real *coal)
{
    if (dim <= 0 || num_pairs < 0 || num_unique < 0)
        return ORACLE_ERR_ARG;
    for (int64_t i = 0; i < num_unique * dim; ++i)
        coal[i] = (real)0;
    for (int64_t i = 0; i < num_pairs; ++i) {
        if (casted_dst[i] < 0 || casted_dst[i] >= num_unique)
            return ORACLE_ERR_ARG;
        if (casted_src[i] < 0 || casted_src[i] >= num_bags)
            return ORACLE_ERR_ARG;
        real *c = coal + (int64_t)casted_dst[i] * dim;
        const real *g = grad_out + (int64_t)casted_src[i] * dim;
        for (int32_t d = 0; d < dim; ++d)
            c[d] = c[d] + g[d];
    }
    return 0;
}

/*
 * Gradient scatter with plain SGD (Sec. II-B): every coalesced gradient G of
 * table row r moves that row by -lr * G; rows without a gradient are left
 * as they are. Order of operations: t = lr * G, then W = W - t.
 */
int oracle_scatter_sgd(int32_t dim, int64_t num_unique, const int64_t *rows, const real *coal,
                       double lr, const int64_t *tbl_ids, int64_t tbl_rows, real *tbl)
{
    if (dim <= 0 || num_unique < 0)
        return ORACLE_ERR_ARG;
    const real rlr = (real)lr;
    for (int64_t u = 0; u < num_unique; ++u) {
        real *w = row_at(tbl, tbl_ids, tbl_rows, dim, rows[u]);
        if (w == NULL)
            return ORACLE_ERR_ROW;
        const real *g = coal + u * dim;
        for (int32_t d = 0; d < dim; ++d) {
            real t = rlr * g[d];
            w[d] = w[d] - t;
        }
    }
    return 0;
}

/*
 * Gradient scatter with Adagrad, Eq. (2): A <- A + G^2, then
 * W <- W - lr * G / sqrt(eps + A), element by element, for the rows that
 * have a coalesced gradient. Order of operations:
 * A = A + G*G; s = sqrt(eps + A); q = G / s; W = W - lr * q.
 * `acc` is stored with the same row set as the table.
 */
int oracle_scatter_adagrad(int32_t dim, int64_t num_unique, const int64_t *rows,
                           const real *coal, double lr, double eps, const int64_t *tbl_ids,
                           int64_t tbl_rows, real *tbl, real *acc)
{
    if (dim <= 0 || num_unique < 0)
        return ORACLE_ERR_ARG;
    const real rlr = (real)lr, reps = (real)eps;
    for (int64_t u = 0; u < num_unique; ++u) {
        real *w = row_at(tbl, tbl_ids, tbl_rows, dim, rows[u]);
        real *a = row_at(acc, tbl_ids, tbl_rows, dim, rows[u]);
        if (w == NULL || a == NULL)
            return ORACLE_ERR_ROW;
        const real *g = coal + u * dim;
        for (int32_t d = 0; d < dim; ++d) {
            real sq = g[d] * g[d];
            a[d] = a[d] + sq;
            real s = real_sqrt(reps + a[d]);
            real q = g[d] / s;
            real step = rlr * q;
            w[d] = w[d] - step;
        }
    }
    return 0;
}

/*
 * Gradient scatter with RMSprop, Eq. (1): the accumulator becomes a running
 * average of squared gradients, A <- gamma*A + (1-gamma)*G^2, and then
 * W <- W - lr * G / sqrt(eps + A), element by element, for the rows that
 * have a coalesced gradient. Rows without a gradient keep W and A (the same
 * lazy update as the Adagrad scatter). Order of operations:
 * t = gamma*A; c = 1 - gamma; A = t + c*(G*G); s = sqrt(eps + A);
 * q = G / s; W = W - lr * q.
 */
int oracle_scatter_rmsprop(int32_t dim, int64_t num_unique, const int64_t *rows,
                           const real *coal, double lr, double eps, double gamma,
                           const int64_t *tbl_ids, int64_t tbl_rows, real *tbl, real *acc)
{
    if (dim <= 0 || num_unique < 0)
        return ORACLE_ERR_ARG;
    const real rlr = (real)lr, reps = (real)eps, rg = (real)gamma;
    const real rc = (real)1 - rg;
    for (int64_t u = 0; u < num_unique; ++u) {
        real *w = row_at(tbl, tbl_ids, tbl_rows, dim, rows[u]);
        real *a = row_at(acc, tbl_ids, tbl_rows, dim, rows[u]);
        if (w == NULL || a == NULL)
            return ORACLE_ERR_ROW;
        const real *g = coal + u * dim;
        for (int32_t d = 0; d < dim; ++d) {
            real t = rg * a[d];
            real sq = g[d] * g[d];
            real m = rc * sq;
            a[d] = t + m;
            real s = real_sqrt(reps + a[d]);
            real q = g[d] / s;
            real step = rlr * q;
            w[d] = w[d] - step;
        }
    }
    return 0;
}

/*
 * Gradient scatter with row-wise Adagrad: Eq. (2) with one accumulator per
 * embedding row instead of one per element, the accumulator growing by the
 * mean of the row's squared gradient. For each row with a coalesced
 * gradient G (dim elements):
 * m = (G_0^2 + G_1^2 + ... + G_{dim-1}^2) / dim, summed in column order
 * from zero; A = A + m; s = sqrt(eps + A); then for every d:
 * q = G_d / s; W_d = W_d - lr * q.
 * `acc` holds one value per row, stored with the same row set as the table.
 */
int oracle_scatter_rowwise_adagrad(int32_t dim, int64_t num_unique, const int64_t *rows,
                                   const real *coal, double lr, double eps,
                                   const int64_t *tbl_ids, int64_t tbl_rows, real *tbl,
                                   real *acc)
{
    if (dim <= 0 || num_unique < 0)
        return ORACLE_ERR_ARG;
    const real rlr = (real)lr, reps = (real)eps, rdim = (real)dim;
    for (int64_t u = 0; u < num_unique; ++u) {
        real *w = row_at(tbl, tbl_ids, tbl_rows, dim, rows[u]);
        real *a = row_at(acc, tbl_ids, tbl_rows, 1, rows[u]);
        if (w == NULL || a == NULL)
            return ORACLE_ERR_ROW;
        const real *g = coal + u * dim;
        real ss = 0;
        for (int32_t d = 0; d < dim; ++d) {
            real sq = g[d] * g[d];
            ss = ss + sq;
        }
        real m = ss / rdim;
        a[0] = a[0] + m;
        real s = real_sqrt(reps + a[0]);
        for (int32_t d = 0; d < dim; ++d) {
            real q = g[d] / s;
            real step = rlr * q;
            w[d] = w[d] - step;
        }
    }
    return 0;
}
