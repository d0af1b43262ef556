/*
 * Multi-threaded CPU baseline of one embedding training step -- a reported
 * baseline for the benchmark, not part of the product and not the oracle.
 *
 * It is the paper's baseline training step on the host CPU (Kwon, Lee,
 * Rhu, arXiv 2010.13100, Sec. II-B and Algorithm 1; the tuned CPU baseline
 * of Sec. V), parallelised with OpenMP over all cores:
 *
 *   forward gather-reduce   one bag per iteration of a parallel loop
 *   gradient expand         one bag per iteration
 *   stable argsort by row   LSD radix sort, 8-bit digits, per-thread
 *                           histograms and ordered per-thread scatter ranges
 *   coalesce (Algorithm 1)  the sorted array cut at segment starts into one
 *                           range per thread; each segment summed in order
 *   sparse update           SGD, or Adagrad as Eq. (2), one row per iteration
 *
 * Every output equals the single-threaded oracle's bit for bit: sums run in
 * the same order (input order within a bag; sorted, then input, order
 * within a segment) and the update takes the same separately rounded fp32
 * operations (built with -ffp-contract=off). It shares no code with the HIP
 * library or with the oracle.
 *
 * Tables are a row set: `table` holds `rows` rows of `dim` floats, and the
 * caller passes each pair's row as an index into it (`pair_row`), so a
 * benchmark can hand over only the rows a batch touches.
 *
 * Returns the number of coalesced rows (>= 0), or -1 on a bad argument,
 * -3 when memory runs out.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

int cpu_threads(void) { return omp_get_max_threads(); }

/* Stable LSD radix sort of (key, value) pairs, keys < 2^bits. */
static int radix_sort(uint32_t *key, int32_t *val, int64_t n, int bits)
{
    const size_t n1 = (size_t)(n > 0 ? n : 1);
    uint32_t *k2 = malloc(n1 * sizeof(uint32_t));
    int32_t *v2 = malloc(n1 * sizeof(int32_t));
    const int nt = omp_get_max_threads();
    int64_t *hist = calloc((size_t)nt * 256, sizeof(int64_t));
    if (!k2 || !v2 || !hist) {
        free(k2); free(v2); free(hist);
        return -3;
    }
    for (int shift = 0; shift < bits; shift += 8) {
        memset(hist, 0, (size_t)nt * 256 * sizeof(int64_t));
#pragma omp parallel num_threads(nt)
        {
            const int t = omp_get_thread_num();
            if (omp_get_num_threads() != nt) abort();
            const int64_t lo = n * t / nt, hi = n * (t + 1) / nt;
            int64_t *h = hist + (size_t)t * 256;
            for (int64_t i = lo; i < hi; ++i) h[(key[i] >> shift) & 255]++;
#pragma omp barrier
#pragma omp single
            {
                /* digit-major, thread-minor exclusive scan: thread t's items
                 * of digit d follow those of threads < t (stability) */
                int64_t run = 0;
                for (int d = 0; d < 256; ++d)
                    for (int u = 0; u < nt; ++u) {
                        const int64_t c = hist[(size_t)u * 256 + d];
                        hist[(size_t)u * 256 + d] = run;
                        run += c;
                    }
            }
            for (int64_t i = lo; i < hi; ++i) {
                const int64_t at = h[(key[i] >> shift) & 255]++;
                k2[at] = key[i];
                v2[at] = val[i];
            }
        }
        memcpy(key, k2, (size_t)n * sizeof(uint32_t));
        memcpy(val, v2, (size_t)n * sizeof(int32_t));
    }
    free(k2); free(v2); free(hist);
    return 0;
}

/*
 * One step. Inputs: num_bags bags in CSR form (bag_offsets[num_bags+1]),
 * pair_row[N] (row of each pair in `table`), grad_out[num_bags x dim].
 * Outputs: out[num_bags x dim]; coal[N x dim] and coal_rows[N] (the first U
 * entries are written: coalesced rows in ascending row order); table (and
 * acc for Adagrad) updated in place. optimizer: 0 SGD, 1 Adagrad.
 * seconds[5] (may be NULL) receives the wall time of the five phases.
 */
int64_t cpu_train_step(int32_t num_bags, const int32_t *bag_offsets, const int32_t *pair_row,
                       int32_t rows, int32_t dim, float *table, float *acc,
                       const float *grad_out, float *out, float *coal, int32_t *coal_rows,
                       int32_t optimizer, float lr, float eps, double *seconds)
{
    if (num_bags < 0 || rows < 0 || dim <= 0 || !bag_offsets || (optimizer == 1 && !acc))
        return -1;
    /* the per-thread ranges below assume every parallel region gets exactly
     * omp_get_max_threads() threads */
    omp_set_dynamic(0);
    const int64_t n = bag_offsets[num_bags];
    double t0 = omp_get_wtime(), t1;
    /* forward: each bag's rows in input order, from +0 */
#pragma omp parallel for schedule(static)
    for (int32_t g = 0; g < num_bags; ++g) {
        float *o = out + (int64_t)g * dim;
        for (int32_t d = 0; d < dim; ++d) o[d] = 0.0f;
        for (int32_t j = bag_offsets[g]; j < bag_offsets[g + 1]; ++j) {
            const float *w = table + (int64_t)pair_row[j] * dim;
            for (int32_t d = 0; d < dim; ++d) o[d] = o[d] + w[d];
        }
    }
    t1 = omp_get_wtime();
    if (seconds) seconds[0] = t1 - t0;
    t0 = t1;
    /* expand: one copy of the bag's gradient per pair */
    const size_t n1 = (size_t)(n > 0 ? n : 1);
    float *exp_grad = malloc(n1 * dim * sizeof(float));
    uint32_t *key = malloc(n1 * sizeof(uint32_t));
    int32_t *pos = malloc(n1 * sizeof(int32_t));
    if (!exp_grad || !key || !pos) {
        free(exp_grad); free(key); free(pos);
        return -3;
    }
#pragma omp parallel for schedule(static)
    for (int32_t g = 0; g < num_bags; ++g)
        for (int32_t j = bag_offsets[g]; j < bag_offsets[g + 1]; ++j)
            memcpy(exp_grad + (int64_t)j * dim, grad_out + (int64_t)g * dim,
                   (size_t)dim * sizeof(float));
    t1 = omp_get_wtime();
    if (seconds) seconds[1] = t1 - t0;
    t0 = t1;
    /* stable argsort of the pairs by row */
    int bits = 0;
    while (bits < 32 && ((int64_t)1 << bits) < rows) bits += 8;
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < n; ++j) {
        key[j] = (uint32_t)pair_row[j];
        pos[j] = (int32_t)j;
    }
    if (radix_sort(key, pos, n, bits) != 0) {
        free(exp_grad); free(key); free(pos);
        return -3;
    }
    t1 = omp_get_wtime();
    if (seconds) seconds[2] = t1 - t0;
    t0 = t1;
    /* Algorithm 1's accumulate: ranges cut at segment starts, one per
     * thread; first count each range's segments, then sum them in order */
    const int nt = omp_get_max_threads();
    int64_t *cut = malloc((size_t)(nt + 1) * sizeof(int64_t));
    int64_t *base = malloc((size_t)(nt + 1) * sizeof(int64_t));
    if (!cut || !base) {
        free(exp_grad); free(key); free(pos); free(cut); free(base);
        return -3;
    }
    for (int t = 0; t <= nt; ++t) {
        int64_t c = n * t / nt;
        while (c > 0 && c < n && key[c] == key[c - 1]) ++c;
        cut[t] = c;
    }
    for (int t = 1; t <= nt; ++t)
        if (cut[t] < cut[t - 1]) cut[t] = cut[t - 1];
#pragma omp parallel num_threads(nt)
    {
        const int t = omp_get_thread_num();
        if (omp_get_num_threads() != nt) abort();
        int64_t segs = 0;
        for (int64_t i = cut[t]; i < cut[t + 1]; ++i)
            if (i == 0 || key[i] != key[i - 1]) ++segs;
        base[t + 1] = segs;
#pragma omp barrier
#pragma omp single
        {
            base[0] = 0;
            for (int u = 1; u <= nt; ++u) base[u] += base[u - 1];
        }
        int64_t u = base[t] - 1;
        for (int64_t i = cut[t]; i < cut[t + 1]; ++i) {
            if (i == 0 || key[i] != key[i - 1]) {
                ++u;
                coal_rows[u] = (int32_t)key[i];
                float *c = coal + u * dim;
                for (int32_t d = 0; d < dim; ++d) c[d] = 0.0f;
            }
            float *c = coal + u * dim;
            const float *e = exp_grad + (int64_t)pos[i] * dim;
            for (int32_t d = 0; d < dim; ++d) c[d] = c[d] + e[d];
        }
    }
    const int64_t num_unique = base[nt];
    free(cut); free(base); free(exp_grad); free(key); free(pos);
    t1 = omp_get_wtime();
    if (seconds) seconds[3] = t1 - t0;
    t0 = t1;
    /* gradient scatter with the optimizer */
#pragma omp parallel for schedule(static)
    for (int64_t u = 0; u < num_unique; ++u) {
        float *w = table + (int64_t)coal_rows[u] * dim;
        const float *gr = coal + u * dim;
        if (optimizer == 0) {
            for (int32_t d = 0; d < dim; ++d) {
                const float s = lr * gr[d];
                w[d] = w[d] - s;
            }
        } else {
            float *a = acc + (int64_t)coal_rows[u] * dim;
            for (int32_t d = 0; d < dim; ++d) {
                const float g2 = gr[d] * gr[d];
                a[d] = a[d] + g2;
                const float s = sqrtf(eps + a[d]);
                const float q = gr[d] / s;
                const float m = lr * q;
                w[d] = w[d] - m;
            }
        }
    }
    t1 = omp_get_wtime();
    if (seconds) seconds[4] = t1 - t0;
    return num_unique;
}
