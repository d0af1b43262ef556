/*
 * tc_workload.h -- device-side fill of synthetic embedding tables.
 *
 * Input generation only; not part of the training step. Tables of tens of
 * GB are filled on the GPU with the counter-based generator SplitMix64
 * (Steele, Lea and Flood, "Fast splittable pseudorandom number generators",
 * OOPSLA 2014): element e of the concatenated table (e = global_row * dim +
 * col) takes output number e+1 of SplitMix64 started at state `seed`,
 *   z = seed + (e+1) * 0x9E3779B97F4A7C15   (mod 2^64)
 *   z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9
 *   z = (z ^ (z >> 27)) * 0x94D049BB133111EB
 *   z =  z ^ (z >> 31)
 * u = (z >> 40) * 2^-24 in [0, 1) and the value is the fp32 lo + (hi-lo)*u,
 * with hi-lo, the product and the sum each rounded to fp32.
 */
#ifndef TC_WORKLOAD_H
#define TC_WORKLOAD_H

#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Fill rows [row_begin, row_begin + num_rows) of a [* x dim] fp32 table.
 * `W` points at row 0 of the table (device). Returns 0, or -1 on a bad
 * argument, -2 if the launch failed. Asynchronous on `stream`.
 */
int tcw_fill_uniform(float *W, int64_t row_begin, int64_t num_rows, int32_t dim, uint64_t seed,
                     float lo, float hi, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* TC_WORKLOAD_H */
