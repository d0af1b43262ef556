// Device-side fill of synthetic tables with SplitMix64 (input generation).
#include <hip/hip_runtime.h>

#include <cstdint>

#include "tc_workload.h"

namespace {

__device__ __forceinline__ uint64_t splitmix64_output(uint64_t seed, uint64_t counter) {
    uint64_t z = seed + counter * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

__global__ __launch_bounds__(256) void k_fill_uniform(float *__restrict__ W, int64_t first,
                                                      int64_t count, uint64_t seed, float lo,
                                                      float span) {
    const int64_t stride = int64_t(gridDim.x) * blockDim.x;
    for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < count; i += stride) {
        const int64_t e = first + i;
        const uint64_t z = splitmix64_output(seed, uint64_t(e) + 1u);
        const float u = float(uint32_t(z >> 40)) * 5.9604644775390625e-08f;  // 2^-24
        const float prod = span * u;
        W[e] = lo + prod;
    }
}

}  // namespace

extern "C" int tcw_fill_uniform(float *W, int64_t row_begin, int64_t num_rows, int32_t dim,
                                uint64_t seed, float lo, float hi, hipStream_t stream) {
    if (row_begin < 0 || num_rows < 0 || dim <= 0) return -1;
    if (num_rows == 0) return 0;
    if (!W) return -1;
    const int64_t count = num_rows * int64_t(dim);
    int64_t blocks = (count + 255) / 256;
    if (blocks > 256 * 64) blocks = 256 * 64;
    const float span = hi - lo;
    k_fill_uniform<<<unsigned(blocks), 256, 0, stream>>>(W, row_begin * int64_t(dim), count, seed,
                                                         lo, span);
    return hipGetLastError() == hipSuccess ? 0 : -2;
}
