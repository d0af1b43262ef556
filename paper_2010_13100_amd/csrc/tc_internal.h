// Internal helpers of libtc: error reporting, argument checks, launch shapes.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>

#include "tc.h"

namespace tc {

// Per-thread message of the last failed call.
void set_error(const char *fmt, ...);
void clear_error();

// Returns TC_ERR_HIP (with a message) if the last launch failed.
tc_status check_launch(const char *what);

constexpr int kWave = 64;          // CDNA wavefront width
constexpr int kBlock = 256;        // threads per block for the streaming kernels
constexpr int kMaxDim = 1024;

// Compute units of the current device (hipDeviceGetAttribute, cached per
// device; 256, an MI355X's count, if the query fails). Grids are sized in
// workgroups per CU from it.
int device_cus();

inline bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Lanes that share one output row: dim/4 float4 columns spread over a
// power-of-two lane group of at most one wavefront; wider rows give each lane
// several float4 chunks.
struct RowShape {
    int lanes;   // lanes per row (1..64, power of two)
    int chunks;  // float4 chunks per lane
};

inline RowShape row_shape(int dim) {
    int d4 = dim / 4;
    int lanes = 1;
    while (lanes < d4 && lanes < kWave) lanes *= 2;
    int chunks = (d4 + lanes - 1) / lanes;
    return {lanes, chunks};
}

// Grid for a grid-stride kernel over `items` work items, `per_block` per
// block, capped at `waves_per_cu` resident blocks' worth on every CU.
inline unsigned grid_for(int64_t items, int64_t per_block, int64_t cap_blocks) {
    int64_t g = (items + per_block - 1) / per_block;
    if (g < 1) g = 1;
    if (g > cap_blocks) g = cap_blocks;
    return static_cast<unsigned>(g);
}

}  // namespace tc

#define TC_REQUIRE(cond, code, ...)        \
    do {                                   \
        if (!(cond)) {                     \
            ::tc::set_error(__VA_ARGS__);  \
            return (code);                 \
        }                                  \
    } while (0)
