// Gradient scatter with an optimizer (Sec. II-B): SGD, Adagrad (Eq. 2),
// RMSprop (Eq. 1) and row-wise Adagrad.
//
// Every coalesced row u has exactly one owner: a group of LANES lanes that
// reads coal_grad[u], reads and writes W[unique_rows[u]] (and the
// accumulator row) with dwordx4 accesses. unique_rows are distinct, so no
// atomics are needed and the result does not depend on scheduling. The
// optimizer arithmetic (tc_optim.h) is separately rounded fp32.
//
// Row-wise Adagrad needs the row's sum of squares in column order. The group
// stages its squares in its own slice of LDS and every lane of the group
// then adds the whole row sequentially (broadcast 16-byte reads), so all
// lanes hold the same accumulator value without a tree reduction that would
// change the rounding.
#include "tc_optim.h"

namespace tc {
namespace {

template <int LANES, int CHUNKS, int OPT>
__global__ __launch_bounds__(kBlock) void k_sparse_update(
    float *__restrict__ W, float *__restrict__ A, int32_t dim,
    const int32_t *__restrict__ rows, const float *__restrict__ coal,
    const int32_t *__restrict__ num_unique_dev, int64_t cap, float lr, float eps, float gamma) {
    constexpr int kGroups = kWave / LANES;
    constexpr int kRowF4 = LANES * CHUNKS;  // float4 capacity of one group's row
    constexpr bool kRowwise = OPT == TC_OPT_ROWWISE_ADAGRAD;
    __shared__ float4 sq_lds[kRowwise ? kBlock / kWave : 1][kRowwise ? kWave * CHUNKS : 1];
    const int lane = threadIdx.x & (kWave - 1);
    const int sub = lane & (LANES - 1);
    const int grp = lane / LANES;
    const int64_t nu = *num_unique_dev;
    const int64_t num = nu < cap ? nu : cap;
    const int64_t wave = (int64_t(blockIdx.x) * blockDim.x + threadIdx.x) / kWave;
    const int64_t nwave = (int64_t(gridDim.x) * blockDim.x) / kWave;
    const int d4 = dim >> 2;
    const float omg = 1.0f - gamma;

    for (int64_t u0 = wave * kGroups; u0 < num; u0 += nwave * kGroups) {
        const int64_t u = u0 + grp;
        if (u >= num) continue;
        const int64_t r = rows[u];
        float *wrow = W + r * int64_t(dim);
        const float *grow = coal + u * int64_t(dim);
        if constexpr (kRowwise) {
            float4 g[CHUNKS];
            float4 *sq = &sq_lds[threadIdx.x / kWave][grp * kRowF4];
#pragma unroll
            for (int c = 0; c < CHUNKS; ++c) {
                const int col4 = sub + c * LANES;
                if (col4 >= d4) continue;
                g[c] = *reinterpret_cast<const float4 *>(grow + 4 * col4);
                sq[col4] = make_float4(g[c].x * g[c].x, g[c].y * g[c].y, g[c].z * g[c].z,
                                       g[c].w * g[c].w);
            }
            // the squares of the whole row are in LDS once this wave's stores
            // are done (one wave: its LDS operations complete in order)
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            float ss = 0.f;
            for (int k = 0; k < d4; ++k) {
                const float4 v = sq[k];
                ss = ss + v.x;
                ss = ss + v.y;
                ss = ss + v.z;
                ss = ss + v.w;
            }
            const float m = ss / float(dim);
            const float a = A[r] + m;
            const float s = sqrtf(eps + a);
            if (sub == 0) A[r] = a;
#pragma unroll
            for (int c = 0; c < CHUNKS; ++c) {
                const int col4 = sub + c * LANES;
                if (col4 >= d4) continue;
                float4 w = stream_load4(wrow + 4 * col4);
                w.x = w.x - lr * (g[c].x / s);
                w.y = w.y - lr * (g[c].y / s);
                w.z = w.z - lr * (g[c].z / s);
                w.w = w.w - lr * (g[c].w / s);
                stream_store4(wrow + 4 * col4, w);
            }
            // this row's reads of the group's LDS slice are issued before the
            // next row's stores to it (program order within the wave)
            __builtin_amdgcn_wave_barrier();
            continue;
        }
#pragma unroll
        for (int c = 0; c < CHUNKS; ++c) {
            const int col4 = sub + c * LANES;
            if (col4 >= d4) continue;
            const float4 g = *reinterpret_cast<const float4 *>(grow + 4 * col4);
            float4 w = stream_load4(wrow + 4 * col4);
            if constexpr (OPT == TC_OPT_SGD) {
                w.x = sgd_step(w.x, g.x, lr);
                w.y = sgd_step(w.y, g.y, lr);
                w.z = sgd_step(w.z, g.z, lr);
                w.w = sgd_step(w.w, g.w, lr);
            } else {
                float *arow = A + r * int64_t(dim);
                float4 a = stream_load4(arow + 4 * col4);
                if constexpr (OPT == TC_OPT_ADAGRAD) {
                    adagrad_step(w.x, a.x, g.x, lr, eps);
                    adagrad_step(w.y, a.y, g.y, lr, eps);
                    adagrad_step(w.z, a.z, g.z, lr, eps);
                    adagrad_step(w.w, a.w, g.w, lr, eps);
                } else {
                    rmsprop_step(w.x, a.x, g.x, lr, eps, gamma, omg);
                    rmsprop_step(w.y, a.y, g.y, lr, eps, gamma, omg);
                    rmsprop_step(w.z, a.z, g.z, lr, eps, gamma, omg);
                    rmsprop_step(w.w, a.w, g.w, lr, eps, gamma, omg);
                }
                stream_store4(arow + 4 * col4, a);
            }
            stream_store4(wrow + 4 * col4, w);
        }
    }
}

template <int OPT>
tc_status launch_update(float *W, float *A, int32_t dim, const int32_t *rows, const float *coal,
                        const int32_t *num_unique, int64_t cap, float lr, float eps,
                        float gamma, hipStream_t stream) {
    const RowShape s = row_shape(dim);
    const int64_t rows_per_block = (kBlock / kWave) * (kWave / s.lanes);
    const unsigned grid = grid_for(cap, rows_per_block, int64_t(device_cus()) * 8);
#define TC_UP_CASE(L, C)                                                                 \
    if (s.lanes == L && s.chunks == C) {                                                 \
        k_sparse_update<L, C, OPT><<<grid, kBlock, 0, stream>>>(                          \
            W, A, dim, rows, coal, num_unique, cap, lr, eps, gamma);                     \
        return check_launch("k_sparse_update");                                          \
    }
    TC_UP_CASE(1, 1)
    TC_UP_CASE(2, 1)
    TC_UP_CASE(4, 1)
    TC_UP_CASE(8, 1)
    TC_UP_CASE(16, 1)
    TC_UP_CASE(32, 1)
    TC_UP_CASE(64, 1)
    TC_UP_CASE(64, 2)
    TC_UP_CASE(64, 3)
    TC_UP_CASE(64, 4)
#undef TC_UP_CASE
    set_error("no update kernel for dim %d", dim);
    return TC_ERR_UNSUPPORTED;
}

}  // namespace
}  // namespace tc

using namespace tc;

extern "C" tc_status tc_sparse_update(float *W, float *opt_state, int64_t total_rows, int32_t dim,
                                      const int32_t *unique_rows, const float *coal_grad,
                                      const int32_t *num_unique, int64_t max_unique,
                                      int32_t opt_kind, float lr, float eps, float gamma,
                                      hipStream_t stream) {
    clear_error();
    TC_REQUIRE(total_rows >= 0 && max_unique >= 0, TC_ERR_INVALID_ARG,
               "tc_sparse_update: negative size");
    TC_REQUIRE(total_rows < (int64_t(1) << 31) && max_unique < (int64_t(1) << 31),
               TC_ERR_INVALID_ARG, "tc_sparse_update: sizes must be below 2^31");
    TC_REQUIRE(dim > 0 && dim % 4 == 0 && dim <= kMaxDim, TC_ERR_UNSUPPORTED,
               "tc_sparse_update: dim %d must be a multiple of 4 in [4, %d]", dim, kMaxDim);
    TC_REQUIRE(opt_kind >= TC_OPT_SGD && opt_kind <= TC_OPT_ROWWISE_ADAGRAD, TC_ERR_INVALID_ARG,
               "tc_sparse_update: unknown optimizer %d", opt_kind);
    TC_REQUIRE((opt_kind == TC_OPT_SGD) == (opt_state == nullptr), TC_ERR_INVALID_ARG,
               "tc_sparse_update: opt_state must be NULL for SGD and given otherwise");
    TC_REQUIRE(opt_kind != TC_OPT_RMSPROP || (gamma >= 0.f && gamma <= 1.f), TC_ERR_INVALID_ARG,
               "tc_sparse_update: RMSprop gamma must lie in [0, 1]");
    if (max_unique == 0) return TC_OK;
    TC_REQUIRE(W && unique_rows && coal_grad && num_unique, TC_ERR_INVALID_ARG,
               "tc_sparse_update: null pointer");
    TC_REQUIRE(aligned16(W) && aligned16(coal_grad) &&
                   (!opt_state || opt_kind == TC_OPT_ROWWISE_ADAGRAD || aligned16(opt_state)),
               TC_ERR_UNSUPPORTED, "tc_sparse_update: float pointers must be 16-byte aligned");
    switch (opt_kind) {
    case TC_OPT_SGD:
        return launch_update<TC_OPT_SGD>(W, nullptr, dim, unique_rows, coal_grad, num_unique,
                                         max_unique, lr, eps, gamma, stream);
    case TC_OPT_ADAGRAD:
        return launch_update<TC_OPT_ADAGRAD>(W, opt_state, dim, unique_rows, coal_grad,
                                             num_unique, max_unique, lr, eps, gamma, stream);
    case TC_OPT_RMSPROP:
        return launch_update<TC_OPT_RMSPROP>(W, opt_state, dim, unique_rows, coal_grad,
                                             num_unique, max_unique, lr, eps, gamma, stream);
    default:
        return launch_update<TC_OPT_ROWWISE_ADAGRAD>(W, opt_state, dim, unique_rows, coal_grad,
                                                     num_unique, max_unique, lr, eps, gamma,
                                                     stream);
    }
}
