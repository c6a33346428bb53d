// Reference streaming kernels for measurement: the rates a plain read and a
// plain copy reach on the device, against which the softmax and top-k
// kernels' bandwidth is judged (they compute nothing of the method).
// Each wavefront streams one contiguous span of 16-byte vectors, RF_U per
// lane in flight, with non-temporal hints (the data are touched once): on
// this chip long sequential streams read faster than a grid-stride
// interleave over the whole buffer.
#include "md.hpp"
#include "kernels.h"

namespace osm {

constexpr int RF_BLOCK = 256, RF_U = 8;

// span of wavefront w of nw over n vectors, in whole steps of 64 * RF_U
__device__ __forceinline__ void rf_span(int64_t n, int64_t nw, int64_t w, int64_t* b,
                                        int64_t* e) {
    constexpr int64_t STEP = 64 * RF_U;
    const int64_t steps = (n + STEP - 1) / STEP;
    const int64_t per = (steps + nw - 1) / nw;
    *b = w * per * STEP;
    *e = (w + 1) * per * STEP < n ? (w + 1) * per * STEP : n;
}

// Reads every vector; the sum is stored only if it equals a value it never
// takes on the benchmark's data, so the loads cannot be dropped.
__global__ __launch_bounds__(RF_BLOCK) void ref_read(const u32x4* __restrict__ x, int64_t n,
                                                    float* __restrict__ sink) {
    const int lane = threadIdx.x & 63;
    int64_t b, e;
    rf_span(n, (int64_t)gridDim.x * (RF_BLOCK / 64),
            (int64_t)blockIdx.x * (RF_BLOCK / 64) + (threadIdx.x >> 6), &b, &e);
    float acc = 0.0f;
    for (int64_t i = b + lane; i < e; i += 64 * RF_U) {
        u32x4 q[RF_U];
#pragma unroll
        for (int u = 0; u < RF_U; ++u) {
            const int64_t j = i + u * 64;
            q[u] = j < e ? __builtin_nontemporal_load(x + j) : u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int u = 0; u < RF_U; ++u) acc += __uint_as_float(q[u].x) + __uint_as_float(q[u].w);
    }
    if (acc == 1.2345678e-30f) sink[threadIdx.x] = acc;
}

__global__ __launch_bounds__(RF_BLOCK) void ref_copy(const u32x4* __restrict__ x,
                                                    u32x4* __restrict__ y, int64_t n) {
    const int lane = threadIdx.x & 63;
    int64_t b, e;
    rf_span(n, (int64_t)gridDim.x * (RF_BLOCK / 64),
            (int64_t)blockIdx.x * (RF_BLOCK / 64) + (threadIdx.x >> 6), &b, &e);
    for (int64_t i = b + lane; i < e; i += 64 * RF_U) {
        u32x4 q[RF_U];
#pragma unroll
        for (int u = 0; u < RF_U; ++u) {
            const int64_t j = i + u * 64;
            if (j < e) q[u] = __builtin_nontemporal_load(x + j);
        }
#pragma unroll
        for (int u = 0; u < RF_U; ++u) {
            const int64_t j = i + u * 64;
            if (j < e) __builtin_nontemporal_store(q[u], y + j);
        }
    }
}

hipError_t launch_ref_stream(int op, const void* x, void* y, int64_t vecs, int cus,
                             hipStream_t st) {
    // one workgroup of four wavefronts per CU (the fastest read shape in a
    // sweep of 4 to 64 wavefronts per CU and 4 to 16 vectors in flight per
    // lane), never more wavefronts than steps
    int64_t waves = (vecs + 64 * RF_U - 1) / (64 * RF_U);
    if (waves > 4 * (int64_t)cus) waves = 4 * (int64_t)cus;
    if (waves < 1) waves = 1;
    const int64_t g = (waves + RF_BLOCK / 64 - 1) / (RF_BLOCK / 64);
    if (op == 0)
        hipLaunchKernelGGL(ref_read, dim3((unsigned)g), dim3(RF_BLOCK), 0, st,
                           static_cast<const u32x4*>(x), vecs, static_cast<float*>(y));
    else
        hipLaunchKernelGGL(ref_copy, dim3((unsigned)g), dim3(RF_BLOCK), 0, st,
                           static_cast<const u32x4*>(x), static_cast<u32x4*>(y), vecs);
    return hipGetLastError();
}

}  // namespace osm
