// Row-resident online softmax for gfx950: the online normalizer (Alg. 3)
// with the row held in registers between its two uses, so every element is
// loaded once and stored once (the paper's online mode loads it twice).
//
// One row per workgroup of BLOCK threads.  Lane t holds R 16-byte vectors
// of the row (vectors t, t + BLOCK, ..., all loaded before any is used, with
// non-temporal hints), plus at most one scalar head and one scalar tail
// element where the row does not start or end on a 16-byte boundary.  When y
// is not congruent with x modulo 16 bytes, the outputs of a vector are
// stored one by one.
//
//   1. the lane's pair: its maximum m_t, then d_t = sum 2^{x log2e - m_t log2e}
//      (Theorem 1's closed form over the lane's elements);
//   2. the row's pair: Eq. 4 over the lanes (wavefront butterflies, then a
//      fixed-order merge of the wavefronts' pairs through LDS);
//   3. y = 2^{x log2e - s} / d from the registers, non-temporal stores.
#include "md.hpp"
#include "kernels.h"

namespace osm {

// Largest of three binary32 values in one instruction (no quieting of
// signalling NaNs: a row holding NaN gives NaN outputs through d anyway).
__device__ __forceinline__ float rmax3(float a, float b, float c) {
    float r;
    asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
    return r;
}

template <typename T>
__device__ __forceinline__ void widen_vec(u32x4 q, float (&x)[Vec<T>::N]) {
    if constexpr (Vec<T>::N == 4) {
        x[0] = __uint_as_float(q.x);
        x[1] = __uint_as_float(q.y);
        x[2] = __uint_as_float(q.z);
        x[3] = __uint_as_float(q.w);
    } else {
        x[0] = bf16_lo(q.x); x[1] = bf16_hi(q.x);
        x[2] = bf16_lo(q.y); x[3] = bf16_hi(q.y);
        x[4] = bf16_lo(q.z); x[5] = bf16_hi(q.z);
        x[6] = bf16_lo(q.w); x[7] = bf16_hi(q.w);
    }
}

// Keep `q` in its registers as-is and make the compiler forget what it
// derived from it, so that each phase widens the packed elements again
// instead of keeping a widened copy live across the phases (for bfloat16
// that copy would need twice the registers).
__device__ __forceinline__ void opaque(u32x4& q) { asm volatile("" : "+v"(q)); }

template <typename T, int BLOCK, int R, bool YVEC>
__global__ __launch_bounds__(BLOCK) void softmax_resident(const T* __restrict__ x,
                                                         T* __restrict__ y, int64_t N,
                                                         int64_t V) {
    constexpr int E = Vec<T>::N;
    __shared__ typename Team<BLOCK>::Smem sm;
    const int t = threadIdx.x;
    const float ninf = -__builtin_inff();
    for (int64_t row = blockIdx.x; row < N; row += gridDim.x) {
        const T* xr = x + row * V;
        T* yr = y + row * V;
        int64_t head = ((16 - (int64_t)(((uintptr_t)xr) & 15)) & 15) / (int64_t)sizeof(T);
        if (head > V) head = V;
        const int64_t nvec = (V - head) / E;
        const int64_t tail0 = head + nvec * E;
        const u32x4* vb = reinterpret_cast<const u32x4*>(xr + head);
        // all loads first; lanes past the row load vector 0 and mask it
        u32x4 buf[R];
        bool ok[R];
#pragma unroll
        for (int i = 0; i < R; ++i) {
            const int64_t v = t + (int64_t)i * BLOCK;
            ok[i] = v < nvec;
            buf[i] = nvec > 0 ? __builtin_nontemporal_load(vb + (ok[i] ? v : 0)) : u32x4{0, 0, 0, 0};
        }
        const bool hok = t < head, tok = tail0 + t < V;
        const float hx = hok ? load1(xr + t) : ninf;
        const float tx = tok ? load1(xr + tail0 + t) : ninf;
        // 1. the lane's pair: its maximum, then the sum relative to it
        float m = rmax3(hx, tx, ninf);
#pragma unroll
        for (int i = 0; i < R; ++i) {
            float xv[E];
            widen_vec<T>(buf[i], xv);
#pragma unroll
            for (int k = 0; k < E; k += 2)
                m = rmax3(m, ok[i] ? xv[k] : ninf, ok[i] ? xv[k + 1] : ninf);
        }
        float s = m * kLog2e;
        if (!(s > kEmptyS)) s = kEmptyS;  // lane without elements (or only -inf)
        float d = exp2_hw(__builtin_fmaf(hx, kLog2e, -s)) + exp2_hw(__builtin_fmaf(tx, kLog2e, -s));
#pragma unroll
        for (int i = 0; i < R; ++i) {
            opaque(buf[i]);
            if (ok[i]) {
                float xv[E];
                widen_vec<T>(buf[i], xv);
#pragma unroll
                for (int k = 0; k < E; ++k) d += exp2_hw(__builtin_fmaf(xv[k], kLog2e, -s));
            }
        }
        // 2. the row's pair (every thread takes part)
        const MD md = Team<BLOCK>::merge(MD{s, d}, sm);
        const float S = md.s, rd = 1.0f / md.d;
        // 3. outputs from the registers
        T* yv = yr + head;
#pragma unroll
        for (int i = 0; i < R; ++i) {
            opaque(buf[i]);
            if (ok[i]) {
                Vec<T> o;
                widen_vec<T>(buf[i], o.v);
                out_vals(o.v, S, rd);
                T* dst = yv + (t + (int64_t)i * BLOCK) * E;
                if constexpr (YVEC) {
                    o.store_nt(dst);
                } else {
#pragma unroll
                    for (int k = 0; k < E; ++k) store1(dst + k, o.v[k]);
                }
            }
        }
        if (hok) store1(yr + t, out_elem(hx, S, rd));
        if (tok) store1(yr + tail0 + t, out_elem(tx, S, rd));
    }
}

namespace {

template <typename T, int BLOCK, int R>
hipError_t launch_res_t(const void* x, void* y, int64_t N, int64_t V, bool vec, hipStream_t st) {
    const unsigned grid = (unsigned)(N < (1ll << 30) ? N : (1ll << 30));
    if (vec)
        hipLaunchKernelGGL((softmax_resident<T, BLOCK, R, true>), dim3(grid), dim3(BLOCK), 0, st,
                           (const T*)x, (T*)y, N, V);
    else
        hipLaunchKernelGGL((softmax_resident<T, BLOCK, R, false>), dim3(grid), dim3(BLOCK), 0, st,
                           (const T*)x, (T*)y, N, V);
    return hipGetLastError();
}

template <typename T>
hipError_t launch_res_d(const void* x, void* y, int64_t N, int64_t V, int block, int r, bool vec,
                        hipStream_t st) {
    if (block == 256 && r == 4) return launch_res_t<T, 256, 4>(x, y, N, V, vec, st);
    if (block == 256 && r == 8) return launch_res_t<T, 256, 8>(x, y, N, V, vec, st);
    if (block == 256 && r == 16) return launch_res_t<T, 256, 16>(x, y, N, V, vec, st);
    if (block == 512 && r == 16) return launch_res_t<T, 512, 16>(x, y, N, V, vec, st);
    if (block == 1024 && r == 16) return launch_res_t<T, 1024, 16>(x, y, N, V, vec, st);
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_softmax_resident(const void* x, void* y, int64_t N, int64_t V, int dtype,
                                   int block, int r, bool vec, hipStream_t st) {
    if (dtype == 0) return launch_res_d<float>(x, y, N, V, block, r, vec, st);
    return launch_res_d<bf16_t>(x, y, N, V, block, r, vec, st);
}

}  // namespace osm
