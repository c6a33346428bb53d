// Row-wise softmax kernels for gfx950: naive (Alg. 1), safe (Alg. 2) and
// online (Alg. 3) normalizer calculation, each doing exactly the paper's
// passes over global memory.
//
//   naive : pass 1 d = sum 2^{x log2e};            pass 2 y      (2 loads, 1 store)
//   safe  : pass 1 m = max x; pass 2 d = sum ...;  pass 3 y      (3 loads, 1 store)
//   online: pass 1 (s, d) by the merge of Eq. 4;   pass 2 y      (2 loads, 1 store)
//
// Work decomposition ("team" = the lanes that share one row):
//   * TEAM in {4, 8, 16, 32}: several rows per wavefront, reduced with
//     quad permutations / swizzles inside the lane group (short rows);
//   * TEAM == 64: one row per wavefront;
//   * TEAM in {128 .. 1024}: one row per workgroup, wavefront butterflies and
//     then a fixed-order merge of the per-wavefront pairs through LDS;
//   * split-V: several workgroups per row; pass 1 of each chunk writes a
//     partial pair to a scratch array, and the output kernel merges the
//     row's partials in a fixed order before its pass over the chunk.  The
//     kernel boundary is the device-wide barrier between the passes.
//
// Every row is a contiguous run of V elements; row offsets are 64-bit.  The
// body of a row's range is read as 16-byte vectors (global_load_dwordx4),
// with scalar head and tail elements where the range does not start or end
// on a 16-byte boundary.  Lane t of a team takes vectors t, t + TEAM, ...,
// so each wavefront instruction touches 1 KiB of consecutive memory.
#include "md.hpp"
#include "kernels.h"

// Load cache policy per pass: a pass whose loads are the last use of the
// data (the output pass) reads with non-temporal hints; earlier passes use
// ordinary loads so their lines can serve the re-read.
#ifndef OSM_NT_FIRST
#define OSM_NT_FIRST 0
#endif
#ifndef OSM_NT_LAST
#define OSM_NT_LAST 1
#endif

namespace osm {

enum { NAIVE = 0, SAFE = 1, ONLINE = 2 };

template <typename T, bool NT>
__device__ __forceinline__ Vec<T> vload(const T* p) {
    if constexpr (NT) return Vec<T>::load_nt(p);
    else return Vec<T>::load(p);
}

// The part of a row a team works on, split into scalar head, aligned vector
// body and scalar tail.
template <typename T>
struct Range {
    const T* xb;  // first element of the range in x
    T* yb;        // same element in y (may be null for read-only passes)
    int64_t n;    // elements in the range
    int64_t head; // scalar elements before the first aligned vector
    int64_t nvec; // aligned 16-byte vectors
    int64_t tail0;// first scalar element after the vectors

    __device__ __forceinline__ Range(const T* x, T* y, int64_t lo, int64_t hi, bool vec) {
        constexpr int E = Vec<T>::N;
        xb = x + lo;
        yb = y ? y + lo : nullptr;
        n = hi > lo ? hi - lo : 0;
        if (vec) {
            int64_t mis = (int64_t)(((uintptr_t)xb) & 15);
            head = ((16 - mis) & 15) / (int64_t)sizeof(T);
            if (head > n) head = n;
            nvec = (n - head) / E;
        } else {
            head = n;
            nvec = 0;
        }
        tail0 = head + nvec * E;
    }
};

// ------------------------------------------------------------ per-lane folds
// Online pass 1 over the lane's share of a range: U independent pairs (one
// per unrolled load) keep U loads in flight and shorten the dependency chain.
template <typename T, int TEAM, int U, bool NT = OSM_NT_FIRST>
__device__ __forceinline__ MD lane_md(const Range<T>& r, int t) {
    constexpr int E = Vec<T>::N;
    MD st[U];
#pragma unroll
    for (int u = 0; u < U; ++u) st[u] = md_empty();
    const T* vb = r.xb + r.head;
    int64_t v = t;
    for (; v + (int64_t)(U - 1) * TEAM < r.nvec; v += (int64_t)U * TEAM) {
        Vec<T> buf[U];
#pragma unroll
        for (int u = 0; u < U; ++u) buf[u] = vload<T, NT>(vb + (v + (int64_t)u * TEAM) * E);
#pragma unroll
        for (int u = 0; u < U; ++u) st[u] = md_fold_lazy(st[u], buf[u].v, vec_max(buf[u].v));
    }
    for (; v < r.nvec; v += TEAM) {
        Vec<T> b = vload<T, NT>(vb + v * E);
        st[0] = md_fold_lazy(st[0], b.v, vec_max(b.v));
    }
    for (int64_t i = t; i < r.head; i += TEAM) st[0] = md_fold1(st[0], load1(r.xb + i));
    for (int64_t i = r.tail0 + t; i < r.n; i += TEAM) st[0] = md_fold1(st[0], load1(r.xb + i));
    MD acc = st[0];
#pragma unroll
    for (int u = 1; u < U; ++u) acc = md_merge(acc, st[u]);
    return acc;
}

template <int N>
__device__ __forceinline__ float vmax(float m, const float (&x)[N]) {
#pragma unroll
    for (int i = 0; i < N; ++i) m = fmaxf(m, x[i]);
    return m;
}

// Safe pass 1: the maximum of the lane's share.
template <typename T, int TEAM, int U, bool NT = OSM_NT_FIRST>
__device__ __forceinline__ float lane_max(const Range<T>& r, int t) {
    constexpr int E = Vec<T>::N;
    float m[U];
#pragma unroll
    for (int u = 0; u < U; ++u) m[u] = -__builtin_inff();
    const T* vb = r.xb + r.head;
    int64_t v = t;
    for (; v + (int64_t)(U - 1) * TEAM < r.nvec; v += (int64_t)U * TEAM) {
        Vec<T> buf[U];
#pragma unroll
        for (int u = 0; u < U; ++u) buf[u] = vload<T, NT>(vb + (v + (int64_t)u * TEAM) * E);
#pragma unroll
        for (int u = 0; u < U; ++u) m[u] = vmax(m[u], buf[u].v);
    }
    for (; v < r.nvec; v += TEAM) m[0] = vmax(m[0], vload<T, NT>(vb + v * E).v);
    for (int64_t i = t; i < r.head; i += TEAM) m[0] = fmaxf(m[0], load1(r.xb + i));
    for (int64_t i = r.tail0 + t; i < r.n; i += TEAM) m[0] = fmaxf(m[0], load1(r.xb + i));
    float acc = m[0];
#pragma unroll
    for (int u = 1; u < U; ++u) acc = fmaxf(acc, m[u]);
    return acc;
}

template <int N>
__device__ __forceinline__ float vsum_exp(float a, const float (&x)[N], float S) {
#pragma unroll
    for (int i = 0; i < N; ++i) a += exp2_hw(__builtin_fmaf(x[i], kLog2e, -S));
    return a;
}

// Sum of 2^{x log2e - S} over the lane's share (naive pass 1 with S = 0,
// safe pass 2 with S = max * log2e).
template <typename T, int TEAM, int U, bool NT = OSM_NT_FIRST>
__device__ __forceinline__ float lane_sum(const Range<T>& r, int t, float S) {
    constexpr int E = Vec<T>::N;
    float a[U];
#pragma unroll
    for (int u = 0; u < U; ++u) a[u] = 0.0f;
    const T* vb = r.xb + r.head;
    int64_t v = t;
    for (; v + (int64_t)(U - 1) * TEAM < r.nvec; v += (int64_t)U * TEAM) {
        Vec<T> buf[U];
#pragma unroll
        for (int u = 0; u < U; ++u) buf[u] = vload<T, NT>(vb + (v + (int64_t)u * TEAM) * E);
#pragma unroll
        for (int u = 0; u < U; ++u) a[u] = vsum_exp(a[u], buf[u].v, S);
    }
    for (; v < r.nvec; v += TEAM) a[0] = vsum_exp(a[0], vload<T, NT>(vb + v * E).v, S);
    for (int64_t i = t; i < r.head; i += TEAM)
        a[0] += exp2_hw(__builtin_fmaf(load1(r.xb + i), kLog2e, -S));
    for (int64_t i = r.tail0 + t; i < r.n; i += TEAM)
        a[0] += exp2_hw(__builtin_fmaf(load1(r.xb + i), kLog2e, -S));
    float acc = a[0];
#pragma unroll
    for (int u = 1; u < U; ++u) acc += a[u];
    return acc;
}

// Output pass: y = 2^{x log2e - S} * (1/d) (subnormal results included, see
// out_vals), stored with non-temporal hints so that the written rows do not
// evict input rows still waiting for this pass.
template <typename T, int TEAM, int U, bool NT = OSM_NT_LAST>
__device__ __forceinline__ void lane_out(const Range<T>& r, int t, float S, float rd) {
    constexpr int E = Vec<T>::N;
    const T* vb = r.xb + r.head;
    T* yb = r.yb + r.head;
    int64_t v = t;
    for (; v + (int64_t)(U - 1) * TEAM < r.nvec; v += (int64_t)U * TEAM) {
        Vec<T> buf[U];
#pragma unroll
        for (int u = 0; u < U; ++u) buf[u] = vload<T, NT>(vb + (v + (int64_t)u * TEAM) * E);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            out_vals(buf[u].v, S, rd);
            buf[u].store_nt(yb + (v + (int64_t)u * TEAM) * E);
        }
    }
    for (; v < r.nvec; v += TEAM) {
        Vec<T> b = vload<T, NT>(vb + v * E);
        out_vals(b.v, S, rd);
        b.store_nt(yb + v * E);
    }
    for (int64_t i = t; i < r.head; i += TEAM) store1(r.yb + i, out_elem(load1(r.xb + i), S, rd));
    for (int64_t i = r.tail0 + t; i < r.n; i += TEAM)
        store1(r.yb + i, out_elem(load1(r.xb + i), S, rd));
}

// --------------------------------------------------------------- row kernels
template <typename T, int MODE, int TEAM, int BLOCK, int U, bool VEC>
__global__ __launch_bounds__(BLOCK) void softmax_rows(const T* __restrict__ x, T* __restrict__ y,
                                                     int64_t N, int64_t V) {
    static_assert(TEAM <= 64 || TEAM == BLOCK, "multi-wave teams span the workgroup");
    constexpr int ROWS = BLOCK / TEAM;
    __shared__ typename Team<TEAM>::Smem sm;
    const int t = threadIdx.x % TEAM;
    for (int64_t row0 = (int64_t)blockIdx.x * ROWS; row0 < N; row0 += (int64_t)gridDim.x * ROWS) {
        const int64_t row = row0 + threadIdx.x / TEAM;
        if constexpr (TEAM <= 64) {
            if (row >= N) return;  // whole lane groups leave together
        }
        Range<T> r(x + row * V, y + row * V, 0, V, VEC);
        float S, rd;
        if constexpr (MODE == ONLINE) {
            MD md = Team<TEAM>::merge(lane_md<T, TEAM, U>(r, t), sm);
            S = md.s;
            rd = 1.0f / md.d;
        } else if constexpr (MODE == SAFE) {
            float m = Team<TEAM>::template reduce<true>(lane_max<T, TEAM, U>(r, t), sm);
            S = m * kLog2e;
            float d = Team<TEAM>::template reduce<false>(lane_sum<T, TEAM, U>(r, t, S), sm);
            rd = 1.0f / d;
        } else {
            S = 0.0f;
            float d = Team<TEAM>::template reduce<false>(lane_sum<T, TEAM, U>(r, t, 0.0f), sm);
            rd = 1.0f / d;
        }
        lane_out<T, TEAM, U>(r, t, S, rd);
    }
}

// ------------------------------------------------------------ split-V kernels
// Chunk c of a row covers [c * chunk, min(V, (c + 1) * chunk)); chunk is a
// multiple of the 16-byte vector width, so when rows start aligned every
// chunk does too.  Block b handles row b / S, chunk b % S.
constexpr int SPLIT_BLOCK = 256;
#ifndef OSM_SPLIT_U
#define OSM_SPLIT_U 2
#endif
constexpr int SPLIT_U = OSM_SPLIT_U;

__device__ __forceinline__ void chunk_bounds(int64_t c, int64_t chunk, int64_t V, int64_t& lo,
                                             int64_t& hi) {
    lo = c * chunk;
    hi = lo + chunk;
    if (lo > V) lo = V;
    if (hi > V) hi = V;
}

// Pass 1 of a chunk.  online: partial pair; safe: partial max; naive: partial
// sum of 2^{x log2e}.  Partials are float2 (s, d) / (max, -) / (sum, -).
template <typename T, int MODE, bool VEC>
__global__ __launch_bounds__(SPLIT_BLOCK) void split_pass1(const T* __restrict__ x,
                                                          float2* __restrict__ part, int64_t V,
                                                          int64_t S, int64_t chunk) {
    using TM = Team<SPLIT_BLOCK>;
    __shared__ TM::Smem sm;
    const int64_t b = blockIdx.x;
    const int64_t row = b / S, c = b % S;
    int64_t lo, hi;
    chunk_bounds(c, chunk, V, lo, hi);
    Range<T> r(x + row * V, nullptr, lo, hi, VEC);
    float2 out;
    if constexpr (MODE == ONLINE) {
        MD md = TM::merge(lane_md<T, SPLIT_BLOCK, SPLIT_U>(r, threadIdx.x), sm);
        out = make_float2(md.s, md.d);
    } else if constexpr (MODE == SAFE) {
        out = make_float2(TM::reduce<true>(lane_max<T, SPLIT_BLOCK, SPLIT_U>(r, threadIdx.x), sm),
                          0.0f);
    } else {
        out = make_float2(
            TM::reduce<false>(lane_sum<T, SPLIT_BLOCK, SPLIT_U>(r, threadIdx.x, 0.0f), sm), 0.0f);
    }
    if (threadIdx.x == 0) part[b] = out;
}

// Merge of a row's S partials, identical in every block of the row: thread i
// folds partials i, i + BLOCK, ... in order, then the fixed reduction tree.
template <int WHAT>  // 0: pair merge, 1: max of .x, 2: sum of .x, 3: sum of .y
__device__ __forceinline__ float2 merge_partials(const float2* __restrict__ p, int64_t S,
                                                 Team<SPLIT_BLOCK>::Smem& sm) {
    using TM = Team<SPLIT_BLOCK>;
    if constexpr (WHAT == 0) {
        MD a = md_empty();
        for (int64_t i = threadIdx.x; i < S; i += SPLIT_BLOCK) {
            float2 q = p[i];
            a = md_merge(a, MD{q.x, q.y});
        }
        MD r = TM::merge(a, sm);
        return make_float2(r.s, r.d);
    } else if constexpr (WHAT == 1) {
        float a = -__builtin_inff();
        for (int64_t i = threadIdx.x; i < S; i += SPLIT_BLOCK) a = fmaxf(a, p[i].x);
        return make_float2(TM::reduce<true>(a, sm), 0.0f);
    } else {
        float a = 0.0f;
        for (int64_t i = threadIdx.x; i < S; i += SPLIT_BLOCK) a += (WHAT == 2 ? p[i].x : p[i].y);
        return make_float2(TM::reduce<false>(a, sm), 0.0f);
    }
}

// Safe pass 2 of a chunk: the row maximum from the partials, then the partial
// sum of 2^{x log2e - S}, stored in .y of the block's own partial.
template <typename T, bool VEC>
__global__ __launch_bounds__(SPLIT_BLOCK) void split_safe_pass2(const T* __restrict__ x,
                                                               float2* __restrict__ part,
                                                               int64_t V, int64_t S,
                                                               int64_t chunk) {
    using TM = Team<SPLIT_BLOCK>;
    __shared__ TM::Smem sm;
    const int64_t b = blockIdx.x;
    const int64_t row = b / S, c = b % S;
    const float m = merge_partials<1>(part + row * S, S, sm).x;
    const float Sx = m * kLog2e;
    int64_t lo, hi;
    chunk_bounds(c, chunk, V, lo, hi);
    Range<T> r(x + row * V, nullptr, lo, hi, VEC);
    float d = TM::reduce<false>(lane_sum<T, SPLIT_BLOCK, SPLIT_U>(r, threadIdx.x, Sx), sm);
    // the sum goes to .y, which no block of this kernel reads, while .x (the
    // maxima every block of the row reads) stays untouched
    if (threadIdx.x == 0) part[b].y = d;
}

// Output pass of a chunk after merging the row's partials.
template <typename T, int MODE, bool VEC>
__global__ __launch_bounds__(SPLIT_BLOCK) void split_out(const T* __restrict__ x,
                                                        T* __restrict__ y,
                                                        const float2* __restrict__ part,
                                                        int64_t V, int64_t S, int64_t chunk) {
    using TM = Team<SPLIT_BLOCK>;
    __shared__ TM::Smem sm;
    const int64_t b = blockIdx.x;
    const int64_t row = b / S, c = b % S;
    const float2* pr = part + row * S;
    float Sx, rd;
    if constexpr (MODE == ONLINE) {
        float2 md = merge_partials<0>(pr, S, sm);
        Sx = md.x;
        rd = 1.0f / md.y;
    } else if constexpr (MODE == SAFE) {
        Sx = merge_partials<1>(pr, S, sm).x * kLog2e;
        rd = 1.0f / merge_partials<3>(pr, S, sm).x;
    } else {
        Sx = 0.0f;
        rd = 1.0f / merge_partials<2>(pr, S, sm).x;
    }
    int64_t lo, hi;
    chunk_bounds(c, chunk, V, lo, hi);
    Range<T> r(x + row * V, y + row * V, lo, hi, VEC);
    lane_out<T, SPLIT_BLOCK, SPLIT_U>(r, threadIdx.x, Sx, rd);
}

// ------------------------------------------------------------------ launchers
namespace {

template <typename T, int MODE, int TEAM, int BLOCK, int U, bool VEC>
hipError_t launch_rows_t(const void* x, void* y, int64_t N, int64_t V, hipStream_t st) {
    constexpr int ROWS = BLOCK / TEAM;
    int64_t blocks = (N + ROWS - 1) / ROWS;
    if (blocks > (1 << 30)) blocks = 1 << 30;
    hipLaunchKernelGGL((softmax_rows<T, MODE, TEAM, BLOCK, U, VEC>), dim3((unsigned)blocks),
                       dim3(BLOCK), 0, st, (const T*)x, (T*)y, N, V);
    return hipGetLastError();
}

template <typename T, int MODE, bool VEC>
hipError_t launch_rows_mv(const void* x, void* y, int64_t N, int64_t V, int team,
                          hipStream_t st) {
    switch (team) {
        case 4: return launch_rows_t<T, MODE, 4, 256, 1, VEC>(x, y, N, V, st);
        case 8: return launch_rows_t<T, MODE, 8, 256, 1, VEC>(x, y, N, V, st);
        case 16: return launch_rows_t<T, MODE, 16, 256, 2, VEC>(x, y, N, V, st);
        case 32: return launch_rows_t<T, MODE, 32, 256, 2, VEC>(x, y, N, V, st);
        case 64: return launch_rows_t<T, MODE, 64, 256, 2, VEC>(x, y, N, V, st);
        case 128: return launch_rows_t<T, MODE, 128, 128, 4, VEC>(x, y, N, V, st);
        case 256: return launch_rows_t<T, MODE, 256, 256, 4, VEC>(x, y, N, V, st);
        case 512: return launch_rows_t<T, MODE, 512, 512, 4, VEC>(x, y, N, V, st);
        case 1024: return launch_rows_t<T, MODE, 1024, 1024, 2, VEC>(x, y, N, V, st);
        default: return hipErrorInvalidValue;
    }
}

template <typename T, int MODE>
hipError_t launch_rows_m(const void* x, void* y, int64_t N, int64_t V, int team, bool vec,
                         hipStream_t st) {
    return vec ? launch_rows_mv<T, MODE, true>(x, y, N, V, team, st)
               : launch_rows_mv<T, MODE, false>(x, y, N, V, team, st);
}

template <typename T>
hipError_t launch_rows_d(const void* x, void* y, int64_t N, int64_t V, int mode, int team,
                         bool vec, hipStream_t st) {
    switch (mode) {
        case NAIVE: return launch_rows_m<T, NAIVE>(x, y, N, V, team, vec, st);
        case SAFE: return launch_rows_m<T, SAFE>(x, y, N, V, team, vec, st);
        case ONLINE: return launch_rows_m<T, ONLINE>(x, y, N, V, team, vec, st);
        default: return hipErrorInvalidValue;
    }
}

template <typename T, int MODE, bool VEC>
hipError_t launch_split_t(const void* x, void* y, float2* part, int64_t N, int64_t V, int64_t S,
                          int64_t chunk, hipStream_t st) {
    const unsigned blocks = (unsigned)(N * S);
    hipLaunchKernelGGL((split_pass1<T, MODE, VEC>), dim3(blocks), dim3(SPLIT_BLOCK), 0, st,
                       (const T*)x, part, V, S, chunk);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if constexpr (MODE == SAFE) {
        hipLaunchKernelGGL((split_safe_pass2<T, VEC>), dim3(blocks), dim3(SPLIT_BLOCK), 0, st,
                           (const T*)x, part, V, S, chunk);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL((split_out<T, MODE, VEC>), dim3(blocks), dim3(SPLIT_BLOCK), 0, st,
                       (const T*)x, (T*)y, (const float2*)part, V, S, chunk);
    return hipGetLastError();
}

template <typename T, bool VEC>
hipError_t launch_split_v(const void* x, void* y, float2* part, int64_t N, int64_t V, int mode,
                          int64_t S, int64_t chunk, hipStream_t st) {
    switch (mode) {
        case NAIVE: return launch_split_t<T, NAIVE, VEC>(x, y, part, N, V, S, chunk, st);
        case SAFE: return launch_split_t<T, SAFE, VEC>(x, y, part, N, V, S, chunk, st);
        case ONLINE: return launch_split_t<T, ONLINE, VEC>(x, y, part, N, V, S, chunk, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_softmax_rows(const void* x, void* y, int64_t N, int64_t V, int dtype, int mode,
                               int team, bool vec, hipStream_t st) {
    if (dtype == 0) return launch_rows_d<float>(x, y, N, V, mode, team, vec, st);
    return launch_rows_d<bf16_t>(x, y, N, V, mode, team, vec, st);
}

hipError_t launch_softmax_split(const void* x, void* y, void* scratch, int64_t N, int64_t V,
                                int dtype, int mode, int64_t S, int64_t chunk, bool vec,
                                hipStream_t st) {
    float2* part = (float2*)scratch;
    if (dtype == 0)
        return vec ? launch_split_v<float, true>(x, y, part, N, V, mode, S, chunk, st)
                   : launch_split_v<float, false>(x, y, part, N, V, mode, S, chunk, st);
    return vec ? launch_split_v<bf16_t, true>(x, y, part, N, V, mode, S, chunk, st)
               : launch_split_v<bf16_t, false>(x, y, part, N, V, mode, S, chunk, st);
}

}  // namespace osm
