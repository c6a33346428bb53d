// Fused online softmax + top-k for gfx950 (Section 4, Alg. 4): one read of
// every element, K (probability, index) pairs written per row.
//
// Alg. 4 keeps, next to the online pair (m, d), a sorted buffer of the K
// largest inputs seen so far and inserts every element into it.  On a
// 64-lane wavefront a per-element insertion would make every lane pay for the
// rare lane that inserts, so the same selection is organised as
// filter + queue + select:
//
//  * Order.  Elements are ranked by the 64-bit key
//        (monotone image of x) << 32 | ~index,
//    so a larger key means a larger x, or an equal x at a lower index: the
//    order Alg. 4's strictly-less insertion produces.  -0.0 is keyed as +0.0.
//  * Filter.  Each wavefront keeps its own top-K list (keys in LDS) and the
//    threshold tau = its K-th key.  Those K elements belong to the row, so
//    the row's K-th key is >= tau, and an element with key <= tau can never
//    enter the row's top-K.  A cheap test on each lane's 16-byte vector maximum
//    (already computed for the online pair) skips whole vectors.
//  * Queue.  Elements that pass are appended to the wavefront's LDS queue
//    (ballot + mbcnt compaction).
//  * Select.  When the queue fills up, or holds enough entries to be worth
//    raising tau, the wavefront selects the K largest keys of list + queue:
//    K rounds of "largest key below the last one taken", each a scan of 5
//    entries per lane and a 6-step butterfly maximum.
//  * Merge.  At the end of the row, the pairs of the wavefronts are merged
//    (Eq. 4) and wavefront 0 selects the K largest keys of all the lists.
//    Outputs are v_i = 2^{x_i log2e - s} / d and z_i = index, in key order.
#include "md.hpp"
#include "kernels.h"

namespace osm {

constexpr int TK_BLOCK = 256;
constexpr int TK_W = TK_BLOCK / 64;
constexpr int TK_KMAX = 64;          // largest supported K (one list slot per lane)
constexpr int TK_QCAP = 256;         // queue entries per wavefront
constexpr int TK_REGION = TK_KMAX + TK_QCAP;
constexpr int TK_PER_LANE = TK_REGION / 64;
constexpr int TK_FLUSH_AT = 128;     // select early once the queue holds this many
constexpr int TK_U = 2;              // 16-byte vectors per lane in flight

static_assert(TK_REGION % 64 == 0, "region must split evenly over 64 lanes");

__device__ __forceinline__ uint64_t make_key(float x, uint32_t idx) {
    uint32_t u = __float_as_uint(x);
    u = (u == 0x80000000u) ? 0u : u;  // -0.0 ranks as +0.0
    uint32_t hi = u ^ ((uint32_t)((int32_t)u >> 31) | 0x80000000u);
    return ((uint64_t)hi << 32) | (uint64_t)(~idx);
}

__device__ __forceinline__ float key_value(uint64_t k) {
    uint32_t hi = (uint32_t)(k >> 32);
    uint32_t u = (hi & 0x80000000u) ? (hi & 0x7FFFFFFFu) : ~hi;
    return __uint_as_float(u);
}

__device__ __forceinline__ int32_t key_index(uint64_t k) { return (int32_t)(~(uint32_t)k); }

// Largest key over the wavefront; every lane gets the same value.
__device__ __forceinline__ uint64_t wave_max_key(uint64_t k) {
    uint32_t hi = (uint32_t)(k >> 32), lo = (uint32_t)k;
#define OSM_KEY_STEP(M)                                                  \
    {                                                                    \
        uint32_t oh = xor_lane_u<M>(hi), ol = xor_lane_u<M>(lo);         \
        bool take = (oh > hi) || (oh == hi && ol > lo);                  \
        hi = take ? oh : hi;                                             \
        lo = take ? ol : lo;                                             \
    }
    OSM_KEY_STEP(1)
    OSM_KEY_STEP(2)
    OSM_KEY_STEP(4)
    OSM_KEY_STEP(8)
    OSM_KEY_STEP(16)
    OSM_KEY_STEP(32)
#undef OSM_KEY_STEP
    return ((uint64_t)hi << 32) | lo;
}

// Selection of the K largest keys among n_per_lane * 64 slots (0 = empty).
// Lane k returns the k-th largest key (0 past the available count); the
// number found is returned in *found.
template <int PER_LANE>
__device__ __forceinline__ uint64_t select_topk(const uint64_t (&e)[PER_LANE], int K,
                                                int* found) {
    const int lane = __lane_id();
    uint64_t last = ~0ull, mine = 0;
    int k = 0;
    for (; k < K; ++k) {
        uint64_t best = 0;
#pragma unroll
        for (int j = 0; j < PER_LANE; ++j) {
            uint64_t c = e[j];
            best = (c < last && c > best) ? c : best;
        }
        best = wave_max_key(best);
        if (best == 0) break;
        if (lane == k) mine = best;
        last = best;
    }
    *found = k;
    return mine;
}

struct TopkWave {
    uint64_t* region;  // [0, KMAX): sorted list; [KMAX, REGION): queue
    int qcount;
    uint64_t tau;
    float tau_v;

    // list + queue -> new list; resets the queue; raises tau.
    __device__ __forceinline__ void flush(int K) {
        const int lane = __lane_id();
        wave_sync();
        uint64_t e[TK_PER_LANE];
#pragma unroll
        for (int j = 0; j < TK_PER_LANE; ++j) e[j] = region[lane + 64 * j];
        int found;
        uint64_t mine = select_topk<TK_PER_LANE>(e, K, &found);
        wave_sync();
        region[lane] = mine;
#pragma unroll
        for (int j = 1; j < TK_PER_LANE; ++j) region[lane + 64 * j] = 0;
        wave_sync();
        qcount = 0;
        if (found == K) {
            // readlane returns int: go through uint32_t so that the low word
            // is zero-extended, not sign-extended
            const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)mine, K - 1);
            const uint32_t hi =
                (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(mine >> 32), K - 1);
            tau = ((uint64_t)hi << 32) | (uint64_t)lo;
            tau_v = key_value(tau);
        }
    }

    // Offer one element per lane (ok = lane holds a real element).
    __device__ __forceinline__ void offer(float x, uint32_t idx, bool ok, int K) {
        uint64_t key = make_key(x, idx);
        bool p = ok && key > tau;
        uint64_t mask = __builtin_amdgcn_ballot_w64(p);
        if (mask == 0) return;
        int cnt = __builtin_popcountll(mask);
        if (qcount + cnt > TK_QCAP) {
            flush(K);
            p = ok && key > tau;
            mask = __builtin_amdgcn_ballot_w64(p);
            cnt = __builtin_popcountll(mask);
        }
        uint32_t below = __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
        if (p) region[TK_KMAX + qcount + below] = key;
        qcount += cnt;
    }
};

template <typename T, bool VEC>
__global__ __launch_bounds__(TK_BLOCK) void topk_fused(const T* __restrict__ x,
                                                      float* __restrict__ vals,
                                                      int32_t* __restrict__ idx, int64_t V,
                                                      int K) {
    constexpr int E = Vec<T>::N;
    __shared__ uint64_t region[TK_W][TK_REGION];
    __shared__ MD wmd[TK_W];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t row = blockIdx.x;
    const T* xr = x + row * V;

    for (int i = tid; i < TK_W * TK_REGION; i += TK_BLOCK) (&region[0][0])[i] = 0;
    __syncthreads();

    TopkWave tw{region[wave], 0, 0ull, -__builtin_inff()};

    // split of the row into scalar head, 16-byte vectors, scalar tail
    int64_t head, nvec;
    if (VEC) {
        int64_t mis = (int64_t)(((uintptr_t)xr) & 15);
        head = ((16 - mis) & 15) / (int64_t)sizeof(T);
        if (head > V) head = V;
        nvec = (V - head) / E;
    } else {
        head = V;
        nvec = 0;
    }
    const int64_t tail0 = head + nvec * E;
    const T* vb = xr + head;

    MD st[TK_U];
#pragma unroll
    for (int u = 0; u < TK_U; ++u) st[u] = md_empty();

    // scalar head and tail: wave-uniform loops, one element per lane
    for (int64_t b0 = 0; b0 < head; b0 += TK_BLOCK) {
        int64_t i = b0 + tid;
        bool ok = i < head;
        float v = ok ? load1(xr + i) : -__builtin_inff();
        if (ok) st[0] = md_fold1(st[0], v);
        tw.offer(v, (uint32_t)i, ok, K);
    }
    for (int64_t b0 = tail0; b0 < V; b0 += TK_BLOCK) {
        int64_t i = b0 + tid;
        bool ok = i < V;
        float v = ok ? load1(xr + i) : -__builtin_inff();
        if (ok) st[0] = md_fold1(st[0], v);
        tw.offer(v, (uint32_t)i, ok, K);
    }

    // vector body: every lane runs the same number of iterations so that the
    // wavefront-wide queue operations see all 64 lanes
    for (int64_t b0 = 0; b0 < nvec; b0 += (int64_t)TK_BLOCK * TK_U) {
        Vec<T> buf[TK_U];
        bool ok[TK_U];
#pragma unroll
        for (int u = 0; u < TK_U; ++u) {
            int64_t vi = b0 + (int64_t)u * TK_BLOCK + tid;
            ok[u] = vi < nvec;
            buf[u] = ok[u] ? Vec<T>::load(vb + vi * E) : Vec<T>::fill(-__builtin_inff());
        }
#pragma unroll
        for (int u = 0; u < TK_U; ++u) {
            float mx = buf[u].v[0];
#pragma unroll
            for (int i = 1; i < E; ++i) mx = fmaxf(mx, buf[u].v[i]);
            st[u] = md_fold(st[u], buf[u].v);
            if (__builtin_amdgcn_ballot_w64(ok[u] && mx >= tw.tau_v) != 0) {
                const int64_t e0 = head + (b0 + (int64_t)u * TK_BLOCK + tid) * E;
#pragma unroll
                for (int i = 0; i < E; ++i) tw.offer(buf[u].v[i], (uint32_t)(e0 + i), ok[u], K);
            }
        }
        if (tw.qcount >= TK_FLUSH_AT) tw.flush(K);
    }
    tw.flush(K);

    // merge of the normalizer pairs: wavefront butterflies, then fixed order
    MD md = st[0];
#pragma unroll
    for (int u = 1; u < TK_U; ++u) md = md_merge(md, st[u]);
    md = group_merge<64>(md);
    if (lane == 0) wmd[wave] = md;
    __syncthreads();
    if (wave == 0) {
        MD r = wmd[0];
#pragma unroll
        for (int w = 1; w < TK_W; ++w) r = md_merge(r, wmd[w]);
        const float S = r.s, rd = 1.0f / r.d;
        uint64_t e[TK_W];
#pragma unroll
        for (int w = 0; w < TK_W; ++w) e[w] = region[w][lane];
        int found;
        uint64_t mine = select_topk<TK_W>(e, K, &found);
        if (lane < K) {
            float xv = key_value(mine);
            vals[row * K + lane] = exp2_hw(__builtin_fmaf(xv, kLog2e, -S)) * rd;
            idx[row * K + lane] = key_index(mine);
        }
    }
}

hipError_t launch_topk_fused(const void* x, float* vals, int32_t* idx, int64_t N, int64_t V,
                             int K, int dtype, bool vec, hipStream_t st) {
    if (K < 1 || K > TK_KMAX) return hipErrorInvalidValue;
    dim3 grid((unsigned)N), block(TK_BLOCK);
    if (dtype == 0) {
        if (vec)
            hipLaunchKernelGGL((topk_fused<float, true>), grid, block, 0, st, (const float*)x,
                               vals, idx, V, K);
        else
            hipLaunchKernelGGL((topk_fused<float, false>), grid, block, 0, st, (const float*)x,
                               vals, idx, V, K);
    } else {
        if (vec)
            hipLaunchKernelGGL((topk_fused<bf16_t, true>), grid, block, 0, st,
                               (const bf16_t*)x, vals, idx, V, K);
        else
            hipLaunchKernelGGL((topk_fused<bf16_t, false>), grid, block, 0, st,
                               (const bf16_t*)x, vals, idx, V, K);
    }
    return hipGetLastError();
}

}  // namespace osm
