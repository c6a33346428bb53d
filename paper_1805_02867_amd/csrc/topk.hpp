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
//  * Threshold.  Each wavefront keeps its own top-K list (keys in LDS); its
//    K-th key is a key of K elements of the row, so the row's K-th key is at
//    least as large, and no element with a key <= that threshold can enter
//    the row's top-K.  When several wavefronts share a row they publish their
//    thresholds in LDS and each filters with the largest one (tau).
//  * Bootstrap.  Before the first selection, tau comes from the first step:
//    the K-th largest distinct value among the lanes' maxima is the value of
//    K distinct elements, so every top-K element is at least as large.
//  * Filter.  Per step, the lane's maximum over its vectors (which also
//    drives the rescale test of the online pair) is compared with tau's
//    value: most steps are skipped with one compare per lane.  Otherwise
//    each vector's maximum, then each element, is compared with tau's value,
//    and only an element at or above it gets its key built and the exact key
//    test (which settles ties by index).
//  * Queue.  Elements that pass are appended to the wavefront's LDS queue
//    right after its list (ballot + mbcnt compaction).  The region holds the
//    list, a trigger's worth of queue and everything that can be appended
//    between two trigger checks (half a step), so appends never overflow and
//    never select.
//  * Select.  After a step, when the queue holds enough entries to be worth
//    raising tau, the wavefront selects the K largest keys of list + queue.
//    Small K: K rounds of "largest key below the last one taken", each a
//    scan of the occupied slots (one per lane per 64 slots) and two 32-bit
//    butterfly maxima.  Large K: the list is kept sorted across the lanes
//    and each 64-key chunk of the queue is sorted by a bitonic network and
//    merged into it.  Either way lane k ends holding the k-th key.
//  * Output.  The normalizer pairs are merged (Eq. 4) and the sorted list
//    gives v_i = 2^{x_i log2e - s} / d and z_i = index, in key order.  With
//    several wavefronts per row, wavefront 0 first selects the K largest keys
//    of their lists.
//
// Three shapes: one, two or four wavefronts per row (four, two or one rows
// per 256-thread workgroup).  Fewer wavefronts per row keep a row's filter
// state in fewer hands (one wavefront needs no barrier at all); more give
// each SIMD more wavefronts to hide the latency of the selection chains, and
// fill the chip when the batch is small.  Each step issues all of a lane's loads
// before processing any, so a wavefront keeps U KiB in flight; loads carry
// non-temporal hints since every element is read exactly once.
#pragma once

#include <type_traits>

#include "md.hpp"
#include "kernels.h"

namespace osm {

constexpr int TK_BLOCK = 256;
constexpr int TK_KMAX = 64;            // largest supported K (one list slot per lane)
constexpr int TK_FLUSH_MAX = 64;       // largest selection trigger (queued keys)
constexpr int TK_PER_LANE = 5;         // rows of 64 slots per K-round selection block
// Selections with more than this many rounds use the sorting network.
#ifndef OSM_TOPK_ROUNDS_MAX
#define OSM_TOPK_ROUNDS_MAX 8
#endif
constexpr int TK_ROUNDS_MAX = OSM_TOPK_ROUNDS_MAX;

// Select early once the queue holds this many (per K): a threshold refreshed
// often saves candidates; the K-round selection costs K rounds, so its
// trigger grows with K, while the sorting-network selection (large K) costs
// one pass per 64 queued keys and runs at one full chunk.
__device__ __forceinline__ int flush_at(int K) {
    if (K > TK_ROUNDS_MAX) return 64;
    return 4 * K > 32 ? 4 * K : 32;
}

// Slots of a wavefront's LDS region (list + queue) when at most `burst`
// keys can be appended between two selection-trigger checks: the queue
// holds fewer than TK_FLUSH_MAX keys at a check, so it never overflows and
// appending never has to select (which keeps the selection code out of the
// unrolled candidate paths).
constexpr int region_slots(int burst) { return TK_KMAX + TK_FLUSH_MAX + burst; }

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

// Largest key over the wavefront; every lane gets the same value.  Two
// 32-bit butterfly maxima (md.hpp steps, DPP-fused where possible): first
// over the value words, then over the index words of the lanes holding that
// value word.  Keys are distinct, so the pair identifies the largest key.
template <int STEP = 0>
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
    if constexpr (STEP < 6) {
        uint32_t a, b;
        bfly_operands<STEP>(v, a, b);
        return wave_max_u32<STEP + 1>(a > b ? a : b);
    } else {
        return v;
    }
}

// The butterflies leave the maximum in every lane; it is read from the first
// lane so that the compiler holds it as a scalar (callers run with every
// lane of the wavefront active), and a test on it is a scalar branch.
__device__ __forceinline__ uint64_t wave_max_key(uint64_t k) {
    const uint32_t hi = (uint32_t)(k >> 32), lo = (uint32_t)k;
    const uint32_t mh = (uint32_t)__builtin_amdgcn_readfirstlane((int)wave_max_u32(hi));
    const uint32_t ml =
        (uint32_t)__builtin_amdgcn_readfirstlane((int)wave_max_u32(hi == mh ? lo : 0u));
    return ((uint64_t)mh << 32) | ml;
}

// ----------------------------------------------------------------- sorting
// Value of lane (lane ^ J) for the sorting networks: DPP quad permutations
// for 1 and 2, the LDS-crossbar swizzle for 4 and 8, and for 16 and 32 the
// operand of the permlane swap pair that came from the other row / half
// (after a 16-lane swap, lanes of even rows hold their partner's value in
// the second result and lanes of odd rows in the first; likewise for the
// 32-lane halves).
template <int J>
__device__ __forceinline__ uint32_t xor_partner(uint32_t v) {
    if constexpr (J == 1) {
        return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false);
    } else if constexpr (J == 2) {
        return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false);
    } else if constexpr (J == 4 || J == 8) {
        return (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, (J << 10) | 0x1F);
    } else if constexpr (J == 16) {
        auto p = __builtin_amdgcn_permlane16_swap(v, v, false, false);
        return (__lane_id() & 16) ? p[0] : p[1];
    } else {
        static_assert(J == 32, "xor partner distance must be a power of two below 64");
        auto p = __builtin_amdgcn_permlane32_swap(v, v, false, false);
        return (__lane_id() & 32) ? p[0] : p[1];
    }
}

template <int J>
__device__ __forceinline__ uint64_t xor_partner_key(uint64_t k) {
    return ((uint64_t)xor_partner<J>((uint32_t)(k >> 32)) << 32) | xor_partner<J>((uint32_t)k);
}

// One compare-exchange stage: the lower lane of each pair keeps the larger
// key when `desc_block` holds, the smaller one otherwise (and the upper lane
// the other one).  A lane that keeps the larger key takes its partner's when
// that is larger, one that keeps the smaller takes it when it is not larger
// (equal keys are the same key either way): one compare and one mask xor,
// where a select between two compares became masked control flow.
template <int J>
__device__ __forceinline__ uint64_t cx_stage(uint64_t v, bool desc_block) {
    const uint64_t p = xor_partner_key<J>(v);
    const bool lower = (__lane_id() & J) == 0;
    const bool take = (p > v) != (lower != desc_block);
    return take ? p : v;
}

// Bitonic sort of one key per lane over the wavefront: lane 0 ends with the
// largest key.
template <int KB, int J>
__device__ __forceinline__ uint64_t bitonic_stage_run(uint64_t v) {
    if constexpr (J >= 1) {
        const bool desc_block = (__lane_id() & KB) == 0;  // KB = 64: the whole wave descends
        v = cx_stage<J>(v, desc_block);
        return bitonic_stage_run<KB, J / 2>(v);
    } else {
        return v;
    }
}

__device__ __forceinline__ uint64_t sort_desc(uint64_t v) {
    v = bitonic_stage_run<2, 1>(v);
    v = bitonic_stage_run<4, 2>(v);
    v = bitonic_stage_run<8, 4>(v);
    v = bitonic_stage_run<16, 8>(v);
    v = bitonic_stage_run<32, 16>(v);
    v = bitonic_stage_run<64, 32>(v);
    return v;
}

// Sort of a bitonic sequence (one key per lane): lane 0 ends with the largest.
__device__ __forceinline__ uint64_t bitonic_merge_desc(uint64_t v) {
    return bitonic_stage_run<64, 32>(v);
}

// Key of lane 63 - lane (xor 63 = mirror within 16 lanes, then xor 16, xor 32).
__device__ __forceinline__ uint64_t reverse_lanes(uint64_t k) {
    uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(k >> 32), 0x140, 0xF,
                                                       0xF, false);
    uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)k, 0x140, 0xF, 0xF,
                                                       false);
    hi = xor_partner<32>(xor_partner<16>(hi));
    lo = xor_partner<32>(xor_partner<16>(lo));
    return ((uint64_t)hi << 32) | lo;
}

// Top 64 keys of (sorted list `cur`, one key per lane, lane 0 largest) and
// (64 more keys, any order), sorted the same way.
__device__ __forceinline__ uint64_t merge_chunk(uint64_t cur, uint64_t q) {
    q = reverse_lanes(sort_desc(q));         // ascending across lanes
    const uint64_t m = cur > q ? cur : q;     // top 64 of the union, a bitonic sequence
    return bitonic_merge_desc(m);
}

// The same 64-bit value on every lane, taken from lane `src` (uniform).
__device__ __forceinline__ uint64_t read_lane_key(uint64_t k, int src) {
    // readlane returns int: go through uint32_t so that the low word is
    // zero-extended, not sign-extended
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)k, src);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(k >> 32), src);
    return ((uint64_t)hi << 32) | (uint64_t)lo;
}

// Selection of the K largest keys among the first `rows` of PER_LANE slots
// per lane (0 = empty).  Lane k returns the k-th largest key (0 past the
// available count); the number found is returned in *found.
template <int PER_LANE>
__device__ __forceinline__ uint64_t select_topk(const uint64_t (&e)[PER_LANE], int rows, int K,
                                                int* found) {
    const int lane = __lane_id();
    uint64_t last = ~0ull, mine = 0;
    int k = 0;
    for (; k < K; ++k) {
        uint64_t best = 0;
#pragma unroll
        for (int j = 0; j < PER_LANE; ++j) {
            if (j < rows) {
                uint64_t c = e[j];
                best = (c < last && c > best) ? c : best;
            }
        }
        best = wave_max_key(best);
        if (best == 0) break;
        if (lane == k) mine = best;
        last = best;
    }
    *found = k;
    return mine;
}

template <int W>  // wavefronts sharing a row
struct TopkWave {
    uint64_t* region;      // [0, K): sorted list; [K, K + qcount): queue
    uint64_t* published;   // thresholds of the wavefronts of the row (W > 1)
    int wave;              // index of this wavefront within its row
    int K;
    int qcount;
    uint64_t tau;
    float tau_v;
    uint64_t mine;         // lane k: k-th key of the list (after a selection)

    __device__ __forceinline__ void raise_tau(uint64_t t) {
        if (t > tau) {
            tau = t;
            tau_v = key_value(t);
        }
    }

    // list + queue -> new list; resets the queue; raises (and publishes) tau.
    // Small K: K rounds of a wavefront maximum.  Large K: the queue in chunks
    // of 64 keys, each sorted and merged into the sorted list (cost
    // independent of K).
    __device__ __forceinline__ void flush() {
        const int lane = __lane_id();
        int found;
        wave_sync();
        if (K <= TK_ROUNDS_MAX) {
            // the occupied slots as rows of 64; the first block takes
            // TK_PER_LANE rows, each further block the current list plus
            // TK_PER_LANE - 1 more rows
            const int used = K + qcount;
            const int rows = (used + 63) >> 6;
            uint64_t e[TK_PER_LANE];
#pragma unroll
            for (int j = 0; j < TK_PER_LANE; ++j)
                e[j] = (j < rows && lane + 64 * j < used) ? region[lane + 64 * j] : 0ull;
            mine = select_topk<TK_PER_LANE>(e, rows, K, &found);
            for (int r0 = TK_PER_LANE; r0 < rows; r0 += TK_PER_LANE - 1) {
                e[0] = lane < K ? mine : 0ull;
#pragma unroll
                for (int j = 1; j < TK_PER_LANE; ++j) {
                    const int r = r0 + j - 1;
                    e[j] = (r < rows && lane + 64 * r < used) ? region[lane + 64 * r] : 0ull;
                }
                mine = select_topk<TK_PER_LANE>(e, TK_PER_LANE, K, &found);
            }
        } else {
            uint64_t cur = lane < K ? region[lane] : 0ull;  // sorted list
            for (int c = 0; c < qcount; c += 64) {
                const uint64_t q = c + lane < qcount ? region[K + c + lane] : 0ull;
                cur = merge_chunk(cur, q);
            }
            mine = lane < K ? cur : 0ull;
            found = (mine != 0) ? lane + 1 : 0;
            found = (int)wave_max_u32((uint32_t)found);
        }
        wave_sync();
        if (lane < K) region[lane] = mine;
        wave_sync();
        qcount = 0;
        if (found == K) {
            raise_tau(read_lane_key(mine, K - 1));
            if constexpr (W > 1) {
                // other wavefronts read this without a barrier: a single-copy
                // atomic 64-bit store keeps them from seeing a torn key
                if (lane == 0)
                    __hip_atomic_store(&published[wave], tau, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_WORKGROUP);
            }
        }
    }

    // Take the largest threshold any wavefront of the row has published.
    __device__ __forceinline__ void pull() {
        if constexpr (W > 1) {
            uint64_t t = 0;
#pragma unroll
            for (int w = 0; w < W; ++w) {
                uint64_t o = __hip_atomic_load(&published[w], __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_WORKGROUP);
                t = o > t ? o : t;
            }
            raise_tau(t);
        }
    }

    // Append the lanes' keys where p holds (the region is sized so that
    // this always fits, see region_slots).
    __device__ __forceinline__ void append(bool p, uint64_t key) {
        uint64_t mask = __builtin_amdgcn_ballot_w64(p);
        if (mask == 0) return;
        int cnt = __builtin_popcountll(mask);
        uint32_t below = __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
        if (p) region[K + qcount + below] = key;
        qcount += cnt;
    }

    // Offer E consecutive elements per lane (indices idx0 .. idx0 + E - 1).
    template <int E>
    __device__ __forceinline__ void offer(const float (&x)[E], uint32_t idx0, bool ok) {
#pragma unroll
        for (int i = 0; i < E; ++i) {
            bool p = ok && x[i] >= tau_v;
            if (__builtin_amdgcn_ballot_w64(p) != 0) {
                uint64_t key = make_key(x[i], idx0 + (uint32_t)i);
                append(p && key > tau, key);
            }
        }
    }
};

// Largest of three binary32 values in one instruction.  fmaxf on loaded
// values makes the compiler quiet possible signalling NaNs first (two extra
// instructions per pair in IEEE mode); here a NaN input may give NaN, which
// only concerns rows holding NaN, whose top-k is unspecified (their outputs
// are NaN through the normalizer in any case).
__device__ __forceinline__ float max3_raw(float a, float b, float c) {
    float r;
    asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
    return r;
}

// max(acc, x[0..N-1]) by a chain of three-input maxima.
template <int N>
__device__ __forceinline__ float vec_max_into(const float (&x)[N], float acc) {
    static_assert(N % 2 == 0, "vectors hold an even number of elements");
    float r = max3_raw(x[0], x[1], acc);
#pragma unroll
    for (int i = 2; i < N; i += 2) r = max3_raw(r, x[i], x[i + 1]);
    return r;
}

// Raw 16-byte vector and its widening to binary32.
template <typename T>
__device__ __forceinline__ void widen(u32x4 q, float (&x)[Vec<T>::N]) {
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

// d += sum_i 2^{x_i log2e - s} with s held fixed (the safe normalizer).
template <int N>
__device__ __forceinline__ float sum_exp_fixed(float d, const float (&x)[N], float s) {
#pragma unroll
    for (int i = 0; i < N; ++i) d += exp2_hw(__builtin_fmaf(x[i], kLog2e, -s));
    return d;
}

// W wavefronts per (virtual) row; TK_BLOCK / (64 W) of them per workgroup;
// U 16-byte vectors per lane per step.
//
// Virtual rows.  Row r of the batch is cut into `segs` chunks of `seg`
// elements (the last one shorter); virtual row v = r * segs + c covers chunk
// c.  With segs = 1 a virtual row is a row.  PART = false writes the final
// outputs (segs must be 1); PART = true writes, per virtual row, its K
// largest keys (indices relative to the start of the row; 0 = fewer than K)
// and its normalizer pair, which topk_merge combines.
// LDS slots of one wavefront's list + queue region for a shape: keys are
// queued by the offer of a batch of candidate vectors (at most 64 E keys) or
// of one scalar element per lane, each followed by a check of the selection
// trigger.
template <typename T, int U>
constexpr int topk_region() {
    return region_slots(64 * Vec<T>::N);
}

// Candidate vectors waiting for their element-wise offer: at most 63 left
// over from the last batch plus 64 appended before the next check.
constexpr int TK_CV_CAP = 128;

// The LDS of a workgroup of the fused top-k kernels.
template <typename T, int U>
struct TopkSmem {
    uint64_t region[TK_BLOCK / 64][topk_region<T, U>()];
    u32x4 cvec[TK_BLOCK / 64][TK_CV_CAP];
    uint32_t cidx[TK_BLOCK / 64][TK_CV_CAP];
    uint64_t published[TK_BLOCK / 64];
    MD wmd[TK_BLOCK / 64];
    float wmx[TK_BLOCK / 64];
    int wq[TK_BLOCK / 64];  // keys queued after the list, per wavefront, at the row's end
};

// One (virtual) row by the W wavefronts of this thread's row group: row vr,
// or with PART chunk vr % segs (seg elements) of row vr / segs, whose K
// largest keys and pair go to pkeys[vr * K ...] and pmd[vr].  The caller has
// emptied the group's lists and thresholds (and, for W > 1, synchronised).
// Returns whether this wavefront holds the row's result (all of them for
// W = 1, the row's first for W > 1).  COH: the partial is stored with
// agent-scope atomic stores, which reach the device's coherence point
// without cache maintenance, for another workgroup of the same kernel.
template <typename T, int W, int U, int VAR, bool PART, bool COH = false>
__device__ __forceinline__ bool topk_vrow(TopkSmem<T, U>& sm, const T* __restrict__ x,
                                          float* __restrict__ vals, int32_t* __restrict__ idx,
                                          uint64_t* __restrict__ pkeys, MD* __restrict__ pmd,
                                          int64_t V, int K, int64_t seg, int64_t segs,
                                          int64_t vr) {
    constexpr int E = Vec<T>::N;
    constexpr int TR = 64 * W;              // threads per row
    constexpr int64_t STEP = (int64_t)TR * U;
    auto& region = sm.region;
    auto& wmd = sm.wmd;
    auto& wmx = sm.wmx;
    uint64_t* const published = sm.published;
    // the wavefront index is uniform: taken as a scalar, so that the row, the
    // step counts and every branch on them stay scalar
    const int tid = threadIdx.x, lane = tid & 63, wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int rw = wv % W;                  // wavefront within the row
    const int tr = tid % TR;                // thread within the row

    const int64_t row = PART ? vr / segs : vr;
    const int64_t start = PART ? (vr - row * segs) * seg : 0;
    const int64_t L = PART ? (V - start < seg ? V - start : seg) : V;
    const uint32_t base = (uint32_t)start;  // index of the chunk's first element
    const T* xr = x + row * V + start;
    TopkWave<W> tw{region[wv], published + (wv / W) * W, rw, K, 0, 0ull, -__builtin_inff(),
                   0ull};

    // split of the chunk into scalar head, 16-byte vectors, scalar tail
    int64_t head = ((16 - (int64_t)(((uintptr_t)xr) & 15)) & 15) / (int64_t)sizeof(T);
    if (head > L) head = L;
    const int64_t nvec = (L - head) / E;
    const int64_t tail0 = head + nvec * E;
    const u32x4* vb = reinterpret_cast<const u32x4*>(xr + head);
    const int fa = flush_at(K);

    const u32x4 ninf = (E == 4) ? u32x4{0xFF800000u, 0xFF800000u, 0xFF800000u, 0xFF800000u}
                                : u32x4{0xFF80FF80u, 0xFF80FF80u, 0xFF80FF80u, 0xFF80FF80u};
    // Full steps (every lane holds U whole vectors) run as a software
    // pipeline over two register buffers: the loads of step t + 1 are issued
    // before step t is processed.  Their addresses are a per-lane pointer plus
    // immediate offsets, so the compiler waits only for the buffer it is
    // about to use.  The remaining vectors (fewer than a step) form one last
    // step with indices clamped into the row and masked after loading.
    const int64_t nfull = nvec / STEP;
    const u32x4* lp = vb + tr;  // this lane's first vector
    // NT: the last read of the data (non-temporal hint)
    auto load_full = [&](u32x4 (&buf)[U], int64_t sidx, auto nt) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if constexpr (decltype(nt)::value)
                buf[u] = __builtin_nontemporal_load(lp + sidx * STEP + u * TR);
            else
                buf[u] = lp[sidx * STEP + u * TR];
        }
        // keep the scheduler from hoisting the next step's work above these
        // loads (that would make it wait for the previous buffer first)
        __builtin_amdgcn_sched_barrier(0);
    };
    auto lane_max_of = [&](const u32x4 (&buf)[U], const bool (&ok)[U], bool masked) {
        float lm = -__builtin_inff();
#pragma unroll
        for (int u = 0; u < U; ++u) {
            float xv[E];
            widen<T>(masked && !ok[u] ? ninf : buf[u], xv);
            lm = vec_max_into(xv, lm);
        }
        return lm;
    };
    bool all_ok[U];
#pragma unroll
    for (int u = 0; u < U; ++u) all_ok[u] = true;

    // The lane's normalizer: one reference sr shared by U partial sums
    // dacc[u] (independent chains for the exponentials of a step), so that
    // d = sum_u dacc[u] relative to sr.
    float sr = kEmptyS;
    float dacc[U];
#pragma unroll
    for (int u = 0; u < U; ++u) dacc[u] = 0.0f;

    // Safe variant: the row's maximum first (plain loads, so that the second
    // read may still find the data in cache), then s = max * log2e is held
    // fixed: the pairs only sum.
    float sfix = 0.0f;
    if constexpr (VAR == TK_SAFE) {
        float mx = -__builtin_inff();
        for (int64_t i = tr; i < head; i += TR) mx = fmaxf(mx, load1(xr + i));
        for (int64_t i = tail0 + tr; i < L; i += TR) mx = fmaxf(mx, load1(xr + i));
        if (nfull > 0) {
            u32x4 ba[U], bb[U];
            load_full(ba, 0, std::false_type{});
            int64_t j = 0;
            for (; j + 2 <= nfull; j += 2) {
                load_full(bb, j + 1, std::false_type{});
                mx = fmaxf(mx, lane_max_of(ba, all_ok, false));
                load_full(ba, (j + 2 < nfull) ? j + 2 : j + 1, std::false_type{});
                mx = fmaxf(mx, lane_max_of(bb, all_ok, false));
            }
            if (j < nfull) mx = fmaxf(mx, lane_max_of(ba, all_ok, false));
        }
        if (nfull * STEP < nvec) {
            const int64_t b0 = nfull * STEP, vlast = nvec - 1;
            u32x4 bt[U];
            bool ok[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t vi = b0 + (int64_t)u * TR + tr;
                ok[u] = vi < nvec;
                bt[u] = vb[vi < nvec ? vi : vlast];
            }
            mx = fmaxf(mx, lane_max_of(bt, ok, true));
        }
        mx = group_max<64>(mx);
        if constexpr (W > 1) {
            if (lane == 0) wmx[wv] = mx;
            __syncthreads();
            const int w0 = wv - rw;
#pragma unroll
            for (int w = 0; w < W; ++w) mx = fmaxf(mx, wmx[w0 + w]);
        }
        // a row of -inf keeps the empty reference (d stays 0); NaN and +inf
        // reach d as NaN, as in the online pair
        sfix = mx * kLog2e;
        if (!(sfix > kEmptyS)) sfix = kEmptyS;
        sr = sfix;
    }
    // Online: move the reference to t (rescaling every partial sum) when t
    // exceeds it by more than kLazy; every term then stays <= 2^kLazy.
    auto raise_ref = [&](float t) {
        if (t > sr + kLazy) {
            const float f = exp2_hw(sr - t);
#pragma unroll
            for (int u = 0; u < U; ++u) dacc[u] *= f;
            sr = t;
        }
    };
    auto fold1 = [&](float v) {
        if constexpr (VAR == TK_ONLINE) raise_ref(v * kLog2e);
        if constexpr (VAR != TK_VALUES) dacc[0] += exp2_hw(__builtin_fmaf(v, kLog2e, -sr));
    };

    // scalar head and tail: wave-uniform loops, one element per lane
    for (int64_t b0 = 0; b0 < head; b0 += TR) {
        int64_t i = b0 + tr;
        bool ok = i < head;
        float v[1] = {ok ? load1(xr + i) : -__builtin_inff()};
        if (ok) fold1(v[0]);
        tw.template offer<1>(v, base + (uint32_t)i, ok);
        if (tw.qcount >= fa) tw.flush();
    }
    for (int64_t b0 = tail0; b0 < L; b0 += TR) {
        int64_t i = b0 + tr;
        bool ok = i < L;
        float v[1] = {ok ? load1(xr + i) : -__builtin_inff()};
        if (ok) fold1(v[0]);
        tw.template offer<1>(v, base + (uint32_t)i, ok);
        if (tw.qcount >= fa) tw.flush();
    }

    // Bootstrap: the K-th largest distinct value among the lanes' maxima
    // over the first step bounds the row's K-th value from below; keys
    // >= (that value, any index) are kept, i.e. keys > (value key with index
    // word 0) - 1.
    // (Large K: the K-th of the lanes' maxima, counted with multiplicity,
    // read off a sort; still a lower bound, as the lanes hold distinct
    // elements.)
    auto bootstrap = [&](const float (&lm)[1]) {
        if (K <= TK_ROUNDS_MAX) {
            float last = __builtin_inff();
            int k = 0;
            for (; k < K; ++k) {
                float c = (lm[0] < last) ? lm[0] : -__builtin_inff();
                c = group_max<64>(c);
                if (!(c > -__builtin_inff())) break;
                last = c;
            }
            if (k == K) tw.raise_tau((make_key(last, 0u) & 0xFFFFFFFF00000000ull) - 1);
        } else {
            // keys with the lane as a stand-in index: only their value words are used
            const uint64_t srt = sort_desc(lm[0] > -__builtin_inff()
                                               ? make_key(lm[0], (uint32_t)lane) : 0ull);
            const uint64_t kth = read_lane_key(srt, K - 1);
            if (kth != 0) tw.raise_tau((kth & 0xFFFFFFFF00000000ull) - 1);
        }
    };
    // Candidate vectors.  A vector whose maximum reaches the threshold is
    // appended whole (its 16 bytes and the index of its first element) to the
    // wavefront's LDS list; each 64 of them are then offered element by
    // element, one vector per lane, so that the per-element tests run on
    // candidates in every lane instead of in the few lanes that hold one.
    u32x4* const cvec = sm.cvec[wv];
    uint32_t* const cidx = sm.cidx[wv];
    int cn = 0;  // entries in the list (wave-uniform)
    auto cv_drain = [&]() {  // offers the first min(cn, 64) entries
        const int n = cn < 64 ? cn : 64;
        const bool has = lane < n;
        wave_sync();
        const u32x4 q = cvec[has ? lane : 0];
        const uint32_t i0 = cidx[has ? lane : 0];
        const int m = cn - n;  // left over, moved to the front
        u32x4 r = q;
        uint32_t ri = 0;
        if (lane < m) {
            r = cvec[64 + lane];
            ri = cidx[64 + lane];
        }
        wave_sync();
        if (lane < m) {
            cvec[lane] = r;
            cidx[lane] = ri;
        }
        cn = m;
        float xv[E];
        widen<T>(has ? q : ninf, xv);
        tw.template offer<E>(xv, base + i0, has);
        if (tw.qcount >= fa) tw.flush();
    };
    auto cv_append = [&](bool p, const u32x4& q, uint32_t i0) {
        const uint64_t mask = __builtin_amdgcn_ballot_w64(p);
        if (mask == 0) return;
        const uint32_t below = __builtin_amdgcn_mbcnt_hi(
            (uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
        if (p) {
            cvec[cn + below] = q;
            cidx[cn + below] = i0;
        }
        cn += __builtin_popcountll(mask);
        if (cn >= 64) cv_drain();
    };

    // One step: the lane's maximum over the step (one rescale test, and one
    // candidate test, per step), the exponentials of every element, then the
    // vectors that may hold a candidate are offered.
    auto step = [&](const u32x4 (&buf)[U], const bool (&ok)[U], int64_t b0, bool masked) {
        const float lane_mx = lane_max_of(buf, ok, masked);
        if constexpr (VAR == TK_ONLINE) {
            // a wave-uniform branch, so that the common case skips the
            // rescale instead of computing it and selecting it away
            const float t = lane_mx * kLog2e;
            if (__builtin_amdgcn_ballot_w64(t > sr + kLazy) != 0) raise_ref(t);
        }
        if constexpr (VAR != TK_VALUES) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                float xv[E];
                widen<T>(masked && !ok[u] ? ninf : buf[u], xv);
                dacc[u] = sum_exp_fixed(dacc[u], xv, sr);
            }
        }
        if (__builtin_amdgcn_ballot_w64(lane_mx >= tw.tau_v) != 0) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                float xv[E];
                widen<T>(masked && !ok[u] ? ninf : buf[u], xv);
                const uint32_t e0 = (uint32_t)(head + (b0 + (int64_t)u * TR + tr) * E);
                cv_append(ok[u] && vec_max(xv) >= tw.tau_v, buf[u], e0);
            }
        }
        tw.pull();
    };

    bool booted = false;
    if (nfull > 0) {
        u32x4 ba[U], bb[U];
        load_full(ba, 0, std::true_type{});
        const float lm[1] = {lane_max_of(ba, all_ok, false)};
        bootstrap(lm);
        booted = true;
        int64_t j = 0;
        for (; j + 2 <= nfull; j += 2) {
            load_full(bb, j + 1, std::true_type{});
            step(ba, all_ok, j * STEP, false);
            load_full(ba, (j + 2 < nfull) ? j + 2 : j + 1, std::true_type{});  // stays inside the row
            step(bb, all_ok, (j + 1) * STEP, false);
        }
        if (j < nfull) step(ba, all_ok, j * STEP, false);
    }
    if (nfull * STEP < nvec) {
        // last, partial step: clamped indices, masked lanes
        const int64_t b0 = nfull * STEP, vlast = nvec - 1;
        u32x4 bt[U];
        bool ok[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t vi = b0 + (int64_t)u * TR + tr;
            ok[u] = vi < nvec;
            bt[u] = __builtin_nontemporal_load(vb + (vi < nvec ? vi : vlast));
        }
        if (!booted) {
            const float lm[1] = {lane_max_of(bt, ok, true)};
            bootstrap(lm);
        }
        step(bt, ok, b0, true);
    }
    while (cn > 0) cv_drain();
    // A row shared by W > 1 wavefronts and K <= TK_ROUNDS_MAX: no final
    // selection per wavefront; the row's first wavefront selects once over
    // every wavefront's list and queue (each under one row of 64 slots, as a
    // selection runs whenever a queue reaches its trigger).
    if (W == 1 || K > TK_ROUNDS_MAX) tw.flush();

    // merge of the normalizer pairs: wavefront butterflies, then (W > 1)
    // a fixed-order merge of the row's wavefronts
    MD md = md_empty();
    if constexpr (VAR != TK_VALUES) {
        float dsum = dacc[0];
#pragma unroll
        for (int u = 1; u < U; ++u) dsum += dacc[u];
        md = group_merge<64>(MD{sr, dsum});
    }
    uint64_t key = tw.mine;
    if constexpr (W > 1) {
        if (lane == 0) {
            wmd[wv] = md;
            sm.wq[wv] = K <= TK_ROUNDS_MAX ? tw.qcount : 0;
        }
        __syncthreads();
        if (rw != 0) return false;
        const int w0 = wv;  // first wavefront of the row
        md = wmd[w0];
#pragma unroll
        for (int w = 1; w < W; ++w) md = md_merge(md, wmd[w0 + w]);
        if (K <= TK_ROUNDS_MAX) {
            uint64_t e[W];
#pragma unroll
            for (int w = 0; w < W; ++w)
                e[w] = (lane < K + sm.wq[w0 + w]) ? region[w0 + w][lane] : 0ull;
            int found;
            key = select_topk<W>(e, W, K, &found);
        } else {
            // the wavefronts' lists are sorted (lane 0 largest, 0 past the K-th):
            // each is merged into the running one by a lane reversal, a maximum
            // per lane and the 6-stage bitonic merge, instead of K rounds
            uint64_t cur = lane < K ? region[w0][lane] : 0ull;
#pragma unroll
            for (int w = 1; w < W; ++w) {
                const uint64_t q = reverse_lanes(lane < K ? region[w0 + w][lane] : 0ull);
                cur = bitonic_merge_desc(cur > q ? cur : q);
            }
            key = lane < K ? cur : 0ull;
        }
    }
    if constexpr (PART) {
        if constexpr (COH) {
            if (lane < K)
                __hip_atomic_store(pkeys + vr * K + lane, key, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
            if (VAR != TK_VALUES && lane == 0)
                __hip_atomic_store(reinterpret_cast<uint64_t*>(pmd + vr),
                                   __builtin_bit_cast(uint64_t, md), __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
        } else {
            if (lane < K) pkeys[vr * K + lane] = key;
            if (VAR != TK_VALUES && lane == 0) pmd[vr] = md;
        }
    } else if (lane < K) {
        if constexpr (VAR == TK_VALUES) {
            vals[row * K + lane] = key_value(key);
        } else {
            const float S = md.s, rd = 1.0f / md.d;
            vals[row * K + lane] = out_elem(key_value(key), S, rd);
        }
        idx[row * K + lane] = key_index(key);
    }
    return true;
}

template <typename T, int W, int U, int VAR, bool PART>
__global__ __launch_bounds__(TK_BLOCK) void topk_fused(const T* __restrict__ x,
                                                      float* __restrict__ vals,
                                                      int32_t* __restrict__ idx,
                                                      uint64_t* __restrict__ pkeys,
                                                      MD* __restrict__ pmd, int64_t N, int64_t V,
                                                      int K, int64_t seg, int64_t segs) {
    constexpr int RB = TK_BLOCK / 64 / W;   // rows per workgroup
    __shared__ TopkSmem<T, U> sm;
    const int lane = threadIdx.x & 63, wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t vr = (int64_t)blockIdx.x * RB + wv / W;
    const bool live = vr < N * segs;        // uniform per wavefront (and per row)
    if (lane < K) sm.region[wv][lane] = 0;  // empty list
    if (lane == 0) sm.published[wv] = 0;
    if constexpr (W > 1) __syncthreads();
    if (!live) return;                      // whole rows leave together
    topk_vrow<T, W, U, VAR, PART>(sm, x, vals, idx, pkeys, pmd, V, K, seg, segs, vr);
}

// Second stage of the split top-k: per row, the K largest of the S * K
// chunk keys (filtered against the running threshold as in the one-pass
// kernel) and the fixed-order merge (Eq. 4) of the S chunk pairs.  One
// wavefront per row.
constexpr int TK_MERGE_B = 8;  // keys per lane in flight

// One row by one wavefront: region holds at least region_slots(64) slots,
// its first K already empty; B keys per lane are in flight, and the
// selection trigger is checked after every 64 appended keys.  The pairs'
// loads are issued with the first keys', so that a row of up to 64 B keys and
// 64 chunks costs one round trip.  COH: the partials are read with
// agent-scope atomic loads (written by other workgroups of the same kernel).
template <int VAR, bool COH = false, int B = TK_MERGE_B>
__device__ __forceinline__ void topk_merge_row(uint64_t* region, const uint64_t* pkeys,
                                               const MD* pmd, float* __restrict__ vals,
                                               int32_t* __restrict__ idx, int64_t row, int64_t S,
                                               int K) {
    const int lane = threadIdx.x & 63;
    TopkWave<1> tw{region, nullptr, 0, K, 0, 0ull, -__builtin_inff(), 0ull};
    const int fa = flush_at(K);
    const int64_t n = S * K;
    const uint64_t* pk = pkeys + row * n;
    const MD* pm = pmd + row * S;
    auto load_md = [&](int64_t j) {
        if constexpr (COH)
            return __builtin_bit_cast(MD, __hip_atomic_load(reinterpret_cast<const uint64_t*>(pm + j),
                                                            __ATOMIC_RELAXED,
                                                            __HIP_MEMORY_SCOPE_AGENT));
        else
            return pm[j];
    };
    // the first pair of this lane (chunk `lane`), requested before the keys
    MD md = md_empty();
    if constexpr (VAR != TK_VALUES) {
        if (lane < S) md = load_md(lane);
    }
    auto load_keys = [&](uint64_t (&k)[B], int64_t c) {
#pragma unroll
        for (int b = 0; b < B; ++b) {
            const int64_t j = c + b * 64 + lane;
            if constexpr (COH)
                k[b] = j < n ? __hip_atomic_load(pk + j, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                             : 0ull;
            else
                k[b] = j < n ? pk[j] : 0ull;
        }
    };
    uint64_t key;
    if (n <= 64 * B && K <= TK_ROUNDS_MAX) {
        // every key in registers at once: K rounds of the wavefront maximum
        // below the last key taken (0 marks a missing key and is never taken)
        uint64_t k[B];
        load_keys(k, 0);
        int found;
        key = select_topk<B>(k, B, K, &found);
    } else {
        for (int64_t c = 0; c < n; c += 64 * B) {
            uint64_t k[B];
            load_keys(k, c);
#pragma unroll
            for (int b = 0; b < B; ++b) {
                tw.append(k[b] > tw.tau, k[b]);  // 0 never passes
                if (tw.qcount >= fa) tw.flush();
            }
        }
        tw.flush();
        key = tw.mine;
    }
    if constexpr (VAR != TK_VALUES) {
        // chunks lane, lane + 64, ... in order, then the butterfly
        for (int64_t j = lane + 64; j < S; j += 64) md = md_merge(md, load_md(j));
        md = group_merge<64>(md);  // every lane takes part
    }
    if (lane < K) {
        if constexpr (VAR == TK_VALUES) {
            vals[row * K + lane] = key_value(key);
        } else {
            const float Sv = md.s, rd = 1.0f / md.d;
            vals[row * K + lane] = out_elem(key_value(key), Sv, rd);
        }
        idx[row * K + lane] = key_index(key);
    }
}

template <int VAR>
__global__ __launch_bounds__(TK_BLOCK) void topk_merge(const uint64_t* __restrict__ pkeys,
                                                      const MD* __restrict__ pmd,
                                                      float* __restrict__ vals,
                                                      int32_t* __restrict__ idx, int64_t N,
                                                      int64_t S, int K) {
    constexpr int WB = TK_BLOCK / 64;
    constexpr int REGION = region_slots(64);
    __shared__ uint64_t region[WB][REGION];
    const int lane = threadIdx.x & 63, wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t row = (int64_t)blockIdx.x * WB + wv;
    if (lane < K) region[wv][lane] = 0;
    if (row >= N) return;
    topk_merge_row<VAR>(region[wv], pkeys, pmd, vals, idx, row, S, K);
}

// Split top-k in one kernel: chunk c of row r is workgroup r * segs + c (four
// wavefronts), which leaves its partial (K keys, pair) at the coherence
// point; the workgroup that completes a row (ctr[r] counts its chunks) merges
// the row's partials there and then, instead of a second kernel.  ctr starts
// at zero and is left at zero (the merger resets its row's count).
template <typename T, int U, int VAR>
__global__ __launch_bounds__(TK_BLOCK) void topk_split1(const T* __restrict__ x,
                                                       float* __restrict__ vals,
                                                       int32_t* __restrict__ idx,
                                                       uint64_t* __restrict__ pkeys,
                                                       MD* __restrict__ pmd, uint32_t* ctr,
                                                       int64_t N, int64_t V, int K, int64_t seg,
                                                       int64_t segs) {
    static_assert(topk_region<T, U>() >= region_slots(64), "the merge appends 64 keys per check");
    __shared__ TopkSmem<T, U> sm;
    const int lane = threadIdx.x & 63, wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t vr = blockIdx.x;
    if (lane < K) sm.region[wv][lane] = 0;
    if (lane == 0) sm.published[wv] = 0;
    __syncthreads();
    if (!topk_vrow<T, 4, U, VAR, true, true>(sm, x, nullptr, nullptr, pkeys, pmd, V, K, seg, segs,
                                             vr))
        return;
    // the partial's coherent stores have completed before the row's count moves
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    const int64_t row = vr / segs;
    uint32_t done = 0;
    if (lane == 0)
        done = __hip_atomic_fetch_add(ctr + row, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    done = __builtin_amdgcn_readfirstlane(done);
    if (done != (uint32_t)segs - 1) return;
    // every chunk of the row is in: its partials are read at the coherence
    // point, after the count that says so
    if (lane < K) sm.region[wv][lane] = 0;
    topk_merge_row<VAR, true>(sm.region[wv], pkeys, pmd, vals, idx, row, segs, K);
    if (lane == 0) __hip_atomic_store(ctr + row, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// 16-byte vectors per lane per step, by shape and element type: enough
// loads in flight per wavefront without pushing the register count (and so
// the occupancy) down; bfloat16 vectors widen to twice the registers.  For
// bfloat16 rows of a wavefront, six vectors (48 elements a lane per step,
// 146 registers, three wavefronts per SIMD) also give the first step's lane
// maxima, and so the starting threshold, three times the reach of two.
#ifndef OSM_TOPK_U1
#define OSM_TOPK_U1 5
#endif
#ifndef OSM_TOPK_U1B
#define OSM_TOPK_U1B 6
#endif
#ifndef OSM_TOPK_U2
#define OSM_TOPK_U2 4
#endif
#ifndef OSM_TOPK_U4
#define OSM_TOPK_U4 2
#endif

#ifndef OSM_TOPK_USPLIT
#define OSM_TOPK_USPLIT 6
#endif

// The split kernels (a chunk per workgroup, for small batches) run only a
// few workgroups per CU, so they can keep more loads in flight per lane.
constexpr int topk_split_unroll() { return OSM_TOPK_USPLIT; }

template <typename T, int W>
constexpr int topk_unroll() {
    if constexpr (W == 1) return std::is_same<T, float>::value ? OSM_TOPK_U1 : OSM_TOPK_U1B;
    else if constexpr (W == 2) return std::is_same<T, float>::value ? OSM_TOPK_U2 : OSM_TOPK_U1B;
    else return OSM_TOPK_U4;
}

// Launch of one variant for one element type (see TopkLaunch).
template <typename T, int VAR>
hipError_t launch_topk_t(const TopkLaunch& a) {
    dim3 block(TK_BLOCK);
    const T* x = static_cast<const T*>(a.x);
    if (a.S <= 1) {
        if (a.waves_per_row == 1) {
            constexpr int RB = TK_BLOCK / 64;
            dim3 grid((unsigned)((a.N + RB - 1) / RB));
            hipLaunchKernelGGL((topk_fused<T, 1, topk_unroll<T, 1>(), VAR, false>), grid, block, 0,
                               a.st, x, a.vals, a.idx, nullptr, nullptr, a.N, a.V, a.K, a.V,
                               (int64_t)1);
        } else if (a.waves_per_row == 2) {
            if constexpr (VAR == TK_ONLINE) {  // the two-wavefront shape is built for Alg. 4 only
                constexpr int RB = TK_BLOCK / 128;
                dim3 grid((unsigned)((a.N + RB - 1) / RB));
                hipLaunchKernelGGL((topk_fused<T, 2, topk_unroll<T, 2>(), VAR, false>), grid,
                                   block, 0, a.st, x, a.vals, a.idx, nullptr, nullptr, a.N, a.V,
                                   a.K, a.V, (int64_t)1);
            } else {
                return hipErrorInvalidValue;
            }
        } else if (a.waves_per_row == 4) {
            dim3 grid((unsigned)a.N);
            hipLaunchKernelGGL((topk_fused<T, 4, topk_unroll<T, 4>(), VAR, false>), grid, block, 0,
                               a.st, x, a.vals, a.idx, nullptr, nullptr, a.N, a.V, a.K, a.V,
                               (int64_t)1);
        } else {
            return hipErrorInvalidValue;
        }
        return hipGetLastError();
    }
    // split: chunks of a.chunk elements, one workgroup (four wavefronts) each
    uint64_t* pkeys = static_cast<uint64_t*>(a.part);
    MD* pmd = reinterpret_cast<MD*>(pkeys + a.N * a.S * a.K);
    dim3 grid((unsigned)(a.N * a.S));
    if (a.ctr) {  // merge by each row's last chunk, in the same kernel
        hipLaunchKernelGGL((topk_split1<T, topk_split_unroll(), VAR>), grid, block, 0, a.st, x,
                           a.vals, a.idx, pkeys, pmd, a.ctr, a.N, a.V, a.K, a.chunk, a.S);
        return hipGetLastError();
    }
    hipLaunchKernelGGL((topk_fused<T, 4, topk_split_unroll(), VAR, true>), grid, block, 0, a.st,
                       x, nullptr, nullptr, pkeys, pmd, a.N, a.V, a.K, a.chunk, a.S);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    constexpr int WB = TK_BLOCK / 64;
    dim3 mgrid((unsigned)((a.N + WB - 1) / WB));
    hipLaunchKernelGGL((topk_merge<VAR>), mgrid, block, 0, a.st, pkeys, pmd, a.vals, a.idx, a.N,
                       a.S, a.K);
    return hipGetLastError();
}

}  // namespace osm
