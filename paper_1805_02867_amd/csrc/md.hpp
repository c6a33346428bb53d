// Device-side building blocks shared by every kernel of the library:
// element I/O for binary32 and bfloat16, the normalizer pair and its merge,
// and lane-group reductions for 64-wide CDNA wavefronts.
//
// The normalizer pair.  Section 3 of the paper carries (m, d) with
// m = max_k x_k and d = sum_j e^{x_j - m}.  On the GPU we carry the same pair
// in base 2, (s, d) with s ~ m * log2(e) and d = sum_j 2^{x_j log2(e) - s},
// because the hardware exponential (v_exp_f32) is 2^x.  Every exponent is
// formed as fma(x, log2(e), -s): x * log2(e) is exact inside the fma and only
// the difference is rounded, once.  Whatever binary32 value s holds, the same
// s is used for d and for the outputs of a row, so it cancels in
// y = 2^{x log2(e) - s} / d; it only has to be >= every x * log2(e) up to a
// rounding, which keeps every term <= 1 (no overflow, the paper's safety
// argument after Theorem 1).
//
// Identity.  An empty pair is (s, d) = (-FLT_MAX, 0) rather than (-inf, 0):
// merging it with anything scales 0 by 2^{finite} = 0 or by 2^0 = 1, so no
// e^{-inf - (-inf)} = NaN can arise from empty lanes, chunks or -inf inputs,
// and no branch is needed in the hot loop.  A row made only of -inf keeps
// d = 0 and then produces 0 * (1/0) = NaN outputs, which is what the safe
// formula (Eq. 2) gives in IEEE arithmetic; +inf or NaN inputs likewise reach
// every output of their row as NaN.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace osm {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kEmptyS = -3.402823466e38f;  // -FLT_MAX: identity of the merge

__device__ __forceinline__ float exp2_hw(float v) { return __builtin_amdgcn_exp2f(v); }

// Outputs y = 2^t * rd (t = x log2e - s, rd = 1/d).  v_exp_f32 returns 0
// where 2^t is below 2^-126 (it produces no binary32 subnormals), which would
// lose outputs that are subnormal but not zero.  There the exponent is raised
// by 64 and the factor 2^-64 moved into rd: 2^{t+64} is normal for every
// t >= -190 and the product rounds once, to the subnormal result.  (rd *
// 2^-64 stays normal for d <= 2^62, which holds for the safe and online
// normalizers: d <= V * 2^8.)
constexpr float kExpMin = -126.0f;

__device__ __forceinline__ float out_scaled(float t, float rd) {
    const bool lo = t < kExpMin;
    return exp2_hw(lo ? t + 64.0f : t) * (lo ? rd * 0x1p-64f : rd);
}

__device__ __forceinline__ float out_elem(float x, float S, float rd) {
    return out_scaled(__builtin_fmaf(x, kLog2e, -S), rd);
}

// The same for N values at once: the common case (no exponent below -126 in
// the wavefront) costs one minimum per element pair and one uniform branch.
template <int N>
__device__ __forceinline__ void out_vals(float (&v)[N], float S, float rd) {
    float t[N];
#pragma unroll
    for (int i = 0; i < N; ++i) t[i] = __builtin_fmaf(v[i], kLog2e, -S);
    float mn = t[0];
#pragma unroll
    for (int i = 1; i < N; ++i) mn = __builtin_fminf(mn, t[i]);
    if (__builtin_amdgcn_ballot_w64(mn < kExpMin) == 0) {
#pragma unroll
        for (int i = 0; i < N; ++i) v[i] = exp2_hw(t[i]) * rd;
    } else {
#pragma unroll
        for (int i = 0; i < N; ++i) v[i] = out_scaled(t[i], rd);
    }
}

// ---------------------------------------------------------------- element I/O
// Native 16-byte vector types (the nontemporal builtins take these).
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// A 16-byte vector: 4 binary32 or 8 bfloat16 elements.
template <typename T> struct Vec;

template <> struct Vec<float> {
    static constexpr int N = 4;
    float v[4];
    __device__ __forceinline__ static Vec load(const float* p) {
        f32x4 q = *reinterpret_cast<const f32x4*>(p);
        return Vec{{q.x, q.y, q.z, q.w}};
    }
    __device__ __forceinline__ static Vec load_nt(const float* p) {
        f32x4 q = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
        return Vec{{q.x, q.y, q.z, q.w}};
    }
    __device__ __forceinline__ static Vec fill(float f) { return Vec{{f, f, f, f}}; }
    __device__ __forceinline__ void store(float* p) const {
        *reinterpret_cast<f32x4*>(p) = f32x4{v[0], v[1], v[2], v[3]};
    }
    __device__ __forceinline__ void store_nt(float* p) const {
        __builtin_nontemporal_store(f32x4{v[0], v[1], v[2], v[3]}, reinterpret_cast<f32x4*>(p));
    }
};

// bfloat16 is stored as its raw 16-bit pattern.  Widening is exact (the
// pattern is the upper half of a binary32); narrowing rounds to nearest even
// with the gfx950 packed conversion instruction.
struct bf16_t {
    uint16_t bits;
};

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    __bf16 ha = (__bf16)a;
    __bf16 hb = (__bf16)b;
    return (uint32_t)__builtin_bit_cast(uint16_t, ha) |
           ((uint32_t)__builtin_bit_cast(uint16_t, hb) << 16);
}

template <> struct Vec<bf16_t> {
    static constexpr int N = 8;
    float v[8];
    __device__ __forceinline__ static Vec unpack(u32x4 q) {
        return Vec{{bf16_lo(q.x), bf16_hi(q.x), bf16_lo(q.y), bf16_hi(q.y),
                    bf16_lo(q.z), bf16_hi(q.z), bf16_lo(q.w), bf16_hi(q.w)}};
    }
    __device__ __forceinline__ static Vec load(const bf16_t* p) {
        return unpack(*reinterpret_cast<const u32x4*>(p));
    }
    __device__ __forceinline__ static Vec load_nt(const bf16_t* p) {
        return unpack(__builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p)));
    }
    __device__ __forceinline__ static Vec fill(float f) {
        return Vec{{f, f, f, f, f, f, f, f}};
    }
    __device__ __forceinline__ u32x4 pack() const {
        return u32x4{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]),
                     pack_bf16x2(v[6], v[7])};
    }
    __device__ __forceinline__ void store(bf16_t* p) const {
        *reinterpret_cast<u32x4*>(p) = pack();
    }
    __device__ __forceinline__ void store_nt(bf16_t* p) const {
        __builtin_nontemporal_store(pack(), reinterpret_cast<u32x4*>(p));
    }
};

__device__ __forceinline__ float load1(const float* p) { return *p; }
__device__ __forceinline__ float load1(const bf16_t* p) {
    return __uint_as_float((uint32_t)p->bits << 16);
}
__device__ __forceinline__ void store1(float* p, float v) { *p = v; }
__device__ __forceinline__ void store1(bf16_t* p, float v) {
    __bf16 h = (__bf16)v;
    p->bits = __builtin_bit_cast(uint16_t, h);
}

// ------------------------------------------------------------ normalizer pair
struct MD {
    float s;  // running maximum, scaled by log2(e)
    float d;  // normalizer relative to s
};

__device__ __forceinline__ MD md_empty() { return MD{kEmptyS, 0.0f}; }

// The merge operator of Eq. 4 in base 2.  Symmetric bit for bit:
// merge(a, b) == merge(b, a), since max and + commute in IEEE arithmetic.
__device__ __forceinline__ MD md_merge(MD a, MD b) {
    float S = fmaxf(a.s, b.s);
    return MD{S, a.d * exp2_hw(a.s - S) + b.d * exp2_hw(b.s - S)};
}

// Fold a vector of elements into a pair: the pair of the vector, in which
// every element enters as (x_j, 1), merged into the running pair.  One
// rescale of the running d per vector, one exponential per element.
template <int N>
__device__ __forceinline__ float vec_max(const float (&x)[N]) {
    float mx = x[0];
#pragma unroll
    for (int i = 1; i < N; ++i) mx = fmaxf(mx, x[i]);
    return mx;
}

// As md_fold, with the vector's maximum already at hand.
template <int N>
__device__ __forceinline__ MD md_fold_mx(MD a, const float (&x)[N], float mx) {
    float S = fmaxf(a.s, mx * kLog2e);
    float acc = a.d * exp2_hw(a.s - S);
#pragma unroll
    for (int i = 0; i < N; ++i) acc += exp2_hw(__builtin_fmaf(x[i], kLog2e, -S));
    return MD{S, acc};
}

// Lazy variant for the one-pass loops: the reference s moves only when a
// vector's maximum exceeds it by more than kLazy (in log2 units), so most
// vectors skip the rescale and its exponential.  d = sum 2^{x log2e - s}
// holds for any s; with s >= max * log2e - kLazy every term stays <= 2^kLazy
// (d <= 2^kLazy * V: no overflow for any V < 2^31).
constexpr float kLazy = 8.0f;

template <int N>
__device__ __forceinline__ MD md_fold_lazy(MD a, const float (&x)[N], float mx) {
    const float t = mx * kLog2e;
    if (t > a.s + kLazy) {  // divergent, rarely taken after a lane's first vectors
        a.d *= exp2_hw(a.s - t);
        a.s = t;
    }
    float acc = a.d;
#pragma unroll
    for (int i = 0; i < N; ++i) acc += exp2_hw(__builtin_fmaf(x[i], kLog2e, -a.s));
    return MD{a.s, acc};
}

template <int N>
__device__ __forceinline__ MD md_fold(MD a, const float (&x)[N]) {
    float mx = vec_max(x);
    float S = fmaxf(a.s, mx * kLog2e);
    float acc = a.d * exp2_hw(a.s - S);
#pragma unroll
    for (int i = 0; i < N; ++i) acc += exp2_hw(__builtin_fmaf(x[i], kLog2e, -S));
    return MD{S, acc};
}

__device__ __forceinline__ MD md_fold1(MD a, float x) {
    float S = fmaxf(a.s, x * kLog2e);
    return MD{S, a.d * exp2_hw(a.s - S) + exp2_hw(__builtin_fmaf(x, kLog2e, -S))};
}

// ------------------------------------------------------- lane-group exchange
// Butterfly reductions over aligned groups of G lanes (G a power of two,
// 1..64) entirely in VALU cross-lane operations, no LDS round trips:
//   step 0: DPP quad_perm [1,0,3,2]      (pairs lanes i, i^1)
//   step 1: DPP quad_perm [2,3,0,1]      (pairs lanes i, i^2)
//   step 2: DPP row_half_mirror          (pairs i, 7-i within 8 lanes)
//   step 3: DPP row_mirror               (pairs i, 15-i within 16 lanes)
//   step 4: v_permlane16_swap            (pairs 16-lane rows 2r, 2r+1)
//   step 5: v_permlane32_swap            (pairs the two 32-lane halves)
// After steps 0..k-1 every lane of an aligned group of 2^k lanes holds the
// same bits: at steps 0-1 values are paired with their xor partner; at steps
// 2-3 all lanes of each half of the group already agree, so a mirror pairs
// the halves; at steps 4-5 each swap hands both lanes of a pair the same two
// operands in the same order.  The operator must be commutative bit for bit
// (max, +, and the merge of Eq. 4 as written below are).  All lanes of a
// group must be active.
template <int STEP>
__device__ __forceinline__ void bfly_operands(uint32_t v, uint32_t& a, uint32_t& b) {
    if constexpr (STEP == 0) {
        a = v;
        b = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false);
    } else if constexpr (STEP == 1) {
        a = v;
        b = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false);
    } else if constexpr (STEP == 2) {
        a = v;
        b = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false);
    } else if constexpr (STEP == 3) {
        a = v;
        b = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false);
    } else if constexpr (STEP == 4) {
        auto p = __builtin_amdgcn_permlane16_swap(v, v, false, false);
        a = p[0];
        b = p[1];
    } else {
        static_assert(STEP == 5, "a 64-lane butterfly has six steps");
        auto p = __builtin_amdgcn_permlane32_swap(v, v, false, false);
        a = p[0];
        b = p[1];
    }
}

template <int STEP>
__device__ __forceinline__ void bfly_operands(float v, float& a, float& b) {
    uint32_t ua, ub;
    bfly_operands<STEP>(__float_as_uint(v), ua, ub);
    a = __uint_as_float(ua);
    b = __uint_as_float(ub);
}

template <int STEP>
__device__ __forceinline__ void bfly_operands(MD v, MD& a, MD& b) {
    bfly_operands<STEP>(v.s, a.s, b.s);
    bfly_operands<STEP>(v.d, a.d, b.d);
}

template <int G, int STEP = 0>
__device__ __forceinline__ MD group_merge(MD v) {
    if constexpr ((1 << STEP) < G) {
        MD a, b;
        bfly_operands<STEP>(v, a, b);
        return group_merge<G, STEP + 1>(md_merge(a, b));
    } else {
        return v;
    }
}

template <int G, int STEP = 0>
__device__ __forceinline__ float group_max(float v) {
    if constexpr ((1 << STEP) < G) {
        float a, b;
        bfly_operands<STEP>(v, a, b);
        return group_max<G, STEP + 1>(fmaxf(a, b));
    } else {
        return v;
    }
}

template <int G, int STEP = 0>
__device__ __forceinline__ float group_sum(float v) {
    if constexpr ((1 << STEP) < G) {
        float a, b;
        bfly_operands<STEP>(v, a, b);
        return group_sum<G, STEP + 1>(a + b);
    } else {
        return v;
    }
}

// ------------------------------------------------------------ team reductions
// TEAM <= 64: butterflies inside the lane group.  TEAM > 64 (= the whole
// workgroup): wavefront butterflies, then every thread merges the W
// per-wavefront values from LDS in wavefront order, so all threads hold the
// same bits.
template <int TEAM>
struct Team {
    static constexpr int W = TEAM > 64 ? TEAM / 64 : 1;
    struct Smem {
        MD md[W];
        float f[W];
    };

    __device__ __forceinline__ static MD merge(MD a, Smem& sm) {
        if constexpr (TEAM <= 64) {
            return group_merge<TEAM>(a);
        } else {
            MD w = group_merge<64>(a);
            int wave = threadIdx.x >> 6;
            if ((threadIdx.x & 63) == 0) sm.md[wave] = w;
            __syncthreads();
            MD r = sm.md[0];
#pragma unroll
            for (int i = 1; i < W; ++i) r = md_merge(r, sm.md[i]);
            __syncthreads();
            return r;
        }
    }

    template <bool IS_MAX>
    __device__ __forceinline__ static float reduce(float a, Smem& sm) {
        if constexpr (TEAM <= 64) {
            return IS_MAX ? group_max<TEAM>(a) : group_sum<TEAM>(a);
        } else {
            float w = IS_MAX ? group_max<64>(a) : group_sum<64>(a);
            int wave = threadIdx.x >> 6;
            if ((threadIdx.x & 63) == 0) sm.f[wave] = w;
            __syncthreads();
            float r = sm.f[0];
#pragma unroll
            for (int i = 1; i < W; ++i) r = IS_MAX ? fmaxf(r, sm.f[i]) : r + sm.f[i];
            __syncthreads();
            return r;
        }
    }
};

// Keep LDS traffic between lanes of one wavefront in program order.
__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

}  // namespace osm
