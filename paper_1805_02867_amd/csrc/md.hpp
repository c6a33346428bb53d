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
__device__ __forceinline__ MD md_fold(MD a, const float (&x)[N]) {
    float mx = x[0];
#pragma unroll
    for (int i = 1; i < N; ++i) mx = fmaxf(mx, x[i]);
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
// Value of lane (lane ^ MASK); MASK < 64.  Quad permutations for 1 and 2,
// the LDS crossbar swizzle (no memory traffic) for 4..16, and a bpermute for
// 32.  All lanes taking part must be active.
template <int MASK>
__device__ __forceinline__ float xor_lane(float v) {
    int i = __float_as_int(v);
    int r;
    if constexpr (MASK == 1) {
        r = __builtin_amdgcn_update_dpp(0, i, 0xB1, 0xF, 0xF, false);  // [1,0,3,2]
    } else if constexpr (MASK == 2) {
        r = __builtin_amdgcn_update_dpp(0, i, 0x4E, 0xF, 0xF, false);  // [2,3,0,1]
    } else if constexpr (MASK == 4 || MASK == 8 || MASK == 16) {
        r = __builtin_amdgcn_ds_swizzle(i, (MASK << 10) | 0x1F);
    } else {
        static_assert(MASK == 32, "xor_lane: mask must be a power of two below 64");
        int src = ((int)__lane_id() ^ 32) << 2;
        r = __builtin_amdgcn_ds_bpermute(src, i);
    }
    return __int_as_float(r);
}

template <int MASK>
__device__ __forceinline__ uint32_t xor_lane_u(uint32_t v) {
    return (uint32_t)__float_as_int(xor_lane<MASK>(__int_as_float((int)v)));
}

// Butterfly reductions over aligned groups of G lanes (G a power of two,
// 1..64).  Every lane of a group ends with the same value bit for bit: each
// step combines a value with its partner's through a symmetric operator.
template <int G, int MASK = 1>
__device__ __forceinline__ MD group_merge(MD a) {
    if constexpr (MASK < G) {
        MD b{xor_lane<MASK>(a.s), xor_lane<MASK>(a.d)};
        return group_merge<G, MASK * 2>(md_merge(a, b));
    } else {
        return a;
    }
}

template <int G, int MASK = 1>
__device__ __forceinline__ float group_max(float a) {
    if constexpr (MASK < G) {
        return group_max<G, MASK * 2>(fmaxf(a, xor_lane<MASK>(a)));
    } else {
        return a;
    }
}

template <int G, int MASK = 1>
__device__ __forceinline__ float group_sum(float a) {
    if constexpr (MASK < G) {
        return group_sum<G, MASK * 2>(a + xor_lane<MASK>(a));
    } else {
        return a;
    }
}

// Keep LDS traffic between lanes of one wavefront in program order.
__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

}  // namespace osm
