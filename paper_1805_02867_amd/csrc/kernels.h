// Host-side launchers of the device kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace osm {

// Row kernels: team = lanes per row (4..64 inside a wavefront, 128..1024 one
// row per workgroup).  vec: x and y rows may be read / written as 16-byte
// vectors (x and y congruent modulo 16 bytes).
hipError_t launch_softmax_rows(const void* x, void* y, int64_t N, int64_t V, int dtype,
                               int mode, int team, bool vec, hipStream_t st);

// Split-V: S chunks of `chunk` elements per row; scratch holds N * S float2.
hipError_t launch_softmax_split(const void* x, void* y, void* scratch, int64_t N, int64_t V,
                                int dtype, int mode, int64_t S, int64_t chunk, bool vec,
                                hipStream_t st);

// Row-resident online softmax: one row per workgroup of `block` threads,
// r 16-byte vectors per lane held in registers; vec: y congruent with x
// modulo 16 bytes (vector stores), else outputs stored one by one.
hipError_t launch_softmax_resident(const void* x, void* y, int64_t N, int64_t V, int dtype,
                                   int block, int r, bool vec, hipStream_t st);

// Projection (bfloat16 h: N x H, w: V x H, H a multiple of 8 and at most
// 2^20, 16-byte aligned): logits = h . w^T in binary32; cus = compute units.
hipError_t launch_proj_logits(const void* h, const void* w, float* out, int64_t N, int64_t H,
                              int64_t V, int cus, hipStream_t st);

// Projection fused with the online softmax and top-k: S vocabulary chunks of
// `tiles` tiles each, `parts` partials per (row, chunk) (proj_topk_shape
// picks all three for a device with `cus` compute units); part holds
// proj_topk_part_bytes(N, S, parts, K) bytes.
void proj_topk_shape(int64_t N, int64_t V, int K, int cus, int64_t* S, int64_t* tiles,
                     int* parts);
size_t proj_topk_part_bytes(int64_t N, int64_t S, int parts, int K);
hipError_t launch_proj_topk(const void* h, const void* w, float* vals, int32_t* idx,
                            void* part, int64_t N, int64_t H, int64_t V, int K, int64_t S,
                            int64_t tiles, int parts, hipStream_t st);

// Reference streaming kernels (measurement only): op 0 reads `vecs` 16-byte
// vectors of x (y: a 1 KB sink, written only for a sum never met), op 1
// copies them to y.
hipError_t launch_ref_stream(int op, const void* x, void* y, int64_t vecs, int cus,
                             hipStream_t st);

// What the top-k kernels compute next to the selection (Section 4, and the
// comparisons of Section 5.2):
//  TK_ONLINE: the online pair, one pass (Alg. 4);
//  TK_SAFE:   a maximum pass over the row first, then the normalizer with
//             that maximum held fixed, in the pass that selects (the safe
//             softmax fused with top-k: two loads per element);
//  TK_VALUES: no softmax; the outputs are the selected inputs themselves
//             (the separate top-k of the unfused comparisons).
enum TopkVar { TK_ONLINE = 0, TK_SAFE = 1, TK_VALUES = 2 };

struct TopkLaunch {
    const void* x;
    float* vals;
    int32_t* idx;
    void* part;          // split scratch (S > 1): topk_part_bytes(N, S, K) bytes
    int64_t N, V;
    int K;
    int waves_per_row;   // S <= 1: 1, 2 (TK_ONLINE only) or 4
    int64_t S, chunk;    // chunks per row and their length in elements (S > 1)
    hipStream_t st;
    // S > 1: N zeroed per-row counters, so that each row's last chunk merges
    // the row in the same kernel (the counters are left zeroed); null: a
    // second kernel merges.
    uint32_t* ctr = nullptr;
};

// Split scratch: N * S * K 64-bit keys, then N * S normalizer pairs.
inline size_t topk_part_bytes(int64_t N, int64_t S, int64_t K) {
    return (size_t)N * (size_t)S * ((size_t)K * 8 + 8);
}

hipError_t launch_topk_online_f32(const TopkLaunch& a);
hipError_t launch_topk_online_bf16(const TopkLaunch& a);
hipError_t launch_topk_safe_f32(const TopkLaunch& a);
hipError_t launch_topk_safe_bf16(const TopkLaunch& a);
hipError_t launch_topk_values_f32(const TopkLaunch& a);
hipError_t launch_topk_values_bf16(const TopkLaunch& a);

inline hipError_t launch_topk(const TopkLaunch& a, int dtype, int var) {
    const bool bf = dtype == 1;
    switch (var) {
        case TK_ONLINE: return bf ? launch_topk_online_bf16(a) : launch_topk_online_f32(a);
        case TK_SAFE: return bf ? launch_topk_safe_bf16(a) : launch_topk_safe_f32(a);
        case TK_VALUES: return bf ? launch_topk_values_bf16(a) : launch_topk_values_f32(a);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace osm
