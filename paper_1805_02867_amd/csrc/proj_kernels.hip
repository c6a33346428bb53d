// Projection kernels: the plain projection (logits written out), and the
// projection with the online softmax and top-k fused into its epilogue, so
// that the logits never leave the chip (the Discussion's proposal).
//
// Fused kernel.  Workgroup (c, b) computes P = W . h^T for the vocabulary
// tiles of chunk c against batch rows [128 b, 128 b + 128): with W as the
// MFMA's A operand, each lane's result registers hold 64 vocabulary entries
// of one batch row (a column of P) per tile, so a lane keeps, for that row,
//  * the online pair (s, d) of the entries it has seen (Alg. 3's update,
//    with the reference moved only when the tile maximum passes it by more
//    than kLazy, as in the other one-pass kernels), and
//  * its own sorted list of the K largest keys it has seen (Alg. 4's buffer),
//    entered only by values at or above the list's K-th value.
// The two holders of a batch row in a workgroup (the two lane halves) each
// write their pair and list as a partial;
// the split top-k merge kernel combines a row's partials (Eq. 4 for the
// pairs, the key order for the lists).
#include "proj.hpp"
#include "topk.hpp"

namespace osm {

// ------------------------------------------------------------ plain logits
// Tiles in grouped order: groups of up to 8 batch strips, each taken across
// all vocabulary tiles before the next group, so that a contiguous block of
// logical ids covers a compact block of tiles.
constexpr int64_t PJ_GROUP = 8;

__global__ __launch_bounds__(PJ_BLOCK) void proj_logits(const uint16_t* __restrict__ h,
                                                       const uint16_t* __restrict__ w,
                                                       float* __restrict__ out, int64_t N,
                                                       int64_t H, int64_t V, int64_t per) {
    __shared__ ProjSmem sm;
    const int64_t nb = (N + PJ_TX - 1) / PJ_TX, nt = (V + PJ_TY - 1) / PJ_TY;
    const int64_t L = xcd_logical(blockIdx.x, per);
    if (L >= nb * nt) return;  // the whole workgroup leaves
    const int64_t in_group = PJ_GROUP * nt;
    const int64_t first = (L / in_group) * PJ_GROUP;
    const int64_t gsize = nb - first < PJ_GROUP ? nb - first : PJ_GROUP;
    const int64_t x0 = (first + (L % in_group) % gsize) * PJ_TX;  // batch
    const int64_t y0 = ((L % in_group) / gsize) * PJ_TY;          // vocabulary
    f32x16 acc[2][2];
    pj_tile<2, 2>(h, N, w, V, H, x0, y0, sm, acc);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wx = wave >> 1, wy = wave & 1;
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int64_t row = x0 + wx * 64 + mi * 32 + row_in_32(i, lane);
                const int64_t col = y0 + wy * 64 + ni * 32 + (lane & 31);
                if (row < N && col < V) out[row * V + col] = acc[mi][ni][i];
            }
}

// ------------------------------------------------------------ fused top-k
// Insert `key` into the lane's list (descending, K valid entries in a
// register array of KC, unused entries 0); the caller has checked that key
// exceeds the K-th entry.  Every entry moves at most one place, computed
// from the old list, so all positions update at once.
template <int KC>
__device__ __forceinline__ void list_insert(uint64_t (&L)[KC], int K, uint64_t key) {
    uint64_t prev = L[0];
    L[0] = key > L[0] ? key : L[0];
#pragma unroll
    for (int i = 1; i < KC; ++i) {
        const uint64_t cur = L[i];
        const uint64_t moved = key > prev ? prev : (key > cur ? key : cur);
        L[i] = i < K ? moved : cur;
        prev = cur;
    }
}

template <int KC>
__device__ __forceinline__ uint64_t list_kth(const uint64_t (&L)[KC], int K) {
    uint64_t t = 0;
#pragma unroll
    for (int i = 0; i < KC; ++i) t = (i == K - 1) ? L[i] : t;
    return t;
}

// One chunk of the vocabulary for one 128-row batch strip.  The four
// wavefronts sit side by side along the batch (each 128 vocabulary entries x
// 32 batch rows, 4 x 1 blocks), so lane l of wavefront w holds, for batch row
// 32 w + l % 32 of the strip, 64 vocabulary entries of each tile: the entries
// 32 mi + row_in_32(i, l) for result register i of block mi.  The two lane
// halves of a batch row each write a partial: 2 S per row (chunk, half), each
// a pair and K keys (0 = none).
template <int KC>
__global__ __launch_bounds__(PJ_BLOCK) __attribute__((amdgpu_waves_per_eu(2, 2))) void proj_topk_part(
    const uint16_t* __restrict__ h, const uint16_t* __restrict__ w, uint64_t* __restrict__ pkeys,
    MD* __restrict__ pmd, int64_t N, int64_t H, int64_t V, int K, int64_t S, int64_t tiles,
    int64_t per) {
    __shared__ ProjSmem sm;
    static_assert(sizeof(ProjSmem) >= PJ_BLOCK * 64 * sizeof(float), "epilogue scratch fits");
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    // logical id = chunk * strips + strip: an XCD's workgroups take all batch
    // strips of the same chunks, so each weight tile is read into its L2 once
    const int64_t nb = (N + PJ_TY - 1) / PJ_TY;
    const int64_t lid = xcd_logical(blockIdx.x, per);
    if (lid >= S * nb) return;  // the whole workgroup leaves
    const int64_t c = lid / nb;
    const int64_t y0 = (lid % nb) * PJ_TY;  // batch strip
    const int64_t v_begin = c * tiles * PJ_TX;
    int64_t v_end = v_begin + tiles * PJ_TX;
    if (v_end > V) v_end = V;

    float sr = kEmptyS, dacc = 0.0f;
    uint64_t L[KC];
    uint64_t tkey = 0ull;  // K-th key of the list (0 while it has fewer)
    float tval = -__builtin_inff();
#pragma unroll
    for (int i = 0; i < KC; ++i) L[i] = 0ull;

    for (int64_t x0 = v_begin; x0 < v_end; x0 += PJ_TX) {
        f32x16 acc[4][1];
        pj_tile<1, 4>(w, V, h, N, H, x0, y0, sm, acc);
        // vocabulary entry of result register i of block mi: vbase + voff(mi, i)
        const int64_t vbase = x0 + 4 * (lane >> 5);
        if (x0 + PJ_TX > v_end) {  // the chunk's last tile runs past its end
            const int64_t lim = v_end - vbase;
#pragma unroll
            for (int mi = 0; mi < 4; ++mi)
#pragma unroll
                for (int i = 0; i < 16; ++i)
                    if (mi * 32 + 8 * (i >> 2) + (i & 3) >= lim) acc[mi][0][i] = -__builtin_inff();
        }
        float lm = -__builtin_inff();
#pragma unroll
        for (int mi = 0; mi < 4; ++mi)
#pragma unroll
            for (int i = 0; i < 16; i += 2) lm = max3_raw(lm, acc[mi][0][i], acc[mi][0][i + 1]);
        const float t = lm * kLog2e;
        if (__builtin_amdgcn_ballot_w64(t > sr + kLazy) != 0) {
            if (t > sr + kLazy) {
                dacc *= exp2_hw(sr - t);
                sr = t;
            }
        }
        float dsum[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int mi = 0; mi < 4; ++mi)
#pragma unroll
            for (int i = 0; i < 16; ++i)
                dsum[mi] += exp2_hw(__builtin_fmaf(acc[mi][0][i], kLog2e, -sr));
        dacc += (dsum[0] + dsum[1]) + (dsum[2] + dsum[3]);
        if (__builtin_amdgcn_ballot_w64(lm >= tval) != 0) {
            // Rare path: the lane's 64 entries go to its own column of the
            // staging LDS (free between tiles: the next tile writes it only
            // after a workgroup barrier), and one loop walks them, so the list
            // insertion exists once rather than per register.
            float* scr = reinterpret_cast<float*>(&sm) + threadIdx.x;
#pragma unroll
            for (int mi = 0; mi < 4; ++mi)
#pragma unroll
                for (int i = 0; i < 16; ++i) scr[(mi * 16 + i) * PJ_BLOCK] = acc[mi][0][i];
            if (lm >= tval) {
#pragma unroll 1
                for (int j = 0; j < 64; ++j) {
                    const float x = scr[j * PJ_BLOCK];
                    // masked entries are -inf; a -inf logit is never a candidate
                    if (x >= tval && x > -__builtin_inff()) {
                        const uint32_t v = (uint32_t)(vbase + (j >> 4) * 32 +
                                                      8 * ((j & 15) >> 2) + (j & 3));
                        const uint64_t key = make_key(x, v);
                        if (key > tkey) {
                            list_insert<KC>(L, K, key);
                            tkey = list_kth<KC>(L, K);
                            tval = tkey != 0 ? key_value(tkey) : -__builtin_inff();
                        }
                    }
                }
            }
        }
    }
    const int64_t Sp = S * 2;
    const int64_t p = c * 2 + (lane >> 5);
    const int64_t row = y0 + wave * 32 + (lane & 31);
    if (row < N) {
        uint64_t* dst = pkeys + (row * Sp + p) * K;
#pragma unroll
        for (int i = 0; i < KC; ++i)
            if (i < K) dst[i] = L[i];
        pmd[row * Sp + p] = MD{sr, dacc};
    }
}

// ---------------------------------------------------------------- launchers
hipError_t launch_proj_logits(const void* h, const void* w, float* out, int64_t N, int64_t H,
                              int64_t V, hipStream_t st) {
    const int64_t total = ((N + PJ_TX - 1) / PJ_TX) * ((V + PJ_TY - 1) / PJ_TY);
    const int64_t per = (total + 7) / 8;
    hipLaunchKernelGGL(proj_logits, dim3((unsigned)(8 * per)), dim3(PJ_BLOCK), 0, st,
                       (const uint16_t*)h, (const uint16_t*)w, out, N, H, V, per);
    return hipGetLastError();
}

size_t proj_topk_part_bytes(int64_t N, int64_t S, int K) {
    return (size_t)N * (size_t)(S * 2) * ((size_t)K * 8 + 8);
}

hipError_t launch_proj_topk(const void* h, const void* w, float* vals, int32_t* idx,
                            void* part, int64_t N, int64_t H, int64_t V, int K, int64_t S,
                            int64_t tiles, hipStream_t st) {
    uint64_t* pkeys = static_cast<uint64_t*>(part);
    MD* pmd = reinterpret_cast<MD*>(pkeys + N * S * 2 * K);
    const int64_t per = (S * ((N + PJ_TY - 1) / PJ_TY) + 7) / 8;
    dim3 grid((unsigned)(8 * per));
    if (K <= 8)
        hipLaunchKernelGGL((proj_topk_part<8>), grid, dim3(PJ_BLOCK), 0, st, (const uint16_t*)h,
                           (const uint16_t*)w, pkeys, pmd, N, H, V, K, S, tiles, per);
    else
        hipLaunchKernelGGL((proj_topk_part<16>), grid, dim3(PJ_BLOCK), 0, st, (const uint16_t*)h,
                           (const uint16_t*)w, pkeys, pmd, N, H, V, K, S, tiles, per);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    constexpr int WB = TK_BLOCK / 64;
    dim3 mgrid((unsigned)((N + WB - 1) / WB));
    hipLaunchKernelGGL((topk_merge<TK_ONLINE>), mgrid, dim3(TK_BLOCK), 0, st, pkeys, pmd, vals,
                       idx, N, S * 2, K);
    return hipGetLastError();
}

}  // namespace osm
