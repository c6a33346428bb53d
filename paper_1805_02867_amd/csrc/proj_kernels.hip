// Projection kernels: the plain projection (logits written out), and the
// projection with the online softmax and top-k fused into its epilogue, so
// that the logits never leave the chip (the Discussion's proposal).
//
// Fused kernel.  Workgroup (c, b) computes P = W . h^T for the vocabulary
// tiles of chunk c against batch rows [128 b, 128 b + 128): with W as the
// MFMA's A operand, each lane's result registers hold 32 vocabulary entries
// of each of two batch rows (columns of P), so a lane keeps, per batch row,
//  * the online pair (s, d) of the entries it has seen (Alg. 3's update,
//    with the reference moved only when the tile maximum passes it by more
//    than kLazy, as in the other one-pass kernels), and
//  * its own sorted list of the K largest keys it has seen (Alg. 4's buffer),
//    entered only by values at or above the list's K-th value.
// The four holders of a batch row in a workgroup (two wavefronts along the
// vocabulary, two lane halves) each write their pair and list as a partial;
// the split top-k merge kernel combines a row's partials (Eq. 4 for the
// pairs, the key order for the lists).
#include "proj.hpp"
#include "topk.hpp"

namespace osm {

// ------------------------------------------------------------ plain logits
__global__ __launch_bounds__(PJ_BLOCK) void proj_logits(const uint16_t* __restrict__ h,
                                                       const uint16_t* __restrict__ w,
                                                       float* __restrict__ out, int64_t N,
                                                       int64_t H, int64_t V) {
    __shared__ ProjSmem sm;
    const int64_t y0 = (int64_t)blockIdx.x * PJ_TY;  // vocabulary
    const int64_t x0 = (int64_t)blockIdx.y * PJ_TX;  // batch
    f32x16 acc[2][2];
    pj_tile(h, N, w, V, H, x0, y0, sm, acc);
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

// One chunk of the vocabulary for one 128-row batch strip.  Partials: per
// batch row, S * 4 of them (chunk c, wavefront wx, lane half), each a pair
// and K keys (0 = none).
template <int KC>
__global__ __launch_bounds__(PJ_BLOCK) void proj_topk_part(
    const uint16_t* __restrict__ h, const uint16_t* __restrict__ w, uint64_t* __restrict__ pkeys,
    MD* __restrict__ pmd, int64_t N, int64_t H, int64_t V, int K, int64_t S, int64_t tiles) {
    __shared__ ProjSmem sm;
    static_assert(sizeof(ProjSmem) >= PJ_BLOCK * 33 * sizeof(float), "epilogue scratch fits");
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wx = wave >> 1, wy = wave & 1;
    const int64_t c = blockIdx.x;
    const int64_t y0 = (int64_t)blockIdx.y * PJ_TY;  // batch strip
    const int64_t v_begin = c * tiles * PJ_TX;
    int64_t v_end = v_begin + tiles * PJ_TX;
    if (v_end > V) v_end = V;

    float sr[2] = {kEmptyS, kEmptyS}, dacc[2] = {0.0f, 0.0f};
    uint64_t L[2][KC];
    uint64_t tkey[2] = {0ull, 0ull};       // K-th key of the list (0 while it has fewer)
    float tval[2] = {-__builtin_inff(), -__builtin_inff()};
#pragma unroll
    for (int ni = 0; ni < 2; ++ni)
#pragma unroll
        for (int i = 0; i < KC; ++i) L[ni][i] = 0ull;

    for (int64_t x0 = v_begin; x0 < v_end; x0 += PJ_TX) {
        f32x16 acc[2][2];
        pj_tile(w, V, h, N, H, x0, y0, sm, acc);
        // vocabulary entry of result register i of block mi: vbase + voff(mi, i)
        const int64_t vbase = x0 + wx * 64 + 4 * (lane >> 5);
        if (x0 + PJ_TX > v_end) {  // the chunk's last tile runs past its end
            const int64_t lim = v_end - vbase;
#pragma unroll
            for (int mi = 0; mi < 2; ++mi)
#pragma unroll
                for (int ni = 0; ni < 2; ++ni)
#pragma unroll
                    for (int i = 0; i < 16; ++i)
                        if (mi * 32 + 8 * (i >> 2) + (i & 3) >= lim) acc[mi][ni][i] = -__builtin_inff();
        }
#pragma unroll
        for (int ni = 0; ni < 2; ++ni) {
            // the lane's 32 entries of batch row (y0 + 64 wy + 32 ni + lane % 32)
            float lm = -__builtin_inff();
#pragma unroll
            for (int mi = 0; mi < 2; ++mi)
#pragma unroll
                for (int i = 0; i < 16; i += 2)
                    lm = max3_raw(lm, acc[mi][ni][i], acc[mi][ni][i + 1]);
            const float t = lm * kLog2e;
            if (__builtin_amdgcn_ballot_w64(t > sr[ni] + kLazy) != 0) {
                if (t > sr[ni] + kLazy) {
                    dacc[ni] *= exp2_hw(sr[ni] - t);
                    sr[ni] = t;
                }
            }
            float dsum = 0.0f;
#pragma unroll
            for (int mi = 0; mi < 2; ++mi)
#pragma unroll
                for (int i = 0; i < 16; ++i)
                    dsum += exp2_hw(__builtin_fmaf(acc[mi][ni][i], kLog2e, -sr[ni]));
            dacc[ni] += dsum;
            if (__builtin_amdgcn_ballot_w64(lm >= tval[ni]) != 0) {
                // Rare path: the lane's 32 entries go to its own slice of the
                // staging LDS (free between tiles: the next tile stores into it
                // only after a workgroup barrier), and one loop walks them, so
                // the list insertion exists once rather than per register.
                float* scr = reinterpret_cast<float*>(&sm) + (wave * 64 + lane) * 33;
#pragma unroll
                for (int mi = 0; mi < 2; ++mi)
#pragma unroll
                    for (int i = 0; i < 16; ++i) scr[mi * 16 + i] = acc[mi][ni][i];
                if (lm >= tval[ni]) {
#pragma unroll 1
                    for (int j = 0; j < 32; ++j) {
                        const float x = scr[j];
                        // masked entries are -inf; a -inf logit is never a candidate
                        if (x >= tval[ni] && x > -__builtin_inff()) {
                            const uint32_t v = (uint32_t)(vbase + (j >> 4) * 32 +
                                                          8 * ((j & 15) >> 2) + (j & 3));
                            const uint64_t key = make_key(x, v);
                            if (key > tkey[ni]) {
                                list_insert<KC>(L[ni], K, key);
                                tkey[ni] = list_kth<KC>(L[ni], K);
                                tval[ni] = tkey[ni] != 0 ? key_value(tkey[ni]) : -__builtin_inff();
                            }
                        }
                    }
                }
            }
        }
    }
    const int64_t Sp = S * 4;
    const int64_t p = c * 4 + wx * 2 + (lane >> 5);
#pragma unroll
    for (int ni = 0; ni < 2; ++ni) {
        const int64_t row = y0 + wy * 64 + ni * 32 + (lane & 31);
        if (row < N) {
            uint64_t* dst = pkeys + (row * Sp + p) * K;
#pragma unroll
            for (int i = 0; i < KC; ++i)
                if (i < K) dst[i] = L[ni][i];
            pmd[row * Sp + p] = MD{sr[ni], dacc[ni]};
        }
    }
}

// ---------------------------------------------------------------- launchers
hipError_t launch_proj_logits(const void* h, const void* w, float* out, int64_t N, int64_t H,
                              int64_t V, hipStream_t st) {
    dim3 grid((unsigned)((V + PJ_TY - 1) / PJ_TY), (unsigned)((N + PJ_TX - 1) / PJ_TX));
    hipLaunchKernelGGL(proj_logits, grid, dim3(PJ_BLOCK), 0, st, (const uint16_t*)h,
                       (const uint16_t*)w, out, N, H, V);
    return hipGetLastError();
}

size_t proj_topk_part_bytes(int64_t N, int64_t S, int K) {
    return (size_t)N * (size_t)(S * 4) * ((size_t)K * 8 + 8);
}

hipError_t launch_proj_topk(const void* h, const void* w, float* vals, int32_t* idx,
                            void* part, int64_t N, int64_t H, int64_t V, int K, int64_t S,
                            int64_t tiles, hipStream_t st) {
    uint64_t* pkeys = static_cast<uint64_t*>(part);
    MD* pmd = reinterpret_cast<MD*>(pkeys + N * S * 4 * K);
    dim3 grid((unsigned)S, (unsigned)((N + PJ_TY - 1) / PJ_TY));
    if (K <= 8)
        hipLaunchKernelGGL((proj_topk_part<8>), grid, dim3(PJ_BLOCK), 0, st, (const uint16_t*)h,
                           (const uint16_t*)w, pkeys, pmd, N, H, V, K, S, tiles);
    else
        hipLaunchKernelGGL((proj_topk_part<16>), grid, dim3(PJ_BLOCK), 0, st, (const uint16_t*)h,
                           (const uint16_t*)w, pkeys, pmd, N, H, V, K, S, tiles);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    constexpr int WB = TK_BLOCK / 64;
    dim3 mgrid((unsigned)((N + WB - 1) / WB));
    hipLaunchKernelGGL((topk_merge<TK_ONLINE>), mgrid, dim3(TK_BLOCK), 0, st, pkeys, pmd, vals,
                       idx, N, S * 4, K);
    return hipGetLastError();
}

}  // namespace osm
