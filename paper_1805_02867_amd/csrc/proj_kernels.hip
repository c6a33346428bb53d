// Projection kernels: the plain projection (logits written out), and the
// projection with the online softmax and top-k fused into its epilogue, so
// that the logits never leave the chip (the Discussion's proposal).
//
// Fused kernel.  Workgroup (c, b) computes P = W . h^T for the vocabulary
// tiles of chunk c against a strip of batch rows: with W as the MFMA's A
// operand, each lane's result registers hold, per tile, a run of vocabulary
// entries of each of its batch rows (columns of P), so a lane keeps, for each
// of those rows,
//  * the online pair (s, d) of the entries it has seen (Alg. 3's update,
//    with the reference moved only when the tile maximum passes it by more
//    than kLazy, as in the other one-pass kernels), and
//  * its own sorted list of the K largest keys it has seen (Alg. 4's buffer),
//    entered only by values at or above the list's K-th value.
// Every holder of a batch row in a workgroup (two lane halves in each
// wavefront along the vocabulary) writes its pair and list as a partial;
// the split top-k merge kernel combines a row's partials (Eq. 4 for the
// pairs, the key order for the lists).
#include "proj.hpp"
#include "topk.hpp"

namespace osm {

// Plain logits: 256 x 256 tiles for eight wavefronts when the tile count
// fills the chip twice over, else 128 x 128 tiles for four (two workgroups
// per CU), which keep small problems spread over more CUs.
using PjBig = PjCfg<256, 256, 2, 4>;
using PjSmall = PjCfg<128, 128, 2, 2>;
// Fused, by batch size and K (the vocabulary tile is 256 entries in all; the
// lanes' top-K lists live in registers):
//  * 256 x 256 (K <= 8, N > 128): 2 x 4 wavefronts, two batch rows per lane;
//    128 result registers and at most 128 others per lane, so two
//    wavefronts share each SIMD and one's epilogue overlaps the other's
//    products;
//  * 256 x 128 in 2 x 4 wavefronts (8 < K <= 16, N > 1024): one batch row per
//    lane, also two wavefronts per SIMD;
//  * 256 x 128 in 1 x 4 wavefronts (otherwise, N > 64): one batch row per
//    lane, one wavefront per SIMD, measured faster than the 2 x 4 layout up
//    to N = 512;
//  * 256 x 64 (N <= 64): 2 x 2 wavefronts, one batch row per lane, so small
//    batches do not pay for a strip of 256 rows.
using PjFused8 = PjCfg<256, 256, 2, 4>;
using PjFused16W = PjCfg<256, 128, 2, 4>;
using PjFused16 = PjCfg<256, 128, 1, 4>;
using PjFusedN = PjCfg<256, 64, 2, 2>;
static int fused_cfg(int64_t N, int K) {
    if (N <= 64) return 3;
    if (K <= 8 && N > 128) return 0;
    return K > 8 && N > 1024 ? 1 : 2;
}

// ------------------------------------------------------------ plain logits
// Tiles in grouped order: groups of up to 8 batch strips, each taken across
// all vocabulary tiles before the next group, so that a contiguous block of
// logical ids covers a compact block of tiles.
constexpr int64_t PJ_GROUP = 8;

template <class C>
__global__ __launch_bounds__(C::NT) void proj_logits(const uint16_t* __restrict__ h,
                                                     const uint16_t* __restrict__ w,
                                                     float* __restrict__ out, int64_t N,
                                                     int64_t H, int64_t V, int64_t per) {
    __shared__ typename C::Smem sm;
    const int64_t nb = (N + C::TX - 1) / C::TX, nt = (V + C::TY - 1) / C::TY;
    const int64_t lid = xcd_logical(blockIdx.x, per);
    if (lid >= nb * nt) return;  // the whole workgroup leaves
    const int64_t in_group = PJ_GROUP * nt;
    const int64_t first = (lid / in_group) * PJ_GROUP;
    const int64_t gsize = nb - first < PJ_GROUP ? nb - first : PJ_GROUP;
    const int64_t bx0 = (first + (lid % in_group) % gsize) * C::TX;  // batch
    const int64_t vy0 = ((lid % in_group) / gsize) * C::TY;          // vocabulary
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wx = wave / C::WY, wy = wave % C::WY;
    pj_run<C>(
        h, N, w, V, H, 0, 1, sm,
        [&](int64_t, int64_t& x0, int64_t& y0) {
            x0 = bx0;
            y0 = vy0;
        },
        [&](int64_t, int64_t x0, int64_t y0, f32x16 (&acc)[C::MI][C::NI]) {
            // streaming stores: the logits are not read again by this kernel
            // (measured 11-12% faster at 4000 x 1024 x 32000, also for a top-k
            // reading them next; neutral at H = 4096)
#pragma unroll
            for (int mi = 0; mi < C::MI; ++mi)
#pragma unroll
                for (int ni = 0; ni < C::NI; ++ni)
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        const int64_t row = x0 + wx * 32 * C::MI + mi * 32 + row_in_32(i, lane);
                        const int64_t col = y0 + wy * 32 * C::NI + ni * 32 + (lane & 31);
                        if (row < N && col < V)
                            __builtin_nontemporal_store(acc[mi][ni][i], out + row * V + col);
                    }
        });
}

// ------------------------------------------------------------ fused top-k
constexpr int64_t PJ_CB = 4, PJ_SB = 8;  // block of chunks x batch strips per XCD

// Insert `key` into a lane's list (descending, K valid entries in a
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

// A copy of an accumulator register made where it is used.  Left to itself
// the compiler moves every accumulator of the tile into vector registers at
// once when the products end (they are read by vector instructions from
// then on), which overflows the register file; reading each one through
// this keeps the accumulators where the products left them.
__device__ __forceinline__ float acc_reread(float a) {
    float r;
    asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(r) : "a"(a));
    return r;
}

// Bit j of a candidate mask for entry x against threshold t, set when x is
// below t: the sign of x - t, moved to bit j in vector registers (a compare
// would give a wave-wide scalar mask per entry, and the compiler keeps many
// of those alive at once).  x == t gives +0, i.e. not below; a NaN
// difference may set either value, and every candidate is checked again
// before it is offered.
__device__ __forceinline__ uint32_t below_bit(float x, float t, int j) {
    return (__float_as_uint(x - t) >> 31) << j;
}

// A lane's top-K list: KC registers of descending keys, K valid, unused
// entries 0.
template <int KC>
struct LaneList {
    uint64_t L[KC];
    __device__ __forceinline__ void init() {
#pragma unroll
        for (int i = 0; i < KC; ++i) L[i] = 0ull;
    }
    // insert (key > K-th entry); returns the new K-th entry
    __device__ __forceinline__ uint64_t insert(int K, uint64_t key) {
        list_insert<KC>(L, K, key);
        return list_kth<KC>(L, K);
    }
};

// One chunk of vocabulary tiles [c * tiles, min((c + 1) * tiles, nt)) for one
// batch strip of TY rows.  Lane l of wavefront (wx, wy) holds, for batch rows
// 32 (NI wy + ni) + l % 32 (ni < NI) of the strip, the entries
// vbase + 32 mi + 8 (i / 4) + i % 4 (vbase = tile start + 32 MI wx + 4 (l / 32),
// mi < MI) in result register i of block (mi, ni).  The partial of a (row, chunk) pair
// written by this lane is p = 2 (WX c + wx) + l / 32: 2 WX S per row, each a
// pair and K keys (0 = none).
template <class C, int KC>
__global__ __launch_bounds__(C::NT) void proj_topk_part(
    const uint16_t* __restrict__ h, const uint16_t* __restrict__ w, uint64_t* __restrict__ pkeys,
    MD* __restrict__ pmd, int64_t N, int64_t H, int64_t V, int K, int64_t S, int64_t tiles,
    int64_t per) {
    constexpr int NI = C::NI;
    constexpr int E = C::MI * 16;  // entries per row per lane and tile
    // entries per pass of the LDS column: the largest power of two that fits a stage
    constexpr int EC = sizeof(typename C::Stage) >= C::NT * 64 * sizeof(float)   ? 64
                       : sizeof(typename C::Stage) >= C::NT * 32 * sizeof(float) ? 32
                                                                                 : 16;
    static_assert(sizeof(typename C::Stage) >= C::NT * EC * sizeof(float), "scratch fits");
    __shared__ typename C::Smem sm;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wx = wave / C::WY, wy = wave % C::WY;
    // Logical ids in blocks of PJ_CB chunks x up to PJ_SB batch strips, so
    // that the workgroups of an XCD (a contiguous range of ids) share few
    // operand tiles in its L2: a block of 4 x 8 reads 12 distinct tiles per
    // step where 2 chunks x 16 strips would read 18.
    const int64_t nb = (N + C::TY - 1) / C::TY, nt = (V + C::TX - 1) / C::TX;
    const int64_t sb = nb < PJ_SB ? nb : PJ_SB, nsb = (nb + sb - 1) / sb;
    const int64_t lid = xcd_logical(blockIdx.x, per);
    const int64_t blk = lid / (PJ_CB * sb), in = lid % (PJ_CB * sb);
    const int64_t c = (blk / nsb) * PJ_CB + in / sb;
    const int64_t strip = (blk % nsb) * sb + in % sb;
    if (c >= S || strip >= nb) return;  // the whole workgroup leaves
    const int64_t y0s = strip * C::TY;  // batch strip
    const int64_t t0 = c * tiles;
    const int64_t t1 = t0 + tiles < nt ? t0 + tiles : nt;

    float sr[NI], dacc[NI], tval[NI];
    uint64_t tkey[NI];  // K-th key of the list (0 while it has fewer)
    LaneList<KC> list[NI];
#pragma unroll
    for (int ni = 0; ni < NI; ++ni) {
        sr[ni] = kEmptyS;
        dacc[ni] = 0.0f;
        tval[ni] = -__builtin_inff();
        tkey[ni] = 0ull;
        list[ni].init();
    }
    float* scr = reinterpret_cast<float*>(&sm.st[1]) + threadIdx.x;  // this thread's column

    pj_run<C>(
        w, V, h, N, H, t0, t1, sm,
        [&](int64_t t, int64_t& x0, int64_t& y0) {
            x0 = t * C::TX;
            y0 = y0s;
        },
        [&](int64_t, int64_t x0, int64_t, f32x16 (&acc)[C::MI][C::NI]) {
            constexpr int E = C::MI * 16;  // entries per row per lane
            // groups of GS consecutive entries: 8, or fewer so that there
            // are at least KC groups (the bootstrap below needs K of them)
            constexpr int GS = E / KC < 8 ? E / KC : 8;
            constexpr int NG = E / GS;
            static_assert(GS % 2 == 0 && NG >= KC, "groups hold whole entry pairs");
            const int64_t vbase = x0 + wx * 32 * C::MI + 4 * (lane >> 5);
            // offset from vbase of entry j (block j / 16, register j % 16)
            auto voff = [](int j) { return (j >> 4) * 32 + 8 * ((j & 15) >> 2) + (j & 3); };
            // Alg. 4's insertion, for an entry already known to be >= tval[ni]
            auto offer = [&](int ni, float xv, int j) {
                const uint64_t key = make_key(xv, (uint32_t)(vbase + voff(j)));
                if (key > tkey[ni]) {
                    tkey[ni] = list[ni].insert(K, key);
                    // until the list holds K keys the threshold stays as it is
                    if (tkey[ni] != 0) tval[ni] = key_value(tkey[ni]);
                }
            };
            // entries [q EC, q EC + EC) of row ni into this thread's LDS column
            auto stage = [&](int ni, int q) {
#pragma unroll
                for (int j = 0; j < EC; ++j)
                    scr[j * C::NT] = acc_reread(acc[(q * EC + j) >> 4][ni][j & 15]);
            };
            // The vocabulary's last tile may run past V (once per chunk at
            // most): entries at offsets >= lim do not exist.
            const bool ragged = x0 + C::TX > V;
            const int lim = ragged ? (int)(V - vbase) : 1 << 30;
#pragma unroll
            for (int ni = 0; ni < NI; ++ni) {
                // 1. One pass over the row's entries (the only code unrolled
                //    over them): the maxima of groups of GS, the terms against
                //    the current reference and the entries below the list's
                //    K-th value (tval only rises, so every entry that can still
                //    enter the list is outside that set).
                float bm[NG];
                float dsum[4] = {0.0f, 0.0f, 0.0f, 0.0f};
                uint32_t cm[E / 32];
#pragma unroll
                for (int g = 0; g < NG; ++g) bm[g] = -__builtin_inff();
#pragma unroll
                for (int u = 0; u < E / 32; ++u) cm[u] = 0u;
                if (!ragged) {
                    const float th = tval[ni];
#pragma unroll
                    for (int j = 0; j < E; j += 2) {
                        const float a0 = acc_reread(acc[j >> 4][ni][j & 15]);
                        const float a1 = acc_reread(acc[(j + 1) >> 4][ni][(j + 1) & 15]);
                        bm[j / GS] = max3_raw(bm[j / GS], a0, a1);
                        dsum[j & 3] += exp2_hw(__builtin_fmaf(a0, kLog2e, -sr[ni]));
                        dsum[(j + 1) & 3] += exp2_hw(__builtin_fmaf(a1, kLog2e, -sr[ni]));
                        cm[j >> 5] |= below_bit(a0, th, j & 31) | below_bit(a1, th, (j + 1) & 31);
                    }
                } else {
#pragma unroll
                    for (int j = 0; j < E; ++j) {
                        const float a = acc_reread(acc[j >> 4][ni][j & 15]);
                        bm[j / GS] = __builtin_fmaxf(bm[j / GS], voff(j) < lim ? a : -__builtin_inff());
                    }
                }
                float lm = bm[0];
#pragma unroll
                for (int g = 1; g < NG; ++g) lm = __builtin_fmaxf(lm, bm[g]);
                // 2. Alg. 3: move the reference when some lane's maximum
                //    passes it by more than kLazy (the chunk's first tile, then
                //    rarely); the terms are then summed again below.
                bool recompute = ragged;
                const float tm = lm * kLog2e;
                if (__builtin_amdgcn_ballot_w64(tm > sr[ni] + kLazy) != 0) {
                    if (tm > sr[ni] + kLazy) {
                        dacc[ni] *= exp2_hw(sr[ni] - tm);
                        sr[ni] = tm;
                    }
                    recompute = true;
                }
                // 3. A chunk's first tile: the list is empty and every entry
                //    would be a candidate.  The group maxima are entries of
                //    distinct groups, so their K-th largest value (ties counted
                //    once, which only lowers it) is a value that at least K of
                //    the lane's entries reach: a valid threshold, shared with
                //    the other lane holding the row.  The candidates are then
                //    found again below.
                bool remask = ragged;
                if (__builtin_amdgcn_ballot_w64(tval[ni] == -__builtin_inff()) != 0) {
                    if (K <= NG && tval[ni] == -__builtin_inff()) {
                        float b[NG], boot = -__builtin_inff();
#pragma unroll
                        for (int g = 0; g < NG; ++g) b[g] = bm[g];
#pragma unroll 1
                        for (int r = 0; r < K; ++r) {
                            float m = b[0];
#pragma unroll
                            for (int g = 1; g < NG; ++g) m = __builtin_fmaxf(m, b[g]);
#pragma unroll
                            for (int g = 0; g < NG; ++g) b[g] = b[g] == m ? -__builtin_inff() : b[g];
                            boot = m;
                        }
                        tval[ni] = boot;
                    }
                    tval[ni] = __builtin_fmaxf(tval[ni], __shfl_xor(tval[ni], 32));
                    remask = true;
                }
                float ds = recompute ? 0.0f : (dsum[0] + dsum[1]) + (dsum[2] + dsum[3]);
                // 4. Per part of EC entries, when anything is left to do, the
                //    part goes to this thread's column of the free LDS stage
                //    (the one copy of the part's registers in the code), and
                //    rolled loops finish the work: the terms again after a
                //    move of the reference, the candidates again after the
                //    bootstrap or on the ragged tile (with the bound), then
                //    Alg. 4's insertion of each candidate.
#pragma unroll
                for (int q = 0; q < E / EC; ++q) {
                    uint64_t m = 0;  // candidates of this part
                    if constexpr (EC >= 32) {
#pragma unroll
                        for (int u = 0; u < EC / 32; ++u)
                            m |= (uint64_t)~cm[q * (EC / 32) + u] << (32 * u);
                    } else {
                        m = (~cm[q * EC / 32] >> (q * EC % 32)) & ((1u << EC) - 1u);
                    }
                    if (!recompute && !remask && __builtin_amdgcn_ballot_w64(m != 0) == 0) continue;
                    stage(ni, q);
                    if (recompute || remask) {
                        const float tv = tval[ni], s = sr[ni];
                        uint64_t nm = 0;
                        float pd = 0.0f;
#pragma unroll 4
                        for (int j = 0; j < EC; ++j) {
                            const float xv = scr[j * C::NT];
                            const bool valid = voff(q * EC + j) < lim;
                            const float e = exp2_hw(__builtin_fmaf(xv, kLog2e, -s));
                            pd += valid ? e : 0.0f;
                            nm |= (uint64_t)(valid && xv >= tv) << j;
                        }
                        if (recompute) ds += pd;
                        if (remask) m = nm;
                    }
                    while (m != 0) {
                        const int j = __builtin_ctzll(m);
                        m &= m - 1;
                        const float xv = scr[j * C::NT];
                        // a -inf logit is never a candidate
                        if (xv >= tval[ni] && xv > -__builtin_inff()) offer(ni, xv, q * EC + j);
                    }
                }
                dacc[ni] += ds;
                // The other lane holding this row saw other entries of it:
                // the larger of the two K-th values also bounds the row's
                // K-th value from below.
                tval[ni] = __builtin_fmaxf(tval[ni], __shfl_xor(tval[ni], 32));
            }
        });

    constexpr int P = 2 * C::WX;  // partials per (row, chunk)
    const int64_t Sp = S * P;
    const int64_t p = c * P + wx * 2 + (lane >> 5);
#pragma unroll
    for (int ni = 0; ni < NI; ++ni) {
        const int64_t row = y0s + wy * 32 * NI + ni * 32 + (lane & 31);
        if (row < N) {
            uint64_t* dst = pkeys + (row * Sp + p) * K;
#pragma unroll
            for (int i = 0; i < KC; ++i)
                if (i < K) dst[i] = list[ni].L[i];
            pmd[row * Sp + p] = MD{sr[ni], dacc[ni]};
        }
    }
}

// ---------------------------------------------------------------- launchers
template <class C>
static hipError_t launch_logits_t(const void* h, const void* w, float* out, int64_t N, int64_t H,
                                  int64_t V, hipStream_t st) {
    const int64_t total = ((N + C::TX - 1) / C::TX) * ((V + C::TY - 1) / C::TY);
    const int64_t per = (total + 7) / 8;
    hipLaunchKernelGGL((proj_logits<C>), dim3((unsigned)(8 * per)), dim3(C::NT), 0, st,
                       (const uint16_t*)h, (const uint16_t*)w, out, N, H, V, per);
    return hipGetLastError();
}

hipError_t launch_proj_logits(const void* h, const void* w, float* out, int64_t N, int64_t H,
                              int64_t V, int cus, hipStream_t st) {
    const int64_t big = ((N + PjBig::TX - 1) / PjBig::TX) * ((V + PjBig::TY - 1) / PjBig::TY);
    if (big >= 2 * (int64_t)cus) return launch_logits_t<PjBig>(h, w, out, N, H, V, st);
    return launch_logits_t<PjSmall>(h, w, out, N, H, V, st);
}

void proj_topk_shape(int64_t N, int64_t V, int K, int cus, int64_t* S, int64_t* tiles,
                     int* parts) {
    const int cfg = fused_cfg(N, K);
    const int64_t TY = cfg == 0 ? PjFused8::TY
                       : cfg == 1 ? PjFused16W::TY
                       : cfg == 2 ? PjFused16::TY
                                  : PjFusedN::TY;
    const int64_t TX = PjFused8::TX;
    *parts = 2 * (cfg == 0 ? PjFused8::WX
                  : cfg == 1 ? PjFused16W::WX
                  : cfg == 2 ? PjFused16::WX
                             : PjFusedN::WX);
    // vocabulary chunks: about one workgroup per CU in all (each takes 80 KB
    // of LDS or more); two per CU for the 256 x 64 tiles at K <= 8 (80 KB
    // each, both fit), where the call streams w and twice the loads in
    // flight pay for the merge of twice the partials (measured 5-7% faster
    // at N <= 64; at K = 16 the larger merge ate the gain)
    const int64_t nb = (N + TY - 1) / TY, nt = (V + TX - 1) / TX;
    const int64_t per_cu = cfg == 3 && K <= 8 ? 2 : 1;
    int64_t s = ((int64_t)cus * per_cu + nb - 1) / nb;
    if (s > nt) s = nt;
    if (s < 1) s = 1;
    const int64_t t = (nt + s - 1) / s;
    *tiles = t;
    *S = (nt + t - 1) / t;
}

size_t proj_topk_part_bytes(int64_t N, int64_t S, int parts, int K) {
    return (size_t)N * (size_t)(S * parts) * ((size_t)K * 8 + 8);
}

template <class C, int KC>
static void launch_part(const void* h, const void* w, uint64_t* pkeys, MD* pmd, int64_t N,
                        int64_t H, int64_t V, int K, int64_t S, int64_t tiles, hipStream_t st) {
    const int64_t nb = (N + C::TY - 1) / C::TY;
    const int64_t sb = nb < PJ_SB ? nb : PJ_SB, nsb = (nb + sb - 1) / sb;
    const int64_t ids = (S + PJ_CB - 1) / PJ_CB * nsb * PJ_CB * sb;  // whole blocks
    const int64_t per = (ids + 7) / 8;
    hipLaunchKernelGGL((proj_topk_part<C, KC>), dim3((unsigned)(8 * per)), dim3(C::NT), 0,
                       st, (const uint16_t*)h, (const uint16_t*)w, pkeys, pmd, N, H, V, K, S,
                       tiles, per);
}

hipError_t launch_proj_topk(const void* h, const void* w, float* vals, int32_t* idx,
                            void* part, int64_t N, int64_t H, int64_t V, int K, int64_t S,
                            int64_t tiles, int parts, hipStream_t st) {
    const int64_t Sp = S * parts;  // partials per row
    uint64_t* pkeys = static_cast<uint64_t*>(part);
    MD* pmd = reinterpret_cast<MD*>(pkeys + N * Sp * K);
    const int cfg = fused_cfg(N, K);
    if (cfg == 0)
        launch_part<PjFused8, 8>(h, w, pkeys, pmd, N, H, V, K, S, tiles, st);
    else if (cfg == 1)
        launch_part<PjFused16W, 16>(h, w, pkeys, pmd, N, H, V, K, S, tiles, st);
    else if (cfg == 2)
        launch_part<PjFused16, 16>(h, w, pkeys, pmd, N, H, V, K, S, tiles, st);
    else
        launch_part<PjFusedN, 16>(h, w, pkeys, pmd, N, H, V, K, S, tiles, st);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    constexpr int WB = TK_BLOCK / 64;
    dim3 mgrid((unsigned)((N + WB - 1) / WB));
    hipLaunchKernelGGL((topk_merge<TK_ONLINE>), mgrid, dim3(TK_BLOCK), 0, st, pkeys, pmd, vals,
                       idx, N, Sp, K);
    return hipGetLastError();
}

}  // namespace osm
