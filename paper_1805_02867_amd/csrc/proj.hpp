// Projection layer on the gfx950 matrix cores: P = X . Y^T for row-major
// bfloat16 X (nx x K) and Y (ny x K), binary32 accumulation.  The projection
// ahead of the softmax (Section 1) is logits = h . W^T; the Discussion's
// fusion runs the softmax (+ top-k) on the tile while it is still on chip.
//
// Tile: 128 x 128 of P per workgroup of 256 threads (four wavefronts, each
// 64 x 64 = 2 x 2 blocks of v_mfma_f32_32x32x16_bf16).  K advances in steps
// of 64 through two pairs of LDS tiles filled by direct-to-LDS loads (no
// staging registers); one barrier per step.
//
// MFMA 32x32x16 lane layout (checked on the hardware): lane l supplies
// A[m = l % 32][k = 8 (l / 32) + j] and B[k = 8 (l / 32) + j][n = l % 32] for
// j < 8, and receives C[m = 8 (r / 4) + 4 (l / 32) + r % 4][n = l % 32] in
// result register r < 16.
#pragma once

#include "md.hpp"

namespace osm {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int PJ_BLOCK = 256;
constexpr int PJ_TX = 128;               // tile rows of P taken from X
constexpr int PJ_TY = 128;               // tile columns of P taken from Y
constexpr int PJ_BK = 64;                // K per step
constexpr int PJ_CHUNKS = PJ_TX * PJ_BK / 8 / PJ_BLOCK;  // 16-byte loads per thread per tile

// LDS: the X and Y tiles of two K steps, 128 rows of 64 bfloat16 (128 B)
// each.  Within a row, 16-byte chunk kc sits in slot kc ^ (row & 7), so the
// eight lanes of each phase of a fragment read (eight consecutive rows, one
// chunk) hit eight different slots, i.e. distinct banks.
struct ProjSmem {
    uint16_t x0[PJ_TX][PJ_BK];
    uint16_t y0[PJ_TY][PJ_BK];
    uint16_t x1[PJ_TX][PJ_BK];
    uint16_t y1[PJ_TY][PJ_BK];
};

// Workgroups are dealt to the eight XCDs in turn (workgroup b to XCD b % 8),
// each with its own L2.  Logical id of workgroup b when XCD k takes the k-th
// contiguous block of `per` logical ids, so that the workgroups sharing an
// L2 work on neighbouring tiles and share their operand tiles there.  The
// grid holds 8 * per workgroups; ids past `total` have no work.
__device__ __forceinline__ int64_t xcd_logical(int64_t b, int64_t per) {
    return (b % 8) * per + b / 8;
}

// Row `r`, result register `i` of a wavefront's 64 x 64 block: the P row
// within the block is 32 mi + row_in_32(i, lane), the column 32 ni + lane % 32.
__device__ __forceinline__ int row_in_32(int i, int lane) {
    return 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
}

// 16 zero bytes in device memory: the source of every chunk that lies outside
// a matrix (the direct-to-LDS load cannot be zeroed after it lands).
__device__ const u32x4 pj_zero16 = {0u, 0u, 0u, 0u};

// Global -> LDS without registers: the 128 x 64 tile of a row-major matrix
// (`rows` x K, K a multiple of 8) at (r0, k0) into `tile`.  Each wavefront
// issues four 16-byte-per-lane direct-to-LDS loads; lane l of load j lands in
// LDS chunk p = 64 (4 j + wave) + l, i.e. row p / 8, slot p % 8, which holds
// the row's chunk (p % 8) ^ (row & 7).
__device__ __forceinline__ void pj_dma(uint16_t (&tile)[PJ_TX][PJ_BK],
                                       const uint16_t* __restrict__ m, int64_t rows, int64_t K,
                                       int64_t r0, int64_t k0) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int j = 0; j < PJ_CHUNKS; ++j) {
        const int base = 64 * (4 * j + wave);  // first chunk of this load (wave-uniform)
        const int p = base + lane;
        const int row = p >> 3, kc = (p & 7) ^ (row & 7);
        const int64_t grow = r0 + row, gcol = k0 + kc * 8;
        const void* src = (grow < rows && gcol < K) ? (const void*)(m + grow * K + gcol)
                                                   : (const void*)&pj_zero16;
        __builtin_amdgcn_global_load_lds(
            (const void __attribute__((address_space(1)))*)src,
            (__attribute__((address_space(3))) void*)(&tile[0][0] + base * 8), 16, 0, 0);
    }
}

// The 16-byte fragment of row r, chunk kc of a tile.
__device__ __forceinline__ bf16x8 pj_frag(const uint16_t (&tile)[PJ_TX][PJ_BK], int r, int kc) {
    return __builtin_bit_cast(
        bf16x8, *reinterpret_cast<const u32x4*>(&tile[r][((kc ^ (r & 7)) * 8)]));
}

// acc[mi][ni] += the wavefront's (32 MI) x (32 NI) block of X-tile . Y-tile^T
// over one K step; the block starts at row bx of the X tile and row by of the
// Y tile.  The fragments of sub-step ks + 1 are read into the other register
// set before the products of sub-step ks are issued, so the LDS latency is
// exposed once per step rather than before every group of products.
template <int MI, int NI>
__device__ __forceinline__ void pj_mma(const uint16_t (&xt)[PJ_TX][PJ_BK],
                                       const uint16_t (&yt)[PJ_TY][PJ_BK], int bx, int by,
                                       f32x16 (&acc)[MI][NI]) {
    const int lane = threadIdx.x & 63;
    const int lr = lane & 31, lh = lane >> 5;
    bf16x8 a[2][MI], b[2][NI];  // [register set][block]
    auto read = [&](int set, int ks) {
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) a[set][mi] = pj_frag(xt, bx + mi * 32 + lr, 2 * ks + lh);
#pragma unroll
        for (int ni = 0; ni < NI; ++ni) b[set][ni] = pj_frag(yt, by + ni * 32 + lr, 2 * ks + lh);
    };
    read(0, 0);
#pragma unroll
    for (int ks = 0; ks < PJ_BK / 16; ++ks) {
        const int cur = ks & 1;
        if (ks + 1 < PJ_BK / 16) read(cur ^ 1, ks + 1);
#pragma unroll
        for (int mi = 0; mi < MI; ++mi)
#pragma unroll
            for (int ni = 0; ni < NI; ++ni)
                acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[cur][mi], b[cur][ni],
                                                                      acc[mi][ni], 0, 0, 0);
    }
    // Keep that order through scheduling: the first fragment reads, then per
    // sub-step the next sub-step's reads ahead of its products (mask 0x100:
    // LDS reads, 0x008: matrix instructions).
    __builtin_amdgcn_sched_group_barrier(0x100, MI + NI, 0);
#pragma unroll
    for (int ks = 0; ks < PJ_BK / 16; ++ks) {
        if (ks + 1 < PJ_BK / 16) __builtin_amdgcn_sched_group_barrier(0x100, MI + NI, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, MI * NI, 0);
    }
}

// The workgroup's 128 x 128 tile of P at (x0, y0), accumulated over all of K,
// by WX x WY wavefronts (WX WY = 4), each a (128 / WX) x (128 / WY) block:
// wavefront w covers X rows 32 MI (w / WY) and Y rows 32 NI (w % WY) on.
// Every thread of the workgroup must call it (it synchronises).  The next
// step's tiles stream straight into the other pair of LDS buffers while the
// current pair is multiplied; the loop is unrolled by two so that each
// buffer's role is fixed in the code (the compiler then knows the loads in
// flight do not alias the tiles being read, and waits for them only before
// the step's barrier).
template <int WX, int WY>
__device__ __forceinline__ void pj_tile(const uint16_t* __restrict__ X, int64_t nx,
                                        const uint16_t* __restrict__ Y, int64_t ny, int64_t K,
                                        int64_t x0, int64_t y0, ProjSmem& sm,
                                        f32x16 (&acc)[PJ_TX / 32 / WX][PJ_TY / 32 / WY]) {
    static_assert(WX * WY == PJ_BLOCK / 64, "one block per wavefront");
    constexpr int MI = PJ_TX / 32 / WX, NI = PJ_TY / 32 / WY;
    const int wave = threadIdx.x >> 6;
    const int bx = (wave / WY) * 32 * MI, by = (wave % WY) * 32 * NI;
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[mi][ni][i] = 0.0f;
    const int64_t nk = (K + PJ_BK - 1) / PJ_BK;
    __syncthreads();  // the previous tile's readers of the buffers are done
    pj_dma(sm.x0, X, nx, K, x0, 0);
    pj_dma(sm.y0, Y, ny, K, y0, 0);
    __syncthreads();
    int64_t kb = 0;
    for (; kb + 2 <= nk; kb += 2) {
        if (kb + 1 < nk) {
            pj_dma(sm.x1, X, nx, K, x0, (kb + 1) * PJ_BK);
            pj_dma(sm.y1, Y, ny, K, y0, (kb + 1) * PJ_BK);
        }
        pj_mma<MI, NI>(sm.x0, sm.y0, bx, by, acc);
        __syncthreads();
        if (kb + 2 < nk) {
            pj_dma(sm.x0, X, nx, K, x0, (kb + 2) * PJ_BK);
            pj_dma(sm.y0, Y, ny, K, y0, (kb + 2) * PJ_BK);
        }
        pj_mma<MI, NI>(sm.x1, sm.y1, bx, by, acc);
        __syncthreads();
    }
    if (kb < nk) {
        pj_mma<MI, NI>(sm.x0, sm.y0, bx, by, acc);
        __syncthreads();
    }
}

}  // namespace osm
