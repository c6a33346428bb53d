// Projection layer on the gfx950 matrix cores: P = X . Y^T for row-major
// bfloat16 X (nx x K) and Y (ny x K), binary32 accumulation.  The projection
// ahead of the softmax (Section 1) is logits = h . W^T; the Discussion's
// fusion runs the softmax (+ top-k) on the tile while it is still on chip.
//
// Tile: 128 x 128 of P per workgroup of 256 threads (four wavefronts, each
// 64 x 64 = 2 x 2 blocks of v_mfma_f32_32x32x16_bf16).  K advances in steps
// of 64 through two LDS buffers (X and Y tiles, rows padded to 144 bytes so
// that each 8-lane phase of a 16-byte LDS read hits distinct banks), fed
// from registers loaded one step ahead; one barrier per step.
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
constexpr int PJ_ROW = PJ_BK + 8;        // bfloat16 elements per LDS row (padding)
constexpr int PJ_CHUNKS = PJ_TX * PJ_BK / 8 / PJ_BLOCK;  // 16-byte loads per thread per tile

struct ProjSmem {
    uint16_t x[2][PJ_TX][PJ_ROW];
    uint16_t y[2][PJ_TY][PJ_ROW];
};

// Row `r`, result register `i` of a wavefront's 64 x 64 block: the P row
// within the block is 32 mi + row_in_32(i, lane), the column 32 ni + lane % 32.
__device__ __forceinline__ int row_in_32(int i, int lane) {
    return 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
}

// Global -> registers: this thread's 16-byte chunks of a 128 x 64 tile of a
// row-major matrix with `rows` rows and K columns (K a multiple of 8), rows
// from r0 and columns from k0.  The loads are unconditional (a chunk outside
// the matrix reads element 0 instead) so that they issue back to back; the
// chunks outside are zeroed when stored (pj_store).
struct PjChunks {
    u32x4 v[PJ_CHUNKS];
    bool ok[PJ_CHUNKS];
};

__device__ __forceinline__ void pj_load(PjChunks& reg, const uint16_t* __restrict__ m,
                                        int64_t rows, int64_t K, int64_t r0, int64_t k0) {
    const int t = threadIdx.x;
#pragma unroll
    for (int i = 0; i < PJ_CHUNKS; ++i) {
        const int c = t + i * PJ_BLOCK;
        const int64_t row = r0 + (c >> 3), col = k0 + (c & 7) * 8;
        reg.ok[i] = row < rows && col < K;
        reg.v[i] = *reinterpret_cast<const u32x4*>(m + (reg.ok[i] ? row * K + col : 0));
    }
}

__device__ __forceinline__ void pj_store(uint16_t (&tile)[PJ_TX][PJ_ROW], const PjChunks& reg) {
    const int t = threadIdx.x;
#pragma unroll
    for (int i = 0; i < PJ_CHUNKS; ++i) {
        const int c = t + i * PJ_BLOCK;
        *reinterpret_cast<u32x4*>(&tile[c >> 3][(c & 7) * 8]) =
            reg.ok[i] ? reg.v[i] : u32x4{0u, 0u, 0u, 0u};
    }
}

// acc[mi][ni] += the wavefront's 64 x 64 block of X-tile . Y-tile^T over one
// K step held in LDS buffer `buf`.
__device__ __forceinline__ void pj_mma(const ProjSmem& sm, int buf, int wx, int wy,
                                       f32x16 (&acc)[2][2]) {
    const int lane = threadIdx.x & 63;
    const int lr = lane & 31, lk = (lane >> 5) * 8;
#pragma unroll
    for (int ks = 0; ks < PJ_BK / 16; ++ks) {
        bf16x8 a[2], b[2];
#pragma unroll
        for (int mi = 0; mi < 2; ++mi)
            a[mi] = __builtin_bit_cast(
                bf16x8, *reinterpret_cast<const u32x4*>(&sm.x[buf][wx * 64 + mi * 32 + lr][ks * 16 + lk]));
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
            b[ni] = __builtin_bit_cast(
                bf16x8, *reinterpret_cast<const u32x4*>(&sm.y[buf][wy * 64 + ni * 32 + lr][ks * 16 + lk]));
#pragma unroll
        for (int mi = 0; mi < 2; ++mi)
#pragma unroll
            for (int ni = 0; ni < 2; ++ni)
                acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mi], b[ni], acc[mi][ni], 0, 0, 0);
    }
}

// The workgroup's 128 x 128 tile of P at (x0, y0), accumulated over all of K.
// Every thread of the workgroup must call it (it synchronises).  The next
// step's tiles are loaded into registers before the current step is
// multiplied and stored to the other LDS buffer after it.  (Loading two steps
// ahead measured no faster and cost the fused kernel half its occupancy.)
__device__ __forceinline__ void pj_tile(const uint16_t* __restrict__ X, int64_t nx,
                                        const uint16_t* __restrict__ Y, int64_t ny, int64_t K,
                                        int64_t x0, int64_t y0, ProjSmem& sm,
                                        f32x16 (&acc)[2][2]) {
    const int wave = threadIdx.x >> 6;
    const int wx = wave >> 1, wy = wave & 1;
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[mi][ni][i] = 0.0f;
    const int64_t nk = (K + PJ_BK - 1) / PJ_BK;
    PjChunks rx, ry;
    pj_load(rx, X, nx, K, x0, 0);
    pj_load(ry, Y, ny, K, y0, 0);
    __syncthreads();  // the previous tile's readers of buffer 0 are done
    pj_store(sm.x[0], rx);
    pj_store(sm.y[0], ry);
    __syncthreads();
    for (int64_t kb = 0; kb < nk; ++kb) {
        const int buf = (int)(kb & 1);
        const bool more = kb + 1 < nk;
        if (more) {
            pj_load(rx, X, nx, K, x0, (kb + 1) * PJ_BK);
            pj_load(ry, Y, ny, K, y0, (kb + 1) * PJ_BK);
        }
        pj_mma(sm, buf, wx, wy, acc);
        if (more) {
            pj_store(sm.x[buf ^ 1], rx);
            pj_store(sm.y[buf ^ 1], ry);
        }
        __syncthreads();
    }
}

}  // namespace osm
