// Projection layer on the gfx950 matrix cores: P = X . Y^T for row-major
// bfloat16 X (nx x K) and Y (ny x K), binary32 accumulation.  The projection
// ahead of the softmax (Section 1) is logits = h . W^T; the Discussion's
// fusion runs the softmax (+ top-k) on the tile while it is still on chip.
//
// Tile: TX x TY of P per workgroup of WX x WY wavefronts, each a block of
// 32 x 32 v_mfma_f32_32x32x16_bf16 products.  K advances in steps of 64
// through two LDS stages.  Operands travel global -> LDS by buffer loads
// with the LDS as destination (no staging registers); the buffer descriptor
// of each operand starts at the tile's first row and ends at the matrix's
// end, so rows past the matrix, and chunks past K (given an offset beyond
// the descriptor), read as zeros without any branch on the load path.  The
// step count is rounded up to even, the extra step reading zeros, so that
// every tile starts in stage 0 and both stages have fixed roles in the code.
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

constexpr int PJ_BK = 64;  // K per step

// Workgroups are dealt to the eight XCDs in turn (workgroup b to XCD b % 8),
// each with its own L2.  Logical id of workgroup b when XCD k takes the k-th
// contiguous block of `per` logical ids, so that the workgroups sharing an
// L2 work on neighbouring tiles and share their operand tiles there.  The
// grid holds 8 * per workgroups; ids past the tile count have no work.
__device__ __forceinline__ int64_t xcd_logical(int64_t b, int64_t per) {
    return (b % 8) * per + b / 8;
}

// P row of result register `i` within a 32 x 32 block: 8 (i / 4) + 4 (l / 32) + i % 4.
__device__ __forceinline__ int row_in_32(int i, int lane) {
    return 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
}

// LDS slot of 16-byte chunk kc of a tile row (rows of 64 bfloat16, 128 B).
// The LDS serves a 16-byte-per-lane read 16 lanes at a time from 64
// four-byte banks (256 B); the 16 lanes of a fragment read hold 16
// consecutive rows and one chunk, two rows per 256 B of banks, so the slot
// is XORed with (row / 2) % 8: the 16 (row parity, slot) pairs are then all
// distinct and the read is free of bank conflicts.
__device__ __forceinline__ int pj_slot(int row, int kc) { return kc ^ ((row >> 1) & 7); }

template <int TX_, int TY_, int WX_, int WY_>
struct PjCfg {
    static constexpr int TX = TX_, TY = TY_, WX = WX_, WY = WY_;
    static constexpr int NW = WX * WY, NT = 64 * NW;            // wavefronts, threads
    static constexpr int MI = TX / 32 / WX, NI = TY / 32 / WY;  // blocks per wavefront
    static constexpr int LX = TX * 8 / NT, LY = TY * 8 / NT;    // loads per thread per stage
    static_assert(LX * NT == TX * 8 && LY * NT == TY * 8, "whole loads");
    // X and Y tiles of the two stages (each stage contiguous)
    struct Stage {
        uint16_t x[TX][PJ_BK];
        uint16_t y[TY][PJ_BK];
    };
    struct Smem {
        Stage st[2];
    };
};

// Buffer descriptor of `m` (rows x K) from row r0 on; reads at byte offsets
// at or past its size return zeros.  Valid offsets in a tile stay below
// 256 K 2 <= 2^29 (K <= 2^20), so the size saturates at 2^31 - 1 harmlessly.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t pj_rsrc(const uint16_t* m, int64_t rows,
                                                         int64_t K, int64_t r0) {
    const int64_t bytes = (rows - r0) * K * 2;
    return __builtin_amdgcn_make_buffer_rsrc((void*)(m + r0 * K), (short)0,
                                             (int)(bytes < 0x7FFFFFFF ? bytes : 0x7FFFFFFF),
                                             0x00020000);
}
constexpr uint32_t PJ_OOB = 0x80000000u;  // an offset past every descriptor

// Per-thread part of the load addressing: load j of a stage covers LDS chunk
// p = 64 (NW j + wave) + lane, i.e. row p / 8, slot p % 8, which holds the
// row's chunk kc = pj_slot(row, p % 8) (the map is an involution).  Row
// p / 8 = 8 (NW j + wave) + lane / 8, so kc does not depend on j, and the
// byte offset of load j is voff + j * jstride.
struct PjAddr {
    uint32_t voff, jstride;
    int kc;
    template <class C>
    __device__ __forceinline__ static PjAddr make(int64_t K) {
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
        const int p = 64 * wave + lane;
        const int row = p >> 3, kc = pj_slot(row, p & 7);
        return PjAddr{(uint32_t)(row * K * 2 + kc * 16), (uint32_t)(8 * C::NW * K * 2), kc};
    }
};

// Loads of step k (elements 64 k ... of each row) of one operand tile.
// Wavefront index, known to the compiler to be uniform (scalar registers).
__device__ __forceinline__ int pj_wave() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

template <class C, int ROWS, int L>
__device__ __forceinline__ void pj_dma(uint16_t (&tile)[ROWS][PJ_BK], __amdgpu_buffer_rsrc_t rs,
                                       const PjAddr& a, int64_t K, int64_t k) {
    const int wave = pj_wave();
    const int64_t k0 = k * PJ_BK;
    // chunks at or past K (the last step of a ragged K, and padded steps) read zeros
    const bool oob = k0 + PJ_BK > K && k0 + a.kc * 8 >= K;
#pragma unroll
    for (int j = 0; j < L; ++j) {
        const int base = 64 * (C::NW * j + wave);  // first chunk of this load (wave-uniform)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            rs, (__attribute__((address_space(3))) void*)(&tile[0][0] + base * 8), 16,
            oob ? PJ_OOB : a.voff + j * a.jstride, (int)(k0 * 2), 0, 0);
    }
}

// Byte offsets, within a tile, of a lane's fragment reads for the blocks of
// a wavefront whose first row is `base` (a multiple of 32): sub-step ks of
// block m reads row base + 32 m + l % 32, chunk 2 ks + l / 32, at byte
// off[ks] + 4096 m.  The row adds a multiple of 16 to (row / 2) for every m,
// so the slot's XOR term is (l % 32) / 2 % 8 for all blocks: one offset per
// sub-step, and the block's part is an instruction offset.
template <int KS>
struct PjFragOff {
    uint32_t off[KS];
    __device__ __forceinline__ static PjFragOff make(int base) {
        const int lane = threadIdx.x & 63, lr = lane & 31, lh = lane >> 5;
        PjFragOff f;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            f.off[ks] = (uint32_t)((base + lr) * PJ_BK * 2 + 16 * pj_slot(lr, 2 * ks + lh));
        return f;
    }
};

template <int ROWS>
__device__ __forceinline__ bf16x8 pj_frag(const uint16_t (&tile)[ROWS][PJ_BK], uint32_t off,
                                          int m) {
    const char* p = reinterpret_cast<const char*>(&tile[0][0]) + off + m * 32 * PJ_BK * 2;
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(p));
}

// acc[mi][ni] += the wavefront's (32 MI) x (32 NI) block of X-tile . Y-tile^T
// over one K step; the block starts at the X-tile row and Y-tile row whose
// fragment offsets are xo and yo.  The fragments of sub-step ks + 1 are read
// into the other register set before the products of sub-step ks are issued.
template <class C>
__device__ __forceinline__ void pj_mma(const uint16_t (&xt)[C::TX][PJ_BK],
                                       const uint16_t (&yt)[C::TY][PJ_BK],
                                       const PjFragOff<PJ_BK / 16>& xo,
                                       const PjFragOff<PJ_BK / 16>& yo,
                                       f32x16 (&acc)[C::MI][C::NI]) {
    constexpr int MI = C::MI, NI = C::NI, KS = PJ_BK / 16;
    bf16x8 a[2][MI], b[2][NI];  // [register set][block]
    auto read = [&](int set, int ks) {
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) a[set][mi] = pj_frag(xt, xo.off[ks], mi);
#pragma unroll
        for (int ni = 0; ni < NI; ++ni) b[set][ni] = pj_frag(yt, yo.off[ks], ni);
    };
    read(0, 0);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        const int cur = ks & 1;
        if (ks + 1 < KS) read(cur ^ 1, ks + 1);
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
    for (int ks = 0; ks < KS; ++ks) {
        if (ks + 1 < KS) __builtin_amdgcn_sched_group_barrier(0x100, MI + NI, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, MI * NI, 0);
    }
}

// Stage hand-over.  The loads of the next stage were issued one step
// earlier; each thread waits for its own, and for its own fragment reads of
// the stage about to be refilled (the compiler may leave the last of them
// in flight, their products scheduled after the barrier), then the
// workgroup barrier makes every thread's loads visible and tells that every
// wavefront has finished reading that stage.  (A plain s_barrier: the fenced
// __syncthreads would also make the compiler wait for everything else.)
__device__ __forceinline__ void pj_handover() {
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Step count of a K: whole steps of 64, rounded up to even.
__device__ __forceinline__ int64_t pj_steps(int64_t K) {
    return ((K + PJ_BK - 1) / PJ_BK + 1) / 2 * 2;
}

// Issue both operands' loads of step k into stage `st`.
template <class C>
__device__ __forceinline__ void pj_issue(typename C::Smem& sm, int st, __amdgpu_buffer_rsrc_t rx,
                                         __amdgpu_buffer_rsrc_t ry, const PjAddr& a, int64_t K,
                                         int64_t k) {
    pj_dma<C, C::TX, C::LX>(sm.st[st].x, rx, a, K, k);
    pj_dma<C, C::TY, C::LY>(sm.st[st].y, ry, a, K, k);
}

// The workgroup's tiles t = t0, t0 + 1, ... < t1, each TX x TY of P at
// coords(t) = (x0, y0) (x0 < nx, y0 < ny), accumulated over all of K;
// epi(t, x0, y0, acc) runs after each tile with stage 1 of the LDS free for
// its own use (every wavefront is past its last read of it, and it is
// refilled only after the next tile's first hand-over).  The next tile's
// first stage is in flight while epi runs.  Every thread of the workgroup
// must call this, with t0 < t1.
template <class C, class Coords, class Epi>
__device__ __forceinline__ void pj_run(const uint16_t* __restrict__ X, int64_t nx,
                                       const uint16_t* __restrict__ Y, int64_t ny, int64_t K,
                                       int64_t t0, int64_t t1, typename C::Smem& sm,
                                       Coords&& coords, Epi&& epi) {
    const int wave = pj_wave();
    const int bx = (wave / C::WY) * 32 * C::MI, by = (wave % C::WY) * 32 * C::NI;
    const PjFragOff<PJ_BK / 16> xo = PjFragOff<PJ_BK / 16>::make(bx),
                                yo = PjFragOff<PJ_BK / 16>::make(by);
    const PjAddr a = PjAddr::make<C>(K);
    const int64_t nk = pj_steps(K);
    int64_t x0, y0;
    coords(t0, x0, y0);
    __amdgpu_buffer_rsrc_t rx = pj_rsrc(X, nx, K, x0), ry = pj_rsrc(Y, ny, K, y0);
    pj_issue<C>(sm, 0, rx, ry, a, K, 0);
    for (int64_t t = t0; t < t1; ++t) {
        const bool more = t + 1 < t1;
        int64_t xn = x0, yn = y0;
        if (more) coords(t + 1, xn, yn);
        const __amdgpu_buffer_rsrc_t rxn = pj_rsrc(X, nx, K, xn), ryn = pj_rsrc(Y, ny, K, yn);
        f32x16 acc[C::MI][C::NI];
#pragma unroll
        for (int mi = 0; mi < C::MI; ++mi)
#pragma unroll
            for (int ni = 0; ni < C::NI; ++ni)
#pragma unroll
                for (int i = 0; i < 16; ++i) acc[mi][ni][i] = 0.0f;
        for (int64_t k = 0; k < nk; k += 2) {
            pj_handover();
            pj_issue<C>(sm, 1, rx, ry, a, K, k + 1);
            pj_mma<C>(sm.st[0].x, sm.st[0].y, xo, yo, acc);
            pj_handover();
            if (k + 2 < nk) pj_issue<C>(sm, 0, rx, ry, a, K, k + 2);
            else if (more) pj_issue<C>(sm, 0, rxn, ryn, a, K, 0);
            pj_mma<C>(sm.st[1].x, sm.st[1].y, xo, yo, acc);
        }
        // every wavefront's last read of stage 1 is done before epi may write it
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        epi(t, x0, y0, acc);
        x0 = xn;
        y0 = yn;
        rx = rxn;
        ry = ryn;
    }
}

}  // namespace osm
