/*
 * osoftmax -- row-wise softmax with the online normalizer, and fused
 * softmax + top-k, for AMD Instinct MI355X (gfx950).
 *
 * Method: M. Milakov and N. Gimelshein, "Online normalizer calculation for
 * softmax" (arXiv:1805.02867, 2018).
 *
 * Conventions shared by every entry point:
 *  - Buffers are device pointers on the current HIP device, owned by the
 *    caller.  Batches are row-major N x V, rows contiguous (row r starts V
 *    elements after row r-1), each pointer aligned to its element size.
 *  - Element types (dtype): OSM_F32 = IEEE binary32, OSM_BF16 = bfloat16
 *    (16-bit patterns).  All arithmetic is binary32; bfloat16 inputs are
 *    widened exactly and bfloat16 outputs are rounded to nearest even.
 *  - Calls are asynchronous: they validate the arguments on the host, enqueue
 *    work on `stream` (NULL = the default stream) and return.  A status other
 *    than OSM_OK means nothing was enqueued, except OSM_EHIP, which reports a
 *    HIP error raised while enqueuing.  Kernel faults surface on the next
 *    synchronising HIP call, as with any HIP kernel.
 *  - N = 0 is a no-op returning OSM_OK.  Sizes must satisfy 1 <= V <= 2^31-1,
 *    0 <= N <= 2^31-1.
 *  - Input and output buffers must not overlap (OSM_EINVAL otherwise).
 *  - Results are deterministic: the same call on the same device gives the
 *    same bits (fixed reduction orders, no floating-point atomics).
 *  - Non-finite inputs: -inf elements give 0 when the row has a finite
 *    element; a row holding NaN or +inf, or only -inf, gives NaN outputs
 *    (IEEE evaluation of the safe formula, Eq. 2).  Finite inputs must stay
 *    below 2.35e38 (x * log2(e) must be finite).  Top-k of a NaN row is
 *    unspecified.
 *  - Thread safety: calls may be made concurrently from several host threads
 *    and streams.  The only shared state is a per-device cache of device
 *    properties and a per-device stream-ordered memory pool.
 */
#ifndef OSOFTMAX_H
#define OSOFTMAX_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#if defined(__GNUC__) || defined(__clang__)
#define OSM_API __attribute__((visibility("default")))
#else
#define OSM_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

/* Element types. */
enum osm_dtype { OSM_F32 = 0, OSM_BF16 = 1 };

/* Normalizer algorithms (Section 2 and 3 of the paper):
 *  OSM_NAIVE : Alg. 1 -- d = sum_j e^{x_j}, y_i = e^{x_i}/d.  Two loads and
 *              one store per element.  Overflows (NaN/inf outputs) once
 *              e^{x} exceeds binary32 range, x > ~88.7, as the paper warns.
 *  OSM_SAFE  : Alg. 2 -- max pass, normalizer pass, output pass.  Three
 *              loads and one store per element.
 *  OSM_ONLINE: Alg. 3 -- one pass carrying the running (max, normalizer)
 *              pair merged with Eq. 4, then the output pass.  Two loads and
 *              one store per element. */
enum osm_mode { OSM_NAIVE = 0, OSM_SAFE = 1, OSM_ONLINE = 2 };

/* Status codes. */
enum osm_status {
    OSM_OK = 0,
    OSM_EINVAL = 1,       /* invalid argument; nothing enqueued */
    OSM_EUNSUPPORTED = 2, /* valid but unsupported configuration */
    OSM_EHIP = 3,         /* HIP reported an error while enqueuing */
    OSM_ENOMEM = 4        /* scratch allocation failed */
};

/* Kernel families for softmax_fwd_ex. */
enum osm_kernel {
    OSM_KERNEL_AUTO = 0,  /* what softmax_fwd uses */
    OSM_KERNEL_ROWS = 1,  /* param = lanes per row: 4, 8, 16, 32 (several rows
                             per wavefront), 64 (a row per wavefront) or
                             128, 256, 512, 1024 (a row per workgroup) */
    OSM_KERNEL_SPLIT = 2  /* param = chunks per row S >= 1: several workgroups
                             per row, partial pairs merged through a scratch
                             array (stream-ordered allocation) */
};

/* Largest K accepted by the top-k entry points. */
#define OSM_TOPK_KMAX 64

/* y = Softmax(x) row by row (Eq. 1, Section 2), for each of N rows of V
 * elements.  x: N*V elements of `dtype`, read only.  y: N*V elements of the
 * same dtype, written.  mode: an osm_mode.  The three modes compute the same
 * function (Theorem 1) and differ in their passes over memory.
 * Errors: OSM_EINVAL for N < 0, V < 1, sizes above the limits, null pointers
 * with N > 0, unknown dtype or mode, misaligned or overlapping buffers.
 * OSM_ENOMEM if the split-V scratch array cannot be allocated. */
OSM_API int softmax_fwd(const void* x, void* y, int64_t N, int64_t V, int dtype, int mode,
                hipStream_t stream);

/* softmax_fwd with an explicit kernel family and parameter (osm_kernel);
 * OSM_KERNEL_AUTO ignores param.  Results agree with softmax_fwd within the
 * library's accuracy (binary32 rounding differs with the reduction tree).
 * Errors: as softmax_fwd, plus OSM_EINVAL for an unknown kernel or a param
 * it does not accept. */
OSM_API int softmax_fwd_ex(const void* x, void* y, int64_t N, int64_t V, int dtype, int mode,
                   int kernel, int64_t param, hipStream_t stream);

/* Fused online softmax + top-k (Alg. 4, Section 4) over binary32 rows.
 * For each row: z = the K indices of the largest x (Eq. 5), larger first,
 * equal values in increasing index order (Alg. 4's strictly-less insertion);
 * vals[i] = softmax(x)[z[i]].  Reads x once; writes only N*K outputs.
 * x: N*V binary32.  vals: N*K binary32.  idx: N*K int32, 0-based.
 * Errors: OSM_EINVAL for K < 1, K > V, K > OSM_TOPK_KMAX, and the softmax_fwd
 * argument errors; vals and idx must not overlap x or each other. */
OSM_API int softmax_topk(const float* x, float* vals, int32_t* idx, int64_t N, int64_t V, int K,
                 hipStream_t stream);

/* softmax_topk for bfloat16 or binary32 rows (dtype: osm_dtype).  vals stay
 * binary32 and are computed from the exact widened inputs. */
OSM_API int softmax_topk_dt(const void* x, float* vals, int32_t* idx, int64_t N, int64_t V, int K,
                    int dtype, hipStream_t stream);

/* softmax_topk_dt with an explicit kernel shape: kernel OSM_KERNEL_AUTO (what
 * softmax_topk_dt uses; param ignored) or OSM_KERNEL_ROWS with param = lanes
 * per row: 64, 128 or 256 (one, two or four wavefronts per row).  Results
 * are identical across shapes except for binary32 rounding of vals.
 * Errors: as softmax_topk_dt, plus OSM_EINVAL for another kernel or param. */
OSM_API int softmax_topk_ex(const void* x, float* vals, int32_t* idx, int64_t N, int64_t V,
                            int K, int dtype, int kernel, int64_t param, hipStream_t stream);

/* Kernel family and parameter softmax_fwd would use for this shape on the
 * current device.  Errors: OSM_EINVAL for bad sizes, dtype or null outputs. */
OSM_API int osm_plan(int64_t N, int64_t V, int dtype, int mode, int* kernel, int64_t* param);

/* Static description of a status code (never NULL). */
OSM_API const char* osm_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* OSOFTMAX_H */
