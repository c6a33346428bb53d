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
 *    and streams, including several threads on one stream.  The shared state
 *    is a per-device cache of device properties, a per-device stream-ordered
 *    memory pool, and the scratch of the split kernels, kept per stream (up
 *    to 64 streams per device; further streams get a buffer per call).  A
 *    call that uses its stream's scratch holds a per-device lock from taking
 *    the buffer until its last kernel is enqueued, so calls on one stream
 *    never interleave their kernels on shared buffers.  A stream's buffer
 *    grows in stream order and is kept until osm_stream_release(stream) or
 *    the end of the process: call osm_stream_release before destroying a
 *    stream that has used the library, so that a later stream given the same
 *    handle starts without a buffer.
 *  - Graph capture: the row kernels allocate nothing; the split kernels
 *    (small batches of long rows) allocate their stream's scratch on its
 *    first use and when it must grow.  Under HIP graph capture, either call
 *    once outside the capture on the same stream with the largest shape to
 *    be captured (the buffer is then reused and nothing is allocated), or use
 *    softmax_topk_ex_noalloc for the top-k: an allocation recorded into a
 *    graph would leave the stream's buffer owned by the graph.
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
 *              one store per element.
 *  OSM_RESIDENT: Alg. 3's pair (per lane, then merged with Eq. 4) with the
 *              row held in registers between the normalizer and the output:
 *              one load and one store per element.  Rows of at most
 *              OSM_RESIDENT_MAX_VEC whole 16-byte vectors (65536 binary32 or
 *              131072 bfloat16 elements, plus up to one partial vector at
 *              each end); longer rows give OSM_EUNSUPPORTED. */
enum osm_mode { OSM_NAIVE = 0, OSM_SAFE = 1, OSM_ONLINE = 2, OSM_RESIDENT = 3 };

/* Longest row of OSM_RESIDENT, in 16-byte vectors. */
#define OSM_RESIDENT_MAX_VEC 16384

/* Status codes. */
enum osm_status {
    OSM_OK = 0,
    OSM_EINVAL = 1,       /* invalid argument; nothing enqueued */
    OSM_EUNSUPPORTED = 2, /* valid but unsupported configuration */
    OSM_EHIP = 3,         /* HIP reported an error while enqueuing */
    OSM_ENOMEM = 4,       /* scratch allocation failed */
    OSM_ESCRATCH = 5      /* needs more than OSM_NOALLOC_SCRATCH_BYTES of
                             fixed scratch (softmax_topk_ex_noalloc) */
};

/* Kernel families for softmax_fwd_ex, softmax_topk_ex and softmax_topk_algo. */
enum osm_kernel {
    OSM_KERNEL_AUTO = 0,  /* what the plain entry points use */
    OSM_KERNEL_ROWS = 1,  /* param = lanes per row.  Softmax: 4, 8, 16, 32
                             (several rows per wavefront), 64 (a row per
                             wavefront) or 128, 256, 512, 1024 (a row per
                             workgroup).  Top-k: 64, 128 or 256 (one, two or
                             four wavefronts per row). */
    OSM_KERNEL_SPLIT = 2  /* param = chunks per row S >= 1: a workgroup per
                             chunk; per-chunk normalizer pairs (and, for
                             top-k, per-chunk top-k keys) go through a
                             scratch array (stream-ordered allocation).
                             Softmax merges them in a second kernel; top-k
                             merges each row in the workgroup that completes
                             it, counted in a per-stream array of N
                             counters that is cleared once when allocated
                             and left cleared by every call (so calls on one
                             stream must not overlap, which stream order
                             guarantees) */
};

/* Softmax + top-k algorithms (Section 4, and the comparisons of Section 5.2):
 *  OSM_TOPK_ONLINE_FUSED  : Alg. 4 -- online pair and top-k in one pass, one
 *                           load per element.  What softmax_topk uses.
 *  OSM_TOPK_SAFE_FUSED    : a maximum pass, then the normalizer (with that
 *                           maximum) and top-k in one pass: two loads per
 *                           element.
 *  OSM_TOPK_SAFE_UNFUSED  : safe softmax (Alg. 2) writes y, then a separate
 *                           top-k over y: five accesses per element.
 *  OSM_TOPK_ONLINE_UNFUSED: online softmax (Alg. 3) writes y, then top-k over
 *                           y: four accesses per element.
 *  OSM_TOPK_VALUES        : top-k of x itself, no softmax (vals = x[z]).
 * The fused algorithms select on x; the unfused ones select on the stored y
 * (Eq. 5), so where distinct inputs round to equal outputs (mostly bfloat16
 * y) their ties go to the lower index among equal y. */
enum osm_topk_algo {
    OSM_TOPK_ONLINE_FUSED = 0,
    OSM_TOPK_SAFE_FUSED = 1,
    OSM_TOPK_SAFE_UNFUSED = 2,
    OSM_TOPK_ONLINE_UNFUSED = 3,
    OSM_TOPK_VALUES = 4
};

/* Largest K accepted by the top-k entry points. */
#define OSM_TOPK_KMAX 64

/* y = Softmax(x) row by row (Eq. 1, Section 2), for each of N rows of V
 * elements.  x: N*V elements of `dtype`, read only.  y: N*V elements of the
 * same dtype, written.  mode: an osm_mode.  The three modes compute the same
 * function (Theorem 1) and differ in their passes over memory.
 * Errors: OSM_EINVAL for N < 0, V < 1, sizes above the limits, null pointers
 * with N > 0, unknown dtype or mode, misaligned or overlapping buffers.
 * OSM_ENOMEM if the split-V scratch array cannot be allocated.
 * OSM_EUNSUPPORTED for OSM_RESIDENT rows longer than it holds. */
OSM_API int softmax_fwd(const void* x, void* y, int64_t N, int64_t V, int dtype, int mode,
                hipStream_t stream);

/* softmax_fwd with an explicit kernel family and parameter (osm_kernel);
 * OSM_KERNEL_AUTO ignores param.  OSM_RESIDENT accepts OSM_KERNEL_AUTO or
 * OSM_KERNEL_ROWS with param = 256, 512 or 1024 threads per row.  Results agree with softmax_fwd within the
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

/* softmax_topk_dt with an explicit kernel: OSM_KERNEL_AUTO (what
 * softmax_topk_dt uses; param ignored), OSM_KERNEL_ROWS with param = lanes
 * per row: 64, 128 or 256 (one, two or four wavefronts per row), or
 * OSM_KERNEL_SPLIT with param = chunks per row (clamped so that every chunk
 * starts inside the row).  Indices are identical across kernels; vals agree
 * within binary32 rounding of the reduction tree.
 * Errors: as softmax_topk_dt, plus OSM_EINVAL for another kernel or param,
 * or N * S >= 2^31 chunks; OSM_ENOMEM if the split scratch (N * S * (8K + 8)
 * bytes) or the row counters (4N bytes) cannot be allocated. */
OSM_API int softmax_topk_ex(const void* x, float* vals, int32_t* idx, int64_t N, int64_t V,
                            int K, int dtype, int kernel, int64_t param, hipStream_t stream);

/* Size of the fixed scratch array behind softmax_topk_ex_noalloc, per device. */
#define OSM_NOALLOC_SCRATCH_BYTES (1u << 20)

/* softmax_topk_ex for callers that cannot allocate device memory (code under
 * HIP graph capture, serving loops that must not call hipMalloc): the same
 * kernels and results, but nothing is allocated or freed, by the library or
 * through any allocating routine.  The split path (OSM_KERNEL_SPLIT, or the
 * plan's choice for small batches of long rows) keeps its per-chunk partials
 * (N * S * (8K + 8) bytes, rounded up to 256) and its N row counters (4N
 * bytes, cleared by a small kernel at each call) in a fixed array of
 * OSM_NOALLOC_SCRATCH_BYTES per device, held until the process ends; the row
 * kernels need no scratch.  Every call on a device shares that array, and it
 * keeps the last call's contents: calls that can overlap on one device (on
 * different streams, or from host threads on different streams) race and
 * must be ordered by the caller; calls on one stream are ordered by the
 * stream.  Arguments, results and errors as softmax_topk_ex, plus
 * OSM_ESCRATCH when the split path would need more than the array holds
 * (nothing enqueued) and OSM_EHIP if the array's device address could not
 * be obtained. */
OSM_API int softmax_topk_ex_noalloc(const void* x, float* vals, int32_t* idx, int64_t N,
                                    int64_t V, int K, int dtype, int kernel, int64_t param,
                                    hipStream_t stream);

/* Softmax + top-k by any osm_topk_algo, with an explicit kernel for the
 * top-k pass (kernel and param as in softmax_topk_ex; the two-wavefront
 * shape, param 128, exists for OSM_TOPK_ONLINE_FUSED only; the softmax pass
 * of the unfused algorithms uses what softmax_fwd uses).
 * y: N*V elements of dtype, written with the softmax for the unfused
 * algorithms (must not overlap x, vals or idx); ignored (may be NULL) by the
 * others.  vals: binary32; for the unfused algorithms and OSM_TOPK_VALUES
 * they are the selected elements of y (resp. x), widened exactly.
 * Errors: as softmax_topk_ex, plus OSM_EINVAL for an unknown algo or a
 * missing / misaligned / overlapping y where one is needed. */
OSM_API int softmax_topk_algo(const void* x, void* y, float* vals, int32_t* idx, int64_t N,
                              int64_t V, int K, int dtype, int algo, int kernel, int64_t param,
                              hipStream_t stream);

/* Top-k of the elements themselves, row by row (the top-k of Eq. 5 applied
 * to x): z = the K indices of the largest x, larger first, equal values in
 * increasing index order; vals = x[z] widened to binary32 (-0.0 is returned
 * as +0.0).  NaN elements are never selected; a row with fewer than K
 * non-NaN elements gets idx -1 and NaN vals in the missing places.
 * Errors: as softmax_topk_dt. */
OSM_API int topk_fwd(const void* x, float* vals, int32_t* idx, int64_t N, int64_t V, int K,
                     int dtype, hipStream_t stream);

/* Largest K of proj_softmax_topk. */
#define OSM_PROJ_KMAX 16

/* The projection ahead of the softmax in a language model (Section 1):
 * logits[n][v] = sum_k h[n][k] * w[v][k], on the matrix cores.
 * h: N*H bfloat16 (hidden vectors, row-major), w: V*H bfloat16 (one row per
 * vocabulary entry), both 16-byte aligned with H a multiple of 8.
 * logits: N*V binary32 (binary32 accumulation; the order of the sums is the
 * kernel's, so results match an exact dot product to within binary32
 * accumulation error).  logits must not overlap h or w.
 * Errors: OSM_EINVAL for N < 0, N > 65535 * 128, V < 1, H < 8, H > 2^20,
 * H not a multiple of 8, sizes above 2^31 - 1, null or misaligned
 * pointers. */
OSM_API int proj_fwd(const void* h, const void* w, float* logits, int64_t N, int64_t H,
                     int64_t V, hipStream_t stream);

/* The projection fused with the online softmax and top-k (the Discussion's
 * proposal): for each row n, z = the K indices of the largest logits (Eq. 5,
 * larger first, equal values in increasing index order) and vals[i] =
 * softmax(logits[n])[z[i]], without writing the logits anywhere.  Each
 * 256 x 256 tile of logits is reduced on chip to per-lane online pairs
 * (Alg. 3) and top-K lists (Alg. 4); partials are merged by Eq. 4 and the key
 * order.  h, w as in proj_fwd; vals: N*K binary32; idx: N*K int32, 0-based.
 * Selection is on the binary32 logits as computed by the kernel.
 * Errors: as proj_fwd, plus OSM_EINVAL for K < 1, K > V, K > OSM_PROJ_KMAX or
 * overlapping outputs; OSM_ENOMEM if the partials' scratch (N * 2S * (8K + 8)
 * bytes, S = vocabulary chunks) cannot be allocated. */
OSM_API int proj_softmax_topk(const void* h, const void* w, float* vals, int32_t* idx,
                              int64_t N, int64_t H, int64_t V, int K, hipStream_t stream);

/* Reference streaming kernels, for measurement only (nothing of the method):
 * op 0 reads `bytes` bytes of x (y: a device buffer of at least 1 KB that
 * the kernel may write, as a sink the compiler cannot remove); op 1 copies
 * `bytes` bytes of x to y, with 16-byte non-temporal accesses: the
 * plain read and copy rates against which the other kernels' bandwidth is
 * judged.  x and y 16-byte aligned, bytes a multiple of 16, x and y not
 * overlapping (op 1).  Each wavefront streams one contiguous span.
 * Errors: OSM_EINVAL for another op, bytes < 0 or not
 * a multiple of 16, null or misaligned pointers, overlap. */
OSM_API int osm_ref_stream(int op, const void* x, void* y, int64_t bytes, hipStream_t stream);

/* Releases the scratch buffers the library keeps for `stream` (split
 * kernels' partials and row counters): they are freed in stream order, behind
 * the work already enqueued on the stream, which still completes normally;
 * the next call on the stream allocates afresh.  Call it before destroying a
 * stream that has used the library.  A stream without buffers is a no-op.
 * Errors: OSM_EHIP if HIP rejects the stream-ordered free (for example a
 * stream already destroyed). */
OSM_API int osm_stream_release(hipStream_t stream);

/* Kernel family and parameter softmax_fwd would use for this shape on the
 * current device (for OSM_RESIDENT: OSM_KERNEL_ROWS and the threads per row).  Errors: OSM_EINVAL for bad sizes, dtype or
 * null outputs; OSM_EUNSUPPORTED for OSM_RESIDENT rows it cannot hold. */
OSM_API int osm_plan(int64_t N, int64_t V, int dtype, int mode, int* kernel, int64_t* param);

/* Kernel family and parameter the top-k entry points would use for this
 * shape on the current device.  Errors: OSM_EINVAL for bad sizes, dtype, K
 * or null outputs. */
OSM_API int osm_topk_plan(int64_t N, int64_t V, int dtype, int K, int* kernel, int64_t* param);

/* Static description of a status code (never NULL). */
OSM_API const char* osm_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* OSOFTMAX_H */
