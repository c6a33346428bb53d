/*
 * Reference oracle for row-wise softmax and softmax+top-k
 * (Milakov & Gimelshein, "Online normalizer calculation for softmax", 2018).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, obviously correct
 * CPU statement of what the GPU library computes.  Only the test suite, the
 * smoke check and the CPU-baseline leg of the benchmark may load it.  It
 * shares no code, header, table or helper with the HIP library, and the HIP
 * library never calls it.
 *
 * All arithmetic is IEEE binary64 with the platform libm exp().  Rows are
 * independent; OpenMP only distributes whole rows over threads, so the result
 * of every row is the same for any thread count.
 *
 * Inputs are row-major N x V arrays of binary32, bfloat16 (raw 16-bit
 * patterns) or binary64.  Every widening to binary64 is exact.
 *
 * Readings of the paper taken here (where it is silent or ambiguous):
 *  - The pair (-inf, 0) is the identity of the merge operator; merging two
 *    pairs whose larger maximum is -inf gives the identity rather than the
 *    NaN that e^{-inf-(-inf)} would produce.
 *  - Non-finite inputs follow plain IEEE evaluation of the safe formula
 *    (Eq. 2): a row holding NaN or +inf, or made only of -inf, gives a row
 *    of NaN; -inf elements next to finite ones give exactly 0.
 *  - Top-k selects on the input values x (the fused algorithm, Alg. 4, keeps
 *    the running top-k of x), under the total order "larger x first, lower
 *    index first among equal x".  Equal here is IEEE equality, so -0.0 and
 *    +0.0 tie.  This is the order Alg. 4's strictly-less insertion test
 *    produces.  NaN inputs make the selection unspecified (they are ordered
 *    last here only so that the sort stays well defined).
 *  - Indices are 0-based.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Input element types understood by the oracle. */
enum { ORC_F32 = 0, ORC_BF16 = 1, ORC_F64 = 2 };

/* Status codes. */
enum { ORC_OK = 0, ORC_EINVAL = 1, ORC_ENOMEM = 2 };

static int g_threads = 0; /* 0: OpenMP default */

void orc_set_threads(int n) { g_threads = n > 0 ? n : 0; }

/* Threads a parallel region of the oracle will use. */
int orc_get_threads(void) {
#ifdef _OPENMP
    return g_threads > 0 ? g_threads : omp_get_max_threads();
#else
    return 1;
#endif
}

/* Exact widening of element i of a row to binary64. */
static double load_elem(const void* row, int dtype, int64_t i) {
    if (dtype == ORC_F32) return (double)((const float*)row)[i];
    if (dtype == ORC_F64) return ((const double*)row)[i];
    /* bfloat16 is the upper half of a binary32 pattern */
    uint32_t bits = (uint32_t)((const uint16_t*)row)[i] << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

static size_t elem_size(int dtype) {
    return dtype == ORC_F32 ? 4 : dtype == ORC_BF16 ? 2 : 8;
}

static const void* row_ptr(const void* x, int dtype, int64_t V, int64_t r) {
    return (const char*)x + (size_t)r * (size_t)V * elem_size(dtype);
}

static int bad_args(const void* x, int dtype, int64_t N, int64_t V) {
    if (N < 0 || V < 1) return 1;
    if (dtype != ORC_F32 && dtype != ORC_BF16 && dtype != ORC_F64) return 1;
    if (N > 0 && !x) return 1;
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Normalizer pair (m, d) by its definition (Theorem 1's closed form):
 *   m = max_k x_k,   d = sum_j e^{x_j - m}.                                 */
static void md_direct_row(const void* row, int dtype, int64_t V, double* m_out,
                          double* d_out) {
    double m = -INFINITY;
    for (int64_t k = 0; k < V; ++k) {
        double v = load_elem(row, dtype, k);
        if (v > m) m = v; /* a NaN never compares greater; it reaches d below */
    }
    double d = 0.0;
    for (int64_t j = 0; j < V; ++j) d += exp(load_elem(row, dtype, j) - m);
    *m_out = m;
    *d_out = d;
}

int orc_md_direct(const void* x, int dtype, int64_t N, int64_t V, double* m,
                  double* d) {
    if (bad_args(x, dtype, N, V) || (N > 0 && (!m || !d))) return ORC_EINVAL;
#pragma omp parallel for schedule(dynamic, 1) num_threads(orc_get_threads())
    for (int64_t r = 0; r < N; ++r)
        md_direct_row(row_ptr(x, dtype, V, r), dtype, V, &m[r], &d[r]);
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* The merge operator on normalizer pairs (Section 3.1, Eq. 4):
 *   (m_i, d_i) (+) (m_j, d_j) = (M, d_i e^{m_i - M} + d_j e^{m_j - M}),
 *   M = max(m_i, m_j),
 * with (-inf, 0) as identity (see the file header).                         */
void orc_md_combine(double mi, double di, double mj, double dj, double* m_out,
                    double* d_out) {
    double M = mi > mj ? mi : mj;
    if (mi != mi || mj != mj) { /* NaN propagates */
        *m_out = NAN;
        *d_out = NAN;
        return;
    }
    if (M == -INFINITY) {
        *m_out = -INFINITY;
        *d_out = 0.0;
        return;
    }
    *m_out = M;
    *d_out = di * exp(mi - M) + dj * exp(mj - M);
}

/* The online normalizer recurrence (Alg. 3, first loop), element by element
 * in index order: m_j = max(m_{j-1}, x_j), d_j = d_{j-1} e^{m_{j-1}-m_j}
 * + e^{x_j - m_j}, from (m_0, d_0) = (-inf, 0).  Each step is the merge of
 * the running pair with (x_j, 1), which is how the identity guard applies. */
static void md_online_row(const void* row, int dtype, int64_t V, double* m_out,
                          double* d_out) {
    double m = -INFINITY, d = 0.0;
    for (int64_t j = 0; j < V; ++j) {
        double xj = load_elem(row, dtype, j);
        orc_md_combine(m, d, xj, 1.0, &m, &d);
    }
    *m_out = m;
    *d_out = d;
}

int orc_md_online(const void* x, int dtype, int64_t N, int64_t V, double* m,
                  double* d) {
    if (bad_args(x, dtype, N, V) || (N > 0 && (!m || !d))) return ORC_EINVAL;
#pragma omp parallel for schedule(dynamic, 1) num_threads(orc_get_threads())
    for (int64_t r = 0; r < N; ++r)
        md_online_row(row_ptr(x, dtype, V, r), dtype, V, &m[r], &d[r]);
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Softmax by the safe formula (Eq. 2): y_i = e^{x_i - m} / sum_j e^{x_j - m},
 * m = max_k x_k.  By Theorem 1 this is exactly what every algorithm of the
 * paper computes, so it is the expected output of every mode.               */
static void softmax_row(const void* row, int dtype, int64_t V, double* y) {
    double m, d;
    md_direct_row(row, dtype, V, &m, &d);
    for (int64_t i = 0; i < V; ++i) y[i] = exp(load_elem(row, dtype, i) - m) / d;
}

int orc_softmax(const void* x, int dtype, int64_t N, int64_t V, double* y) {
    if (bad_args(x, dtype, N, V) || (N > 0 && !y)) return ORC_EINVAL;
#pragma omp parallel for schedule(dynamic, 1) num_threads(orc_get_threads())
    for (int64_t r = 0; r < N; ++r)
        softmax_row(row_ptr(x, dtype, V, r), dtype, V, y + (size_t)r * (size_t)V);
    return ORC_OK;
}

/* Softmax by the unprotected formula (Eq. 1 evaluated as Alg. 1):
 * d = sum_j e^{x_j}, y_i = e^{x_i} / d.  Overflows for large x, which is the
 * failure the safe and online forms avoid.                                  */
int orc_softmax_naive(const void* x, int dtype, int64_t N, int64_t V, double* y) {
    if (bad_args(x, dtype, N, V) || (N > 0 && !y)) return ORC_EINVAL;
#pragma omp parallel for schedule(dynamic, 1) num_threads(orc_get_threads())
    for (int64_t r = 0; r < N; ++r) {
        const void* row = row_ptr(x, dtype, V, r);
        double* yr = y + (size_t)r * (size_t)V;
        double d = 0.0;
        for (int64_t j = 0; j < V; ++j) d += exp(load_elem(row, dtype, j));
        for (int64_t i = 0; i < V; ++i) yr[i] = exp(load_elem(row, dtype, i)) / d;
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Top-k (Eq. 5) by a full sort of the indices under the total order of the
 * file header; z = the first K indices, v_i = softmax(x)_{z_i}.             */
typedef struct {
    double x;
    int32_t i;
} keyed;

static int keyed_cmp(const void* a, const void* b) {
    const keyed* p = (const keyed*)a;
    const keyed* q = (const keyed*)b;
    int pn = p->x != p->x, qn = q->x != q->x;
    if (pn != qn) return pn - qn; /* NaN last */
    if (!pn) {
        if (p->x > q->x) return -1;
        if (p->x < q->x) return 1;
    }
    return (p->i > q->i) - (p->i < q->i);
}

int orc_topk(const void* x, int dtype, int64_t N, int64_t V, int K, double* v,
             int32_t* z) {
    if (bad_args(x, dtype, N, V) || K < 1 || K > V || V > INT32_MAX)
        return ORC_EINVAL;
    if (N > 0 && (!v || !z)) return ORC_EINVAL;
    int err = 0;
#pragma omp parallel num_threads(orc_get_threads())
    {
        keyed* buf = (keyed*)malloc((size_t)V * sizeof(keyed));
        if (!buf) {
#pragma omp atomic write
            err = 1;
        }
#pragma omp for schedule(dynamic, 1)
        for (int64_t r = 0; r < N; ++r) {
            if (!buf) continue;
            const void* row = row_ptr(x, dtype, V, r);
            for (int64_t j = 0; j < V; ++j) {
                buf[j].x = load_elem(row, dtype, j);
                buf[j].i = (int32_t)j;
            }
            qsort(buf, (size_t)V, sizeof(keyed), keyed_cmp);
            double m, d;
            md_direct_row(row, dtype, V, &m, &d);
            for (int k = 0; k < K; ++k) {
                z[r * K + k] = buf[k].i;
                v[r * K + k] = exp(buf[k].x - m) / d;
            }
        }
        free(buf);
    }
    return err ? ORC_ENOMEM : ORC_OK;
}

/* Top-k (Eq. 5) by repeated selection, a second route to orc_topk's result
 * used to pin it: pass k scans the whole row for the first element, under the
 * total order of the file header, among those ranked after the element pass
 * k-1 took (pass 0: among all).  Its normalizer comes from the online
 * recurrence (Alg. 3, each step an Eq. 4 merge), not from the closed form
 * orc_topk uses.  Output v_k = e^{x_{z_k} - m}/d.                           */
static int ranks_before(double xa, int64_t ia, double xb, int64_t ib) {
    int an = xa != xa, bn = xb != xb;
    if (an != bn) return bn; /* every number before every NaN */
    if (!an && xa != xb) return xa > xb;
    return ia < ib;          /* equal values (or two NaN): lower index first */
}

int orc_topk_select(const void* x, int dtype, int64_t N, int64_t V, int K, double* v,
                    int32_t* z) {
    if (bad_args(x, dtype, N, V) || K < 1 || K > V || V > INT32_MAX) return ORC_EINVAL;
    if (N > 0 && (!v || !z)) return ORC_EINVAL;
#pragma omp parallel for schedule(dynamic, 1) num_threads(orc_get_threads())
    for (int64_t r = 0; r < N; ++r) {
        const void* row = row_ptr(x, dtype, V, r);
        double m, d;
        md_online_row(row, dtype, V, &m, &d);
        double prev_x = 0.0;
        int64_t prev_i = -1;
        for (int k = 0; k < K; ++k) {
            int64_t best = -1;
            double best_x = 0.0;
            for (int64_t j = 0; j < V; ++j) {
                double xj = load_elem(row, dtype, j);
                if (prev_i >= 0 && !ranks_before(prev_x, prev_i, xj, j)) continue;
                if (best < 0 || ranks_before(xj, j, best_x, best)) {
                    best = j;
                    best_x = xj;
                }
            }
            z[r * K + k] = (int32_t)best;
            v[r * K + k] = exp(best_x - m) / d;
            prev_x = best_x;
            prev_i = best;
        }
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Round binary64 values to the nearest bfloat16, ties to even, in one step
 * (no intermediate binary32 rounding).  bfloat16 keeps 8 significant bits and
 * the binary32 exponent range; below 2^-126 its spacing stays 2^-133.       */
static uint16_t bf16_from_f64(double a) {
    if (a != a) return 0x7FC0;
    uint16_t sign = signbit(a) ? 0x8000 : 0;
    a = fabs(a);
    if (isinf(a)) return sign | 0x7F80;
    if (a == 0.0) return sign;
    int e;
    frexp(a, &e); /* a in [2^(e-1), 2^e) */
    int ex = e - 1;
    if (ex < -126) ex = -126;
    double q = ldexp(1.0, ex - 7); /* spacing of bfloat16 values near a */
    double r = rint(a / q) * q;    /* default rounding mode: ties to even */
    if (r >= ldexp(1.0, 128)) return sign | 0x7F80;
    float f = (float)r; /* exact: r has at most 8 significant bits */
    uint32_t bits;
    memcpy(&bits, &f, sizeof bits);
    return sign | (uint16_t)(bits >> 16);
}

void orc_bf16_round(const double* y, int64_t n, uint16_t* out) {
    for (int64_t i = 0; i < n; ++i) out[i] = bf16_from_f64(y[i]);
}

/* bfloat16 bit patterns to binary64, exactly: the widening every bfloat16
 * input of the oracle goes through (load_elem). */
void orc_bf16_widen(const uint16_t* bits, int64_t n, double* out) {
    for (int64_t i = 0; i < n; ++i) out[i] = load_elem(bits, ORC_BF16, i);
}

/* ------------------------------------------------------------ projection */
/* The projection layer that precedes the softmax in a language model
 * (Section 1; the Discussion proposes fusing the softmax into it):
 *   logits[n][v] = sum_{k < H} h[n][k] * w[v][k]
 * for hidden vectors h (N x H) and a weight matrix w (V x H, one row per
 * vocabulary entry), accumulated in binary64 with k ascending.  Products of
 * bfloat16 or binary32 inputs are exact in binary64. */
int orc_proj(const void* h, int hdtype, const void* w, int wdtype, int64_t N, int64_t H,
             int64_t V, double* out) {
    if (bad_args(h, hdtype, N, H) || bad_args(w, wdtype, V, H) || (N > 0 && !out))
        return ORC_EINVAL;
#pragma omp parallel for schedule(dynamic, 1) num_threads(orc_get_threads())
    for (int64_t n = 0; n < N; ++n) {
        const void* hr = row_ptr(h, hdtype, H, n);
        double* o = out + (size_t)n * (size_t)V;
        for (int64_t v = 0; v < V; ++v) {
            const void* wr = row_ptr(w, wdtype, H, v);
            double acc = 0.0;
            for (int64_t k = 0; k < H; ++k) acc += load_elem(hr, hdtype, k) * load_elem(wr, wdtype, k);
            o[v] = acc;
        }
    }
    return ORC_OK;
}
