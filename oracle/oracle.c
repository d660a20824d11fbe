/*
 * oracle.c -- fp64 CPU reference for the dense contraction.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may call, link or
 * load this file or the library built from it; only the tests, the smoke check
 * and the benchmark's CPU-baseline leg do.  It shares no code, header, table or
 * helper with the HIP library: it is written from the operator definitions in
 * the paper, not from the kernels.
 *
 * What it computes
 * ----------------
 * matmul (paper, Sec. 3.1, Fig. 2: the untransformed loop nest
 *   C[I][J] += A[I][K] * B[K][J] over hyper-rectangular I, J, K):
 *     C[i][j] = sum_{k=0}^{K-1} A[i][k] * B[k][j]
 *   with C overwritten (the accumulation starts from zero), every product and
 *   partial sum held in IEEE double, and k ascending.  A is row-major with row
 *   stride lda, B row-major with stride ldb, C row-major with stride ldc.
 *   Inputs are fp32 values, or bf16 bit patterns widened exactly to fp32.
 *
 * conv2d (paper, Sec. 3.1 lists conv2d among the operators but prints no
 * formula; the reading used here is the usual cross-correlation with zero
 * padding inside the operator, no dilation, one group, no bias):
 *     Y[n][oc][oh][ow] = sum_{ic<C} sum_{kh<R} sum_{kw<S}
 *         X[n][ic][oh*sh - ph + kh][ow*sw - pw + kw] * W[oc][ic][kh][kw]
 *   where input positions outside [0,H) x [0,W) contribute zero,
 *   OH = (H + 2*ph - R)/sh + 1 and OW = (W + 2*pw - S)/sw + 1 (floor),
 *   X is NCHW, W is OIHW, Y is NCHW, all contiguous.  Terms are summed in
 *   double, in ascending (ic, kh, kw) order.
 *
 * Loop order.  The "full" matmul runs the i-k-j order with a double row
 * accumulator: each C[i][j] still receives its K products in ascending k, so
 * it is bit-identical to the per-entry dot product of the "sampled" routine
 * (loop interchange that keeps every element's summation order; the paper,
 * Sec. 3.2, "Interchange").  Threads split the outermost loop only.
 *
 * Pins: see the not-gpu tests (identity, all-ones, rank-1, exact small
 * integers, hand-worked 2x2/3x3, library float64 matmul/conv, conv special
 * cases and planted-mistake checks).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ---------------------------------------------------------------- inputs */

/* Exact widening of a bf16 bit pattern: the 16 bits are the top half of an
 * fp32 word. */
static double bf16_to_double(uint16_t bits)
{
    uint32_t w = ((uint32_t)bits) << 16;
    float f;
    memcpy(&f, &w, sizeof f);
    return (double)f;
}

/* Element fetch for an operand that is either fp32 (is_bf16 == 0) or bf16
 * bits (is_bf16 != 0). */
static double load_elem(const void *p, int64_t idx, int is_bf16)
{
    if (is_bf16)
        return bf16_to_double(((const uint16_t *)p)[idx]);
    return (double)((const float *)p)[idx];
}

static void set_threads(int nthreads)
{
#ifdef _OPENMP
    if (nthreads > 0)
        omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
}

/* ---------------------------------------------------------------- matmul */

/* Full matmul, rows [row_begin, row_end) of C only (the whole product when
 * row_begin = 0, row_end = M).  Returns 0, or -1 on allocation failure. */
int xo_matmul_rows(int64_t M, int64_t N, int64_t K,
                   const void *A, int64_t lda, const void *B, int64_t ldb,
                   double *C, int64_t ldc, int is_bf16,
                   int64_t row_begin, int64_t row_end, int nthreads)
{
    if (row_begin < 0) row_begin = 0;
    if (row_end > M) row_end = M;
    if (row_end <= row_begin || N <= 0) return 0;
    set_threads(nthreads);
    int failed = 0;
#pragma omp parallel
    {
        double *acc = (double *)malloc((size_t)N * sizeof(double));
        if (!acc) {
#pragma omp atomic write
            failed = 1;
        }
#pragma omp for schedule(dynamic, 1)
        for (int64_t i = row_begin; i < row_end; ++i) {
            if (!acc) continue;
            for (int64_t j = 0; j < N; ++j) acc[j] = 0.0;
            for (int64_t k = 0; k < K; ++k) {
                double a = load_elem(A, i * lda + k, is_bf16);
                for (int64_t j = 0; j < N; ++j)
                    acc[j] += a * load_elem(B, k * ldb + j, is_bf16);
            }
            for (int64_t j = 0; j < N; ++j) C[i * ldc + j] = acc[j];
        }
        free(acc);
    }
    return failed ? -1 : 0;
}

/* C[I[s]][J[s]] for s < S, each a plain dot product in ascending k. */
void xo_matmul_sampled(int64_t M, int64_t N, int64_t K,
                       const void *A, int64_t lda, const void *B, int64_t ldb,
                       int is_bf16, const int64_t *I, const int64_t *J,
                       int64_t S, double *out, int nthreads)
{
    (void)M; (void)N;
    set_threads(nthreads);
#pragma omp parallel for schedule(static)
    for (int64_t s = 0; s < S; ++s) {
        double acc = 0.0;
        for (int64_t k = 0; k < K; ++k)
            acc += load_elem(A, I[s] * lda + k, is_bf16) *
                   load_elem(B, k * ldb + J[s], is_bf16);
        out[s] = acc;
    }
}

/* ---------------------------------------------------------------- conv2d */

static double conv_point(int64_t C, int64_t H, int64_t W, int64_t R, int64_t S,
                         int64_t sh, int64_t sw, int64_t ph, int64_t pw,
                         const void *X, const void *Wt, int is_bf16,
                         int64_t n, int64_t oc, int64_t oh, int64_t ow)
{
    double acc = 0.0;
    for (int64_t ic = 0; ic < C; ++ic)
        for (int64_t kh = 0; kh < R; ++kh)
            for (int64_t kw = 0; kw < S; ++kw) {
                int64_t ih = oh * sh - ph + kh;
                int64_t iw = ow * sw - pw + kw;
                if (ih < 0 || ih >= H || iw < 0 || iw >= W)
                    continue; /* zero padding contributes nothing */
                double x = load_elem(X, ((n * C + ic) * H + ih) * W + iw, is_bf16);
                double w = load_elem(Wt, ((oc * C + ic) * R + kh) * S + kw, is_bf16);
                acc += x * w;
            }
    return acc;
}

static int64_t out_extent(int64_t in, int64_t k, int64_t stride, int64_t pad)
{
    return (in + 2 * pad - k) / stride + 1;
}

/* Full direct convolution: the 7-loop nest n, oc, oh, ow, ic, kh, kw. */
void xo_conv2d_full(int64_t N, int64_t C, int64_t H, int64_t W,
                    int64_t OC, int64_t R, int64_t S,
                    int64_t sh, int64_t sw, int64_t ph, int64_t pw,
                    const void *X, const void *Wt, int is_bf16,
                    double *Y, int nthreads)
{
    int64_t OH = out_extent(H, R, sh, ph), OW = out_extent(W, S, sw, pw);
    if (OH <= 0 || OW <= 0) return;
    set_threads(nthreads);
#pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int64_t n = 0; n < N; ++n)
        for (int64_t oc = 0; oc < OC; ++oc)
            for (int64_t oh = 0; oh < OH; ++oh)
                for (int64_t ow = 0; ow < OW; ++ow)
                    Y[((n * OC + oc) * OH + oh) * OW + ow] =
                        conv_point(C, H, W, R, S, sh, sw, ph, pw, X, Wt, is_bf16,
                                   n, oc, oh, ow);
}

/* Y at flat NCHW output indices F[s], s < S_count. */
void xo_conv2d_sampled(int64_t N, int64_t C, int64_t H, int64_t W,
                       int64_t OC, int64_t R, int64_t S,
                       int64_t sh, int64_t sw, int64_t ph, int64_t pw,
                       const void *X, const void *Wt, int is_bf16,
                       const int64_t *F, int64_t S_count, double *out,
                       int nthreads)
{
    (void)N;
    int64_t OH = out_extent(H, R, sh, ph), OW = out_extent(W, S, sw, pw);
    set_threads(nthreads);
#pragma omp parallel for schedule(static)
    for (int64_t s = 0; s < S_count; ++s) {
        int64_t f = F[s];
        int64_t ow = f % OW;
        int64_t oh = (f / OW) % OH;
        int64_t oc = (f / (OW * OH)) % OC;
        int64_t n = f / (OW * OH * OC);
        out[s] = conv_point(C, H, W, R, S, sh, sw, ph, pw, X, Wt, is_bf16,
                            n, oc, oh, ow);
    }
}

/* Number of OpenMP threads a parallel region would use. */
int xo_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
