/*
 * xtc.h -- C ABI of libxtc.so, the MI355X (gfx950) tiled dense contraction.
 *
 * One function per operator, inputs before outputs, every tensor a raw
 * pointer to contiguous memory (the paper's module ABI, Sec. 4.1, "Module":
 * a function named after the operator that takes the operator's inputs and
 * outputs as contiguous raw pointers).  The schedule is an explicit struct so
 * that schedules can be swept: its fields are the GPU forms of the paper's
 * scheduling primitives (Sec. 3.2, Table 1): strip-mine/tile (block_*,
 * wave_*), vectorize (mfma_*), pack with padding (lds_stages, lds_pad),
 * unroll (unroll_k), parallelize (the workgroup grid) and interchange of the
 * parallel tile loops (raster, xcd_remap).
 *
 * Plain C: no HIP header is needed to use it.  The stream is an opaque
 * hipStream_t passed as void* (NULL = the null stream).
 *
 * Common rules for every entry point
 * ----------------------------------
 * - Tensor pointers are DEVICE pointers, allocated and owned by the caller.
 *   The library allocates nothing, keeps no pointer after it returns and
 *   holds no mutable global state except a thread-local last HIP error code.
 * - Outputs must not overlap inputs (the paper declares its operands
 *   noalias, Fig. 5).  This is not checked.
 * - Every argument and schedule check happens on the host BEFORE any HIP
 *   call, so invalid calls return an error without touching the device.
 * - Kernels are enqueued on `stream`; calls are asynchronous and never
 *   synchronise.  Faults during execution surface at the caller's next
 *   synchronisation on that stream, not in the return value.
 * - The return value is the only error channel.
 * - Element offsets are 32-bit inside the kernels: every operand's span
 *   (bytes from its first to its last addressed element) must be at most
 *   0x7FFFFFD0 bytes (2^31 - 48), else XTC_ERR_TOO_LARGE.  Elements
 *   outside an operand (ragged edges, zero padding) are read through a
 *   buffer offset of 0x7FFFFFF0, which this limit keeps past every operand,
 *   so they read as zero.
 */
#ifndef XTC_H
#define XTC_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Element types.  XTC_BF16: inputs are bf16 bit patterns (uint16), products
 * are exact in fp32, accumulation and output are fp32. */
typedef enum { XTC_F32 = 0, XTC_BF16 = 1 } xtc_dtype;

typedef enum { XTC_OP_MATMUL = 0, XTC_OP_CONV2D = 1 } xtc_op;

typedef enum {
    XTC_OK = 0,
    XTC_ERR_NULL_POINTER = 1,         /* a tensor or output pointer is NULL   */
    XTC_ERR_BAD_SHAPE = 2,            /* negative or inconsistent extents     */
    XTC_ERR_BAD_LEADING_DIM = 3,      /* lda < K, ldb < N or ldc < N          */
    XTC_ERR_BAD_DTYPE = 4,            /* unknown dtype, or not supported here */
    XTC_ERR_BAD_SCHEDULE = 5,         /* illegal field values / combination   */
    XTC_ERR_UNSUPPORTED_SCHEDULE = 6, /* legal but not among compiled ones    */
    XTC_ERR_TOO_LARGE = 7,            /* an operand span above 0x7FFFFFD0     */
                                      /* bytes, or a conv stride/pad/extent   */
                                      /* above 2^30                           */
    XTC_ERR_HIP = 8,                  /* a HIP call failed (see below)        */
    XTC_ERR_MISALIGNED = 9            /* a tensor pointer is not aligned to   */
                                      /* its element size                     */
} xtc_status;

/*
 * Schedule of one contraction C[M,N] = A[M,K] B[K,N] (for conv2d the implicit
 * GEMM: M = OC, N = batch*OH*OW, K = C*R*S; see xtc_conv2d_nchw).
 *
 *  size          sizeof(xtc_sched) as known to the caller (ABI versioning).
 *  block_m/n/k   workgroup tile: the outer strip-mine of M and N (one
 *                workgroup per tile, parallelized over the CUs) and the
 *                K-step staged in LDS per pipeline stage (channels per
 *                stage for the k_order = 2 conv kernels).  Powers of two,
 *                except block_n and wave_n of the k_order = 2 conv kernels
 *                (multiples of 16).
 *  wave_m/n      tile of one 64-lane wavefront inside the workgroup tile
 *                (second strip-mine level); the workgroup has
 *                (block_m/wave_m)*(block_n/wave_n) waves.
 *  mfma_m/n/k    matrix-core instruction tile (the vectorize primitive):
 *                fp32: 32x32x2 or 16x16x4; bf16: 32x32x16 or 16x16x32.
 *  lds_stages    LDS buffers per operand (pack + software pipelining), 1-5;
 *                0 = no LDS staging (the k_split kernels).
 *  lds_pad       LDS row padding in elements (pack with padding against bank
 *                conflicts); -1 selects an XOR-swizzled layout instead.
 *  unroll_k      MFMA k-steps unrolled per LDS stage (0 = the whole stage).
 *  raster        order of the parallel tile loops (interchange): 0 row-major
 *                (N fastest), 1 column-major (M fastest), 2 <= g <= 64
 *                grouped: bands of g tile-rows, walked column by column (a
 *                band taller than the tile grid is the whole grid).  Values
 *                outside 0..64 are XTC_ERR_BAD_SCHEDULE.
 *  xcd_remap     1: renumber workgroups so that each of the 8 XCDs (which
 *                receive workgroups round-robin and each own an L2) works on
 *                one contiguous band of the tile order; 0: hardware order.
 *  k_order       conv2d only (0 for matmul): order of the reduction over
 *                (ic, kh, kw).  0: channel-major, k = (ic*R + kh)*S + kw (the
 *                OIHW weight layout; with block_m = 16, for few output
 *                channels, the workgroup's input patch is staged in LDS
 *                once when it fits, and its two halves of K are reduced by
 *                two groups of waves and added in a fixed order); 1:
 *                tap-major, k = (kh*S + kw)*C + ic
 *                (needs C % 32 == 0, else the channel-major kernel with the
 *                same tiles runs); 2: chunks of channels, and inside a
 *                chunk the R*S taps, with each chunk's input patch staged
 *                once for all taps, for 3x3 stride-1 layers with rows of
 *                about 56 pixels (OW >= 51):
 *                  fp32: chunks of 8, k = ((ic/8)*R*S + kh*S + kw)*8 + ic%8;
 *                  block_n = 256 needs C % 16 == 0 and W + pad_w <= 60;
 *                  block_n = 208 (16x16x4 instructions) needs C % 8 == 0
 *                  and covers at most 208 pixels per workgroup, the count
 *                  chosen per launch so that workgroups split evenly;
 *                  block_n = 416 is the same with two such pixel halves
 *                  per workgroup (8 waves) sharing one input patch;
 *                  other shapes run the tap-major kernel;
 *                  bf16: chunks of 16, k = ((ic/16)*R*S + kh*S + kw)*16 +
 *                  ic%16, needs C % 16 == 0, even W, pad_w <= 2,
 *                  OW - pad_w <= 60, a 4-byte-aligned X and a 16-byte-
 *                  aligned W; other shapes run the channel-major kernel;
 *                3: bf16 only, row streaming for 3x3 stride-1 layers of 64
 *                input channels: a workgroup walks down a band of output
 *                rows of one image with all C*R*S weights of its 64 output
 *                channels resident; k = ((kw*4 + ic/16)*3 + kh)*16 + ic%16
 *                per output row.  Needs C == 64, even W, OW % 4 == 0,
 *                OW <= 64, pad_w <= 2, OW + 3 - pad_w <= 63, a 4-byte-
 *                aligned X and 16-byte-aligned W and Y; other shapes run the
 *                k_order 2 kernel.
 *                Results differ only by rounding order.
 *  k_split       waves that share one workgroup tile, each reducing every
 *                k_split-th group of block_k reduction steps (a parallel
 *                split of the reduction for problems with too few tiles to
 *                fill the chip); their partial sums are added in a fixed
 *                order through LDS, so results stay deterministic.  1 = no
 *                split.  With lds_stages = 0 each wave covers the whole
 *                workgroup tile (wave_m = block_m, wave_n = block_n) and
 *                operands go from memory straight to the matrix-core
 *                registers, double-buffered in registers.  With
 *                lds_stages >= 1 (matmul only) k_split groups of
 *                (block_m/wave_m)*(block_n/wave_n) waves each run the
 *                LDS-staged pipeline on every k_split-th K-step of the
 *                tile, each group on its own LDS ring.
 *
 * block_*, wave_*, mfma_*, lds_stages, lds_pad, unroll_k, k_order and k_split
 * select a compiled kernel instance; raster and xcd_remap are run-time choices valid
 * for all.
 */
typedef struct {
    int32_t size;
    int32_t block_m, block_n, block_k;
    int32_t wave_m, wave_n;
    int32_t mfma_m, mfma_n, mfma_k;
    int32_t lds_stages;
    int32_t lds_pad;
    int32_t unroll_k;
    int32_t raster;
    int32_t xcd_remap;
    int32_t k_order;
    int32_t k_split;
} xtc_sched;

/*
 * xtc_matmul -- C = A * B  (paper Sec. 3.1, Fig. 2: C[i][j] accumulates
 * A[i][k]*B[k][j] over k; here C is overwritten, i.e. accumulation starts
 * from zero).
 *
 *  M, N, K   extents, >= 0.  M == 0 or N == 0: no-op returning XTC_OK.
 *            K == 0: C[0:M, 0:N] is set to zero.
 *  A         device, row-major M x K with row stride lda >= max(K,1)
 *            (elements); fp32 (XTC_F32) or bf16 bits (XTC_BF16).
 *  B         device, row-major K x N with row stride ldb >= max(N,1).
 *  C         device, fp32, row-major M x N with row stride ldc >= max(N,1).
 *            Only C[i*ldc + j] for i < M, j < N is written; columns
 *            N <= j < ldc are never touched.
 *  dtype     XTC_F32 or XTC_BF16 (applies to A and B; C is always fp32).
 *            A, B and C are aligned to their element size (4 bytes fp32,
 *            2 bytes bf16); any row stride is accepted.
 *  sched     NULL selects xtc_default_schedule(); otherwise must pass
 *            xtc_sched_check().
 *  stream    hipStream_t or NULL.
 * Errors: XTC_ERR_NULL_POINTER (A, B or C NULL while M, N > 0),
 * XTC_ERR_BAD_SHAPE (negative extent), XTC_ERR_BAD_LEADING_DIM,
 * XTC_ERR_BAD_DTYPE, XTC_ERR_MISALIGNED (a pointer not aligned to its
 * element size), XTC_ERR_BAD_SCHEDULE, XTC_ERR_UNSUPPORTED_SCHEDULE,
 * XTC_ERR_TOO_LARGE, XTC_ERR_HIP (launch failed).
 */
xtc_status xtc_matmul(int64_t M, int64_t N, int64_t K,
                      const void *A, int64_t lda,
                      const void *B, int64_t ldb,
                      float *C, int64_t ldc,
                      xtc_dtype dtype, const xtc_sched *sched, void *stream);

/*
 * xtc_conv2d_nchw -- 2-D convolution (the paper's conv2d operator, Sec. 3.1)
 * read as zero-padded cross-correlation without dilation, groups or bias:
 *   Y[n][oc][oh][ow] = sum_{ic<C, kh<R, kw<S}
 *        X[n][ic][oh*stride_h - pad_h + kh][ow*stride_w - pad_w + kw]
 *        * Wt[oc][ic][kh][kw],
 * input positions outside [0,H) x [0,W) contributing zero, with
 *   OH = (H + 2*pad_h - R)/stride_h + 1,  OW = (W + 2*pad_w - S)/stride_w + 1.
 * Computed as an implicit GEMM (no im2col buffer): M = OC, N = N*OH*OW,
 * K = C*R*S, reduced in the order the schedule's k_order selects.
 *
 *  X    device, NCHW contiguous; Wt device, OIHW contiguous; both fp32
 *       (XTC_F32) or both bf16 bit patterns (XTC_BF16, products exact in
 *       fp32, fp32 accumulation).
 *  Y    device, N x OC x OH x OW contiguous fp32 (overwritten).
 *  X, Wt and Y are aligned to their element size (else XTC_ERR_MISALIGNED).
 *  N, C, H, W, OC, R, S >= 1 except that N == 0 or OC == 0 is a no-op;
 *  stride >= 1, pad >= 0, OH >= 1 and OW >= 1, else XTC_ERR_BAD_SHAPE.
 *  stride_h, stride_w, pad_h, pad_w, H, W, H + 2*pad_h and W + 2*pad_w are
 *  at most 2^30 (input coordinates stay in 32-bit arithmetic), else
 *  XTC_ERR_TOO_LARGE.
 *  dtype XTC_F32 or XTC_BF16 (else XTC_ERR_BAD_DTYPE); each reduces in
 *  the order its schedule's k_order selects (bf16: 0, 2 or 3).
 *  sched NULL selects the default conv schedule.
 * Errors as for xtc_matmul; XTC_ERR_TOO_LARGE also when C*R*S exceeds the
 * kernel's k-offset table capacity (xtc_conv_max_k()).
 */
xtc_status xtc_conv2d_nchw(int64_t N, int64_t C, int64_t H, int64_t W,
                           int64_t OC, int64_t R, int64_t S,
                           int64_t stride_h, int64_t stride_w,
                           int64_t pad_h, int64_t pad_w,
                           const void *X, const void *Wt, float *Y,
                           xtc_dtype dtype, const xtc_sched *sched, void *stream);

/*
 * xtc_matmul_relu, xtc_conv2d_nchw_relu -- the contraction followed by its
 * consumer relu, fused into the epilogue (the paper's matmul+relu graph,
 * Sec. 5.2, Fig. 9, and its "fusion of consumer", Sec. 3.2): every output
 * element is written once, as relu(v) = (v < 0 ? 0 : v) of the value v that
 * xtc_matmul / xtc_conv2d_nchw would write (a NaN stays NaN, -0.0 stays
 * -0.0).  Arguments, layouts, ownership, schedules and errors are exactly
 * those of xtc_matmul / xtc_conv2d_nchw; the same kernel instances run, so
 * no extra pass over the output and no extra memory traffic is added.
 */
xtc_status xtc_matmul_relu(int64_t M, int64_t N, int64_t K,
                           const void *A, int64_t lda,
                           const void *B, int64_t ldb,
                           float *C, int64_t ldc,
                           xtc_dtype dtype, const xtc_sched *sched, void *stream);

xtc_status xtc_conv2d_nchw_relu(int64_t N, int64_t C, int64_t H, int64_t W,
                                int64_t OC, int64_t R, int64_t S,
                                int64_t stride_h, int64_t stride_w,
                                int64_t pad_h, int64_t pad_w,
                                const void *X, const void *Wt, float *Y,
                                xtc_dtype dtype, const xtc_sched *sched, void *stream);

/*
 * xtc_default_schedule -- the schedule used when sched == NULL, chosen from
 * the problem shape (the paper's default_schedule of an exploration
 * strategy, Sec. 5.2).  For op == XTC_OP_CONV2D pass the implicit-GEMM
 * extents.  Pure host function.  Errors: XTC_ERR_NULL_POINTER (out NULL),
 * XTC_ERR_BAD_DTYPE, XTC_ERR_BAD_SHAPE.
 */
xtc_status xtc_default_schedule(xtc_op op, xtc_dtype dtype,
                                int64_t M, int64_t N, int64_t K, xtc_sched *out);

/*
 * xtc_sched_check -- XTC_OK if `s` can run op/dtype: its fields are legal
 * (XTC_ERR_BAD_SCHEDULE otherwise) and they name a compiled instance
 * (XTC_ERR_UNSUPPORTED_SCHEDULE otherwise).  This is the membership test of
 * the design space a scheduling strategy samples from (Sec. 5.2: a strategy
 * defines a design space over a scheduling template and turns a sample into
 * a schedule); the fields are the primitives of Table 1 (Sec. 3.2).
 * Pure host function; `s` is only read.  Errors: XTC_ERR_NULL_POINTER (s
 * NULL), XTC_ERR_BAD_DTYPE, XTC_ERR_BAD_SCHEDULE (also an unknown op),
 * XTC_ERR_UNSUPPORTED_SCHEDULE.
 */
xtc_status xtc_sched_check(xtc_op op, xtc_dtype dtype, const xtc_sched *s);

/*
 * xtc_sched_list -- the compiled part of the design space (Sec. 5.2: the
 * grid a strategy samples from): writes up to `cap` compiled schedules for
 * op/dtype into the caller-owned array `out` (may be NULL when cap is 0;
 * each entry has raster = 0, xcd_remap = 1) and returns how many exist in
 * total (call with cap = 0 to size the array).  Combined with every raster
 * and xcd_remap value they span the schedules an exploration can sample.
 * Returns -1 for an unknown op/dtype.  Pure host function.
 */
int32_t xtc_sched_list(xtc_op op, xtc_dtype dtype, xtc_sched *out, int32_t cap);

/*
 * xtc_sched_occupancy -- how many workgroups of the kernel instance `s`
 * names one CU holds at once (an input of the per-schedule traffic model
 * evaluated against hardware counters, the GPU form of the cache-model
 * study of Sec. 6.3: the tiles resident together decide what the caches
 * share) (the hardware limit set by the kernel's
 * registers, LDS and threads), for reduction length K (matmul: K; conv2d:
 * C*R*S, which sizes the conv kernels' LDS k-offset table).  For a conv
 * tap-major instance the figure is that of the tap-major kernel itself, not
 * of the channel-major kernel it falls back to when C % 32 != 0.  Queries
 * the current HIP device; enqueues nothing.  Errors: XTC_ERR_NULL_POINTER,
 * the codes of xtc_sched_check, XTC_ERR_BAD_SHAPE (K < 0),
 * XTC_ERR_TOO_LARGE (conv K above xtc_conv_max_k(), or K > 2^30),
 * XTC_ERR_HIP.
 */
xtc_status xtc_sched_occupancy(xtc_op op, xtc_dtype dtype, int64_t K,
                               const xtc_sched *s, int32_t *wg_per_cu);

/*
 * xtc_status_str -- static, NUL-terminated description of a status code, for
 * the harness that reports why a generated operator could not run (Sec. 4.2:
 * the Executor validates results, the Evaluator runs the code and collects
 * metrics).  Never NULL ("unknown status" for a value outside the enum); the
 * string is owned by the library and must not be freed.
 */
const char *xtc_status_str(xtc_status s);

/*
 * xtc_last_hip_error -- hipError_t value of the last failed HIP call made by
 * this thread inside the library, 0 if none (the detail behind XTC_ERR_HIP,
 * for the harness of Sec. 4.2).  Thread-local; not reset by later
 * successful calls.
 */
int32_t xtc_last_hip_error(void);

/*
 * xtc_conv_max_k -- largest reduction length C*R*S that xtc_conv2d_nchw
 * accepts (the capacity of the conv kernels' k-offset table; the conv2d
 * operator of Sec. 3.1 lowered to an implicit GEMM).  Pure host function.
 */
int64_t xtc_conv_max_k(void);

/*
 * xtc_version -- library version, major*10000 + minor*100 + patch, so that a
 * caller loading the module (Sec. 4.1, "Module": a shared library loaded at
 * run time) can check the ABI it binds to.  Pure host function.
 */
int32_t xtc_version(void);

#ifdef __cplusplus
}
#endif

#endif /* XTC_H */
