// Host side of the C ABI declared in include/xtc.h: argument and schedule
// validation (before any HIP call), compiled-instance lookup, default
// schedules and the launch on the caller's stream.
#include <string.h>

#include "xtc_internal.h"

namespace {

using namespace xtc;

thread_local int32_t g_last_hip_error = 0;

// Largest operand span in bytes.  Kernels use 32-bit buffer offsets, and
// an element outside an operand is read through the offset kOOB
// (0x7FFFFFF0): the span stays 32 bytes below it, so that offset (plus a
// 16-byte chunk, plus the 16-byte alignment slack of the shifted bf16 loads)
// always lies past the operand's buffer range and reads zero.
constexpr int64_t kMaxSpan = 0x7FFFFFF0 - 32;
// Largest raster group; the kernels also clamp it to the tile rows.
constexpr int kMaxRaster = 64;
// Largest stride or padding, and padded extent, of a convolution: keeps
// every input coordinate oh*stride - pad + kh within 32-bit arithmetic.
constexpr int64_t kMaxConvExtent = int64_t(1) << 30;
constexpr int kLdsBytes = 160 * 1024;                  // LDS per CU on gfx950

// Products and sums of non-negative extents, saturated at INT64_MAX: the
// entry points take any int64 sizes, and a product that wrapped around
// would pass the span limits.
int64_t sat_mul(int64_t a, int64_t b) {
    int64_t r;
    return __builtin_mul_overflow(a, b, &r) ? INT64_MAX : r;
}
int64_t sat_add(int64_t a, int64_t b) {
    int64_t r;
    return __builtin_add_overflow(a, b, &r) ? INT64_MAX : r;
}
int64_t cdiv(int64_t a, int64_t b) { return a / b + (a % b != 0); }   // a >= 0, b > 0

// Bytes from the first to one past the last addressed element of a
// rows x cols row-major operand with row stride ld (0 if empty; saturated).
int64_t span_bytes(int64_t rows, int64_t cols, int64_t ld, int64_t elt) {
    if (rows <= 0 || cols <= 0) return 0;
    return sat_mul(sat_add(sat_mul(rows - 1, ld), cols), elt);
}

bool same_instance(const xtc_sched &a, const xtc_sched &b) {
    return a.block_m == b.block_m && a.block_n == b.block_n && a.block_k == b.block_k &&
           a.wave_m == b.wave_m && a.wave_n == b.wave_n && a.mfma_m == b.mfma_m &&
           a.mfma_n == b.mfma_n && a.mfma_k == b.mfma_k && a.lds_stages == b.lds_stages &&
           a.lds_pad == b.lds_pad && a.unroll_k == b.unroll_k && a.k_order == b.k_order &&
           a.k_split == b.k_split;
}

bool pow2(int v) { return v > 0 && (v & (v - 1)) == 0; }

// Structural legality of a schedule for op/dtype, independent of whether it
// was compiled.
xtc_status legal(xtc_op op, xtc_dtype dt, const xtc_sched &s) {
    if (s.size != (int32_t)sizeof(xtc_sched)) return XTC_ERR_BAD_SCHEDULE;
    // Tile sizes are powers of two, except the pixel dimension of the conv
    // kernels that stage an input patch (k_order 2), whose workgroups cover
    // a whole number of 16-pixel instruction blocks.
    const bool any_n = op == XTC_OP_CONV2D && s.k_order == 2 && s.block_n > 0 && s.block_n % 16 == 0 &&
                       s.wave_n > 0 && s.wave_n % 16 == 0;
    if (!pow2(s.block_m) || !pow2(s.block_k) || !pow2(s.wave_m) ||
        (!any_n && (!pow2(s.block_n) || !pow2(s.wave_n))))
        return XTC_ERR_BAD_SCHEDULE;
    if (s.block_m % s.wave_m || s.block_n % s.wave_n) return XTC_ERR_BAD_SCHEDULE;
    if (s.k_split != 1 && s.k_split != 2 && s.k_split != 4 && s.k_split != 8)
        return XTC_ERR_BAD_SCHEDULE;
    const int waves = (s.block_m / s.wave_m) * (s.block_n / s.wave_n) * s.k_split;
    if (waves < 1 || waves > 16) return XTC_ERR_BAD_SCHEDULE;  // <= 1024 threads
    // k_split > 1: either waves that each cover the whole tile with operands
    // straight to registers (lds_stages 0), or groups of waves that each run
    // the LDS-staged pipeline on their share of the K-steps (lds_stages >= 1)
    if (s.k_split > 1 && (op != XTC_OP_MATMUL ||
                          (s.lds_stages == 0 && (s.wave_m != s.block_m || s.wave_n != s.block_n))))
        return XTC_ERR_BAD_SCHEDULE;
    // instruction tiles the matrix cores offer for this dtype
    if (s.mfma_m != s.mfma_n) return XTC_ERR_BAD_SCHEDULE;
    if (dt == XTC_F32) {
        if (!((s.mfma_m == 32 && s.mfma_k == 2) || (s.mfma_m == 16 && s.mfma_k == 4)))
            return XTC_ERR_BAD_SCHEDULE;
    } else {
        if (!((s.mfma_m == 32 && s.mfma_k == 16) || (s.mfma_m == 16 && s.mfma_k == 32)))
            return XTC_ERR_BAD_SCHEDULE;
    }
    if (s.wave_m % s.mfma_m || s.wave_n % s.mfma_n) return XTC_ERR_BAD_SCHEDULE;
    // block_k: a whole number of fragment sets (fp32: 4 k per lane group);
    // for the patch-staging conv kernels it counts channels per stage, a
    // whole number of instruction k-steps
    const int kchunk = (op == XTC_OP_CONV2D && s.k_order == 2) ? s.mfma_k
                       : dt == XTC_F32 ? 4 * (64 / s.mfma_m) : s.mfma_k;
    if (s.block_k % kchunk) return XTC_ERR_BAD_SCHEDULE;
    // lds_stages 0: operands straight to registers (the k_split matmul
    // kernels and the few-output-channel conv kernel)
    const bool regs_ok = s.k_split > 1 || (op == XTC_OP_CONV2D && s.block_m == s.wave_m);
    if (s.lds_stages < (regs_ok ? 0 : 1) || s.lds_stages > 5) return XTC_ERR_BAD_SCHEDULE;
    if (s.lds_pad < -1 || s.lds_pad > 64) return XTC_ERR_BAD_SCHEDULE;
    if (s.unroll_k < 0) return XTC_ERR_BAD_SCHEDULE;
    if (s.raster < 0 || s.raster > kMaxRaster || s.xcd_remap < 0 || s.xcd_remap > 1)
        return XTC_ERR_BAD_SCHEDULE;
    if (s.k_order < 0 || s.k_order > 3 || (op == XTC_OP_MATMUL && s.k_order != 0))
        return XTC_ERR_BAD_SCHEDULE;
    // LDS budget of the staged tiles
    const int elt = dt == XTC_F32 ? 4 : 2;
    const int pad = s.lds_pad > 0 ? s.lds_pad : 0;
    // swizzled unpadded rows (lds_pad = -1) or rows padded by lds_pad (A) and 8 (B)
    const int bpad = s.lds_pad < 0 ? 0 : 8;
    int64_t lds = (int64_t)s.lds_stages * elt *
                  ((int64_t)s.block_m * (s.block_k + pad) + (int64_t)s.block_n * (s.block_k + bpad));
    if (s.k_split > 1) lds += (int64_t)s.k_split * s.block_m * s.block_n * 4;  // partial sums
    if (lds > kLdsBytes) return XTC_ERR_BAD_SCHEDULE;
    return XTC_OK;
}

const GemmInstance *find_gemm(xtc_dtype dt, const xtc_sched &s) {
    int n = 0;
    const GemmInstance *tab = dt == XTC_F32 ? gemm_f32_instances(&n) : gemm_bf16_instances(&n);
    for (int i = 0; i < n; ++i)
        if (same_instance(tab[i].sched, s)) return &tab[i];
    return nullptr;
}

const ConvInstance *find_conv(xtc_dtype dt, const xtc_sched &s) {
    int n = 0;
    const ConvInstance *tab = dt == XTC_F32 ? conv2d_f32_instances(&n) : conv2d_bf16_instances(&n);
    for (int i = 0; i < n; ++i)
        if (same_instance(tab[i].sched, s)) return &tab[i];
    return nullptr;
}

xtc_status hip_status(hipError_t e) {
    if (e == hipSuccess) return XTC_OK;
    g_last_hip_error = (int32_t)e;
    return XTC_ERR_HIP;
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }
bool aligned_to(const void *p, int64_t bytes) {
    return (reinterpret_cast<uintptr_t>(p) & (uintptr_t)(bytes - 1)) == 0;
}

}  // namespace

extern "C" {

const char *xtc_status_str(xtc_status s) {
    switch (s) {
        case XTC_OK: return "ok";
        case XTC_ERR_NULL_POINTER: return "null pointer";
        case XTC_ERR_BAD_SHAPE: return "bad shape";
        case XTC_ERR_BAD_LEADING_DIM: return "bad leading dimension";
        case XTC_ERR_BAD_DTYPE: return "bad or unsupported dtype";
        case XTC_ERR_BAD_SCHEDULE: return "illegal schedule";
        case XTC_ERR_UNSUPPORTED_SCHEDULE: return "schedule not among the compiled instances";
        case XTC_ERR_TOO_LARGE: return "operand too large for 32-bit offsets";
        case XTC_ERR_HIP: return "HIP error";
        case XTC_ERR_MISALIGNED: return "pointer not aligned to its element size";
    }
    return "unknown status";
}

int32_t xtc_last_hip_error(void) { return g_last_hip_error; }

int64_t xtc_conv_max_k(void) { return kConvMaxK; }

int32_t xtc_version(void) { return 100; }

xtc_status xtc_default_schedule(xtc_op op, xtc_dtype dt, int64_t M, int64_t N, int64_t K,
                                xtc_sched *out) {
    if (!out) return XTC_ERR_NULL_POINTER;
    if (dt != XTC_F32 && dt != XTC_BF16) return XTC_ERR_BAD_DTYPE;
    if (op != XTC_OP_MATMUL && op != XTC_OP_CONV2D) return XTC_ERR_BAD_SHAPE;
    if (M < 0 || N < 0 || K < 0) return XTC_ERR_BAD_SHAPE;
    const int64_t cus = 256;
    auto tiles = [&](int bm, int bn) { return sat_mul(cdiv(M, bm), cdiv(N, bn)); };
    if (op == XTC_OP_CONV2D && dt == XTC_BF16) {
        // the row-streaming kernel (3x3 stride 1, 64 input channels, rows of
        // at most 64 pixels; 32x64x56x56 -> 64: 15.3 us kernel span against
        // 17 us for the halo-tiled kernel), which runs the halo-tiled kernel
        // outside its class, and that one the 64x128 gather kernel outside
        // its own (not 3x3 stride 1, odd widths, rows far from 56 pixels);
        // the gather kernel with 128x128 tiles for more than 64 output
        // channels, 64x64 when 64x128 tiles leave CUs idle
        *out = make_sched(64, 64, 16, 32, 32, 32, 32, 16, 2, -1, 0, 3);
        if (M > 64)
            *out = make_sched(128, 128, 32, 64, 64, 32, 32, 16, 2, 8, 0);
        else if (tiles(64, 128) < cus)
            *out = make_sched(64, 64, 32, 32, 32, 32, 32, 16, 2, 8, 0);
        out->raster = 0;
        return XTC_OK;
    }
    if (op == XTC_OP_CONV2D) {
        // The balanced halo-tiled kernel where the shape allows it (3x3,
        // stride 1, rows of about 56 pixels): 64 output channels x at most
        // 208 (or 416) pixels per workgroup, the pixel tile sized so that the
        // workgroups split evenly over the CUs; else the tap-major kernel's
        // 64x256 tiles of 4 waves (64x64 each) with a two-stage ring, two
        // workgroups per CU, so up to 512 tiles run in a single wave.  When
        // that leaves CUs idle (a small image batch), 64x64 tiles of four
        // 32x32 waves give four times as many workgroups.
        if (M <= 16) {
            // few output channels (the paper's 7x7 stride-2 layer into 16
            // channels: 11.9 us with 64x64 tiles)
            *out = make_sched(16, 64, 128, 16, 16, 16, 16, 4, 0, 0, 0, 0);
            out->raster = 0;
            return XTC_OK;
        }
        *out = make_sched(64, 208, 8, 16, 208, 16, 16, 4, 2, -1, 0, 2);
        // two pixel halves per workgroup (one patch and one weight copy for
        // 416 pixels) once that still gives about a workgroup per CU
        // (32x64x56x56 layer: 65.6 -> 63.6 us)
        if (tiles(64, 416) >= cus - cus / 8)
            *out = make_sched(64, 416, 8, 16, 208, 16, 16, 4, 2, -1, 0, 2);
        if (M > 64)
            *out = make_sched(128, 128, 32, 64, 64, 32, 32, 2, 2, -1, 0, 1);
        else if (tiles(64, 256) < cus)
            *out = make_sched(64, 64, 32, 32, 32, 32, 32, 2, 2, -1, 0, 1);
        out->raster = 0;
        return XTC_OK;
    }
    bool mid = false, big = false;
    if (dt == XTC_F32) {
        // Direct-to-LDS tiles from 256x256 (a tile per CU) through 256x128
        // and 128x128 (two tiles per CU); the reduction-split kernels for
        // long reductions with a narrow operand; 64x64 direct-to-LDS tiles
        // down to half a tile per CU (these won from 512x1024x128 to
        // 2048^3); below that, the largest reduction-split tile that still
        // gives one tile per CU (measured over 16x16 .. 128x128 tiles on
        // shapes from 256^3 to 4096^3 and skinny ones such as 128x128x4096
        // and 64x4096x1024).
        if (tiles(256, 256) >= cus) {
            // eight 128x64 waves, one workgroup per CU: half the copy
            // traffic per FLOP of 256x128 tiles (4096^3: 141.3 -> 145.3
            // TFLOP/s in one sweep)
            *out = make_sched(256, 256, 32, 128, 64, 32, 32, 2, 2, -1, 0);
            big = true;
        } else if (tiles(256, 128) >= 2 * cus) {
            // eight 64x64 waves: a quarter less copy traffic per FLOP than
            // 128x128 (4096^3: 139.6 -> 142.5 TFLOP/s)
            *out = make_sched(256, 128, 32, 64, 64, 32, 32, 2, 2, -1, 0);
            big = true;
        } else if (tiles(128, 128) >= 2 * cus) {
            *out = make_sched(128, 128, 32, 64, 64, 32, 32, 2, 2, -1, 0);
        } else if (K >= 2048 && (M < N ? M : N) <= 32 && tiles(32, 32) >= cus) {
            // One operand has at most 32 rows (or columns) and the
            // reduction is long: the product streams the other operand from
            // HBM.  The reduction-split kernels read it straight into
            // registers, with more loads in flight per CU than the
            // direct-to-LDS ring holds (32768x16x4096: 3.2 -> 5.0 TB/s).
            // Tiles and orders as measured on 32768x16, 16x32768 and
            // 32768x32 (K = 4096).
            if (N <= 16) {
                // 32x16 tiles: each workgroup's reads of B serve 32 rows
                *out = make_sched(32, 16, 32, 32, 16, 16, 16, 4, 0, 0, 0, 0, 8);
                out->raster = 0;
            } else if (M <= 16) {
                *out = make_sched(32, 32, 32, 32, 32, 32, 32, 2, 0, 0, 0, 0, 4);
                out->raster = 0;
            } else {
                *out = make_sched(32, 32, 32, 32, 32, 32, 32, 2, 0, 0, 0, 0, 8);
                out->raster = 4;
            }
            return XTC_OK;
        } else if (tiles(64, 64) >= cus / 2) {
            *out = make_sched(64, 64, 32, 32, 32, 32, 32, 2, 2, -1, 0);
            // at most one tile per CU and a long reduction: two groups of
            // four waves per tile, each on half of the K-steps, so that each
            // SIMD holds two waves (1000^3: 24.3 -> 22.2 us, 1024^3: 23.7 ->
            // 22.5 us; no gain with several tiles per CU, a loss for K = 128)
            if (tiles(64, 64) <= cus && K >= 512) out->k_split = 2;
            mid = true;
        } else if (tiles(64, 32) >= cus)
            *out = make_sched(64, 32, 16, 64, 32, 32, 32, 2, 0, 0, 0, 0, 4);
        else if (tiles(32, 32) >= cus)
            *out = make_sched(32, 32, 32, 32, 32, 32, 32, 2, 0, 0, 0, 0, K >= 1024 ? 8 : 4);
        else
            *out = make_sched(16, 16, 32, 16, 16, 16, 16, 4, 0, 0, 0, 0, 4);
    } else {
        // direct-to-LDS tiles from 256x256 down to 64x128 (half a tile per
        // CU), then the register-staged 64x64 tiles
        if (tiles(256, 256) >= cus)
            *out = make_sched(256, 256, 32, 128, 64, 32, 32, 16, 4, -1, 0);
        else if (tiles(128, 128) >= cus)
            *out = make_sched(128, 128, 32, 64, 64, 32, 32, 16, 4, -1, 0);
        else if (tiles(64, 128) >= cus / 2)
            *out = make_sched(64, 128, 64, 32, 64, 32, 32, 16, 2, -1, 0);
        else
            *out = make_sched(64, 64, 64, 32, 32, 32, 32, 16, 2, 8, 0);
    }
    const int64_t t = tiles(out->block_m, out->block_n);
    out->raster = (mid || big) ? 4 : (t >= 64 ? 8 : 0);
    // The register-fed reduction-split tiles: column-major order (graph
    // replays interleaved on one machine: 256^3 3.36 -> 3.25 us, 256x258x512
    // 5.77 -> 5.57 us, the 256x1024x128 matmul+relu 4.91 -> 4.78 us)
    if (out->k_split > 1 && out->lds_stages == 0) out->raster = 1;
    if (dt == XTC_BF16 && out->block_m == 256 && out->block_n == 256) {
        // Column-major tiles dealt round-robin to the XCDs: at any moment all
        // eight XCDs read the same few B column-panels, which the shared
        // last-level cache then serves once (measured on 8192^3: 2% faster
        // than grouped raster 8 with the XCD remap).
        out->raster = 1;
        out->xcd_remap = 0;
    }
    return XTC_OK;
}

xtc_status xtc_sched_check(xtc_op op, xtc_dtype dt, const xtc_sched *s) {
    if (!s) return XTC_ERR_NULL_POINTER;
    if (dt != XTC_F32 && dt != XTC_BF16) return XTC_ERR_BAD_DTYPE;
    if (op != XTC_OP_MATMUL && op != XTC_OP_CONV2D) return XTC_ERR_BAD_SCHEDULE;
    const xtc_status st = legal(op, dt, *s);
    if (st != XTC_OK) return st;
    if (op == XTC_OP_MATMUL) return find_gemm(dt, *s) ? XTC_OK : XTC_ERR_UNSUPPORTED_SCHEDULE;
    return find_conv(dt, *s) ? XTC_OK : XTC_ERR_UNSUPPORTED_SCHEDULE;
}

xtc_status xtc_sched_occupancy(xtc_op op, xtc_dtype dt, int64_t K, const xtc_sched *s,
                               int32_t *wg_per_cu) {
    if (!s || !wg_per_cu) return XTC_ERR_NULL_POINTER;
    const xtc_status st = xtc_sched_check(op, dt, s);
    if (st != XTC_OK) return st;
    if (K < 0) return XTC_ERR_BAD_SHAPE;
    if (op == XTC_OP_CONV2D && K > kConvMaxK) return XTC_ERR_TOO_LARGE;
    if (K > (int64_t)1 << 30) return XTC_ERR_TOO_LARGE;
    OccupancyFn fn =
        op == XTC_OP_MATMUL ? find_gemm(dt, *s)->occupancy : find_conv(dt, *s)->occupancy;
    int n = 0;
    const xtc_status hs = hip_status(fn((int)K, &n));
    if (hs != XTC_OK) return hs;
    *wg_per_cu = n;
    return XTC_OK;
}

int32_t xtc_sched_list(xtc_op op, xtc_dtype dt, xtc_sched *out, int32_t cap) {
    int n = 0;
    if (op == XTC_OP_MATMUL && dt == XTC_F32) {
        const GemmInstance *t = gemm_f32_instances(&n);
        for (int i = 0; i < n && i < cap && out; ++i) out[i] = t[i].sched;
    } else if (op == XTC_OP_MATMUL && dt == XTC_BF16) {
        const GemmInstance *t = gemm_bf16_instances(&n);
        for (int i = 0; i < n && i < cap && out; ++i) out[i] = t[i].sched;
    } else if (op == XTC_OP_CONV2D && (dt == XTC_F32 || dt == XTC_BF16)) {
        const ConvInstance *t = dt == XTC_F32 ? conv2d_f32_instances(&n) : conv2d_bf16_instances(&n);
        for (int i = 0; i < n && i < cap && out; ++i) out[i] = t[i].sched;
    } else {
        return -1;
    }
    return n;
}

}  // extern "C"

namespace {

xtc_status matmul_impl(int64_t M, int64_t N, int64_t K, const void *A, int64_t lda, const void *B,
                       int64_t ldb, float *C, int64_t ldc, xtc_dtype dtype, const xtc_sched *sched,
                       void *stream, int relu) {
    if (dtype != XTC_F32 && dtype != XTC_BF16) return XTC_ERR_BAD_DTYPE;
    if (M < 0 || N < 0 || K < 0) return XTC_ERR_BAD_SHAPE;
    if (lda < (K > 1 ? K : 1) || ldb < (N > 1 ? N : 1) || ldc < (N > 1 ? N : 1))
        return XTC_ERR_BAD_LEADING_DIM;
    xtc_sched s;
    if (sched) {
        const xtc_status st = xtc_sched_check(XTC_OP_MATMUL, dtype, sched);
        if (st != XTC_OK) return st;
        s = *sched;
    } else {
        xtc_default_schedule(XTC_OP_MATMUL, dtype, M, N, K, &s);
    }
    if (M == 0 || N == 0) return XTC_OK;
    if (!C || (K > 0 && (!A || !B))) return XTC_ERR_NULL_POINTER;
    const int64_t elt = dtype == XTC_F32 ? 4 : 2;
    if (!aligned_to(A, elt) || !aligned_to(B, elt) || !aligned_to(C, 4)) return XTC_ERR_MISALIGNED;
    if (span_bytes(M, K, lda, elt) > kMaxSpan || span_bytes(K, N, ldb, elt) > kMaxSpan ||
        span_bytes(M, N, ldc, 4) > kMaxSpan || lda > kMaxSpan / elt || ldb > kMaxSpan / elt ||
        ldc > kMaxSpan / 4)
        return XTC_ERR_TOO_LARGE;
    const GemmInstance *inst = find_gemm(dtype, s);
    if (!inst) return XTC_ERR_UNSUPPORTED_SCHEDULE;

    GemmArgs a;
    a.M = (int)M; a.N = (int)N; a.K = (int)K;
    a.A = A; a.lda = (int)lda; a.B = B; a.ldb = (int)ldb; a.C = C; a.ldc = (int)ldc;
    a.raster = s.raster; a.xcd_remap = s.xcd_remap;
    a.relu = relu;
    const bool a_rows = aligned16(A) && (lda * elt) % 16 == 0;
    const bool b_rows = aligned16(B) && (ldb * elt) % 16 == 0;
    bool vec;
    switch (inst->vec_rule) {
        case kARowsOnly: vec = K == 0 || (a_rows && (K * elt) % 16 == 0); break;
        case kWholeChunks:
            vec = K == 0 || (a_rows && b_rows && (K * elt) % 16 == 0 && (N * elt) % 16 == 0);
            break;
        default: vec = K == 0 || (a_rows && b_rows); break;
    }
    const GemmLaunch fn = vec ? inst->vec_launch : inst->any_launch;
    return hip_status(fn(a, static_cast<hipStream_t>(stream)));
}

xtc_status conv_impl(int64_t N, int64_t C, int64_t H, int64_t W, int64_t OC, int64_t R,
                     int64_t S, int64_t stride_h, int64_t stride_w, int64_t pad_h, int64_t pad_w,
                     const void *X, const void *Wt, float *Y, xtc_dtype dtype,
                     const xtc_sched *sched, void *stream, int relu) {
    if (dtype != XTC_F32 && dtype != XTC_BF16) return XTC_ERR_BAD_DTYPE;
    if (N < 0 || OC < 0 || C < 1 || H < 1 || W < 1 || R < 1 || S < 1 || stride_h < 1 ||
        stride_w < 1 || pad_h < 0 || pad_w < 0)
        return XTC_ERR_BAD_SHAPE;
    if (stride_h > kMaxConvExtent || stride_w > kMaxConvExtent || pad_h > kMaxConvExtent ||
        pad_w > kMaxConvExtent || H > kMaxConvExtent || W > kMaxConvExtent ||
        H + 2 * pad_h > kMaxConvExtent || W + 2 * pad_w > kMaxConvExtent)
        return XTC_ERR_TOO_LARGE;
    if (H + 2 * pad_h < R || W + 2 * pad_w < S) return XTC_ERR_BAD_SHAPE;
    const int64_t OH = (H + 2 * pad_h - R) / stride_h + 1;
    const int64_t OW = (W + 2 * pad_w - S) / stride_w + 1;
    const int64_t Mg = OC, Ng = sat_mul(sat_mul(N, OH), OW), Kg = sat_mul(sat_mul(C, R), S);
    xtc_sched s;
    if (sched) {
        const xtc_status st = xtc_sched_check(XTC_OP_CONV2D, dtype, sched);
        if (st != XTC_OK) return st;
        s = *sched;
    } else {
        xtc_default_schedule(XTC_OP_CONV2D, dtype, Mg, Ng, Kg, &s);
    }
    if (N == 0 || OC == 0) return XTC_OK;
    if (!X || !Wt || !Y) return XTC_ERR_NULL_POINTER;
    const int64_t xelt = dtype == XTC_F32 ? 4 : 2;
    if (!aligned_to(X, xelt) || !aligned_to(Wt, xelt) || !aligned_to(Y, 4)) return XTC_ERR_MISALIGNED;
    const int64_t elt = dtype == XTC_F32 ? 4 : 2;
    if (sat_mul(sat_mul(sat_mul(sat_mul(N, C), H), W), elt) > kMaxSpan ||
        sat_mul(sat_mul(OC, Kg), elt) > kMaxSpan || sat_mul(sat_mul(OC, Ng), 4) > kMaxSpan)
        return XTC_ERR_TOO_LARGE;
    if (Kg > kConvMaxK) return XTC_ERR_TOO_LARGE;
    const ConvInstance *inst = find_conv(dtype, s);
    if (!inst) return XTC_ERR_UNSUPPORTED_SCHEDULE;

    ConvArgs a;
    a.Nb = (int)N; a.C = (int)C; a.H = (int)H; a.W = (int)W; a.OC = (int)OC;
    a.R = (int)R; a.S = (int)S;
    a.sh = (int)stride_h; a.sw = (int)stride_w; a.ph = (int)pad_h; a.pw = (int)pad_w;
    a.OH = (int)OH; a.OW = (int)OW;
    a.X = static_cast<const float *>(X);
    a.Wt = static_cast<const float *>(Wt);
    a.Y = Y;
    a.raster = s.raster; a.xcd_remap = s.xcd_remap;
    a.relu = relu;
    a.tile_px = 0;
    return hip_status(inst->launch(a, static_cast<hipStream_t>(stream)));
}

}  // namespace

extern "C" {

xtc_status xtc_matmul(int64_t M, int64_t N, int64_t K, const void *A, int64_t lda, const void *B,
                      int64_t ldb, float *C, int64_t ldc, xtc_dtype dtype, const xtc_sched *sched,
                      void *stream) {
    return matmul_impl(M, N, K, A, lda, B, ldb, C, ldc, dtype, sched, stream, 0);
}

xtc_status xtc_matmul_relu(int64_t M, int64_t N, int64_t K, const void *A, int64_t lda,
                           const void *B, int64_t ldb, float *C, int64_t ldc, xtc_dtype dtype,
                           const xtc_sched *sched, void *stream) {
    return matmul_impl(M, N, K, A, lda, B, ldb, C, ldc, dtype, sched, stream, 1);
}

xtc_status xtc_conv2d_nchw(int64_t N, int64_t C, int64_t H, int64_t W, int64_t OC, int64_t R,
                           int64_t S, int64_t stride_h, int64_t stride_w, int64_t pad_h,
                           int64_t pad_w, const void *X, const void *Wt, float *Y, xtc_dtype dtype,
                           const xtc_sched *sched, void *stream) {
    return conv_impl(N, C, H, W, OC, R, S, stride_h, stride_w, pad_h, pad_w, X, Wt, Y, dtype, sched,
                     stream, 0);
}

xtc_status xtc_conv2d_nchw_relu(int64_t N, int64_t C, int64_t H, int64_t W, int64_t OC, int64_t R,
                                int64_t S, int64_t stride_h, int64_t stride_w, int64_t pad_h,
                                int64_t pad_w, const void *X, const void *Wt, float *Y,
                                xtc_dtype dtype, const xtc_sched *sched, void *stream) {
    return conv_impl(N, C, H, W, OC, R, S, stride_h, stride_w, pad_h, pad_w, X, Wt, Y, dtype, sched,
                     stream, 1);
}

}  // extern "C"
