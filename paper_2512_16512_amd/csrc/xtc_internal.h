// Internal interface between the host API (xtc_api.cpp) and the kernel
// families (gemm_f32.hip, gemm_bf16.hip, conv2d_f32.hip).  Not installed.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/xtc.h"

namespace xtc {

// Arguments of one matmul launch.  Offsets are in elements and fit in
// 32 bits (checked on the host).
struct GemmArgs {
    int M, N, K;
    const void *A;
    int lda;
    const void *B;
    int ldb;
    float *C;
    int ldc;
    int raster;     // 0 row-major, 1 column-major, g >= 2 grouped by g tile-rows
    int xcd_remap;  // 1: give each XCD a contiguous band of the tile order
    int relu;       // 1: the epilogue writes relu(acc) = (acc < 0 ? 0 : acc) (fused consumer)
};

// Arguments of one conv2d launch (implicit GEMM: M = OC, N = Nb*OH*OW,
// K = C*R*S, k = (ic*R + kh)*S + kw).
struct ConvArgs {
    int Nb, C, H, W, OC, R, S;
    int sh, sw, ph, pw;
    int OH, OW;
    const float *X;   // bf16 bit patterns for the bf16 kernels
    const float *Wt;  // (the kernels reinterpret the pointers)
    float *Y;
    int raster;
    int xcd_remap;
    int relu;       // 1: the epilogue writes relu(acc) = (acc < 0 ? 0 : acc) (fused consumer)
    int tile_px;    // output pixels per workgroup tile (set by launchers that choose it)
};

using GemmLaunch = hipError_t (*)(const GemmArgs &, hipStream_t);
using ConvLaunch = hipError_t (*)(const ConvArgs &, hipStream_t);

// Resident workgroups per CU of one kernel (the hardware limit set by its
// registers, LDS and threads) at reduction length K, which sizes the dynamic
// LDS of the conv kernels' k-offset table.
using OccupancyFn = hipError_t (*)(int K, int *wg_per_cu);
template <auto KERNEL, int THREADS, int DYN_BYTES_PER_K>
hipError_t occupancy_of(int K, int *wg_per_cu) {
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(
        wg_per_cu, reinterpret_cast<const void *>(KERNEL), THREADS,
        (size_t)DYN_BYTES_PER_K * (size_t)K);
}

// What `vec_launch` of an instance requires; `any_launch` has no
// requirement.
enum VecRule {
    kRowsAligned = 0,  // 16-byte aligned A and B rows (base pointers and leading dimensions)
    kWholeChunks = 1,  // that, and K and N multiples of 16 bytes of elements
    kARowsOnly = 2,    // 16-byte aligned A rows and K a multiple of 16 bytes (B read per element)
};

// One compiled kernel instance.
struct GemmInstance {
    xtc_sched sched;
    GemmLaunch vec_launch;
    GemmLaunch any_launch;
    VecRule vec_rule;
    OccupancyFn occupancy;  // of the kernel vec_launch runs
};

struct ConvInstance {
    xtc_sched sched;
    ConvLaunch launch;
    OccupancyFn occupancy;  // of the instance's own kernel (not its fallbacks)
};

const GemmInstance *gemm_f32_instances(int *count);
const GemmInstance *gemm_bf16_instances(int *count);
const ConvInstance *conv2d_f32_instances(int *count);
const ConvInstance *conv2d_bf16_instances(int *count);

// Largest implicit-GEMM K the conv kernels' LDS k-offset table holds.
constexpr int kConvMaxK = 4096;

// Fills the fields of a schedule descriptor.
inline xtc_sched make_sched(int bm, int bn, int bk, int wm, int wn, int mm, int mn, int mk,
                            int stages, int pad, int unroll, int k_order = 0,
                            int k_split = 1) {
    xtc_sched s;
    s.size = (int32_t)sizeof(xtc_sched);
    s.block_m = bm; s.block_n = bn; s.block_k = bk;
    s.wave_m = wm; s.wave_n = wn;
    s.mfma_m = mm; s.mfma_n = mn; s.mfma_k = mk;
    s.lds_stages = stages; s.lds_pad = pad; s.unroll_k = unroll;
    s.raster = 0; s.xcd_remap = 1;
    s.k_order = k_order;
    s.k_split = k_split;
    return s;
}

}  // namespace xtc
