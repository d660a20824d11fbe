// fp32 matrix-core helpers shared by the fp32 GEMM and the fp32 implicit-GEMM
// conv2d: instruction wrappers with their accumulator layouts, vector types
// and predicated loads.
#pragma once

#include <hip/hip_runtime.h>

namespace xtc {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

template <int MI>
struct F32Mfma;

template <>
struct F32Mfma<32> {
    static constexpr int KG = 2;     // lane groups (k values) per instruction
    static constexpr int NACC = 16;  // accumulator registers per lane
    typedef f32x16 acc_t;
    static __device__ __forceinline__ acc_t mma(float a, float b, const acc_t &c) {
        return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
    }
    // Row inside the 32x32 tile of accumulator register r of lane `lane`
    // (the column is lane % 32).
    static __device__ __forceinline__ int row(int lane, int r) {
        return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
    }
};

template <>
struct F32Mfma<16> {
    static constexpr int KG = 4;
    static constexpr int NACC = 4;
    typedef f32x4 acc_t;
    static __device__ __forceinline__ acc_t mma(float a, float b, const acc_t &c) {
        return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
    }
    static __device__ __forceinline__ int row(int lane, int r) { return 4 * (lane >> 4) + r; }
};

template <int W>
struct VecF32;
template <>
struct VecF32<4> {
    typedef f32x4 t;
};
template <>
struct VecF32<1> {
    typedef float t;
};

// Predicated load of W consecutive floats starting at p, of which only the
// first `valid` (0..W) exist; the rest read as zero.
template <int W>
__device__ __forceinline__ typename VecF32<W>::t load_pred(const float *p, int valid);

template <>
__device__ __forceinline__ f32x4 load_pred<4>(const float *p, int valid) {
    if (valid >= 4) return *reinterpret_cast<const f32x4 *>(p);
    f32x4 v = {0.f, 0.f, 0.f, 0.f};
    if (valid > 0) v[0] = p[0];
    if (valid > 1) v[1] = p[1];
    if (valid > 2) v[2] = p[2];
    return v;
}

template <>
__device__ __forceinline__ float load_pred<1>(const float *p, int valid) {
    return valid > 0 ? *p : 0.f;
}

}  // namespace xtc
