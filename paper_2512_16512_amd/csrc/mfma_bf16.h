// bf16 matrix-core helpers shared by the bf16 GEMM and the bf16 implicit-GEMM
// conv2d: instruction wrappers with their accumulator layouts, the gfx950
// transpose read, vector types and predicated loads.
#pragma once

#include <hip/hip_runtime.h>

namespace xtc {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));

// ds_read_b64_tr_b16: within each group of 16 lanes, lane 4u + t receives as
// its element r the t-th 16-bit element of the 8 bytes addressed by lane
// 4r + u.  Lane 4r + u pointing at row k0 + r, columns n0 + 4u .. n0 + 4u + 3
// of a row-major [k][n] tile therefore hands lane (4u + t) the four values
// B[k0 .. k0 + 3][n0 + 4u + t]: a column of four consecutive k.
__device__ __forceinline__ u16x4 ds_read_tr16(const unsigned short *p) {
    typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
    const i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(p));
    return __builtin_bit_cast(u16x4, v);
}

template <int MI>
struct Bf16Mfma;

template <>
struct Bf16Mfma<32> {
    static constexpr int KG = 2;     // lane groups along k
    static constexpr int NACC = 16;
    typedef f32x16 acc_t;
    static __device__ __forceinline__ acc_t mma(const u16x8 &a, const u16x8 &b, const acc_t &c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                       __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    }
    static __device__ __forceinline__ int row(int lane, int r) {
        return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
    }
};

template <>
struct Bf16Mfma<16> {
    static constexpr int KG = 4;
    static constexpr int NACC = 4;
    typedef f32x4 acc_t;
    static __device__ __forceinline__ acc_t mma(const u16x8 &a, const u16x8 &b, const acc_t &c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                       __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    }
    static __device__ __forceinline__ int row(int lane, int r) { return 4 * (lane >> 4) + r; }
};

template <int W>
struct VecU16;
template <>
struct VecU16<8> {
    typedef u16x8 t;
};
template <>
struct VecU16<1> {
    typedef unsigned short t;
};

template <int W>
__device__ __forceinline__ typename VecU16<W>::t load_pred_u16(const unsigned short *p, int valid);

template <>
__device__ __forceinline__ u16x8 load_pred_u16<8>(const unsigned short *p, int valid) {
    if (valid >= 8) return *reinterpret_cast<const u16x8 *>(p);
    u16x8 v = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int e = 0; e < 7; ++e)
        if (e < valid) v[e] = p[e];
    return v;
}

template <>
__device__ __forceinline__ unsigned short load_pred_u16<1>(const unsigned short *p, int valid) {
    return valid > 0 ? *p : (unsigned short)0;
}

}  // namespace xtc
