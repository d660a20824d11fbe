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

// Eight consecutive bf16 values starting at element e of a buffer whose base
// address is 16-byte aligned, for any position e: the two aligned 16-byte
// chunks that cover them are loaded (a chunk past the buffer's end reads
// zero) and funnel-shifted into place.  Values from position `valid` on are
// zero.  This lets rows that start at any 2-byte boundary be read with
// 16-byte loads.
__device__ __forceinline__ u16x8 load_shifted_u16x8(__amdgpu_buffer_rsrc_t rs, int e, int valid) {
    typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
    const int o = 2 * e;
    const int ob = o & ~15;
    const u32x4 v0 = __builtin_amdgcn_raw_buffer_load_b128(rs, ob, 0, 0);
    const u32x4 v1 = __builtin_amdgcn_raw_buffer_load_b128(rs, ob + 16, 0, 0);
    const unsigned w[8] = {v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]};
    const int d = (o >> 2) & 3;  // whole dwords to skip
    const bool half = (o & 2) != 0;
    u32x4 r;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const unsigned lo = d == 0 ? w[i] : d == 1 ? w[i + 1] : d == 2 ? w[i + 2] : w[i + 3];
        const unsigned hi = d == 0 ? w[i + 1] : d == 1 ? w[i + 2] : d == 2 ? w[i + 3] : w[i + 4];
        r[i] = half ? __builtin_amdgcn_alignbyte(hi, lo, 2) : lo;   // (hi:lo) >> 16
    }
    u16x8 v = __builtin_bit_cast(u16x8, r);
#pragma unroll
    for (int k = 0; k < 8; ++k)
        if (k >= valid) v[k] = 0;
    return v;
}

// Buffer resource covering `bytes` bytes from p, with its base rounded down
// and its end rounded up to 16 bytes, so a 16-byte chunk holding any of the
// bytes is wholly inside it (such a chunk never crosses a page, so it is
// mapped) and a chunk past the end reads zero; *first receives p's position
// in elements of `elt` bytes from that base.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t aligned_rsrc(const void *p, long long bytes,
                                                               int elt, int *first) {
    const unsigned long long a = reinterpret_cast<unsigned long long>(p);
    const unsigned mis = (unsigned)(a & 15);
    *first = (int)(mis / elt);
    return __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void *>(a - mis), 0,
                                             (int)((bytes + mis + 15) & ~15ll), 0x00020000);
}

}  // namespace xtc
