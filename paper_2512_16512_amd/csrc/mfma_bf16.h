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
// chunks that cover them are funnel-shifted into place.  Values from
// position `valid` on are zero.  This lets rows that start at any 2-byte
// boundary be read with 16-byte loads.
//
// Lanes call it in runs: within a run, lane l + 1 asks for the eight values
// after lane l's, so lane l's second chunk is lane l + 1's first and comes
// from that lane; only the last lane of a run (`run_end`, which must hold
// for lane 63) loads it itself.  Loads past the buffer's end read zero.
__device__ __forceinline__ u16x8 load_shifted_u16x8(__amdgpu_buffer_rsrc_t rs, int e, int valid,
                                                    bool run_end) {
    typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
    const int o = 2 * e;
    const int ob = o & ~15;
    const u32x4 v0 = __builtin_amdgcn_raw_buffer_load_b128(rs, ob, 0, 0);
    // lanes inside a run ask for an offset past any buffer (zero, no fetch)
    const u32x4 own = __builtin_amdgcn_raw_buffer_load_b128(rs, run_end ? ob + 16 : 0x7FFFFFF0, 0, 0);
    // the shuffle runs in every lane (a lane reading an inactive lane gets
    // nothing), and only then is the lane's own load chosen where it applies
    u32x4 v1;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const unsigned next = (unsigned)__shfl_down((int)v0[q], 1, 64);
        v1[q] = run_end ? own[q] : next;
    }
    const unsigned w[8] = {v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]};
    // Shift right by (o & 15) bytes: 8, then 4 bytes as the position asks
    // (bitwise selects, no branches), then 2 bytes with v_alignbyte, whose
    // shift is 0 or 2.
    const unsigned m8 = (o & 8) ? ~0u : 0u, m4 = (o & 4) ? ~0u : 0u;
    unsigned w1[6], w2[5];
#pragma unroll
    for (int i = 0; i < 6; ++i) w1[i] = w[i] ^ ((w[i] ^ w[i + 2]) & m8);
#pragma unroll
    for (int i = 0; i < 5; ++i) w2[i] = w1[i] ^ ((w1[i] ^ w1[i + 1]) & m4);
    const unsigned sh = (unsigned)(o & 2);
    u32x4 r;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        // values 2i and 2i + 1 kept only below `valid`
        const unsigned keep = (2 * i < valid ? 0xFFFFu : 0u) | (2 * i + 1 < valid ? 0xFFFF0000u : 0u);
        r[i] = __builtin_amdgcn_alignbyte(w2[i + 1], w2[i], sh) & keep;   // (hi:lo) >> 8*sh
    }
    return __builtin_bit_cast(u16x8, r);
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
