// bf16 GEMM on the gfx950 matrix cores: C[M,N] = A[M,K] * B[K,N] with A and B
// bf16 (row-major), products exact in fp32, fp32 accumulation, fp32 C
// (overwritten).
//
// Schedule structure as in gemm_f32.hip (workgroup tile, wave tile, MFMA
// instruction tile, double-buffered padded LDS staging, predicated edges).
//
// Operand fragments.  The bf16 MFMAs (32x32x16, 16x16x32) take, per lane,
// 8 consecutive-k values of one A row (row lane%MI, k-group lane/MI) and 8
// consecutive-k values of one B column.  A is row-major (k-contiguous), so
// its fragment is one ds_read_b128 from a k-contiguous LDS row.  B is
// row-major too (n-contiguous) and is staged in LDS as it is (16-byte
// writes, rows padded by 32 elements); its fragment is gathered with two
// gfx950 transpose reads (ds_read_b64_tr_b16).  Within each group of 16
// lanes that instruction returns to lane 4u+t, as its element r, element t
// of the 8 bytes addressed by lane 4r+u of the group.  So when lane 4r+u
// addresses B[k0+r][n0+4u .. n0+4u+3], lane a of the group receives
// B[k0 .. k0+3][n0+a]: four consecutive k of its own column, which is the
// MFMA B-operand layout.  Two such reads (k0 and k0+4) give the 8 values.
#include "tile_map.h"
#include "xtc_internal.h"

namespace xtc {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));

// Transpose read of 4 x 16 bits (see the file comment for the lane mapping).
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

template <int BM, int BN, int BK, int WM, int WN, int MI, int PAD, bool VEC>
struct GemmBf16Cfg {
    static constexpr int NWM = BM / WM, NWN = BN / WN;
    static constexpr int NT = NWM * NWN * 64;
    static constexpr int TM = WM / MI, TN = WN / MI;
    typedef Bf16Mfma<MI> MF;
    static constexpr int KG = MF::KG;
    static constexpr int KCH = 8 * KG;      // k per MFMA instruction
    static constexpr int AS = BK + PAD;     // LDS row stride of the A tile (elements)
    static constexpr int BS = BN + 32;      // LDS row stride of the B tile (elements)
    static constexpr int W = VEC ? 8 : 1;   // elements per global load
    static constexpr int A_CPR = BK / W;
    static constexpr int B_CPR = BN / W;
    static constexpr int A_LOADS = BM * BK / (W * NT);
    static constexpr int B_LOADS = BK * BN / (W * NT);
    typedef typename VecU16<W>::t vec_t;
    static_assert(BM % WM == 0 && BN % WN == 0, "wave tile must divide the block tile");
    static_assert(WM % MI == 0 && WN % MI == 0, "MFMA tile must divide the wave tile");
    static_assert(BK % KCH == 0, "block_k must be a multiple of the MFMA k");
    static_assert(A_LOADS * W * NT == BM * BK, "A tile must split evenly over threads");
    static_assert(B_LOADS * W * NT == BK * BN, "B tile must split evenly over threads");
    static_assert(PAD % 8 == 0, "padding must keep 16-byte alignment");
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

template <int BM, int BN, int BK, int WM, int WN, int MI, int PAD, bool VEC>
__global__ void __launch_bounds__((BM / WM) * (BN / WN) * 64)
gemm_bf16_kernel(GemmArgs p) {
    typedef GemmBf16Cfg<BM, BN, BK, WM, WN, MI, PAD, VEC> G;
    typedef typename G::MF MF;
    typedef typename G::vec_t vec_t;
    constexpr int W = G::W;

    __shared__ __attribute__((aligned(16))) unsigned short As[2][BM * G::AS];
    __shared__ __attribute__((aligned(16))) unsigned short Bs[2][BK * G::BS];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave / G::NWN, wn = wave % G::NWN;
    const int lrow = lane % MI, lgrp = lane / MI;

    const int M = p.M, N = p.N, K = p.K;
    const int tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
    int tm, tn;
    tile_coords(blockIdx.x, gridDim.x, tiles_m, tiles_n, p.raster, p.xcd_remap, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;

    const unsigned short *__restrict__ A = static_cast<const unsigned short *>(p.A);
    const unsigned short *__restrict__ B = static_cast<const unsigned short *>(p.B);
    const int lda = p.lda, ldb = p.ldb;

    vec_t ra[G::A_LOADS], rb[G::B_LOADS];

    auto load_tiles = [&](int kt) {
        const int k0 = kt * BK;
#pragma unroll
        for (int i = 0; i < G::A_LOADS; ++i) {
            const int idx = tid + i * G::NT;
            const int r = idx / G::A_CPR, c = (idx % G::A_CPR) * W;
            const int gm = m0 + r, gk = k0 + c;
            const int valid = gm < M ? K - gk : 0;
            ra[i] = load_pred_u16<W>(A + (gm < M ? gm : 0) * lda + (valid > 0 ? gk : 0), valid);
        }
#pragma unroll
        for (int i = 0; i < G::B_LOADS; ++i) {
            const int idx = tid + i * G::NT;
            const int r = idx / G::B_CPR, c = (idx % G::B_CPR) * W;
            const int gk = k0 + r, gn = n0 + c;
            const int valid = gk < K ? N - gn : 0;
            rb[i] = load_pred_u16<W>(B + (gk < K ? gk : 0) * ldb + (valid > 0 ? gn : 0), valid);
        }
    };

    auto store_tiles = [&](int st) {
#pragma unroll
        for (int i = 0; i < G::A_LOADS; ++i) {
            const int idx = tid + i * G::NT;
            const int r = idx / G::A_CPR, c = (idx % G::A_CPR) * W;
            *reinterpret_cast<vec_t *>(&As[st][r * G::AS + c]) = ra[i];
        }
#pragma unroll
        for (int i = 0; i < G::B_LOADS; ++i) {
            const int idx = tid + i * G::NT;
            const int r = idx / G::B_CPR, c = (idx % G::B_CPR) * W;
            *reinterpret_cast<vec_t *>(&Bs[st][r * G::BS + c]) = rb[i];
        }
    };

    typename MF::acc_t acc[G::TM][G::TN];
#pragma unroll
    for (int i = 0; i < G::TM; ++i)
#pragma unroll
        for (int j = 0; j < G::TN; ++j)
#pragma unroll
            for (int r = 0; r < MF::NACC; ++r) acc[i][j][r] = 0.f;

    const int KT = (K + BK - 1) / BK;
    if (KT > 0) {
        load_tiles(0);
        store_tiles(0);
        __syncthreads();
    }
    for (int kt = 0; kt < KT; ++kt) {
        const int cur = kt & 1;
        const bool has_next = kt + 1 < KT;
        if (has_next) load_tiles(kt + 1);

        const unsigned short *as = &As[cur][(wm * WM + lrow) * G::AS + 8 * lgrp];
        // transpose-read base: row 8*(k-group) + (lane%16)/4, column
        // (lane%MI rounded down to 16) + 4*(lane%4)
        const unsigned short *bs =
            &Bs[cur][(8 * lgrp + ((lane & 15) >> 2)) * G::BS + wn * WN + (lrow & ~15) + 4 * (lane & 3)];
#pragma unroll
        for (int kk = 0; kk < BK; kk += G::KCH) {
            u16x8 a[G::TM], b[G::TN];
#pragma unroll
            for (int i = 0; i < G::TM; ++i)
                a[i] = *reinterpret_cast<const u16x8 *>(as + i * MI * G::AS + kk);
#pragma unroll
            for (int j = 0; j < G::TN; ++j) {
                const u16x4 lo = ds_read_tr16(bs + kk * G::BS + j * MI);
                const u16x4 hi = ds_read_tr16(bs + (kk + 4) * G::BS + j * MI);
                b[j] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
            }
#pragma unroll
            for (int i = 0; i < G::TM; ++i)
#pragma unroll
                for (int j = 0; j < G::TN; ++j) acc[i][j] = MF::mma(a[i], b[j], acc[i][j]);
        }

        if (has_next) store_tiles(cur ^ 1);
        __syncthreads();
    }

    float *__restrict__ C = p.C;
    const int ldc = p.ldc;
#pragma unroll
    for (int i = 0; i < G::TM; ++i)
#pragma unroll
        for (int j = 0; j < G::TN; ++j) {
            const int col = n0 + wn * WN + j * MI + lrow;
#pragma unroll
            for (int r = 0; r < MF::NACC; ++r) {
                const int row = m0 + wm * WM + i * MI + MF::row(lane, r);
                if (row < M && col < N) C[row * ldc + col] = acc[i][j][r];
            }
        }
}

template <int BM, int BN, int BK, int WM, int WN, int MI, int PAD, bool VEC>
hipError_t launch_bf16(const GemmArgs &a, hipStream_t s) {
    typedef GemmBf16Cfg<BM, BN, BK, WM, WN, MI, PAD, VEC> G;
    const unsigned tiles = (unsigned)(((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN));
    GemmArgs args = a;
    void *kargs[] = {&args};
    return hipLaunchKernel(
        reinterpret_cast<const void *>(&gemm_bf16_kernel<BM, BN, BK, WM, WN, MI, PAD, VEC>),
        dim3(tiles), dim3(G::NT), kargs, 0, s);
}

#define XTC_BF16_INSTANCE(BM, BN, BK, WM, WN, MI, PAD)                                        \
    GemmInstance {                                                                            \
        make_sched(BM, BN, BK, WM, WN, MI, MI, (MI == 32 ? 16 : 32), 2, PAD, 0),               \
            &launch_bf16<BM, BN, BK, WM, WN, MI, PAD, true>,                                  \
            &launch_bf16<BM, BN, BK, WM, WN, MI, PAD, false>                                  \
    }

const GemmInstance kBf16Instances[] = {
    XTC_BF16_INSTANCE(256, 256, 64, 128, 64, 32, 8),  // default for large problems
    XTC_BF16_INSTANCE(128, 128, 64, 64, 64, 32, 8),
    XTC_BF16_INSTANCE(64, 64, 64, 32, 32, 32, 8),     // small problems
    XTC_BF16_INSTANCE(128, 128, 64, 64, 64, 16, 8),   // 16x16x32 instruction tile
};

}  // namespace

const GemmInstance *gemm_bf16_instances(int *count) {
    *count = (int)(sizeof(kBf16Instances) / sizeof(kBf16Instances[0]));
    return kBf16Instances;
}

}  // namespace xtc
