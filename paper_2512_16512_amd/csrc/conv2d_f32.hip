// fp32 conv2d (NCHW input, OIHW weights, NCHW output) as an implicit GEMM on
// the gfx950 matrix cores, with no im2col buffer.
//
// Orientation.  Per image the convolution is Y_n[OC, OH*OW] = W[OC, K] *
// col_n[K, OH*OW] with K = C*R*S and k = (ic*R + kh)*S + kw.  The GEMM here is
// M = OC (rows of the row-major weight matrix, k-contiguous), N = Nb*OH*OW
// pixels across the batch (column q = n*OH*OW + p), and K as above.  For a
// fixed k, consecutive output pixels read (mostly) consecutive input
// addresses, so the B gather and the NCHW output stores are coalesced along
// the pixel dimension.  This is the same tiled contraction as gemm_f32.hip
// (same workgroup / wave / MFMA tiling and double-buffered padded LDS
// staging); only the B loader (a gather with zero-padding predicates fused
// into the pack step) and the epilogue (NCHW addressing) differ.
//
// k-offset table.  At kernel start each workgroup builds, in LDS, a table
// mapping k to (ic*H*W + kh*W + kw, kh, kw), so the gather needs no integer
// division in the main loop: an element (k, q) is X[base(q) + off(k)] when
// 0 <= ih0(q) + kh < H and 0 <= iw0(q) + kw < W, else zero.
#include "mfma_f32.h"
#include "tile_map.h"
#include "xtc_internal.h"

namespace xtc {
namespace {

template <int BM, int BN, int BK, int WM, int WN, int MI, int PAD, bool VEC>
struct ConvF32Cfg {
    static constexpr int NWM = BM / WM, NWN = BN / WN;
    static constexpr int NT = NWM * NWN * 64;
    static constexpr int TM = WM / MI, TN = WN / MI;
    typedef F32Mfma<MI> MF;
    static constexpr int KG = MF::KG;
    static constexpr int KCH = 4 * KG;
    static constexpr int AS = BK + PAD;
    static constexpr int BS = BN + (MI == 32 ? 8 : 4);
    static constexpr int WA = VEC ? 4 : 1;          // weight elements per global load
    static constexpr int A_CPR = BK / WA;
    static constexpr int A_LOADS = BM * BK / (WA * NT);
    static constexpr int B_ROWS_PER_PASS = NT / BN; // gather: thread owns one pixel column
    static constexpr int B_LOADS = BK / B_ROWS_PER_PASS;
    typedef typename VecF32<WA>::t vec_t;
    static_assert(NT % BN == 0 && BK % B_ROWS_PER_PASS == 0, "gather split");
    static_assert(A_LOADS * WA * NT == BM * BK, "weight tile must split evenly");
    static_assert(BK % KCH == 0, "block_k must be a multiple of the fragment k-chunk");
};

template <int BM, int BN, int BK, int WM, int WN, int MI, int PAD, bool VEC>
__global__ void __launch_bounds__((BM / WM) * (BN / WN) * 64)
conv2d_f32_kernel(ConvArgs p) {
    typedef ConvF32Cfg<BM, BN, BK, WM, WN, MI, PAD, VEC> G;
    typedef typename G::MF MF;
    typedef typename G::vec_t vec_t;
    constexpr int WA = G::WA;

    __shared__ __attribute__((aligned(16))) float As[2][BM * G::AS];
    __shared__ __attribute__((aligned(16))) float Bs[2][BK * G::BS];
    extern __shared__ int2 ktab[];  // [K]: {ic*H*W + kh*W + kw, kh | kw << 16}

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave / G::NWN, wn = wave % G::NWN;
    const int lrow = lane % MI, lgrp = lane / MI;

    const int C = p.C, H = p.H, Wd = p.W, R = p.R, S = p.S;
    const int OC = p.OC, OHW = p.OH * p.OW;
    const int M = OC, N = p.Nb * OHW, K = C * R * S;
    const int HW = H * Wd;

    const int tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
    int tm, tn;
    tile_coords(blockIdx.x, gridDim.x, tiles_m, tiles_n, p.raster, p.xcd_remap, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;

    // k-offset table for the whole K range.
    const int RS = R * S;
    for (int k = tid; k < K; k += G::NT) {
        const int ic = k / RS, rem = k - ic * RS;
        const int kh = rem / S, kw = rem - kh * S;
        ktab[k] = make_int2(ic * HW + kh * Wd + kw, kh | (kw << 16));
    }

    // This thread's gather column (fixed for the whole K loop).
    const int bcol = tid % BN, brow0 = tid / BN;
    const int q = n0 + bcol;
    const bool qok = q < N;
    int xbase = 0, ih0 = 0, iw0 = 0;
    if (qok) {
        const int img = q / OHW, pix = q - img * OHW;
        const int oh = pix / p.OW, ow = pix - oh * p.OW;
        ih0 = oh * p.sh - p.ph;
        iw0 = ow * p.sw - p.pw;
        xbase = img * C * HW + ih0 * Wd + iw0;
    }

    const float *__restrict__ Wt = p.Wt;
    const float *__restrict__ X = p.X;

    vec_t ra[G::A_LOADS];
    float rb[G::B_LOADS];

    auto load_tiles = [&](int kt) {
        const int k0 = kt * BK;
#pragma unroll
        for (int i = 0; i < G::A_LOADS; ++i) {
            const int idx = tid + i * G::NT;
            const int r = idx / G::A_CPR, c = (idx % G::A_CPR) * WA;
            const int gm = m0 + r, gk = k0 + c;
            const int valid = gm < M ? K - gk : 0;
            ra[i] = load_pred<WA>(Wt + (gm < M ? gm : 0) * K + (valid > 0 ? gk : 0), valid);
        }
#pragma unroll
        for (int i = 0; i < G::B_LOADS; ++i) {
            const int k = k0 + brow0 + i * G::B_ROWS_PER_PASS;
            float v = 0.f;
            if (qok && k < K) {
                const int2 t = ktab[k];
                const int ih = ih0 + (t.y & 0xffff), iw = iw0 + (t.y >> 16);
                if ((unsigned)ih < (unsigned)H && (unsigned)iw < (unsigned)Wd) v = X[xbase + t.x];
            }
            rb[i] = v;
        }
    };

    auto store_tiles = [&](int st) {
#pragma unroll
        for (int i = 0; i < G::A_LOADS; ++i) {
            const int idx = tid + i * G::NT;
            const int r = idx / G::A_CPR, c = (idx % G::A_CPR) * WA;
            *reinterpret_cast<vec_t *>(&As[st][r * G::AS + c]) = ra[i];
        }
#pragma unroll
        for (int i = 0; i < G::B_LOADS; ++i)
            Bs[st][(brow0 + i * G::B_ROWS_PER_PASS) * G::BS + bcol] = rb[i];
    };

    typename MF::acc_t acc[G::TM][G::TN];
#pragma unroll
    for (int i = 0; i < G::TM; ++i)
#pragma unroll
        for (int j = 0; j < G::TN; ++j)
#pragma unroll
            for (int r = 0; r < MF::NACC; ++r) acc[i][j][r] = 0.f;

    __syncthreads();  // k-offset table ready
    const int KT = (K + BK - 1) / BK;
    load_tiles(0);
    store_tiles(0);
    __syncthreads();
    for (int kt = 0; kt < KT; ++kt) {
        const int cur = kt & 1;
        const bool has_next = kt + 1 < KT;
        if (has_next) load_tiles(kt + 1);

        const float *as = &As[cur][(wm * WM + lrow) * G::AS + 4 * lgrp];
        const float *bs = &Bs[cur][(4 * lgrp) * G::BS + wn * WN + lrow];
#pragma unroll
        for (int kk = 0; kk < BK; kk += G::KCH) {
            f32x4 a[G::TM];
            float b[G::TN][4];
#pragma unroll
            for (int i = 0; i < G::TM; ++i)
                a[i] = *reinterpret_cast<const f32x4 *>(as + i * MI * G::AS + kk);
#pragma unroll
            for (int j = 0; j < G::TN; ++j)
#pragma unroll
                for (int s = 0; s < 4; ++s) b[j][s] = bs[(kk + s) * G::BS + j * MI];
#pragma unroll
            for (int s = 0; s < 4; ++s)
#pragma unroll
                for (int i = 0; i < G::TM; ++i)
#pragma unroll
                    for (int j = 0; j < G::TN; ++j) acc[i][j] = MF::mma(a[i][s], b[j][s], acc[i][j]);
        }

        if (has_next) store_tiles(cur ^ 1);
        __syncthreads();
    }

    // Epilogue: (oc, q) -> Y[img][oc][pix], masked on the edges.
    float *__restrict__ Y = p.Y;
#pragma unroll
    for (int j = 0; j < G::TN; ++j) {
        const int col = n0 + wn * WN + j * MI + lrow;
        if (col >= N) continue;
        const int img = col / OHW, pix = col - img * OHW;
        float *ybase = Y + img * OC * OHW + pix;
#pragma unroll
        for (int i = 0; i < G::TM; ++i)
#pragma unroll
            for (int r = 0; r < MF::NACC; ++r) {
                const int oc = m0 + wm * WM + i * MI + MF::row(lane, r);
                if (oc < M) ybase[oc * OHW] = acc[i][j][r];
            }
    }
}

template <int BM, int BN, int BK, int WM, int WN, int MI, int PAD>
hipError_t launch_conv_f32(const ConvArgs &a, hipStream_t s) {
    const int M = a.OC, N = a.Nb * a.OH * a.OW, K = a.C * a.R * a.S;
    const unsigned tiles = (unsigned)(((M + BM - 1) / BM) * ((N + BN - 1) / BN));
    const size_t dyn = (size_t)K * sizeof(int2);
    ConvArgs args = a;
    void *kargs[] = {&args};
    const bool vec = (K % 4 == 0) && ((reinterpret_cast<uintptr_t>(a.Wt) & 15) == 0);
    const void *fn = vec ? reinterpret_cast<const void *>(&conv2d_f32_kernel<BM, BN, BK, WM, WN, MI, PAD, true>)
                         : reinterpret_cast<const void *>(&conv2d_f32_kernel<BM, BN, BK, WM, WN, MI, PAD, false>);
    return hipLaunchKernel(fn, dim3(tiles), dim3((BM / WM) * (BN / WN) * 64), kargs, dyn, s);
}

#define XTC_CONV_INSTANCE(BM, BN, BK, WM, WN, MI, PAD)                                        \
    ConvInstance {                                                                            \
        make_sched(BM, BN, BK, WM, WN, MI, MI, (MI == 32 ? 2 : 4), 2, PAD, 0),                 \
            &launch_conv_f32<BM, BN, BK, WM, WN, MI, PAD>                                     \
    }

const ConvInstance kConvInstances[] = {
    XTC_CONV_INSTANCE(64, 128, 32, 32, 64, 32, 4),   // default: OC = 64 in one tile row
    XTC_CONV_INSTANCE(64, 64, 32, 32, 32, 32, 4),
    XTC_CONV_INSTANCE(128, 128, 32, 64, 64, 32, 4),
    XTC_CONV_INSTANCE(64, 128, 32, 32, 64, 16, 4),
};

}  // namespace

const ConvInstance *conv2d_f32_instances(int *count) {
    *count = (int)(sizeof(kConvInstances) / sizeof(kConvInstances[0]));
    return kConvInstances;
}

}  // namespace xtc
