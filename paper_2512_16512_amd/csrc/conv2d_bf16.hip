// bf16 conv2d on the gfx950 matrix cores: X (NCHW) and W (OIHW) hold bf16
// bit patterns, products are exact in fp32, accumulation and Y (NCHW) are
// fp32.  The same zero-padded cross-correlation as the fp32 kernels, computed
// as an implicit GEMM with M = OC, N = batch*OH*OW, K = C*R*S in OIHW order
// (k = (ic*R + kh)*S + kw).
//
// Register-staged, double-buffered LDS tiles, as the fp32 channel-major conv
// kernel: each thread owns one output pixel of the B tile for the whole K
// loop and gathers its input values through a per-workgroup LDS table of
// k -> (input offset, kh, kw), so the gather needs no integer division; an
// input position in the padding is a zero.  The weights are the row-major
// A[OC][K] operand (16-byte loads when K is a multiple of 8 and the base is
// 16-byte aligned).  The fragments are those of the bf16 GEMM: one
// ds_read_b128 per A fragment from k-contiguous padded rows, and two gfx950
// transpose reads per B fragment from the pixel-contiguous B tile.
#include "mfma_bf16.h"
#include "tile_map.h"
#include "xtc_internal.h"

namespace xtc {
namespace {

template <int BM, int BN, int BK, int WM, int WN, int MI, int PAD, bool VEC>
struct ConvBf16Cfg {
    static constexpr int NWM = BM / WM, NWN = BN / WN;
    static constexpr int NT = NWM * NWN * 64;
    static constexpr int TM = WM / MI, TN = WN / MI;
    typedef Bf16Mfma<MI> MF;
    static constexpr int KG = MF::KG;
    static constexpr int KCH = 8 * KG;              // k per MFMA instruction
    static constexpr int AS = BK + PAD;             // LDS row stride of the weight tile
    static constexpr int BS = BN + 32;              // LDS row stride of the pixel tile
    static constexpr int WA = VEC ? 8 : 1;          // weight elements per global load
    static constexpr int A_CPR = BK / WA;
    static constexpr int A_LOADS = BM * BK / (WA * NT);
    static constexpr int B_ROWS_PER_PASS = NT / BN; // gather: a thread owns one pixel column
    static constexpr int B_LOADS = BK / B_ROWS_PER_PASS;
    typedef typename VecU16<WA>::t vec_t;
    static_assert(BM % WM == 0 && BN % WN == 0, "wave tile must divide the block tile");
    static_assert(WM % MI == 0 && WN % MI == 0, "MFMA tile must divide the wave tile");
    static_assert(NT % BN == 0 && BK % B_ROWS_PER_PASS == 0, "gather split");
    static_assert(A_LOADS * WA * NT == BM * BK, "weight tile must split evenly");
    static_assert(BK % KCH == 0, "block_k must be a multiple of the MFMA k");
    static_assert(PAD % 8 == 0, "padding must keep 16-byte alignment");
};

template <int BM, int BN, int BK, int WM, int WN, int MI, int PAD, bool VEC>
__global__ void __launch_bounds__((BM / WM) * (BN / WN) * 64)
conv2d_bf16_kernel(ConvArgs p) {
    typedef ConvBf16Cfg<BM, BN, BK, WM, WN, MI, PAD, VEC> G;
    typedef typename G::MF MF;
    typedef typename G::vec_t vec_t;
    constexpr int WA = G::WA;

    __shared__ __attribute__((aligned(16))) unsigned short As[2][BM * G::AS];
    __shared__ __attribute__((aligned(16))) unsigned short Bs[2][BK * G::BS];
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

    const int RS = R * S;
    for (int k = tid; k < K; k += G::NT) {
        const int ic = k / RS, rem = k - ic * RS;
        const int kh = rem / S, kw = rem - kh * S;
        ktab[k] = make_int2(ic * HW + kh * Wd + kw, kh | (kw << 16));
    }

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

    const unsigned short *__restrict__ Wt = reinterpret_cast<const unsigned short *>(p.Wt);
    const unsigned short *__restrict__ X = reinterpret_cast<const unsigned short *>(p.X);

    vec_t ra[G::A_LOADS];
    unsigned short rb[G::B_LOADS];

    auto load_tiles = [&](int kt) {
        const int k0 = kt * BK;
#pragma unroll
        for (int i = 0; i < G::A_LOADS; ++i) {
            const int idx = tid + i * G::NT;
            const int r = idx / G::A_CPR, c = (idx % G::A_CPR) * WA;
            const int gm = m0 + r, gk = k0 + c;
            const int valid = gm < M ? K - gk : 0;
            ra[i] = load_pred_u16<WA>(Wt + (gm < M ? gm : 0) * K + (valid > 0 ? gk : 0), valid);
        }
#pragma unroll
        for (int i = 0; i < G::B_LOADS; ++i) {
            const int k = k0 + brow0 + i * G::B_ROWS_PER_PASS;
            unsigned short v = 0;
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
                if (oc < M) ybase[oc * OHW] = (p.relu && acc[i][j][r] < 0.f) ? 0.f : acc[i][j][r];
            }
    }
}

template <int BM, int BN, int BK, int WM, int WN, int MI, int PAD>
hipError_t launch_conv_bf16(const ConvArgs &a, hipStream_t s) {
    const int M = a.OC, N = a.Nb * a.OH * a.OW, K = a.C * a.R * a.S;
    const unsigned tiles = (unsigned)(((M + BM - 1) / BM) * ((N + BN - 1) / BN));
    const size_t dyn = (size_t)K * sizeof(int2);
    ConvArgs args = a;
    void *kargs[] = {&args};
    const bool vec = (K % 8 == 0) && ((reinterpret_cast<uintptr_t>(a.Wt) & 15) == 0);
    const void *fn =
        vec ? reinterpret_cast<const void *>(&conv2d_bf16_kernel<BM, BN, BK, WM, WN, MI, PAD, true>)
            : reinterpret_cast<const void *>(&conv2d_bf16_kernel<BM, BN, BK, WM, WN, MI, PAD, false>);
    return hipLaunchKernel(fn, dim3(tiles), dim3((BM / WM) * (BN / WN) * 64), kargs, dyn, s);
}

#define XTC_CONV_BF16_INSTANCE(BM, BN, BK, WM, WN, MI, PAD)                                   \
    ConvInstance {                                                                            \
        make_sched(BM, BN, BK, WM, WN, MI, MI, (MI == 32 ? 16 : 32), 2, PAD, 0),               \
            &launch_conv_bf16<BM, BN, BK, WM, WN, MI, PAD>,                                   \
            &occupancy_of<&conv2d_bf16_kernel<BM, BN, BK, WM, WN, MI, PAD, true>,             \
                          (BM / WM) * (BN / WN) * 64, (int)sizeof(int2)>                      \
    }

const ConvInstance kConvBf16Instances[] = {
    XTC_CONV_BF16_INSTANCE(64, 128, 32, 32, 64, 32, 8),   // default for OC <= 64
    XTC_CONV_BF16_INSTANCE(128, 128, 32, 64, 64, 32, 8),  // default for OC > 64
    XTC_CONV_BF16_INSTANCE(64, 64, 32, 32, 32, 32, 8),    // few output pixels
    XTC_CONV_BF16_INSTANCE(64, 128, 64, 32, 64, 32, 8),
    XTC_CONV_BF16_INSTANCE(64, 128, 64, 32, 64, 16, 8),   // 16x16x32 instruction tile
};

}  // namespace

const ConvInstance *conv2d_bf16_instances(int *count) {
    *count = (int)(sizeof(kConvBf16Instances) / sizeof(kConvBf16Instances[0]));
    return kConvBf16Instances;
}

}  // namespace xtc
