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
#include "lds_dma.h"
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

// ---------------------------------------------------------------------------
// Halo-tiled bf16 kernel (k_order = 2) for stride-1 3x3 convolutions of rows
// of about 56 pixels.  The gather above loads every input value once per
// tap; here a stage stages a 16-channel input patch once for all nine taps:
//  - a workgroup computes 64 output channels x 256 consecutive output pixels
//    of one image (four 64x64 waves of 32x32x16 instructions).  The pixels
//    span at most 6 output rows when OW >= 51, so their inputs fit in a patch
//    of PR = 8 input rows;
//  - the patch is stored channel-innermost, [half][row][column][8 channels],
//    16 bytes per cell: the B fragment of a lane (8 channels of one pixel at
//    one tap) is then one 16-byte read of the cell the tap points at, for
//    any column shift.  Input column iw sits at patch column iw + CO;
//    columns and rows outside the image hold zeros;
//  - bank layout: gfx950 serves a ds_read_b128 in four phases of 16 lanes
//    ({0-3, 12-15, 20-23, 24-27}, {4-11, 16-19, 28-31} and the same + 32),
//    and a 16-byte cell occupies one of 16 bank groups.  Patch row r (64
//    columns) is stored rotated by (r * OW) mod 16 cells inside a row of 80
//    cells, so the 32 pixels of a fragment stay on consecutive bank groups
//    also when they wrap to the next output row (unrotated, the wrap moved
//    them by OW - 64 groups onto other lanes' banks).  Output channel rows
//    of the weights hold their two 8-channel halves swapped when bit 3 of
//    the channel is set, which puts the rows a phase reads on distinct
//    groups.  Stores are served 8 lanes at a time over 32 banks (128
//    bytes), so a thread writes its two patch cells in an order that keeps
//    each group of 8 lanes on 8 distinct 16-byte slots;
//  - the patch is filled through registers: a thread loads one dword (two
//    neighbouring input columns) of each of the 16 channels and repacks them
//    into the two columns' cells.  NCHW rows of even width keep every pair
//    dword-aligned;
//  - the weights of a stage, W[oc][c0 .. c0+15][kh][kw], are 144 contiguous
//    values per output channel (16-byte aligned when C % 16 == 0); a thread
//    loads one 8-channel slab (72 values) and repacks it into the
//    [tap][oc][16 channels] cells of the A fragments;
//  - the reduction runs over 16-channel chunks and, inside a chunk, over the
//    taps; an instruction's two k lane groups take channels 0-7 and 8-15 of
//    the tap.
namespace halo_bf16 {
constexpr int BM = 64, BN = 256, WM = 64, WN = 64, NWAVES = 4, NT = 256;
constexpr int MI = 32, TM = WM / MI, TN = WN / MI;
constexpr int CC = 16;                        // channels per stage
constexpr int NTAP = 9;
constexpr int PR = 8;                         // patch rows
constexpr int PC = 64;                        // patch columns
constexpr int PCA = 80;                       // cells per stored patch row (PC + the rotation)
constexpr int CO = 2;                         // patch column of input column 0 (even)
constexpr int CELL = 16;                      // bytes: 8 channels of one (row, column)
constexpr int HALF = PR * PCA * CELL;         // one 8-channel half of the patch
constexpr int P_BYTES = 2 * HALF;
constexpr int W_BYTES = NTAP * BM * CC * 2;   // [tap][oc][16 channels]
constexpr int STAGE_BYTES = P_BYTES + W_BYTES;
static_assert(NT == PR * PC / 2, "one patch column pair per thread");
static_assert(2 * BM <= NT, "one weight slab per thread");
}  // namespace halo_bf16

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

__global__ void __launch_bounds__(halo_bf16::NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
conv2d_bf16_halo_kernel(ConvArgs p) {
    using namespace halo_bf16;
    typedef Bf16Mfma<MI> MF;
    __shared__ __attribute__((aligned(16))) unsigned char smem[2 * STAGE_BYTES];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int lrow = lane % MI, lgrp = lane / MI;   // lgrp: channel half of the fragments

    const int C = p.C, H = p.H, Wd = p.W;
    const int OC = p.OC, OW = p.OW, OHW = p.OH * p.OW;
    const int chunks = (OHW + BN - 1) / BN;   // per image
    const int tiles_m = (OC + BM - 1) / BM, tiles_n = p.Nb * chunks;
    int tm, tn;
    tile_coords(blockIdx.x, gridDim.x, tiles_m, tiles_n, p.raster, p.xcd_remap, tm, tn);
    const int m0 = tm * BM;
    const int img = tn / chunks, p0 = (tn - img * chunks) * BN;
    const int oh0 = p0 / OW;                  // first output row of the tile
    const int ih0 = oh0 - p.ph;               // input row of patch row 0
    const int KT = C / CC;

    // Patch loads: patch row pr, column pair cp (input columns 2cp - CO, +1),
    // through a buffer resource: one offset per thread, the channel step in a
    // scalar offset, and pairs outside the image at an out-of-range offset,
    // which reads zeros.
    const int pr = tid >> 5, cp = tid & 31;
    const int prot = (pr * OW) & 15;            // rotation of this patch row
    const bool sw = (cp >> 2) & 1;              // store order of the two cells
    const int cell0 = (pr * PCA + 2 * cp + prot + (sw ? 1 : 0)) * CELL;
    const int cell1 = (pr * PCA + 2 * cp + prot + (sw ? 0 : 1)) * CELL;
    const int ih = ih0 + pr, iw = 2 * cp - CO;
    const bool pok = ih >= 0 && ih < H && iw >= 0 && iw + 1 < Wd;
    // dwords per channel plane; read into a scalar register, since the
    // compiler otherwise recomputes it on both sides of the divergent select
    // below and then holds it per lane, which turns every buffer load that
    // takes it as a scalar offset into a loop over lanes
    const int HW2 = __builtin_amdgcn_readfirstlane(H * Wd / 2);
    const int xoff = pok ? (img * C * HW2 + (ih * Wd + iw) / 2) * 4 : kOOB;
    const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<unsigned short *>(reinterpret_cast<const unsigned short *>(p.X)), 0,
        p.Nb * C * HW2 * 4, 0x00020000);
    // Weight loads (threads 0 .. 2*BM-1): output channel m0 + woc, channels
    // 8*wh .. 8*wh+7 of the stage, all nine taps: nine 16-byte chunks.
    const int woc = tid >> 1, wh = tid & 1;
    // byte offset of this thread's 8-channel half in an output channel row
    // (halves swapped when bit 3 of the channel is set)
    const int wslot = (woc * CC + 8 * (wh ^ ((woc >> 3) & 1))) * 2;
    const bool wthr = tid < 2 * BM;
    const bool wok = wthr && m0 + woc < OC;
    const int woff = wok ? ((m0 + woc) * C + 8 * wh) * NTAP * 2 : kOOB;
    const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<unsigned short *>(reinterpret_cast<const unsigned short *>(p.Wt)), 0,
        OC * C * NTAP * 2, 0x00020000);

    // two register sets, so that the loads of a stage are in flight for two
    // stages' worth of matrix work before they are stored
    unsigned xs[2][CC];
    u32x4_t ws[2][NTAP];
    // Loads of stage kt into set S.  Past the last stage (live false) the
    // offsets are out of range: the loads return zeros without touching
    // memory.  Loads under a branch would make the compiler's wait before
    // each store count conservatively, and wait for loads it does not need.
    auto gload = [&](auto S, int kt, bool live) __attribute__((always_inline)) {
        const int c0 = live ? kt * CC : 0;
        const int xo = live ? xoff : kOOB, wo = live ? woff : kOOB;
#pragma unroll
        for (int c = 0; c < CC; ++c)
            xs[S][c] = __builtin_amdgcn_raw_buffer_load_b32(rx, xo, (c0 + c) * HW2 * 4, 0);
        // every thread issues the weight loads (threads without a slab at an
        // out-of-range offset), so that all waves count the same loads
#pragma unroll
        for (int q = 0; q < NTAP; ++q)
            ws[S][q] = __builtin_amdgcn_raw_buffer_load_b128(rw, wo, c0 * NTAP * 2 + q * 16, 0);
    };
    // halfword e (0 .. 71) of the weight slab in set S
    auto wv = [&](auto S, int e) __attribute__((always_inline)) {
        return (ws[S][e >> 3][(e >> 1) & 3] >> (16 * (e & 1))) & 0xffffu;
    };
    auto lstore = [&](auto S) __attribute__((always_inline)) {
        unsigned char *P = smem + S * STAGE_BYTES;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            u32x4_t lo, hi;   // columns 2cp and 2cp + 1
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const unsigned a = xs[S][8 * h + 2 * j], b = xs[S][8 * h + 2 * j + 1];
                lo[j] = (a & 0xffffu) | (b << 16);
                hi[j] = (a >> 16) | (b & 0xffff0000u);
            }
            // writes are served 8 lanes at a time over 128 bytes of banks:
            // threads whose column pair has bit 2 set write their odd cell
            // first, so each group of 8 lanes covers 8 distinct 16-byte slots
            const u32x4_t c0 = sw ? hi : lo, c1 = sw ? lo : hi;
            *reinterpret_cast<u32x4_t *>(P + h * HALF + cell0) = c0;
            *reinterpret_cast<u32x4_t *>(P + h * HALF + cell1) = c1;
        }
        if (wthr) {
            unsigned char *Wl = P + P_BYTES;
#pragma unroll
            for (int t = 0; t < NTAP; ++t) {
                u32x4_t v;
#pragma unroll
                for (int d = 0; d < 4; ++d)
                    v[d] = wv(S, 2 * d * NTAP + t) | (wv(S, (2 * d + 1) * NTAP + t) << 16);
                *reinterpret_cast<u32x4_t *>(Wl + t * BM * CC * 2 + wslot) = v;
            }
        }
    };

    // Fragment bases.  A: output channel i*32 + lrow, channels 8*lgrp .. +7
    // (halves swapped when bit 3 of the channel is set).  B: this lane's
    // pixel of column block j, one base per kernel row kh (the rotation
    // depends on the patch row); patch position (0, 0) past the image.
    const int a_base = P_BYTES + (lrow * CC + 8 * (lgrp ^ ((lrow >> 3) & 1))) * 2;
    int b_base[TN][3];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int pix = p0 + wave * WN + j * MI + lrow;
        int r = 0, c = 0;
        if (pix < OHW) {
            const int oh = pix / OW, ow = pix - oh * OW;
            r = oh - oh0;
            c = ow - p.pw + CO;
        }
#pragma unroll
        for (int kh = 0; kh < 3; ++kh)
            b_base[j][kh] = lgrp * HALF + ((r + kh) * PCA + c + (((r + kh) * OW) & 15)) * CELL;
    }

    typename MF::acc_t acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < MF::NACC; ++r) acc[i][j][r] = 0.f;

    u16x8 af[2][TM], bfr[2][TN];
    auto load_frags = [&](int buf, int t, int fb) __attribute__((always_inline)) {
        const unsigned char *P = smem + buf * STAGE_BYTES;
        const int kh = t / 3, kw = t - 3 * kh;
#pragma unroll
        for (int i = 0; i < TM; ++i)
            af[fb][i] = *reinterpret_cast<const u16x8 *>(P + a_base + ((t * BM + i * MI) * CC) * 2);
#pragma unroll
        for (int j = 0; j < TN; ++j)
            bfr[fb][j] = *reinterpret_cast<const u16x8 *>(P + b_base[j][kh] + kw * CELL);
    };
    auto mfmas = [&](int fb) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc[i][j] = MF::mma(af[fb][i], bfr[fb][j], acc[i][j]);
    };

    // Stage kt is computed from LDS buffer kt % 2, which register set kt % 2
    // filled; that set then takes the loads of stage kt + 2, and set
    // (kt + 1) % 2, loaded a stage earlier, is stored into the other buffer
    // after the nine taps.
    const std::integral_constant<int, 0> S0;
    const std::integral_constant<int, 1> S1;
    auto stage = [&](auto S, int kt) __attribute__((always_inline)) {
        constexpr int NS = 1 - decltype(S)::value;
        gload(S, kt + 2, kt + 2 < KT);
        // keep the loads ahead of the taps (the scheduler would otherwise sink
        // them to the end of the stage, one stage before their use)
        __builtin_amdgcn_sched_barrier(0);
        load_frags(S, 0, 0);
#pragma unroll
        for (int t = 0; t < NTAP; ++t) {
            if (t + 1 < NTAP) load_frags(S, t + 1, (t + 1) & 1);
            mfmas(t & 1);
        }
        if (kt + 1 < KT) lstore(std::integral_constant<int, NS>());
        __syncthreads();
    };
    gload(S0, 0, true);
    gload(S1, 1, KT > 1);
    lstore(S0);
    __syncthreads();
    for (int kt = 0; kt < KT; kt += 2) {
        stage(S0, kt);
        if (kt + 1 < KT) stage(S1, kt + 1);
    }

    float *__restrict__ Y = p.Y + (size_t)img * OC * OHW;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int pix = p0 + wave * WN + j * MI + lrow;
        if (pix >= OHW) continue;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int r = 0; r < MF::NACC; ++r) {
                const int oc = m0 + i * MI + MF::row(lane, r);
                if (oc < OC)
                    __builtin_nontemporal_store((p.relu && acc[i][j][r] < 0.f) ? 0.f : acc[i][j][r],
                                                &Y[oc * OHW + pix]);
            }
    }
}

// Shapes the halo kernel covers; anything else runs the gather kernel with
// 64x128 tiles.
inline bool bf16_halo_eligible(const ConvArgs &a) {
    using namespace halo_bf16;
    if (a.R != 3 || a.S != 3 || a.sh != 1 || a.sw != 1) return false;
    if (a.C % CC != 0 || a.W % 2 != 0 || a.pw > CO) return false;
    if (a.OW - a.pw + 3 > PC - 1) return false;            // last patch column used
    if ((reinterpret_cast<uintptr_t>(a.X) & 3) != 0 || (reinterpret_cast<uintptr_t>(a.Wt) & 15) != 0)
        return false;
    const int span = (BN - 1 + a.OW - 1) / a.OW + 1;      // output rows a tile can touch
    return span + 2 <= PR;
}

hipError_t launch_conv_bf16_halo(const ConvArgs &a, hipStream_t s) {
    if (!bf16_halo_eligible(a)) return launch_conv_bf16<64, 128, 32, 32, 64, 32, 8>(a, s);
    const int OHW = a.OH * a.OW;
    const unsigned tiles = (unsigned)(((a.OC + halo_bf16::BM - 1) / halo_bf16::BM) * a.Nb *
                                      ((OHW + halo_bf16::BN - 1) / halo_bf16::BN));
    ConvArgs args = a;
    void *kargs[] = {&args};
    return hipLaunchKernel(reinterpret_cast<const void *>(&conv2d_bf16_halo_kernel), dim3(tiles),
                           dim3(halo_bf16::NT), kargs, 0, s);
}

// ---------------------------------------------------------------------------
// Row-streaming bf16 kernel (k_order = 3) for stride-1 3x3 convolutions of 64
// input channels with output rows of at most 64 pixels.  With bf16 inputs such
// a layer does about 190 FLOP per HBM byte, below the matrix cores' ridge
// (about 315), so the kernel is laid out for streaming X in and Y out at HBM
// rate rather than for matrix-core reuse:
//  - a workgroup owns 64 output channels of one image and a band of
//    consecutive output rows, and walks down the band RO = 2 output rows per
//    step, so that each input row enters LDS once per band and the output
//    of a step is written while the following rows are computed;
//  - all C*R*S = 576 weights of its 64 output channels stay in LDS for the
//    whole band (72 KiB, loaded once);
//  - input rows pass through a ring of NR = 8 LDS rows: the four rows a step
//    reads, the two the next step adds (stored at the end of the step,
//    published by the step's barrier) and two slots free for refilling; the
//    loads of the rows a step adds are issued during the step before (so
//    that the first step's own instructions cover the arrival of those
//    rows), into one of two register sets;
//  - wave w computes 32 output channels (half w & 1) x 32 pixels (half
//    w >> 1) of both output rows with 32x32x16 instructions, pixels as the
//    row operand and output channels as the column operand;
//  - one fragment of input row r (32 pixels, 8 channels, one column shift
//    kw) serves every output row of the step that reads row r, one per
//    kernel row kh: four input rows feed the 2 x 3 (output row, kh) pairs.
//    Per 16-channel k-step a wave reads 4 + 3 fragments for 6 instructions,
//    which keeps LDS below the matrix cores' rate and a group's reads within
//    the 15 the LDS counter can wait past;
//  - an input row is stored channel-innermost, one 16-byte cell of 8
//    channels per (column, 8-channel group), 64 columns with input column iw
//    at column iw + CO and zeros outside the image.  Group g of column c sits
//    at slot g ^ h(c), h(c) = ((c >> 1) ^ (c & ~3)) & 7, which keeps both the
//    fragment reads (each phase: 16 lanes of a 32-column run, one group) and
//    the staging writes (8 lanes of consecutive column pairs per phase, each
//    lane writing its two cells in an order that alternates every four
//    lanes) free of bank conflicts at every column shift;
//  - a weight cell holds 8 channels of one (tap, output channel); the eight
//    cells of output channel o sit at slots g ^ h(o), the same pattern, since
//    a weight fragment (32 output channels x two groups) is addressed like a
//    pixel fragment;
//  - each wave turns its output rows around through a 4 KiB LDS area of its
//    own before storing them, so that a store instruction writes runs of 128
//    bytes of one channel row (ring 64 KiB + weights 72 KiB + 4 x 4 KiB:
//    152 KiB, one workgroup per CU).
namespace rows_bf16 {
constexpr int NT = 256;                   // four waves
constexpr int BM = 64;                    // output channels per workgroup
constexpr int CH = 64;                    // input channels (all resident)
constexpr int NCG = CH / 8;               // 8-channel cells per column
constexpr int NKS = CH / 16;              // 16-channel instruction k-steps per tap
constexpr int NTAP = 9;
constexpr int RO = 2;                     // output rows per step
constexpr int NR = 8;                     // input rows in the ring
constexpr int PC = 64;                    // stored columns per input row
constexpr int CO = 2;                     // stored column of input column 0 (even)
constexpr int ROWB = PC * NCG * 16;       // bytes per stored input row
constexpr int RING_BYTES = NR * ROWB;
constexpr int W_BYTES = NTAP * BM * NCG * 16;
constexpr int STG_BYTES = 32 * 128;       // per wave: one output row, 32 channels x 32 pixels
constexpr int LDS_BYTES = RING_BYTES + W_BYTES + (NT / 64) * STG_BYTES;
static_assert(NT == 32 * NCG, "one (column pair, cell group) per thread");
static_assert(2 * NT == BM * NCG, "two weight slabs per thread");
static_assert(NR >= 3 * RO + 2, "ring: a step's rows, the next step's, and the slots being refilled");
// slot swizzle of the cells of one column (or output channel)
__device__ __forceinline__ int swz(int c) { return ((c >> 1) ^ (c & ~3)) & 7; }
}  // namespace rows_bf16

__global__ void __launch_bounds__(rows_bf16::NT)
conv2d_bf16_rows_kernel(ConvArgs p) {
    using namespace rows_bf16;
    typedef Bf16Mfma<32> MF;
    __shared__ __attribute__((aligned(16))) unsigned char smem[LDS_BYTES];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int l32 = lane & 31, lg = lane >> 5;

    const int H = p.H, Wd = p.W, OC = p.OC, OH = p.OH, OW = p.OW;
    const int band_rows = p.tile_px;
    const int nbands = (OH + band_rows - 1) / band_rows;
    const int tiles_m = (OC + BM - 1) / BM, tiles_n = p.Nb * nbands;
    int tm, tn;
    tile_coords(blockIdx.x, gridDim.x, tiles_m, tiles_n, p.raster, p.xcd_remap, tm, tn);
    const int m0 = tm * BM;
    const int img = tn / nbands, band = tn - img * nbands;
    const int oh_a = band * band_rows;
    const int rows = min(band_rows, OH - oh_a);   // output rows of the band
    const int nsteps = (rows + RO - 1) / RO;
    const int ih0 = oh_a - p.ph;                   // input row of band row 0
    const int nin = RO * nsteps + 2;               // input rows the band reads

    // ---- input rows: thread (q, g) loads column pair q (input columns
    // 2q - CO, +1) of channels 8g .. 8g+7, one dword per channel; rows and
    // pairs outside the image are read at an out-of-range offset (zeros).
    const int q = tid & 31, g = tid >> 5;
    const int iwp = 2 * q - CO;
    const bool colok = iwp >= 0 && iwp + 1 < Wd;
    const int plane = __builtin_amdgcn_readfirstlane(H * Wd * 2);      // bytes per channel plane
    const int xcol = ((img * CH + 8 * g) * H) * Wd * 2 + iwp * 2;
    const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float *>(p.X), 0, p.Nb * CH * plane, 0x00020000);
    // Two register sets.  Loads and output stores are unconditional
    // (out-of-range offsets instead of branches), so the compiler's counted
    // waits before a set is stored do not include the stores issued after
    // its loads.
    unsigned xv[2][RO][8];
    auto load_rows = [&](auto S, int r0) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < RO; ++i) {
            const int r = r0 + i, ih = ih0 + r;
            const bool ok = colok & (r < nin) & (ih >= 0) & (ih < H);
            const int o = ok ? xcol + ih * Wd * 2 : kOOB;
#pragma unroll
            for (int c = 0; c < 8; ++c)
                xv[S][i][c] = __builtin_amdgcn_raw_buffer_load_b32(rx, o, c * plane, 0);
        }
    };
    // the thread's two cells; lanes with bit 2 of q set write their odd
    // column first
    const bool wodd = (q >> 2) & 1;
    const int c0 = 2 * q + (wodd ? 1 : 0), c1 = 2 * q + (wodd ? 0 : 1);
    const int cell0 = c0 * (NCG * 16) + ((g ^ swz(c0)) << 4);
    const int cell1 = c1 * (NCG * 16) + ((g ^ swz(c1)) << 4);
    auto store_rows = [&](auto S, int r0) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < RO; ++i) {
            unsigned char *R = smem + ((r0 + i) % NR) * ROWB;
            u32x4_t ev, od;   // columns 2q and 2q + 1
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const unsigned a = xv[S][i][2 * j], b = xv[S][i][2 * j + 1];
                ev[j] = (a & 0xffffu) | (b << 16);
                od[j] = (a >> 16) | (b & 0xffff0000u);
            }
            *reinterpret_cast<u32x4_t *>(R + cell0) = wodd ? od : ev;
            *reinterpret_cast<u32x4_t *>(R + cell1) = wodd ? ev : od;
        }
    };

    // ---- weights: slab s (= tid, tid + NT) is output channel s >> 3,
    // channels 8(s & 7) .. +7, all nine taps: 72 contiguous values of the
    // OIHW row, nine 16-byte loads, repacked into one cell per tap.
    const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float *>(p.Wt), 0, OC * CH * NTAP * 2, 0x00020000);
    unsigned char *const Wl = smem + RING_BYTES;
    const std::integral_constant<int, 0> S0;
    const std::integral_constant<int, 1> S1;
    // prologue: the weights first (they come from L2, and the in-order
    // memory counter would otherwise make their wait include the input
    // rows' HBM latency), then band rows 0 .. 3; rows 4, 5 (set 0), which
    // the first step stores at its end, stay in flight
    u32x4_t ws[2][NTAP];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int s = tid + h * NT;
        const int oc = s >> 3, wg = s & 7;
        const int off = m0 + oc < OC ? ((m0 + oc) * CH + 8 * wg) * NTAP * 2 : kOOB;
#pragma unroll
        for (int t = 0; t < NTAP; ++t) ws[h][t] = __builtin_amdgcn_raw_buffer_load_b128(rw, off, 16 * t, 0);
    }
    load_rows(S0, 0);
    load_rows(S1, RO);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int s = tid + h * NT;
        const int oc = s >> 3, wg = s & 7;
        auto wv = [&](int e) __attribute__((always_inline)) {   // halfword e = channel e / 9, tap e % 9
            return (ws[h][e >> 3][(e >> 1) & 3] >> (16 * (e & 1))) & 0xffffu;
        };
        const int slot = oc * (NCG * 16) + ((wg ^ swz(oc)) << 4);
#pragma unroll
        for (int t = 0; t < NTAP; ++t) {
            u32x4_t v;
#pragma unroll
            for (int d = 0; d < 4; ++d) v[d] = wv(2 * d * NTAP + t) | (wv((2 * d + 1) * NTAP + t) << 16);
            *reinterpret_cast<u32x4_t *>(Wl + t * BM * NCG * 16 + slot) = v;
        }
    }
    store_rows(S0, 0);
    store_rows(S1, RO);
    load_rows(S0, 2 * RO);
    __syncthreads();

    // ---- fragment offsets.  B (weights): output channel 32*(wave & 1) +
    // l32, group 2*kstep + lg.  A (pixels): pixel 32*(wave >> 1) + l32 of the
    // output row (lanes past OW read a valid cell and are not stored),
    // column shift kw, group 2*kstep + lg.
    const int oc_l = 32 * (wave & 1) + l32;
    // lanes past OW take the pixel 32 to the left (same banks, so the read
    // stays conflict-free), or the last pixel when there is none
    int px_l = 32 * (wave >> 1) + l32;
    if (px_l >= OW) px_l = px_l >= 32 && px_l - 32 < OW ? px_l - 32 : OW - 1;
    int b_off[NKS], a_off[3][NKS];
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
        b_off[ks] = oc_l * (NCG * 16) + (((2 * ks + lg) ^ swz(oc_l)) << 4);
#pragma unroll
        for (int kw = 0; kw < 3; ++kw) {
            const int col = px_l + kw - p.pw + CO;
            a_off[kw][ks] = col * (NCG * 16) + (((2 * ks + lg) ^ swz(col)) << 4);
        }
    }

    // ---- output: lane (l32, lg) of wave w holds, per output row, pixels
    // 32*(w >> 1) + 8i + 4lg .. +3 (i = 0..3) of output channel m0 + oc_l.
    // Stored as they are, each 16-byte store instruction would write 32
    // pieces of 32 bytes (one per channel).  Instead each row goes through
    // the wave's own LDS area ([channel][8 chunks of 4 pixels], chunk slot
    // c ^ (channel & 7): conflict-free both ways) and is read back so that
    // lane j holds chunk j & 7 of channel 8s + (j >> 3): four stores per row,
    // each of 8 runs of 128 bytes.  A store whose channel, row or pixels lie
    // outside Y goes to an out-of-range offset and is dropped.
    const __amdgpu_buffer_rsrc_t ry = __builtin_amdgcn_make_buffer_rsrc(
        p.Y, 0, p.Nb * OC * OH * OW * 4, 0x00020000);
    unsigned char *const stg = smem + RING_BYTES + W_BYTES + wave * STG_BYTES;
    const int ch_rd = lane & 7, oc_rd = lane >> 3;   // chunk and channel (within 8) read back
    const int px_rd = 32 * (wave >> 1) + 4 * ch_rd;
    // byte offset in Y of band row 0 for each of the lane's four stores of a
    // row (out of range where the channel or the pixels lie outside Y); a
    // row adds its row offset, which keeps an out-of-range offset out of
    // range (unsigned, and Y spans less than 2^31 bytes)
    unsigned soff[4];
#pragma unroll
    for (int s4 = 0; s4 < 4; ++s4) {
        const int oc = m0 + 32 * (wave & 1) + 8 * s4 + oc_rd;
        soff[s4] = (oc < OC) & (px_rd < OW) ? (unsigned)((((img * OC + oc) * OH + oh_a) * OW + px_rd) * 4)
                                             : (unsigned)kOOB;
    }
    // relu as a lower bound (-inf: none); accumulators start at +0, so a
    // -0 result, which the bound would not keep, cannot occur
    const float lo = p.relu ? 0.f : -__builtin_inff();
    // A step's outputs are stored during the next step, one store per
    // k-step group, and its row loads are spread the same way: with one
    // wave per SIMD a burst of memory instructions stalls the wave at the
    // memory queue while its matrix instructions wait behind them.
    constexpr int NPART = RO * 4;               // output stores (and load pairs) per step
    f32x4 pend[NPART];
    int pend_off[NPART];
#pragma unroll
    for (int k = 0; k < NPART; ++k) pend_off[k] = kOOB;
    auto store_part = [&](int k) __attribute__((always_inline)) {
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, pend[k]), ry, pend_off[k], 0, 0);
    };
    // loads of band rows r0, r0 + 1 into set S, part k: row k / 4, channels
    // 2(k % 4), +1
    auto load_part = [&](auto S, int r0, int k) __attribute__((always_inline)) {
        const int i = k / 4, r = r0 + i, ih = ih0 + r;
        const bool ok = colok & (r < nin) & (ih >= 0) & (ih < H);
        const int o = ok ? xcol + ih * Wd * 2 : kOOB;
#pragma unroll
        for (int c = 2 * (k % 4); c < 2 * (k % 4) + 2; ++c)
            xv[S][i][c] = __builtin_amdgcn_raw_buffer_load_b32(rx, o, c * plane, 0);
    };

    // Fragments: the (kw, k-step) groups of a step in order, double-buffered
    // in registers.  The reads of the next group are issued between the
    // matrix instructions of the current one (a run of reads would likewise
    // stall the wave at the LDS queue), and the last group of a step reads
    // the first group of the next step.
    constexpr int NGRP = 3 * NKS;
    constexpr int NREAD = 3 + RO + 2;            // reads per group
    constexpr int NMMA = 3 * RO;                 // instructions per group
    static_assert(NGRP % 2 == 0 && NREAD >= NMMA && NGRP - 1 >= NPART, "group parity and interleave");
    u16x8 af[2][RO + 2], bf[2][3];
    auto frags = [&](int fb, int grp, int st) __attribute__((always_inline)) {
        const int kw = grp / NKS, ks = grp % NKS;
#pragma unroll
        for (int kh = 0; kh < 3; ++kh)
            bf[fb][kh] = *reinterpret_cast<const u16x8 *>(Wl + (kh * 3 + kw) * BM * NCG * 16 + b_off[ks]);
#pragma unroll
        for (int i = 0; i < RO + 2; ++i)
            af[fb][i] = *reinterpret_cast<const u16x8 *>(smem + ((RO * st + i) % NR) * ROWB + a_off[kw][ks]);
    };
    auto interleave = [&](bool mem) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < NMMA; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one LDS read
            if (mem && i == 1) __builtin_amdgcn_sched_group_barrier(0x040, 1, 0);   // the store
            if (mem && i == 3) __builtin_amdgcn_sched_group_barrier(0x020, 2, 0);   // the loads
        }
        __builtin_amdgcn_sched_group_barrier(0x100, NREAD - NMMA, 0);
        __builtin_amdgcn_sched_barrier(0);
    };

    // step st: its groups load, into set SL, the rows the next step stores;
    // at its end it stores, from set SS, the rows the step after it adds
    auto step = [&](auto SL, auto SS, int st) __attribute__((always_inline)) {
        typename MF::acc_t acc[RO];
#pragma unroll
        for (int o = 0; o < RO; ++o)
#pragma unroll
            for (int r = 0; r < MF::NACC; ++r) acc[o][r] = 0.f;
        auto mmas = [&](int fb) __attribute__((always_inline)) {
#pragma unroll
            for (int kh = 0; kh < 3; ++kh)
#pragma unroll
                for (int o = 0; o < RO; ++o) acc[o] = MF::mma(af[fb][o + kh], bf[fb][kh], acc[o]);
        };
#pragma unroll
        for (int grp = 0; grp + 1 < NGRP; ++grp) {
            frags((grp + 1) & 1, grp + 1, st);
            mmas(grp & 1);
            if (grp < NPART) {
                store_part(grp);
                load_part(SL, RO * st + 2 * RO + 2, grp);
            }
            interleave(grp < NPART);
        }
        // the next step's new rows into the ring (loaded during the previous
        // step; their slots were last read two steps ago), then a barrier:
        // every wave has stored them and finished the previous step's reads
        store_rows(SS, RO * st + RO + 2);
        __syncthreads();
        frags(0, 0, st + 1);
        mmas(1);
        interleave(false);
        // this step's outputs, through the staging area, stored during the
        // next step (write-back stores: nontemporal ones of lines that other
        // workgroups' stores complete would cost whole lines of HBM writes).
        // The wave's LDS operations run in order, so row 1 may overwrite
        // the area row 0 was read from.
#pragma unroll
        for (int o = 0; o < RO; ++o) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                f32x4 v;
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = __builtin_fmaxf(acc[o][4 * i + r], lo);
                *reinterpret_cast<f32x4 *>(stg + l32 * 128 + (((2 * i + lg) ^ (l32 & 7)) << 4)) = v;
            }
            const bool rok = RO * st + o < rows;   // uniform
            const unsigned roff = (unsigned)((RO * st + o) * OW * 4);
#pragma unroll
            for (int s4 = 0; s4 < 4; ++s4) {
                const int k = 4 * o + s4;
                pend[k] = *reinterpret_cast<const f32x4 *>(stg + (8 * s4 + oc_rd) * 128 + ((ch_rd ^ oc_rd) << 4));
                pend_off[k] = rok ? (int)(soff[s4] + roff) : kOOB;
            }
        }
    };
    frags(0, 0, 0);
    for (int st = 0; st < nsteps; st += 2) {
        step(S1, S0, st);
        if (st + 1 < nsteps) step(S0, S1, st + 1);
    }
#pragma unroll
    for (int k = 0; k < NPART; ++k) store_part(k);
}

// Shapes the row-streaming kernel covers; anything else runs the halo-tiled
// kernel (which itself falls back to the gather kernel).
inline bool bf16_rows_eligible(const ConvArgs &a) {
    using namespace rows_bf16;
    if (a.R != 3 || a.S != 3 || a.sh != 1 || a.sw != 1) return false;
    if (a.C != CH || a.W % 2 != 0 || a.pw > CO || a.OW % 4 != 0 || a.OW > 64) return false;
    if (a.OW + 1 - a.pw + CO > PC - 1) return false;   // last stored column a fragment reads
    if ((reinterpret_cast<uintptr_t>(a.X) & 3) != 0 || (reinterpret_cast<uintptr_t>(a.Wt) & 15) != 0 ||
        (reinterpret_cast<uintptr_t>(a.Y) & 15) != 0)
        return false;
    return true;
}

hipError_t launch_conv_bf16_rows(const ConvArgs &a, hipStream_t s) {
    if (!bf16_rows_eligible(a)) return launch_conv_bf16_halo(a, s);
    // bands sized so that the workgroups (one per CU: the LDS holds one)
    // cover the 256 CUs about once, rounded up to whole steps: a band's
    // time is its step count, so a last step with one row does the work of
    // two (32x64x56x56: 7 bands of 8 rows, 224 workgroups, against 8 bands
    // of 7: 18.9 -> 18.5 us between events)
    const int octiles = (a.OC + rows_bf16::BM - 1) / rows_bf16::BM;
    const int per_img = octiles * a.Nb;
    int nb = (256 + per_img - 1) / per_img;
    ConvArgs args = a;
    args.tile_px = (a.OH + nb - 1) / nb;   // output rows per band, whole steps
    args.tile_px = (args.tile_px + rows_bf16::RO - 1) / rows_bf16::RO * rows_bf16::RO;
    const int nbands = (a.OH + args.tile_px - 1) / args.tile_px;
    args.xcd_remap = 1;
    void *kargs[] = {&args};
    return hipLaunchKernel(reinterpret_cast<const void *>(&conv2d_bf16_rows_kernel),
                           dim3((unsigned)(per_img * nbands)), dim3(rows_bf16::NT), kargs, 0, s);
}

#define XTC_CONV_BF16_INSTANCE(BM, BN, BK, WM, WN, MI, PAD)                                   \
    ConvInstance {                                                                            \
        make_sched(BM, BN, BK, WM, WN, MI, MI, (MI == 32 ? 16 : 32), 2, PAD, 0),               \
            &launch_conv_bf16<BM, BN, BK, WM, WN, MI, PAD>,                                   \
            &occupancy_of<&conv2d_bf16_kernel<BM, BN, BK, WM, WN, MI, PAD, true>,             \
                          (BM / WM) * (BN / WN) * 64, (int)sizeof(int2)>                      \
    }

const ConvInstance kConvBf16Instances[] = {
    ConvInstance{make_sched(64, 256, 16, 64, 64, 32, 32, 16, 2, -1, 0, 2),  // halo, 3x3 stride 1
                 &launch_conv_bf16_halo,
                 &occupancy_of<&conv2d_bf16_halo_kernel, halo_bf16::NT, 0>},
    ConvInstance{make_sched(64, 64, 16, 32, 32, 32, 32, 16, 2, -1, 0, 3),  // row streaming, 3x3 s1, C 64
                 &launch_conv_bf16_rows,
                 &occupancy_of<&conv2d_bf16_rows_kernel, rows_bf16::NT, 0>},
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
