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
#include <type_traits>

#include "lds_dma.h"
#include "mfma_f32.h"
#include "tile_map.h"
#include "unroll.h"
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
                if (oc < M) ybase[oc * OHW] = (p.relu && acc[i][j][r] < 0.f) ? 0.f : acc[i][j][r];
            }
    }
}

template <int BM, int BN, int BK, int WM, int WN, int MI, int PAD>
hipError_t launch_conv_f32(const ConvArgs &a, hipStream_t s);

// ---------------------------------------------------------------------------
// Direct-to-LDS variant.  Both operands reach LDS through buffer loads with
// the `lds` modifier, into a ring of STAGES buffers:
//  - weights (the GEMM A operand, row-major [OC][C*R*S]): 16-byte copies of
//    128-byte tile rows, chunk c of row m stored at slot c ^ ((m ^ m>>3) & 7);
//  - the im2col gather (the B operand): one 4-byte copy per lane per k row,
//    64 consecutive output pixels per instruction.  Each lane's buffer
//    offset is base(pixel) + off(k) from the k-offset table, or an offset
//    past the end of X when the tap falls in the zero padding (or the pixel
//    or k is past the end), which the hardware returns as zero: the padding
//    predicate costs no branch and no register staging.  Inside each group
//    of 64 columns, rows whose (k >> 2) is odd store column c at c ^ 32, so
//    the two halves of a wave (k rows 4 apart in the MFMA operand layout)
//    read different bank halves.
// The main loop is the same ping-pong as the bf16 direct-to-LDS GEMM: the
// fragments of k-step s+1 are read while the MFMAs of step s run, and the
// barrier that publishes stage kt+1 is taken inside the last step of stage
// kt.  Needs C*R*S to be a multiple of 4 and a 16-byte aligned weight
// pointer (else the register-staged kernel above runs).
template <int BM, int BN, int BK, int WM, int WN, int STAGES>
struct ConvDmaCfg {
    static constexpr int MI = 32;
    static constexpr int NWM = BM / WM, NWN = BN / WN;
    static constexpr int NWAVES = NWM * NWN;
    static constexpr int NT = NWAVES * 64;
    static constexpr int TM = WM / MI, TN = WN / MI;
    typedef F32Mfma<MI> MF;
    static constexpr int KCH = 4 * MF::KG;          // k per fragment set (8)
    static constexpr int NS = BK / KCH;             // fragment sets per stage
    static constexpr int RA = BK * 4, CA = BK / 4;  // weight tile row bytes / chunks
    static constexpr int A_BYTES = BM * RA;
    static constexpr int A_BLOCKS = A_BYTES / 1024;
    static constexpr int A_PER_WAVE = A_BLOCKS / NWAVES;
    static constexpr int NCG = BN / 64;             // 64-column groups of the B tile
    static constexpr int B_BYTES = BK * BN * 4;
    static constexpr int B_INSTR = BK * NCG;
    static constexpr int B_PER_WAVE = B_INSTR / NWAVES;
    static constexpr int ROWS_PER_WAVE = BK / NWAVES;
    static constexpr int LOADS = A_PER_WAVE + B_PER_WAVE;
    static constexpr int STAGE_BYTES = A_BYTES + B_BYTES;
    static_assert(CA == 8, "block_k must be 32 (128-byte weight rows)");
    static_assert(A_PER_WAVE * NWAVES == A_BLOCKS && A_PER_WAVE >= 1, "weight tile split");
    static_assert(B_PER_WAVE * NWAVES == B_INSTR, "gather split");
    static_assert(ROWS_PER_WAVE % 8 == 0, "each wave gathers whole groups of 8 k rows");
    static_assert(NS % 2 == 0, "an even number of fragment sets per stage");
    static_assert((STAGES - 1) * LOADS < 64, "vmcnt range");
};

template <int BM, int BN, int BK, int WM, int WN, int STAGES>
__global__ void __launch_bounds__((BM / WM) * (BN / WN) * 64)
conv2d_f32_dma_kernel(ConvArgs p) {
    typedef ConvDmaCfg<BM, BN, BK, WM, WN, STAGES> G;
    typedef typename G::MF MF;
    constexpr int MI = G::MI;
    __shared__ __attribute__((aligned(1024))) unsigned char smem[STAGES * G::STAGE_BYTES];
    extern __shared__ int2 ktab[];  // [K]: {ic*H*W + kh*W + kw, kh | kw << 16}

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave / G::NWN, wn = wave % G::NWN;
    const int lrow = lane % MI, lgrp = lane / MI;

    const int C = p.C, H = p.H, Wd = p.W, R = p.R, S = p.S;
    const int OC = p.OC, OW = p.OW, OHW = p.OH * p.OW;
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

    const i32x4 rw = make_rsrc(p.Wt, OC * K * 4);
    const i32x4 rx = make_rsrc(p.X, p.Nb * C * HW * 4);
    const int wave_u = __builtin_amdgcn_readfirstlane(wave);
    const unsigned smem_base = lds_address(smem);

    // Weight copies: this wave's blocks of 8 rows x 8 chunks.
    int a_row[G::A_PER_WAVE], a_col[G::A_PER_WAVE];
#pragma unroll
    for (int q = 0; q < G::A_PER_WAVE; ++q) {
        const int row = (wave * G::A_PER_WAVE + q) * 8 + lane / 8;
        a_row[q] = row;
        a_col[q] = 4 * ((lane & 7) ^ ((row ^ (row >> 3)) & 7));
    }

    // Gather: this wave owns k rows [wave*ROWS_PER_WAVE, ...) of every
    // stage, all NCG column groups.  Its lane covers pixel column
    // cg*64 + (lane ^ 32x) with x = (k row >> 2) & 1.
    int g_xb[G::NCG][2], g_ih[G::NCG][2], g_iw[G::NCG][2];
#pragma unroll
    for (int cg = 0; cg < G::NCG; ++cg)
#pragma unroll
        for (int x = 0; x < 2; ++x) {
            const int q = n0 + cg * 64 + (lane ^ (32 * x));
            if (q < N) {
                const int img = q / OHW, pix = q - img * OHW;
                const int oh = pix / OW, ow = pix - oh * OW;
                g_ih[cg][x] = oh * p.sh - p.ph;
                g_iw[cg][x] = ow * p.sw - p.pw;
                g_xb[cg][x] = img * C * HW + g_ih[cg][x] * Wd + g_iw[cg][x];
            } else {
                g_ih[cg][x] = -(1 << 28);  // fails the row-range test: reads zero
                g_iw[cg][x] = 0;
                g_xb[cg][x] = 0;
            }
        }

    __syncthreads();  // k-offset table ready

    // Copies of one stage are split in two halves: prepare() computes every
    // buffer offset (k-offset table reads and predicates, no LDS writes), so
    // it can run early, overlapped with the MFMAs of the current stage;
    // fire() issues the copies once the target slot is free.
    int offA[G::A_PER_WAVE], offB[G::ROWS_PER_WAVE][G::NCG];
    auto prepare = [&](int kt) {
        const int k0 = kt * BK;
#pragma unroll
        for (int q = 0; q < G::A_PER_WAVE; ++q) {
            const int gm = m0 + a_row[q], gk = k0 + a_col[q];
            offA[q] = (gm < M && gk < K) ? (gm * K + gk) * 4 : kOOB;
        }
        int2 t[G::ROWS_PER_WAVE];
#pragma unroll
        for (int r = 0; r < G::ROWS_PER_WAVE; ++r) {
            const int k = k0 + wave_u * G::ROWS_PER_WAVE + r;
            t[r] = ktab[k < K ? k : K - 1];
        }
#pragma unroll
        for (int r = 0; r < G::ROWS_PER_WAVE; ++r) {
            const int k = k0 + wave_u * G::ROWS_PER_WAVE + r;
            const int kh = t[r].y & 0xffff, kw = t[r].y >> 16;
            const int x = (r >> 2) & 1;  // == (k row >> 2) & 1 since ROWS_PER_WAVE % 8 == 0
#pragma unroll
            for (int cg = 0; cg < G::NCG; ++cg) {
                const int ih = g_ih[cg][x] + kh, iw = g_iw[cg][x] + kw;
                const bool ok = k < K && (unsigned)ih < (unsigned)H && (unsigned)iw < (unsigned)Wd;
                offB[r][cg] = ok ? (g_xb[cg][x] + t[r].x) * 4 : kOOB;
            }
        }
    };
    auto fire = [&](int st) {
        const unsigned base = smem_base + st * G::STAGE_BYTES;
#pragma unroll
        for (int q = 0; q < G::A_PER_WAVE; ++q)
            dma16(rw, base + (wave_u * G::A_PER_WAVE + q) * 1024, offA[q]);
#pragma unroll
        for (int r = 0; r < G::ROWS_PER_WAVE; ++r)
#pragma unroll
            for (int cg = 0; cg < G::NCG; ++cg)
                dma4(rx, base + G::A_BYTES + ((wave_u * G::ROWS_PER_WAVE + r) * BN + cg * 64) * 4,
                     offB[r][cg]);
    };

    // Fragment addressing (byte offsets inside a stage).
    int a_off[G::TM], a_swz[G::TM];
#pragma unroll
    for (int i = 0; i < G::TM; ++i) {
        const int row = wm * WM + i * MI + lrow;
        a_off[i] = row * G::RA;
        a_swz[i] = (row ^ (row >> 3)) & 7;
    }
    // B: row kk + 4*lgrp + s has (row >> 2) & 1 == lgrp & 1 for kk % 8 == 0.
    int b_off[G::TN];
#pragma unroll
    for (int j = 0; j < G::TN; ++j)
        b_off[j] = (4 * lgrp * BN + ((wn * WN + j * MI + lrow) ^ (32 * (lgrp & 1)))) * 4;

    typename MF::acc_t acc[G::TM][G::TN];
#pragma unroll
    for (int i = 0; i < G::TM; ++i)
#pragma unroll
        for (int j = 0; j < G::TN; ++j)
#pragma unroll
            for (int r = 0; r < MF::NACC; ++r) acc[i][j][r] = 0.f;

    f32x4 af[2][G::TM];
    float bfr[2][G::TN][4];

    auto load_frags = [&](int st, int step, int buf) {
        const unsigned char *As = smem + st * G::STAGE_BYTES;
        const unsigned char *Bs = As + G::A_BYTES;
        const int kk = step * G::KCH;
#pragma unroll
        for (int i = 0; i < G::TM; ++i) {
            const int slot = ((kk >> 2) + lgrp) ^ a_swz[i];
            af[buf][i] = *reinterpret_cast<const f32x4 *>(As + a_off[i] + slot * 16);
        }
#pragma unroll
        for (int j = 0; j < G::TN; ++j)
#pragma unroll
            for (int s = 0; s < 4; ++s)
                bfr[buf][j][s] = *reinterpret_cast<const float *>(Bs + (kk + s) * BN * 4 + b_off[j]);
    };

    auto mfmas = [&](int buf) {
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int i = 0; i < G::TM; ++i)
#pragma unroll
                for (int j = 0; j < G::TN; ++j)
                    acc[i][j] = MF::mma(af[buf][i][s], bfr[buf][j][s], acc[i][j]);
    };

    // Branch-free main loop (zero-fill copies past the end of K keep the
    // number of copies in flight constant; see the GEMM kernels).
    const int KT = (K + BK - 1) / BK;
#pragma unroll
    for (int s = 0; s < STAGES; ++s) {
        prepare(s);
        fire(s);
    }
    wait_vmcnt<(STAGES - 1) * G::LOADS>();
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    load_frags(0, 0, 0);
    for (int kt = 0; kt < KT; ++kt) {
        const int st = kt % STAGES;
        prepare(kt + STAGES);
#pragma unroll
        for (int s = 0; s + 1 < G::NS; ++s) {
            load_frags(st, s + 1, (s + 1) & 1);
            mfmas(s & 1);
        }
        wait_vmcnt_and_lds<(STAGES - 2) * G::LOADS>();
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        fire(st);
        load_frags((kt + 1) % STAGES, 0, 0);
        mfmas((G::NS - 1) & 1);
    }
    wait_vmcnt<0>();  // no copy may still be writing LDS when the workgroup ends

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

template <int BM, int BN, int BK, int WM, int WN, int STAGES>
hipError_t launch_conv_f32_dma(const ConvArgs &a, hipStream_t s) {
    typedef ConvDmaCfg<BM, BN, BK, WM, WN, STAGES> G;
    const int M = a.OC, N = a.Nb * a.OH * a.OW, K = a.C * a.R * a.S;
    const unsigned tiles = (unsigned)(((M + BM - 1) / BM) * ((N + BN - 1) / BN));
    const size_t dyn = (size_t)K * sizeof(int2);
    if (K % 4 != 0 || (reinterpret_cast<uintptr_t>(a.Wt) & 15) != 0)
        return launch_conv_f32<BM, BN, BK, WM, WN, 32, 4>(a, s);  // register-staged fallback
    ConvArgs args = a;
    void *kargs[] = {&args};
    return hipLaunchKernel(reinterpret_cast<const void *>(&conv2d_f32_dma_kernel<BM, BN, BK, WM, WN, STAGES>),
                           dim3(tiles), dim3(G::NT), kargs, dyn, s);
}

// ---------------------------------------------------------------------------
// Tap-major direct-to-LDS variant (channel counts that are a multiple of 32).
// The reduction runs over k = (kh*S + kw)*C + ic instead of (ic*R + kh)*S +
// kw: the sum is the same up to rounding order.  One LDS stage then holds 32
// consecutive input channels of a single tap (kh, kw), so
//  - the padding predicate and the pixel part of the input offset are the
//    same for every channel of the stage: each lane computes them once per
//    stage, and the channel goes into the copy's scalar offset (soffset), so
//    a gather copy needs no vector arithmetic at all;
//  - the weights of the stage, W[oc][ic0 .. ic0+31][kh][kw], are a strided
//    gather too: each lane owns one (oc, channel) slot of the weight tile for
//    the whole K loop (a fixed vector offset) and the stage moves the scalar
//    offset to (ic0*R*S + tap).
// LDS layouts and fragment reads are those of the variant above (128-byte
// weight rows with 16-byte chunks swizzled by (m ^ m>>3) & 7; 64-column
// pixel groups with columns XOR 32 on rows whose (k >> 2) is odd).
template <int BM, int BN, int WM, int WN, int STAGES>
struct ConvTapCfg {
    static constexpr int BK = 32, MI = 32;
    static constexpr int NWM = BM / WM, NWN = BN / WN;
    static constexpr int NWAVES = NWM * NWN;
    static constexpr int NT = NWAVES * 64;
    static constexpr int TM = WM / MI, TN = WN / MI;
    typedef F32Mfma<MI> MF;
    static constexpr int KCH = 4 * MF::KG;
    static constexpr int NS = BK / KCH;
    static constexpr int RA = BK * 4;                // weight tile row bytes
    static constexpr int A_BYTES = BM * RA;
    static constexpr int A_INSTR = BM * BK / 64;     // dword copies (two weight rows each)
    static constexpr int A_PER_WAVE = A_INSTR / NWAVES;
    static constexpr int NCG = BN / 64;
    static constexpr int B_BYTES = BK * BN * 4;
    static constexpr int ROWS_PER_WAVE = BK / NWAVES;
    static constexpr int B_PER_WAVE = ROWS_PER_WAVE * NCG;
    static constexpr int LOADS = A_PER_WAVE + B_PER_WAVE;
    static constexpr int STAGE_BYTES = A_BYTES + B_BYTES;
    static_assert(A_PER_WAVE * NWAVES == A_INSTR && A_PER_WAVE >= 1, "weight tile split");
    static_assert(ROWS_PER_WAVE * NWAVES == BK && ROWS_PER_WAVE >= 1, "gather split");
    static_assert(NS % 2 == 0, "an even number of fragment sets per stage");
    static_assert((STAGES - 1) * LOADS < 64, "vmcnt range");
    static_assert(STAGES * STAGE_BYTES <= 160 * 1024, "LDS budget");
};

template <int BM, int BN, int WM, int WN, int STAGES>
__global__ void __launch_bounds__((BM / WM) * (BN / WN) * 64)
conv2d_f32_tap_kernel(ConvArgs p) {
    typedef ConvTapCfg<BM, BN, WM, WN, STAGES> G;
    typedef typename G::MF MF;
    constexpr int MI = G::MI, BK = G::BK;
    __shared__ __attribute__((aligned(1024))) unsigned char smem[STAGES * G::STAGE_BYTES];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave / G::NWN, wn = wave % G::NWN;
    const int lrow = lane % MI, lgrp = lane / MI;

    const int C = p.C, H = p.H, Wd = p.W, R = p.R, S = p.S;
    const int OC = p.OC, OW = p.OW, OHW = p.OH * p.OW;
    const int M = OC, N = p.Nb * OHW;
    const int HW = H * Wd, RS = R * S;
    const int CB = C / BK;                 // channel chunks per tap
    const int KT = RS * CB;                // LDS stages

    const int tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
    int tm, tn;
    tile_coords(blockIdx.x, gridDim.x, tiles_m, tiles_n, p.raster, p.xcd_remap, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;

    const i32x4 rw = make_rsrc(p.Wt, OC * C * RS * 4);
    const i32x4 rx = make_rsrc(p.X, p.Nb * C * HW * 4);
    const int wave_u = __builtin_amdgcn_readfirstlane(wave);
    const unsigned smem_base = lds_address(smem);

    // Weight copies: copy q of this wave fills tile rows 2*(wave*A_PER_WAVE+q)
    // and +1; lane i lands at row position i % 32, i.e. chunk slot (i%32)/4
    // holding channel chunk slot ^ swizzle(row).
    int voffA[G::A_PER_WAVE];
#pragma unroll
    for (int q = 0; q < G::A_PER_WAVE; ++q) {
        const int row = 2 * (wave * G::A_PER_WAVE + q) + lane / 32;
        const int pos = lane % 32;
        const int kl = 4 * ((pos >> 2) ^ ((row ^ (row >> 3)) & 7)) + (pos & 3);
        const int oc = m0 + row;
        voffA[q] = oc < M ? (oc * C * RS + kl * RS) * 4 : kOOB;
    }

    // Gather columns (as in the variant above).
    int g_xb[G::NCG][2], g_ih[G::NCG][2], g_iw[G::NCG][2];
#pragma unroll
    for (int cg = 0; cg < G::NCG; ++cg)
#pragma unroll
        for (int x = 0; x < 2; ++x) {
            const int q = n0 + cg * 64 + (lane ^ (32 * x));
            if (q < N) {
                const int img = q / OHW, pix = q - img * OHW;
                const int oh = pix / OW, ow = pix - oh * OW;
                g_ih[cg][x] = oh * p.sh - p.ph;
                g_iw[cg][x] = ow * p.sw - p.pw;
                g_xb[cg][x] = img * C * HW + g_ih[cg][x] * Wd + g_iw[cg][x];
            } else {
                g_ih[cg][x] = -(1 << 28);  // fails the row-range test: reads zero
                g_iw[cg][x] = 0;
                g_xb[cg][x] = 0;
            }
        }

    // Stage walk: (tap, channel chunk) of the next stage to prepare.  prepare()
    // is called once per stage, in stage order.
    // prepare(live): a stage past the end of K (live == false) copies only
    // zeros: every vector offset out of range and the scalar offsets 0, so
    // no address of it depends on the (then meaningless) walk state.
    int nx_c0 = 0, nx_kh = 0, nx_kw = 0;
    int voffA_st[G::A_PER_WAVE];
    int voffB[G::NCG][2];
    int so_a = 0, so_b = 0;
    bool st_live = true;
    auto prepare = [&](bool live) {
        const int kh = nx_kh, kw = nx_kw, c0 = nx_c0;
        st_live = live;
#pragma unroll
        for (int cg = 0; cg < G::NCG; ++cg)
#pragma unroll
            for (int x = 0; x < 2; ++x) {
                const int ih = g_ih[cg][x] + kh, iw = g_iw[cg][x] + kw;
                const bool ok = live && (unsigned)ih < (unsigned)H && (unsigned)iw < (unsigned)Wd;
                voffB[cg][x] = ok ? (g_xb[cg][x] + kh * Wd + kw) * 4 : kOOB;
            }
#pragma unroll
        for (int q = 0; q < G::A_PER_WAVE; ++q) voffA_st[q] = live ? voffA[q] : kOOB;
        so_a = live ? (c0 * RS + kh * S + kw) * 4 : 0;
        so_b = live ? (c0 + wave_u * G::ROWS_PER_WAVE) * HW * 4 : 0;
        // advance to the next stage: channels, then kw, then kh
        nx_c0 = c0 + BK;
        if (nx_c0 == C) {
            nx_c0 = 0;
            nx_kw = kw + 1;
            if (nx_kw == S) {
                nx_kw = 0;
                nx_kh = kh + 1;
            }
        }
    };
    auto fire = [&](int st) {
        const unsigned base = smem_base + st * G::STAGE_BYTES;
#pragma unroll
        for (int q = 0; q < G::A_PER_WAVE; ++q)
            dma4_so(rw, base + (wave_u * G::A_PER_WAVE + q) * 256, voffA_st[q], so_a);
#pragma unroll
        for (int r = 0; r < G::ROWS_PER_WAVE; ++r) {
            // column swizzle of this k row (a constant when each wave owns a
            // multiple of 8 rows, else a wave-uniform select)
            const int x = ((wave_u * G::ROWS_PER_WAVE + r) >> 2) & 1;
#pragma unroll
            for (int cg = 0; cg < G::NCG; ++cg)
                dma4_so(rx, base + G::A_BYTES + ((wave_u * G::ROWS_PER_WAVE + r) * BN + cg * 64) * 4,
                        x ? voffB[cg][1] : voffB[cg][0], st_live ? so_b + r * HW * 4 : 0);
        }
    };

    int a_off[G::TM], a_swz[G::TM];
#pragma unroll
    for (int i = 0; i < G::TM; ++i) {
        const int row = wm * WM + i * MI + lrow;
        a_off[i] = row * G::RA;
        a_swz[i] = (row ^ (row >> 3)) & 7;
    }
    int b_off[G::TN];
#pragma unroll
    for (int j = 0; j < G::TN; ++j)
        b_off[j] = (4 * lgrp * BN + ((wn * WN + j * MI + lrow) ^ (32 * (lgrp & 1)))) * 4;

    typename MF::acc_t acc[G::TM][G::TN];
#pragma unroll
    for (int i = 0; i < G::TM; ++i)
#pragma unroll
        for (int j = 0; j < G::TN; ++j)
#pragma unroll
            for (int r = 0; r < MF::NACC; ++r) acc[i][j][r] = 0.f;

    f32x4 af[2][G::TM];
    float bfr[2][G::TN][4];

    auto load_frags = [&](int st, int step, int buf) {
        const unsigned char *As = smem + st * G::STAGE_BYTES;
        const unsigned char *Bs = As + G::A_BYTES;
        const int kk = step * G::KCH;
#pragma unroll
        for (int i = 0; i < G::TM; ++i) {
            const int slot = ((kk >> 2) + lgrp) ^ a_swz[i];
            af[buf][i] = *reinterpret_cast<const f32x4 *>(As + a_off[i] + slot * 16);
        }
#pragma unroll
        for (int j = 0; j < G::TN; ++j)
#pragma unroll
            for (int s = 0; s < 4; ++s)
                bfr[buf][j][s] = *reinterpret_cast<const float *>(Bs + (kk + s) * BN * 4 + b_off[j]);
    };

    auto mfmas = [&](int buf) {
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int i = 0; i < G::TM; ++i)
#pragma unroll
                for (int j = 0; j < G::TN; ++j)
                    acc[i][j] = MF::mma(af[buf][i][s], bfr[buf][j][s], acc[i][j]);
    };

    // Branch-free main loop (see the GEMM kernels); stages past the end are
    // zero-fill copies.
#pragma unroll
    for (int s = 0; s < STAGES; ++s) {
        prepare(s < KT);
        fire(s);
    }
    wait_vmcnt<(STAGES - 1) * G::LOADS>();
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    load_frags(0, 0, 0);
    for (int kt = 0; kt < KT; ++kt) {
        const int st = kt % STAGES;
        prepare(kt + STAGES < KT);
#pragma unroll
        for (int s = 0; s + 1 < G::NS; ++s) {
            load_frags(st, s + 1, (s + 1) & 1);
            mfmas(s & 1);
        }
        wait_vmcnt_and_lds<(STAGES - 2) * G::LOADS>();
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        fire(st);
        load_frags((kt + 1) % STAGES, 0, 0);
        mfmas((G::NS - 1) & 1);
    }
    wait_vmcnt<0>();  // no copy may still be writing LDS when the workgroup ends

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

// Tap-major kernel when the channel count is a multiple of 32, else the
// k-table kernel with the same tiles (which itself falls back to the
// register-staged one when C*R*S is not a multiple of 4).
template <int BM, int BN, int WM, int WN, int STAGES, int FALLBACK_STAGES>
hipError_t launch_conv_f32_tap(const ConvArgs &a, hipStream_t s) {
    typedef ConvTapCfg<BM, BN, WM, WN, STAGES> G;
    if (a.C % G::BK != 0) return launch_conv_f32_dma<BM, BN, 32, WM, WN, FALLBACK_STAGES>(a, s);
    const int M = a.OC, N = a.Nb * a.OH * a.OW;
    const unsigned tiles = (unsigned)(((M + BM - 1) / BM) * ((N + BN - 1) / BN));
    ConvArgs args = a;
    void *kargs[] = {&args};
    return hipLaunchKernel(reinterpret_cast<const void *>(&conv2d_f32_tap_kernel<BM, BN, WM, WN, STAGES>),
                           dim3(tiles), dim3(G::NT), kargs, 0, s);
}

// ---------------------------------------------------------------------------
// Halo-tiled kernel (k_order = 2) for stride-1 3x3 convolutions of rows about
// 56 pixels wide.  The tap-major kernel gathers every input value once per
// tap (nine gather copies per input value for 3x3); here a stage holds an
// 8-channel input patch that all nine taps read from LDS:
//  - a workgroup computes 64 output channels x 256 consecutive output pixels
//    of one image (flat oh*OW + ow order, four 64x64 waves).  Those pixels
//    span at most 6 output rows when OW >= 51, so their inputs fit in a patch
//    of PR = 8 input rows per channel;
//  - the patch stores input row ih of channel c at LDS row (c, ih - ih0),
//    64 columns wide, input column iw at column iw + 4 (left and right
//    padding and rows outside the image read as zero).  One dword copy of 64
//    lanes fills one patch row: lane l fetches column l - 4, a fixed vector
//    offset, and (image, channel, row) go into the scalar offset;
//  - the stage's weights W[oc][c0 .. c0+7][kh][kw] are a dword gather into
//    [tap][oc][8 channels] (one 16-byte read per MFMA A fragment, as in the
//    tap-major kernel);
//  - the reduction runs over channel chunks, and inside a chunk over the nine
//    taps: a tap is one MFMA k-step of 8 channels.  An output pixel's B value
//    for (channel, tap) is patch[(c, r + kh, ow - pw + kw + 4)], so every
//    B fragment read is one ds_read_b32 at a per-lane base plus a constant.
// Patch planes are 8*64 + 8 floats apart, which puts the two lane groups of
// a fragment read (channels c and c + 4) 32 banks apart.
namespace halo {
constexpr int BM = 64, BN = 256, WM = 64, WN = 64, NWAVES = 4, NT = 256;
constexpr int MI = 32, TM = WM / MI, TN = WN / MI;
constexpr int CC = 8;                         // channels per stage
constexpr int NTAP = 9;                       // 3x3 taps, one MFMA k-step each
constexpr int PR = 8;                         // patch rows per channel
constexpr int PLANE = PR * 64 + 8;            // floats per channel plane
constexpr int A_FLOATS = NTAP * BM * CC;      // [tap][oc][c]
constexpr int A_BYTES = A_FLOATS * 4;
constexpr int B_BYTES = CC * PLANE * 4;
constexpr int STAGE_BYTES = A_BYTES + B_BYTES;
constexpr int A_COPIES = A_FLOATS / 64;       // 72
constexpr int A_PER_WAVE = A_COPIES / NWAVES; // 18
constexpr int B_COPIES = CC * PR;             // 64
constexpr int B_PER_WAVE = B_COPIES / NWAVES; // 16: two channels x eight rows
constexpr int LOADS = A_PER_WAVE + B_PER_WAVE;
constexpr int CO = 4;                         // LDS column of input column 0
constexpr unsigned kOffNone = 0x80000000u;    // scalar offset that puts any lane out of range
static_assert(A_PER_WAVE * NWAVES == A_COPIES && B_PER_WAVE * NWAVES == B_COPIES, "copy split");
static_assert((PLANE * 4) % 64 == 32, "lane groups 32 banks apart");
}  // namespace halo

template <int STAGES>
__global__ void __launch_bounds__(halo::NT)
conv2d_f32_halo_kernel(ConvArgs p) {
    using namespace halo;
    typedef F32Mfma<MI> MF;
    static_assert((STAGES - 1) * LOADS < 64, "vmcnt range");
    static_assert(STAGES * STAGE_BYTES <= 80 * 1024, "two workgroups per CU");
    __shared__ __attribute__((aligned(1024))) unsigned char smem[STAGES * STAGE_BYTES];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int lrow = lane % MI, lgrp = lane / MI;
    const int wave_u = __builtin_amdgcn_readfirstlane(wave);

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
    const int KT = C / CC;                    // stages (even: C % 16 == 0)

    const i32x4 rw = make_rsrc(p.Wt, OC * C * NTAP * 4);
    const i32x4 rx = make_rsrc(p.X, p.Nb * C * H * Wd * 4);
    const unsigned smem_base = lds_address(smem);

    // Copy offsets.  Every copy's address is a fixed per-lane vector offset
    // plus a scalar offset that moves by a constant per stage, so a stage's
    // copies need one scalar add each and no conditions:
    //  - weights: lane l fills slot (oc = 8*ocb + l/8, channel l%8) of a copy;
    //    a row past OC reads zero through the buffer range check;
    //  - patch: lane l fills column l (input column l - CO, zero outside the
    //    row); a patch row outside the image uses the out-of-range vector
    //    offset (its scalar offset is clamped to a real row so the sum stays
    //    below 2^32).
    // Stages past the end (the ring's tail) load whatever their offsets hit
    // -- in range or zero, never outside the buffers -- and are never used.
    const int voffA = ((lane >> 3) * C * NTAP + (lane & 7) * NTAP) * 4;
    const int iwl = lane - CO;
    const int voffB = (iwl >= 0 && iwl < Wd) ? iwl * 4 : kOOB;
    int voffR[PR];
#pragma unroll
    for (int r = 0; r < PR; ++r) voffR[r] = (ih0 + r >= 0 && ih0 + r < H) ? voffB : kOOB;
    const int HW4 = H * Wd * 4;
    const int a_stage = CC * NTAP * 4;       // scalar-offset step per stage
    const int b_stage = CC * HW4;
    const int a_base0 = (m0 * C * NTAP) * 4;
    const int b_base0 = (img * C + wave_u * (CC / NWAVES)) * HW4;

    int so_a = a_base0, so_b = b_base0;      // offsets of the next stage to fire
    // Copy q (0 .. LOADS-1) of the stage in slot st: weights first, then the
    // patch rows.
    auto copy = [&](int st, int q) __attribute__((always_inline)) {
        const unsigned base = smem_base + st * STAGE_BYTES;
        if (q < A_PER_WAVE) {
            const int cq = wave_u * A_PER_WAVE + q;          // copy index: tap-major
            const int tap = cq / 8, ocb = cq % 8;
            dma4_so(rw, base + (tap * BM * CC + ocb * 64) * 4, voffA,
                    so_a + (ocb * 8 * C * NTAP + tap) * 4);
        } else {
            const int cl = (q - A_PER_WAVE) / PR, row = (q - A_PER_WAVE) % PR;  // channel, patch row
            const int ihc = min(max(ih0 + row, 0), H - 1);
            dma4_so(rx, base + A_BYTES + ((wave_u * (CC / NWAVES) + cl) * PLANE + row * 64) * 4,
                    voffR[row], so_b + cl * HW4 + ihc * Wd * 4);
        }
    };
    auto advance = [&]() {
        so_a += a_stage;
        so_b += b_stage;
    };
    auto fire = [&](int st) {
#pragma unroll
        for (int q = 0; q < LOADS; ++q) copy(st, q);
        advance();
    };

    // Per-lane fragment bases.  A: row (i*32 + lrow), channels 4*lgrp .. +3.
    // B: this lane's pixel of column block j (clamped to patch position 0 when
    // past the image; such columns are not stored).
    const int a_base = ((lrow * CC) + 4 * lgrp) * 4;
    int b_base[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int pix = p0 + wave * WN + j * MI + lrow;
        int off = 0;
        if (pix < OHW) {
            const int oh = pix / OW, ow = pix - oh * OW;
            off = (oh - oh0) * 64 + ow - p.pw + CO;
        }
        b_base[j] = (4 * lgrp * PLANE + off) * 4;
    }

    typename MF::acc_t acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < MF::NACC; ++r) acc[i][j][r] = 0.f;

    f32x4 af[2][TM];
    float bfr[2][TN][4];
    auto load_frags = [&](int st, int tap, int buf) {
        const unsigned char *As = smem + st * STAGE_BYTES;
        const unsigned char *Bs = As + A_BYTES;
        const int kh = tap / 3, kw = tap - 3 * kh;
#pragma unroll
        for (int i = 0; i < TM; ++i)
            af[buf][i] = *reinterpret_cast<const f32x4 *>(As + a_base + (tap * BM * CC + i * MI * CC) * 4);
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            // an opaque base per column block keeps the compiler from pairing
            // the two blocks' reads into ds_read2_b32, whose second address
            // would collide with the other lane group's banks
            int bb = b_base[j];
            asm volatile("" : "+v"(bb));
#pragma unroll
            for (int s = 0; s < 4; ++s)
                bfr[buf][j][s] = *reinterpret_cast<const float *>(Bs + bb + (s * PLANE + kh * 64 + kw) * 4);
        }
    };
    auto mfmas = [&](int buf) {
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = MF::mma(af[buf][i][s], bfr[buf][j][s], acc[i][j]);
    };
    // The last tap's MFMAs with the copies of the stage STAGES ahead spread
    // between them: issued all at once right after the barrier, the copies of
    // every wave queue at the texture unit and stall the issuing waves.
    auto mfmas_with_copies = [&](int buf, int st) __attribute__((always_inline)) {
        constexpr int NM = 4 * TM * TN;
#pragma unroll
        for (int m = 0; m < NM; ++m) {
            const int s = m / (TM * TN), i = (m / TN) % TM, j = m % TN;
            acc[i][j] = MF::mma(af[buf][i][s], bfr[buf][j][s], acc[i][j]);
            const int q0 = m * LOADS / NM, q1 = (m + 1) * LOADS / NM;
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int q = q0; q < q1; ++q) copy(st, q);
            __builtin_amdgcn_sched_barrier(0);
        }
        advance();
    };

    // One stage: nine taps, fragments of tap t + 1 read while tap t runs;
    // the barrier that frees this stage's slot sits before the last tap.  P
    // is the fragment buffer of the stage's first tap: with nine taps it
    // alternates between stages, so the loop body runs two stages.
    auto stage = [&](int kt, auto par) {
        constexpr int P = decltype(par)::value;
        const int st = kt % STAGES;
#pragma unroll
        for (int t = 0; t + 1 < NTAP; ++t) {
            load_frags(st, t + 1, (P + t + 1) & 1);
            mfmas((P + t) & 1);
        }
        wait_vmcnt_and_lds<(STAGES - 2) * LOADS>();
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        load_frags((kt + 1) % STAGES, 0, (P + NTAP) & 1);
        mfmas_with_copies((P + NTAP - 1) & 1, st);
    };

#pragma unroll
    for (int s = 0; s < STAGES; ++s) fire(s);
    wait_vmcnt<(STAGES - 1) * LOADS>();
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    load_frags(0, 0, 0);
    for (int kt = 0; kt < KT; kt += 2) {
        stage(kt, std::integral_constant<int, 0>());
        stage(kt + 1, std::integral_constant<int, NTAP & 1>());
    }
    wait_vmcnt<0>();  // no copy may still be writing LDS when the workgroup ends

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
                if (oc < OC) Y[oc * OHW + pix] = (p.relu && acc[i][j][r] < 0.f) ? 0.f : acc[i][j][r];
            }
    }
}

// Balanced halo-tiled kernel (k_order = 2, 16x16x4 instruction tile).  The
// same input-patch staging as the kernel above, with tiles sized so that the
// workgroups of a launch split evenly over the CUs: a workgroup computes 64
// output channels x PT consecutive output pixels of one image, where the
// launcher picks PT <= 208 as OHW divided into the fewest tiles per image
// (3136 pixels -> 16 tiles of 196; 32 images -> 512 workgroups, two per CU).
// Each of the four waves owns 16 output channels and all thirteen 16-pixel
// column blocks, so every wave does the same work whatever PT is; columns
// past the tile are computed and not stored.  For the 16x16x4 instruction a
// lane holds the weight of (channel 4s + lane/16, output channel lane%16)
// and the input value of (channel 4s + lane/16, pixel lane%16), so the four
// lane groups read four channel planes.  gfx950 serves a ds_read_b32 in two
// phases of 32 lanes (two lane groups each), and within a phase two lanes
// conflict when their dword addresses are equal modulo 32 (measured):
//  - patch planes are PR*64 + 16 floats apart, so the two groups of a phase
//    sit 16 banks apart and a 16-pixel block within one image row reads 32
//    distinct banks.  A block that wraps to the next image row still
//    collides with the other group; avoiding that needs patch rows of 72
//    floats, which does not fit two workgroups per CU;
//  - the weights of a stage are [tap][oc][8 channels]; a phase reads two
//    channels of 16 output channels, and with plain rows output channels
//    oc, oc + 4, oc + 8, oc + 12 share banks, so output channel oc holds its
//    channel c at slot c ^ (2 * ((oc >> 2) & 3)).
namespace halo16 {
constexpr int BM = 64;
constexpr int NB = 13;                        // 16-pixel column blocks per wave
constexpr int CC = 8, NTAP = 9, CO = 4;
constexpr int NSTEP = NTAP * CC / 4;          // instruction k-steps per stage (18)
constexpr int A_FLOATS = NTAP * BM * CC;      // [tap][oc][c]
constexpr int A_BYTES = A_FLOATS * 4;
constexpr int A_COPIES = A_FLOATS / 64;       // 72
static_assert(NSTEP % 2 == 0, "fragment buffers keep their parity from stage to stage");

// NH pixel halves per workgroup: 4*NH waves, wave w owns output channels
// 16*(w % 4) .. +15 and the 16*NB pixels of half w / 4.  Two halves (8
// waves, up to 416 pixels) share one patch of 10 rows and one copy of the
// stage's weights, where two one-half workgroups load 8 rows and the
// weights each.
template <int NH>
struct Cfg {
    static constexpr int NWAVES = 4 * NH, NT = 64 * NWAVES;
    static constexpr int BN = 16 * NB * NH;       // largest pixel tile
    static constexpr int PR = NH == 1 ? 8 : 10;   // patch rows
    static constexpr int PLANE = PR * 64 + 16;
    static constexpr int B_BYTES = CC * PLANE * 4;
    static constexpr int STAGE_BYTES = A_BYTES + B_BYTES;
    static constexpr int A_PER_WAVE = A_COPIES / NWAVES;   // 18 or 9
    static constexpr int B_COPIES = CC * PR;               // one per (channel, patch row)
    static constexpr int B_PER_WAVE = B_COPIES / NWAVES;   // 16 (two channels) or 10 (one)
    static constexpr int LOADS = A_PER_WAVE + B_PER_WAVE;
    static_assert(A_PER_WAVE * NWAVES == A_COPIES && B_PER_WAVE * NWAVES == B_COPIES, "copy split");
    static_assert(B_PER_WAVE % PR == 0, "a wave copies whole channels");
    static_assert((PLANE % 32) == 16, "the two lane groups of a phase 16 of 32 banks apart");
};
}  // namespace halo16

template <int STAGES, int NH>
__global__ void __launch_bounds__(halo16::Cfg<NH>::NT)
conv2d_f32_halo16_kernel(ConvArgs p) {
    using namespace halo16;
    typedef Cfg<NH> G;
    constexpr int NWAVES = G::NWAVES, PR = G::PR, PLANE = G::PLANE, STAGE_BYTES = G::STAGE_BYTES;
    constexpr int A_PER_WAVE = G::A_PER_WAVE, LOADS = G::LOADS;
    typedef F32Mfma<16> MF;
    static_assert((STAGES - 1) * LOADS < 64, "vmcnt range");
    static_assert(STAGES * STAGE_BYTES <= 80 * 1024, "two workgroups per CU");
    __shared__ __attribute__((aligned(1024))) unsigned char smem[STAGES * STAGE_BYTES];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wq = wave & 3, half = wave >> 2;   // output-channel group, pixel half
    const int lcol = lane & 15, lgrp = lane >> 4;
    const int wave_u = __builtin_amdgcn_readfirstlane(wave);

    const int C = p.C, H = p.H, Wd = p.W;
    const int OC = p.OC, OW = p.OW, OHW = p.OH * p.OW;
    const int PT = p.tile_px;
    const int chunks = (OHW + PT - 1) / PT;   // per image
    const int tiles_m = (OC + BM - 1) / BM, tiles_n = p.Nb * chunks;
    int tm, tn;
    tile_coords(blockIdx.x, gridDim.x, tiles_m, tiles_n, p.raster, p.xcd_remap, tm, tn);
    const int m0 = tm * BM;
    const int img = tn / chunks, p0 = (tn - img * chunks) * PT;
    const int pend = min(p0 + PT, OHW);
    const int oh0 = p0 / OW;                  // first output row of the tile
    const int ih0 = oh0 - p.ph;               // input row of patch row 0
    const int KT = C / CC;                    // stages

    const i32x4 rw = make_rsrc(p.Wt, OC * C * NTAP * 4);
    const i32x4 rx = make_rsrc(p.X, p.Nb * C * H * Wd * 4);
    const unsigned smem_base = lds_address(smem);

    // Copies as in the 64x256 halo kernel: a fixed per-lane vector offset
    // plus a scalar offset that moves by a constant per stage; padding and
    // rows outside the image are out-of-range offsets that read zero, and
    // stages past the end read in range or zero and are never used.
    // A copy fills 8 output channels x 8 channel slots of one tap: lane l
    // writes slot l % 8 of output channel 8 * block + l / 8, which holds
    // channel (l % 8) ^ (2 * ((oc >> 2) & 3)) (the weight swizzle); the XOR
    // is 2 * (l >> 5) for even blocks and 2 * (2 + (l >> 5)) for odd ones.
    const int voffA0 = ((lane >> 3) * C * NTAP + ((lane & 7) ^ ((lane >> 5) << 1)) * NTAP) * 4;
    const int voffA1 = ((lane >> 3) * C * NTAP + ((lane & 7) ^ ((2 | (lane >> 5)) << 1)) * NTAP) * 4;
    const int iwl = lane - CO;
    const int voffB = (iwl >= 0 && iwl < Wd) ? iwl * 4 : kOOB;
    int voffR[PR];
#pragma unroll
    for (int r = 0; r < PR; ++r) voffR[r] = (ih0 + r >= 0 && ih0 + r < H) ? voffB : kOOB;
    const int HW4 = H * Wd * 4;
    const int a_stage = CC * NTAP * 4;
    const int b_stage = CC * HW4;
    int so_a = (m0 * C * NTAP) * 4;
    int so_b = (img * C + wave_u * (CC / NWAVES)) * HW4;
    auto copy = [&](int st, int q) __attribute__((always_inline)) {
        const unsigned base = smem_base + st * STAGE_BYTES;
        if (q < A_PER_WAVE) {
            const int cq = wave_u * A_PER_WAVE + q;          // copy index: tap-major
            const int tap = cq / 8, ocb = cq % 8;
            dma4_so(rw, base + (tap * BM * CC + ocb * 64) * 4, (ocb & 1) ? voffA1 : voffA0,
                    so_a + (ocb * 8 * C * NTAP + tap) * 4);
        } else {
            const int cl = (q - A_PER_WAVE) / PR, row = (q - A_PER_WAVE) % PR;
            const int ihc = min(max(ih0 + row, 0), H - 1);
            dma4_so(rx, base + A_BYTES + ((wave_u * (CC / NWAVES) + cl) * PLANE + row * 64) * 4,
                    voffR[row], so_b + cl * HW4 + ihc * Wd * 4);
        }
    };
    auto advance = [&]() {
        so_a += a_stage;
        so_b += b_stage;
    };

    // The waves of the second half run NB - 1 column blocks when the tile's
    // second half fits in them (PT <= 16 * (2 * NB - 1) pixels, 392 for
    // 56 x 56 images): on each SIMD, which holds one wave of each half, that
    // is 25 instead of 26 blocks of MFMAs.  Each instance runs the same copy
    // and barrier sequence.
    auto body = [&](auto nbc) __attribute__((always_inline)) {
        constexpr int NBW = decltype(nbc)::value;
        // Fragment bases.  A: output channel 16*wq + lcol, channel lgrp + 4s
        // (one base per s: the swizzle may flip bit 2 of the slot).
        // B: pixel pw0 + 16j + lcol of the patch (clamped to position 0 past the
        // tile; such columns are not stored), channel plane lgrp (+4s).
        const int a_sw = ((lcol >> 2) & 3) << 1;
        const int a_base[2] = {((wq * 16 + lcol) * CC + (lgrp ^ a_sw)) * 4,
                               ((wq * 16 + lcol) * CC + ((lgrp + 4) ^ a_sw)) * 4};
        const int pw0 = p0 + 16 * NB * half;     // first pixel of this wave's half
        int b_base[NBW];
#pragma unroll
        for (int j = 0; j < NBW; ++j) {
            const int pix = pw0 + 16 * j + lcol;
            int off = 0;
            if (pix < pend) {
                const int oh = pix / OW, ow = pix - oh * OW;
                off = (oh - oh0) * 64 + ow - p.pw + CO;
            }
            b_base[j] = (lgrp * PLANE + off) * 4;
        }

        typename MF::acc_t acc[NBW];
#pragma unroll
        for (int j = 0; j < NBW; ++j)
#pragma unroll
            for (int r = 0; r < MF::NACC; ++r) acc[j][r] = 0.f;

        float af[2], bfr[2][NBW];
        // k-step t of a stage: tap t / 2, channels 4 * (t % 2) .. + 3
        auto load_frags = [&](int st, int t, int buf) __attribute__((always_inline)) {
            const unsigned char *As = smem + st * STAGE_BYTES;
            const unsigned char *Bs = As + A_BYTES;
            const int tap = t >> 1, s = t & 1;
            const int kh = tap / 3, kw = tap - 3 * kh;
            af[buf] = *reinterpret_cast<const float *>(As + a_base[s] + tap * BM * CC * 4);
#pragma unroll
            for (int j = 0; j < NBW; ++j)
                bfr[buf][j] = *reinterpret_cast<const float *>(Bs + b_base[j] + (4 * s * PLANE + kh * 64 + kw) * 4);
        };
        auto mfmas = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
            for (int j = 0; j < NBW; ++j) acc[j] = MF::mma(af[buf], bfr[buf][j], acc[j]);
        };
        // K-step t of the stage in slot st, one MFMA at a time, each followed by
        // one fragment read of k-step t + 1 and its share of the copies of the
        // next stage into slot nx.  A stage's copies are spread over its first
        // CSTEPS k-steps: issued together, the copies of all waves would queue at
        // the texture unit and stall the issuing waves.  The fences keep the
        // order (and keep the compiler from hoisting the reads).
        static_assert(STAGES == 2, "the next stage is copied into the other slot of a two-slot ring");
        constexpr int CSTEPS = 12;
        auto step = [&](int st, auto tc, int nx) __attribute__((always_inline)) {
            constexpr int t = decltype(tc)::value;   // a constant: the copy split is fixed per k-step
            const int cur = t & 1, nxt = (t + 1) & 1;
            const unsigned char *As = smem + st * STAGE_BYTES;
            const unsigned char *Bs = As + A_BYTES;
            const int tap = (t + 1) >> 1, s = (t + 1) & 1;
            const int kh = tap / 3, kw = tap - 3 * kh;
            constexpr int q0 = t < CSTEPS ? t * LOADS / CSTEPS : LOADS;
            constexpr int q1 = t < CSTEPS ? (t + 1) * LOADS / CSTEPS : LOADS;
#pragma unroll
            for (int m = 0; m < NBW; ++m) {
                acc[m] = MF::mma(af[cur], bfr[cur][m], acc[m]);
                if (m == 0)
                    af[nxt] = *reinterpret_cast<const float *>(As + a_base[s] + tap * BM * CC * 4);
                bfr[nxt][m] =
                    *reinterpret_cast<const float *>(Bs + b_base[m] + (4 * s * PLANE + kh * 64 + kw) * 4);
#pragma unroll
                for (int q = q0 + m * (q1 - q0) / NBW; q < q0 + (m + 1) * (q1 - q0) / NBW; ++q) copy(nx, q);
                __builtin_amdgcn_sched_barrier(0);
            }
        };

        // Stage 0 into slot 0; then every iteration computes stage kt from slot
        // kt % 2 while copying stage kt + 1 into the other slot (stages past the
        // end read in range or zero and are never used).
#pragma unroll
        for (int q = 0; q < LOADS; ++q) copy(0, q);
        advance();
        wait_vmcnt<0>();
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        load_frags(0, 0, 0);
        for (int kt = 0; kt < KT; ++kt) {
            const int st = kt & 1, nx = st ^ 1;
            each_index([&](auto tc) __attribute__((always_inline)) { step(st, tc, nx); },
                       std::make_integer_sequence<int, NSTEP - 1>());
            advance();
            // this wave's copies of stage kt + 1 have landed, then everyone's; every
            // wave has also issued its last read of slot st (k-step NSTEP - 1's
            // fragments, now in registers)
            wait_vmcnt_and_lds<0>();
            __builtin_amdgcn_s_barrier();
            asm volatile("" ::: "memory");
            load_frags(nx, 0, 0);
            mfmas((NSTEP - 1) & 1);
        }
        wait_vmcnt<0>();  // no copy may still be writing LDS when the workgroup ends

        float *__restrict__ Y = p.Y + (size_t)img * OC * OHW;
#pragma unroll
        for (int j = 0; j < NBW; ++j) {
            const int pix = pw0 + 16 * j + lcol;
            if (pix >= pend) continue;
#pragma unroll
            for (int r = 0; r < MF::NACC; ++r) {
                const int oc = m0 + 16 * wq + MF::row(lane, r);
                if (oc < OC) Y[oc * OHW + pix] = (p.relu && acc[j][r] < 0.f) ? 0.f : acc[j][r];
            }
        }
    };
    if (NH == 2 && half == 1 && PT <= 16 * (2 * NB - 1))
        body(std::integral_constant<int, NB - 1>());
    else
        body(std::integral_constant<int, NB>());
}

// ---------------------------------------------------------------------------
// Few output channels (block_m = 16, lds_stages = 0): layers such as the
// paper's 7x7 stride-2 conv of 3 input channels into 16 (K = 147), where
// 64-row tiles leave three quarters of the matrix cores idle and the
// reduction is too short to amortise LDS staging.  A workgroup covers 16
// output channels x 16*NB*4 pixels with four waves; each wave owns NB blocks
// of 16 pixels and runs 16x16x4 instructions.  Both operands go straight
// from memory into the instruction's registers: a lane holds, per k-step
// s, the weight W[oc0 + lane % 16][4s + lane / 16] and the input value of
// its pixel at that k, gathered through the LDS k-offset table.  Elements
// outside the image, past K or past the output channels are buffer loads
// at an out-of-range offset, which read zero, so there are no predicated
// loads and K needs no particular multiple.  The k-steps are processed in
// chunks of KC, the loads of chunk c + 1 in flight while chunk c's MFMAs
// run (two register sets: for K up to 8 * KC every load is issued before
// the first MFMA waits); MFMAs of k-steps past K are skipped, and even and
// odd k-steps accumulate into two chains, added at the end, which halves
// the dependent MFMA chain.
namespace smallm {
constexpr int WAVES = 4, NT = 64 * WAVES;
}

template <int NB, int KC>
__global__ void __launch_bounds__(smallm::NT)
conv2d_f32_smallm_kernel(ConvArgs p) {
    typedef F32Mfma<16> MF;
    constexpr int KCH = 4 * KC;                  // k per chunk
    constexpr int BN = 16 * NB * smallm::WAVES;
    extern __shared__ int2 ktab[];  // [KP]: {ic*H*W + kh*W + kw, kh | kw << 16}

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int l16 = lane & 15, g = lane >> 4;

    const int C = p.C, H = p.H, Wd = p.W, R = p.R, S = p.S;
    const int OC = p.OC, OHW = p.OH * p.OW;
    const int N = p.Nb * OHW, K = C * R * S;
    const int HW = H * Wd, RS = R * S;
    const int NC = (K + KCH - 1) / KCH;          // chunks
    const int KP = NC * KCH;                     // table entries

    const int tiles_m = (OC + 15) / 16, tiles_n = (N + BN - 1) / BN;
    int tm, tn;
    tile_coords(blockIdx.x, gridDim.x, tiles_m, tiles_n, p.raster, p.xcd_remap, tm, tn);
    const int m0 = tm * 16, n0 = tn * BN + wave * 16 * NB;

    for (int k = tid; k < KP; k += smallm::NT) {
        int2 e = make_int2(0, 0);
        if (k < K) {
            const int ic = k / RS, rem = k - ic * RS;
            const int kh = rem / S, kw = rem - kh * S;
            e = make_int2(ic * HW + kh * Wd + kw, kh | (kw << 16));
        }
        ktab[k] = e;
    }

    const __amdgpu_buffer_rsrc_t rw =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(p.Wt), 0, OC * K * 4, 0x00020000);
    const __amdgpu_buffer_rsrc_t rx =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(p.X), 0, p.Nb * C * HW * 4, 0x00020000);
    const int oc = m0 + l16;
    const int woff = oc < OC ? oc * K : 0;

    // this lane's pixel of each of its blocks
    int xb[NB], ih0[NB], iw0[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        const int q = n0 + 16 * j + l16;
        xb[j] = 0;
        ih0[j] = -(1 << 30);    // a pixel past the end: every tap out of range
        iw0[j] = 0;
        if (q < N) {
            const int img = q / OHW, pix = q - img * OHW;
            const int oh = pix / p.OW, ow = pix - oh * p.OW;
            ih0[j] = oh * p.sh - p.ph;
            iw0[j] = ow * p.sw - p.pw;
            xb[j] = img * C * HW + ih0[j] * Wd + iw0[j];
        }
    }

    float a[2][KC], b[2][NB][KC];
    auto load = [&](int buf, int k0) __attribute__((always_inline)) {
#pragma unroll
        for (int s = 0; s < KC; ++s) {
            const int k = k0 + 4 * s + g;
            const bool kok = k < K;
            a[buf][s] = __builtin_bit_cast(
                float, __builtin_amdgcn_raw_buffer_load_b32(rw, (kok && oc < OC) ? (woff + k) * 4 : kOOB, 0, 0));
            const int2 t = ktab[k];
            const int kh = t.y & 0xffff, kw = t.y >> 16;
#pragma unroll
            for (int j = 0; j < NB; ++j) {
                const bool in = kok && (unsigned)(ih0[j] + kh) < (unsigned)H &&
                                (unsigned)(iw0[j] + kw) < (unsigned)Wd;
                b[buf][j][s] = __builtin_bit_cast(
                    float, __builtin_amdgcn_raw_buffer_load_b32(rx, in ? (xb[j] + t.x) * 4 : kOOB, 0, 0));
            }
        }
    };

    typename MF::acc_t acc[2][NB];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int j = 0; j < NB; ++j)
#pragma unroll
            for (int r = 0; r < MF::NACC; ++r) acc[h][j][r] = 0.f;
    auto mfmas = [&](int buf, int k0) __attribute__((always_inline)) {
#pragma unroll
        for (int s = 0; s < KC; ++s)
            if (k0 + 4 * s < K)   // uniform
#pragma unroll
                for (int j = 0; j < NB; ++j)
                    acc[s & 1][j] = MF::mma(a[buf][s], b[buf][j][s], acc[s & 1][j]);
    };

    __syncthreads();  // k-offset table ready
    // Ring of two register sets over the NC chunks (a uniform trip count);
    // k-steps past K in the last chunk load zeros and add nothing.
    load(0, 0);
    for (int c = 0; c < NC; c += 2) {
        if (c + 1 < NC) load(1, (c + 1) * KCH);
        mfmas(0, c * KCH);
        if (c + 1 >= NC) break;
        if (c + 2 < NC) load(0, (c + 2) * KCH);
        mfmas(1, (c + 1) * KCH);
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[0][j] += acc[1][j];

    float *__restrict__ Y = p.Y;
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        const int q = n0 + 16 * j + l16;
        if (q >= N) continue;
        const int img = q / OHW, pix = q - img * OHW;
#pragma unroll
        for (int r = 0; r < MF::NACC; ++r) {
            const int o = m0 + MF::row(lane, r);
            if (o < OC) Y[((size_t)img * OC + o) * OHW + pix] = (p.relu && acc[0][j][r] < 0.f) ? 0.f : acc[0][j][r];
        }
    }
}

// Patch-staged variant of the few-output-channel kernel, for layers whose
// input patch fits in LDS (at most 48 KiB with the weights, 256 padded
// columns and 256 k) (the paper's 7x7 stride-2 layer: 3 channels x 9
// rows x 229 columns, 24.7 KB).  A workgroup covers 64 consecutive output
// pixels of one image (one or two output rows).  It stages, with coalesced
// loads in one round trip to memory:
//  - its input patch: every channel, the input rows those output rows reach
//    (rows outside the image as zeros) and every padded column, so that
//    patch[c][r][col] holds X[c][ih_lo + r][col - pad_w] or zero;
//  - the weights of its 16 output channels, [oc][K] (zero past OC);
//  - the k-offset table relative to the patch, k -> c*PR*WP + kh*WP + kw.
// An output pixel's B value at k is then patch[pix_base + ktab[k]] with
// pix_base = (oh*stride_h - pad_h - ih_lo)*WP + ow*stride_w: no bounds
// checks in the K loop, which reads only LDS.  Eight waves stage (16-byte
// chunks of the input rows where the width allows); waves 0-3 and 4-7 then
// reduce the two halves of K for the same pixel blocks, and the second
// half's partial sums reach the first through the patch area.
namespace smallm {
constexpr int PATCH_MAX_BYTES = 48 * 1024;
constexpr int PWAVES = 8, PNT = 64 * PWAVES;   // patch-staged kernel: two reduction halves of 4 waves

// Geometry of the patch-staged kernel for a launch: rows PR and width WP
// of the patch and the patch column PADL of input column 0, or PR = 0 when
// the patch does not fit.  With 16-byte row loads (vec) PADL and WP are
// multiples of 4, so that every 4-column chunk of the patch is one aligned
// chunk of an input row or lies wholly outside it.
struct PatchGeom {
    int PR, WP, PADL, bytes;
};
__host__ __device__ inline PatchGeom patch_geom(const ConvArgs &a, int bn, bool vec) {
    const int span = (bn - 1 + a.OW - 1) / a.OW + 1;   // output rows a tile can touch
    PatchGeom g;
    g.PR = (span - 1) * a.sh + a.R;
    g.PADL = vec ? (a.pw + 3) / 4 * 4 : a.pw;
    g.WP = (a.OW - 1) * a.sw + a.S - a.pw + g.PADL;
    if (vec) g.WP = (g.WP + 3) / 4 * 4;
    const long long K = (long long)a.C * a.R * a.S;
    const long long kp = (K + 31) / 32 * 32;
    // the patch area also holds the second half's partial sums at the end
    // (4 waves x 64 lanes x 2 chains x bn / 64 blocks x 4 floats)
    const long long area = max((long long)a.C * g.PR * g.WP, 32LL * bn);
    const long long bytes = 4LL * (area + 16 * (kp + 2)) + 4 * kp;
    // the staging loops cover up to 256 padded columns and 256 k
    g.bytes = (bytes <= PATCH_MAX_BYTES && g.WP <= 256 && kp <= 256) ? (int)bytes : 0;
    if (g.bytes == 0) g.PR = 0;
    return g;
}
}  // namespace smallm

template <int NB, int NCH, bool VEC>
__global__ void __launch_bounds__(smallm::PNT)
conv2d_f32_smallm_patch_kernel(ConvArgs p) {
    typedef F32Mfma<16> MF;
    constexpr int BN = 16 * NB * smallm::WAVES;
    extern __shared__ __attribute__((aligned(16))) float sm[];   // 16-byte patch rows and partial sums

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int l16 = lane & 15, g = lane >> 4;
    // waves 0-3 and 4-7 take the two halves of the reduction over the same
    // pixel blocks (two waves per SIMD); all eight stage
    const int half = wave >> 2, wq = wave & 3;

    const int C = p.C, H = p.H, Wd = p.W, R = p.R, S = p.S;
    const int OC = p.OC, OW = p.OW, OHW = p.OH * OW;
    const int K = C * R * S, KP = (K + 31) / 32 * 32;
    const int RS = R * S;
    const smallm::PatchGeom geo = smallm::patch_geom(p, BN, VEC);
    const int PR = geo.PR, WP = geo.WP, PADL = geo.PADL, PLANE = PR * WP;

    const int chunks = (OHW + BN - 1) / BN;   // tiles per image
    const int tiles_m = (OC + 15) / 16, tiles_n = p.Nb * chunks;
    int tm, tn;
    tile_coords(blockIdx.x, gridDim.x, tiles_m, tiles_n, p.raster, p.xcd_remap, tm, tn);
    const int m0 = tm * 16;
    const int img = tn / chunks, p0 = (tn - img * chunks) * BN;
    const int ih_lo = (p0 / OW) * p.sh - p.ph;

    // weight rows are KP + 2 floats apart: a phase of a ds_read_b32 (16
    // output channels x 2 lane groups) then covers 32 distinct banks (KP is
    // a multiple of 32, so rows KP apart would all share one bank)
    const int WS = KP + 2;
    const int AREA = max(C * PLANE, 32 * BN);           // the patch, later the partial sums
    float *patch = sm;                                  // [C][PR][WP]
    float *wl = sm + AREA;                              // [16][WS]
    int *ktab = reinterpret_cast<int *>(wl + 16 * WS);  // [KP]

    const __amdgpu_buffer_rsrc_t rw =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(p.Wt), 0, OC * K * 4, 0x00020000);
    const __amdgpu_buffer_rsrc_t rx =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(p.X), 0, p.Nb * C * H * Wd * 4, 0x00020000);

    // Stage the patch, the weights and the table (zeros where out of range).
    // Wave w takes patch rows w, w + 8, ...; lane l takes columns l + 64q
    // (WP <= 256), or with 16-byte loads columns 4l .. 4l + 3; every load of
    // a batch is issued before its LDS stores.
    const int xb = img * C * H * Wd;
    const int nrows = C * PR;
    constexpr int RPW = 4;   // rows per wave per batch
    // Weights first (wave w takes output channels w and w + 8), so that
    // their loads and the patch's are in flight together: one round trip to
    // memory for the whole staging.
    float wv[2][4];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int o = wave + smallm::PWAVES * i;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int k = lane + 64 * q;
            const bool in = m0 + o < OC && k < K;
            wv[i][q] = __builtin_bit_cast(
                float, __builtin_amdgcn_raw_buffer_load_b32(rw, in ? ((m0 + o) * K + k) * 4 : kOOB, 0, 0));
        }
    }
    // this thread's table entry (KP <= 256 threads), computed while the
    // loads are in flight; k >= K: any in-range entry (its weight is zero)
    int tk = 0;
    if (tid < K) {
        const int ic = tid / RS, rem = tid - ic * RS;
        const int kh = rem / S, kw = rem - kh * S;
        tk = ic * PLANE + kh * WP + kw;
    }
    // (channel, patch row) of row `wave`, stepped by 8 rows without division
    int c_next = wave / PR, r_next = wave - c_next * PR;
    for (int rb = wave; rb < nrows; rb += smallm::PWAVES * RPW) {
        float v[RPW][4];
        int c = c_next, r = r_next;
#pragma unroll
        for (int i = 0; i < RPW; ++i) {
            const int row = rb + smallm::PWAVES * i;
            if (i > 0) {
                r += smallm::PWAVES;
                while (r >= PR) {   // uniform
                    r -= PR;
                    ++c;
                }
            }
            const int ih = ih_lo + r;
            const bool rok = row < nrows && (unsigned)ih < (unsigned)H;
            if constexpr (VEC) {
                // W and PADL are multiples of 4: a chunk is wholly inside the row or outside it
                const int iw = 4 * lane - PADL;
                const bool in = rok && 4 * lane < WP && (unsigned)iw < (unsigned)Wd;
                const f32x4 t = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                              rx, in ? (xb + (c * H + ih) * Wd + iw) * 4 : kOOB, 0, 0));
#pragma unroll
                for (int q = 0; q < 4; ++q) v[i][q] = t[q];
            } else {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int iw = lane + 64 * q - PADL;
                    const bool in = rok && lane + 64 * q < WP && (unsigned)iw < (unsigned)Wd;
                    v[i][q] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                                            rx, in ? (xb + (c * H + ih) * Wd + iw) * 4 : kOOB, 0, 0));
                }
            }
        }
#pragma unroll
        for (int i = 0; i < RPW; ++i) {
            const int row = rb + smallm::PWAVES * i;
            if constexpr (VEC) {
                if (row < nrows && 4 * lane < WP) {
                    f32x4 t;
#pragma unroll
                    for (int q = 0; q < 4; ++q) t[q] = v[i][q];
                    *reinterpret_cast<f32x4 *>(patch + row * WP + 4 * lane) = t;
                }
            } else {
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    if (row < nrows && lane + 64 * q < WP) patch[row * WP + lane + 64 * q] = v[i][q];
            }
        }
        r += smallm::PWAVES;   // the next batch's first row
        while (r >= PR) {
            r -= PR;
            ++c;
        }
        c_next = c;
        r_next = r;
    }
    // the weights' stores, after the patch: their loads were issued first
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q)
            if (lane + 64 * q < KP) wl[(wave + smallm::PWAVES * i) * WS + lane + 64 * q] = wv[i][q];
    if (tid < KP) ktab[tid] = tk;

    // this lane's pixel of each of its blocks (position 0 past the image)
    const int n0 = p0 + wq * 16 * NB;
    int pb[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        const int pix = n0 + 16 * j + l16;
        pb[j] = 0;
        if (pix < OHW) {
            const int oh = pix / OW, ow = pix - oh * OW;
            pb[j] = (oh * p.sh - p.ph - ih_lo) * WP + ow * p.sw + PADL - p.pw;
        }
    }

    typename MF::acc_t acc[2][NB];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int j = 0; j < NB; ++j)
#pragma unroll
            for (int r = 0; r < MF::NACC; ++r) acc[h][j][r] = 0.f;
    __syncthreads();

    // k-step s: lane group g takes k = 4s + g.  Steps run in NCH chunks of
    // 8 (KP = 32 * NCH: padded steps have zero weights); the first half of
    // the waves takes chunks 0 .. NC0 - 1, the second half the rest.  A
    // half's table entries are read first, in one batch, so that no input
    // read waits on a table read: the input values and weights of chunk
    // c + 1 are then read while chunk c's MFMAs run.  Even and odd steps
    // accumulate into two chains.
    constexpr int NC0 = (NCH + 1) / 2;
    const float *wrow = wl + l16 * WS + g;
    auto reduce_chunks = [&](auto C0, auto C1) __attribute__((always_inline)) {
        constexpr int CA = decltype(C0)::value, CB = decltype(C1)::value;
        if constexpr (CB > CA) {
            int tv[CB - CA][8];
#pragma unroll
            for (int c = CA; c < CB; ++c)
#pragma unroll
                for (int i = 0; i < 8; ++i) tv[c - CA][i] = ktab[32 * c + 4 * i + g];
            float av[2][8], bv[2][NB][8];
            auto rd = [&](int buf, int c) __attribute__((always_inline)) {
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    av[buf][i] = wrow[32 * c + 4 * i];
#pragma unroll
                    for (int j = 0; j < NB; ++j) bv[buf][j][i] = patch[pb[j] + tv[c - CA][i]];
                }
            };
            auto mm = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
                for (int i = 0; i < 8; ++i)
#pragma unroll
                    for (int j = 0; j < NB; ++j) acc[i & 1][j] = MF::mma(av[buf][i], bv[buf][j][i], acc[i & 1][j]);
            };
            rd(0, CA);
#pragma unroll
            for (int c = CA; c < CB; ++c) {
                if (c + 1 < CB) rd((c + 1 - CA) & 1, c + 1);
                mm((c - CA) & 1);
                if (c + 1 < CB) {
                    // the next chunk's reads between this chunk's instructions: in
                    // one run they would exceed the 15 reads the LDS counter can
                    // wait past, and each instruction would wait for some of them
#pragma unroll
                    for (int i = 0; i < 8; ++i) {
                        __builtin_amdgcn_sched_group_barrier(0x008, NB, 0);          // MFMA
                        __builtin_amdgcn_sched_group_barrier(0x100, 1 + NB, 0);      // LDS reads
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
        }
    };
    if (half == 0)
        reduce_chunks(std::integral_constant<int, 0>(), std::integral_constant<int, NC0>());
    else
        reduce_chunks(std::integral_constant<int, NC0>(), std::integral_constant<int, NCH>());

    // the second half's partial sums through the patch area (every wave is
    // done reading the patch), added by the first half in a fixed order
    __syncthreads();
    f32x4 *part = reinterpret_cast<f32x4 *>(patch);   // [wq][chain][block][lane]
    if (half == 1) {
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int j = 0; j < NB; ++j) part[((wq * 2 + h) * NB + j) * 64 + lane] = acc[h][j];
    }
    __syncthreads();
    if (half == 1) return;

    float *__restrict__ Y = p.Y + (size_t)img * OC * OHW;
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        const int pix = n0 + 16 * j + l16;
        const f32x4 q0 = part[((wq * 2 + 0) * NB + j) * 64 + lane];
        const f32x4 q1 = part[((wq * 2 + 1) * NB + j) * 64 + lane];
        if (pix >= OHW) continue;
#pragma unroll
        for (int r = 0; r < MF::NACC; ++r) {
            const int o = m0 + MF::row(lane, r);
            const float v = (acc[0][j][r] + acc[1][j][r]) + (q0[r] + q1[r]);
            if (o < OC) Y[(size_t)o * OHW + pix] = (p.relu && v < 0.f) ? 0.f : v;
        }
    }
}

template <int NB, int KC>
hipError_t launch_conv_f32_smallm(const ConvArgs &a, hipStream_t s) {
    constexpr int BN = 16 * NB * smallm::WAVES, KCH = 4 * KC;
    // 16-byte patch loads need 16-byte aligned input rows
    bool vec = a.W % 4 == 0 && (reinterpret_cast<uintptr_t>(a.X) & 15) == 0;
    smallm::PatchGeom geo = smallm::patch_geom(a, BN, vec);
    if (vec && geo.PR == 0) {
        vec = false;
        geo = smallm::patch_geom(a, BN, false);
    }
    if (geo.PR > 0) {
        const int OHW = a.OH * a.OW;
        const unsigned tiles =
            (unsigned)(((a.OC + 15) / 16) * a.Nb * ((OHW + BN - 1) / BN));
        ConvArgs args = a;
        void *kargs[] = {&args};
#define XTC_PATCH_FNS(V)                                                                    \
    {reinterpret_cast<const void *>(&conv2d_f32_smallm_patch_kernel<NB, 1, V>),               \
     reinterpret_cast<const void *>(&conv2d_f32_smallm_patch_kernel<NB, 2, V>),               \
     reinterpret_cast<const void *>(&conv2d_f32_smallm_patch_kernel<NB, 3, V>),               \
     reinterpret_cast<const void *>(&conv2d_f32_smallm_patch_kernel<NB, 4, V>),               \
     reinterpret_cast<const void *>(&conv2d_f32_smallm_patch_kernel<NB, 5, V>),               \
     reinterpret_cast<const void *>(&conv2d_f32_smallm_patch_kernel<NB, 6, V>),               \
     reinterpret_cast<const void *>(&conv2d_f32_smallm_patch_kernel<NB, 7, V>),               \
     reinterpret_cast<const void *>(&conv2d_f32_smallm_patch_kernel<NB, 8, V>)}
        static const void *const fns[2][8] = {XTC_PATCH_FNS(false), XTC_PATCH_FNS(true)};
#undef XTC_PATCH_FNS
        // patch_geom admits K up to 256 (KP / 32 = 1 .. 8 chunks)
        const int nch = (a.C * a.R * a.S + 31) / 32;
        return hipLaunchKernel(fns[vec ? 1 : 0][nch - 1], dim3(tiles), dim3(smallm::PNT), kargs,
                               (size_t)geo.bytes, s);
    }
    const int N = a.Nb * a.OH * a.OW, K = a.C * a.R * a.S;
    const unsigned tiles = (unsigned)(((a.OC + 15) / 16) * ((N + BN - 1) / BN));
    const size_t dyn = (size_t)(((K + KCH - 1) / KCH) * KCH) * sizeof(int2);
    ConvArgs args = a;
    void *kargs[] = {&args};
    return hipLaunchKernel(reinterpret_cast<const void *>(&conv2d_f32_smallm_kernel<NB, KC>),
                           dim3(tiles), dim3(smallm::NT), kargs, dyn, s);
}

// Shapes the halo kernel covers; anything else runs the tap-major kernel
// with the same 64x256 tiles.
inline bool halo_eligible(const ConvArgs &a) {
    using namespace halo;
    if (a.R != 3 || a.S != 3 || a.sh != 1 || a.sw != 1) return false;
    if (a.C % (2 * CC) != 0 || a.pw > CO) return false;
    if (a.OW - a.pw + 5 > 63) return false;              // last patch column used (W + pw <= 60)
    const int span = (BN - 1 + a.OW - 1) / a.OW + 1;      // output rows a tile can touch
    return span + 2 <= PR;
}

template <int STAGES>
hipError_t launch_conv_f32_halo(const ConvArgs &a, hipStream_t s) {
    if (!halo_eligible(a)) return launch_conv_f32_tap<64, 256, 64, 64, 2, 2>(a, s);
    const int OHW = a.OH * a.OW;
    const unsigned tiles = (unsigned)(((a.OC + halo::BM - 1) / halo::BM) * a.Nb *
                                      ((OHW + halo::BN - 1) / halo::BN));
    ConvArgs args = a;
    void *kargs[] = {&args};
    return hipLaunchKernel(reinterpret_cast<const void *>(&conv2d_f32_halo_kernel<STAGES>),
                           dim3(tiles), dim3(halo::NT), kargs, 0, s);
}

// Pixels per tile for the balanced halo kernel with NH halves: the fewest
// tiles per image that keep a tile within 208*NH pixels; 0 when the shape is
// outside the kernel's class (then the 64x256 halo kernel, or the tap-major
// kernel, runs).
template <int NH>
inline int halo16_tile_px(const ConvArgs &a) {
    using namespace halo16;
    typedef Cfg<NH> G;
    if (a.R != 3 || a.S != 3 || a.sh != 1 || a.sw != 1) return 0;
    if (a.C % CC != 0 || a.pw > CO) return 0;
    if (a.OW - a.pw + 5 > 63) return 0;                  // last patch column used (W + pw <= 60)
    const int OHW = a.OH * a.OW;
    const int t = (OHW + G::BN - 1) / G::BN;
    const int pt = (OHW + t - 1) / t;
    const int span = (pt - 1 + a.OW - 1) / a.OW + 1;      // output rows a tile can touch
    return span + 2 <= G::PR ? pt : 0;
}

template <int STAGES, int NH>
hipError_t launch_conv_f32_halo16(const ConvArgs &a, hipStream_t s) {
    const int pt = halo16_tile_px<NH>(a);
    if (pt == 0) return launch_conv_f32_halo<STAGES>(a, s);
    ConvArgs args = a;
    args.tile_px = pt;
    const int OHW = a.OH * a.OW;
    const unsigned tiles = (unsigned)(((a.OC + halo16::BM - 1) / halo16::BM) * a.Nb *
                                      ((OHW + pt - 1) / pt));
    void *kargs[] = {&args};
    return hipLaunchKernel(reinterpret_cast<const void *>(&conv2d_f32_halo16_kernel<STAGES, NH>),
                           dim3(tiles), dim3(halo16::Cfg<NH>::NT), kargs, 0, s);
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
            &launch_conv_f32<BM, BN, BK, WM, WN, MI, PAD>,                                    \
            &occupancy_of<&conv2d_f32_kernel<BM, BN, BK, WM, WN, MI, PAD, true>,              \
                          (BM / WM) * (BN / WN) * 64, (int)sizeof(int2)>                      \
    }

#define XTC_CONV_DMA_INSTANCE(BM, BN, BK, WM, WN, STAGES)                                     \
    ConvInstance {                                                                            \
        make_sched(BM, BN, BK, WM, WN, 32, 32, 2, STAGES, -1, 0),                             \
            &launch_conv_f32_dma<BM, BN, BK, WM, WN, STAGES>,                                 \
            &occupancy_of<&conv2d_f32_dma_kernel<BM, BN, BK, WM, WN, STAGES>,                 \
                          (BM / WM) * (BN / WN) * 64, (int)sizeof(int2)>                      \
    }

// Tap-major direct-to-LDS instances (k_order = 1).
#define XTC_CONV_TAP_INSTANCE(BM, BN, WM, WN, STAGES, FB)                                     \
    ConvInstance {                                                                            \
        make_sched(BM, BN, 32, WM, WN, 32, 32, 2, STAGES, -1, 0, 1),                          \
            &launch_conv_f32_tap<BM, BN, WM, WN, STAGES, FB>,                                 \
            &occupancy_of<&conv2d_f32_tap_kernel<BM, BN, WM, WN, STAGES>,                     \
                          (BM / WM) * (BN / WN) * 64, 0>                                      \
    }

const ConvInstance kConvInstances[] = {
    ConvInstance{make_sched(64, 208, 8, 16, 208, 16, 16, 4, 2, -1, 0, 2),  // balanced halo, 3x3 stride 1
                 &launch_conv_f32_halo16<2, 1>,
                 &occupancy_of<&conv2d_f32_halo16_kernel<2, 1>, halo16::Cfg<1>::NT, 0>},
    ConvInstance{make_sched(64, 416, 8, 16, 208, 16, 16, 4, 2, -1, 0, 2),  // the same, two pixel halves
                 &launch_conv_f32_halo16<2, 2>,
                 &occupancy_of<&conv2d_f32_halo16_kernel<2, 2>, halo16::Cfg<2>::NT, 0>},
    ConvInstance{make_sched(64, 256, 8, 64, 64, 32, 32, 2, 2, -1, 0, 2),   // halo, 3x3 stride 1
                 &launch_conv_f32_halo<2>,
                 &occupancy_of<&conv2d_f32_halo_kernel<2>, halo::NT, 0>},
    XTC_CONV_TAP_INSTANCE(64, 256, 64, 64, 2, 2),    // the halo instance's fallback
    XTC_CONV_TAP_INSTANCE(64, 128, 32, 64, 2, 3),
    XTC_CONV_TAP_INSTANCE(64, 64, 32, 32, 2, 4),
    XTC_CONV_TAP_INSTANCE(128, 128, 64, 64, 2, 3),   // default for OC > 64
    XTC_CONV_DMA_INSTANCE(64, 128, 32, 32, 64, 3),
    XTC_CONV_DMA_INSTANCE(64, 64, 32, 32, 32, 3),
    XTC_CONV_DMA_INSTANCE(128, 128, 32, 64, 64, 3),
    XTC_CONV_INSTANCE(64, 128, 32, 32, 64, 32, 4),
    XTC_CONV_INSTANCE(64, 64, 32, 32, 32, 32, 4),
    XTC_CONV_INSTANCE(128, 128, 32, 64, 64, 32, 4),
    XTC_CONV_INSTANCE(64, 128, 32, 32, 64, 16, 4),
    // few output channels: 16 x 64 tiles, operands straight to registers
    ConvInstance{make_sched(16, 64, 128, 16, 16, 16, 16, 4, 0, 0, 0, 0),
                 &launch_conv_f32_smallm<1, 32>,
                 &occupancy_of<&conv2d_f32_smallm_kernel<1, 32>, smallm::NT, (int)sizeof(int2)>},
};

}  // namespace

const ConvInstance *conv2d_f32_instances(int *count) {
    *count = (int)(sizeof(kConvInstances) / sizeof(kConvInstances[0]));
    return kConvInstances;
}

}  // namespace xtc
