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
#include "lds_dma.h"
#include "mfma_bf16.h"
#include "tile_map.h"
#include "xtc_internal.h"

namespace xtc {
namespace {

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
    static constexpr int W = 8;             // elements per global load
    static constexpr int A_CPR = BK / W;    // 16-byte chunks per tile row
    static constexpr int B_CPR = BN / W;
    static_assert(64 % A_CPR == 0 && 64 % B_CPR == 0, "a tile row's chunks stay in one wave");
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

    // VEC: 16-byte aligned rows, read with plain 16-byte loads.  Otherwise
    // rows may start at any 2-byte boundary: 16-byte loads of the aligned
    // chunks that cover each group of eight, shifted into place.
    int a_first, b_first;
    const __amdgpu_buffer_rsrc_t rsa = aligned_rsrc(A, ((long long)(M - 1) * lda + K) * 2, 2, &a_first);
    const __amdgpu_buffer_rsrc_t rsb = aligned_rsrc(B, ((long long)(K - 1) * ldb + N) * 2, 2, &b_first);
    auto load_tiles = [&](int kt) {
        const int k0 = kt * BK;
#pragma unroll
        for (int i = 0; i < G::A_LOADS; ++i) {
            const int idx = tid + i * G::NT;
            const int r = idx / G::A_CPR, c = (idx % G::A_CPR) * W;
            const int gm = m0 + r, gk = k0 + c;
            const int valid = gm < M ? K - gk : 0;
            if constexpr (VEC) {
                ra[i] = load_pred_u16<W>(A + (valid > 0 ? gm * lda + gk : 0), valid);
            } else {
                // a run is one tile row: its lanes' chunks are consecutive,
                // also past K (those values are read but zeroed)
                const int e = gm < M ? gm * lda + gk : 0;
                ra[i] = load_shifted_u16x8(rsa, a_first + e, valid, idx % G::A_CPR == G::A_CPR - 1);
            }
        }
#pragma unroll
        for (int i = 0; i < G::B_LOADS; ++i) {
            const int idx = tid + i * G::NT;
            const int r = idx / G::B_CPR, c = (idx % G::B_CPR) * W;
            const int gk = k0 + r, gn = n0 + c;
            const int valid = gk < K ? N - gn : 0;
            if constexpr (VEC) {
                rb[i] = load_pred_u16<W>(B + (valid > 0 ? gk * ldb + gn : 0), valid);
            } else {
                const int e = gk < K ? gk * ldb + gn : 0;
                rb[i] = load_shifted_u16x8(rsb, b_first + e, valid, idx % G::B_CPR == G::B_CPR - 1);
            }
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
                if (row < M && col < N) C[row * ldc + col] = (p.relu && acc[i][j][r] < 0.f) ? 0.f : acc[i][j][r];
            }
        }
}

// ---------------------------------------------------------------------------
// Direct-to-LDS variant.  Global tiles are copied straight into LDS with
// buffer_load_dwordx4 ... lds (16 bytes per lane, no register staging), into
// a ring of STAGES LDS buffers, so STAGES-1 K-steps are in flight while the
// matrix cores work on the oldest one.  One such instruction writes 1 KiB of
// LDS contiguously (lane i at byte 16*i of the block), so the layout is
// chosen on the global side: each 16-byte chunk of a tile row is placed at
// slot = chunk ^ swizzle(row) of its LDS row, which keeps the fragment reads
// free of bank conflicts with unpadded rows (swz_a, swz_b below).  Out-of-range chunks (rows >= M
// or >= K, columns >= N or k >= K) are fetched through a buffer offset past
// the end of the buffer, which the hardware returns as zero: this variant
// needs K and N to be multiples of 8 and 16-byte aligned rows, and otherwise
// the register-staged kernel above runs.

// A rows hold CA = BK/8 chunks of 16 bytes; chunk c of row m sits at slot
// c ^ swz_a(m), and an A fragment (16 bytes per lane) is one ds_read_b128.
// gfx950 serves a ds_read_b128 in four phases of 16 lanes: lanes
// {0-3, 12-15, 20-23, 24-27}, {4-11, 16-19, 28-31} and the same sets + 32
// (measured with a per-lane-pair conflict probe).  Lane l of a fragment
// read takes row l % 32, so a phase holds rows r with (r >> 2) in
// {0, 3, 5, 6} or in {1, 2, 4, 7}; the swizzles below give those rows
// distinct 16-byte bank groups (64 banks of 4 bytes), so every phase is
// conflict-free for the 32x32x16 reads, and for the 16x16x32 reads at
// block_k 64.
template <int CA>
__device__ __forceinline__ int swz_a(int row) {
    return CA == 4 ? (row >> 2) & 3 : (row >> 1) & 7;
}

// B rows (one k each) are read four consecutive rows at a time by the
// transpose reads, which gfx950 serves in two phases of 32 lanes (0-31,
// 32-63); XOR values {0, 6, 10, 12} on k % 4 spread the four rows a phase
// reads over distinct bank groups.  With the 16x16x32 instruction one phase
// also reads rows k and k + 8 (lane groups 0 and 1), which XOR 2 on bit 3
// of k separates (with the 32x32x16 instruction that term costs 0.6% on
// 8192^3 and is left out).
template <int MI>
__device__ __forceinline__ int swz_b(int k) {
    return ((k & 1) * 6) ^ ((k & 2) * 5) ^ (MI == 16 ? ((k >> 3) & 1) * 2 : 0);
}


template <int BM, int BN, int BK, int WM, int WN, int MI, int STAGES>
struct Bf16DmaCfg {
    static constexpr int NWM = BM / WM, NWN = BN / WN;
    static constexpr int NWAVES = NWM * NWN;
    static constexpr int NT = NWAVES * 64;
    static constexpr int TM = WM / MI, TN = WN / MI;
    typedef Bf16Mfma<MI> MF;
    static constexpr int KG = MF::KG;
    static constexpr int KCH = 8 * KG;                  // k per MFMA
    static constexpr int NS = BK / KCH;                 // MFMA k-steps per LDS stage
    static constexpr int RA = BK * 2, CA = BK / 8;      // A row bytes / chunks
    static constexpr int RB = BN * 2, CB = BN / 8;      // B row bytes / chunks
    static constexpr int A_BYTES = BM * RA, B_BYTES = BK * RB;
    static constexpr int A_BLOCKS = A_BYTES / 1024, B_BLOCKS = B_BYTES / 1024;
    static constexpr int A_PER_WAVE = A_BLOCKS / NWAVES, B_PER_WAVE = B_BLOCKS / NWAVES;
    static constexpr int LOADS = A_PER_WAVE + B_PER_WAVE;   // copies per wave per stage
    static constexpr int STAGE_BYTES = A_BYTES + B_BYTES;
    static_assert(A_PER_WAVE * NWAVES == A_BLOCKS && B_PER_WAVE * NWAVES == B_BLOCKS,
                  "tiles must split into whole 1 KiB blocks per wave");
    static_assert(CA == 4 || CA == 8, "block_k must be 32 or 64");
    static_assert(CB >= 16 && RB <= 1024, "block_n must be 128..512");
    static_assert(BK % KCH == 0 && NS % 2 == 0, "an even number of MFMA k-steps per stage");
    static_assert(STAGES >= 2 && STAGES * STAGE_BYTES <= 160 * 1024, "LDS budget");
    static_assert((STAGES - 1) * LOADS < 64, "vmcnt range");
};

// Main loop (per workgroup).  Iteration kt computes stage kt from slot
// kt % STAGES; for each k-step s it reads the fragments of step s+1 (two
// register sets alternate) while the MFMAs of step s run.  Barrier B(kt), in
// front of the last k-step's MFMAs, publishes stage kt+1 (each wave first
// waits for its own copies of it).  Copies only enter a slot whose reads
// every wave has completed, by one of two orders:
//   STAGES >= 3 (lagged ring): after B(kt) the copies of stage
//     kt+STAGES-1 go into slot (kt-1) % STAGES.  Every read of that slot
//     fed an MFMA of iteration kt-1, and a wave only reaches B(kt) after
//     those MFMAs have taken their operands (the register wait in front of
//     each MFMA), in the previous trip of the loop.  STAGES-2 stages are in
//     flight while one is computed.
//   STAGES == 2: the first MFMAs of the last k-step take every fragment of
//     slot kt's last read set; each wave then waits for all its LDS reads
//     (lgkmcnt 0) before B(kt), and the copies of stage kt+2 into slot kt
//     follow B(kt).
// Either way the ring's reuse is ordered by waits and the barrier, not by
// the latency of the copies.  Scheduling-group barriers interleave the LDS
// reads of the next k-step with the MFMAs of the current one.
template <int BM, int BN, int BK, int WM, int WN, int MI, int STAGES>
__global__ void __launch_bounds__((BM / WM) * (BN / WN) * 64)
gemm_bf16_dma_kernel(GemmArgs p) {
    typedef Bf16DmaCfg<BM, BN, BK, WM, WN, MI, STAGES> G;
    typedef typename G::MF MF;
    __shared__ __attribute__((aligned(1024))) unsigned char smem[STAGES * G::STAGE_BYTES];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave / G::NWN, wn = wave % G::NWN;
    const int lrow = lane % MI, lgrp = lane / MI;

    const int M = p.M, N = p.N, K = p.K;
    const int tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
    int tm, tn;
    tile_coords(blockIdx.x, gridDim.x, tiles_m, tiles_n, p.raster, p.xcd_remap, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;

    const i32x4 ra = make_rsrc(p.A, ((M - 1) * p.lda + K) * 2);
    const i32x4 rb = make_rsrc(p.B, ((K - 1) * p.ldb + N) * 2);
    const int wave_u = __builtin_amdgcn_readfirstlane(wave);
    const unsigned smem_base = lds_address(smem);

    // Per-lane source coordinates of this wave's copy blocks (fixed over K).
    int a_row[G::A_PER_WAVE], a_col[G::A_PER_WAVE];
#pragma unroll
    for (int q = 0; q < G::A_PER_WAVE; ++q) {
        const int blk = wave * G::A_PER_WAVE + q;
        const int row = blk * (1024 / G::RA) + lane / G::CA;
        a_row[q] = row;
        a_col[q] = 8 * ((lane % G::CA) ^ swz_a<G::CA>(row));
    }
    int b_row[G::B_PER_WAVE], b_col[G::B_PER_WAVE];
#pragma unroll
    for (int q = 0; q < G::B_PER_WAVE; ++q) {
        const int blk = wave * G::B_PER_WAVE + q;
        const int row = blk * (1024 / G::RB) + lane / G::CB;
        b_row[q] = row;
        b_col[q] = 8 * ((lane % G::CB) ^ swz_b<MI>(row));
    }

    // Copies of one stage: prepare() computes the buffer offsets (out of
    // range, i.e. zero fill, for a stage past the end of K), fire() issues
    // them once the target slot is free.  Every stage index issues exactly
    // LOADS copies per wave, so the number of copies in flight is the same in
    // every iteration and one vmcnt value is exact throughout.
    int offA[G::A_PER_WAVE], offB[G::B_PER_WAVE];
    auto prepare = [&](int kt) {
        const int k0 = kt * BK;
#pragma unroll
        for (int q = 0; q < G::A_PER_WAVE; ++q) {
            const int gm = m0 + a_row[q], gk = k0 + a_col[q];
            offA[q] = (gm < M && gk < K) ? (gm * p.lda + gk) * 2 : kOOB;
        }
#pragma unroll
        for (int q = 0; q < G::B_PER_WAVE; ++q) {
            const int gk = k0 + b_row[q], gn = n0 + b_col[q];
            offB[q] = (gk < K && gn < N) ? (gk * p.ldb + gn) * 2 : kOOB;
        }
    };
    auto fire = [&](int st) {
        const unsigned base = smem_base + st * G::STAGE_BYTES;
#pragma unroll
        for (int q = 0; q < G::A_PER_WAVE; ++q)
            dma16(ra, base + (wave_u * G::A_PER_WAVE + q) * 1024, offA[q]);
#pragma unroll
        for (int q = 0; q < G::B_PER_WAVE; ++q)
            dma16(rb, base + G::A_BYTES + (wave_u * G::B_PER_WAVE + q) * 1024, offB[q]);
    };

    // Fragment addressing inside one stage (byte offsets).
    int a_off[G::TM], a_swz[G::TM];
#pragma unroll
    for (int i = 0; i < G::TM; ++i) {
        const int row = wm * WM + i * MI + lrow;
        a_off[i] = row * G::RA;
        a_swz[i] = swz_a<G::CA>(row);
    }
    const int rsub = (lane & 15) >> 2;  // transpose-read row inside the group of four
    // the rows this lane reads are kk + 8*lgrp + rsub (+ 4) with kk a multiple
    // of 16: == rsub (mod 4), with bit 3 equal to bit 0 of lgrp
    const int bsw = swz_b<MI>(8 * (lgrp & 1) + rsub);
    int b_chunk[G::TN];
#pragma unroll
    for (int j = 0; j < G::TN; ++j)
        b_chunk[j] = (((wn * WN + j * MI + (lrow & ~15) + 4 * (lane & 3)) >> 3) ^ bsw) * 16 +
                     8 * (lane & 1);

    typename MF::acc_t acc[G::TM][G::TN];
#pragma unroll
    for (int i = 0; i < G::TM; ++i)
#pragma unroll
        for (int j = 0; j < G::TN; ++j)
#pragma unroll
            for (int r = 0; r < MF::NACC; ++r) acc[i][j][r] = 0.f;

    u16x8 af[2][G::TM], bfr[2][G::TN];

    auto load_frags = [&](int st, int step, int buf) {
        const unsigned char *As = smem + st * G::STAGE_BYTES;
        const unsigned char *Bs = As + G::A_BYTES;
        const int kk = step * G::KCH;
#pragma unroll
        for (int i = 0; i < G::TM; ++i) {
            const int slot = ((kk >> 3) + lgrp) ^ a_swz[i];
            af[buf][i] = *reinterpret_cast<const u16x8 *>(As + a_off[i] + slot * 16);
        }
#pragma unroll
        for (int j = 0; j < G::TN; ++j) {
            const unsigned char *q0 = Bs + (kk + 8 * lgrp + rsub) * G::RB + b_chunk[j];
            const u16x4 lo = ds_read_tr16(reinterpret_cast<const unsigned short *>(q0));
            const u16x4 hi = ds_read_tr16(reinterpret_cast<const unsigned short *>(q0 + 4 * G::RB));
            bfr[buf][j] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        }
    };

    auto mfmas = [&](int buf) {
#pragma unroll
        for (int i = 0; i < G::TM; ++i)
#pragma unroll
            for (int j = 0; j < G::TN; ++j) acc[i][j] = MF::mma(af[buf][i], bfr[buf][j], acc[i][j]);
    };

    // The last k-step of a stage (lagged ring): its MFMAs with the copies
    // of the stage AHEAD ahead spread between them, so that the copies of
    // all waves do not queue at the texture unit at once right after the
    // barrier (which stalls the issuing waves, MFMAs included); the fences
    // keep the compiler from regrouping them.
    auto mfmas_with_copies = [&](int buf, int st) {
        const unsigned base = smem_base + st * G::STAGE_BYTES;
        constexpr int NM = G::TM * G::TN;
#pragma unroll
        for (int m = 0; m < NM; ++m) {
            acc[m / G::TN][m % G::TN] =
                MF::mma(af[buf][m / G::TN], bfr[buf][m % G::TN], acc[m / G::TN][m % G::TN]);
            const int q0 = m * G::LOADS / NM, q1 = (m + 1) * G::LOADS / NM;
            if (q1 > q0) {
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int q = q0; q < q1; ++q) {
                    if (q < G::A_PER_WAVE)
                        dma16(ra, base + (wave_u * G::A_PER_WAVE + q) * 1024, offA[q]);
                    else
                        dma16(rb, base + G::A_BYTES + (wave_u * G::B_PER_WAVE + q - G::A_PER_WAVE) * 1024,
                              offB[q - G::A_PER_WAVE]);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    };

    // The last k-step of a stage in the two-slot ring, in two parts.  mfmas_head: the MFMAs of
    // the first A fragment against every B fragment.  They need the set's
    // last LDS read (the last B fragment), and LDS reads return in order, so
    // once they are issued every read of the slot being retired has
    // returned and the wave's lgkmcnt(0) wait in front of the barrier costs
    // nothing more.  mfmas_tail: the remaining MFMAs, with the copies of
    // the stage STAGES ahead spread between them, so that the copies of all
    // waves do not queue at the texture unit at once right after the
    // barrier (which stalls the issuing waves, MFMAs included); the fences
    // keep the compiler from regrouping them.
    auto mfmas_head = [&](int buf) {
#pragma unroll
        for (int j = 0; j < G::TN; ++j) acc[0][j] = MF::mma(af[buf][0], bfr[buf][j], acc[0][j]);
    };
    auto mfmas_tail = [&](int buf, int st) {
        const unsigned base = smem_base + st * G::STAGE_BYTES;
        constexpr int NM = (G::TM - 1) * G::TN;
        if constexpr (NM == 0) fire(st);  // one A fragment: the head was the whole step
#pragma unroll
        for (int m = 0; m < NM; ++m) {
            const int i = 1 + m / G::TN, j = m % G::TN;
            acc[i][j] = MF::mma(af[buf][i], bfr[buf][j], acc[i][j]);
            const int q0 = m * G::LOADS / NM, q1 = (m + 1) * G::LOADS / NM;
            if (q1 > q0) {
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int q = q0; q < q1; ++q) {
                    if (q < G::A_PER_WAVE)
                        dma16(ra, base + (wave_u * G::A_PER_WAVE + q) * 1024, offA[q]);
                    else
                        dma16(rb, base + G::A_BYTES + (wave_u * G::B_PER_WAVE + q - G::A_PER_WAVE) * 1024,
                              offB[q - G::A_PER_WAVE]);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    };

    // One MFMA followed by its share of the next step's LDS reads.
    auto interleave = [&]() {
        constexpr int NM = G::TM * G::TN;
        constexpr int ND = G::TM + 2 * G::TN;
        constexpr int PER = (ND + NM - 1) / NM;
#pragma unroll
        for (int m = 0; m < NM; ++m) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
            if (m * PER < ND) __builtin_amdgcn_sched_group_barrier(0x100, PER, 0);  // DS read
        }
    };

    // The loop body is branch-free: the tail iterations copy zeros into
    // slots nobody reads any more and read fragments they do not use, which
    // keeps the compiler's LDS-wait analysis exact (no conservative waits at
    // control-flow merges in front of the last k-step's MFMAs).
    constexpr bool LAG = STAGES >= 3;
    constexpr int AHEAD = LAG ? STAGES - 1 : STAGES;   // stages copied before stage 0 is computed
    const int KT = (K + BK - 1) / BK;
#pragma unroll
    for (int s = 0; s < AHEAD; ++s) {
        prepare(s);
        fire(s);
    }
    wait_vmcnt<(AHEAD - 1) * G::LOADS>();
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    load_frags(0, 0, 0);
    for (int kt = 0; kt < KT; ++kt) {
        const int st = kt % STAGES;
        prepare(kt + AHEAD);
#pragma unroll
        for (int s = 0; s + 1 < G::NS; ++s) {
            load_frags(st, s + 1, (s + 1) & 1);
            mfmas(s & 1);
            interleave();
        }
        if constexpr (LAG) {
            // stage kt+1 has landed (this wave's copies, then everyone's);
            // slot (kt-1) % STAGES was last read by iteration kt-1
            wait_vmcnt<(AHEAD - 2) * G::LOADS>();
            __builtin_amdgcn_s_barrier();
            asm volatile("" ::: "memory");
            load_frags((kt + 1) % STAGES, 0, 0);
            mfmas_with_copies((G::NS - 1) & 1, (kt + AHEAD) % STAGES);
        } else {
            mfmas_head((G::NS - 1) & 1);
            // This wave's copies of stage kt+1 have landed and all its LDS
            // reads (the last ones of slot st) have returned; after the
            // barrier the same holds for every wave, so slot st is free and
            // stage kt+1 is visible.  The empty asm keeps every LDS read of
            // slot st in front of the wait.
            __builtin_amdgcn_sched_barrier(0);
            asm volatile("" ::: "memory");
            wait_vmcnt_and_lds<(STAGES - 2) * G::LOADS>();
            __builtin_amdgcn_s_barrier();
            asm volatile("" ::: "memory");
            load_frags((kt + 1) % STAGES, 0, 0);
            mfmas_tail((G::NS - 1) & 1, st);
        }
    }
    wait_vmcnt<0>();  // no copy may still be writing LDS when the workgroup ends

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
                if (row < M && col < N)
                    __builtin_nontemporal_store((p.relu && acc[i][j][r] < 0.f) ? 0.f : acc[i][j][r],
                                                &C[row * ldc + col]);
            }
        }
}

template <int BM, int BN, int BK, int WM, int WN, int MI, int STAGES>
hipError_t launch_bf16_dma(const GemmArgs &a, hipStream_t s) {
    typedef Bf16DmaCfg<BM, BN, BK, WM, WN, MI, STAGES> G;
    const unsigned tiles = (unsigned)(((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN));
    GemmArgs args = a;
    void *kargs[] = {&args};
    return hipLaunchKernel(
        reinterpret_cast<const void *>(
            &gemm_bf16_dma_kernel<BM, BN, BK, WM, WN, MI, STAGES>),
        dim3(tiles), dim3(G::NT), kargs, 0, s);
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
            &launch_bf16<BM, BN, BK, WM, WN, MI, PAD, false>, kRowsAligned,                   \
            &occupancy_of<&gemm_bf16_kernel<BM, BN, BK, WM, WN, MI, PAD, true>,               \
                          (BM / WM) * (BN / WN) * 64, 0>                                      \
    }

// Direct-to-LDS ring (lds_pad = -1: swizzled, unpadded LDS rows), b128 A
// reads, MFMA / LDS-read interleaving.  The fallback for unaligned or
// non-16-byte-granular operands is the register-staged kernel with the same
// tiles.
#define XTC_BF16_DMA_INSTANCE(BM, BN, BK, WM, WN, MI, STAGES)                                 \
    GemmInstance {                                                                            \
        make_sched(BM, BN, BK, WM, WN, MI, MI, (MI == 32 ? 16 : 32), STAGES, -1, 0),           \
            &launch_bf16_dma<BM, BN, BK, WM, WN, MI, STAGES>,                                 \
            &launch_bf16<BM, BN, BK, WM, WN, MI, 8, false>, kWholeChunks,                     \
            &occupancy_of<&gemm_bf16_dma_kernel<BM, BN, BK, WM, WN, MI, STAGES>,              \
                          (BM / WM) * (BN / WN) * 64, 0>                                      \
    }

const GemmInstance kBf16Instances[] = {
    XTC_BF16_DMA_INSTANCE(256, 256, 32, 128, 64, 32, 4),  // default for large problems
    XTC_BF16_DMA_INSTANCE(256, 256, 64, 128, 64, 32, 2),
    XTC_BF16_DMA_INSTANCE(256, 256, 64, 128, 128, 32, 2), // 4 waves of 128x128
    XTC_BF16_DMA_INSTANCE(256, 128, 32, 128, 64, 32, 4),
    XTC_BF16_DMA_INSTANCE(128, 128, 32, 64, 64, 32, 4),   // medium problems
    XTC_BF16_DMA_INSTANCE(64, 128, 32, 32, 64, 32, 4),
    XTC_BF16_DMA_INSTANCE(64, 128, 64, 32, 64, 32, 2),
    XTC_BF16_DMA_INSTANCE(128, 128, 64, 64, 64, 16, 2),
    XTC_BF16_INSTANCE(256, 256, 64, 128, 64, 32, 8),
    XTC_BF16_INSTANCE(128, 128, 64, 64, 64, 32, 8),
    XTC_BF16_INSTANCE(64, 64, 64, 32, 32, 32, 8),         // small problems
    XTC_BF16_INSTANCE(128, 128, 64, 64, 64, 16, 8),       // 16x16x32 instruction tile
};

}  // namespace

const GemmInstance *gemm_bf16_instances(int *count) {
    *count = (int)(sizeof(kBf16Instances) / sizeof(kBf16Instances[0]));
    return kBf16Instances;
}

}  // namespace xtc
