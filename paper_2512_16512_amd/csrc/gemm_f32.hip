// fp32 GEMM on the gfx950 matrix cores: C[M,N] = A[M,K] * B[K,N], row-major,
// fp32 in, fp32 accumulate, fp32 out (C overwritten).
//
// How the paper's scheduling primitives (Sec. 3.2) appear here:
//  - strip-mine / tile + parallelize: one workgroup per BM x BN tile of C,
//    the tile grid spread over the CUs (tile_map.h for the order);
//  - second tiling level: each 64-lane wave owns a WM x WN sub-tile;
//  - vectorize: the innermost tile is one MFMA instruction tile
//    (32x32x2 or 16x16x4 fp32), accumulators stay in registers
//    (bufferize: they are written to C once, at the end);
//  - pack (with padding): each K-step of A (BM x BK) and B (BK x BN) is
//    copied to LDS in padded rows, double-buffered so that the global loads
//    of step t+1 overlap the matrix-core work of step t;
//  - split: the last K-step and the edge tiles use predicated loads that
//    zero-fill outside the matrix, and predicated stores.
//
// Operand fragments.  An fp32 MFMA of shape MIxMIxKG takes, per lane, one
// A value (row lane%MI, k-group lane/MI) and one B value (column lane%MI,
// k-group lane/MI).  Any assignment of the K-step's k values to
// (instruction, k-group) works as long as A and B agree; here lane group g
// of instruction s takes k = kk + 4g + s, so one ds_read_b128 per lane
// fetches the A values of four consecutive instructions from a k-contiguous
// LDS row, and B (n-contiguous in LDS) is read with conflict-free
// ds_read_b32 (lanes of one group read consecutive columns).
#include "lds_dma.h"
#include "mfma_f32.h"
#include "tile_map.h"
#include "xtc_internal.h"

namespace xtc {
namespace {

template <int BM, int BN, int BK, int WM, int WN, int MI, int PAD, bool VEC>
struct GemmF32Cfg {
    static constexpr int NWM = BM / WM, NWN = BN / WN;
    static constexpr int NT = NWM * NWN * 64;
    static constexpr int TM = WM / MI, TN = WN / MI;
    typedef F32Mfma<MI> MF;
    static constexpr int KG = MF::KG;
    static constexpr int KCH = 4 * KG;                 // k consumed per A fragment read
    static constexpr int AS = BK + PAD;                // A tile LDS row stride (floats)
    static constexpr int BS = BN + (MI == 32 ? 8 : 4); // B tile LDS row stride (floats)
    static constexpr int W = VEC ? 4 : 1;              // elements per global load
    static constexpr int A_CPR = BK / W;               // loads per A tile row
    static constexpr int B_CPR = BN / W;               // loads per B tile row
    static constexpr int A_LOADS = BM * BK / (W * NT);
    static constexpr int B_LOADS = BK * BN / (W * NT);
    typedef typename VecF32<W>::t vec_t;
    static_assert(BM % WM == 0 && BN % WN == 0, "wave tile must divide the block tile");
    static_assert(WM % MI == 0 && WN % MI == 0, "MFMA tile must divide the wave tile");
    static_assert(BK % KCH == 0, "block_k must be a multiple of the fragment k-chunk");
    static_assert(A_LOADS * W * NT == BM * BK, "A tile must split evenly over threads");
    static_assert(B_LOADS * W * NT == BK * BN, "B tile must split evenly over threads");
    static_assert(PAD % 4 == 0, "A padding must keep 16-byte alignment");
};

template <int BM, int BN, int BK, int WM, int WN, int MI, int PAD, bool VEC>
__global__ void __launch_bounds__((BM / WM) * (BN / WN) * 64)
gemm_f32_kernel(GemmArgs p) {
    typedef GemmF32Cfg<BM, BN, BK, WM, WN, MI, PAD, VEC> G;
    typedef typename G::MF MF;
    typedef typename G::vec_t vec_t;
    constexpr int W = G::W;

    __shared__ __attribute__((aligned(16))) float As[2][BM * G::AS];
    __shared__ __attribute__((aligned(16))) float Bs[2][BK * G::BS];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave / G::NWN, wn = wave % G::NWN;
    const int lrow = lane % MI, lgrp = lane / MI;

    const int M = p.M, N = p.N, K = p.K;
    const int tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
    int tm, tn;
    tile_coords(blockIdx.x, gridDim.x, tiles_m, tiles_n, p.raster, p.xcd_remap, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;

    const float *__restrict__ A = static_cast<const float *>(p.A);
    const float *__restrict__ B = static_cast<const float *>(p.B);
    const int lda = p.lda, ldb = p.ldb;

    vec_t ra[G::A_LOADS], rb[G::B_LOADS];

    // Global -> registers for K-step kt (zero-filled outside the matrix).
    auto load_tiles = [&](int kt) {
        const int k0 = kt * BK;
#pragma unroll
        for (int i = 0; i < G::A_LOADS; ++i) {
            const int idx = tid + i * G::NT;
            const int r = idx / G::A_CPR, c = (idx % G::A_CPR) * W;
            const int gm = m0 + r, gk = k0 + c;
            const int valid = gm < M ? K - gk : 0;
            ra[i] = load_pred<W>(A + (gm < M ? gm : 0) * lda + (valid > 0 ? gk : 0), valid);
        }
#pragma unroll
        for (int i = 0; i < G::B_LOADS; ++i) {
            const int idx = tid + i * G::NT;
            const int r = idx / G::B_CPR, c = (idx % G::B_CPR) * W;
            const int gk = k0 + r, gn = n0 + c;
            const int valid = gk < K ? N - gn : 0;
            rb[i] = load_pred<W>(B + (gk < K ? gk : 0) * ldb + (valid > 0 ? gn : 0), valid);
        }
    };

    // Registers -> LDS stage `st`.
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

    // Epilogue: accumulators -> C, masked on the edges.
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

template <int BM, int BN, int BK, int WM, int WN, int MI, int PAD, bool VEC>
hipError_t launch_f32(const GemmArgs &a, hipStream_t s) {
    typedef GemmF32Cfg<BM, BN, BK, WM, WN, MI, PAD, VEC> G;
    const unsigned tiles = (unsigned)(((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN));
    GemmArgs args = a;
    void *kargs[] = {&args};
    return hipLaunchKernel(reinterpret_cast<const void *>(&gemm_f32_kernel<BM, BN, BK, WM, WN, MI, PAD, VEC>),
                           dim3(tiles), dim3(G::NT), kargs, 0, s);
}

// ---------------------------------------------------------------------------
// Direct-to-LDS variant: A and B tiles reach a ring of STAGES LDS buffers
// through 16-byte buffer loads with the `lds` modifier (no register
// staging); out-of-range chunks read as zero through the buffer range check
// (needs K and N multiples of 4 and 16-byte aligned rows, else the
// register-staged kernel above runs).
//  - A rows (BK floats, 16-byte chunks) store chunk c of row m at slot
//    c ^ swizzle(m).  gfx950 serves a ds_read_b128 in four phases of 16
//    lanes ({0-3, 12-15, 20-23, 24-27}, {4-11, 16-19, 28-31} and the same
//    + 32) over 64 banks; the swizzles give the rows of each phase distinct
//    16-byte bank groups for both instruction tiles (checked for every
//    instance with the LDS model, paper_2512_16512_amd/lds_model.py);
//  - B rows (n-contiguous) store chunk c of row k at c ^ 8*((k >> 2) & 1):
//    a ds_read_b32 of the B operand reads rows k and k+4 with the two halves
//    of the wave, which then land 128 bytes apart (different bank halves).
// Main loop: the ping-pong of the bf16 direct-to-LDS kernel.
template <int CA>
__device__ __forceinline__ int swz_a_f32(int row) {
    return CA == 4 ? (row >> 2) & 3 : (row >> 1) & 7;
}

template <int BM, int BN, int BK, int WM, int WN, int MI_, int STAGES>
struct F32DmaCfg {
    static constexpr int MI = MI_;
    static constexpr int NWM = BM / WM, NWN = BN / WN;
    static constexpr int NWAVES = NWM * NWN;
    static constexpr int NT = NWAVES * 64;
    static constexpr int TM = WM / MI, TN = WN / MI;
    typedef F32Mfma<MI> MF;
    static constexpr int KG = MF::KG;               // lane groups along k (2 or 4)
    static constexpr int KCH = 4 * KG;              // k per fragment set (8 or 16)
    static constexpr int SWB = 16 / KG;             // B chunk XOR step between lane groups
    static constexpr int NS = BK / KCH;
    static constexpr int RA = BK * 4, CA = BK / 4;  // A row bytes / chunks
    static constexpr int RB = BN * 4, CB = BN / 4;  // B row bytes / chunks
    static constexpr int A_BYTES = BM * RA, B_BYTES = BK * RB;
    static constexpr int A_BLOCKS = A_BYTES / 1024, B_BLOCKS = B_BYTES / 1024;
    static constexpr int A_PER_WAVE = A_BLOCKS / NWAVES, B_PER_WAVE = B_BLOCKS / NWAVES;
    static constexpr int LOADS = A_PER_WAVE + B_PER_WAVE;
    static constexpr int STAGE_BYTES = A_BYTES + B_BYTES;
    static_assert(A_PER_WAVE * NWAVES == A_BLOCKS && B_PER_WAVE * NWAVES == B_BLOCKS,
                  "tiles must split into whole 1 KiB blocks per wave");
    static_assert(CA == 4 || CA == 8, "block_k must be 16 or 32");
    static_assert(CB >= 16 && RB <= 1024, "block_n must be 64..256");
    static_assert(SWB * (KG - 1) < CB, "B swizzle stays inside a row");
    static_assert(NS % 2 == 0, "an even number of fragment sets per stage");
    static_assert(STAGES >= 2 && STAGES * STAGE_BYTES <= 160 * 1024, "LDS budget");
    static_assert((STAGES - 1) * LOADS < 64, "vmcnt range");
};

// KSW > 1: the workgroup holds KSW groups of waves, each running the whole
// pipeline below on its own LDS ring over every KSW-th K-step (group g takes
// K-steps g, g + KSW, ...), with the same number of iterations in every
// group (zero-filled K-steps past the end), so that each SIMD holds KSW
// waves and one wave's LDS and barrier waits overlap another's matrix
// instructions.  At the end the groups' accumulators are added through LDS
// in the fixed order 0, 1, ..., KSW-1 (deterministic results).
template <int BM, int BN, int BK, int WM, int WN, int MI_, int STAGES, int KSW = 1>
__global__ void __launch_bounds__((BM / WM) * (BN / WN) * 64 * KSW)
gemm_f32_dma_kernel(GemmArgs p) {
    typedef F32DmaCfg<BM, BN, BK, WM, WN, MI_, STAGES> G;
    typedef typename G::MF MF;
    constexpr int MI = G::MI;
    static_assert(KSW * STAGES * G::STAGE_BYTES <= 160 * 1024, "LDS budget");
    __shared__ __attribute__((aligned(1024))) unsigned char smem_all[KSW * STAGES * G::STAGE_BYTES];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int kg = __builtin_amdgcn_readfirstlane((tid >> 6) / G::NWAVES);   // K group of this wave
    const int wave = (tid >> 6) % G::NWAVES;        // wave inside its group
    unsigned char *const smem = smem_all + kg * STAGES * G::STAGE_BYTES;
    const int wm = wave / G::NWN, wn = wave % G::NWN;
    const int lrow = lane % MI, lgrp = lane / MI;

    const int M = p.M, N = p.N, K = p.K;
    const int tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
    int tm, tn;
    tile_coords(blockIdx.x, gridDim.x, tiles_m, tiles_n, p.raster, p.xcd_remap, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;

    const i32x4 ra = make_rsrc(p.A, ((M - 1) * p.lda + K) * 4);
    const i32x4 rb = make_rsrc(p.B, ((K - 1) * p.ldb + N) * 4);
    const int wave_u = __builtin_amdgcn_readfirstlane(wave);
    const unsigned smem_base = lds_address(smem);

    int a_row[G::A_PER_WAVE], a_col[G::A_PER_WAVE];
#pragma unroll
    for (int q = 0; q < G::A_PER_WAVE; ++q) {
        const int row = (wave * G::A_PER_WAVE + q) * (1024 / G::RA) + lane / G::CA;
        a_row[q] = row;
        a_col[q] = 4 * ((lane % G::CA) ^ swz_a_f32<G::CA>(row));
    }
    int b_row[G::B_PER_WAVE], b_col[G::B_PER_WAVE];
#pragma unroll
    for (int q = 0; q < G::B_PER_WAVE; ++q) {
        const int row = (wave * G::B_PER_WAVE + q) * (1024 / G::RB) + lane / G::CB;
        b_row[q] = row;
        b_col[q] = 4 * ((lane % G::CB) ^ (G::SWB * ((row >> 2) & (G::KG - 1))));
    }

    int offA[G::A_PER_WAVE], offB[G::B_PER_WAVE];
    auto prepare = [&](int kt) {
        const int k0 = (kt * KSW + kg) * BK;
#pragma unroll
        for (int q = 0; q < G::A_PER_WAVE; ++q) {
            const int gm = m0 + a_row[q], gk = k0 + a_col[q];
            offA[q] = (gm < M && gk < K) ? (gm * p.lda + gk) * 4 : kOOB;
        }
#pragma unroll
        for (int q = 0; q < G::B_PER_WAVE; ++q) {
            const int gk = k0 + b_row[q], gn = n0 + b_col[q];
            offB[q] = (gk < K && gn < N) ? (gk * p.ldb + gn) * 4 : kOOB;
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

    int a_off[G::TM], a_swz[G::TM];
#pragma unroll
    for (int i = 0; i < G::TM; ++i) {
        const int row = wm * WM + i * MI + lrow;
        a_off[i] = row * G::RA;
        a_swz[i] = swz_a_f32<G::CA>(row);
    }
    // B row kk + 4*lgrp + s has (row >> 2) % KG == lgrp (kk % (4*KG) == 0).
    int b_off[G::TN];
#pragma unroll
    for (int j = 0; j < G::TN; ++j)
        b_off[j] = (4 * lgrp * BN + ((wn * WN + j * MI + lrow) ^ (4 * G::SWB * lgrp))) * 4;

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
                bfr[buf][j][s] = *reinterpret_cast<const float *>(Bs + (kk + s) * G::RB + b_off[j]);
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

    // The last fragment set of a stage: its MFMAs with the copies of the
    // stage STAGES ahead spread between them (copies issued all at once by
    // every wave right after the barrier queue at the texture unit and
    // stall the issuing waves); the fences keep the order.
    auto mfmas_with_copies = [&](int buf, int st) {
        const unsigned base = smem_base + st * G::STAGE_BYTES;
        constexpr int NM = 4 * G::TM * G::TN;
#pragma unroll
        for (int m = 0; m < NM; ++m) {
            const int s = m / (G::TM * G::TN), i = (m / G::TN) % G::TM, j = m % G::TN;
            acc[i][j] = MF::mma(af[buf][i][s], bfr[buf][j][s], acc[i][j]);
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

    // Branch-free main loop: every stage index issues LOADS copies per wave
    // (zero-fill copies past the end of K), so one vmcnt value is exact in
    // every iteration and the compiler's LDS waits stay tight.
    const int KT = ((K + BK - 1) / BK + KSW - 1) / KSW;   // iterations of every group
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
            // one MFMA, then one LDS read of the next fragment set
#pragma unroll
            for (int m = 0; m < 4 * G::TM * G::TN; ++m) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                if (m < G::TM + 4 * G::TN) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            }
        }
        wait_vmcnt_and_lds<(STAGES - 2) * G::LOADS>();
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        load_frags((kt + 1) % STAGES, 0, 0);
        mfmas_with_copies((G::NS - 1) & 1, st);
    }
    wait_vmcnt<0>();  // no copy may still be writing LDS when the workgroup ends

    if constexpr (KSW > 1) {
        // groups 1 .. KSW-1 leave their sums in LDS (each lane its own
        // registers, lane-contiguous); group 0 adds them in group order
        constexpr int NREG = G::TM * G::TN * MF::NACC;
        static_assert((KSW - 1) * G::NWAVES * NREG * 64 * 4 <= KSW * STAGES * G::STAGE_BYTES,
                      "partial sums fit in the rings");
        float *red = reinterpret_cast<float *>(smem_all);
        __syncthreads();   // every group's last fragment reads are done
        if (kg > 0) {
#pragma unroll
            for (int i = 0; i < G::TM; ++i)
#pragma unroll
                for (int j = 0; j < G::TN; ++j)
#pragma unroll
                    for (int r = 0; r < MF::NACC; ++r)
                        red[((((kg - 1) * G::NWAVES + wave) * G::TM + i) * G::TN + j) * MF::NACC * 64 + r * 64 + lane] =
                            acc[i][j][r];
        }
        __syncthreads();
        if (kg > 0) return;
#pragma unroll
        for (int g = 1; g < KSW; ++g)
#pragma unroll
            for (int i = 0; i < G::TM; ++i)
#pragma unroll
                for (int j = 0; j < G::TN; ++j)
#pragma unroll
                    for (int r = 0; r < MF::NACC; ++r)
                        acc[i][j][r] += red[((((g - 1) * G::NWAVES + wave) * G::TM + i) * G::TN + j) * MF::NACC * 64 +
                                            r * 64 + lane];
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

template <int BM, int BN, int BK, int WM, int WN, int MI, int STAGES, int KSW = 1>
hipError_t launch_f32_dma(const GemmArgs &a, hipStream_t s) {
    typedef F32DmaCfg<BM, BN, BK, WM, WN, MI, STAGES> G;
    const unsigned tiles = (unsigned)(((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN));
    GemmArgs args = a;
    void *kargs[] = {&args};
    return hipLaunchKernel(
        reinterpret_cast<const void *>(&gemm_f32_dma_kernel<BM, BN, BK, WM, WN, MI, STAGES, KSW>),
        dim3(tiles), dim3(G::NT * KSW), kargs, 0, s);
}

// ---------------------------------------------------------------------------
// Reduction-split kernel (k_split = KS > 1) for problems with too few output
// tiles to fill the chip.  KS waves share one BM x BN tile (BM = MI*TM,
// BN = MI*TN); wave g reduces the K-steps g, g + KS, g + 2KS, ... of
// BK = U*KCH k values each.  Operands go from memory straight to the MFMA
// operand registers (a small problem is L2-resident, and no LDS round trip
// sits on the latency path) through a ring of D register buffers: the loads
// of the wave's K-step t + D - 1 are issued before the MFMAs of step t, so
// that D - 1 steps of loads are in flight behind the matrix-core work.  At the
// end every wave writes its partial accumulators to LDS and the KS partials
// are added in the fixed order g = 0, 1, ..., KS-1 (deterministic results),
// each wave finishing an interleaved share of the tile's registers, with the
// epilogue applied to the sum.
template <int MI, int TM, int TN, int KS, int U, int D, bool VEC>
__global__ void __launch_bounds__(KS * 64)
gemm_f32_ksplit_kernel(GemmArgs p) {
    typedef F32Mfma<MI> MF;
    constexpr int KCH = 4 * MF::KG;  // k values of one fragment set (4 instructions)
    constexpr int BK = U * KCH;      // k values of one K-step
    constexpr int BM = MI * TM, BN = MI * TN;
    constexpr int NREG = TM * TN * MF::NACC;
    __shared__ float red[KS][NREG][64];

    const int lane = threadIdx.x & 63, g = threadIdx.x >> 6;
    const int lrow = lane % MI, lgrp = lane / MI;
    const int M = p.M, N = p.N, K = p.K;
    const int tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
    int tm, tn;
    tile_coords(blockIdx.x, gridDim.x, tiles_m, tiles_n, p.raster, p.xcd_remap, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;

    const float *__restrict__ A = static_cast<const float *>(p.A);
    const float *__restrict__ B = static_cast<const float *>(p.B);
    const int lda = p.lda, ldb = p.ldb;

    // Branch-free loads: buffer loads whose offset is moved past the end of
    // the operand (kOOB) when the element lies outside the matrix read zero.
    // VEC (K a multiple of 4, 16-byte aligned A rows): one 16-byte load per A
    // row segment; otherwise one 4-byte load per element.
    const __amdgpu_buffer_rsrc_t ra =
        __builtin_amdgcn_make_buffer_rsrc((void *)A, (short)0, ((M - 1) * lda + K) * 4, 0x00020000);
    const __amdgpu_buffer_rsrc_t rb =
        __builtin_amdgcn_make_buffer_rsrc((void *)B, (short)0, K > 0 ? ((K - 1) * ldb + N) * 4 : 0,
                                          0x00020000);
    // Per-lane byte offsets of this lane's A rows and B columns, moved out of
    // range when the row or column lies outside the matrix.  B rows at or
    // past K are out of range by themselves (K*ldb + n >= (K-1)*ldb + N), so
    // the k index of B is only clamped to K (which also keeps the unsigned
    // offset from wrapping); A, whose next row follows row i directly, tests
    // k < K.
    unsigned aoff[TM], boff[TN];
#pragma unroll
    for (int i = 0; i < TM; ++i) {
        const int r = m0 + i * MI + lrow;
        aoff[i] = r < M ? (unsigned)(r * lda) * 4u : (unsigned)kOOB;
    }
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int c = n0 + j * MI + lrow;
        boff[j] = c < N ? (unsigned)c * 4u : (unsigned)kOOB;
    }

    // Lane group lgrp of instruction s takes k = kb + s with kb = k0 + 4*lgrp
    // (as in the LDS-staged kernels): one 16-byte row segment of A and four
    // column values of B per fragment set.
    f32x4 fa[D][U][TM];
    float fb[D][U][TN][4];
    auto load = [&](const int buf, const int kt) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int kb = kt * BK + u * KCH + 4 * lgrp;
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                if (VEC) {
                    const unsigned off = kb < K ? aoff[i] + (unsigned)kb * 4u : (unsigned)kOOB;
                    fa[buf][u][i] = __builtin_bit_cast(
                        f32x4, __builtin_amdgcn_raw_buffer_load_b128(ra, (int)off, 0, 0));
                } else {
#pragma unroll
                    for (int s = 0; s < 4; ++s) {
                        const unsigned off =
                            kb + s < K ? aoff[i] + (unsigned)(kb + s) * 4u : (unsigned)kOOB;
                        fa[buf][u][i][s] = __builtin_bit_cast(
                            float, __builtin_amdgcn_raw_buffer_load_b32(ra, (int)off, 0, 0));
                    }
                }
            }
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const unsigned roff = (unsigned)(min(kb + s, K) * ldb) * 4u;
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    fb[buf][u][j][s] = __builtin_bit_cast(
                        float, __builtin_amdgcn_raw_buffer_load_b32(rb, (int)(roff + boff[j]), 0, 0));
            }
        }
    };

    typename MF::acc_t acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < MF::NACC; ++r) acc[i][j][r] = 0.f;

    auto compute = [&](const int buf) {
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int s = 0; s < 4; ++s)
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = MF::mma(fa[buf][u][i][s], fb[buf][u][j][s], acc[i][j]);
    };

    // D K-steps per iteration (unrolled) so that every register buffer is
    // named by a constant.  This wave's steps are g, g + KS, ...  The loads
    // are branch-free: steps past the end are loaded (as zeros, every offset
    // being out of range), so every step issues the same loads and the
    // compiler's wait counts stay exact.  Only the matrix instructions of
    // steps past the end are skipped (a uniform branch with no memory
    // instruction in it): with a short reduction most of an iteration's
    // steps can lie past it (K = 128 on 32x32 tiles: three of four).
    const int KT = (K + BK - 1) / BK;
#pragma unroll
    for (int d = 0; d + 1 < D; ++d) load(d, g + d * KS);
    for (int base = g; base < KT; base += D * KS) {
#pragma unroll
        for (int d = 0; d < D; ++d) {
            load((d + D - 1) % D, base + (d + D - 1) * KS);
            if (d == 0 || base + d * KS < KT) compute(d);
        }
    }

    // Fixed-order reduction of the KS partial tiles through LDS.
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < MF::NACC; ++r) red[g][(i * TN + j) * MF::NACC + r][lane] = acc[i][j][r];
    __syncthreads();
    float *__restrict__ C = p.C;
    const int ldc = p.ldc;
    for (int q = g; q < NREG; q += KS) {
        float v = red[0][q][lane];
#pragma unroll
        for (int h = 1; h < KS; ++h) v += red[h][q][lane];
        const int i = q / (TN * MF::NACC), j = (q / MF::NACC) % TN, r = q % MF::NACC;
        const int row = m0 + i * MI + MF::row(lane, r);
        const int col = n0 + j * MI + lrow;
        if (row < M && col < N) C[row * ldc + col] = (p.relu && v < 0.f) ? 0.f : v;
    }
}

template <int MI, int TM, int TN, int KS, int U, int D, bool VEC>
hipError_t launch_f32_ksplit(const GemmArgs &a, hipStream_t s) {
    constexpr int BM = MI * TM, BN = MI * TN;
    const unsigned tiles = (unsigned)(((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN));
    GemmArgs args = a;
    void *kargs[] = {&args};
    return hipLaunchKernel(
        reinterpret_cast<const void *>(&gemm_f32_ksplit_kernel<MI, TM, TN, KS, U, D, VEC>),
        dim3(tiles), dim3(KS * 64), kargs, 0, s);
}

#define XTC_F32_INSTANCE(BM, BN, BK, WM, WN, MI, PAD)                                         \
    GemmInstance {                                                                            \
        make_sched(BM, BN, BK, WM, WN, MI, MI, (MI == 32 ? 2 : 4), 2, PAD, 0),                 \
            &launch_f32<BM, BN, BK, WM, WN, MI, PAD, true>,                                   \
            &launch_f32<BM, BN, BK, WM, WN, MI, PAD, false>, kRowsAligned,                    \
            &occupancy_of<&gemm_f32_kernel<BM, BN, BK, WM, WN, MI, PAD, true>,                \
                          (BM / WM) * (BN / WN) * 64, 0>                                      \
    }

// Direct-to-LDS ring (lds_pad = -1); register-staged fallback, same tiles.
#define XTC_F32_DMA_INSTANCE(BM, BN, BK, WM, WN, STAGES) XTC_F32_DMA_MI_INSTANCE(BM, BN, BK, WM, WN, 32, STAGES)
#define XTC_F32_DMA_MI_INSTANCE(BM, BN, BK, WM, WN, MI, STAGES)                               \
    GemmInstance {                                                                            \
        make_sched(BM, BN, BK, WM, WN, MI, MI, (MI == 32 ? 2 : 4), STAGES, -1, 0),             \
            &launch_f32_dma<BM, BN, BK, WM, WN, MI, STAGES>,                                  \
            &launch_f32<BM, BN, BK, WM, WN, MI, 4, false>, kWholeChunks,                      \
            &occupancy_of<&gemm_f32_dma_kernel<BM, BN, BK, WM, WN, MI, STAGES>,               \
                          (BM / WM) * (BN / WN) * 64, 0>                                      \
    }

// In-workgroup reduction split: KSW groups of waves on one tile (k_split =
// KSW with LDS staging); the fallback is the unsplit register-staged kernel.
#define XTC_F32_DMA_KSW_INSTANCE(BM, BN, BK, WM, WN, STAGES, KSW)                             \
    GemmInstance {                                                                            \
        make_sched(BM, BN, BK, WM, WN, 32, 32, 2, STAGES, -1, 0, 0, KSW),                     \
            &launch_f32_dma<BM, BN, BK, WM, WN, 32, STAGES, KSW>,                             \
            &launch_f32<BM, BN, BK, WM, WN, 32, 4, false>, kWholeChunks,                      \
            &occupancy_of<&gemm_f32_dma_kernel<BM, BN, BK, WM, WN, 32, STAGES, KSW>,          \
                          (BM / WM) * (BN / WN) * 64 * KSW, 0>                                \
    }

// 256x256 tiles: the register-staged kernel with the same tiles would spill,
// so the fallback runs 128x128 tiles of four 64x64 waves.
#define XTC_F32_DMA_BIG_INSTANCE(BM, BN, BK, WM, WN, STAGES)                                  \
    GemmInstance {                                                                            \
        make_sched(BM, BN, BK, WM, WN, 32, 32, 2, STAGES, -1, 0),                             \
            &launch_f32_dma<BM, BN, BK, WM, WN, 32, STAGES>,                                  \
            &launch_f32<128, 128, 32, 64, 64, 32, 4, false>, kWholeChunks,                    \
            &occupancy_of<&gemm_f32_dma_kernel<BM, BN, BK, WM, WN, 32, STAGES>,               \
                          (BM / WM) * (BN / WN) * 64, 0>                                      \
    }

// Reduction-split instances: KS waves per MI*TM x MI*TN tile, U fragment
// sets per K-step, D K-steps in flight per wave, no LDS staging.
#define XTC_F32_KSPLIT_INSTANCE(MI, TM, TN, KS, U, D)                                         \
    GemmInstance {                                                                            \
        make_sched(MI * TM, MI * TN, U * 4 * (64 / MI), MI * TM, MI * TN, MI, MI,             \
                   (MI == 32 ? 2 : 4), 0, 0, 0, 0, KS),                                       \
            &launch_f32_ksplit<MI, TM, TN, KS, U, D, true>,                                   \
            &launch_f32_ksplit<MI, TM, TN, KS, U, D, false>, kARowsOnly,                      \
            &occupancy_of<&gemm_f32_ksplit_kernel<MI, TM, TN, KS, U, D, true>, KS * 64, 0>    \
    }

const GemmInstance kF32Instances[] = {
    XTC_F32_DMA_INSTANCE(256, 128, 16, 128, 64, 3),
    XTC_F32_DMA_INSTANCE(256, 128, 32, 128, 64, 2),
    XTC_F32_DMA_INSTANCE(128, 128, 32, 64, 64, 2),
    XTC_F32_DMA_INSTANCE(128, 128, 16, 64, 64, 4),
    XTC_F32_DMA_MI_INSTANCE(128, 128, 32, 64, 64, 16, 2),   // 16x16x4 instruction tile
    XTC_F32_DMA_INSTANCE(256, 128, 32, 64, 64, 2),   // 8 waves of 64x64
    XTC_F32_DMA_INSTANCE(128, 256, 32, 64, 64, 2),
    XTC_F32_DMA_BIG_INSTANCE(256, 256, 32, 128, 64, 2),   // default for large problems
    XTC_F32_DMA_BIG_INSTANCE(256, 256, 32, 64, 64, 2),    // 16 waves of 64x64
    XTC_F32_DMA_INSTANCE(64, 128, 32, 32, 64, 3),    // mid-size problems
    XTC_F32_DMA_INSTANCE(64, 64, 32, 32, 32, 4),
    XTC_F32_DMA_INSTANCE(64, 64, 32, 32, 32, 2),
    XTC_F32_DMA_KSW_INSTANCE(64, 64, 32, 32, 32, 2, 2),   // two K groups of four 32x32 waves
    XTC_F32_DMA_KSW_INSTANCE(64, 64, 32, 32, 32, 2, 4),
    XTC_F32_INSTANCE(128, 128, 32, 64, 64, 32, 4),
    XTC_F32_INSTANCE(128, 128, 16, 64, 64, 32, 4),
    XTC_F32_INSTANCE(64, 64, 32, 32, 32, 32, 4),     // small problems: more tiles
    XTC_F32_INSTANCE(128, 128, 32, 64, 64, 16, 8),   // 16x16x4 instruction tile (A rows padded by
                                                     // 8: conflict-free fragment reads)
    XTC_F32_INSTANCE(256, 128, 16, 128, 64, 32, 4),
    XTC_F32_KSPLIT_INSTANCE(32, 1, 1, 4, 4, 4),      // 32x32 tiles, 4 waves
    XTC_F32_KSPLIT_INSTANCE(32, 1, 1, 8, 4, 4),      // 32x32 tiles, 8 waves
    XTC_F32_KSPLIT_INSTANCE(32, 2, 1, 4, 2, 4),      // 64x32 tiles
    XTC_F32_KSPLIT_INSTANCE(32, 2, 2, 4, 2, 3),      // 64x64 tiles
    XTC_F32_KSPLIT_INSTANCE(16, 1, 1, 4, 2, 4),      // 16x16 tiles, 16x16x4 instruction
    XTC_F32_KSPLIT_INSTANCE(16, 1, 1, 8, 2, 4),      // 16x16 tiles, 8 waves
    XTC_F32_KSPLIT_INSTANCE(16, 2, 1, 8, 2, 4),      // 32x16 tiles: tall-skinny products
};

}  // namespace

const GemmInstance *gemm_f32_instances(int *count) {
    *count = (int)(sizeof(kF32Instances) / sizeof(kF32Instances[0]));
    return kF32Instances;
}

}  // namespace xtc
