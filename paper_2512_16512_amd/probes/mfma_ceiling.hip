// Sustained matrix-core throughput with no memory traffic: the ceiling a
// contraction kernel on this chip can approach when every operand is already
// in registers.
//
// Every wave keeps a 128x64 accumulator tile and
// issues back-to-back MFMAs on operands held in registers, rotating which
// operand registers feed which accumulator so that no instruction repeats its
// inputs.  The operands are uniform [-1, 1) values (rounded to bf16 for the
// bf16 modes), or all zero with --zeros: the chip's power draw, and with it
// the clock under its power limit, depends on how many operand bits toggle.
//
// usage: mfma_ceiling [--zeros] [workgroups=2048] [iterations=20000]
// Prints, per instruction, the median TFLOP/s of five timed launches and its
// fraction of the MI355X dense peak (bf16 2516.6, fp32 157.3 TFLOP/s).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));

#define CHECK(x)                                                                      \
    do {                                                                              \
        hipError_t e_ = (x);                                                          \
        if (e_ != hipSuccess) {                                                       \
            fprintf(stderr, "%s: %s\n", #x, hipGetErrorString(e_));                  \
            exit(1);                                                                  \
        }                                                                             \
    } while (0)

constexpr int kWords = 65536;   // operand table: 65536 groups of 8 values

// MODE 0: v_mfma_f32_32x32x16_bf16, 4x2 accumulators (a 128x64 tile);
// MODE 1: v_mfma_f32_16x16x32_bf16, 8x4 accumulators (128x64);
// MODE 2: v_mfma_f32_32x32x2_f32,  4x2 accumulators (128x64);
// MODE 3: v_mfma_f32_16x16x4_f32,  8x4 accumulators (128x64).
template <int MODE>
__global__ __launch_bounds__(256) void mfma_loop(const u16x8 *in, float *out, int iters) {
    const int t = blockIdx.x * 256 + threadIdx.x;
    u16x8 a[4], b[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        a[i] = in[(t * 8 + i) & (kWords - 1)];
        b[i] = in[(t * 8 + 4 + i) & (kWords - 1)];
    }
    float s = 0.f;
    if constexpr (MODE == 0) {
        f32x16 acc[4][2] = {};
        for (int it = 0; it < iters; it += 4)
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                            __builtin_bit_cast(bf16x8, a[(i + u) & 3]),
                            __builtin_bit_cast(bf16x8, b[(j + u) & 3]), acc[i][j], 0, 0, 0);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) s += acc[i][j][r];
    } else if constexpr (MODE == 1) {
        f32x4 acc[8][4] = {};
        for (int it = 0; it < iters; it += 4)
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int i = 0; i < 8; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                            __builtin_bit_cast(bf16x8, a[(i + u) & 3]),
                            __builtin_bit_cast(bf16x8, b[(j + u + (i >> 2)) & 3]), acc[i][j], 0, 0, 0);
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int r = 0; r < 4; ++r) s += acc[i][j][r];
    } else {
        // fp32 operands with 23 random mantissa bits, uniform in [-0.5, 0.5)
        // (zero where the table is zero), from pairs of table entries
        float fa[8], fb[8];
        auto widen = [](unsigned hi, unsigned lo) {
            const unsigned bits = (hi << 16) | lo;
            const unsigned u = 0x3F800000u | (bits & 0x7FFFFFu);
            float f;
            memcpy(&f, &u, 4);
            return bits ? f - 1.5f : 0.f;
        };
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            fa[i] = widen(a[i >> 1][4 * (i & 1)], a[i >> 1][4 * (i & 1) + 1]);
            fb[i] = widen(b[i >> 1][4 * (i & 1) + 2], b[i >> 1][4 * (i & 1) + 3]);
        }
        if constexpr (MODE == 2) {
            f32x16 acc[4][2] = {};
            for (int it = 0; it < iters; it += 4)
#pragma unroll
                for (int u = 0; u < 4; ++u)
#pragma unroll
                    for (int i = 0; i < 4; ++i)
#pragma unroll
                        for (int j = 0; j < 2; ++j)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[(2 * u + i) & 7], fb[(2 * u + j + 1) & 7],
                                                                             acc[i][j], 0, 0, 0);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
#pragma unroll
                    for (int r = 0; r < 16; ++r) s += acc[i][j][r];
        } else {
            f32x4 acc[8][4] = {};
            for (int it = 0; it < iters; it += 4)
#pragma unroll
                for (int u = 0; u < 4; ++u)
#pragma unroll
                    for (int i = 0; i < 8; ++i)
#pragma unroll
                        for (int j = 0; j < 4; ++j)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[(u + i) & 7], fb[(u + j + 3) & 7],
                                                                             acc[i][j], 0, 0, 0);
#pragma unroll
            for (int i = 0; i < 8; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
#pragma unroll
                    for (int r = 0; r < 4; ++r) s += acc[i][j][r];
        }
    }
    out[t] = s;   // keeps the loop live
}

static unsigned short to_bf16(float f) {
    unsigned u;
    memcpy(&u, &f, 4);
    return (unsigned short)((u + 0x7FFF + ((u >> 16) & 1)) >> 16);
}

int main(int argc, char **argv) {
    bool zeros = false;
    int pos[2] = {2048, 20000}, np = 0;
    for (int i = 1; i < argc; ++i) {
        if (!strcmp(argv[i], "--zeros")) zeros = true;
        else if (np < 2) pos[np++] = atoi(argv[i]);
    }
    const int wgs = pos[0], iters = pos[1] / 4 * 4;
    if (wgs < 1 || iters < 4) {
        fprintf(stderr, "usage: mfma_ceiling [--zeros] [workgroups>=1] [iterations>=4]\n");
        return 2;
    }
    std::vector<unsigned short> h((size_t)kWords * 8);
    unsigned long long st = 0x2512165120ull;
    for (auto &v : h) {
        st = st * 6364136223846793005ull + 1442695040888963407ull;
        const float f = (float)(st >> 40) * (1.0f / 8388608.0f) - 1.0f;   // uniform [-1, 1)
        v = zeros ? 0 : to_bf16(f);
    }
    u16x8 *din;
    float *dout;
    CHECK(hipMalloc(&din, h.size() * 2));
    CHECK(hipMalloc(&dout, (size_t)wgs * 256 * 4));
    CHECK(hipMemcpy(din, h.data(), h.size() * 2, hipMemcpyHostToDevice));
    hipEvent_t e0, e1;
    CHECK(hipEventCreate(&e0));
    CHECK(hipEventCreate(&e1));
    struct Mode {
        const char *name;
        void (*kern)(const u16x8 *, float *, int);
        double flop_per_iter;   // per wave
        double peak;
    } modes[4] = {
        {"v_mfma_f32_32x32x16_bf16", mfma_loop<0>, 8.0 * 2 * 32 * 32 * 16, 2516.6},
        {"v_mfma_f32_16x16x32_bf16", mfma_loop<1>, 32.0 * 2 * 16 * 16 * 32, 2516.6},
        {"v_mfma_f32_32x32x2_f32", mfma_loop<2>, 8.0 * 2 * 32 * 32 * 2, 157.3},
        {"v_mfma_f32_16x16x4_f32", mfma_loop<3>, 32.0 * 2 * 16 * 16 * 4, 157.3},
    };
    printf("operands %s, %d workgroups of 4 waves, %d iterations\n", zeros ? "all zero" : "uniform [-1,1)",
           wgs, iters);
    for (const Mode &m : modes) {
        const int it = m.peak < 1000 ? iters / 8 * 4 : iters;   // fp32: 512 or 1024 MFMA cycles per iteration
        hipLaunchKernelGGL(m.kern, dim3(wgs), dim3(256), 0, 0, din, dout, it);   // warm-up
        CHECK(hipDeviceSynchronize());
        std::vector<double> tf;
        for (int rep = 0; rep < 5; ++rep) {
            CHECK(hipEventRecord(e0));
            hipLaunchKernelGGL(m.kern, dim3(wgs), dim3(256), 0, 0, din, dout, it);
            CHECK(hipEventRecord(e1));
            CHECK(hipEventSynchronize(e1));
            float ms;
            CHECK(hipEventElapsedTime(&ms, e0, e1));
            tf.push_back(m.flop_per_iter * it * wgs * 4.0 / ms / 1e9);
        }
        std::sort(tf.begin(), tf.end());
        printf("%-26s %8.1f TFLOP/s  %.3f of %.1f\n", m.name, tf[2], tf[2] / m.peak, m.peak);
    }
    CHECK(hipGetLastError());
    CHECK(hipFree(din));
    CHECK(hipFree(dout));
    return 0;
}
