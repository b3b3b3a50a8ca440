// roofline_probe.hip -- attainable ceilings of the two bounds the lookup kernels are rated against.
//
// A standalone executable (built beside liblacache.so) that prints one JSON line:
//   mfma_random_tflops    sustained bf16 matrix-core throughput on random bf16 operands (the data the stage-1
//                         GEMM multiplies): the better of the two forms below;
//   mfma_random_32x32x16_tflops, mfma_random_16x16x32_tflops  each form alone (v_mfma_f32_32x32x16_bf16, the
//                         form the GEMM uses, and v_mfma_f32_16x16x32_bf16);
//   mfma_constant_tflops  the 32x32x16 loop with constant operands;
//   hbm_read_gbs          best of several passes of three streaming reads of a 4 GiB buffer (grid-stride,
//                         contiguous per-wave runs, and the runs with non-temporal loads);
//   hbm_read_plain_gbs    the best of the two with plain loads.
// MFMA power depends on the operand bits, so the sustained clock, and with it the matrix-core rate, is lower
// for random data than for constant data; the datasheet peak assumes the maximum clock.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <cstdio>
#include <cstdlib>
#include <vector>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kTab = 4096;  // u32x4 entries of the operand table

__device__ inline f32x16 mfma(u32x4 a, u32x4 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                   0, 0, 0);
}

// 8 independent accumulators per wave, 16 MFMAs per iteration.  RANDOM: the operands are 8 registers per
// lane loaded from a table of random bf16 pairs and rotated between the MFMAs; else constant operands.
template <bool RANDOM>
__global__ __launch_bounds__(512) void k_mfma(int iters, const u32x4* __restrict__ tab, float* __restrict__ out) {
    const int lane = threadIdx.x & 63;
    u32x4 r[8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
        r[i] = RANDOM ? tab[(i * 64 + lane + (int)blockIdx.x * 7) & (kTab - 1)] : u32x4{1u, 2u, 3u, 4u};
    f32x16 acc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = f32x16{};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] = mfma(r[i], r[(i + 3) & 7], acc[i]);
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] = mfma(r[(i + 5) & 7], r[(i + 1) & 7], acc[i]);
    }
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) s += acc[i][lane & 15];
    out[blockIdx.x * 512 + threadIdx.x] = s;  // keeps every MFMA live
}

// The same work as k_mfma<true> (random operands) in v_mfma_f32_16x16x32_bf16: half the FLOPs per
// instruction, so 16 independent accumulators and 32 MFMAs per iteration.
__global__ __launch_bounds__(512) void k_mfma16(int iters, const u32x4* __restrict__ tab, float* __restrict__ out) {
    const int lane = threadIdx.x & 63;
    u32x4 r[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = tab[(i * 64 + lane + (int)blockIdx.x * 7) & (kTab - 1)];
    f32x4 acc[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[i] = f32x4{};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int i = 0; i < 16; ++i)
            acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, r[i & 7]),
                                                             __builtin_bit_cast(bf16x8, r[(i + 3) & 7]), acc[i], 0, 0, 0);
#pragma unroll
        for (int i = 0; i < 16; ++i)
            acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, r[(i + 5) & 7]),
                                                             __builtin_bit_cast(bf16x8, r[(i + 1) & 7]), acc[i], 0, 0, 0);
    }
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) s += acc[i][lane & 3];
    out[blockIdx.x * 512 + threadIdx.x] = s;  // keeps every MFMA live
}

// Grid-stride streaming read of n 16-byte words; one word per thread is written so the loads stay live.
__global__ __launch_bounds__(256) void k_read(const u32x4* __restrict__ src, int64_t n, u32x4* __restrict__ out) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    u32x4 x = {0u, 0u, 0u, 0u};
    for (; i + 3 * stride < n; i += 4 * stride) {
        const u32x4 a = src[i], b = src[i + stride], c = src[i + 2 * stride], d = src[i + 3 * stride];
        x ^= a ^ b ^ c ^ d;
    }
    for (; i < n; i += stride) x ^= src[i];
    out[(int64_t)blockIdx.x * blockDim.x + threadIdx.x] = x;
}

// Contiguous per-wave runs: wave w of the grid reads words [w * per_wave, (w + 1) * per_wave) as 1 KiB
// coalesced wave loads, eight in flight (per_wave is a multiple of 512 words).  NT: non-temporal loads (the
// data is not kept in the caches), as the streaming stage-1 kernel reads its keys.
template <bool NT>
__global__ __launch_bounds__(1024) void k_read_runs(const u32x4* __restrict__ src, int64_t per_wave,
                                                    u32x4* __restrict__ out) {
    const int lane = threadIdx.x & 63;
    const int64_t w = (int64_t)blockIdx.x * (blockDim.x / 64) + (threadIdx.x >> 6);
    const u32x4* p = src + w * per_wave + lane;
    u32x4 x = {0u, 0u, 0u, 0u};
    for (int64_t j = 0; j < per_wave; j += 512) {
        u32x4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = NT ? __builtin_nontemporal_load(p + j + u * 64) : p[j + u * 64];
#pragma unroll
        for (int u = 0; u < 8; ++u) x ^= v[u];
    }
    out[(int64_t)blockIdx.x * blockDim.x + threadIdx.x] = x;
}

#define CK(x)                                                                              \
    do {                                                                                   \
        hipError_t e_ = (x);                                                               \
        if (e_ != hipSuccess) {                                                            \
            fprintf(stderr, "roofline_probe: %s failed: %s\n", #x, hipGetErrorString(e_)); \
            return 1;                                                                      \
        }                                                                                  \
    } while (0)

}  // namespace

int main() {
    hipDeviceProp_t prop;
    CK(hipGetDeviceProperties(&prop, 0));
    const int ncu = prop.multiProcessorCount;

    // random bf16 pairs in [-2^-4, 2^-4): random sign, exponent 119..126, random mantissa
    std::vector<uint32_t> h(kTab * 4);
    srand(12345);
    for (auto& x : h) {
        const uint32_t lo = (uint32_t)(((rand() & 1) << 15) | ((119 + rand() % 8) << 7) | (rand() & 127));
        const uint32_t hi = (uint32_t)(((rand() & 1) << 15) | ((119 + rand() % 8) << 7) | (rand() & 127));
        x = lo | (hi << 16);
    }
    u32x4* tab = nullptr;
    float* out = nullptr;
    const int grid = 2 * ncu;
    CK(hipMalloc(&tab, h.size() * 4));
    CK(hipMalloc(&out, (size_t)grid * 512 * sizeof(float)));
    CK(hipMemcpy(tab, h.data(), h.size() * 4, hipMemcpyHostToDevice));
    hipEvent_t e0, e1;
    CK(hipEventCreate(&e0));
    CK(hipEventCreate(&e1));

    const int iters = 60000;  // ~50-75 ms per launch: long enough for the clock to settle
    double tf[3];  // random 32x32x16, constant 32x32x16, random 16x16x32: the same FLOPs each
    for (int v = 0; v < 3; ++v) {
        float ms = 0.f;
        CK(hipEventRecord(e0));
        if (v == 0)
            k_mfma<true><<<dim3(grid), dim3(512)>>>(iters, tab, out);
        else if (v == 1)
            k_mfma<false><<<dim3(grid), dim3(512)>>>(iters, tab, out);
        else
            k_mfma16<<<dim3(grid), dim3(512)>>>(iters, tab, out);
        CK(hipGetLastError());
        CK(hipEventRecord(e1));
        CK(hipEventSynchronize(e1));
        CK(hipEventElapsedTime(&ms, e0, e1));
        const double flop = 2.0 * 32 * 32 * 16 * 16.0 * iters * grid * 8;
        tf[v] = flop / (ms * 1e-3) / 1e12;
    }

    const int64_t bytes = (int64_t)4 << 30;
    const int64_t n = bytes / 16;
    u32x4 *src = nullptr, *sink = nullptr;
    const int rgrid = 8 * ncu * 4;
    CK(hipMalloc(&src, (size_t)bytes));
    CK(hipMalloc(&sink, (size_t)(rgrid * 256 > 2 * ncu * 1024 ? rgrid * 256 : 2 * ncu * 1024) * 16));
    CK(hipMemset(src, 0x3C, (size_t)bytes));
    // runs: 2 workgroups of 16 waves per CU; words per wave rounded down to whole 8 KiB steps
    const int run_grid = 2 * ncu, run_waves = run_grid * 16;
    const int64_t per_wave = n / run_waves / 512 * 512;
    double best_gbs = 0.0, best_plain = 0.0;
    for (int rep = 0; rep < 18; ++rep) {
        float ms = 0.f;
        const int kind = rep / 6;  // 0 grid-stride, 1 runs, 2 runs with non-temporal loads
        CK(hipEventRecord(e0));
        if (kind == 0)
            k_read<<<dim3(rgrid), dim3(256)>>>(src, n, sink);
        else if (kind == 1)
            k_read_runs<false><<<dim3(run_grid), dim3(1024)>>>(src, per_wave, sink);
        else
            k_read_runs<true><<<dim3(run_grid), dim3(1024)>>>(src, per_wave, sink);
        CK(hipGetLastError());
        CK(hipEventRecord(e1));
        CK(hipEventSynchronize(e1));
        CK(hipEventElapsedTime(&ms, e0, e1));
        const double moved = kind ? (double)per_wave * run_waves * 16 : (double)bytes;
        const double gbs = moved / (ms * 1e-3) / 1e9;
        if (rep % 6 == 0) continue;  // the first pass of each kind warms up
        if (gbs > best_gbs) best_gbs = gbs;
        if (kind < 2 && gbs > best_plain) best_plain = gbs;
    }
    printf("{\"mfma_random_tflops\": %.1f, \"mfma_random_32x32x16_tflops\": %.1f, "
           "\"mfma_random_16x16x32_tflops\": %.1f, \"mfma_constant_tflops\": %.1f, \"hbm_read_gbs\": %.1f, "
           "\"hbm_read_plain_gbs\": %.1f, \"cus\": %d}\n",
           tf[0] > tf[2] ? tf[0] : tf[2], tf[0], tf[2], tf[1], best_gbs, best_plain, ncu);
    CK(hipFree(tab));
    CK(hipFree(out));
    CK(hipFree(src));
    CK(hipFree(sink));
    return 0;
}
