// k_calibrate.hip -- threshold calibration from benign pairs: pair cosines, then an exact percentile.
//
// Appendix A.2 sets each threshold to a percentile of the cosine similarities
// of benign pairs, capped from above (tau_c = min(0.80, P5) over paraphrase
// query pairs, tau_a = min(0.70, P10) over their response prefixes).  The pair
// cosine is the one the lookup computes: both vectors normalised in double and
// rounded once to bfloat16 (the same routine as every stored vector), their
// products accumulated in float32, clamped to [-1, 1].  The percentile is
// linear between the closest ranks, h = (n - 1) p / 100 (the paper does not
// say; this is numpy's default), from the two order statistics floor(h) and
// floor(h) + 1, which an exact radix select finds without sorting: three
// histogram passes over the orderable 32-bit keys of the similarities (11,
// 11 and 10 bits), each followed by a one-workgroup scan that fixes those
// bits of both ranks' keys.
#include <mutex>

#include "common.hpp"
#include "launch.hpp"

namespace lacache {

namespace {

constexpr int kBins = 2048;  // histogram bins of the widest pass (11 bits)
constexpr int kPasses = 3;
__constant__ const int kShift[kPasses] = {21, 10, 0};
__constant__ const int kBits[kPasses] = {11, 11, 10};

}  // namespace

// One wave per pair (grid-stride over the pairs): normalise a[j] and b[j] as stored vectors are, and dot the
// rounded values in column order per lane, then across the wave.  The rounded values are used as float32
// directly (a bfloat16 is a float32 with zero low bits); products of two are exact.  NC > 0: d <= 512 NC and each lane keeps its 8 NC columns of
// both rows in registers, read once; the norms are summed in the order row_norm uses, so the rounded values
// are those of the stored vectors.  NC = 0: any d, the rows read once for the norms and once for the dot.
template <int NC>
__device__ __forceinline__ void pair_cosine(const void* __restrict__ a, const void* __restrict__ b, int dtype, int d,
                                   int64_t j, float* __restrict__ sims) {
    const int lane = threadIdx.x & 63;
    const size_t esz = dtype == 0 ? 4 : 2;
    const char* ra = (const char*)a + j * d * esz;
    const char* rb = (const char*)b + j * d * esz;
    float acc = 0.0f;
    if constexpr (NC > 0) {
        float xa[NC][8], xb[NC][8];
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            load8f(ra, dtype, d, lane * 8 + 512 * c, xa[c]);
            load8f(rb, dtype, d, lane * 8 + 512 * c, xb[c]);
        }
        double sa = 0.0, sb = 0.0;
#pragma unroll
        for (int c = 0; c < NC; ++c)
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                sa += (double)xa[c][e] * (double)xa[c][e];
                sb += (double)xb[c][e] * (double)xb[c][e];
            }
        const double na = __builtin_sqrt(wave_sum_f64(sa)), nb = __builtin_sqrt(wave_sum_f64(sb));
        if (na != 0.0 && nb != 0.0) {  // a zero vector normalises to zero and scores 0
            const float rna = quotient_rcp_f32(na), rnb = quotient_rcp_f32(nb);
#pragma unroll
            for (int c = 0; c < NC; ++c)
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    if (lane * 8 + 512 * c + e >= d) continue;
                    acc += bf16_rne_quotient_f32(xa[c][e], na, rna) * bf16_rne_quotient_f32(xb[c][e], nb, rnb);
                }
        }
    } else {
        const double na = row_norm(ra, dtype, d, true, lane);
        const double nb = row_norm(rb, dtype, d, true, lane);
        if (na != 0.0 && nb != 0.0) {
            const float rna = quotient_rcp_f32(na), rnb = quotient_rcp_f32(nb);
            for (int j0 = lane * 8; j0 < d; j0 += 512) {
                float va[8], vb[8];
                load8f(ra, dtype, d, j0, va);
                load8f(rb, dtype, d, j0, vb);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    if (j0 + e >= d) continue;
                    acc += bf16_rne_quotient_f32(va[e], na, rna) * bf16_rne_quotient_f32(vb[e], nb, rnb);
                }
            }
        }
    }
    acc = wave_sum_f32(acc);
    if (lane == 0) sims[j] = fminf(fmaxf(acc, -1.0f), 1.0f);
}

// LOOP: grid-stride over the pairs, for more pairs than one grid holds; else one pair per wave (the loop's
// carried state costs registers, and with them occupancy, on this latency-bound kernel).
template <int NC, bool LOOP>
__global__ __launch_bounds__(256) void k_pair_cosine(const void* __restrict__ a, const void* __restrict__ b,
                                                     int dtype, int d, int64_t n, float* __restrict__ sims) {
    const int64_t j0 = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if constexpr (LOOP) {
        for (int64_t j = j0; j < n; j += (int64_t)gridDim.x * 4) pair_cosine<NC>(a, b, dtype, d, j, sims);
    } else {
        if (j0 >= n) return;
        pair_cosine<NC>(a, b, dtype, d, j0, sims);
    }
}

// state[0..1]: the key bits found so far for rank 0 / rank 1; state[2..3]: the ranks still to skip inside
// the current prefix.  hist: [2][kBins] counts.
__global__ __launch_bounds__(256) void k_select_init(uint32_t* __restrict__ state, uint32_t* __restrict__ hist,
                                                     uint32_t r0, uint32_t r1) {
    for (int i = threadIdx.x; i < 2 * kBins; i += blockDim.x) hist[i] = 0u;
    if (threadIdx.x == 0) {
        state[0] = 0u;
        state[1] = 0u;
        state[2] = r0;
        state[3] = r1;
    }
}

// Histogram of bits [shift, shift + bits) of the keys whose higher bits equal each rank's prefix.
__global__ __launch_bounds__(256) void k_select_hist(const float* __restrict__ sims, int64_t n, int pass,
                                                     const uint32_t* __restrict__ state,
                                                     uint32_t* __restrict__ hist) {
    __shared__ uint32_t h[2 * kBins];
    for (int i = threadIdx.x; i < 2 * kBins; i += blockDim.x) h[i] = 0u;
    __syncthreads();
    const int shift = kShift[pass], bits = kBits[pass];
    const int hi = shift + bits;  // bits above hi are fixed by the earlier passes
    const uint32_t p0 = state[0], p1 = state[1];
    const uint32_t mask = (uint32_t)((1u << bits) - 1u);
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        const uint32_t key = order_f32(sims[i]);
        const uint32_t bin = (key >> shift) & mask;
        const bool m0 = hi >= 32 || (key >> hi) == (p0 >> hi);
        const bool m1 = hi >= 32 || (key >> hi) == (p1 >> hi);
        if (m0) atomicAdd(&h[bin], 1u);
        if (m1) atomicAdd(&h[kBins + bin], 1u);
    }
    __syncthreads();
    for (int i = threadIdx.x; i < 2 * kBins; i += blockDim.x)
        if (h[i] != 0u) atomicAdd(&hist[i], h[i]);
}

// One workgroup: for each rank, the bin holding it (counts scanned in bin order) fixes this pass's bits of its
// key; the counts of the bins before it are skipped.  Each thread takes nb / 256 consecutive bins, a block-wide
// exclusive scan gives the count before them, and the one thread whose bins hold the rank walks them.  The
// histogram is cleared for the next pass.
__global__ __launch_bounds__(256) void k_select_scan(int pass, uint32_t* __restrict__ state,
                                                     uint32_t* __restrict__ hist) {
    constexpr int kPer = kBins / 256;  // bins per thread in the widest pass
    __shared__ uint32_t wsum[2][4];
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int shift = kShift[pass], per = (1 << kBits[pass]) / 256;
    const uint32_t rank[2] = {state[2], state[3]};
    uint32_t cnt[2][kPer], tot[2] = {0u, 0u};
#pragma unroll
    for (int k = 0; k < 2; ++k)
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            cnt[k][i] = i < per ? hist[k * kBins + tid * per + i] : 0u;
            tot[k] += cnt[k][i];
        }
    uint32_t incl[2];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        incl[k] = tot[k];
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const uint32_t t = __shfl_up(incl[k], o, kWave);
            if (lane >= o) incl[k] += t;
        }
        if (lane == 63) wsum[k][wid] = incl[k];
    }
    __syncthreads();  // every thread has read the ranks before any is rewritten
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        uint32_t run = incl[k] - tot[k];
        for (int w = 0; w < wid; ++w) run += wsum[k][w];
        if (run <= rank[k] && rank[k] < run + tot[k]) {
            bool found = false;
#pragma unroll
            for (int i = 0; i < kPer; ++i) {
                if (found || i >= per) continue;
                if (rank[k] < run + cnt[k][i]) {
                    state[k] |= (uint32_t)(tid * per + i) << shift;
                    state[2 + k] = rank[k] - run;
                    found = true;
                } else {
                    run += cnt[k][i];
                }
            }
        }
    }
#pragma unroll
    for (int k = 0; k < 2; ++k)
        for (int i = 0; i < per; ++i) hist[k * kBins + tid * per + i] = 0u;
}

// P = x_lo + (h - lo) (x_hi - x_lo) in double from the two order statistics; out[0] = P, out[1] = min(cap, P).
__global__ void k_select_final(const uint32_t* __restrict__ state, double frac, float cap, float* __restrict__ out) {
    if (threadIdx.x != 0) return;
    const double lo = (double)unorder_f32(state[0]);
    const double hi = (double)unorder_f32(state[1]);
    const double P = lo + frac * (hi - lo);
    out[0] = (float)P;
    out[1] = (float)fmin((double)cap, P);
}

// Scratch of the allocation-free calibration entry point (lacache_calibrate_noalloc): the selection's state
// and histograms, kCalibScratchWords words.  Every GPU the library runs on holds its own copy for the life of
// the process; all such calls on one GPU share it (k_select_init clears it at the start of each call, so calls
// ordered on one stream are independent; calls that overlap on one GPU race).
static __device__ __align__(256) uint32_t scratch[kCalibScratchWords];

hipError_t calibrate_static_scratch(uint32_t** out) {
    // the array's device address, taken once per device with that device current (the host-side name of the
    // array is no device address); devices past the cache's range look it up on every call
    static std::mutex mu;
    static uint32_t* addr[64] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    std::lock_guard<std::mutex> lock(mu);
    if (dev >= 0 && dev < 64 && addr[dev]) {
        *out = addr[dev];
        return hipSuccess;
    }
    uint32_t* p = nullptr;
    e = hipGetSymbolAddress((void**)&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (dev >= 0 && dev < 64) addr[dev] = p;
    *out = p;
    return hipSuccess;
}

hipError_t launch_calibrate(const void* a, const void* b, int dtype, int d, int64_t n, float percentile, float cap,
                            float* sims, float* tau, uint32_t* scratch, int num_cu, hipStream_t s) {
    if (n <= 0) return hipErrorInvalidValue;
    const double h = (double)(n - 1) * ((double)percentile / 100.0);
    int64_t lo = (int64_t)h;  // h >= 0: truncation is floor
    if (lo > n - 1) lo = n - 1;
    const int64_t hi = lo + 1 < n ? lo + 1 : lo;
    const double frac = lo == hi ? 0.0 : h - (double)lo;
    uint32_t* state = scratch;
    uint32_t* hist = scratch + 64;
    const dim3 pc_grid((unsigned)grid_blocks((n + 3) / 4)), pc_block(256);
    if ((n + 3) / 4 > kMaxGridBlocks) {
        if (d <= 512)
            k_pair_cosine<1, true><<<pc_grid, pc_block, 0, s>>>(a, b, dtype, d, n, sims);
        else if (d <= 1024)
            k_pair_cosine<2, true><<<pc_grid, pc_block, 0, s>>>(a, b, dtype, d, n, sims);
        else if (d <= 2048)
            k_pair_cosine<4, true><<<pc_grid, pc_block, 0, s>>>(a, b, dtype, d, n, sims);
        else
            k_pair_cosine<0, true><<<pc_grid, pc_block, 0, s>>>(a, b, dtype, d, n, sims);
    } else {
        if (d <= 512)
            k_pair_cosine<1, false><<<pc_grid, pc_block, 0, s>>>(a, b, dtype, d, n, sims);
        else if (d <= 1024)
            k_pair_cosine<2, false><<<pc_grid, pc_block, 0, s>>>(a, b, dtype, d, n, sims);
        else if (d <= 2048)
            k_pair_cosine<4, false><<<pc_grid, pc_block, 0, s>>>(a, b, dtype, d, n, sims);
        else
            k_pair_cosine<0, false><<<pc_grid, pc_block, 0, s>>>(a, b, dtype, d, n, sims);
    }
    k_select_init<<<dim3(1), dim3(256), 0, s>>>(state, hist, (uint32_t)lo, (uint32_t)hi);
    // at least 16 similarities per thread: each workgroup adds its non-zero bins to the global histogram
    int64_t blocks = (n + 256 * 16 - 1) / (256 * 16);
    if (blocks > num_cu) blocks = num_cu;
    for (int pass = 0; pass < kPasses; ++pass) {
        k_select_hist<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(sims, n, pass, state, hist);
        k_select_scan<<<dim3(1), dim3(256), 0, s>>>(pass, state, hist);
    }
    k_select_final<<<dim3(1), dim3(64), 0, s>>>(state, frac, cap, tau);
    return hipGetLastError();
}

}  // namespace lacache
