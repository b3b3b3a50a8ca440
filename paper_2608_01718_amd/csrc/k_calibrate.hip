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
// 11 and 10 bits), each followed by a one-wave scan that fixes those bits of
// both ranks' keys.
#include "common.hpp"
#include "launch.hpp"

namespace lacache {

namespace {

constexpr int kBins = 2048;  // histogram bins of the widest pass (11 bits)
constexpr int kPasses = 3;
__constant__ const int kShift[kPasses] = {21, 10, 0};
__constant__ const int kBits[kPasses] = {11, 11, 10};

}  // namespace

// One wave per pair: normalise a[j] and b[j] as stored vectors are, and dot the rounded values.
__global__ __launch_bounds__(256) void k_pair_cosine(const void* __restrict__ a, const void* __restrict__ b,
                                                     int dtype, int d, int64_t n, float* __restrict__ sims) {
    const int lane = threadIdx.x & 63;
    const int64_t j = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (j >= n) return;
    const size_t esz = dtype == 0 ? 4 : 2;
    const char* ra = (const char*)a + j * d * esz;
    const char* rb = (const char*)b + j * d * esz;
    const double na = row_norm(ra, dtype, d, true, lane);
    const double nb = row_norm(rb, dtype, d, true, lane);
    float acc = 0.0f;
    for (int j0 = lane * 8; j0 < d; j0 += 512)
        acc = dot8_bf16(quantise8(ra, dtype, d, j0, na, true), quantise8(rb, dtype, d, j0, nb, true), acc);
    acc = wave_sum_f32(acc);
    if (lane == 0) sims[j] = fminf(fmaxf(acc, -1.0f), 1.0f);
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

// One wave: for each rank, the bin holding it (counts scanned in bin order) fixes this pass's bits of its
// key; the counts of the bins before it are skipped.  The histogram is cleared for the next pass.
__global__ __launch_bounds__(64) void k_select_scan(int pass, uint32_t* __restrict__ state,
                                                    uint32_t* __restrict__ hist) {
    const int lane = threadIdx.x;
    const int shift = kShift[pass], nb = 1 << kBits[pass];
    for (int k = 0; k < 2; ++k) {
        const uint32_t rank = state[2 + k];
        uint32_t before = 0u;  // count of the bins already passed
        int bin = -1;
        uint32_t skip = 0u;
        for (int c = 0; c < nb && bin < 0; c += 64) {
            const uint32_t v = hist[k * kBins + c + lane];
            uint32_t incl = v;
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const uint32_t t = __shfl_up(incl, o, kWave);
                if (lane >= o) incl += t;
            }
            const uint32_t excl = incl - v;
            const bool here = before + excl <= rank && rank < before + incl;
            const uint64_t hit = __ballot(here);
            if (hit != 0ull) {
                const int l = __ffsll((unsigned long long)hit) - 1;
                bin = c + l;
                skip = before + __shfl(excl, l, kWave);
            }
            before += __shfl(incl, 63, kWave);
        }
        if (lane == 0 && bin >= 0) {
            state[k] |= (uint32_t)bin << shift;
            state[2 + k] = rank - skip;
        }
    }
    for (int i = lane; i < 2 * kBins; i += 64) hist[i] = 0u;
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
    k_pair_cosine<<<dim3((unsigned)((n + 3) / 4)), dim3(256), 0, s>>>(a, b, dtype, d, n, sims);
    k_select_init<<<dim3(1), dim3(256), 0, s>>>(state, hist, (uint32_t)lo, (uint32_t)hi);
    int64_t blocks = (n + 255) / 256;
    if (blocks > 4 * num_cu) blocks = 4 * num_cu;
    for (int pass = 0; pass < kPasses; ++pass) {
        k_select_hist<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(sims, n, pass, state, hist);
        k_select_scan<<<dim3(1), dim3(64), 0, s>>>(pass, state, hist);
    }
    k_select_final<<<dim3(1), dim3(64), 0, s>>>(state, frac, cap, tau);
    return hipGetLastError();
}

}  // namespace lacache
