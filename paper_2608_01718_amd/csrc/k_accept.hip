// k_accept.hip -- speculative-decoding acceptance: target probabilities of the draft tokens, leading run.
//
// After a miss or a rejected lookahead the k draft tokens of the draft model
// g are verified by the target model f in one forward pass (Section 4.3,
// speculative decoding): token t_j is accepted when P_f(t_j) >= P_g(t_j),
// starting from the first token, and f takes over at the first failure.
// P_f(t_j) is the softmax probability of t_j under f's logits at position j,
// so each (query, position) row of V logits is read once: a workgroup keeps a
// running (maximum, sum of exponentials relative to it) per thread over
// 16-byte chunks of the row, merges the pairs across the workgroup, and
// divides the token's exponential by the sum.  The kernel is bound by reading
// the logits, which it reads once, with non-temporal loads.  A second kernel finds, per query, the first rejected position
// with a wave ballot.
#include "common.hpp"
#include "launch.hpp"

namespace lacache {

namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 4;  // 16-byte chunks in flight per thread

// merge two (max, sum of exp(x - max)) pairs; -inf maxima carry an empty sum
__device__ inline void lse_merge(float& m, float& s, float m2, float s2) {
    const float M = fmaxf(m, m2);
    if (M == -__builtin_inff()) return;
    s = (m == -__builtin_inff() ? 0.0f : s * __expf(m - M)) + (m2 == -__builtin_inff() ? 0.0f : s2 * __expf(m2 - M));
    m = M;
}

// fold up to 8 logits into the running pair
__device__ inline void lse_add8(float& m, float& s, const float x[8]) {
    float cm = x[0];
#pragma unroll
    for (int e = 1; e < 8; ++e) cm = fmaxf(cm, x[e]);
    if (cm > m) {
        s = (m == -__builtin_inff()) ? 0.0f : s * __expf(m - cm);
        m = cm;
    }
    if (m == -__builtin_inff()) return;
#pragma unroll
    for (int e = 0; e < 8; ++e) s += __expf(x[e] - m);
}

// 8 logits from 16-byte aligned memory, by non-temporal loads (each logit is read once)
__device__ inline void load_chunk(const char* p, int dtype, float x[8]) {
    if (dtype == 0) {
        const u32x4 a = __builtin_nontemporal_load((const u32x4*)p), b = __builtin_nontemporal_load((const u32x4*)p + 1);
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            x[t] = __uint_as_float(a[t]);
            x[4 + t] = __uint_as_float(b[t]);
        }
    } else {
        const u32x4 a = __builtin_nontemporal_load((const u32x4*)p);
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            x[2 * t] = __uint_as_float(a[t] << 16);
            x[2 * t + 1] = __uint_as_float(a[t] & 0xFFFF0000u);
        }
    }
}

__device__ inline float load_one(const char* row, int dtype, int v) {
    return dtype == 0 ? ((const float*)row)[v] : bf16_to_f32(((const uint16_t*)row)[v]);
}

}  // namespace

// One workgroup per (query, position) row, grid-stride over the rows.
__global__ __launch_bounds__(kThreads) void k_token_prob(const void* __restrict__ logits, int dtype, int V,
                                                         const int32_t* __restrict__ tokens, int64_t rows,
                                                         float* __restrict__ p_target) {
    __shared__ float sm[kThreads / 64], ss[kThreads / 64];
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const size_t esz = dtype == 0 ? 4 : 2;
    for (int64_t row = blockIdx.x; row < rows; row += gridDim.x) {
        const char* r = (const char*)logits + row * (int64_t)V * esz;
        float m = -__builtin_inff(), s = 0.0f;
        int tail0 = 0;  // first element not covered by whole aligned chunks
        if (((uintptr_t)r & 15) == 0) {
            const int nchunks = V / 8;
            int c = tid;
            for (; c + (kUnroll - 1) * kThreads < nchunks; c += kUnroll * kThreads) {
                float x[kUnroll][8];
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) load_chunk(r + (size_t)(c + u * kThreads) * 8 * esz, dtype, x[u]);
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) lse_add8(m, s, x[u]);
            }
            for (; c < nchunks; c += kThreads) {
                float x[8];
                load_chunk(r + (size_t)c * 8 * esz, dtype, x);
                lse_add8(m, s, x);
            }
            tail0 = nchunks * 8;
        }
        for (int v = tail0 + tid; v < V; v += kThreads) {
            float x[8];
            x[0] = load_one(r, dtype, v);
#pragma unroll
            for (int e = 1; e < 8; ++e) x[e] = -__builtin_inff();
            lse_add8(m, s, x);
        }
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) {
            const float m2 = __shfl_xor(m, o, kWave), s2 = __shfl_xor(s, o, kWave);
            lse_merge(m, s, m2, s2);
        }
        if (lane == 0) {
            sm[wid] = m;
            ss[wid] = s;
        }
        __syncthreads();
        if (tid == 0) {
            for (int w = 1; w < kThreads / 64; ++w) lse_merge(m, s, sm[w], ss[w]);
            const int t = tokens[row];
            float p = 0.0f;
            if (t >= 0 && t < V) p = __expf(load_one(r, dtype, t) - m) / s;
            p_target[row] = p;
        }
        __syncthreads();  // sm / ss are rewritten by the next row
    }
}

// One wave per query: the accepted length is the first position whose target probability is below the
// draft's (k if none).
__global__ __launch_bounds__(256) void k_accept_len(const float* __restrict__ p_target,
                                                    const float* __restrict__ p_draft, int B, int k,
                                                    int32_t* __restrict__ accept_len) {
    const int lane = threadIdx.x & 63;
    for (int64_t b = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); b < B; b += (int64_t)gridDim.x * 4) {
        int len = k;
        for (int j0 = 0; j0 < k; j0 += 64) {
            const int j = j0 + lane;
            const bool reject = j < k && !(p_target[b * k + j] >= p_draft[b * k + j]);
            const uint64_t rej = __ballot(reject);
            if (rej != 0ull) {
                len = j0 + __ffsll((unsigned long long)rej) - 1;
                break;
            }
        }
        if (lane == 0) accept_len[b] = len;
    }
}

hipError_t launch_accept_length(const void* logits, int dtype, int V, const int32_t* tokens, const float* p_draft,
                                int B, int k, int32_t* accept_len, float* p_target, hipStream_t s) {
    const int64_t rows = (int64_t)B * k;
    if (rows <= 0) return hipSuccess;
    k_token_prob<<<dim3((unsigned)grid_blocks(rows)), dim3(kThreads), 0, s>>>(logits, dtype, V, tokens, rows,
                                                                              p_target);
    k_accept_len<<<dim3((unsigned)grid_blocks(((int64_t)B + 3) / 4)), dim3(256), 0, s>>>(p_target, p_draft, B, k,
                                                                                         accept_len);
    return hipGetLastError();
}

}  // namespace lacache
