// k_lsh.hip -- stage 1 through a locality-sensitive index: random-hyperplane signatures, a Hamming-radius
// candidate scan, and exact re-ranking of the candidates.
//
// Section 3 models the cache key as an LSH h(z) of the embedding with the
// gapped collision property of Eq. (1), and Algorithm 1 searches the cache
// with it.  For cosine distance the hash family is random hyperplanes: bit i
// of h(z) is 1 when r_i . z >= 0, so vectors at angle theta agree on a bit
// with probability 1 - theta / pi.  Signatures of the stored (normalised,
// bfloat16-rounded) keys are kept beside the store; a query's candidates are
// the entries within a Hamming radius of its signature (radius 0 is equality
// of hash keys), found by one pass over the signatures (bits / 8 bytes per
// entry instead of the key's d * 2), and re-ranked by their exact similarity.
#include "verify.hpp"

namespace lacache {

namespace {
constexpr int kScanQueries = 1024;  // query signatures held in LDS per scan launch
}

// Copy a row-major [rows][d] bfloat16 matrix into the tiled layout with d_pad columns (zero padded), as is.
__global__ __launch_bounds__(256) void k_tile_rows(const uint16_t* __restrict__ src, int rows, int d, int d_pad,
                                                   uint16_t* __restrict__ dst) {
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (t >= (int64_t)rows * d_pad) return;
    const int r = (int)(t / d_pad), c = (int)(t - (int64_t)r * d_pad);
    dst[tiled_offset(r, c, d_pad >> 5)] = c < d ? src[(int64_t)r * d + c] : (uint16_t)0;
}

// One wave per (16-row group of a tiled matrix, run of `wpw` signature words): the projections of its rows on
// the hyperplanes of those words (16 at a time, v_mfma_f32_16x16x32_bf16 with the rows as the row operand; the
// two 16-hyperplane halves of a word accumulate side by side), packed into sign bits.  Lane l holds, for
// hyperplane 16 hg + l % 16, the rows 4 (l / 16) + j (j = 0..3); a ballot per j gathers the 16 bits of each
// row.  Rows outside [row0, row0 + n) are not written.  Grid-stride over the waves.
__global__ __launch_bounds__(256) void k_simhash(const u32x4* __restrict__ rows_tiled, int kc, int64_t row0,
                                                 int64_t n, const u32x4* __restrict__ hp_tiled, int bits, int wpw,
                                                 uint32_t* __restrict__ sig) {
    const int lane = threadIdx.x & 63;
    const int words = bits >> 5;
    const int chunks = words / wpw;  // word runs per group
    // grid-stride over the waves; groups grow with the wave index, so the first one past the rows ends the loop
    for (int64_t wave = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);; wave += (int64_t)gridDim.x * 4) {
        const int64_t g = (row0 >> 4) + wave / chunks;  // 16-row group
        const int w0 = (int)(wave % chunks) * wpw;
        if (g * 16 >= row0 + n) break;
        const u32x4* a = rows_tiled + g * kc * 64 + lane;
        for (int w = w0; w < w0 + wpw; ++w) {
            f32x4 lo = f32x4{0.f, 0.f, 0.f, 0.f}, hi = f32x4{0.f, 0.f, 0.f, 0.f};
            const u32x4* b0 = hp_tiled + (int64_t)(2 * w) * kc * 64 + lane;
            const u32x4* b1 = b0 + (int64_t)kc * 64;
            for (int c = 0; c < kc; c += 4) {  // kc is a multiple of 4: twelve loads in flight per step
                u32x4 x[4], y0[4], y1[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    x[u] = a[(c + u) * 64];
                    y0[u] = b0[(c + u) * 64];
                    y1[u] = b1[(c + u) * 64];
                }
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    lo = mfma16x16x32(x[u], y0[u], lo);
                    hi = mfma16x16x32(x[u], y1[u], hi);
                }
            }
            uint32_t word = 0u;
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                const f32x4 acc = half ? hi : lo;
                uint64_t m[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) m[j] = __ballot(acc[j] >= 0.0f);
                // lane l < 16 owns row 4 (l / 4) + l % 4 = l of the group: its bits sit in m[l % 4] at 16 (l / 4)
                const uint64_t mine =
                    (lane & 3) == 0 ? m[0] : (lane & 3) == 1 ? m[1] : (lane & 3) == 2 ? m[2] : m[3];
                word |= ((uint32_t)(mine >> (16 * ((lane >> 2) & 3))) & 0xFFFFu) << (16 * half);
            }
            const int64_t row = g * 16 + lane;
            if (lane < 16 && row >= row0 && row < row0 + n) sig[row * words + w] = word;
        }
    }
}

// Signature word of 16 rounded queries against hyperplanes b0 (bits 0..15 of the word) and b1 (16..31): S
// column chunks c0 .. c0+S-1, every operand load of the batch issued before its first MFMA.  xat(c) gives the
// lane's piece of query chunk c.
template <int S, class X>
__device__ __forceinline__ void simhash_batch(X xat, const u32x4* __restrict__ b0, const u32x4* __restrict__ b1,
                                              int c0, f32x4& lo, f32x4& hi) {
    u32x4 x[S], y0[S], y1[S];
#pragma unroll
    for (int u = 0; u < S; ++u) {
        x[u] = xat(c0 + u);
        y0[u] = b0[(c0 + u) * 64];
        y1[u] = b1[(c0 + u) * 64];
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < S; ++u) {
        lo = mfma16x16x32(x[u], y0[u], lo);
        hi = mfma16x16x32(x[u], y1[u], hi);
    }
}

// Query preparation for the LSH lookup, one workgroup of 16 waves per 16 queries: wave w normalises and
// rounds query 16 g + w into the tiled scratch exactly as stored vectors are (zeros past the batch) and
// clears its candidate count; after the barrier wave w < bits / 32 computes signature word w of the 16
// queries with the MFMA sequence of k_simhash (so a query equal to a stored key gets its signature).
// NC > 0 (d_pad <= 512 NC): the query row is read once into registers, and the rounded queries are also
// kept in LDS (the tiled chunk layout), where the signature MFMAs read them; the hyperplane chunks are
// loaded eight at a time.  NC = 0: any d, the rows read twice and the queries read back from the scratch.
template <int NC>
__global__ __launch_bounds__(1024) void k_lsh_prep(const void* __restrict__ queries, int dtype, int nb, int d,
                                                   int d_pad, uint16_t* __restrict__ qt,
                                                   const u32x4* __restrict__ hp_tiled, int bits,
                                                   uint32_t* __restrict__ sigq, uint32_t* __restrict__ cnt) {
    __shared__ u32x4 qs[NC > 0 ? 16 * 64 * NC : 1];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int g = blockIdx.x;
    const int r = g * 16 + wv;
    const bool live = r < nb;
    const int kc = d_pad >> 5;
    const char* src = (const char*)queries + (live ? (int64_t)r * d * (dtype == 0 ? 4 : 2) : 0);
    if constexpr (NC > 0) {
        float x[NC][8];
        row_to_regs<NC>(src, dtype, d, live, lane, x);
        const double n = regs_norm<NC>(x);
        const float rnf = quotient_rcp_f32(n);
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const int j0 = lane * 8 + 512 * c, J = j0 >> 3;
            if (j0 < d_pad) {
                const u32x4 w = regs_quantise8(x[c], j0, d, n, rnf, live);
                *(u32x4*)(qt + tiled_offset(r, j0, kc)) = w;
                qs[(J >> 2) * 64 + (J & 3) * 16 + wv] = w;
            }
        }
    } else {
        normalise_row(src, dtype, d, d_pad, live, lane,
                      [&](int j0, u32x4 w) { *(u32x4*)(qt + tiled_offset(r, j0, kc)) = w; });
    }
    if (live && lane == 0) cnt[r] = 0u;
    __syncthreads();
    const int words = bits >> 5;
    if (wv >= words) return;
    const u32x4* a = (const u32x4*)qt + (int64_t)g * kc * 64 + lane;
    const u32x4* b0 = hp_tiled + (int64_t)(2 * wv) * kc * 64 + lane;
    const u32x4* b1 = b0 + (int64_t)kc * 64;
    f32x4 lo = f32x4{0.f, 0.f, 0.f, 0.f}, hi = f32x4{0.f, 0.f, 0.f, 0.f};
    auto xat = [&](int c) { return NC > 0 ? qs[c * 64 + lane] : a[c * 64]; };
    int c = 0;
    for (; c + 8 <= kc; c += 8) simhash_batch<8>(xat, b0, b1, c, lo, hi);
    if (c < kc) simhash_batch<4>(xat, b0, b1, c, lo, hi);  // kc is a multiple of 4
    uint32_t word = 0u;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
        const f32x4 acc = half ? hi : lo;
        uint64_t m[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) m[j] = __ballot(acc[j] >= 0.0f);
        const uint64_t mine = (lane & 3) == 0 ? m[0] : (lane & 3) == 1 ? m[1] : (lane & 3) == 2 ? m[2] : m[3];
        word |= ((uint32_t)(mine >> (16 * ((lane >> 2) & 3))) & 0xFFFFu) << (16 * half);
    }
    const int row = g * 16 + lane;
    if (lane < 16 && row < nb) sigq[(int64_t)row * words + wv] = word;
}

// Candidates of queries q0 .. q0+nq-1: every entry whose signature differs from the query's in at most `radius`
// bits is appended to the query's list (at most max_cand kept; cnt counts them all).  Each thread takes
// kScanKeys entries at a time (the query signatures, in LDS sized to the nq queries of the launch, are read
// once for all of them).
constexpr int kScanKeys = 4;
__global__ __launch_bounds__(256) void k_lsh_scan(const uint32_t* __restrict__ sig_keys, int64_t n_rows,
                                                  const uint32_t* __restrict__ sig_q, int q0, int nq, int words,
                                                  int radius, int max_cand, uint32_t* __restrict__ cnt,
                                                  int32_t* __restrict__ cand) {
    extern __shared__ uint32_t sq[];  // [nq][words]
    for (int i = threadIdx.x; i < nq * words; i += 256) sq[i] = sig_q[(int64_t)q0 * words + i];
    __syncthreads();
    const int64_t stride = (int64_t)gridDim.x * 256;
    for (int64_t i0 = (int64_t)blockIdx.x * 256 + threadIdx.x; i0 < n_rows; i0 += kScanKeys * stride) {
        uint32_t k[kScanKeys][8];
#pragma unroll
        for (int e = 0; e < kScanKeys; ++e) {
            const int64_t i = i0 + e * stride;
            if ((words & 3) == 0) {  // 16-byte loads (signature rows are 16-byte aligned then)
                const uint4* p = (const uint4*)(sig_keys + i * words);
#pragma unroll
                for (int v = 0; v < 2; ++v) {
                    const uint4 x = (v * 4 < words && i < n_rows) ? p[v] : uint4{0u, 0u, 0u, 0u};
                    k[e][4 * v] = x.x, k[e][4 * v + 1] = x.y, k[e][4 * v + 2] = x.z, k[e][4 * v + 3] = x.w;
                }
            } else {
#pragma unroll
                for (int w = 0; w < 8; ++w) k[e][w] = (w < words && i < n_rows) ? sig_keys[i * words + w] : 0u;
            }
        }
        for (int b = 0; b < nq; ++b) {
            int h[kScanKeys] = {};
#pragma unroll
            for (int w = 0; w < 8; ++w) {
                if (w < words) {
                    const uint32_t qw = sq[b * words + w];
#pragma unroll
                    for (int e = 0; e < kScanKeys; ++e) h[e] += __popc(k[e][w] ^ qw);
                }
            }
#pragma unroll
            for (int e = 0; e < kScanKeys; ++e) {
                const int64_t i = i0 + e * stride;
                if (i < n_rows && h[e] <= radius) {
                    const uint32_t pos = atomicAdd(&cnt[q0 + b], 1u);
                    if (pos < (uint32_t)max_cand) cand[(int64_t)(q0 + b) * max_cand + pos] = (int32_t)i;
                }
            }
        }
    }
}

// One wave per query: the exact similarity of each candidate (the query and the entry read from their tiled
// stores, bf16 products summed in float32), the best as a packed top-1 (order-free: highest score, lowest
// index), then the threshold and stage 2 (verify_query); n_cand receives the candidate count.
__global__ __launch_bounds__(256) void k_lsh_verify(const u32x4* __restrict__ keys_tiled,
                                                    const u32x4* __restrict__ qt, int kc, int B,
                                                    const uint32_t* __restrict__ cnt,
                                                    const int32_t* __restrict__ cand, int max_cand,
                                                    int32_t* __restrict__ n_cand, int n_rows, int dtype,
                                                    const PrefixModels M, const int32_t* __restrict__ la_tok,
                                                    int k, const int32_t* __restrict__ tokens, int k_cap,
                                                    float tau_q, int32_t* __restrict__ idx_out,
                                                    float* __restrict__ score_out, float* __restrict__ resp_out,
                                                    int32_t* __restrict__ dec_out) {
    const int lane = threadIdx.x & 63;
    const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (b >= B) return;
    const uint32_t c_all = cnt[b];
    const int nc = c_all < (uint32_t)max_cand ? (int)c_all : max_cand;
    const int d_pad = kc * 32;
    uint64_t best = 0ull;
    for (int t = 0; t < nc; ++t) {
        const int32_t i = cand[(int64_t)b * max_cand + t];
        float acc = 0.0f;
        for (int j0 = lane * 8; j0 < d_pad; j0 += 512) {
            const u32x4 kv = *(const u32x4*)((const uint16_t*)keys_tiled + tiled_offset(i, j0, kc));
            const u32x4 qv = *(const u32x4*)((const uint16_t*)qt + tiled_offset(b, j0, kc));
            acc = dot8_bf16(qv, kv, acc);
        }
        acc = wave_sum_f32(acc);
        best = umax64(best, pack_top1(acc, i));
    }
    if (lane == 0) n_cand[b] = (int32_t)c_all;
    verify_query(b, best, unpack_idx(best), unpack_score(best), n_rows, dtype, M, la_tok, k, tokens, k_cap, tau_q,
                 idx_out, score_out, resp_out, dec_out, lane);
}

hipError_t launch_tile_rows(const uint16_t* src, int rows, int d, int d_pad, uint16_t* dst, hipStream_t s) {
    const int64_t total = (int64_t)rows * d_pad;
    if (total <= 0) return hipSuccess;
    k_tile_rows<<<dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s>>>(src, rows, d, d_pad, dst);
    return hipGetLastError();
}

hipError_t launch_simhash(const uint16_t* rows_tiled, int d_pad, int64_t row0, int64_t n, const uint16_t* hp_tiled,
                          int bits, uint32_t* sig, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    const int64_t g0 = row0 >> 4, g1 = (row0 + n + 15) >> 4;
    const int words = bits >> 5;
    // few rows (a query batch): one wave per signature word, so the words of a group are computed in parallel;
    // many rows (building the index): one wave per group, reading its rows once for every word
    const int wpw = (g1 - g0) * words <= 4096 ? 1 : words;
    const int64_t waves = (g1 - g0) * (words / wpw);
    k_simhash<<<dim3((unsigned)grid_blocks((waves + 3) / 4)), dim3(256), 0, s>>>(
        (const u32x4*)rows_tiled, d_pad >> 5, row0, n, (const u32x4*)hp_tiled, bits, wpw, sig);
    return hipGetLastError();
}

hipError_t launch_lsh_lookup(const void* queries, int dtype, int nb, int d, int d_pad, uint16_t* qt,
                             const uint16_t* hp_tiled, int bits, uint32_t* sigq, const uint16_t* keys_tiled,
                             const uint32_t* sig_keys, int64_t n_rows, int radius, int max_cand, uint32_t* cnt,
                             int32_t* cand, int32_t* n_cand, const PrefixModels& models, const int32_t* la_tok,
                             int k, const int32_t* tokens, int k_cap, float tau_q, int32_t* idx, float* score,
                             float* resp_score, int32_t* decision, int num_cu, hipStream_t s) {
    if (nb <= 0) return hipSuccess;
    const int words = bits >> 5;
    if (words < 1 || words > 8) return hipErrorInvalidValue;
    const dim3 pg((unsigned)((nb + 15) / 16)), pb(1024);
    const u32x4* hp = (const u32x4*)hp_tiled;
    if (d_pad <= 512)
        k_lsh_prep<1><<<pg, pb, 0, s>>>(queries, dtype, nb, d, d_pad, qt, hp, bits, sigq, cnt);
    else if (d_pad <= 1024)
        k_lsh_prep<2><<<pg, pb, 0, s>>>(queries, dtype, nb, d, d_pad, qt, hp, bits, sigq, cnt);
    else if (d_pad <= 2048)
        k_lsh_prep<4><<<pg, pb, 0, s>>>(queries, dtype, nb, d, d_pad, qt, hp, bits, sigq, cnt);
    else
        k_lsh_prep<0><<<pg, pb, 0, s>>>(queries, dtype, nb, d, d_pad, qt, hp, bits, sigq, cnt);
    // every thread a whole run of kScanKeys entries (no idle slots), at most 8 workgroups per CU
    int64_t blocks = (n_rows + 256 * kScanKeys - 1) / (256 * kScanKeys);
    if (blocks > 8 * num_cu) blocks = 8 * num_cu;
    if (blocks < 1) blocks = 1;
    for (int q0 = 0; q0 < nb && n_rows > 0; q0 += kScanQueries) {
        const int nq = nb - q0 < kScanQueries ? nb - q0 : kScanQueries;
        k_lsh_scan<<<dim3((unsigned)blocks), dim3(256), (size_t)nq * words * 4, s>>>(
            sig_keys, n_rows, sigq, q0, nq, words, radius, max_cand, cnt, cand);
    }
    k_lsh_verify<<<dim3((unsigned)((nb + 3) / 4)), dim3(256), 0, s>>>(
        (const u32x4*)keys_tiled, (const u32x4*)qt, d_pad >> 5, nb, cnt, cand, max_cand, n_cand, (int)n_rows,
        dtype, models, la_tok, k, tokens, k_cap, tau_q, idx, score, resp_score, decision);
    return hipGetLastError();
}

}  // namespace lacache
