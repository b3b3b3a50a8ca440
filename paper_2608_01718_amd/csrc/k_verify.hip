// k_verify.hip -- end of stage 1 (merge, threshold) and stage 2 (gather and verify), one wave per query.
//
// Stage 1 ends with the best entry over all partial candidates; it is a hit
// when the clamped similarity is >= tau_q (Section 5.1, cache check).  Only
// then does stage 2 run (Algorithm 1: the lookahead check sits inside the
// hit branch): the matched entry's stored prefix -- its embedding row and its
// first k token IDs (Section 4.2, cache structure <h(x), [h(f_k(x)), f(x)]>)
// -- is gathered and compared with the query's lookahead.  The check passes
// on identical tokens, or on a prefix-embedding cosine >= tau_r (Section 5.1,
// lookahead check).  Decisions: 0 MISS, 1 REJECT, 2 HIT, 3 HIT_EXACT.
#include "common.hpp"
#include "launch.hpp"

namespace lacache {

// Exact row of query b inside the 32-row group g that the GEMM path reported: replay the group against
// the same 32-query fragment with the same MFMA sequence (v_mfma_f32_32x32x16_bf16 over the 16-column
// steps in order, from a zero accumulator), which reproduces the GEMM's float32 scores bit for bit, and
// take the lowest stored row whose score equals s.  Returns -1 if none does.
__device__ int32_t replay_group(const u32x4* __restrict__ keys, const u32x4* __restrict__ qt, int kc, int b, int g,
                                float s, int n_rows, int lane) {
    const int kr = g * 32 + (lane & 31);       // key row this lane feeds (row operand)
    const int qr = (b & ~31) + (lane & 31);    // query row of the fragment (column operand)
    const u32x4* kp = keys + (int64_t)(kr >> 4) * kc * 64 + (kr & 15);
    const u32x4* qp = qt + (int64_t)(qr >> 4) * kc * 64 + (qr & 15);
    f32x16 acc = f32x16{};
    for (int st = 0; st < 2 * kc; ++st) {
        const int off = (st >> 1) * 64 + (((st & 1) << 1) + (lane >> 5)) * 16;
        acc = mfma32x32x16(kp[off], qp[off], st == 0 ? f32x16{} : acc);
    }
    int row = 0x7FFFFFFF;
    if ((lane & 31) == (b & 31)) {
#pragma unroll
        for (int j = 15; j >= 0; --j) {
            const int r = g * 32 + 8 * (j >> 2) + 4 * (lane >> 5) + (j & 3);
            if (acc[j] == s && r < n_rows) row = r;
        }
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) row = min(row, __shfl_xor(row, m, kWave));
    return row == 0x7FFFFFFF ? -1 : row;
}

__global__ __launch_bounds__(256) void k_finalize_verify(
    const uint64_t* __restrict__ part, int P, int part_groups, const u32x4* __restrict__ keys_tiled,
    const u32x4* __restrict__ qt, int kc, int B, int n_rows, const void* __restrict__ la, int dtype, int d,
    const int32_t* __restrict__ la_tok, int k, const uint16_t* __restrict__ emb, int d_pad,
    const int32_t* __restrict__ tokens, int k_cap, float tau_q, float tau_r, int32_t* __restrict__ idx_out,
    float* __restrict__ score_out, float* __restrict__ resp_out, int32_t* __restrict__ dec_out) {
    const int lane = threadIdx.x & 63;
    const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (b >= B) return;
    const float qnan = __uint_as_float(0x7FC00000u);
    if (n_rows <= 0) {
        if (lane == 0) {
            idx_out[b] = -1;
            score_out[b] = qnan;
            resp_out[b] = qnan;
            dec_out[b] = 0;
        }
        return;
    }
    uint64_t m = 0;
    for (int p = lane; p < P; p += kWave) m = umax64(m, part[(int64_t)b * P + p]);
    m = wave_max_u64(m);
    int32_t i = unpack_idx(m);
    const float s_raw = unpack_score(m);
    if (part_groups && m != 0ull) i = replay_group(keys_tiled, qt, kc, b, i, s_raw, n_rows, lane);
    const float score = fminf(fmaxf(s_raw, -1.0f), 1.0f);
    // every stored row yields a candidate, so m != 0 here; the range check keeps the gathers in bounds regardless
    if (m == 0ull || i < 0 || i >= n_rows || !(score >= tau_q)) {
        if (lane == 0) {
            idx_out[b] = (m == 0ull) ? -1 : i;
            score_out[b] = (m == 0ull) ? qnan : score;
            resp_out[b] = qnan;
            dec_out[b] = 0;
        }
        return;
    }

    // normalise the lookahead embedding exactly as stored vectors are, and dot it with the entry's prefix row
    const char* src = (const char*)la + (int64_t)b * d * (dtype == 0 ? 4 : 2);
    const u32x4* er = (const u32x4*)(emb + (int64_t)i * d_pad);
    float acc = 0.0f;
    normalise_row(src, dtype, d, d_pad, true, lane, [&](int j0, u32x4 w) {
        const u32x4 e = er[j0 >> 3];
        const uint32_t av[4] = {w.x, w.y, w.z, w.w}, ev[4] = {e.x, e.y, e.z, e.w};
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            // bf16 x bf16 products are exact in float; padded columns are zero on both sides
            acc += __uint_as_float(av[t] << 16) * __uint_as_float(ev[t] << 16);
            acc += __uint_as_float(av[t] & 0xFFFF0000u) * __uint_as_float(ev[t] & 0xFFFF0000u);
        }
    });
    acc = wave_sum_f32(acc);
    const float r = fminf(fmaxf(acc, -1.0f), 1.0f);

    // first k tokens: lane j compares token j, 64 at a time
    bool tok_eq = true;
    const int32_t* ut = la_tok + (int64_t)b * k;
    const int32_t* tt = tokens + (int64_t)i * k_cap;
    for (int j0 = 0; j0 < k; j0 += kWave) {
        const int j = j0 + lane;
        const bool differ = (j < k) && (ut[j] != tt[j]);
        if (__ballot(differ) != 0ull) tok_eq = false;
    }
    if (lane == 0) {
        idx_out[b] = i;
        score_out[b] = score;
        resp_out[b] = r;
        dec_out[b] = tok_eq ? 3 : (r >= tau_r ? 2 : 1);
    }
}

hipError_t launch_finalize_verify(const uint64_t* part, int P, bool part_groups, const uint16_t* keys_tiled,
                                  const uint16_t* qt, int B, int n_rows, const void* la, int dtype, int d,
                                  const int32_t* la_tok, int k, const uint16_t* emb, int d_pad,
                                  const int32_t* tokens, int k_cap, float tau_q, float tau_r, int32_t* idx,
                                  float* score, float* resp_score, int32_t* decision, hipStream_t s) {
    if (B <= 0) return hipSuccess;
    k_finalize_verify<<<dim3((B + 3) / 4), dim3(256), 0, s>>>(
        part, P, part_groups ? 1 : 0, (const u32x4*)keys_tiled, (const u32x4*)qt, d_pad / 32, B, n_rows, la, dtype,
        d, la_tok, k, emb, d_pad, tokens, k_cap, tau_q, tau_r, idx, score, resp_score, decision);
    return hipGetLastError();
}

}  // namespace lacache
