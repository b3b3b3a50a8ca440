// verify.hpp -- the end of stage 1 and stage 2 for one query, shared by the kernels that produce a stage-1
// candidate (the merge of the exact partials, and the re-rank of LSH candidates).
//
// A candidate is a hit when its clamped similarity is >= tau_q (Section 5.1,
// cache check).  Only then does stage 2 run (Algorithm 1: the lookahead check
// sits inside the hit branch): the matched entry's stored prefix -- its
// embedding row(s) and its first k token IDs (Section 4.2, cache structure
// <h(x), [h(f_k(x)), f(x)]>) -- is gathered and compared with the query's
// lookahead.  The check passes on identical tokens, or on a prefix-embedding
// cosine >= tau_r (Section 5.1, lookahead check) -- under every one of the m
// prefix models when the cache holds an ensemble of lookahead checks
// (Section 4.4).  Decisions: 0 MISS, 1 REJECT, 2 HIT, 3 HIT_EXACT.
#pragma once

#include "common.hpp"
#include "launch.hpp"

namespace lacache {

// Exact row of query b inside the 32-row group g that the GEMM path reported: replay the group against
// the same 32-query fragment with the same MFMA sequence (v_mfma_f32_32x32x16_bf16 over the 16-column
// steps in order, from a zero accumulator), which reproduces the GEMM's float32 scores bit for bit, and
// take the lowest stored row whose score equals s.  Returns -1 if none does.  The operand fragments are
// loaded 16 steps at a time (the 2 kc steps are a multiple of 8: full batches of 16, then at most one of 8),
// each batch without branches, so the chain of MFMAs waits for memory about kc / 8 times rather than once per
// step.
template <int S>
__device__ __forceinline__ void replay_batch(const u32x4* __restrict__ kp, const u32x4* __restrict__ qp, bool qlane,
                                             int st0, int lane, f32x16& acc) {
    u32x4 ka[S], qa[S];
#pragma unroll
    for (int u = 0; u < S; ++u) {
        const int st = st0 + u;
        const int off = (st >> 1) * 64 + (((st & 1) << 1) + (lane >> 5)) * 16;
        ka[u] = kp[off];
        qa[u] = qlane ? qp[off] : u32x4{0u, 0u, 0u, 0u};
    }
    __builtin_amdgcn_sched_barrier(0);  // every load of the batch issued before the first MFMA waits
#pragma unroll
    for (int u = 0; u < S; ++u) acc = mfma32x32x16(ka[u], qa[u], acc);
}

__device__ inline int32_t replay_group(const u32x4* __restrict__ keys, const u32x4* __restrict__ qt, int kc, int b, int g,
                                float s, int n_rows, int lane) {
    const int kr = g * 32 + (lane & 31);       // key row this lane feeds (row operand)
    const int qr = (b & ~31) + (lane & 31);    // query row of the fragment (column operand)
    const u32x4* kp = keys + (int64_t)(kr >> 4) * kc * 64 + (kr & 15);
    const u32x4* qp = qt + (int64_t)(qr >> 4) * kc * 64 + (qr & 15);
    // only query b's column of the fragment is needed: every output column of the MFMA depends on its own
    // column of the column operand alone, so the other lanes feed zeros instead of loading their queries
    const bool qlane = (lane & 31) == (b & 31);
    f32x16 acc = f32x16{};
    const int n = 2 * kc;
    int st0 = 0;
    for (; st0 + 16 <= n; st0 += 16) replay_batch<16>(kp, qp, qlane, st0, lane, acc);
    if (st0 < n) replay_batch<8>(kp, qp, qlane, st0, lane, acc);
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

// One wave: outputs of query b for the packed stage-1 result m (0: no candidate) naming entry i with raw
// score s_raw.
__device__ inline void verify_query(int b, uint64_t m, int32_t i, float s_raw, int n_rows, int dtype,
                                    const PrefixModels& M, const int32_t* __restrict__ la_tok, int k,
                                    const int32_t* __restrict__ tokens, int k_cap, float tau_q,
                                    int32_t* __restrict__ idx_out, float* __restrict__ score_out,
                                    float* __restrict__ resp_out, int32_t* __restrict__ dec_out, int lane) {
    const float qnan = __uint_as_float(0x7FC00000u);
    const float score = fminf(fmaxf(s_raw, -1.0f), 1.0f);
    // every stored row yields a candidate, so m != 0 here; the range check keeps the gathers in bounds regardless
    if (m == 0ull || i < 0 || i >= n_rows || !(score >= tau_q)) {
        if (lane == 0) {
            idx_out[b] = (m == 0ull) ? -1 : i;
            score_out[b] = (m == 0ull) ? qnan : score;
            dec_out[b] = 0;
        }
        if (lane < M.m) resp_out[(int64_t)b * M.m + lane] = qnan;
        return;
    }

    // the first 64 of the first k tokens (lane j: token j), loaded with the first model's rows below
    const int32_t* ut = la_tok + (int64_t)b * k;
    const int32_t* tt = tokens + (int64_t)i * k_cap;
    const bool has0 = lane < k;
    const int32_t u0 = has0 ? ut[lane] : 0, t0 = has0 ? tt[lane] : 0;

    // for every prefix model: normalise the lookahead embedding exactly as stored vectors are and dot it with
    // the entry's stored prefix row; the embedding check passes only if every model reaches its threshold
    // (Section 4.4: with m lookahead checks a hit needs all of them)
    const size_t esz = dtype == 0 ? 4 : 2;
    bool all_pass = true;
    for (int mi = 0; mi < M.m; ++mi) {
        const int d = M.d[mi], d_pad = M.d_pad[mi];
        const char* src = (const char*)M.la[mi] + (int64_t)b * d * esz;
        const u32x4* er = (const u32x4*)(M.emb[mi] + (int64_t)i * d_pad);
        float acc = 0.0f;
        // padded columns are zero on both sides
        if (d_pad <= 1024) {
            // both rows loaded at once, the lookahead row kept in registers: the same norm, rounding and
            // dot order as normalise_row, one wait for memory instead of three
            float x[2][8];
            u32x4 e[2];
#pragma unroll
            for (int c = 0; c < 2; ++c) {
                const int j0 = lane * 8 + 512 * c;
                e[c] = j0 < d_pad ? er[j0 >> 3] : u32x4{0u, 0u, 0u, 0u};
            }
            row_to_regs<2>(src, dtype, d, true, lane, x);
            const double n = regs_norm<2>(x);
            const float rnf = quotient_rcp_f32(n);
#pragma unroll
            for (int c = 0; c < 2; ++c) {
                const int j0 = lane * 8 + 512 * c;
                if (j0 < d_pad) acc = dot8_bf16(regs_quantise8(x[c], j0, d, n, rnf, true), e[c], acc);
            }
        } else {
            normalise_row(src, dtype, d, d_pad, true, lane,
                          [&](int j0, u32x4 w) { acc = dot8_bf16(w, er[j0 >> 3], acc); });
        }
        acc = wave_sum_f32(acc);
        const float r = fminf(fmaxf(acc, -1.0f), 1.0f);
        if (lane == 0) resp_out[(int64_t)b * M.m + mi] = r;
        all_pass = all_pass && (r >= M.tau[mi]);
    }

    // first k tokens: lane j compares token j, 64 at a time
    bool tok_eq = __ballot(has0 && u0 != t0) == 0ull;
    for (int j0 = kWave; j0 < k; j0 += kWave) {
        const int j = j0 + lane;
        const bool differ = (j < k) && (ut[j] != tt[j]);
        if (__ballot(differ) != 0ull) tok_eq = false;
    }
    if (lane == 0) {
        idx_out[b] = i;
        score_out[b] = score;
        dec_out[b] = tok_eq ? 3 : (all_pass ? 2 : 1);
    }
}

}  // namespace lacache
