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

// The row a group replay names, and the rule that picks it (host-callable, so the rule itself is checked on the
// CPU): the lowest row whose replayed score equals the stage-1 score; if none does (the replay did not
// reproduce the stage-1 arithmetic), the lowest row at the replay's own maximum, flagged as a fallback, so that
// a valid entry of the group is always returned.  Rows are offered one at a time (replay_pick_add) and the
// partial picks of several lanes merged in any order (replay_pick_merge).
struct ReplayPick {
    int exact;    // lowest row whose replayed score equals the stage-1 score (0x7FFFFFFF: none)
    float top;    // highest replayed score seen
    int top_row;  // lowest row holding it (0x7FFFFFFF: no row seen)
};
__host__ __device__ inline ReplayPick replay_pick_none() { return ReplayPick{0x7FFFFFFF, -__builtin_inff(), 0x7FFFFFFF}; }
__host__ __device__ inline ReplayPick replay_pick_add(ReplayPick p, int row, float v, float s) {
    if (v == s && row < p.exact) p.exact = row;
    if (v > p.top || (v == p.top && row < p.top_row)) {
        p.top = v;
        p.top_row = row;
    }
    return p;
}
__host__ __device__ inline ReplayPick replay_pick_merge(ReplayPick a, ReplayPick b) {
    ReplayPick r;
    r.exact = a.exact < b.exact ? a.exact : b.exact;
    const bool take_b = b.top > a.top || (b.top == a.top && b.top_row < a.top_row);
    r.top = take_b ? b.top : a.top;
    r.top_row = take_b ? b.top_row : a.top_row;
    return r;
}
// The named row (-1 when no row was offered); *fallback is set when no replayed score matched.
__host__ __device__ inline int replay_pick_row(ReplayPick p, bool* fallback) {
    *fallback = p.exact == 0x7FFFFFFF;
    const int r = *fallback ? p.top_row : p.exact;
    return r == 0x7FFFFFFF ? -1 : r;
}

// Exact row of query b inside the 16-row group g that the GEMM path reported: replay the group against query
// b with the stage-1 instruction sequence (v_mfma_f32_16x16x32_bf16 over the 32-column steps in order, from a
// zero accumulator), which reproduces the GEMM's float32 scores bit for bit, and pick the row with
// replay_pick_*.  The key operand is the group's 1 KiB chunk of each step; only query b's column of the query
// operand is loaded (every output column of the MFMA depends on its own column alone), the other lanes feed
// zeros.  The operand fragments are loaded 8 steps at a time (kc is a multiple of 4: full batches of 8, then at
// most one of 4), each batch without branches, so the chain of MFMAs waits for memory about kc / 8 times.
template <int S>
__device__ __forceinline__ void replay16_batch(const u32x4* __restrict__ kp, const u32x4* __restrict__ qp, bool qlane,
                                               int st0, f32x4& acc) {
    u32x4 ka[S], qa[S];
#pragma unroll
    for (int u = 0; u < S; ++u) {
        ka[u] = kp[(int64_t)(st0 + u) * 64];
        qa[u] = qlane ? qp[(int64_t)(st0 + u) * 64] : u32x4{0u, 0u, 0u, 0u};
    }
    __builtin_amdgcn_sched_barrier(0);  // every load of the batch issued before the first MFMA waits
#pragma unroll
    for (int u = 0; u < S; ++u) acc = mfma16x16x32(ka[u], qa[u], acc);
}

__device__ inline int32_t replay_group16(const u32x4* __restrict__ keys, const u32x4* __restrict__ qt, int kc, int b,
                                         int g, float s, int n_rows, int lane, bool* fallback) {
    const u32x4* kp = keys + (int64_t)g * kc * 64 + lane;          // chunk (g, j) at kp + 64 j
    const u32x4* qp = qt + (int64_t)(b >> 4) * kc * 64 + lane;     // query rows (b & ~15) .. + 15
    const bool qlane = (lane & 15) == (b & 15);
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
    int st0 = 0;
    for (; st0 + 8 <= kc; st0 += 8) replay16_batch<8>(kp, qp, qlane, st0, acc);
    if (st0 < kc) replay16_batch<4>(kp, qp, qlane, st0, acc);
    // lane l holds rows 4 (l / 16) + i of the group for query column l % 16
    ReplayPick p = replay_pick_none();
    if (qlane) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = g * 16 + 4 * (lane >> 4) + i;
            if (r < n_rows) p = replay_pick_add(p, r, acc[i], s);
        }
    }
#pragma unroll
    for (int m = 16; m <= 32; m <<= 1) {
        ReplayPick o;
        o.exact = __shfl_xor(p.exact, m, kWave);
        o.top = __shfl_xor(p.top, m, kWave);
        o.top_row = __shfl_xor(p.top_row, m, kWave);
        p = replay_pick_merge(p, o);
    }
    // lane b % 16 now holds the merged pick of the four lanes of query b
    p.exact = __shfl(p.exact, b & 15, kWave);
    p.top = __shfl(p.top, b & 15, kWave);
    p.top_row = __shfl(p.top_row, b & 15, kWave);
    return replay_pick_row(p, fallback);
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
