// k_verify.hip -- end of stage 1 (merge, threshold) and stage 2 (gather and verify), one wave per query.
//
// Stage 1 ends with the best entry over all partial candidates (for the GEMM
// path, whose partials name 16-row groups, the exact row is recovered by
// replaying the group; a replay that does not reproduce the stage-1 score
// still names a valid row of the group and is counted in *fallbacks); the
// threshold and stage 2 follow in verify_query.
#include "verify.hpp"

namespace lacache {

__global__ __launch_bounds__(256) void k_finalize_verify(
    const uint64_t* __restrict__ part, int P, int part_groups, const u32x4* __restrict__ keys_tiled,
    const u32x4* __restrict__ qt, int kc, int B, int n_rows, int dtype, const PrefixModels M,
    const int32_t* __restrict__ la_tok, int k, const int32_t* __restrict__ tokens, int k_cap, float tau_q,
    int32_t* __restrict__ idx_out, float* __restrict__ score_out, float* __restrict__ resp_out,
    int32_t* __restrict__ dec_out, uint32_t* __restrict__ fallbacks) {
    const int lane = threadIdx.x & 63;
    const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (b >= B) return;
    uint64_t m = 0;
    if (n_rows > 0) {
        for (int p = lane; p < P; p += kWave) m = umax64(m, part[(int64_t)b * P + p]);
        m = wave_max_u64(m);
    }
    int32_t i = unpack_idx(m);
    const float s_raw = unpack_score(m);
    if (part_groups && m != 0ull) {
        bool fb = false;
        i = replay_group16(keys_tiled, qt, kc, b, i, s_raw, n_rows, lane, &fb);
        if (fb && lane == 0) atomicAdd(fallbacks, 1u);
    }
    verify_query(b, m, i, s_raw, n_rows, dtype, M, la_tok, k, tokens, k_cap, tau_q, idx_out, score_out, resp_out,
                 dec_out, lane);
}

hipError_t launch_finalize_verify(const uint64_t* part, int P, bool part_groups, const uint16_t* keys_tiled,
                                  const uint16_t* qt, int B, int n_rows, int dtype, int d_keys,
                                  const PrefixModels& models, const int32_t* la_tok, int k, const int32_t* tokens,
                                  int k_cap, float tau_q, int32_t* idx, float* score, float* resp_score,
                                  int32_t* decision, uint32_t* fallbacks, hipStream_t s) {
    if (B <= 0) return hipSuccess;
    const int d_pad = (d_keys + 127) / 128 * 128;
    k_finalize_verify<<<dim3((B + 3) / 4), dim3(256), 0, s>>>(
        part, P, part_groups ? 1 : 0, (const u32x4*)keys_tiled, (const u32x4*)qt, d_pad / 32, B, n_rows, dtype,
        models, la_tok, k, tokens, k_cap, tau_q, idx, score, resp_score, decision, fallbacks);
    return hipGetLastError();
}

}  // namespace lacache
