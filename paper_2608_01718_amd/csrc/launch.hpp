// launch.hpp -- host-side launchers of the gfx950 kernels (called by the C ABI in lacache.cpp).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>
#include <tuple>
#include <utility>

namespace lacache {

// Workgroups of a grid-stride launch: at most 2^20, so that a grid's work-items (blocks x threads, up to
// 1024 threads) stay far below the 2^32 one dispatch can describe, whatever the row or pair count.
constexpr int64_t kMaxGridBlocks = int64_t(1) << 20;
inline int64_t grid_blocks(int64_t want) { return want < 1 ? 1 : (want > kMaxGridBlocks ? kMaxGridBlocks : want); }

// Allow kernel `fn` `bytes` of dynamic LDS on the current device, once per device (bit d of `done`; devices
// past 63 set it on every call).  Safe to call from several threads.
inline hipError_t allow_dynamic_lds(const void* fn, int bytes, std::atomic<uint64_t>& done) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    const uint64_t bit = dev < 64 ? (uint64_t(1) << dev) : 0;
    if (bit && (done.load(std::memory_order_acquire) & bit)) return hipSuccess;
    e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e == hipSuccess && bit) done.fetch_or(bit, std::memory_order_acq_rel);
    return e;
}

// Launch `kernel` on stream s.  With events e0 and e1 (both or neither) the launch goes through
// hipExtLaunchKernel, which takes the kernel's own start and end times into them from its dispatch: no
// event packets of their own on the stream, so timing a kernel does not change the gaps around it.
template <typename... P, typename... A>
hipError_t launch_timed(void (*kernel)(P...), dim3 grid, dim3 block, size_t lds, hipStream_t s, hipEvent_t e0,
                        hipEvent_t e1, A... args) {
    static_assert(sizeof...(P) == sizeof...(A), "one argument per kernel parameter");
    if (!e0) {
        kernel<<<grid, block, lds, s>>>(static_cast<P>(args)...);
        return hipGetLastError();
    }
    std::tuple<P...> t{static_cast<P>(args)...};
    return std::apply(
        [&](auto&... v) {
            void* a[] = {(void*)&v...};
            return hipExtLaunchKernel((const void*)kernel, grid, block, a, lds, s, e0, e1, 0);
        },
        t);
}

// Normalise `rows` input rows (dtype 0 f32 / 1 bf16, row-major [rows][d]) and
// store them as bfloat16 at destination rows row0 .. row0+rows-1, zero-filling
// up to rows_pad rows and d_pad columns; `tiled` selects the key layout,
// otherwise row-major [.][d_pad].
hipError_t launch_normalise(const void* in, int dtype, int64_t rows, int64_t rows_pad, int d, int d_pad,
                            uint16_t* out, int64_t row0, bool tiled, hipStream_t s);

// Dense [n][d] copy of stored rows first .. first+n-1.
hipError_t launch_export(const uint16_t* src, int64_t first, int n, int d, int d_pad, uint16_t* dst, bool tiled,
                         hipStream_t s);

// Stage 1, bandwidth-bound path: queries qt (tiled; up to 16 * stream_max_qg rows as one group, zero-padded to
// a multiple of 16, or up to four such groups, zero-padded to whole groups) against n_rows tiled keys.  Writes, for every query b
// and every workgroup p of the launch, the packed top-1 candidate
// part[b * P + p] (P <= kMaxPartials).  Returns the number of partials P through *P_out.
// With events e0 / e1 the kernel's run time is recorded into them (launch_timed).  With qraw (the caller's
// [B][d] query rows, dtype 0 f32 / 1 bf16) the kernel normalises the queries itself and qt is not read; this
// takes d_pad <= 2048 (stream_fused_ncq(d_pad) > 0).
hipError_t launch_stage1_stream(const uint16_t* keys, const uint16_t* qt, int B, int n_rows, int d_pad,
                                uint64_t* part, int num_cu, int* P_out, hipStream_t s, hipEvent_t e0 = nullptr,
                                hipEvent_t e1 = nullptr, const void* qraw = nullptr, int dtype = 0, int d = 0);
int stream_fused_ncq(int d_pad);

// Stage 1, compute-bound path (matrix-core GEMM with a fused row maximum): queries qt (tiled, rows zero-padded
// to a multiple of kGemmQueryTile) against n_rows keys.  The key store must hold whole tiles of kGemmKeyTile
// rows plus one spare tile past the last one (the kernel prefetches into it; its rows are never scored).  Its
// partials name the 16-row group of the candidate (global row / 16) instead of the row; the finalize step
// recovers the row by replaying that group (part_groups = true).
constexpr int kGemmKeyTile = 512;
constexpr int kGemmQueryTile = 128;
hipError_t launch_stage1_gemm(const uint16_t* keys, const uint16_t* qt, int B, int n_rows, int d_pad,
                              uint64_t* part, int num_cu, int* P_out, hipStream_t s, hipEvent_t e0 = nullptr,
                              hipEvent_t e1 = nullptr);

// The response-prefix embedding models of stage 2 (one per lookahead check of an ensemble).
constexpr int kMaxModels = 8;
struct PrefixModels {
    int m;                             // number of models, 1 .. kMaxModels
    const void* la[kMaxModels];        // [B][d_i] lookahead embeddings of the batch (cache dtype)
    const uint16_t* emb[kMaxModels];   // [capacity][d_pad_i] stored normalised prefix embeddings
    int d[kMaxModels], d_pad[kMaxModels];
    float tau[kMaxModels];             // stage-2 threshold of each model
};

// Merge the P partial candidates of each query (rows, or 16-row groups to replay against keys_tiled and
// the tiled queries qt), threshold, and run stage 2 on hits.  resp_score is [B][models.m].  Every query whose
// group replay does not reproduce its stage-1 score adds 1 to *fallbacks (device memory).
hipError_t launch_finalize_verify(const uint64_t* part, int P, bool part_groups, const uint16_t* keys_tiled,
                                  const uint16_t* qt, int B, int n_rows, int dtype, int d_keys,
                                  const PrefixModels& models, const int32_t* la_tok, int k, const int32_t* tokens,
                                  int k_cap, float tau_q, int32_t* idx, float* score, float* resp_score,
                                  int32_t* decision, uint32_t* fallbacks, hipStream_t s);

// Threshold calibration over n pairs (a[j], b[j]) of d-dimensional input vectors: sims[j] = the lookup's
// cosine of the pair; tau[0] = the percentile (linear between the closest ranks), tau[1] = min(cap, tau[0]).
// scratch: kCalibScratchWords words of device memory.
constexpr int kCalibScratchWords = 64 + 2 * 2048;
hipError_t launch_calibrate(const void* a, const void* b, int dtype, int d, int64_t n, float percentile, float cap,
                            float* sims, float* tau, uint32_t* scratch, int num_cu, hipStream_t s);

// Device address, on the current device, of the library's static calibration scratch (kCalibScratchWords words,
// one copy per device, shared by every allocation-free calibration on that device).  Allocates nothing.
hipError_t calibrate_static_scratch(uint32_t** out);

// Speculative-decoding acceptance: p_target[b][j] = softmax(logits[b][j])[tokens[b][j]] (0 for an
// out-of-range token); accept_len[b] = the number of leading positions with p_target >= p_draft.
hipError_t launch_accept_length(const void* logits, int dtype, int V, const int32_t* tokens, const float* p_draft,
                                int B, int k, int32_t* accept_len, float* p_target, hipStream_t s);

// LSH index (random hyperplanes): tiled copy of the raw hyperplanes, signatures of rows row0 .. row0+n-1 of a
// tiled matrix ([rows][bits / 32] words, bit i of a row is 1 when its projection on hyperplane i is >= 0),
// and the whole LSH lookup of a query batch (query preparation, Hamming-radius candidate scan, exact re-rank,
// threshold and stage 2).
hipError_t launch_tile_rows(const uint16_t* src, int rows, int d, int d_pad, uint16_t* dst, hipStream_t s);
hipError_t launch_simhash(const uint16_t* rows_tiled, int d_pad, int64_t row0, int64_t n, const uint16_t* hp_tiled,
                          int bits, uint32_t* sig, hipStream_t s);
hipError_t launch_lsh_lookup(const void* queries, int dtype, int nb, int d, int d_pad, uint16_t* qt,
                             const uint16_t* hp_tiled, int bits, uint32_t* sigq, const uint16_t* keys_tiled,
                             const uint32_t* sig_keys, int64_t n_rows, int radius, int max_cand, uint32_t* cnt,
                             int32_t* cand, int32_t* n_cand, const PrefixModels& models, const int32_t* la_tok,
                             int k, const int32_t* tokens, int k_cap, float tau_q, int32_t* idx, float* score,
                             float* resp_score, int32_t* decision, int num_cu, hipStream_t s);

// Most partials a stage-1 launch may write per query.
constexpr int kMaxPartials = 1024;

}  // namespace lacache
