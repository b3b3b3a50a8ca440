// lacache.cpp -- the C ABI (include/lacache.h): handle, argument checks, dispatch onto the caller's stream.
#include "../../include/lacache.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdlib>
#include <new>
#include <utility>
#include <vector>

#include "launch.hpp"

namespace lacache {
int stream_max_qg(int d_pad);
int stream_max_batch(int d_pad);

// Default crossover, from per-call times of both kernels for 64-256 queries on random bf16 keys:
// - 1M x 768, 1M x 1024 and 500k x 2048 keys: the GEMM kernel wins as soon as a second query group is
//   needed (by 3-6 % against two groups, up to 24 % against three or four);
// - 300k x 1536: two streaming groups still win (by 6 %), three lose (by 24 %);
// - 100k x 768: three streaming groups win (by 11-15 %), four lose.
// Each added group costs the streaming kernel a share of the contraction on every CU, while the GEMM
// kernel's time for one or two query tiles is its pass over the keys; the fewer the keys, the longer the
// streaming kernel stays ahead.
int stream_auto_batch(int d_pad, int64_t n_rows) {
    const int64_t elems = n_rows * (int64_t)d_pad;
    const int groups = elems >= (int64_t(1) << 29) ? 1 : elems >= (int64_t(1) << 27) ? 2 : 3;
    return groups * 16 * stream_max_qg(d_pad);
}
}  // namespace lacache

using namespace lacache;

struct lacache_s {
    int device = 0;
    int64_t cap = 0, cap_pad = 0, size = 0;
    int d = 0, d_pad = 0, k_cap = 0, dtype = 0, max_batch = 0, mb_pad = 0;
    int num_cu = 0, b_small = -1;  // -1: the crossover follows the cache size (stream_auto_batch)
    int m = 1;                 // prefix models (lookahead checks) per entry
    int d_resp[kMaxModels] = {}, d_pad_resp[kMaxModels] = {};
    uint16_t* keys = nullptr;  // tiled [cap_pad][d_pad]: whole GEMM key tiles plus one spare tile of zero rows
    uint16_t* emb[kMaxModels] = {};  // row-major [cap][d_pad_resp[i]], one per prefix model
    int32_t* tokens = nullptr; // [cap][k_cap]
    uint16_t* qt = nullptr;    // tiled [mb_pad][d_pad] normalised queries
    uint64_t* part = nullptr;  // [max_batch][kMaxPartials] packed top-1 candidates
    uint32_t* calib = nullptr; // [kCalibScratchWords] state and histograms of the calibration select
    uint32_t* fallbacks = nullptr;  // [1] queries whose stage-1 group replay missed its score (see k_verify.hip)
    // LSH index (lacache_enable_lsh): hyperplanes, key and query signatures, candidate lists
    int lsh_bits = 0, lsh_max_cand = 0;
    uint16_t* hp = nullptr;        // tiled [lsh_bits][d_pad] raw hyperplanes
    uint32_t* sig = nullptr;       // [cap][lsh_bits / 32]
    uint32_t* sigq = nullptr;      // [max_batch][lsh_bits / 32]
    uint32_t* lsh_cnt = nullptr;   // [max_batch]
    int32_t* lsh_cand = nullptr;   // [max_batch][lsh_max_cand]
    int prof_every = 0;        // lacache_profile: time every prof_every-th stage-1 launch (0: off)
    uint64_t prof_tick = 0;    // stage-1 launches since profiling was enabled
    // event pairs of the timed stage-1 launches: created when profiling is enabled (more only if a window
    // outgrows them) and reused across windows, so a timed lookup only records two events
    std::vector<std::pair<hipEvent_t, hipEvent_t>> prof;
    size_t prof_used = 0;
};

namespace {

constexpr int64_t kMaxCapacity = (int64_t(1) << 31) - 256;
constexpr int kRowTile = 256;  // query scratch rows are padded to it

int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// Runs `body` with the handle's device current and restores the caller's device.
struct DeviceGuard {
    int prev = -1;
    bool ok = false;
    explicit DeviceGuard(int dev) {
        if (hipGetDevice(&prev) != hipSuccess) return;
        ok = (prev == dev) || hipSetDevice(dev) == hipSuccess;
    }
    ~DeviceGuard() {
        if (ok && prev >= 0) (void)hipSetDevice(prev);
    }
};

void free_lsh(lacache_s* h) {
    (void)hipFree(h->hp);
    (void)hipFree(h->sig);
    (void)hipFree(h->sigq);
    (void)hipFree(h->lsh_cnt);
    (void)hipFree(h->lsh_cand);
    h->hp = nullptr;
    h->sig = h->sigq = h->lsh_cnt = nullptr;
    h->lsh_cand = nullptr;
    h->lsh_bits = h->lsh_max_cand = 0;
}

void free_all(lacache_s* h) {
    free_lsh(h);
    (void)hipFree(h->keys);
    for (int i = 0; i < kMaxModels; ++i) (void)hipFree(h->emb[i]);
    (void)hipFree(h->tokens);
    (void)hipFree(h->qt);
    (void)hipFree(h->part);
    (void)hipFree(h->calib);
    (void)hipFree(h->fallbacks);
    for (auto& p : h->prof) {
        (void)hipEventDestroy(p.first);
        (void)hipEventDestroy(p.second);
    }
    h->prof.clear();
}

int alloc_zero(void** p, size_t bytes) {
    if (hipMalloc(p, bytes) != hipSuccess) {
        *p = nullptr;
        (void)hipGetLastError();
        return LACACHE_ENOMEM;
    }
    return hipMemset(*p, 0, bytes) == hipSuccess ? LACACHE_OK : LACACHE_EHIP;
}

void clear_prof(lacache_s* h) { h->prof_used = 0; }

// Makes sure at least n event pairs exist.
int reserve_prof(lacache_s* h, size_t n) {
    while (h->prof.size() < n) {
        hipEvent_t e0 = nullptr, e1 = nullptr;
        if (hipEventCreate(&e0) != hipSuccess) return LACACHE_EHIP;
        if (hipEventCreate(&e1) != hipSuccess) {
            (void)hipEventDestroy(e0);
            return LACACHE_EHIP;
        }
        h->prof.emplace_back(e0, e1);
    }
    return LACACHE_OK;
}

}  // namespace

extern "C" {

const char* lacache_strerror(int code) {
    switch (code) {
        case LACACHE_OK: return "ok";
        case LACACHE_EINVAL: return "invalid argument";
        case LACACHE_EFULL: return "cache capacity exceeded";
        case LACACHE_ENOMEM: return "device allocation failed";
        case LACACHE_EHIP: return "HIP runtime error";
        default: return "unknown error code";
    }
}

int lacache_create_ensemble(lacache_t* out, int64_t capacity, int32_t d, int32_t k_cap, lacache_dtype in_dtype,
                            int32_t max_batch, int32_t device, int32_t m, const int32_t* d_resp) {
    if (!out) return LACACHE_EINVAL;
    *out = nullptr;
    if (capacity < 1 || capacity > kMaxCapacity || d < 1 || d > 16384 || k_cap < 1 || k_cap > 4096 ||
        (in_dtype != LACACHE_F32 && in_dtype != LACACHE_BF16) || max_batch < 1 || max_batch > 65536 ||
        device < 0 || m < 1 || m > kMaxModels || !d_resp)
        return LACACHE_EINVAL;
    for (int i = 0; i < m; ++i)
        if (d_resp[i] < 1 || d_resp[i] > 16384) return LACACHE_EINVAL;
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess) {
        (void)hipGetLastError();
        return LACACHE_EHIP;
    }
    if (device >= ndev) return LACACHE_EINVAL;
    DeviceGuard g(device);
    if (!g.ok) return LACACHE_EHIP;

    lacache_s* h = new (std::nothrow) lacache_s();
    if (!h) return LACACHE_ENOMEM;
    h->device = device;
    h->cap = capacity;
    h->cap_pad = round_up(capacity, kGemmKeyTile) + kGemmKeyTile;
    h->d = d;
    h->d_pad = (int)round_up(d, 128);
    h->m = m;
    for (int i = 0; i < m; ++i) {
        h->d_resp[i] = d_resp[i];
        h->d_pad_resp[i] = (int)round_up(d_resp[i], 128);
    }
    h->k_cap = k_cap;
    h->dtype = (int)in_dtype;
    h->max_batch = max_batch;
    h->mb_pad = (int)round_up(max_batch, kRowTile);
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, device) != hipSuccess) {
        delete h;
        return LACACHE_EHIP;
    }
    h->num_cu = prop.multiProcessorCount;
    h->b_small = -1;

    int rc = LACACHE_OK;
    if (rc == LACACHE_OK) rc = alloc_zero((void**)&h->keys, (size_t)h->cap_pad * h->d_pad * 2);
    for (int i = 0; i < m && rc == LACACHE_OK; ++i)
        rc = alloc_zero((void**)&h->emb[i], (size_t)h->cap * h->d_pad_resp[i] * 2);
    if (rc == LACACHE_OK) rc = alloc_zero((void**)&h->tokens, (size_t)h->cap * h->k_cap * 4);
    if (rc == LACACHE_OK) rc = alloc_zero((void**)&h->qt, (size_t)h->mb_pad * h->d_pad * 2);
    if (rc == LACACHE_OK) rc = alloc_zero((void**)&h->part, (size_t)h->max_batch * kMaxPartials * 8);
    if (rc == LACACHE_OK) rc = alloc_zero((void**)&h->calib, (size_t)kCalibScratchWords * 4);
    if (rc == LACACHE_OK) rc = alloc_zero((void**)&h->fallbacks, 4);
    if (rc == LACACHE_OK && hipDeviceSynchronize() != hipSuccess) rc = LACACHE_EHIP;
    if (rc != LACACHE_OK) {
        free_all(h);
        delete h;
        return rc;
    }
    *out = h;
    return LACACHE_OK;
}

int lacache_create(lacache_t* out, int64_t capacity, int32_t d, int32_t k_cap, lacache_dtype in_dtype,
                   int32_t max_batch, int32_t device) {
    return lacache_create_ensemble(out, capacity, d, k_cap, in_dtype, max_batch, device, 1, &d);
}

int lacache_destroy(lacache_t h) {
    if (!h) return LACACHE_OK;
    int rc = LACACHE_OK;
    {
        DeviceGuard g(h->device);
        if (!g.ok || hipDeviceSynchronize() != hipSuccess) rc = LACACHE_EHIP;
        free_all(h);
    }
    delete h;
    return rc;
}

int64_t lacache_size(lacache_t h) { return h ? h->size : -1; }

int lacache_insert_ensemble(lacache_t h, const void* keys, const void* const* resp_emb, const int32_t* resp_tokens,
                            int32_t n, int64_t* first_idx, void* stream) {
    if (!h || n < 0) return LACACHE_EINVAL;
    if (n == 0) {
        if (first_idx) *first_idx = h->size;
        return LACACHE_OK;
    }
    if (!keys || !resp_emb || !resp_tokens) return LACACHE_EINVAL;
    for (int i = 0; i < h->m; ++i)
        if (!resp_emb[i]) return LACACHE_EINVAL;
    if ((int64_t)n > h->cap - h->size) return LACACHE_EFULL;
    DeviceGuard g(h->device);
    if (!g.ok) return LACACHE_EHIP;
    hipStream_t s = (hipStream_t)stream;
    const int64_t first = h->size;
    if (launch_normalise(keys, h->dtype, n, n, h->d, h->d_pad, h->keys, first, true, s) != hipSuccess)
        return LACACHE_EHIP;
    for (int i = 0; i < h->m; ++i)
        if (launch_normalise(resp_emb[i], h->dtype, n, n, h->d_resp[i], h->d_pad_resp[i], h->emb[i], first, false,
                             s) != hipSuccess)
            return LACACHE_EHIP;
    if (hipMemcpyAsync(h->tokens + first * h->k_cap, resp_tokens, (size_t)n * h->k_cap * 4,
                       hipMemcpyDeviceToDevice, s) != hipSuccess)
        return LACACHE_EHIP;
    if (h->lsh_bits && launch_simhash(h->keys, h->d_pad, first, n, h->hp, h->lsh_bits, h->sig, s) != hipSuccess)
        return LACACHE_EHIP;
    h->size += n;
    if (first_idx) *first_idx = first;
    return LACACHE_OK;
}

int lacache_insert(lacache_t h, const void* keys, const void* resp_emb, const int32_t* resp_tokens, int32_t n,
                   int64_t* first_idx, void* stream) {
    if (h && h->m != 1) return LACACHE_EINVAL;
    return lacache_insert_ensemble(h, keys, &resp_emb, resp_tokens, n, first_idx, stream);
}

static int lookup_chunk(lacache_t h, const char* queries, const PrefixModels& models, const int32_t* la_tok, int B,
                        float tau_q, int k, int32_t* idx, float* score, float* resp, int32_t* dec, hipStream_t s) {
    const int n_rows = (int)h->size;
    int P = 0;
    const bool small = B <= (h->b_small >= 0 ? h->b_small : stream_auto_batch(h->d_pad, n_rows));
    if (n_rows > 0) {
        // the streaming kernel runs more than one query group on whole groups of 16 * stream_max_qg rows
        const int64_t grp = 16 * (int64_t)stream_max_qg(h->d_pad);
        const int64_t rows_pad =
            small ? (B <= grp ? round_up(B, 16) : round_up(B, grp)) : round_up(B, kGemmQueryTile);
        // up to 32 queries (at most two rows per wave) and d_pad = 2048 the streaming kernel normalises its queries
        // itself, saving the staging launch; with more rows per wave its prologue would cost more than that launch
        // (64 queries on 10k x 384 keys: ~5.7 us of prologue against ~4 us of staging), so they are staged
        const bool fused = small && B <= 32 && stream_fused_ncq(h->d_pad) > 0;
        if (!fused && launch_normalise(queries, h->dtype, B, rows_pad, h->d, h->d_pad, h->qt, 0, true, s) != hipSuccess)
            return LACACHE_EHIP;
        hipEvent_t e0 = nullptr, e1 = nullptr;
        if (h->prof_every > 0 && h->prof_tick++ % h->prof_every == 0) {
            if (h->prof_used == h->prof.size() && reserve_prof(h, 2 * h->prof.size() + 64) != LACACHE_OK)
                return LACACHE_EHIP;
            e0 = h->prof[h->prof_used].first;
            e1 = h->prof[h->prof_used].second;
            ++h->prof_used;
        }
        // with profiling on, the events take the stage-1 kernel's own start and end times (launch_timed)
        hipError_t e = small ? launch_stage1_stream(h->keys, h->qt, B, n_rows, h->d_pad, h->part, h->num_cu, &P, s,
                                                    e0, e1, fused ? queries : nullptr, h->dtype, h->d)
                             : launch_stage1_gemm(h->keys, h->qt, B, n_rows, h->d_pad, h->part, h->num_cu, &P, s,
                                                  e0, e1);
        if (e != hipSuccess) return LACACHE_EHIP;
    }
    if (launch_finalize_verify(h->part, P, !small, h->keys, h->qt, B, n_rows, h->dtype, h->d, models, la_tok, k,
                               h->tokens, h->k_cap, tau_q, idx, score, resp, dec, h->fallbacks, s) != hipSuccess)
        return LACACHE_EHIP;
    return LACACHE_OK;
}

int lacache_lookup_ensemble(lacache_t h, const void* queries, const void* const* lookahead_emb,
                            const int32_t* lookahead_tokens, int32_t B, float tau_q, const float* tau_r, int32_t k,
                            int32_t* idx, float* score, float* resp_score, int32_t* decision, void* stream) {
    if (!h || B < 0 || k < 1 || k > h->k_cap || !std::isfinite(tau_q) || !tau_r) return LACACHE_EINVAL;
    for (int i = 0; i < h->m; ++i)
        if (!std::isfinite(tau_r[i])) return LACACHE_EINVAL;
    if (B == 0) return LACACHE_OK;
    if (!queries || !lookahead_emb || !lookahead_tokens || !idx || !score || !resp_score || !decision)
        return LACACHE_EINVAL;
    for (int i = 0; i < h->m; ++i)
        if (!lookahead_emb[i]) return LACACHE_EINVAL;
    DeviceGuard g(h->device);
    if (!g.ok) return LACACHE_EHIP;
    const size_t esz = h->dtype == LACACHE_F32 ? 4 : 2;
    for (int b0 = 0; b0 < B; b0 += h->max_batch) {
        const int nb = (B - b0) < h->max_batch ? (B - b0) : h->max_batch;
        PrefixModels models{};
        models.m = h->m;
        for (int i = 0; i < h->m; ++i) {
            models.la[i] = (const char*)lookahead_emb[i] + (size_t)b0 * h->d_resp[i] * esz;
            models.emb[i] = h->emb[i];
            models.d[i] = h->d_resp[i];
            models.d_pad[i] = h->d_pad_resp[i];
            models.tau[i] = tau_r[i];
        }
        const int rc = lookup_chunk(h, (const char*)queries + (size_t)b0 * h->d * esz, models,
                                    lookahead_tokens + (size_t)b0 * k, nb, tau_q, k, idx + b0, score + b0,
                                    resp_score + (size_t)b0 * h->m, decision + b0, (hipStream_t)stream);
        if (rc != LACACHE_OK) return rc;
    }
    return LACACHE_OK;
}

int lacache_lookup(lacache_t h, const void* queries, const void* lookahead_emb, const int32_t* lookahead_tokens,
                   int32_t B, float tau_q, float tau_r, int32_t k, int32_t* idx, float* score, float* resp_score,
                   int32_t* decision, void* stream) {
    if (h && h->m != 1) return LACACHE_EINVAL;
    return lacache_lookup_ensemble(h, queries, &lookahead_emb, lookahead_tokens, B, tau_q, &tau_r, k, idx, score,
                                   resp_score, decision, stream);
}

int lacache_export(lacache_t h, int64_t first, int32_t n, uint16_t* keys_bf16, uint16_t* emb_bf16, int32_t* tokens,
                   void* stream) {
    if (!h || first < 0 || n < 0 || first + n > h->size) return LACACHE_EINVAL;
    if (n == 0) return LACACHE_OK;
    DeviceGuard g(h->device);
    if (!g.ok) return LACACHE_EHIP;
    hipStream_t s = (hipStream_t)stream;
    if (keys_bf16 && launch_export(h->keys, first, n, h->d, h->d_pad, keys_bf16, true, s) != hipSuccess)
        return LACACHE_EHIP;
    if (emb_bf16 && launch_export(h->emb[0], first, n, h->d_resp[0], h->d_pad_resp[0], emb_bf16, false, s) !=
                        hipSuccess)
        return LACACHE_EHIP;
    if (tokens && hipMemcpyAsync(tokens, h->tokens + first * h->k_cap, (size_t)n * h->k_cap * 4,
                                 hipMemcpyDeviceToDevice, s) != hipSuccess)
        return LACACHE_EHIP;
    return LACACHE_OK;
}

int lacache_export_prefix(lacache_t h, int32_t model, int64_t first, int32_t n, uint16_t* emb_bf16, void* stream) {
    if (!h || model < 0 || model >= h->m || first < 0 || n < 0 || first + n > h->size) return LACACHE_EINVAL;
    if (n == 0) return LACACHE_OK;
    if (!emb_bf16) return LACACHE_EINVAL;
    DeviceGuard g(h->device);
    if (!g.ok) return LACACHE_EHIP;
    if (launch_export(h->emb[model], first, n, h->d_resp[model], h->d_pad_resp[model], emb_bf16, false,
                      (hipStream_t)stream) != hipSuccess)
        return LACACHE_EHIP;
    return LACACHE_OK;
}

int32_t lacache_models(lacache_t h) { return h ? h->m : -1; }

int lacache_calibrate(lacache_t h, int32_t which, const void* a, const void* b, int64_t n, float percentile, float cap,
                      float* sims, float* tau, void* stream) {
    if (!h || which < -1 || which >= h->m || n < 1 || n > (int64_t)UINT32_MAX || !std::isfinite(percentile) ||
        percentile < 0.0f || percentile > 100.0f || !std::isfinite(cap) || !a || !b || !sims || !tau)
        return LACACHE_EINVAL;
    DeviceGuard g(h->device);
    if (!g.ok) return LACACHE_EHIP;
    const int dim = which < 0 ? h->d : h->d_resp[which];
    if (launch_calibrate(a, b, h->dtype, dim, n, percentile, cap, sims, tau, h->calib, h->num_cu,
                         (hipStream_t)stream) != hipSuccess)
        return LACACHE_EHIP;
    return LACACHE_OK;
}

int lacache_calibrate_noalloc(const void* a, const void* b, lacache_dtype dtype, int32_t d, int64_t n, float percentile,
                              float cap, float* sims, float* tau, void* stream) {
    if ((dtype != LACACHE_F32 && dtype != LACACHE_BF16) || d < 1 || d > 16384 || n < 1 || n > (int64_t)UINT32_MAX ||
        !std::isfinite(percentile) || percentile < 0.0f || percentile > 100.0f || !std::isfinite(cap) || !a || !b ||
        !sims || !tau)
        return LACACHE_EINVAL;
    int dev = 0, num_cu = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&num_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return LACACHE_EHIP;
    uint32_t* scratch = nullptr;
    if (calibrate_static_scratch(&scratch) != hipSuccess) return LACACHE_EHIP;
    if (launch_calibrate(a, b, (int)dtype, d, n, percentile, cap, sims, tau, scratch, num_cu, (hipStream_t)stream) !=
        hipSuccess)
        return LACACHE_EHIP;
    return LACACHE_OK;
}

int lacache_accept_length(const void* logits, lacache_dtype dtype, int32_t V, const int32_t* draft_tokens,
                          const float* p_draft, int32_t B, int32_t k, int32_t* accept_len, float* p_target,
                          void* stream) {
    if (V < 1 || B < 0 || k < 1 || k > 4096 || (dtype != LACACHE_F32 && dtype != LACACHE_BF16)) return LACACHE_EINVAL;
    if (B == 0) return LACACHE_OK;
    if (!logits || !draft_tokens || !p_draft || !accept_len || !p_target) return LACACHE_EINVAL;
    if (launch_accept_length(logits, (int)dtype, V, draft_tokens, p_draft, B, k, accept_len, p_target,
                             (hipStream_t)stream) != hipSuccess)
        return LACACHE_EHIP;
    return LACACHE_OK;
}

int lacache_enable_lsh(lacache_t h, int32_t bits, const uint16_t* hyperplanes, int32_t max_candidates,
                       void* stream) {
    if (!h || bits < 32 || bits > 256 || bits % 32 != 0 || !hyperplanes || max_candidates < 1 ||
        max_candidates > 65536)
        return LACACHE_EINVAL;
    DeviceGuard g(h->device);
    if (!g.ok) return LACACHE_EHIP;
    hipStream_t s = (hipStream_t)stream;
    // earlier work on the handle may still read the old index
    if (hipStreamSynchronize(s) != hipSuccess) return LACACHE_EHIP;
    free_lsh(h);
    const int words = bits / 32;
    int rc = LACACHE_OK;
    if (rc == LACACHE_OK) rc = alloc_zero((void**)&h->hp, (size_t)bits * h->d_pad * 2);
    if (rc == LACACHE_OK) rc = alloc_zero((void**)&h->sig, (size_t)h->cap * words * 4);
    if (rc == LACACHE_OK) rc = alloc_zero((void**)&h->sigq, (size_t)h->mb_pad * words * 4);
    if (rc == LACACHE_OK) rc = alloc_zero((void**)&h->lsh_cnt, (size_t)h->max_batch * 4);
    if (rc == LACACHE_OK) rc = alloc_zero((void**)&h->lsh_cand, (size_t)h->max_batch * max_candidates * 4);
    if (rc != LACACHE_OK) {
        free_lsh(h);
        return rc;
    }
    h->lsh_bits = bits;
    h->lsh_max_cand = max_candidates;
    if (launch_tile_rows(hyperplanes, bits, h->d, h->d_pad, h->hp, s) != hipSuccess ||
        launch_simhash(h->keys, h->d_pad, 0, h->size, h->hp, bits, h->sig, s) != hipSuccess)
        return LACACHE_EHIP;
    return LACACHE_OK;
}

int lacache_lookup_lsh(lacache_t h, const void* queries, const void* lookahead_emb, const int32_t* lookahead_tokens,
                       int32_t B, float tau_q, float tau_r, int32_t k, int32_t radius, int32_t* idx, float* score,
                       float* resp_score, int32_t* decision, int32_t* n_cand, void* stream) {
    if (!h || h->m != 1 || !h->lsh_bits || B < 0 || k < 1 || k > h->k_cap || radius < 0 || radius > h->lsh_bits ||
        !std::isfinite(tau_q) || !std::isfinite(tau_r))
        return LACACHE_EINVAL;
    if (B == 0) return LACACHE_OK;
    if (!queries || !lookahead_emb || !lookahead_tokens || !idx || !score || !resp_score || !decision || !n_cand)
        return LACACHE_EINVAL;
    DeviceGuard g(h->device);
    if (!g.ok) return LACACHE_EHIP;
    hipStream_t s = (hipStream_t)stream;
    const size_t esz = h->dtype == LACACHE_F32 ? 4 : 2;
    for (int b0 = 0; b0 < B; b0 += h->max_batch) {
        const int nb = (B - b0) < h->max_batch ? (B - b0) : h->max_batch;
        const char* q = (const char*)queries + (size_t)b0 * h->d * esz;
        PrefixModels models{};
        models.m = 1;
        models.la[0] = (const char*)lookahead_emb + (size_t)b0 * h->d_resp[0] * esz;
        models.emb[0] = h->emb[0];
        models.d[0] = h->d_resp[0];
        models.d_pad[0] = h->d_pad_resp[0];
        models.tau[0] = tau_r;
        if (launch_lsh_lookup(q, h->dtype, nb, h->d, h->d_pad, h->qt, h->hp, h->lsh_bits, h->sigq, h->keys, h->sig,
                              h->size, radius, h->lsh_max_cand, h->lsh_cnt, h->lsh_cand, n_cand + b0, models,
                              lookahead_tokens + (size_t)b0 * k, k, h->tokens, h->k_cap, tau_q, idx + b0,
                              score + b0, resp_score + b0, decision + b0, h->num_cu, s) != hipSuccess)
            return LACACHE_EHIP;
    }
    return LACACHE_OK;
}

int lacache_export_signatures(lacache_t h, int64_t first, int32_t n, uint32_t* sig, void* stream) {
    if (!h || !h->lsh_bits || first < 0 || n < 0 || first + n > h->size) return LACACHE_EINVAL;
    if (n == 0) return LACACHE_OK;
    if (!sig) return LACACHE_EINVAL;
    DeviceGuard g(h->device);
    if (!g.ok) return LACACHE_EHIP;
    const size_t words = (size_t)h->lsh_bits / 32;
    if (hipMemcpyAsync(sig, h->sig + first * words, (size_t)n * words * 4, hipMemcpyDeviceToDevice,
                       (hipStream_t)stream) != hipSuccess)
        return LACACHE_EHIP;
    return LACACHE_OK;
}

int lacache_replay_fallbacks(lacache_t h, int64_t* count) {
    if (!h || !count) return LACACHE_EINVAL;
    DeviceGuard g(h->device);
    if (!g.ok) return LACACHE_EHIP;
    uint32_t v = 0;
    if (hipDeviceSynchronize() != hipSuccess || hipMemcpy(&v, h->fallbacks, 4, hipMemcpyDeviceToHost) != hipSuccess)
        return LACACHE_EHIP;
    *count = v;
    return LACACHE_OK;
}

int lacache_set_small_batch(lacache_t h, int32_t b_small) {
    if (!h || b_small < -1 || b_small > stream_max_batch(h->d_pad)) return LACACHE_EINVAL;
    h->b_small = b_small;
    return LACACHE_OK;
}

int lacache_profile(lacache_t h, int32_t every) {
    if (!h || every < 0) return LACACHE_EINVAL;
    DeviceGuard g(h->device);
    if (!g.ok) return LACACHE_EHIP;
    clear_prof(h);
    h->prof_every = every;
    h->prof_tick = 0;
    // the events of a typical timing window, created now rather than inside it
    return every > 0 ? reserve_prof(h, 256) : LACACHE_OK;
}

int lacache_profile_read(lacache_t h, double* stage1_ms, int64_t* lookups) {
    if (!h || !stage1_ms || !lookups) return LACACHE_EINVAL;
    DeviceGuard g(h->device);
    if (!g.ok) return LACACHE_EHIP;
    double total = 0.0;
    int64_t cnt = 0;
    int rc = LACACHE_OK;
    for (size_t i = 0; i < h->prof_used; ++i) {
        const auto& p = h->prof[i];
        float ms = 0.f;
        if (hipEventSynchronize(p.second) != hipSuccess || hipEventElapsedTime(&ms, p.first, p.second) != hipSuccess) {
            rc = LACACHE_EHIP;
            break;
        }
        total += ms;
        ++cnt;
    }
    clear_prof(h);
    *stage1_ms = total;
    *lookups = cnt;
    return rc;
}

}  // extern "C"
