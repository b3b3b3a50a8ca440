/*
 * lacache.h -- C ABI of the LaCache two-stage semantic-cache lookup for
 * AMD Instinct MI355X (gfx950).
 *
 * The method (LaCache, "Robust Semantic Caching for LLM Serving"):
 *   - Each cache entry is <h(x), [h(f_k(x)), f(x)]> (Section 4.2, cache
 *     structure): the key of the cached query x, a lookahead key of the first
 *     k tokens of its response, and the response itself.  Here the key is the
 *     L2-normalised query embedding, the lookahead key is the normalised
 *     embedding of the response prefix plus the k prefix token IDs, and the
 *     response f(x) stays with the caller, addressed by the entry index.
 *   - A query is processed in two stages (Algorithm 1, Section 4.2 query
 *     processing).  Stage 1 searches the cache with the query key: the entry
 *     of highest cosine similarity is the candidate, a hit when its
 *     similarity is >= tau_q (Section 5.1: cache check sim(x, x') >= tau_c).
 *     Stage 2 runs only on a stage-1 hit: the lookahead of the new query
 *     (its first k speculatively decoded tokens and their embedding) is
 *     compared with the stored prefix of the matched entry; it passes when
 *     the k tokens are identical or the prefix-embedding cosine is >= tau_r
 *     (Section 5.1: lookahead check sim(f_k(x), f_k(x')) >= tau_a).  Only
 *     when both pass is the cached response served; otherwise the caller
 *     decodes and inserts (Algorithm 1, fallback branch).
 *   - With an ensemble of m lookahead checks (Section 4.4: m prefix
 *     embedding models, a hit needs every check to pass) each entry stores m
 *     prefix embeddings, one per model and each of its own dimension, and
 *     the embedding branch of stage 2 passes only when every model's cosine
 *     reaches that model's threshold.  The single-model functions are the
 *     case m = 1, with the prefix model of the key's dimension.
 *
 * Conventions for every function below:
 *   - Every array argument is a DEVICE pointer on the handle's device (for
 *     example a PyTorch ROCm tensor's data_ptr()), row-major and contiguous,
 *     unless marked "host".  Pointers may be NULL only when the matching
 *     count is 0.
 *   - `stream` is a hipStream_t (NULL = the default stream).  insert, lookup
 *     and export only enqueue work on it and return without waiting; the
 *     caller keeps every buffer alive until the stream has passed the call.
 *     Work on one handle must be ordered on one stream (or by events): calls
 *     share the handle's store and scratch buffers.
 *   - A handle is not thread-safe.
 *   - Errors are returned as negative codes and nothing is enqueued when an
 *     argument check fails.  No C++ exception crosses this interface.
 *   - Vector inputs must be finite; non-finite components give unspecified
 *     (but memory-safe) results.
 */
#ifndef LACACHE_H
#define LACACHE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct lacache_s *lacache_t;

/* largest number of prefix models (lookahead checks) of an ensemble cache */
#define LACACHE_MAX_MODELS 8

/* dtype of every input vector of a cache (keys, prefix embeddings, queries, lookahead embeddings) */
typedef enum { LACACHE_F32 = 0, LACACHE_BF16 = 1 } lacache_dtype;

/* decision[b] of a lookup */
enum {
    LACACHE_MISS = 0,      /* stage 1 found no entry with similarity >= tau_q; stage 2 did not run */
    LACACHE_REJECT = 1,    /* stage-1 hit whose lookahead check failed: a collision, decode and insert */
    LACACHE_HIT = 2,       /* both checks passed through the prefix-embedding similarity */
    LACACHE_HIT_EXACT = 3  /* both checks passed with identical first-k prefix tokens */
};

/* return codes */
enum {
    LACACHE_OK = 0,
    LACACHE_EINVAL = -1,   /* bad argument (null pointer, size out of range, non-finite threshold) */
    LACACHE_EFULL = -2,    /* insert would exceed the capacity; nothing was inserted */
    LACACHE_ENOMEM = -3,   /* device allocation failed */
    LACACHE_EHIP = -4      /* a HIP runtime call or kernel launch failed */
};

/*
 * Create a cache on `device` for up to `capacity` entries (1 <= capacity <
 * 2^31 - 256) of dimension d (1 <= d <= 16384), each storing k_cap prefix
 * tokens (1 <= k_cap <= 4096).  Every input vector has dtype in_dtype.
 * max_batch (1 <= max_batch <= 65536) sizes the lookup scratch; lookups with
 * more queries are processed in chunks of max_batch.  All device memory
 * (store and scratch) is allocated here, once, and zero-filled: the store
 * takes capacity * (2 * d_pad * 2 + 4 * k_cap) bytes with d_pad = d rounded
 * up to a multiple of 128.  On success *out receives the handle.
 */
int lacache_create(lacache_t *out, int64_t capacity, int32_t d, int32_t k_cap, lacache_dtype in_dtype,
                   int32_t max_batch, int32_t device);

/*
 * Create a cache whose entries carry an ensemble of m response-prefix
 * embeddings (Section 4.4, m lookahead checks), 1 <= m <= LACACHE_MAX_MODELS.
 * d_resp (host, [m]) gives each prefix model's dimension, 1 .. 16384; the
 * other arguments are those of lacache_create, which equals this call with
 * m = 1 and d_resp = {d}.  The store takes capacity * (2 * d_pad + sum over
 * i of 2 * d_pad_i + 4 * k_cap) bytes, d_pad_i = d_resp[i] rounded up to a
 * multiple of 128.
 */
int lacache_create_ensemble(lacache_t *out, int64_t capacity, int32_t d, int32_t k_cap, lacache_dtype in_dtype,
                            int32_t max_batch, int32_t device, int32_t m, const int32_t *d_resp);

/* Number of prefix models m of the cache; -1 for a NULL handle. */
int32_t lacache_models(lacache_t h);

/* Wait for the device, free everything the handle owns, and the handle itself. NULL is a no-op. */
int lacache_destroy(lacache_t h);

/*
 * Append n entries (Algorithm 1: after decoding, the new entry is added to
 * the cache).  keys and resp_emb are [n][d] of the cache's dtype (the query
 * key and the embedding of the first k_cap response tokens, both from the
 * same embedding model); resp_tokens is [n][k_cap] int32.  Keys and
 * embeddings are L2-normalised (in double) and rounded once, to nearest-even,
 * to bfloat16 as they are stored; a zero vector is stored as zero.
 * Entries get indices size .. size+n-1 in order; *first_idx (host) receives
 * the first.  The entry count is updated immediately, so later lookups on
 * the same stream see the new entries.  n == 0 is a no-op.  Returns
 * LACACHE_EFULL, inserting nothing, if n > capacity - size.  Only for a
 * cache with m = 1 (else LACACHE_EINVAL).
 */
int lacache_insert(lacache_t h, const void *keys, const void *resp_emb, const int32_t *resp_tokens, int32_t n,
                   int64_t *first_idx, void *stream);

/*
 * lacache_insert for any m: resp_emb is a HOST array of m device pointers,
 * resp_emb[i] being [n][d_resp[i]] (cache dtype), the prefix embedding of
 * each entry under model i.  Each is normalised and rounded as keys are.
 */
int lacache_insert_ensemble(lacache_t h, const void *keys, const void *const *resp_emb, const int32_t *resp_tokens,
                            int32_t n, int64_t *first_idx, void *stream);

/*
 * Two-stage lookup of B queries (Algorithm 1).
 *   queries          [B][d]  query embeddings (cache dtype)
 *   lookahead_emb    [B][d]  embedding of each query's first k decoded tokens (cache dtype)
 *   lookahead_tokens [B][k]  int32 token IDs of that prefix
 *   tau_q, tau_r     finite thresholds of stage 1 and stage 2 (compared with >=)
 *   k                1 <= k <= k_cap: number of prefix tokens compared
 * Outputs, each [B]:
 *   idx         entry of highest cosine similarity (lowest index among exact
 *               ties), reported even on a miss; -1 only when the cache is empty
 *   score       that similarity, clamped to [-1, 1]; NaN when the cache is empty
 *   resp_score  prefix-embedding cosine with entry idx, clamped to [-1, 1];
 *               quiet NaN (0x7FC00000) when stage 2 did not run
 *   decision    LACACHE_MISS / REJECT / HIT / HIT_EXACT
 * Similarities are dot products of the bfloat16-rounded normalised vectors,
 * accumulated in float32.  B == 0 is a no-op.  Only for a cache with m = 1
 * (else LACACHE_EINVAL).
 * A lookup (this call and lacache_lookup_ensemble) only enqueues kernels on
 * the stream: no allocation, memory set, copy or host synchronisation.  It
 * can therefore be captured into a HIP graph (with profiling off) and
 * replayed.  A captured lookup keeps what was fixed at capture time: the
 * argument pointers, B, k, the thresholds, the number of stored entries and
 * the stage-1 kernel chosen for them.  Entries inserted after the capture
 * are not searched until the lookup is captured again.
 */
int lacache_lookup(lacache_t h, const void *queries, const void *lookahead_emb, const int32_t *lookahead_tokens,
                   int32_t B, float tau_q, float tau_r, int32_t k, int32_t *idx, float *score, float *resp_score,
                   int32_t *decision, void *stream);

/*
 * lacache_lookup for any m (Section 4.4 ensemble):
 *   lookahead_emb  HOST array of m device pointers, lookahead_emb[i] being
 *                  [B][d_resp[i]] (cache dtype): the lookahead prefix under model i
 *   tau_r          HOST array of m finite stage-2 thresholds, one per model
 *   resp_score     [B][m]: cosine of each model's prefix embeddings, clamped to
 *                  [-1, 1]; quiet NaN in every column when stage 2 did not run
 * decision is HIT_EXACT when the k tokens are identical, HIT when every
 * model's cosine is >= its tau_r[i], REJECT otherwise, MISS on a stage-1
 * miss.  Every other argument and output is as in lacache_lookup.
 */
int lacache_lookup_ensemble(lacache_t h, const void *queries, const void *const *lookahead_emb,
                            const int32_t *lookahead_tokens, int32_t B, float tau_q, const float *tau_r, int32_t k,
                            int32_t *idx, float *score, float *resp_score, int32_t *decision, void *stream);

/* Number of entries inserted so far (host-side count); -1 for a NULL handle. */
int64_t lacache_size(lacache_t h);

/*
 * Copy entries first .. first+n-1 of the store out, as stored: keys_bf16 is
 * [n][d] and emb_bf16 [n][d_resp[0]] bfloat16 bit patterns (prefix model 0),
 * tokens [n][k_cap] int32.  Any of the three may be NULL to skip it.
 * Requires 0 <= first, n >= 0, first + n <= size.  For inspection and tests.
 */
int lacache_export(lacache_t h, int64_t first, int32_t n, uint16_t *keys_bf16, uint16_t *emb_bf16, int32_t *tokens,
                   void *stream);

/* As lacache_export, for the stored prefix embeddings of model 0 <= model < m: emb_bf16 is [n][d_resp[model]]. */
int lacache_export_prefix(lacache_t h, int32_t model, int64_t first, int32_t n, uint16_t *emb_bf16, void *stream);

/*
 * Threshold calibration from benign pairs (Appendix A.2: tau_c = min(0.80, P5)
 * over the cosines of benign paraphrase pairs, tau_a = min(0.70, P10) over the
 * cosines of their response prefixes).
 *   which       -1: the pairs are key-model vectors (dimension d);
 *               0 <= which < m: vectors of prefix model `which` (d_resp[which])
 *   a, b        [n][dim] (cache dtype): pair j is (a[j], b[j]);
 *               1 <= n <= 2^32 - 1 (the selection counts ranks in 32 bits)
 *   percentile  0 .. 100; the percentile is linear between the closest ranks,
 *               h = (n - 1) * percentile / 100, from the order statistics
 *               floor(h) and floor(h) + 1 (computed in double)
 *   cap         finite upper cap of the threshold
 * Outputs (device): sims [n] float, the pair cosines exactly as the lookup
 * computes similarities (normalised, bfloat16-rounded vectors, float32 sums,
 * clamped to [-1, 1]); tau [2] float: tau[0] = the percentile of sims,
 * tau[1] = min(cap, tau[0]).  Uses the handle's calibration scratch, so
 * calls on one handle must be ordered on one stream.  EINVAL for an invalid
 * which, n, percentile or cap, or a NULL pointer.
 */
int lacache_calibrate(lacache_t h, int32_t which, const void *a, const void *b, int64_t n, float percentile,
                      float cap, float *sims, float *tau, void *stream);

/*
 * lacache_calibrate without a handle and without allocating: for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation).  The same pair cosines, selection
 * and outputs as lacache_calibrate, for n pairs of d-dimensional vectors of
 * the given dtype, on the calling thread's current device and on `stream`.
 * The selection's scratch (its state and two 2048-bin histograms, 16.6 KB)
 * is a static array of the library's device image: one copy per GPU, held
 * until the process ends, its size fixed whatever n and d are; it is cleared
 * by the call itself, so calls ordered on one stream are independent, while
 * calls that overlap on one GPU (other streams, other threads) race on it.
 *   1 <= d <= 16384; 1 <= n <= 2^32 - 1; 0 <= percentile <= 100; cap finite;
 * EINVAL otherwise or for a NULL pointer; EHIP for a HIP failure.
 */
int lacache_calibrate_noalloc(const void *a, const void *b, lacache_dtype dtype, int32_t d, int64_t n,
                              float percentile, float cap, float *sims, float *tau, void *stream);

/*
 * Speculative-decoding acceptance after a miss or a rejected lookahead
 * (Section 4.3): the k draft tokens of the draft model g are verified by the
 * target model f in one forward pass; token t_j is accepted when
 * P_f(t_j) >= P_g(t_j), from the first token on, and f takes over at the
 * first failure.  Needs no cache handle; runs on the calling thread's current
 * device.
 *   logits        [B][k][V] (dtype): f's logits at each draft position
 *   draft_tokens  [B][k] int32 draft token IDs; an ID outside [0, V) has probability 0
 *   p_draft       [B][k] float: P_g of each draft token
 *   1 <= V, 0 <= B, 1 <= k <= 4096
 * Outputs: p_target [B][k] float = softmax(logits[b][j])[t_j] (float32
 * arithmetic, max-shifted exponentials); accept_len [B] int32 = the number
 * of leading positions with p_target >= p_draft (0 .. k).  Every row needs at
 * least one finite logit.  B == 0 is a no-op.
 */
int lacache_accept_length(const void *logits, lacache_dtype dtype, int32_t V, const int32_t *draft_tokens,
                          const float *p_draft, int32_t B, int32_t k, int32_t *accept_len, float *p_target,
                          void *stream);

/*
 * Locality-sensitive index for stage 1 (Section 3, Eq. (1): the cache key is
 * an LSH of the embedding, colliding with probability above p1 for close
 * pairs and below p2 for far ones; Algorithm 1 searches the cache with it).
 * Random hyperplanes, the LSH family of cosine distance: bit i of a stored or
 * query vector z (normalised and bfloat16-rounded) is 1 when the projection
 * r_i . z (bf16 products, float32 sums) is >= 0; bits are packed 32 to a word,
 * bit i in word i / 32 at position i % 32.
 *
 * lacache_enable_lsh: hyperplanes [bits][d] bfloat16 (device; not
 * normalised; their entries are the random numbers the index draws), bits a
 * multiple of 32 in 32 .. 256, max_candidates 1 .. 65536 entries kept per
 * query.  Allocates the index (signatures [capacity][bits / 32] and per-query
 * candidate lists), waits for `stream`, and computes the signatures of every
 * stored entry; later inserts add theirs.  Calling it again replaces the index.
 */
int lacache_enable_lsh(lacache_t h, int32_t bits, const uint16_t *hyperplanes, int32_t max_candidates, void *stream);

/*
 * lacache_lookup with the LSH index as stage 1 (caches with one prefix model):
 * the candidates of a query are the entries whose signature differs from the
 * query's in at most `radius` bits (0 .. bits; 0 is equality of hash keys,
 * bits makes every entry a candidate); among them the entry of highest exact
 * similarity (lowest index on ties) is the stage-1 result, then the
 * threshold and stage 2 as in lacache_lookup.  With no candidate: idx -1,
 * score NaN, MISS.  n_cand [B] int32 receives each query's candidate count;
 * a count above max_candidates means only max_candidates of them (in no
 * particular order) were ranked.  Other arguments and outputs as in
 * lacache_lookup.  LACACHE_EINVAL if the index is not enabled.
 */
int lacache_lookup_lsh(lacache_t h, const void *queries, const void *lookahead_emb, const int32_t *lookahead_tokens,
                       int32_t B, float tau_q, float tau_r, int32_t k, int32_t radius, int32_t *idx, float *score,
                       float *resp_score, int32_t *decision, int32_t *n_cand, void *stream);

/* Copy the LSH signatures of entries first .. first+n-1 ([n][bits / 32] uint32, device) out. */
int lacache_export_signatures(lacache_t h, int64_t first, int32_t n, uint32_t *sig, void *stream);

/*
 * Batch-size crossover of stage 1: batches of at most b_small queries use the
 * bandwidth-bound streaming kernel, larger ones the matrix-core GEMM kernel.
 * The streaming kernel runs up to four groups of 64 queries (fewer queries
 * per group for d > 1152).  b_small is -1, or from 0 up to the streaming
 * kernel's largest batch (256 for d <= 1152); anything else is EINVAL.
 * 0 sends every batch to the GEMM kernel.  -1 (the default) lets each call
 * choose from the number of stored entries n and the padded dimension d_pad:
 * one query group when n * d_pad >= 2^29, two when n * d_pad >= 2^27, three
 * below that.  Each added group costs the streaming kernel a share of the
 * contraction on every CU, so the more keys there are, the sooner the GEMM
 * kernel is faster.  Both kernels accumulate every score with the same
 * matrix instruction sequence, so their results are bit-identical.
 */
int lacache_set_small_batch(lacache_t h, int32_t b_small);

/*
 * Timing of the stage-1 kernel.  With every = n > 0, the 1st, (n+1)-th,
 * (2n+1)-th ... stage-1 launch from now on (one per lookup, or per chunk of
 * max_batch queries) is timed: the launch goes through hipExtLaunchKernel
 * with a HIP event pair that takes the kernel's own start and end times, on
 * the lookup's stream.  every = 0 stops timing.  profile_read waits for
 * those events, returns the total elapsed milliseconds and the number of
 * launches timed (host pointers), and clears the record; calling
 * lacache_profile also clears it.  The events are created here (256 pairs,
 * more only when a window outgrows them) and reused.  Timing every launch
 * costs a few microseconds per lookup, which matters only for lookups that
 * take tens of microseconds; sampling every n-th launch spreads that cost.
 * Errors: EINVAL for a null handle or pointer or every < 0, EHIP.
 */
int lacache_profile(lacache_t h, int32_t every);
int lacache_profile_read(lacache_t h, double *stage1_ms, int64_t *lookups);

/*
 * Health counter of the large-batch stage 1.  Its GEMM kernel reports, per
 * query, the 16-row group holding the best score; the exact row is then
 * recovered by recomputing that group's 16 scores with the same matrix
 * instruction sequence and taking the lowest row whose score equals the
 * reported one (lowest index on ties, Algorithm 1's single hit entry).  If no
 * row reproduces the score, the lowest row at the recomputed maximum is
 * taken instead, so the lookup still names a valid entry, and this counter
 * is incremented.  *count (host pointer) receives the number of such queries
 * since create; it is 0 in correct operation.  Synchronises the device.
 * Errors: EINVAL for a null handle or pointer, EHIP.
 */
int lacache_replay_fallbacks(lacache_t h, int64_t *count);

/* Static text for a return code. */
const char *lacache_strerror(int code);

#ifdef __cplusplus
}
#endif

#endif /* LACACHE_H */
