/*
 * lacache_oracle.c -- plain CPU oracle for the LaCache two-stage cache lookup.
 *
 * TEST INFRASTRUCTURE ONLY.  The product library never links, loads or calls
 * this file; only the test-suite, the smoke check and the benchmark's CPU
 * baseline do.  It shares no code, header, table or helper with the HIP path.
 *
 * Everything here is computed in IEEE double, slowly and in the most direct
 * order, so that it can be checked against the paper by eye:
 *
 *   quantise  Cosine similarity (Section 3: the distance between embeddings is
 *             e.g. cosine distance; Section 5.1: a hit needs sim >= tau) is the
 *             dot product of L2-normalised vectors.  A vector is normalised in
 *             double and rounded ONCE, to nearest-even, to bfloat16 -- the
 *             precision the cache stores.  A zero vector stays zero.
 *   stage 1   The cached entry whose key has the largest dot product with the
 *             query (lowest index on exact ties) is "the hit" candidate
 *             (Algorithm 1: search the cache with h(x)); it is a hit when the
 *             score, clamped to [-1, 1], is >= tau_q (Section 5.1, cache check
 *             sim(x, x') >= tau_c).
 *   stage 2   Run only for a stage-1 hit (Algorithm 1: the lookahead check sits
 *             inside the hit branch).  The matched entry stores the lookahead
 *             key of its own response prefix (Section 4.2, cache structure
 *             <h(x), [h(f_k(x)), f(x)]>): here the first k token IDs and the
 *             embedding of that prefix.  The lookahead passes when the k tokens
 *             are identical (a deterministic hash of identical input always
 *             agrees) or when the prefix-embedding cosine is >= tau_r
 *             (Section 5.1, lookahead check sim(f_k(x), f_k(x')) >= tau_a).
 *
 *   calibrate Thresholds from benign pairs (Appendix A.2): the p-th percentile
 *             of the pair cosines, capped from above.
 *   accept    Speculative-decoding acceptance after a miss or rejection
 *             (Section 4.3): leading draft tokens with P_f(t) >= P_g(t).
 *   lsh       Stage 1 through a locality-sensitive index (Eq. (1)): random
 *             hyperplane signatures, candidates within a Hamming radius,
 *             exact re-ranking of the candidates.
 *
 * Decision codes: 0 MISS, 1 REJECT (collision detected), 2 HIT, 3 HIT_EXACT.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define LCO_MISS 0
#define LCO_REJECT 1
#define LCO_HIT 2
#define LCO_HIT_EXACT 3

static float quiet_nan(void)
{
    uint32_t u = 0x7FC00000u;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

/* bfloat16 bit pattern -> the exact double it denotes. */
static double widen_bf16(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/*
 * Round a double to the nearest bfloat16 (8 significant bits, 8 exponent
 * bits), ties to even, in ONE rounding step.  The representable grid near |v|
 * has spacing 2^(e-7) where 2^e is the leading bit of |v|; below the smallest
 * normal binade (e < -126) the spacing stays 2^-133 (subnormals).  Scaling by
 * a power of two is exact, so nearbyint() (default mode: to nearest, ties to
 * even) does the only rounding.
 */
uint16_t lco_bf16_rne(double v)
{
    if (isnan(v))
        return 0x7FC0;
    if (isinf(v))
        return signbit(v) ? 0xFF80 : 0x7F80;
    if (v == 0.0)
        return signbit(v) ? 0x8000 : 0x0000;
    int ex;
    frexp(fabs(v), &ex); /* |v| = m * 2^ex with m in [0.5, 1) */
    int lead = ex - 1;   /* weight of the leading bit */
    if (lead < -126)
        lead = -126;
    double r = nearbyint(ldexp(v, 7 - lead));
    double w = ldexp(r, lead - 7);
    if (fabs(w) >= 0x1p128)
        return signbit(v) ? 0xFF80 : 0x7F80;
    float f = (float)w; /* exact: at most 8 significant bits, within float range */
    uint32_t bits;
    memcpy(&bits, &f, sizeof bits);
    return (uint16_t)(bits >> 16);
}

/* Element j of row r of an input matrix, as a double.  dtype 0 = float32, 1 = bfloat16. */
static double read_in(const void *in, int32_t dtype, int64_t r, int32_t d, int32_t j)
{
    if (dtype == 0)
        return (double)((const float *)in)[r * (int64_t)d + j];
    return widen_bf16(((const uint16_t *)in)[r * (int64_t)d + j]);
}

/*
 * L2-normalise each of `rows` rows of length d in double and round each
 * component once to bfloat16.  A zero row gives an all-zero (+0) row.
 * out is [rows][d] bfloat16 bit patterns.
 */
void lco_quantise(const void *in, int32_t dtype, int64_t rows, int32_t d, uint16_t *out)
{
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < rows; ++r) {
        double ss = 0.0;
        for (int32_t j = 0; j < d; ++j) {
            double v = read_in(in, dtype, r, d, j);
            ss += v * v;
        }
        double n = sqrt(ss);
        for (int32_t j = 0; j < d; ++j) {
            uint16_t q = 0;
            if (n != 0.0)
                q = lco_bf16_rne(read_in(in, dtype, r, d, j) / n);
            out[r * (int64_t)d + j] = q;
        }
    }
}

/* Dot product of two bfloat16 rows, accumulated in double in index order. */
double lco_dot(const uint16_t *x, const uint16_t *y, int32_t d)
{
    double s = 0.0;
    for (int32_t j = 0; j < d; ++j)
        s += widen_bf16(x[j]) * widen_bf16(y[j]);
    return s;
}

static float clamp_unit(double s)
{
    float f = (float)s; /* one rounding to float, to nearest */
    if (f < -1.0f)
        f = -1.0f;
    if (f > 1.0f)
        f = 1.0f;
    return f;
}

/*
 * Steps after the top-1 search, for query b against an arbitrary entry i:
 * stage-1 threshold, and stage 2 if it passes.  Returns the decision and
 * writes the clamped stage-1 score and the stage-2 score (NaN if stage 2 did
 * not run).
 */
static int32_t decide_one(const uint16_t *keys, const uint16_t *emb, const int32_t *tokens, int32_t d,
                          int32_t k_cap, const uint16_t *q, const uint16_t *a, const int32_t *u,
                          float tau_q, float tau_r, int32_t k, int64_t i, double *s_out, float *score_out,
                          float *resp_out)
{
    double s = lco_dot(q, keys + i * (int64_t)d, d);
    float score = clamp_unit(s);
    *s_out = s;
    *score_out = score;
    *resp_out = quiet_nan();
    if (!(score >= tau_q))
        return LCO_MISS;
    float r = clamp_unit(lco_dot(a, emb + i * (int64_t)d, d));
    *resp_out = r;
    int tok_eq = 1;
    for (int32_t j = 0; j < k; ++j)
        if (u[j] != tokens[i * (int64_t)k_cap + j])
            tok_eq = 0;
    if (tok_eq)
        return LCO_HIT_EXACT;
    return (r >= tau_r) ? LCO_HIT : LCO_REJECT;
}

/* A scan in index order replaces its best only on a strictly larger score: the lowest index wins exact ties. */
static int better(double s, double best)
{
    return s > best;
}

/*
 * Stage 1 (Algorithm 1, search with the query key): the entry of highest
 * similarity, scanning entries in index order and replacing the best only on a
 * strictly larger score, so the lowest index wins exact ties.  *second
 * receives the best score over every other entry (-inf when N == 1).
 */
static int64_t top1(const uint16_t *keys, int64_t N, int32_t d, const uint16_t *qb, double *best_out,
                    double *second_out)
{
    double best = -INFINITY, second = -INFINITY;
    int64_t bi = -1;
    for (int64_t i = 0; i < N; ++i) {
        double s = lco_dot(qb, keys + i * (int64_t)d, d);
        if (better(s, best)) {
            second = best;
            best = s;
            bi = i;
        } else if (s > second) {
            second = s;
        }
    }
    *best_out = best;
    *second_out = second;
    return bi;
}

/*
 * The full two-stage lookup over quantised inputs.
 *   keys, emb : [N][d]     quantised cache keys and response-prefix embeddings
 *   tokens    : [N][k_cap] stored response-prefix token IDs
 *   q, a      : [B][d]     quantised queries and lookahead embeddings
 *   u         : [B][k]     lookahead token IDs
 * Outputs per query: idx (argmax, -1 when N == 0), score (clamped maximum,
 * NaN when N == 0), resp_score (NaN unless stage 2 ran), decision, and the
 * unclamped double maximum s_best and top-2 margin (best minus the best over
 * every other entry; +inf when N == 1, 0 for exact ties).
 */
void lco_lookup(const uint16_t *keys, const uint16_t *emb, const int32_t *tokens, int64_t N, int32_t d,
                int32_t k_cap, const uint16_t *q, const uint16_t *a, const int32_t *u, int32_t B, float tau_q,
                float tau_r, int32_t k, int32_t *idx, float *score, float *resp_score, int32_t *decision,
                double *s_best, double *margin)
{
#pragma omp parallel for schedule(dynamic, 1)
    for (int32_t b = 0; b < B; ++b) {
        const uint16_t *qb = q + (int64_t)b * d;
        if (N == 0) {
            idx[b] = -1;
            score[b] = quiet_nan();
            resp_score[b] = quiet_nan();
            decision[b] = LCO_MISS;
            s_best[b] = (double)quiet_nan();
            margin[b] = (double)quiet_nan();
            continue;
        }
        double best, second;
        int64_t bi = top1(keys, N, d, qb, &best, &second);
        idx[b] = (int32_t)bi;
        margin[b] = best - second;
        double s;
        decision[b] = decide_one(keys, emb, tokens, d, k_cap, qb, a + (int64_t)b * d, u + (int64_t)b * k, tau_q,
                                 tau_r, k, bi, &s, &score[b], &resp_score[b]);
        s_best[b] = s;
    }
}

/*
 * The same post-search steps evaluated at a caller-chosen entry at[b] for
 * each query b (used to judge a result whose index differs on a near-tie).
 */
void lco_decide(const uint16_t *keys, const uint16_t *emb, const int32_t *tokens, int64_t N, int32_t d,
                int32_t k_cap, const uint16_t *q, const uint16_t *a, const int32_t *u, int32_t B, float tau_q,
                float tau_r, int32_t k, const int32_t *at, double *s_at, float *score, float *resp_score,
                int32_t *decision)
{
#pragma omp parallel for schedule(static)
    for (int32_t b = 0; b < B; ++b) {
        if (at[b] < 0 || at[b] >= N) {
            s_at[b] = (double)quiet_nan();
            score[b] = quiet_nan();
            resp_score[b] = quiet_nan();
            decision[b] = LCO_MISS;
            continue;
        }
        decision[b] = decide_one(keys, emb, tokens, d, k_cap, q + (int64_t)b * d, a + (int64_t)b * d,
                                 u + (int64_t)b * k, tau_q, tau_r, k, at[b], &s_at[b], &score[b], &resp_score[b]);
    }
}

/* Lowest index j <= i whose quantised key is bitwise identical to key i. */
int64_t lco_first_identical(const uint16_t *keys, int64_t N, int32_t d, int64_t i)
{
    if (i < 0 || i >= N)
        return -1;
    const uint16_t *ki = keys + i * (int64_t)d;
    for (int64_t j = 0; j < i; ++j)
        if (memcmp(keys + j * (int64_t)d, ki, (size_t)d * sizeof(uint16_t)) == 0)
            return j;
    return i;
}

/* Element-wise lco_bf16_rne over an array (for the tests of the rounding rule). */
void lco_bf16_rne_array(const double *in, int64_t n, uint16_t *out)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = lco_bf16_rne(in[i]);
}

/* Threads the following parallel regions use (n >= 1); for timing the oracle on one thread. */
void lco_set_num_threads(int n)
{
    if (n >= 1)
        omp_set_num_threads(n);
}

/* Threads an OpenMP parallel region of the oracle uses (reported beside its timings). */
int lco_num_threads(void)
{
    int n = 1;
#pragma omp parallel
    {
#pragma omp single
        n = omp_get_num_threads();
    }
    return n;
}

/*
 * The lookup with an ensemble of m lookahead checks (Section 4.4: m independent
 * indexing functions h_1..h_m; a cache hit is valid only if the key check
 * passes and every h_i(f_k(x)) agrees with h_i(f_k(x'))).  Each entry stores
 * one response-prefix embedding per model i (emb[i], [N][d_i]); each query
 * brings its lookahead embedding under every model (a[i], [B][d_i]) and there
 * is one threshold tau_r[i] per model.  Stage 1 is the same top-1 as
 * lco_lookup.  Stage 2 (on a stage-1 hit only) passes when the first k tokens
 * are identical, or when the cosine under every model reaches its threshold.
 * resp_score is [B][m] (NaN where stage 2 did not run).
 */
void lco_lookup_ensemble(const uint16_t *keys, int64_t N, int32_t d, const uint16_t *q, int32_t B, float tau_q,
                         int32_t m, const uint16_t *const *emb, const int32_t *d_m, const uint16_t *const *a,
                         const float *tau_r, const int32_t *tokens, int32_t k_cap, const int32_t *u, int32_t k,
                         int32_t *idx, float *score, float *resp_score, int32_t *decision)
{
#pragma omp parallel for schedule(dynamic, 1)
    for (int32_t b = 0; b < B; ++b) {
        for (int32_t i = 0; i < m; ++i)
            resp_score[(int64_t)b * m + i] = quiet_nan();
        decision[b] = LCO_MISS;
        if (N == 0) {
            idx[b] = -1;
            score[b] = quiet_nan();
            continue;
        }
        double best, second;
        int64_t bi = top1(keys, N, d, q + (int64_t)b * d, &best, &second);
        idx[b] = (int32_t)bi;
        score[b] = clamp_unit(best);
        if (!(score[b] >= tau_q))
            continue;
        int all_pass = 1;
        for (int32_t i = 0; i < m; ++i) {
            float r = clamp_unit(lco_dot(a[i] + (int64_t)b * d_m[i], emb[i] + bi * (int64_t)d_m[i], d_m[i]));
            resp_score[(int64_t)b * m + i] = r;
            if (!(r >= tau_r[i]))
                all_pass = 0;
        }
        int tok_eq = 1;
        for (int32_t j = 0; j < k; ++j)
            if (u[(int64_t)b * k + j] != tokens[bi * (int64_t)k_cap + j])
                tok_eq = 0;
        decision[b] = tok_eq ? LCO_HIT_EXACT : (all_pass ? LCO_HIT : LCO_REJECT);
    }
}

/*
 * Threshold calibration (Appendix A.2): a threshold is the p-th percentile of
 * the cosine similarities of benign pairs, capped from above --
 * tau_c = min(0.80, P5) over paraphrase-pair query cosines, tau_a = min(0.70,
 * P10) over their response-prefix cosines.  The paper does not say how a
 * percentile between two order statistics is formed; this uses linear
 * interpolation between the closest ranks (h = (n - 1) p / 100, the default
 * of numpy.percentile).
 *
 * lco_threshold_rule: sims[0..n-1] (any order; a sorted copy is made),
 * n >= 1, 0 <= p <= 100.  *P_out receives the percentile, *tau_out min(cap, P).
 */
static int cmp_double_asc(const void *x, const void *y)
{
    double a = *(const double *)x, b = *(const double *)y;
    return (a > b) - (a < b);
}

void lco_threshold_rule(const double *sims, int64_t n, double p, double cap, double *P_out, double *tau_out)
{
    double *x = (double *)malloc((size_t)n * sizeof(double));
    memcpy(x, sims, (size_t)n * sizeof(double));
    qsort(x, (size_t)n, sizeof(double), cmp_double_asc);
    double h = (double)(n - 1) * (p / 100.0);
    int64_t lo = (int64_t)floor(h);
    double P;
    if (lo >= n - 1)
        P = x[n - 1];
    else
        P = x[lo] + (h - (double)lo) * (x[lo + 1] - x[lo]);
    free(x);
    *P_out = P;
    *tau_out = fmin(cap, P);
}

/*
 * The calibration over n pairs of quantised vectors a[j], b[j] ([n][d]): the
 * pair similarity is the cosine the lookup uses (dot product of the
 * normalised, bfloat16-rounded vectors, clamped to [-1, 1]), then the rule above.
 */
void lco_calibrate(const uint16_t *a, const uint16_t *b, int64_t n, int32_t d, double p, double cap,
                   double *sims, double *P_out, double *tau_out)
{
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < n; ++j) {
        double s = lco_dot(a + j * (int64_t)d, b + j * (int64_t)d, d);
        sims[j] = s > 1.0 ? 1.0 : (s < -1.0 ? -1.0 : s);
    }
    lco_threshold_rule(sims, n, p, cap, P_out, tau_out);
}

/*
 * Speculative-decoding acceptance (Section 4.3, speculative decoding): after a
 * miss or a rejected lookahead, the k draft tokens t_1..t_k of the draft model
 * g are verified by the target model f in one forward pass; token t_j is
 * accepted when P_f(t_j) >= P_g(t_j), starting from the first token, and f
 * takes over at the first token that fails.  P_f(t) is the softmax probability
 * of t under f's logits at that position.  The accepted length is the number
 * of leading accepted tokens (0 .. k).
 *
 *   logits      [B][k][V] (dtype 0 float32, 1 bfloat16): f's logits at each draft position
 *   tokens      [B][k] draft token IDs; an ID outside [0, V) has probability 0
 *   p_draft     [B][k] P_g of each draft token (float32)
 * Outputs: accept_len [B]; p_target [B][k] = P_f(t_j) in double (max-shifted
 * exponentials summed in index order).
 */
void lco_accept_length(const void *logits, int32_t dtype, int32_t V, const int32_t *tokens, const float *p_draft,
                       int32_t B, int32_t k, int32_t *accept_len, double *p_target)
{
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t row = 0; row < (int64_t)B * k; ++row) {
        double m = -INFINITY;
        for (int32_t v = 0; v < V; ++v) {
            double x = read_in(logits, dtype, row, V, v);
            if (x > m)
                m = x;
        }
        double s = 0.0;
        for (int32_t v = 0; v < V; ++v)
            s += exp(read_in(logits, dtype, row, V, v) - m);
        int32_t t = tokens[row];
        p_target[row] = (t >= 0 && t < V) ? exp(read_in(logits, dtype, row, V, t) - m) / s : 0.0;
    }
    for (int32_t b = 0; b < B; ++b) {
        int32_t len = 0;
        while (len < k && p_target[(int64_t)b * k + len] >= (double)p_draft[(int64_t)b * k + len])
            ++len;
        accept_len[b] = len;
    }
}

/*
 * Locality-sensitive index for stage 1 (Section 3, Eq. (1): the cache key is an
 * LSH h(z) of the embedding, with collision probability above p1 for close
 * pairs and below p2 for far ones; Algorithm 1 searches the cache with it).
 * For cosine distance the hash family is random hyperplanes: bit i of h(z) is
 * 1 when r_i . z >= 0 (the hyperplanes r_i are inputs, bfloat16 [bits][d]),
 * so two vectors at angle theta agree on a bit with probability 1 - theta/pi.
 * z is the stored (normalised, bfloat16-rounded) vector.  Bits are packed 32
 * to a word, bit i in word i / 32 at position i % 32.
 *
 * lco_simhash: sig [n][bits/32], proj [n][bits] (the projections, in double).
 */
void lco_simhash(const uint16_t *z, int64_t n, int32_t d, const uint16_t *r, int32_t bits, uint32_t *sig,
                 double *proj)
{
    const int32_t words = bits / 32;
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < n; ++j) {
        for (int32_t w = 0; w < words; ++w)
            sig[j * words + w] = 0u;
        for (int32_t i = 0; i < bits; ++i) {
            double p = lco_dot(r + (int64_t)i * d, z + j * (int64_t)d, d);
            proj[j * (int64_t)bits + i] = p;
            if (p >= 0.0)
                sig[j * words + i / 32] |= 1u << (i % 32);
        }
    }
}

/* Number of differing bits of two signatures of `words` words. */
static int32_t hamming(const uint32_t *a, const uint32_t *b, int32_t words)
{
    int32_t h = 0;
    for (int32_t w = 0; w < words; ++w)
        h += __builtin_popcount(a[w] ^ b[w]);
    return h;
}

/*
 * The lookup with the LSH index as stage 1: the candidates of a query are the
 * entries whose signature differs from the query's in at most `radius` bits
 * (radius 0: equal hash keys, as in Algorithm 1; radius = bits: every entry).
 * Among the candidates the entry of highest exact similarity (lowest index on
 * ties) is the stage-1 result; then the threshold and stage 2 as in
 * lco_lookup.  No candidate: idx -1, score NaN, MISS.  n_cand[b] receives the
 * candidate count.
 */
void lco_lookup_lsh(const uint16_t *keys, const uint16_t *emb, const int32_t *tokens, const uint32_t *sig_keys,
                    int64_t N, int32_t d, int32_t k_cap, int32_t bits, const uint16_t *q, const uint32_t *sig_q,
                    const uint16_t *a, const int32_t *u, int32_t B, int32_t radius, float tau_q, float tau_r,
                    int32_t k, int32_t *idx, float *score, float *resp_score, int32_t *decision, int32_t *n_cand)
{
    const int32_t words = bits / 32;
#pragma omp parallel for schedule(dynamic, 1)
    for (int32_t b = 0; b < B; ++b) {
        const uint16_t *qb = q + (int64_t)b * d;
        double best = -INFINITY;
        int64_t bi = -1;
        int32_t cnt = 0;
        for (int64_t i = 0; i < N; ++i) {
            if (hamming(sig_q + (int64_t)b * words, sig_keys + i * words, words) > radius)
                continue;
            ++cnt;
            double s = lco_dot(qb, keys + i * (int64_t)d, d);
            if (better(s, best)) {
                best = s;
                bi = i;
            }
        }
        n_cand[b] = cnt;
        if (bi < 0) {
            idx[b] = -1;
            score[b] = quiet_nan();
            resp_score[b] = quiet_nan();
            decision[b] = LCO_MISS;
            continue;
        }
        idx[b] = (int32_t)bi;
        double s;
        decision[b] = decide_one(keys, emb, tokens, d, k_cap, qb, a + (int64_t)b * d, u + (int64_t)b * k, tau_q,
                                 tau_r, k, bi, &s, &score[b], &resp_score[b]);
    }
}
