"""Seeded synthetic workloads shaped like the paper's lookup traffic.

The paper evaluates pairwise on MS MARCO / Natural Questions with BGE-large
(1024-d) and MiniLM (384-d) embeddings (Section 5.1); none of those inputs are
available, so every array here is synthetic:

* cache keys and response-prefix embeddings: unit(N(0, I)) rows (or, for the
  clustered variant, unit(0.8 c_m + 0.6 u) around 10,000 random centroids);
* token IDs: uniform over the vocabulary;
* queries, one of three classes --
  benign    : a planted near-duplicate of entry i at cosine c, whose lookahead
              is entry i's own response prefix (same tokens, same embedding);
  collision : a planted near-duplicate of entry i whose lookahead is unrelated
              (random tokens, independent embedding) -- the cache-collision
              attack of Section 3 in its simplest form;
  miss      : a fresh vector.
  A planted query is q = c*x + sqrt(1-c^2)*v with x = unit(key_i) and v a
  random unit vector orthogonal to x, so cos(q, key_i) = c before rounding.

Randomness: NumPy PCG64, one independent stream per (array, 4096-row chunk),
derived from SeedSequence(seed, spawn_key=(stream, chunk)), so the arrays do
not depend on how the caller batches or threads the generation.

Input dtypes: float32, or bfloat16 passed as uint16 bit patterns (rounded to
nearest-even from float32 by torch's CPU conversion).
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

GEN_CHUNK = 4096
F32, BF16 = 0, 1
CLS_MISS, CLS_BENIGN, CLS_COLLISION = 0, 1, 2

# stream identifiers for SeedSequence spawn keys
_S_KEYS, _S_EMB, _S_TOK, _S_CENT, _S_ASSIGN = 0, 1, 2, 3, 4
_S_QCLASS, _S_QVEC, _S_QLOOK, _S_DUP = 10, 11, 12, 13
_S_ENS_EMB, _S_ENS_LOOK = 20, 40       # + model index

# Prefix-embedding dimensions of the lookahead ensemble the paper evaluates
# (Section 5.4, number of lookahead checks): BGE-large, MiniLM, MPNet,
# Qwen3-Embedding-0.6B.
ENSEMBLE_DIMS = (1024, 384, 768, 1024)


@dataclasses.dataclass(frozen=True)
class Spec:
    name: str
    N: int
    d: int
    in_dtype: int          # F32 or BF16
    k_cap: int
    vocab: int
    B: int
    frac_benign: float
    frac_collision: float
    cos_lo: float
    cos_hi: float
    tau_q: float
    tau_r: float
    k: int
    seed: int
    n_dup: int = 0             # exact-duplicate key pairs (j < i, key_i is a bit copy of key_j)
    n_dup_queries: int = 0     # benign queries aimed at duplicate pairs (expect entry j)
    n_centroids: int = 0       # >0: clustered keys unit(0.8 c + 0.6 u)
    paper_shaped: bool = False  # benign / collision lookahead distributions from the paper's statistics


# The five workloads the lookup is measured and checked on, plus one whose
# value distributions follow the statistics the paper prints:
#   benign paraphrase cosine P5 = 0.857 (Appendix A.2, tau_c calibration),
#   benign response-prefix cosine P10 = 0.734 (Appendix A.2, tau_a table),
#   adaptive-attack prefix similarity mean 0.49 (Table 3),
#   thresholds tau_c = 0.80, tau_a = 0.70, k = 20 (Appendix A.2; Section 5.1).
CONFIGS = {
    "tiny": Spec("tiny", 10_000, 384, F32, 8, 32000, 64, 1 / 3, 1 / 3, 0.95, 0.95, 0.9, 0.85, 8, 0),
    "mid": Spec("mid", 100_000, 768, BF16, 8, 32000, 256, 1 / 3, 1 / 3, 0.85, 0.99, 0.9, 0.85, 8, 1),
    "mid_paper": Spec("mid_paper", 100_000, 1024, BF16, 20, 128256, 256, 1 / 3, 1 / 3, 0.86, 0.99, 0.80, 0.70,
                      20, 5, paper_shaped=True),
    "serve_small": Spec("serve_small", 1_000_000, 768, BF16, 16, 128256, 4096, 0.4, 0.1, 0.92, 0.99, 0.9, 0.85,
                        16, 2),
    "serve_large": Spec("serve_large", 1_000_000, 768, BF16, 16, 128256, 4096, 0.4, 0.1, 0.92, 0.99, 0.9, 0.85,
                        16, 3, n_dup=1000, n_dup_queries=256),
    "large": Spec("large", 4_000_000, 1024, BF16, 32, 128256, 1024, 0.4, 0.1, 0.92, 0.99, 0.9, 0.85, 32, 4,
                  n_centroids=10_000),
}
# serve_small is timed in calls of 16 queries drawn from its pool of 4096.
SERVE_SMALL_CALL_B = 16


def spec(name: str, **overrides) -> Spec:
    return dataclasses.replace(CONFIGS[name], **overrides)


@dataclasses.dataclass
class Workload:
    spec: Spec
    keys: np.ndarray        # [N][d] float32 or uint16 (bf16 bits)
    emb: np.ndarray         # [N][d]
    tokens: np.ndarray      # [N][k_cap] int32
    queries: np.ndarray     # [B][d]
    la_emb: np.ndarray      # [B][d]
    la_tok: np.ndarray      # [B][k] int32
    cls: np.ndarray         # [B] CLS_*
    target: np.ndarray      # [B] planted entry (-1 for misses)
    cos: np.ndarray         # [B] planted cosine (nan for misses)
    dup_pairs: np.ndarray   # [n_dup][2] (j, i), j < i

    @property
    def in_dtype(self) -> int:
        return self.spec.in_dtype


def _rng(seed: int, stream: int, chunk: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=(stream, chunk))))


def _unit_rows(x: np.ndarray) -> np.ndarray:
    x = x.astype(np.float64)
    n = np.linalg.norm(x, axis=-1, keepdims=True)
    n[n == 0] = 1.0
    return x / n


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float -> bfloat16 bit patterns (uint16) via torch's CPU conversion (nearest-even)."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def bf16_bits_to_f64(h: np.ndarray) -> np.ndarray:
    return (np.asarray(h, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _cast(x64: np.ndarray, in_dtype: int) -> np.ndarray:
    if in_dtype == F32:
        return x64.astype(np.float32)
    return to_bf16_bits(x64.astype(np.float32))


def as_f64(x: np.ndarray, in_dtype: int) -> np.ndarray:
    return bf16_bits_to_f64(x) if in_dtype == BF16 else np.asarray(x, np.float64)


def _centroids(sp: Spec) -> np.ndarray:
    g = _rng(sp.seed, _S_CENT).standard_normal((sp.n_centroids, sp.d))
    return _unit_rows(g)


def _orth_unit(rng: np.random.Generator, x: np.ndarray) -> np.ndarray:
    """Random unit vectors orthogonal to the unit rows of x."""
    g = rng.standard_normal(x.shape)
    g -= np.sum(g * x, axis=-1, keepdims=True) * x
    return _unit_rows(g)


def _entry_chunk(sp: Spec, c: int, cent: np.ndarray | None, rows: int):
    r0 = c * GEN_CHUNK
    n = min(GEN_CHUNK, rows - r0)
    if cent is None:
        kx = _unit_rows(_rng(sp.seed, _S_KEYS, c).standard_normal((GEN_CHUNK, sp.d), dtype=np.float32)[:n])
    else:
        m = _rng(sp.seed, _S_ASSIGN, c).integers(0, sp.n_centroids, GEN_CHUNK)[:n]
        cm = cent[m]
        kx = 0.8 * cm + 0.6 * _orth_unit(_rng(sp.seed, _S_KEYS, c), cm)
    ex = _unit_rows(_rng(sp.seed, _S_EMB, c).standard_normal((GEN_CHUNK, sp.d), dtype=np.float32)[:n])
    tok = _rng(sp.seed, _S_TOK, c).integers(0, sp.vocab, (GEN_CHUNK, sp.k_cap), dtype=np.int32)[:n]
    return r0, _cast(kx, sp.in_dtype), _cast(ex, sp.in_dtype), tok


def entries(sp: Spec, first: int, n: int, threads: int | None = None):
    """Rows [first, first+n) of the entry stream: (keys, emb, tokens).

    The stream extends past N: rows >= N are the entries of later insert batches.
    """
    dt = np.float32 if sp.in_dtype == F32 else np.uint16
    keys = np.empty((n, sp.d), dt)
    emb = np.empty((n, sp.d), dt)
    tok = np.empty((n, sp.k_cap), np.int32)
    cent = _centroids(sp) if sp.n_centroids else None
    c0, c1 = first // GEN_CHUNK, (first + n + GEN_CHUNK - 1) // GEN_CHUNK
    end = first + n

    def work(c):
        r0, k, e, t = _entry_chunk(sp, c, cent, (c + 1) * GEN_CHUNK)
        lo, hi = max(r0, first), min(r0 + GEN_CHUNK, end)
        keys[lo - first:hi - first] = k[lo - r0:hi - r0]
        emb[lo - first:hi - first] = e[lo - r0:hi - r0]
        tok[lo - first:hi - first] = t[lo - r0:hi - r0]

    threads = threads or min(16, os.cpu_count() or 1)
    if c1 - c0 <= 1:
        for c in range(c0, c1):
            work(c)
    else:
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(work, range(c0, c1)))
    return keys, emb, tok


def _dup_pairs(sp: Spec) -> np.ndarray:
    if not sp.n_dup:
        return np.zeros((0, 2), np.int64)
    rng = _rng(sp.seed, _S_DUP)
    picks = rng.choice(sp.N, size=2 * sp.n_dup, replace=False)
    a, b = picks[:sp.n_dup], picks[sp.n_dup:]
    return np.stack([np.minimum(a, b), np.maximum(a, b)], axis=1)


def _class_counts(sp: Spec, B: int):
    nb = int(round(B * sp.frac_benign))
    nc = int(round(B * sp.frac_collision))
    return nb, nc, B - nb - nc


def queries(sp: Spec, keys: np.ndarray, emb: np.ndarray, tokens: np.ndarray, dup_pairs: np.ndarray,
            B: int | None = None, N: int | None = None, stream_chunk: int = 0, recent=None, recent_frac=0.1):
    """Draw B queries with their lookahead inputs against the first N entries.

    recent = (lo, hi): a fraction recent_frac of the planted queries aims at rows lo .. hi-1 (the latest
    insert batch of an interleaved insert/lookup schedule).
    """
    B = sp.B if B is None else B
    N = keys.shape[0] if N is None else N
    d, k = sp.d, sp.k
    rng = _rng(sp.seed, _S_QCLASS, stream_chunk)
    vrng = _rng(sp.seed, _S_QVEC, stream_chunk)
    lrng = _rng(sp.seed, _S_QLOOK, stream_chunk)
    nb, nc, nm = _class_counts(sp, B)
    cls = np.array([CLS_BENIGN] * nb + [CLS_COLLISION] * nc + [CLS_MISS] * nm, np.int32)
    target = np.full(B, -1, np.int64)
    expect = np.full(B, -1, np.int64)
    planted = cls != CLS_MISS
    np_ = int(planted.sum())
    target[planted] = rng.integers(0, max(N, 1), np_) if N > 0 else -1
    if len(dup_pairs):
        # a random target that is the later copy of a duplicate pair is the earlier copy's key too
        later = dict(zip(dup_pairs[:, 1].tolist(), dup_pairs[:, 0].tolist()))
        target = np.array([later.get(int(t), int(t)) for t in target], np.int64)
    if recent is not None and np_:
        pl_idx = np.nonzero(planted)[0]
        nr = int(round(recent_frac * np_))
        sel = rng.choice(pl_idx, size=nr, replace=False)
        target[sel] = rng.integers(recent[0], recent[1], nr)
    # benign queries aimed at exact-duplicate pairs: near key i (== key j), carrying j's lookahead
    nd = min(sp.n_dup_queries, nb, len(dup_pairs))
    dsel = rng.choice(len(dup_pairs), size=nd, replace=False) if nd else np.zeros(0, np.int64)
    if nd:
        target[:nd] = dup_pairs[dsel, 1]
    cos = np.full(B, np.nan)
    cos[planted] = rng.uniform(sp.cos_lo, sp.cos_hi, np_) if sp.cos_hi > sp.cos_lo else sp.cos_lo
    if sp.paper_shaped:
        # attack queries land in the adaptive-attack band rather than the benign paraphrase band
        cos[cls == CLS_COLLISION] = rng.uniform(0.80, 0.95, nc)

    qv = np.empty((B, d))
    if np_:
        x = _unit_rows(as_f64(keys[target[planted]], sp.in_dtype))
        c = cos[planted][:, None]
        qv[planted] = c * x + np.sqrt(1 - c * c) * _orth_unit(vrng, x)
    if nm:
        if sp.n_centroids:
            cent = _centroids(sp)
            cm = cent[vrng.integers(0, sp.n_centroids, nm)]
            qv[~planted] = 0.8 * cm + 0.6 * _orth_unit(vrng, cm)
        else:
            qv[~planted] = _unit_rows(vrng.standard_normal((nm, d)))

    la_tok = lrng.integers(0, sp.vocab, (B, k), dtype=np.int32)
    la = _unit_rows(lrng.standard_normal((B, d)))
    ben = np.nonzero(cls == CLS_BENIGN)[0]
    src = target.copy()
    if nd:
        src[:nd] = dup_pairs[dsel, 0]       # j's prefix: the tie must resolve to the lower index
    expect[planted] = src[planted]
    if len(ben):
        la_tok[ben] = tokens[src[ben], :k]
        e_src = as_f64(emb[src[ben]], sp.in_dtype)
        if sp.paper_shaped:
            pos = lrng.integers(0, k, len(ben))
            la_tok[ben, pos] = (la_tok[ben, pos] + 1 + lrng.integers(0, sp.vocab - 1, len(ben))) % sp.vocab
            e = _unit_rows(e_src)
            rho = lrng.uniform(0.70, 0.98, len(ben))[:, None]
            la[ben] = rho * e + np.sqrt(1 - rho * rho) * _orth_unit(lrng, e)
        else:
            la[ben] = e_src
    col = np.nonzero(cls == CLS_COLLISION)[0]
    if sp.paper_shaped and len(col):
        e = _unit_rows(as_f64(emb[target[col]], sp.in_dtype))
        rho = np.clip(lrng.normal(0.49, 0.09, len(col)), -0.99, 0.99)[:, None]
        la[col] = rho * e + np.sqrt(1 - rho * rho) * _orth_unit(lrng, e)

    perm = rng.permutation(B)
    return dict(queries=_cast(qv[perm], sp.in_dtype), la_emb=_cast(la[perm], sp.in_dtype), la_tok=la_tok[perm],
                cls=cls[perm], target=expect[perm], cos=cos[perm])


def ensemble_entries(sp: Spec, d_models, first: int, n: int, threads: int | None = None):
    """Rows [first, first+n) of each prefix model's stored embeddings: one [n][d_i] array per model,
    unit(N(0, I)) rows cast to the spec's input dtype."""
    out = [np.empty((n, di), np.float32 if sp.in_dtype == F32 else np.uint16) for di in d_models]
    c0, c1 = first // GEN_CHUNK, (first + n + GEN_CHUNK - 1) // GEN_CHUNK

    def work(job):
        i, c = job
        r0 = c * GEN_CHUNK
        x = _rng(sp.seed, _S_ENS_EMB + i, c).standard_normal((GEN_CHUNK, d_models[i]), dtype=np.float32)
        lo, hi = max(r0, first), min(r0 + GEN_CHUNK, first + n)
        out[i][lo - first:hi - first] = _cast(_unit_rows(x[lo - r0:hi - r0]), sp.in_dtype)

    jobs = [(i, c) for i in range(len(d_models)) for c in range(c0, c1)]
    if len(jobs) <= 1:
        for j in jobs:
            work(j)
    else:
        with ThreadPoolExecutor(threads or min(16, os.cpu_count() or 1)) as ex:
            list(ex.map(work, jobs))
    return out


def ensemble_lookahead(sp: Spec, d_models, stored, tokens, q: dict, stream_chunk: int = 0, frac_substituted=0.5,
                       frac_fooled=0.3):
    """Lookahead embeddings of a query batch under each prefix model of an ensemble.

    q is the dict queries() returns (its cls, target and la_tok); stored[i] holds model i's prefix
    embeddings of every entry and tokens the entries' prefix tokens.  Per query and model the lookahead is rho * e + sqrt(1 - rho^2) * v around
    the target entry's stored prefix e (v a random unit vector orthogonal to e): benign queries draw
    rho ~ U[0.70, 0.98] (the benign prefix-cosine band, P10 near the 0.70 threshold, Appendix A.2);
    collisions draw rho ~ N(0.49, 0.09) (Table 3), except that a fraction frac_fooled of them has one
    model, chosen at random, fooled at rho ~ U[0.75, 0.95] -- the case an ensemble exists for
    (Section 4.4).  Misses get unrelated vectors.  Benign queries carry their target's first k tokens,
    except that a fraction frac_substituted of them has one token replaced, so that the embedding models,
    not identical tokens, decide them.
    Returns (list of [B][d_i] arrays, la_tok).
    """
    rng = _rng(sp.seed, _S_ENS_LOOK, stream_chunk)
    cls, target = q["cls"], q["target"]
    la_tok = np.array(q["la_tok"], np.int32, copy=True)
    B, k = la_tok.shape
    m = len(d_models)
    ben = cls == CLS_BENIGN
    col = cls == CLS_COLLISION
    la_tok[ben] = tokens[target[ben], :k]
    sub = ben & (rng.random(B) < frac_substituted)
    pos = rng.integers(0, k, B)
    bump = 1 + rng.integers(0, sp.vocab - 1, B)
    la_tok[sub, pos[sub]] = (la_tok[sub, pos[sub]] + bump[sub]) % sp.vocab
    fooled = np.where(col & (rng.random(B) < frac_fooled), rng.integers(0, m, B), -1)
    out = []
    for i, di in enumerate(d_models):
        lrng = _rng(sp.seed, _S_ENS_LOOK + 1 + i, stream_chunk)
        la = _unit_rows(lrng.standard_normal((B, di)))
        planted = ben | col
        if planted.any():
            e = _unit_rows(as_f64(stored[i][target[planted]], sp.in_dtype))
            rho = np.where(ben[planted], lrng.uniform(0.70, 0.98, B)[planted],
                           np.clip(lrng.normal(0.49, 0.09, B)[planted], -0.99, 0.99))
            hit = fooled[planted] == i
            rho = np.where(hit, lrng.uniform(0.75, 0.95, B)[planted], rho)[:, None]
            la[planted] = rho * e + np.sqrt(1 - rho * rho) * _orth_unit(lrng, e)
        out.append(_cast(la, sp.in_dtype))
    return out, la_tok


_S_CAL_X, _S_CAL_V, _S_CAL_C = 60, 61, 62


def calibration_pairs(n: int, d: int, cos_lo: float, cos_hi: float, seed: int, in_dtype: int = BF16,
                      threads: int | None = None):
    """n benign pairs for threshold calibration: x_j = unit(N(0, I)) and y_j = c_j x_j + sqrt(1 - c_j^2) v_j
    with v_j a random unit vector orthogonal to x_j and c_j ~ U[cos_lo, cos_hi], so cos(x_j, y_j) = c_j before
    rounding (the paraphrase-pair query cosines of Appendix A.2 lie in such a band: P5 = 0.857 for BGE).
    Returns (a, b), [n][d] in the given input dtype."""
    dt = np.float32 if in_dtype == F32 else np.uint16
    a = np.empty((n, d), dt)
    b = np.empty((n, d), dt)

    def work(c):
        r0 = c * GEN_CHUNK
        r1 = min(n, r0 + GEN_CHUNK)
        m = r1 - r0
        x = _unit_rows(_rng(seed, _S_CAL_X, c).standard_normal((m, d), dtype=np.float32))
        v = _orth_unit(_rng(seed, _S_CAL_V, c), x)
        cs = _rng(seed, _S_CAL_C, c).uniform(cos_lo, cos_hi, (m, 1))
        a[r0:r1] = _cast(x, in_dtype)
        b[r0:r1] = _cast(cs * x + np.sqrt(1 - cs * cs) * v, in_dtype)

    chunks = range((n + GEN_CHUNK - 1) // GEN_CHUNK)
    with ThreadPoolExecutor(threads or min(16, os.cpu_count() or 1)) as ex:
        list(ex.map(work, chunks))
    return a, b


_S_SD_LOG, _S_SD_TOP, _S_SD_TOK, _S_SD_PD = 70, 71, 72, 73


def draft_verification(B: int, k: int, V: int, seed: int, in_dtype: int = BF16, frac_top: float = 0.9,
                       threads: int | None = None):
    """Inputs of the speculative-decoding acceptance step (Section 4.3) for B queries with k draft tokens.

    The target model's logits at each draft position are N(0, 1) over the vocabulary with one favoured
    token raised by U[12, 16] (a peaked next-token distribution).  A fraction frac_top of the draft tokens
    is the favoured token, drawn with a draft probability U[0.1, 0.6]; the rest are uniform random tokens
    with draft probability U[0, 2e-6].  Returns (logits [B][k][V] in the input dtype, tokens [B][k] int32,
    p_draft [B][k] float32)."""
    rows = B * k
    logits = np.empty((rows, V), np.float32 if in_dtype == F32 else np.uint16)
    top = _rng(seed, _S_SD_TOP).integers(0, V, rows)
    boost = _rng(seed, _S_SD_TOP, 1).uniform(12.0, 16.0, rows)
    chunk = max(1, (1 << 22) // V)

    def work(c):
        r0, r1 = c * chunk, min(rows, (c + 1) * chunk)
        x = _rng(seed, _S_SD_LOG, c).standard_normal((r1 - r0, V), dtype=np.float32)
        x[np.arange(r1 - r0), top[r0:r1]] += boost[r0:r1].astype(np.float32)
        logits[r0:r1] = x if in_dtype == F32 else to_bf16_bits(x)

    with ThreadPoolExecutor(threads or min(16, os.cpu_count() or 1)) as ex:
        list(ex.map(work, range((rows + chunk - 1) // chunk)))
    g = _rng(seed, _S_SD_TOK)
    fav = g.random(rows) < frac_top
    tokens = np.where(fav, top, g.integers(0, V, rows)).astype(np.int32)
    pr = _rng(seed, _S_SD_PD)
    p_draft = np.where(fav, pr.uniform(0.1, 0.6, rows), pr.uniform(0.0, 2e-6, rows)).astype(np.float32)
    return logits.reshape(B, k, V), tokens.reshape(B, k), p_draft.reshape(B, k)


_S_HYP = 80


def hyperplanes(bits: int, d: int, seed: int) -> np.ndarray:
    """Random hyperplanes of a locality-sensitive index for cosine distance: [bits][d] N(0, 1) entries as
    bfloat16 bit patterns (uint16).  They are the random numbers the index draws, passed in as an input."""
    return to_bf16_bits(_rng(seed, _S_HYP).standard_normal((bits, d), dtype=np.float32))


def generate(sp: Spec | str, threads: int | None = None, **overrides) -> Workload:
    """Build the cache contents and one batch of queries for a spec."""
    if isinstance(sp, str):
        sp = spec(sp, **overrides)
    elif overrides:
        sp = dataclasses.replace(sp, **overrides)
    keys, emb, tok = entries(sp, 0, sp.N, threads)
    dup = _dup_pairs(sp) if sp.N > 1 else np.zeros((0, 2), np.int64)
    if len(dup):
        keys[dup[:, 1]] = keys[dup[:, 0]]
    q = queries(sp, keys, emb, tok, dup)
    return Workload(spec=sp, keys=keys, emb=emb, tokens=tok, queries=q["queries"], la_emb=q["la_emb"],
                    la_tok=q["la_tok"], cls=q["cls"], target=q["target"], cos=q["cos"], dup_pairs=dup)


__all__ = ["Spec", "Workload", "CONFIGS", "spec", "generate", "entries", "queries", "to_bf16_bits",
           "bf16_bits_to_f64", "as_f64", "CLS_MISS", "CLS_BENIGN", "CLS_COLLISION",
           "F32", "BF16", "GEN_CHUNK", "SERVE_SMALL_CALL_B", "ENSEMBLE_DIMS", "ensemble_entries",
           "ensemble_lookahead", "calibration_pairs", "draft_verification", "hyperplanes"]
