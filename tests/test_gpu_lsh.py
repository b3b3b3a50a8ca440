"""GPU parity of stage 1 through the random-hyperplane LSH index (Section 3, Eq. (1)) through the C ABI,
against the CPU oracle's signatures and LSH lookup on the same seeded inputs.

A signature bit is a float decision (the sign of a projection): the GPU sums in float32, the oracle in
double, so a bit whose projection lies within EPS of zero may legitimately differ.  Signatures are compared
bit for bit outside that band; a query's result is compared exactly unless such a near-zero bit could move
an entry across the Hamming radius and that entry could be the top-1 (then it is exempt and counted)."""
from __future__ import annotations

import sys

import numpy as np
import pytest

import oracle
import synth
from tests.compare import MARGIN, SCORE_TOL, compare
from tests.gpu_util import gpu_cache, gpu_lookup, oracle_store, sample_rows, to_dev

pytestmark = pytest.mark.gpu

EPS = 1e-3  # bound on |float32 - double| of a projection (d <= 1024, |r| entries ~ N(0, 1))


@pytest.fixture(scope="module")
def lc():
    import torch
    assert torch.cuda.is_available()
    import paper_2608_01718_amd as m
    return m


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _popcount_rows(x):
    return np.unpackbits(x.view(np.uint8), axis=-1).sum(axis=-1)


def _hamming(sq, sk):
    return np.stack([_popcount_rows(np.bitwise_xor(sk, s[None, :])) for s in sq])


def _lsh_run(lc, sp, w, bits, radius, max_cand=512, rows=None, insert_chunk=None, enable_first=False):
    hp = synth.hyperplanes(bits, sp.d, seed=sp.seed + bits)
    N = w.keys.shape[0]
    if enable_first:
        c = lc.LaCache(max(1, N), sp.d, sp.k_cap, sp.in_dtype, 4096, 0)
        c.enable_lsh(bits, to_dev(hp), max_cand)
        step = insert_chunk or max(1, N)
        for r0 in range(0, N, step):
            c.insert(to_dev(w.keys[r0:r0 + step]), to_dev(w.emb[r0:r0 + step]), to_dev(w.tokens[r0:r0 + step]))
    else:
        c = gpu_cache(lc, sp, w.keys, w.emb, w.tokens, insert_chunk=insert_chunk)
        c.enable_lsh(bits, to_dev(hp), max_cand)
    B = w.queries.shape[0]
    out = c.lookup_lsh(to_dev(w.queries), to_dev(w.la_emb), to_dev(np.ascontiguousarray(w.la_tok[:, :sp.k])),
                       sp.tau_q, sp.tau_r, sp.k, radius)
    g = [t.cpu().numpy() for t in out]
    gsig = c.export_signatures(0, N).cpu().numpy().view(np.uint32) if N else np.zeros((0, bits // 32), np.uint32)
    c.close()
    kq, eq, tok = oracle_store(sp, w.keys, w.emb, w.tokens)
    qq = oracle.quantise(w.queries, sp.in_dtype)
    aq = oracle.quantise(w.la_emb, sp.in_dtype)
    u = np.ascontiguousarray(w.la_tok[:, :sp.k])
    sk, pk = oracle.simhash(kq, hp, bits) if N else (np.zeros((0, bits // 32), np.uint32), np.zeros((0, bits)))
    sq, pq = oracle.simhash(qq, hp, bits)
    o = oracle.lookup_lsh(kq, eq, tok, sk, qq, sq, aq, u, radius, sp.tau_q, sp.tau_r, sp.k)
    return dict(idx=g[0], score=g[1], resp_score=g[2], decision=g[3], n_cand=g[4]), o, gsig, sk, pk, sq, pq, kq, qq


def _check_signatures(gsig, sk, pk):
    """Bits equal wherever the oracle's projection is farther than EPS from zero."""
    if gsig.size == 0:
        return 0
    diff = np.unpackbits((gsig ^ sk).view(np.uint8), axis=-1, bitorder="little").astype(bool)
    near = np.abs(pk) < EPS
    assert not np.any(diff & ~near), f"{int(np.sum(diff & ~near))} signature bits differ away from zero"
    return int(diff.sum())


def _check_lookup(g, o, sk, pk, sq, pq, kq, qq, radius, sp):
    """Exact agreement per query unless a near-zero bit could change the candidate set in a way that matters."""
    B = qq.shape[0]
    if kq.shape[0] == 0:
        assert np.all(g["idx"] == -1) and np.all(g["decision"] == oracle.MISS) and np.all(g["n_cand"] == 0)
        return 0
    H = _hamming(sq, sk)
    nz_k = (np.abs(pk) < EPS).sum(axis=1)
    nz_q = (np.abs(pq) < EPS).sum(axis=1)
    S = (synth.bf16_bits_to_f64(qq) @ synth.bf16_bits_to_f64(kq).T)
    exempt = 0
    for b in range(B):
        border = np.abs(H[b] - radius) <= nz_q[b] + nz_k
        border &= ~((H[b] <= radius) & (H[b] + nz_q[b] + nz_k <= radius))
        best = S[b, o["idx"][b]] if o["idx"][b] >= 0 else -np.inf
        if np.any(border & (S[b] >= best - MARGIN)):
            exempt += 1
            continue
        assert g["n_cand"][b] == o["n_cand"][b] or np.any(border), (b, g["n_cand"][b], o["n_cand"][b])
        assert g["idx"][b] == o["idx"][b], (b, g["idx"][b], o["idx"][b])
        if o["idx"][b] < 0:
            assert np.isnan(g["score"][b]) and g["decision"][b] == oracle.MISS
            continue
        assert abs(float(g["score"][b]) - float(o["score"][b])) <= SCORE_TOL
        near_thr = abs(float(g["score"][b]) - sp.tau_q) < MARGIN or (
            not np.isnan(o["resp_score"][b]) and abs(float(o["resp_score"][b]) - sp.tau_r) < MARGIN)
        if not near_thr:
            assert g["decision"][b] == o["decision"][b], (b, g["decision"][b], o["decision"][b])
            assert np.isnan(g["resp_score"][b]) == np.isnan(o["resp_score"][b])
    return exempt


# d = 1280 and 2176: the query preparation's widest register-resident form and its two-pass form
@pytest.mark.parametrize("name,N,bits,radius,d", [("tiny", 3000, 64, 12, None), ("mid", 20000, 256, 64, None),
                                                  ("mid_paper", 10000, 128, 30, None),
                                                  ("serve_small", 30000, 256, 64, None), ("mid", 4000, 128, 30, 1280),
                                                  ("mid", 3000, 128, 30, 2176)])
def test_lsh_parity(lc, name, N, bits, radius, d):
    extra = {} if d is None else {"d": d}
    sp = synth.spec(name, N=N, B=300, **extra) if name != "serve_small" else synth.spec(name, N=N, B=500)
    w = synth.generate(sp)
    say(f"[case] lsh {name} N={N} d={sp.d} bits={bits} radius={radius}")
    g, o, gsig, sk, pk, sq, pq, kq, qq = _lsh_run(lc, sp, w, bits, radius, insert_chunk=7777)
    flips = _check_signatures(gsig, sk, pk)
    ex = _check_lookup(g, o, sk, pk, sq, pq, kq, qq, radius, sp)
    say(f"[ok] lsh {name}: bit flips near zero {flips}, exempt queries {ex}, mean candidates "
        f"{o['n_cand'].mean():.1f}, hits {int(np.sum(g['decision'] >= 2))}")
    assert ex <= 2


def test_lsh_full_radius_is_the_exact_lookup(lc):
    """radius = bits: every entry is a candidate, so the result is the exact top-1 (judged by the oracle's
    exact lookup with the usual rules)."""
    sp = synth.spec("mid", N=6000, B=200)
    w = synth.generate(sp)
    g, o, *_ = _lsh_run(lc, sp, w, 64, 64, max_cand=sp.N)
    assert np.all(g["n_cand"] == sp.N)
    kq, eq, tok = oracle_store(sp, w.keys, w.emb, w.tokens)
    qq = oracle.quantise(w.queries, sp.in_dtype)
    aq = oracle.quantise(w.la_emb, sp.in_dtype)
    u = np.ascontiguousarray(w.la_tok[:, :sp.k])
    e = oracle.lookup(kq, eq, tok, qq, aq, u, sp.tau_q, sp.tau_r, sp.k)
    compare(g, e, kq, eq, tok, qq, aq, u, sp.tau_q, sp.tau_r, sp.k)


def test_lsh_radius_zero_self_queries_and_inserts_after_enable(lc):
    """Radius 0 is equality of hash keys: a query equal to a stored key always finds it (or the lowest
    identical copy).  Signatures of entries inserted after the index was enabled are maintained."""
    sp = synth.spec("mid", N=5000, B=64)
    w = synth.generate(sp)
    w.queries[:] = w.keys[np.arange(0, 5000, 5000 // 64)[:64]]
    g, o, gsig, sk, pk, sq, pq, kq, qq = _lsh_run(lc, sp, w, 128, 0, enable_first=True, insert_chunk=999)
    _check_signatures(gsig, sk, pk)
    want = np.arange(0, 5000, 5000 // 64)[:64]
    for b in range(64):
        assert g["idx"][b] == oracle.first_identical(kq, int(want[b])), b
        assert g["score"][b] >= 1 - 2 ** -7
    _check_lookup(g, o, sk, pk, sq, pq, kq, qq, 0, sp)


def test_lsh_edges(lc):
    import torch
    sp = synth.spec("tiny", N=10, B=7)
    w = synth.generate(sp)
    hp = to_dev(synth.hyperplanes(64, sp.d, seed=5))
    c = lc.LaCache(100, sp.d, sp.k_cap, sp.in_dtype, 64, 0)
    q, a, t = to_dev(w.queries), to_dev(w.la_emb), to_dev(np.ascontiguousarray(w.la_tok[:, :sp.k]))
    with pytest.raises(lc.LaCacheError):                       # index not enabled
        lc.lacache_lookup_lsh(c, q, a, t, 0.9, 0.85, sp.k, 10)
    c.enable_lsh(64, hp, 8)
    g = [x.cpu().numpy() for x in c.lookup_lsh(q, a, t, 0.9, 0.85, sp.k, 10)]   # empty cache
    assert np.all(g[0] == -1) and np.all(g[3] == 0) and np.all(g[4] == 0) and np.all(np.isnan(g[1]))
    for bad in (-1, 65):
        with pytest.raises(lc.LaCacheError):
            lc.lacache_lookup_lsh(c, q, a, t, 0.9, 0.85, sp.k, bad)
    for bits, mc in ((48, 8), (288, 8), (64, 0)):
        with pytest.raises(lc.LaCacheError):
            lc.lacache_enable_lsh(c, bits, to_dev(synth.hyperplanes(max(bits, 32), sp.d, seed=1)), mc)
    c.close()
    # candidate overflow is reported through n_cand
    sp = synth.spec("tiny", N=2000, B=20)
    w = synth.generate(sp)
    c = gpu_cache(lc, sp, w.keys, w.emb, w.tokens)
    c.enable_lsh(64, hp, 4)
    g = [x.cpu().numpy() for x in c.lookup_lsh(to_dev(w.queries), to_dev(w.la_emb),
                                                to_dev(np.ascontiguousarray(w.la_tok[:, :sp.k])), 0.9, 0.85,
                                                sp.k, 64)]
    assert np.all(g[4] == 2000) and np.all(g[0] >= 0)
    c.close()
    # ensemble caches have no LSH lookup
    c = lc.LaCache(10, sp.d, sp.k_cap, sp.in_dtype, 16, 0, d_resp=(sp.d, 32))
    c.enable_lsh(64, hp, 4)
    with pytest.raises(lc.LaCacheError):
        lc.lacache_lookup_lsh(c, q, a, t, 0.9, 0.85, sp.k, 10)
    c.close()


def test_lsh_recall_full_size_serve(lc):
    """The serving workload at full size (1M x 768, 4096 queries): 256-bit signatures, radius 64.  Against
    the exact lookup every stage-1 hit is found (same entry, same decision) and the candidate lists stay
    short; the exported signatures of all 1M entries and a stratified sample of 48 queries (every class) are
    checked against the oracle's signatures and LSH lookup."""
    sp = synth.spec("serve_small")
    w = synth.generate(sp)
    bits, radius = 256, 64
    hp = synth.hyperplanes(bits, sp.d, seed=77)
    say("[case] lsh full size 1M x 768, B=4096, bits 256, radius 64")
    c = gpu_cache(lc, sp, w.keys, w.emb, w.tokens, insert_chunk=1 << 18)
    ex = gpu_lookup(c, w.queries, w.la_emb, w.la_tok, sp.tau_q, sp.tau_r, sp.k)
    c.enable_lsh(bits, to_dev(hp), 256)
    out = c.lookup_lsh(to_dev(w.queries), to_dev(w.la_emb), to_dev(np.ascontiguousarray(w.la_tok[:, :sp.k])),
                       sp.tau_q, sp.tau_r, sp.k, radius)
    g = [t.cpu().numpy() for t in out]
    gsig = c.export_signatures(0, sp.N).cpu().numpy().view(np.uint32)
    c.close()
    hit = ex["decision"] >= 1                                 # exact stage-1 hits
    found = (g[0] == ex["idx"]) & (g[3] == ex["decision"])
    recall_hits = float(found[hit].mean())
    miss_ok = float(np.mean(g[3][~hit] == 0))
    say(f"[ok] recall of stage-1 hits {recall_hits:.4f} ({int(hit.sum())} hits), misses kept {miss_ok:.4f}, "
        f"mean candidates {g[4].mean():.2f}, max {g[4].max()}")
    assert recall_hits >= 0.999 and miss_ok == 1.0 and g[4].max() <= 256
    # the oracle's LSH lookup on a stratified sample
    rows = sample_rows(w.cls, w.target, 48)
    kq, eq, tok = oracle_store(sp, w.keys, w.emb, w.tokens)
    qq = oracle.quantise(w.queries[rows], sp.in_dtype)
    aq = oracle.quantise(w.la_emb[rows], sp.in_dtype)
    u = np.ascontiguousarray(w.la_tok[rows, :sp.k])
    sk, pk = oracle.simhash(kq, hp, bits)
    flips = _check_signatures(gsig, sk, pk)
    sq, pq = oracle.simhash(qq, hp, bits)
    o = oracle.lookup_lsh(kq, eq, tok, sk, qq, sq, aq, u, radius, sp.tau_q, sp.tau_r, sp.k)
    gs = dict(idx=g[0][rows], score=g[1][rows], resp_score=g[2][rows], decision=g[3][rows], n_cand=g[4][rows])
    exempt = _check_lookup(gs, o, sk, pk, sq, pq, kq, qq, radius, sp)
    say(f"[ok] lsh full size vs oracle: {len(rows)} sampled queries, exempt {exempt}, signature bit flips near "
        f"zero {flips}, hits {int(np.sum(gs['decision'] >= 2))}")
    assert exempt <= 2
