"""GPU parity: the HIP path through the C ABI against the CPU oracle on the same seeded inputs."""
from __future__ import annotations

import sys

import numpy as np
import pytest

import oracle
import synth
from tests.compare import compare
from tests.gpu_util import gpu_cache, gpu_lookup, oracle_store, sample_rows, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lc():
    import torch
    assert torch.cuda.is_available()
    import paper_2608_01718_amd as m
    return m


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _run(lc, sp, w=None, call_b=None, b_small=None, rows=None, insert_chunk=None, max_batch=4096):
    w = w or synth.generate(sp)
    say(f"[case] {sp.name} N={sp.N} d={sp.d} B={w.queries.shape[0]} k={sp.k} call_b={call_b} b_small={b_small}")
    c = gpu_cache(lc, sp, w.keys, w.emb, w.tokens, max_batch=max_batch, insert_chunk=insert_chunk)
    if b_small is not None:
        c.set_small_batch(b_small)
    g = gpu_lookup(c, w.queries, w.la_emb, w.la_tok, sp.tau_q, sp.tau_r, sp.k, call_b)
    kq, eq, tok = oracle_store(sp, w.keys, w.emb, w.tokens)
    qq = oracle.quantise(w.queries, sp.in_dtype)
    aq = oracle.quantise(w.la_emb, sp.in_dtype)
    u = np.ascontiguousarray(w.la_tok[:, :sp.k])
    rows = np.arange(w.queries.shape[0]) if rows is None else rows
    o = oracle.lookup(kq, eq, tok, qq[rows], aq[rows], u[rows], sp.tau_q, sp.tau_r, sp.k)
    stats = compare(g, o, kq, eq, tok, qq, aq, u, sp.tau_q, sp.tau_r, sp.k, rows)
    # every large-batch group replay reproduced its stage-1 score (no fallback row was taken)
    assert c.replay_fallbacks() == 0
    say(f"[ok] {sp.name}: {stats}")
    c.close()
    return w, g, o, stats


def test_store_matches_oracle_quantisation(lc):
    for name, N in [("tiny", 3000), ("mid", 3000), ("mid_paper", 1000)]:
        sp = synth.spec(name, N=N)
        w = synth.generate(sp)
        c = gpu_cache(lc, sp, w.keys, w.emb, w.tokens, capacity=N + 5, insert_chunk=777)
        k, e, t = (x.cpu().numpy() for x in c.export(0, N))
        kq, eq, tok = oracle_store(sp, w.keys, w.emb, w.tokens)
        for got, want in ((k.view(np.uint16), kq), (e.view(np.uint16), eq)):
            diff = got != want
            # the float64 normalisation may sum in another order; a 1-ulp flip at a rounding tie is allowed
            assert diff.mean() <= 1e-3
            ulp = np.abs(got.astype(np.int32) - want.astype(np.int32))
            assert np.all(ulp[diff] <= 1)
        np.testing.assert_array_equal(t, tok)
        c.close()


@pytest.mark.parametrize("N,chunk", [(1000, 777), (9000, 9000)])
@pytest.mark.parametrize("d", [64, 384, 512, 520, 768, 1000, 1152, 2048, 2100])
@pytest.mark.parametrize("dtype", [oracle.F32, oracle.BF16])
def test_keys_and_prefix_rows_store_identically(lc, N, chunk, d, dtype):
    """The same vectors inserted as keys (tiled layout) and as prefix embeddings (row-major layout) are stored
    bit-identically: every normaliser sums the norm in one order and rounds every element alike.  Keys of
    calls up to 8192 rows take a wave per row (rows held in registers up to d = 2048), larger calls a norm
    pass and a rounding pass; prefix rows are held in registers up to d = 2048, two passes beyond.  Inserts
    in chunks of 777 rows (groups of 16 rows straddle calls) or one insert of 9000; among the rows, zero
    vectors, vectors of subnormal float32 components and vectors near the top of the float32 range (their
    reciprocal norms are no normal float32); against the oracle's quantisation as the store test checks it."""
    rng = np.random.default_rng(1000 + d)
    x = rng.standard_normal((N, d)).astype(np.float32)
    x[5] = 0.0
    x[17] *= np.float32(1e-41)
    x[300] *= np.float32(2e37)
    x[301] *= np.float32(1e-30)
    src = x if dtype == oracle.F32 else (x.view(np.uint32) >> 16).astype(np.uint16)
    tok = rng.integers(0, 1000, (N, 4), dtype=np.int32)
    say(f"[case] keys vs prefix rows, N={N} chunk={chunk} d={d} dtype={dtype}")
    c = lc.LaCache(N, d, 4, dtype, 16, 0)
    for r0 in range(0, N, chunk):
        assert c.insert(to_dev(src[r0:r0 + chunk]), to_dev(src[r0:r0 + chunk]), to_dev(tok[r0:r0 + chunk])) == r0
    k, e, _ = (t.cpu().numpy() for t in c.export(0, N))
    c.close()
    np.testing.assert_array_equal(k.view(np.uint16), e.view(np.uint16))
    want = oracle.quantise(src, dtype)
    got = k.view(np.uint16)
    diff = got != want
    assert diff.mean() <= 1e-3
    assert np.all(np.abs(got.astype(np.int32) - want.astype(np.int32))[diff] <= 1)
    assert not got[5].any()


def test_single_insert_and_export_beyond_one_grid(lc):
    """One insert of 4.3M rows (more rows than one launch of the normaliser covers: its waves loop) and one
    export of all of them (4.3M x 80 values, more than one launch of the export covers: its threads loop),
    checked against the oracle's quantisation as the store test checks it."""
    rng = np.random.default_rng(77)
    N, d = 4_300_000, 80
    keys = rng.standard_normal((N, d), dtype=np.float32)
    emb = rng.standard_normal((N, d), dtype=np.float32)
    tok = rng.integers(0, 1000, (N, 2), dtype=np.int32)
    say(f"[case] one insert of N={N} d={d} f32, then one export")
    c = lc.LaCache(N, d, 2, oracle.F32, 16, 0)
    assert c.insert(to_dev(keys), to_dev(emb), to_dev(tok)) == 0
    k, e, t = (x.cpu().numpy() for x in c.export(0, N))
    for got, src in ((k, keys), (e, emb)):
        want = oracle.quantise(src, oracle.F32)
        diff = got.view(np.uint16) != want
        assert diff.mean() <= 1e-3
        ulp = np.abs(got.view(np.uint16).astype(np.int32) - want.astype(np.int32))
        assert np.all(ulp[diff] <= 1)
    np.testing.assert_array_equal(t, tok)
    c.close()


@pytest.mark.parametrize("name", ["tiny", "mid", "mid_paper"])
def test_parity_full_config(lc, name):
    _run(lc, synth.spec(name))


def test_parity_serve_small_reduced(lc):
    sp = synth.spec("serve_small", N=60_000, B=256)
    _run(lc, sp, call_b=synth.SERVE_SMALL_CALL_B)


def test_parity_serve_large_reduced(lc):
    sp = synth.spec("serve_large", N=40_000, n_dup=200, n_dup_queries=64)
    w, g, o, _ = _run(lc, sp)
    # duplicate-aimed benign queries resolve to the earlier copy and are served from its prefix
    dq = np.nonzero(np.isin(w.target, w.dup_pairs[:, 0]) & (w.cls == synth.CLS_BENIGN))[0]
    assert len(dq) >= 32
    np.testing.assert_array_equal(g["idx"][dq], w.target[dq])
    np.testing.assert_array_equal(g["decision"][dq], oracle.HIT_EXACT)


def test_parity_large_clustered_reduced(lc):
    sp = synth.spec("large", N=30_000, B=512)
    _run(lc, sp)


def test_parity_serve_small_full_size_sampled(lc):
    """The 1M x 768 workload in 16-query calls (the streaming kernel) at full size: 1024 queries, 512
    or more stratified rows of them (every collision query, 256 benign and 256 miss) against the oracle."""
    sp = synth.spec("serve_small", B=1024)
    w = synth.generate(sp)
    rows = sample_rows(w.cls, w.target, 768)
    assert len(rows) >= 512
    _run(lc, sp, w=w, call_b=synth.SERVE_SMALL_CALL_B, rows=rows)


def test_parity_serve_large_full_size_sampled(lc):
    """The 1M x 768, 4096-query workload at full size: 512 stratified rows (every class: benign, collision and
    miss, the misses holding the closest runner-up scores) and 16 duplicate-aimed rows against the oracle; the
    whole batch against the planted truth."""
    sp = synth.spec("serve_large")
    w = synth.generate(sp)
    dq = np.nonzero(np.isin(w.target, w.dup_pairs[:, 0]) & (w.cls == synth.CLS_BENIGN))[0][:16]
    rows = np.unique(np.concatenate([sample_rows(w.cls, w.target, 768), dq]))
    assert len(rows) >= 512
    _, g, _, _ = _run(lc, sp, w=w, rows=rows)
    # the whole batch: every duplicate-aimed query resolves to the earlier copy
    dq = np.nonzero(np.isin(w.target, w.dup_pairs[:, 0]) & (w.cls == synth.CLS_BENIGN))[0]
    np.testing.assert_array_equal(g["idx"][dq], w.target[dq])
    # synthetic hit-rate analogues over the whole batch: benign plants served, collisions rejected
    ben = w.cls == synth.CLS_BENIGN
    col = w.cls == synth.CLS_COLLISION
    assert np.all(np.isin(g["decision"][ben], [oracle.HIT, oracle.HIT_EXACT]))
    assert np.all(g["decision"][col] == oracle.REJECT)
    assert np.all(g["decision"][w.cls == synth.CLS_MISS] == oracle.MISS)


# ------------------------------------------------------------------------------------------- edge cases


def _edge(lc, N, d, B, k_cap, k, dtype=oracle.F32, seed=0, b_small=None, neg=False, zero_rows=(), dup=0,
          zero_queries=()):
    rng = np.random.default_rng(seed)
    sp = synth.Spec("edge", N, d, dtype, k_cap, 50, B, 0, 0, 0, 0, 0.3, 0.2, k, seed)
    dt = np.float32
    keys = rng.standard_normal((N, d)).astype(dt)
    if neg:
        # every key close to one direction, every query opposite to it: all real scores are near -1
        keys = (rng.standard_normal(d) + 0.2 * keys).astype(dt)
    emb = rng.standard_normal((N, d)).astype(dt)
    tok = rng.integers(0, 50, (N, k_cap), dtype=np.int32)
    for r in zero_rows:
        if r < N:
            keys[r] = 0
    if dup and N > 2:
        keys[rng.integers(N // 2, N, dup)] = keys[rng.integers(0, N // 2, dup)]
    q = rng.standard_normal((B, d)).astype(dt)
    pick = rng.integers(0, max(N, 1), B)
    if N:
        q[: B // 2] = keys[pick[: B // 2]] + 0.05 * rng.standard_normal((B // 2, d)).astype(dt)
        if neg:
            q[:] = -keys[pick]
    for r in zero_queries:
        q[r] = 0
    a = rng.standard_normal((B, d)).astype(dt)
    u = rng.integers(0, 50, (B, k), dtype=np.int32)
    if N:
        u[: B // 4] = tok[pick[: B // 4], :k]
        a[B // 4: B // 2] = emb[pick[B // 4: B // 2]]
    if dtype == oracle.BF16:
        keys, emb, q, a = (synth.to_bf16_bits(x) for x in (keys, emb, q, a))
    w = synth.Workload(sp, keys, emb, tok, q, a, u, np.zeros(B, np.int32), np.full(B, -1), np.full(B, np.nan),
                       np.zeros((0, 2), np.int64))
    say(f"[edge] N={N} d={d} B={B} k_cap={k_cap} k={k} dtype={dtype} b_small={b_small} neg={neg}")
    c = gpu_cache(lc, sp, keys, emb, tok, capacity=max(N, 1) + 3)
    if b_small is not None:
        c.set_small_batch(b_small)
    g = gpu_lookup(c, q, a, u, sp.tau_q, sp.tau_r, k)
    kq, eq, tq = oracle_store(sp, keys, emb, tok)
    qq, aq = oracle.quantise(q, dtype), oracle.quantise(a, dtype)
    o = oracle.lookup(kq, eq, tq, qq, aq, u, sp.tau_q, sp.tau_r, k)
    compare(g, o, kq, eq, tq, qq, aq, u, sp.tau_q, sp.tau_r, k)
    assert c.replay_fallbacks() == 0
    c.close()
    return w, g, o


# b_small None keeps the default crossover, which for caches this small (n * d_pad < 2^27) is three streaming
# query groups, 192 queries for d <= 1152
@pytest.mark.parametrize("N,d,B,k_cap,k,b_small", [
    (1, 64, 5, 1, 1, None),          # a single entry
    (17, 64, 16, 8, 8, None),        # one live row in the last 16-row group
    (255, 100, 17, 150, 150, None),  # d not a multiple of 128, k > 64 (two ballot rounds), ragged B
    (257, 384, 63, 20, 1, None),     # k = 1
    (1000, 384, 65, 64, 64, None),   # B just past one streaming query group: two groups of 64
    (2000, 768, 128, 16, 16, None),  # two full streaming query groups
    (1000, 384, 129, 64, 64, None),  # three streaming query groups, the last holding one query
    (1000, 384, 193, 64, 64, None),  # just past the default limit: the GEMM path
    (1500, 768, 200, 16, 16, 256),   # four streaming query groups, the last one ragged
    (1000, 1152, 256, 64, 64, 256),  # the largest streaming batch, at the largest d it holds
    (900, 1280, 150, 8, 8, 192),     # d > 1152: groups of 48 queries, four of them, the last holding 6
    (4097, 768, 300, 16, 16, None),  # ragged everything on the large-batch path
    (300, 1024, 1, 32, 32, None),    # B = 1
    (600, 2100, 40, 8, 8, None),     # d_pad > 2048: queries staged by the normaliser, two 32-query groups
    (300, 6000, 40, 8, 8, None),     # d_pad > 4992: no streaming query group fits LDS, every batch on the GEMM
    (150, 16384, 20, 4, 4, None),    # the largest d a cache takes
    (40, 1, 9, 4, 4, None),          # d = 1: every key normalises to +-1, whole halves of the store tie exactly
    (40, 1, 200, 4, 4, None),        # the same ties on the GEMM path: the first 16-row group, then its lowest row
    (3000, 1, 300, 4, 4, None),      # ties spread over six key tiles and several workgroups' ranges
    (50, 64, 8, 4096, 4096, None),   # k = k_cap = 4096, the largest prefix a cache takes (64 ballot rounds)
])
@pytest.mark.parametrize("dtype", [oracle.F32, oracle.BF16])
def test_edge_shapes(lc, N, d, B, k_cap, k, b_small, dtype):
    _edge(lc, N, d, B, k_cap, k, dtype, b_small=b_small)


def test_crossover_limits_for_wide_rows(lc):
    """Where not even one 16-query group of the streaming kernel fits LDS (d_pad > 4992), no batch size can be
    sent to it: setting the crossover above 0 is EINVAL, 0 and -1 are accepted, and lookups run (on the GEMM
    kernel) either way."""
    import torch
    c = lc.LaCache(64, 6000, 4, oracle.F32, 64, 0)
    x = torch.randn(64, 6000, device="cuda")
    tok = torch.zeros(64, 4, dtype=torch.int32, device="cuda")
    c.insert(x, x, tok)
    with pytest.raises(lc.LaCacheError) as e:
        c.set_small_batch(16)
    assert e.value.code == lc.EINVAL
    for b_small in (0, -1):
        c.set_small_batch(b_small)
        idx, score, _, dec = c.lookup(x[:5], x[:5], tok[:5], 0.5, 0.5, 4)
        assert torch.equal(idx.cpu(), torch.arange(5, dtype=torch.int32))
        assert torch.all(dec.cpu() == oracle.HIT_EXACT)
    c.close()


@pytest.mark.parametrize("b_small,B", [(0, 40), (64, 40), (128, 100), (256, 200)])
def test_all_negative_scores_never_pick_padding(lc, b_small, B):
    # every real score is negative; padded rows (zeros) would score 0 if they were not masked
    for N in (1, 17, 250):
        _, g, o = _edge(lc, N, 64, B, 4, 4, neg=True, b_small=b_small, seed=N)
        assert np.all(g["idx"] < N) and np.all(g["score"] < 0)


def test_zero_vectors_and_duplicates(lc):
    _edge(lc, 500, 128, 70, 8, 8, zero_rows=(0, 3, 499), dup=40)
    # a zero query scores 0 against everything: index 0, score 0
    _, g, _ = _edge(lc, 50, 32, 4, 2, 2, seed=9, zero_queries=(1, 3))
    assert g["idx"][1] == 0 and g["score"][1] == 0 and g["idx"][3] == 0 and g["score"][3] == 0


def test_empty_cache(lc):
    import torch
    c = lc.LaCache(10, 32, 4, oracle.F32, 16, 0)
    q = torch.randn(5, 32, device="cuda")
    t = torch.zeros(5, 4, dtype=torch.int32, device="cuda")
    idx, score, resp, dec = (x.cpu().numpy() for x in c.lookup(q, q, t, 0.5, 0.5, 4))
    assert np.all(idx == -1) and np.all(np.isnan(score)) and np.all(np.isnan(resp)) and np.all(dec == 0)
    assert np.all(resp.view(np.uint32) == 0x7FC00000)
    # a lookup of no queries is a no-op, on an empty cache and on a filled one
    e = c.lookup(q[:0], q[:0], t[:0], 0.5, 0.5, 4)
    assert all(x.numel() == 0 for x in e)
    c.insert(q, q, t)
    e = c.lookup(q[:0], q[:0], t[:0], 0.5, 0.5, 4)
    assert all(x.numel() == 0 for x in e)
    torch.cuda.synchronize()
    c.close()


@pytest.mark.parametrize("B,b_small", [(256, None), (150, None), (256, 0)])
def test_near_tie_exemption_exercised(lc, B, b_small):
    """Pairs of entries whose scores against a query are equal in exact arithmetic but whose keys differ: entry
    j is entry i with two components (one in the first 32-column step, one in the last) swapped, and the query,
    planted near entry i, carries equal values in those two components.  The two float32 scores may round apart
    in either direction, so the GPU may name either entry: the oracle's top-2 margin is (near) zero, every query
    falls in the near-tie set and the idx rule is set membership.  Streaming and GEMM paths."""
    rng = np.random.default_rng(31)
    N, d, k = 4000, 768, 8
    keys = rng.standard_normal((N, d)).astype(np.float32)
    pairs = rng.choice(N // 2, size=B, replace=False) * 2           # entry i = 2m, its swapped copy j = 2m + 1
    p_col, q_col = rng.integers(0, 32, B), rng.integers(d - 32, d, B)
    for n, i in enumerate(pairs):
        keys[i + 1] = keys[i]
        keys[i + 1, p_col[n]], keys[i + 1, q_col[n]] = keys[i, q_col[n]], keys[i, p_col[n]]
    q = keys[pairs] + 0.3 * rng.standard_normal((B, d)).astype(np.float32)
    for n in range(B):
        m = 0.5 * (q[n, p_col[n]] + q[n, q_col[n]])
        q[n, p_col[n]] = q[n, q_col[n]] = m
    emb = rng.standard_normal((N, d)).astype(np.float32)
    tok = rng.integers(0, 50, (N, k), dtype=np.int32)
    a = rng.standard_normal((B, d)).astype(np.float32)
    u = rng.integers(0, 50, (B, k), dtype=np.int32)
    sp = synth.Spec("near_tie", N, d, oracle.F32, k, 50, B, 0, 0, 0, 0, 0.3, 0.2, k, 31)
    say(f"[case] near-tie pairs N={N} B={B} b_small={b_small}")
    c = gpu_cache(lc, sp, keys, emb, tok)
    if b_small is not None:
        c.set_small_batch(b_small)
    g = gpu_lookup(c, q, a, u, sp.tau_q, sp.tau_r, k)
    kq, eq, tq = oracle_store(sp, keys, emb, tok)
    qq, aq = oracle.quantise(q, oracle.F32), oracle.quantise(a, oracle.F32)
    o = oracle.lookup(kq, eq, tq, qq, aq, u, sp.tau_q, sp.tau_r, k)
    stats = compare(g, o, kq, eq, tq, qq, aq, u, sp.tau_q, sp.tau_r, k)
    assert c.replay_fallbacks() == 0
    c.close()
    say(f"[ok] near-tie pairs: {stats}")
    # every query's winner is one of its pair, and the exemption governs (nearly) every query
    assert np.all((g["idx"] == pairs) | (g["idx"] == pairs + 1))
    assert stats["near_set"] >= B * 0.9


@pytest.mark.parametrize("B", [64, 100, 128, 200, 256])
def test_determinism_and_paths_agree(lc, B):
    """Ten repeats give identical outputs, and the streaming and GEMM stage-1 paths give identical outputs."""
    import torch
    sp = synth.spec("mid", N=20_000, B=B)
    w = synth.generate(sp)
    c = gpu_cache(lc, sp, w.keys, w.emb, w.tokens)
    runs = [gpu_lookup(c, w.queries, w.la_emb, w.la_tok, sp.tau_q, sp.tau_r, sp.k) for _ in range(10)]
    for r in runs[1:]:
        for n in runs[0]:
            np.testing.assert_array_equal(r[n].view(np.uint32) if r[n].dtype == np.float32 else r[n],
                                          runs[0][n].view(np.uint32) if runs[0][n].dtype == np.float32
                                          else runs[0][n])
    c.set_small_batch(0)
    g = gpu_lookup(c, w.queries, w.la_emb, w.la_tok, sp.tau_q, sp.tau_r, sp.k)
    s = runs[0]
    # both stage-1 kernels accumulate every score with the same instruction sequence (16x16x32 bf16 MFMAs over
    # the 32-column steps in order, from zero): the two paths agree bit for bit
    for n in ("idx", "score", "resp_score", "decision"):
        np.testing.assert_array_equal(g[n].view(np.uint32) if g[n].dtype == np.float32 else g[n],
                                      s[n].view(np.uint32) if s[n].dtype == np.float32 else s[n])
    assert c.replay_fallbacks() == 0
    c.close()
    torch.cuda.synchronize()


def test_calls_enqueued_on_side_streams(lc):
    """Inserts and lookups of two independent caches enqueued on two side streams (default priority), with no
    host synchronisation between the calls: a lookup sees every insert enqueued before it on its stream, and
    the results equal those of the same calls on the default stream bit for bit."""
    import torch
    sp = synth.spec("mid", N=20_000, B=300)
    w = synth.generate(sp)
    ref_cache = gpu_cache(lc, sp, w.keys, w.emb, w.tokens)
    ref = gpu_lookup(ref_cache, w.queries, w.la_emb, w.la_tok, sp.tau_q, sp.tau_r, sp.k)
    ref_cache.close()
    keys, emb, tok = to_dev(w.keys), to_dev(w.emb), to_dev(w.tokens)
    q, a = to_dev(w.queries), to_dev(w.la_emb)
    t = to_dev(np.ascontiguousarray(w.la_tok[:, :sp.k]))
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    caches, outs = [], []
    half = sp.N // 2
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
        c = lc.LaCache(sp.N, sp.d, sp.k_cap, sp.in_dtype, 4096, 0)
        with torch.cuda.stream(s):
            assert c.insert(keys[:half], emb[:half], tok[:half], stream=s) == 0
            assert c.insert(keys[half:], emb[half:], tok[half:], stream=s) == half
            outs.append(c.lookup(q, a, t, sp.tau_q, sp.tau_r, sp.k, stream=s))
        caches.append(c)
    for s in streams:
        s.synchronize()
    for out in outs:
        g = dict(zip(("idx", "score", "resp_score", "decision"), (x.cpu().numpy() for x in out)))
        for name in ("idx", "decision"):
            np.testing.assert_array_equal(g[name], ref[name])
        for name in ("score", "resp_score"):
            np.testing.assert_array_equal(g[name].view(np.uint32), ref[name].view(np.uint32))
    for c in caches:
        c.close()


def test_lookup_graph_capture_and_replay(lc):
    """Lookups of both stage-1 paths (64 queries on the streaming kernel, 300 on the GEMM kernel) captured into
    one HIP graph and replayed: the lookup enqueues only kernels, so the capture holds it whole.  Every replay,
    with new query contents copied into the captured inputs and the outputs overwritten by eager work
    between replays, equals an eager lookup on the same inputs bit for bit."""
    import torch
    sp = synth.spec("mid", N=20_000, B=364)
    w = synth.generate(sp)
    c = gpu_cache(lc, sp, w.keys, w.emb, w.tokens)
    q_all, a_all = to_dev(w.queries), to_dev(w.la_emb)
    t_all = to_dev(np.ascontiguousarray(w.la_tok[:, :sp.k]))
    q, a, t = q_all.clone(), a_all.clone(), t_all.clone()
    calls = ((64, 0), (300, 64))  # (B, first row): streaming path, then GEMM path (n * d_pad < 2^27: 192 stream)
    dts = (torch.int32, torch.float32, torch.float32, torch.int32)
    outs = {B: tuple(torch.empty(B, dtype=dt, device="cuda") for dt in dts) for B, _ in calls}

    def run(o):
        for B, r0 in calls:
            c.lookup(q[r0:r0 + B], a[r0:r0 + B], t[r0:r0 + B], sp.tau_q, sp.tau_r, sp.k, out=o[B])

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run(outs)  # first use outside the capture (kernel attributes are set once)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        run(outs)
    rng = np.random.default_rng(5)
    for rep in range(4):
        perm = torch.as_tensor(rng.permutation(sp.B), device="cuda")
        q.copy_(q_all[perm])
        a.copy_(a_all[perm])
        t.copy_(t_all[perm])
        for o in outs.values():
            for x in o:
                x.fill_(-7)
        graph.replay()
        torch.cuda.synchronize()
        got = {B: [x.clone() for x in outs[B]] for B, _ in calls}
        ref = {B: tuple(torch.empty(B, dtype=dt, device="cuda") for dt in dts) for B, _ in calls}
        run(ref)
        torch.cuda.synchronize()
        for B, _ in calls:
            for g_, r_ in zip(got[B], ref[B]):
                gb, rb = g_.cpu().numpy(), r_.cpu().numpy()
                np.testing.assert_array_equal(gb.view(np.uint32), rb.view(np.uint32), err_msg=f"replay {rep}, B={B}")
        say(f"[ok] graph replay {rep}: hits {int((ref[300][3] >= 2).sum().item())} of 300")
    assert c.replay_fallbacks() == 0
    graph.reset()
    c.close()


def test_interleaved_inserts(lc):
    """A query planted near an entry is a miss before that entry is inserted and a hit after it."""
    sp = synth.spec("large", N=12_288, B=256)
    keys, emb, tok = synth.entries(sp, 0, sp.N)
    base = 8192
    c = gpu_cache(lc, sp, keys[:base], emb[:base], tok[:base], capacity=sp.N, insert_chunk=4096)
    late = synth.queries(sp, keys, emb, tok, np.zeros((0, 2), np.int64), B=256, N=sp.N, stream_chunk=7)
    aimed_late = (late["target"] >= base) & (late["cls"] == synth.CLS_BENIGN)
    assert aimed_late.sum() > 10
    g0 = gpu_lookup(c, late["queries"], late["la_emb"], late["la_tok"], sp.tau_q, sp.tau_r, sp.k)
    assert np.all(g0["idx"][aimed_late] < base)
    assert np.all(g0["decision"][aimed_late] == oracle.MISS)
    for r0 in range(base, sp.N, 4096):
        assert c.insert(to_dev(keys[r0:r0 + 4096]), to_dev(emb[r0:r0 + 4096]), to_dev(tok[r0:r0 + 4096])) == r0
    g1 = gpu_lookup(c, late["queries"], late["la_emb"], late["la_tok"], sp.tau_q, sp.tau_r, sp.k)
    np.testing.assert_array_equal(g1["idx"][aimed_late], late["target"][aimed_late])
    assert np.all(g1["decision"][aimed_late] == oracle.HIT_EXACT)
    kq, eq, tq = oracle_store(sp, keys, emb, tok)
    qq, aq = oracle.quantise(late["queries"], sp.in_dtype), oracle.quantise(late["la_emb"], sp.in_dtype)
    u = np.ascontiguousarray(late["la_tok"][:, :sp.k])
    o = oracle.lookup(kq, eq, tq, qq, aq, u, sp.tau_q, sp.tau_r, sp.k)
    compare(g1, o, kq, eq, tq, qq, aq, u, sp.tau_q, sp.tau_r, sp.k)
    c.close()


def test_errors_with_live_handle(lc):
    import torch
    c = lc.LaCache(100, 16, 4, oracle.F32, 8, 0)
    x = torch.randn(60, 16, device="cuda")
    t = torch.zeros(60, 4, dtype=torch.int32, device="cuda")
    assert c.insert(x, x, t) == 0
    with pytest.raises(lc.LaCacheError) as e:
        c.insert(x, x, t)                       # 60 + 60 > 100: nothing inserted
    assert e.value.code == lc.EFULL and c.size() == 60
    q = x[:4]
    with pytest.raises(lc.LaCacheError) as e:
        c.lookup(q, q, torch.zeros(4, 5, dtype=torch.int32, device="cuda"), 0.5, 0.5, 5)   # k > k_cap
    assert e.value.code == lc.EINVAL
    with pytest.raises(lc.LaCacheError) as e:
        c.lookup(q, q, t[:4], float("nan"), 0.5, 4)
    assert e.value.code == lc.EINVAL
    with pytest.raises(lc.LaCacheError):
        c.lookup(q, q, t[:4], 0.5, float("inf"), 4)
    with pytest.raises(lc.LaCacheError):
        c.set_small_batch(257)
    with pytest.raises(lc.LaCacheError):
        c.set_small_batch(-2)
    c.set_small_batch(-1)  # back to the size-dependent default
    with pytest.raises(ValueError):
        c.lookup(q.double(), q, t[:4], 0.5, 0.5, 4)
    # a lookup with more queries than max_batch runs in chunks and matches chunk-by-chunk lookups
    q2 = torch.randn(21, 16, device="cuda")
    t2 = torch.zeros(21, 4, dtype=torch.int32, device="cuda")
    whole = [z.cpu() for z in c.lookup(q2, q2, t2, 0.1, 0.1, 4)]
    parts = [[z.cpu() for z in c.lookup(q2[i:i + 8], q2[i:i + 8], t2[i:i + 8], 0.1, 0.1, 4)] for i in (0, 8, 16)]
    for j in range(4):
        assert torch.equal(whole[j].view(torch.int32), torch.cat([p[j] for p in parts]).view(torch.int32))
    c.close()


def test_profile_times_every_stage1_launch(lc):
    """lacache_profile: every lookup of a window is timed (streaming and GEMM stage 1 alike), a window longer
    than the events made at enable time still counts every call, reading clears the window, sampling every
    n-th launch times exactly those, and lookups made while profiling is off are not counted."""
    import torch
    c = lc.LaCache(5000, 256, 4, oracle.BF16, 512, 0)
    x = torch.randn(5000, 256, device="cuda", dtype=torch.bfloat16)
    tok = torch.zeros(5000, 4, dtype=torch.int32, device="cuda")
    c.insert(x, x, tok)
    q16, q300 = x[:16], x[:300]
    c.lookup(q16, q16, tok[:16], 0.5, 0.5, 4)
    c.profile(True)
    c.lookup(q16, q16, tok[:16], 0.5, 0.5, 4)       # streaming kernel
    c.lookup(q300, q300, tok[:300], 0.5, 0.5, 4)    # GEMM kernel
    ms, n = c.profile_read()
    assert n == 2 and ms > 0
    ms, n = c.profile_read()
    assert n == 0 and ms == 0
    for _ in range(700):                            # more than the event pairs made when profiling was enabled
        c.lookup(q16, q16, tok[:16], 0.5, 0.5, 4)
    ms, n = c.profile_read()
    assert n == 700 and ms > 0
    c.profile(3)                                    # every third launch: the 1st, 4th, 7th of 8
    for _ in range(8):
        c.lookup(q16, q16, tok[:16], 0.5, 0.5, 4)
    ms, n = c.profile_read()
    assert n == 3 and ms > 0
    c.profile(False)
    c.lookup(q16, q16, tok[:16], 0.5, 0.5, 4)
    ms, n = c.profile_read()
    assert n == 0
    with pytest.raises(lc.LaCacheError):
        c.profile(-1)
    c.close()


def test_create_out_of_memory(lc):
    """A store that no device can hold (the largest capacity at d = 16384: about 70 TB of keys) is refused with
    ENOMEM; so is an ensemble whose last prefix store does not fit, with the stores allocated before it
    released; the device still serves a cache created afterwards."""
    import torch
    cap = (1 << 31) - 512
    with pytest.raises(lc.LaCacheError) as e:
        lc.LaCache(cap, 16384, 4, oracle.BF16, 16, 0)
    assert e.value.code == lc.ENOMEM

    def serve_small_cache():
        c = lc.LaCache(1000, 64, 4, oracle.F32, 16, 0)
        x = torch.randn(10, 64, device="cuda")
        tok = torch.zeros(10, 4, dtype=torch.int32, device="cuda")
        assert c.insert(x, x, tok) == 0
        idx, _, _, _ = c.lookup(x, x, tok, 0.5, 0.5, 4)
        assert torch.equal(idx.cpu(), torch.arange(10, dtype=torch.int32))
        c.close()

    # the first use loads the library's kernels and fills torch's allocator pool: the device memory before and
    # after the failed create is compared only after that
    serve_small_cache()
    torch.cuda.synchronize()
    free0 = torch.cuda.mem_get_info(0)[0]
    # an ensemble whose second prefix store cannot be allocated (134M x 16384 bf16) after its keys and first
    # prefix store (32 GB each) were: those are released again
    with pytest.raises(lc.LaCacheError) as e:
        lc.LaCache(1 << 27, 128, 4, oracle.BF16, 16, 0, d_resp=(128, 16384))
    assert e.value.code == lc.ENOMEM
    torch.cuda.synchronize()
    assert abs(torch.cuda.mem_get_info(0)[0] - free0) < (64 << 20)
    serve_small_cache()


LARGE_STEPS, LARGE_BATCH = 3, 4096


@pytest.fixture(scope="module")
def large_state(lc):
    """The large clustered workload at full size, shared by the serving steps below: 4,000,000 x 1024 keys
    generated with room for LARGE_STEPS insert batches, the oracle's quantised store, and the cache."""
    import time
    sp = synth.spec("large")
    total = sp.N + LARGE_STEPS * LARGE_BATCH
    t0 = time.time()
    keys, emb, tok = synth.entries(sp, 0, total)
    say(f"[case] large full size: generated {total} entries in {time.time() - t0:.1f}s")
    kq, eq, tq = oracle_store(sp, keys, emb, tok)
    say(f"[case] large full size: oracle store quantised ({time.time() - t0:.1f}s)")
    c = gpu_cache(lc, sp, keys[:sp.N], emb[:sp.N], tok[:sp.N], capacity=total, max_batch=sp.B,
                  insert_chunk=1 << 18)
    st = dict(sp=sp, keys=keys, emb=emb, tok=tok, kq=kq, eq=eq, tq=tq, c=c, n=sp.N, done=-1)
    yield st
    c.close()


@pytest.mark.parametrize("step", list(range(LARGE_STEPS + 1)))
def test_parity_large_full_size_interleaved(lc, large_state, step):
    """The large clustered workload at full size: 4,000,000 x 1024 keys (top-2 margins often below 2e-3),
    k = 32, 1024 queries per lookup, an insert batch of 4096 entries between lookups (one test per serving
    step, in order, on one cache), 10% of the planted queries aimed at the latest batch.  At every step 512
    stratified rows (the misses, whose top-2 margins sit near 2e-3, among them) and the latest-batch-aimed rows
    against the oracle; the rows whose oracle top-2 margin is below 2e-3 -- the near-tie set, where the idx rule
    becomes set membership -- are counted and must occur."""
    st = large_state
    assert st["done"] == step - 1, "the serving steps run in order"
    sp, keys, emb, tok, kq, eq, tq, c = (st[k] for k in ("sp", "keys", "emb", "tok", "kq", "eq", "tq", "c"))
    n = st["n"]
    if step > 0:
        first = c.insert(to_dev(keys[n:n + LARGE_BATCH]), to_dev(emb[n:n + LARGE_BATCH]),
                         to_dev(tok[n:n + LARGE_BATCH]))
        assert first == n
        n += LARGE_BATCH
        st["n"] = n
    recent = (n - LARGE_BATCH, n) if step > 0 else None
    q = synth.queries(sp, keys, emb, tok, np.zeros((0, 2), np.int64), B=sp.B, N=n, stream_chunk=100 + step,
                      recent=recent)
    g = gpu_lookup(c, q["queries"], q["la_emb"], q["la_tok"], sp.tau_q, sp.tau_r, sp.k)
    rows = sample_rows(q["cls"], q["target"], 640, seed=step)
    if recent is not None:
        aimed = np.nonzero((q["target"] >= recent[0]) & (q["cls"] == synth.CLS_BENIGN))[0][:8]
        rows = np.unique(np.concatenate([rows, aimed]))
    qq, aq = oracle.quantise(q["queries"], sp.in_dtype), oracle.quantise(q["la_emb"], sp.in_dtype)
    u = np.ascontiguousarray(q["la_tok"][:, :sp.k])
    o = oracle.lookup(kq[:n], eq[:n], tq[:n], qq[rows], aq[rows], u[rows], sp.tau_q, sp.tau_r, sp.k)
    stats = compare(g, o, kq[:n], eq[:n], tq[:n], qq, aq, u, sp.tau_q, sp.tau_r, sp.k, rows)
    say(f"[ok] large step {step} N={n}: {stats}")
    assert stats["n"] >= 512
    assert stats["near_set"] > 0, "no sampled row had a top-2 margin below 2e-3"
    # the whole batch: planted benign queries are served, collisions rejected
    ben, col = q["cls"] == synth.CLS_BENIGN, q["cls"] == synth.CLS_COLLISION
    assert np.all(np.isin(g["decision"][ben], [oracle.HIT, oracle.HIT_EXACT]))
    assert np.all(g["decision"][col] == oracle.REJECT)
    assert c.replay_fallbacks() == 0
    st["done"] = step
