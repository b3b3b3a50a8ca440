"""GPU parity of the m-ensemble lookahead check (Section 4.4: a hit needs every one of m prefix-embedding
checks to pass) through the C ABI, against the CPU oracle's ensemble lookup on the same seeded inputs."""
from __future__ import annotations

import sys

import numpy as np
import pytest

import oracle
import synth
from tests.compare import compare_ensemble
from tests.gpu_util import gpu_cache, gpu_ensemble_cache, gpu_lookup, gpu_lookup_ensemble, sample_rows, to_dev

pytestmark = pytest.mark.gpu

TAU_R = (0.70, 0.72, 0.68, 0.71, 0.69, 0.70, 0.73, 0.70)


@pytest.fixture(scope="module")
def lc():
    import torch
    assert torch.cuda.is_available()
    import paper_2608_01718_amd as m
    return m


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _workload(sp, dims, B=None, stream_chunk=0):
    w = synth.generate(sp) if B is None else synth.generate(sp, B=B)
    embs = synth.ensemble_entries(sp, dims, 0, sp.N)
    q = dict(cls=w.cls, target=w.target, la_tok=w.la_tok)
    las, la_tok = synth.ensemble_lookahead(sp, dims, embs, w.tokens, q, stream_chunk)
    return w, embs, las, la_tok


def _oracle(sp, w, embs, las, la_tok, tau_r, rows):
    kq = oracle.quantise(w.keys, sp.in_dtype)
    qq = oracle.quantise(w.queries, sp.in_dtype)[rows]
    u = np.ascontiguousarray(la_tok[rows, :sp.k])
    eq = [oracle.quantise(e, sp.in_dtype) for e in embs]
    aq = [oracle.quantise(a, sp.in_dtype)[rows] for a in las]
    o = oracle.lookup_ensemble(kq, qq, sp.tau_q, eq, aq, tau_r, w.tokens, u, sp.k)
    # stage-1 margins for the near-tie rule (the prefix arguments of this call are placeholders)
    s1 = oracle.lookup(kq, kq, w.tokens, qq, qq, u, sp.tau_q, 0.0, sp.k)
    return o, s1


def _run(lc, sp, dims, B=None, call_b=None, b_small=None, rows=None, insert_chunk=None):
    tau_r = TAU_R[:len(dims)]
    w, embs, las, la_tok = _workload(sp, dims, B)
    Bq = w.queries.shape[0]
    say(f"[case] ensemble {sp.name} N={sp.N} d={sp.d} m={len(dims)} dims={dims} B={Bq} call_b={call_b} "
        f"b_small={b_small}")
    c = gpu_ensemble_cache(lc, sp, dims, w.keys, embs, w.tokens, insert_chunk=insert_chunk)
    assert c.m == len(dims) and lc.lacache_models(c) == len(dims)
    if b_small is not None:
        c.set_small_batch(b_small)
    g = gpu_lookup_ensemble(c, w.queries, las, la_tok, sp.tau_q, tau_r, sp.k, call_b)
    rows = np.arange(Bq) if rows is None else rows
    o, s1 = _oracle(sp, w, embs, las, la_tok, tau_r, rows)
    stats = compare_ensemble(g, o, s1, sp.tau_q, tau_r, rows)
    say(f"[ok] ensemble {sp.name} m={len(dims)}: {stats}")
    c.close()
    return g, o, stats


def test_ensemble_store_matches_oracle_quantisation(lc):
    sp = synth.spec("mid_paper", N=1500)
    dims = (1024, 384, 768, 200)
    w = synth.generate(sp)
    embs = synth.ensemble_entries(sp, dims, 0, sp.N)
    c = gpu_ensemble_cache(lc, sp, dims, w.keys, embs, w.tokens, capacity=sp.N + 3, insert_chunk=511)
    for i, e in enumerate(embs):
        got = c.export_prefix(i, 0, sp.N).cpu().numpy().view(np.uint16)
        want = oracle.quantise(e, sp.in_dtype)
        assert got.shape == (sp.N, dims[i])
        diff = got != want
        assert diff.mean() <= 1e-3, (i, diff.mean())
        assert np.abs(got.astype(np.int32) - want.astype(np.int32)).max() <= 1, i
    # export() reports model 0
    _, e0, _ = c.export(0, sp.N)
    assert np.array_equal(e0.cpu().numpy().view(np.uint16), c.export_prefix(0, 0, sp.N).cpu().numpy().view(np.uint16))
    c.close()


def test_ensemble_of_one_is_the_plain_lookup(lc):
    """An ensemble cache of one model with the key dimension gives the plain lookup's outputs bit for bit."""
    for name, B in (("mid", 40), ("serve_large", 300)):
        sp = synth.spec(name, N=8000, B=B, n_dup=30, n_dup_queries=10) if name == "serve_large" else \
            synth.spec(name, N=8000, B=B)
        w = synth.generate(sp)
        say(f"[case] ensemble-of-one {name} B={B}")
        plain = gpu_cache(lc, sp, w.keys, w.emb, w.tokens)
        gp = gpu_lookup(plain, w.queries, w.la_emb, w.la_tok, sp.tau_q, sp.tau_r, sp.k)
        plain.close()
        ens = gpu_ensemble_cache(lc, sp, (sp.d,), w.keys, [w.emb], w.tokens)
        ge = gpu_lookup_ensemble(ens, w.queries, [w.la_emb], w.la_tok, sp.tau_q, [sp.tau_r], sp.k)
        ens.close()
        assert np.array_equal(gp["idx"], ge["idx"]) and np.array_equal(gp["decision"], ge["decision"])
        assert np.array_equal(gp["score"].view(np.uint32), ge["score"].view(np.uint32))
        assert np.array_equal(gp["resp_score"].view(np.uint32), ge["resp_score"][:, 0].view(np.uint32))


@pytest.mark.parametrize("m", [2, 3, 4])
def test_ensemble_parity_small_batch(lc, m):
    sp = synth.spec("mid_paper", N=20000, B=60)
    _, _, st = _run(lc, sp, synth.ENSEMBLE_DIMS[:m])
    assert st["idx_exact"] == st["n"]


@pytest.mark.parametrize("m", [2, 4])
def test_ensemble_parity_gemm_batch(lc, m):
    sp = synth.spec("mid_paper", N=20000, B=300)
    _, _, st = _run(lc, sp, synth.ENSEMBLE_DIMS[:m])
    assert st["idx_exact"] == st["n"]
    # the ensemble must decide: embedding hits, token hits and rejections all occur
    assert st["decisions"][2] > 0 and st["decisions"][3] > 0 and st["decisions"][1] > 0


def test_ensemble_parity_f32_ragged_dims_and_chunking(lc):
    """float32 inputs, prefix dimensions that are not multiples of 128 or 8, eight models (the limit), a
    lookup split over max_batch chunks and calls of several sizes."""
    sp = synth.spec("tiny", N=7000, B=333)
    dims = (384, 1, 7, 129, 250, 513, 64, 1000)
    tau_r = TAU_R[:len(dims)]
    w, embs, las, la_tok = _workload(sp, dims)
    say(f"[case] ensemble f32 ragged dims={dims} B=333 max_batch=100")
    c = lc.LaCache(sp.N, sp.d, sp.k_cap, sp.in_dtype, 100, 0, d_resp=dims)
    for r0 in range(0, sp.N, 2500):
        r1 = min(sp.N, r0 + 2500)
        assert c.insert_ensemble(to_dev(w.keys[r0:r1]), [to_dev(e[r0:r1]) for e in embs],
                                 to_dev(w.tokens[r0:r1])) == r0
    for call_b in (333, 50, 7):
        g = gpu_lookup_ensemble(c, w.queries, las, la_tok, sp.tau_q, tau_r, sp.k, call_b)
        o, s1 = _oracle(sp, w, embs, las, la_tok, tau_r, np.arange(333))
        st = compare_ensemble(g, o, s1, sp.tau_q, tau_r)
        say(f"[ok] call_b={call_b}: {st}")
    c.close()


def test_ensemble_threshold_order_and_extremes(lc):
    """Per-model thresholds are applied to their own model: raising one model's threshold above 1 rejects
    every embedding hit, -1 everywhere accepts every stage-1 hit, and swapping two models' thresholds
    matches the oracle with the same swap."""
    sp = synth.spec("mid_paper", N=6000, B=200)
    dims = (1024, 384, 768)
    w, embs, las, la_tok = _workload(sp, dims)
    c = gpu_ensemble_cache(lc, sp, dims, w.keys, embs, w.tokens)
    rows = np.arange(200)
    for tau_r in ((0.70, 1.5, 0.70), (-1.0, -1.0, -1.0), (0.9, 0.3, 0.6), (0.3, 0.9, 0.6)):
        say(f"[case] ensemble thresholds {tau_r}")
        g = gpu_lookup_ensemble(c, w.queries, las, la_tok, sp.tau_q, tau_r, sp.k)
        o, s1 = _oracle(sp, w, embs, las, la_tok, tau_r, rows)
        compare_ensemble(g, o, s1, sp.tau_q, tau_r)
        if tau_r[1] > 1:
            assert not np.any(g["decision"] == lc.HIT)
        if max(tau_r) < -0.5:
            assert not np.any(g["decision"] == lc.REJECT)
    c.close()


def test_ensemble_empty_cache_and_errors(lc):
    import torch
    sp = synth.spec("mid", N=10, B=5)
    dims = (768, 384)
    c = lc.LaCache(100, sp.d, sp.k_cap, sp.in_dtype, 64, 0, d_resp=dims)
    w, embs, las, la_tok = _workload(sp, dims)
    g = gpu_lookup_ensemble(c, w.queries, las, la_tok, sp.tau_q, (0.7, 0.7), sp.k)
    assert np.all(g["idx"] == -1) and np.all(g["decision"] == lc.MISS)
    assert np.all(np.isnan(g["score"])) and np.all(np.isnan(g["resp_score"]))
    assert g["resp_score"].shape == (5, 2)
    assert np.all(g["resp_score"].view(np.uint32) == 0x7FC00000)
    keys, tok = to_dev(w.keys), to_dev(w.tokens)
    e0 = to_dev(embs[0])
    with pytest.raises(lc.LaCacheError) as ei:      # the single-model insert is for m = 1 only
        lc.lacache_insert(c, keys, e0, tok)
    assert ei.value.code == lc.EINVAL
    c.insert_ensemble(keys, [to_dev(e) for e in embs], tok)
    q, t = to_dev(w.queries), to_dev(np.ascontiguousarray(la_tok[:, :sp.k]))
    a = [to_dev(x) for x in las]
    for tau in ((0.7, float("nan")), (float("inf"), 0.7)):
        with pytest.raises(lc.LaCacheError) as ei:
            c.lookup_ensemble(q, a, t, sp.tau_q, tau, sp.k)
        assert ei.value.code == lc.EINVAL
    with pytest.raises(lc.LaCacheError) as ei:
        lc.lacache_lookup(c, q, a[0], t, sp.tau_q, 0.7, sp.k)
    assert ei.value.code == lc.EINVAL
    with pytest.raises(ValueError):
        c.export_prefix(2, 0, 1)
    raw = lc.raw_library()
    buf = torch.empty(768, dtype=torch.int16, device="cuda:0")
    assert raw.lacache_export_prefix(c.handle, 2, 0, 1, buf.data_ptr(), None) == lc.EINVAL
    assert raw.lacache_export_prefix(c.handle, 0, 9, 5, buf.data_ptr(), None) == lc.EINVAL
    assert c.size() == 10
    c.close()


def test_ensemble_full_size_serve_sampled(lc):
    """The serving workload at full size (1M x 768 keys, the paper's four prefix models) with the batch of
    4096 queries the GEMM path serves, checked on a stratified sample."""
    sp = synth.spec("serve_large")
    dims = synth.ENSEMBLE_DIMS
    tau_r = TAU_R[:4]
    w, embs, las, la_tok = _workload(sp, dims)
    say(f"[case] ensemble full-size serve_large m=4 B={w.queries.shape[0]}")
    c = gpu_ensemble_cache(lc, sp, dims, w.keys, embs, w.tokens, insert_chunk=250_000)
    g = gpu_lookup_ensemble(c, w.queries, las, la_tok, sp.tau_q, tau_r, sp.k)
    rows = sample_rows(w.cls, w.target, 150, seed=7)
    o, s1 = _oracle(sp, w, embs, las, la_tok, tau_r, rows)
    st = compare_ensemble(g, o, s1, sp.tau_q, tau_r, rows)
    say(f"[ok] full-size ensemble: {st}")
    c.close()
