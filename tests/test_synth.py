"""The seeded input generator (synth/workloads.py) produces what the workload recipes state: planted queries at
their drawn cosine to their target, the stated class counts, bitwise-identical duplicate keys, and the same
arrays however the entry stream is requested (windows of any size, any thread count)."""
from __future__ import annotations

import numpy as np
import pytest

import synth


def _cos(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return np.sum(a * b, axis=-1) / (np.linalg.norm(a, axis=-1) * np.linalg.norm(b, axis=-1))


@pytest.mark.parametrize("name", ["tiny", "mid", "serve_large", "large"])
def test_planted_cosines_before_rounding(name):
    """A planted query is c * x + sqrt(1 - c^2) * v with v a unit vector orthogonal to the unit target x:
    with float32 input (one rounding of each component, relative error 2^-24) its cosine to the target is c
    within 1e-6; the drawn c lie in the recipe's range."""
    sp = synth.spec(name, N=3000, B=600, in_dtype=synth.F32, n_dup=min(synth.spec(name).n_dup, 50),
                    n_dup_queries=min(synth.spec(name).n_dup_queries, 20))
    w = synth.generate(sp)
    pl = w.cls != synth.CLS_MISS
    tgt = w.target[pl]
    got = _cos(w.queries[pl], w.keys[tgt])
    assert np.max(np.abs(got - w.cos[pl])) < 1e-6
    assert np.all(w.cos[pl] >= sp.cos_lo) and np.all(w.cos[pl] <= sp.cos_hi)
    assert np.all(np.isnan(w.cos[~pl])) and np.all(w.target[~pl] == -1)


@pytest.mark.parametrize("name,B", [("tiny", 64), ("mid", 256), ("serve_small", 4096), ("serve_large", 4096),
                                    ("large", 1024), ("mid_paper", 256)])
def test_class_counts_are_exact(name, B):
    """Benign / collision / miss counts are round(B * fraction) for the planted classes and the rest misses
    (C3-C5: 40% benign, 10% collision, 50% miss; C1, C2: thirds)."""
    sp = synth.spec(name, N=2000, B=B, n_dup=0, n_dup_queries=0)
    w = synth.generate(sp)
    nb, nc = int(round(B * sp.frac_benign)), int(round(B * sp.frac_collision))
    counts = [int(np.sum(w.cls == c)) for c in (synth.CLS_BENIGN, synth.CLS_COLLISION, synth.CLS_MISS)]
    assert counts == [nb, nc, B - nb - nc]
    if name in ("serve_small", "serve_large"):
        assert counts == [1638, 410, 2048]


def test_duplicate_keys_are_bit_identical():
    """The serving workload's 1,000 exact-duplicate pairs (j < i): key i is a bit copy of key j, the 2,000 rows
    are distinct, prefixes and tokens stay independent; duplicate-aimed benign queries expect the earlier copy."""
    sp = synth.spec("serve_large", N=60_000, B=2048)
    w = synth.generate(sp)
    d = w.dup_pairs
    assert d.shape == (sp.n_dup, 2) == (1000, 2)
    assert np.all(d[:, 0] < d[:, 1]) and len(np.unique(d)) == 2 * sp.n_dup
    np.testing.assert_array_equal(w.keys[d[:, 1]], w.keys[d[:, 0]])
    assert not np.any(np.all(w.emb[d[:, 1]] == w.emb[d[:, 0]], axis=1))
    aimed = np.isin(w.target, d[:, 0]) & (w.cls == synth.CLS_BENIGN)
    assert aimed.sum() >= sp.n_dup_queries
    assert not np.any(np.isin(w.target, d[:, 1]))          # no query expects a later copy


@pytest.mark.parametrize("name", ["mid", "large"])
def test_entry_stream_independent_of_windows_and_threads(name):
    """Rows [0, n) of the entry stream are the same arrays whether drawn at once on one thread, at once on
    several, or in windows of ragged sizes that straddle the generator's chunks."""
    sp = synth.spec(name, N=20_000)
    n = 15_000
    k1, e1, t1 = synth.entries(sp, 0, n, threads=1)
    k4, e4, t4 = synth.entries(sp, 0, n, threads=4)
    parts = []
    r = 0
    for size in (1234, synth.GEN_CHUNK, 7777, n):
        size = min(size, n - r)
        if size <= 0:
            break
        parts.append(synth.entries(sp, r, size, threads=3))
        r += size
    kw, ew, tw = (np.concatenate([p[i] for p in parts]) for i in range(3))
    for a, b in ((k1, k4), (e1, e4), (t1, t4), (k1, kw), (e1, ew), (t1, tw)):
        np.testing.assert_array_equal(a, b)


def test_queries_reproducible():
    """The same spec draws the same query batch; another query stream chunk draws another."""
    sp = synth.spec("mid", N=5000, B=256)
    a, b = synth.generate(sp), synth.generate(sp)
    for f in ("queries", "la_emb", "la_tok", "cls", "target"):
        np.testing.assert_array_equal(getattr(a, f), getattr(b, f))
    q2 = synth.queries(sp, a.keys, a.emb, a.tokens, a.dup_pairs, stream_chunk=1)
    assert not np.array_equal(q2["queries"], a.queries)
