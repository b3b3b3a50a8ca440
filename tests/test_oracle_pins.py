"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each group below fixes one part of the oracle by something independent of it:
a library routine (torch's float->bfloat16 conversion), exact rational
arithmetic, hand-derived closed forms, a brute-force score matrix, or an
invariant the lookup must satisfy.  Sizes keep the whole module to seconds.
"""
import math
from decimal import Decimal, getcontext
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
import synth
from tests import bruteforce as bf

MISS, REJECT, HIT, HIT_EXACT = oracle.MISS, oracle.REJECT, oracle.HIT, oracle.HIT_EXACT
U = 2.0 ** -8  # bfloat16 unit roundoff


def torch_bf16(x32: np.ndarray) -> np.ndarray:
    return torch.from_numpy(np.ascontiguousarray(x32, np.float32)).to(torch.bfloat16).view(torch.int16).numpy() \
        .view(np.uint16)


# --------------------------------------------------------------------------- bf16 rounding


def test_bf16_rne_matches_torch_on_float32_values():
    """On float32 inputs (exact in double) one rounding == torch's nearest-even float->bf16."""
    rng = np.random.default_rng(123)
    bits = rng.integers(0, 2 ** 32, 1_000_000, dtype=np.uint64).astype(np.uint32)
    # force a large share of exact ties (low 16 bits == 0x8000) and near-ties
    bits[:200_000] = (bits[:200_000] & 0xFFFF0000) | 0x8000
    bits[200_000:250_000] = (bits[200_000:250_000] & 0xFFFF0000) | 0x7FFF
    bits[250_000:300_000] = (bits[250_000:300_000] & 0xFFFF0000) | 0x8001
    bits[300_000:350_000] &= 0x807FFFFF  # subnormals
    x = bits.view(np.float32)
    x = x[~np.isnan(x)]
    got = oracle.bf16_rne(x.astype(np.float64))
    want = torch_bf16(x)
    np.testing.assert_array_equal(got, want)


def test_bf16_rne_closed_forms():
    cases = [
        (1.0, 0x3F80),
        (1 + 2 ** -8, 0x3F80),          # halfway between 1 and 1+2^-7: ties to even (down)
        (1 + 3 * 2 ** -8, 0x3F82),      # halfway between 0x3F81 and 0x3F82: ties to even (up)
        (1 + 2 ** -8 + 2 ** -30, 0x3F81),  # just above halfway: up.  (Rounding through float32 first
                                           # would land exactly on the tie and go down: one rounding only.)
        (-0.0, 0x8000),
        (0.0, 0x0000),
        (2.0 ** -133, 0x0001),          # smallest bf16 subnormal
        (2.0 ** -134, 0x0000),          # half of it: tie to even (zero)
        (1.5 * 2.0 ** -134, 0x0001),
        (3.0e38, 0x7F62),
        (3.4e38, 0x7F80),               # beyond the largest finite bf16 (3.3895e38) by more than half an ulp
        (float("inf"), 0x7F80),
        (-float("inf"), 0xFF80),
    ]
    got = oracle.bf16_rne(np.array([v for v, _ in cases]))
    for (v, want), g in zip(cases, got):
        assert g == want, (v, hex(g), hex(want))


# --------------------------------------------------------------------------- quantisation


def _exact_bf16_of(x: Fraction) -> int:
    """bfloat16 bits of the exact rational x, rounded to nearest, ties to even (normal range only)."""
    if x == 0:
        return 0
    s = 0x8000 if x < 0 else 0
    a = abs(x)
    e = math.floor(math.log2(a))
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    ulp = Fraction(2) ** (e - 7)
    m = a / ulp                      # in [128, 256)
    fl = math.floor(m)
    rem = m - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    val = float(fl * ulp)
    return s | (int(np.array(val, np.float32).view(np.uint32)) >> 16)


def test_quantise_matches_exact_normalisation():
    """Normalise exactly (60-digit decimal sqrt, rational division) and round once: the oracle agrees."""
    getcontext().prec = 60
    rng = np.random.default_rng(7)
    x = rng.standard_normal((40, 16)).astype(np.float32)
    x[3] *= 1e-20
    x[4] *= 1e20
    got = oracle.quantise(x, oracle.F32)
    for r in range(x.shape[0]):
        ss = sum(Fraction(float(v)) ** 2 for v in x[r])
        n = Fraction(Decimal(ss.numerator) / Decimal(ss.denominator)).limit_denominator(10 ** 55)
        n = Fraction(Decimal(n.numerator / Decimal(n.denominator)).sqrt())
        for j in range(x.shape[1]):
            want = _exact_bf16_of(Fraction(float(x[r, j])) / n)
            assert got[r, j] == want, (r, j)


def test_quantise_closed_forms():
    q = oracle.quantise(np.array([[3, 4, 0, 0], [0, 0, 7.5, 0], [1, 1, 1, 1], [0, 0, 0, 0],
                                  [-2, 0, 0, 0]], np.float32), oracle.F32)
    np.testing.assert_array_equal(q[0], [0x3F1A, 0x3F4D, 0, 0])     # 0.6 -> 0.6015625, 0.8 -> 0.80078125
    np.testing.assert_array_equal(q[1], [0, 0, 0x3F80, 0])           # a basis vector normalises to 1.0
    np.testing.assert_array_equal(q[2], [0x3F00] * 4)                # 1/2 each, exact
    np.testing.assert_array_equal(q[3], [0, 0, 0, 0])                # zero stays zero
    np.testing.assert_array_equal(q[4], [0xBF80, 0, 0, 0])


def test_quantise_invariances_and_dtypes():
    rng = np.random.default_rng(11)
    x = rng.standard_normal((64, 96)).astype(np.float32)
    q = oracle.quantise(x, oracle.F32)
    # scaling by a power of two is exact and must not change the result
    np.testing.assert_array_equal(oracle.quantise(x * np.float32(2.0 ** 37), oracle.F32), q)
    np.testing.assert_array_equal(oracle.quantise(x * np.float32(2.0 ** -41), oracle.F32), q)
    # negation flips exactly the sign bits
    np.testing.assert_array_equal(oracle.quantise(-x, oracle.F32), q ^ np.uint16(0x8000))
    # a bfloat16 input reads as the float it denotes
    xb = torch_bf16(x)
    np.testing.assert_array_equal(oracle.quantise(xb, oracle.BF16),
                                  oracle.quantise(bf.widen(xb).astype(np.float32), oracle.F32))
    # the quantised rows are unit vectors up to the bf16 rounding of each component
    n = np.linalg.norm(bf.widen(q), axis=1)
    assert np.all(np.abs(n - 1) <= U)


# --------------------------------------------------------------------------- hand-derived lookup


def test_handworked_example():
    """A d=4 cache whose normalised vectors and scores are exact in bfloat16 and float.

    keys   k0 = (1,1,1,1)      -> (1/2,1/2,1/2,1/2)
           k1 = (1,1,1,-1)     -> (1/2,1/2,1/2,-1/2)
           k2 = (2,0,0,0)      -> (1,0,0,0)
           k3 = (3,3,3,3)      -> same as k0 (an exact duplicate after normalisation)
           k4 = (0,0,0,0)      -> zero vector, scores 0 against everything
    queries and their exact scores against k0..k4:
      q0 = (1,1,1,1)           1, 1/2, 1/2, 1, 0      -> idx 0 (tie with 3: lowest), score 1
      q1 = 5*(1,1,1,-1)        1/2, 1, 1/2, 1/2, 0    -> idx 1, score 1
      q2 = (-1,0,0,0)          -1/2,-1/2,-1,-1/2, 0   -> idx 4 (the zero key wins with 0), score 0
      q3 = (0,0,0,0)           0 everywhere            -> idx 0, score 0
      q4 = (1,-1,1,-1)         0, 1/2, 1/2, 0, 0      -> idx 1 (tie with 2: lowest), score 1/2
    tau_q = 1/2: q0, q1, q4 hit (q4 exactly at the threshold: ">="), q2, q3 miss.
    stage 2 (tau_r = 1/2, k = 2):
      q0 -> entry 0: tokens equal                              -> HIT_EXACT, r = e0.a0 = 1
      q1 -> entry 1: tokens differ, r = e1.a1 = 1/2 (= tau_r)  -> HIT
      q4 -> entry 1: tokens differ, r = e1.a4 = -1             -> REJECT
    """
    keys = np.array([[1, 1, 1, 1], [1, 1, 1, -1], [2, 0, 0, 0], [3, 3, 3, 3], [0, 0, 0, 0]], np.float32)
    emb = np.array([[1, 0, 0, 0], [1, 1, 1, 1], [0, 1, 0, 0], [0, 0, 1, 0], [0, 0, 0, 1]], np.float32)
    tokens = np.array([[5, 6, 7], [8, 9, 10], [1, 2, 3], [5, 6, 7], [0, 0, 0]], np.int32)
    queries = np.array([[1, 1, 1, 1], [5, 5, 5, -5], [-1, 0, 0, 0], [0, 0, 0, 0], [1, -1, 1, -1]], np.float32)
    la = np.array([[1, 0, 0, 0], [1, 1, 1, -1], [1, 0, 0, 0], [1, 0, 0, 0], [-1, -1, -1, -1]], np.float32)
    la_tok = np.array([[5, 6], [8, 0], [1, 2], [0, 0], [8, 9 + 1]], np.int32)
    c = oracle.OracleCache(4, 3, oracle.F32)
    assert c.insert(keys, emb, tokens) == 0
    out = c.lookup(queries, la, la_tok, 0.5, 0.5, 2)
    np.testing.assert_array_equal(out["idx"], [0, 1, 4, 0, 1])
    np.testing.assert_array_equal(out["score"], np.float32([1, 1, 0, 0, 0.5]))
    np.testing.assert_array_equal(out["decision"], [HIT_EXACT, HIT, MISS, MISS, REJECT])
    r = out["resp_score"]
    assert r[0] == 1.0 and r[1] == 0.5 and r[4] == -1.0
    assert np.isnan(r[2]) and np.isnan(r[3])
    np.testing.assert_array_equal(out["margin"], [0.0, 0.5, 0.5, 0.0, 0.0])


# --------------------------------------------------------------------------- brute force


def _random_case(rng, N, d, B, k_cap, dup=0):
    keys = oracle.quantise(rng.standard_normal((N, d)).astype(np.float32), oracle.F32)
    if dup and N > 1:
        src = rng.integers(0, N, dup)
        dst = rng.integers(0, N, dup)
        keys[dst] = keys[src]
    emb = oracle.quantise(rng.standard_normal((N, d)).astype(np.float32), oracle.F32)
    tokens = rng.integers(0, 50, (N, k_cap), dtype=np.int32)
    q = oracle.quantise(rng.standard_normal((B, d)).astype(np.float32), oracle.F32)
    a = oracle.quantise(rng.standard_normal((B, d)).astype(np.float32), oracle.F32)
    return keys, emb, tokens, q, a


@pytest.mark.parametrize("N,d,B,k_cap,k", [(1, 32, 5, 1, 1), (2, 32, 9, 8, 8), (7, 64, 16, 20, 20),
                                           (300, 64, 33, 64, 64), (2000, 384, 64, 150, 150),
                                           (1500, 96, 40, 150, 65)])
def test_lookup_matches_bruteforce(N, d, B, k_cap, k):
    rng = np.random.default_rng(N * 1000 + d)
    keys, emb, tokens, q, a = _random_case(rng, N, d, B, k_cap, dup=N // 10)
    # plant: some queries equal to stored keys (hits) with stored tokens (exact) or a near-far embedding
    pick = rng.integers(0, N, B)
    half = B // 2
    q[:half] = keys[pick[:half]]
    u = rng.integers(0, 50, (B, k), dtype=np.int32)
    u[: half // 2] = tokens[pick[: half // 2], :k]
    a[half // 2: half] = emb[pick[half // 2: half]]
    for tau_q, tau_r in [(0.9, 0.85), (-1.0, -1.0), (0.0, 0.3), (1.5, 0.0)]:
        o = oracle.lookup(keys, emb, tokens, q, a, u, tau_q, tau_r, k)
        w = bf.lookup(keys, emb, tokens, q, a, u, tau_q, tau_r, k)
        np.testing.assert_array_equal(o["idx"], w["idx"])
        np.testing.assert_array_equal(o["score"], w["score"])
        np.testing.assert_array_equal(o["decision"], w["decision"])
        np.testing.assert_array_equal(o["resp_score"], w["resp_score"])  # NaN positions match too
        S = w["S"]
        best = S.max(axis=1)
        second = np.where(S == best[:, None], -np.inf, S).max(axis=1)
        n_best = (S == best[:, None]).sum(axis=1)
        want_margin = np.where(n_best > 1, 0.0, best - second)
        np.testing.assert_array_equal(o["margin"], want_margin)


def test_decide_at_arbitrary_entry_matches_bruteforce():
    rng = np.random.default_rng(5)
    keys, emb, tokens, q, a = _random_case(rng, 50, 32, 20, 8)
    u = rng.integers(0, 50, (20, 8), dtype=np.int32)
    at = rng.integers(0, 50, 20).astype(np.int32)
    q[:10] = keys[at[:10]]
    u[:5] = tokens[at[:5]]
    o = oracle.decide(keys, emb, tokens, q, a, u, 0.5, 0.1, 8, at)
    S = bf.scores(q, keys)
    np.testing.assert_array_equal(o["s"], S[np.arange(20), at])
    for b in range(20):
        one = bf.lookup(keys[at[b]:at[b] + 1], emb[at[b]:at[b] + 1], tokens[at[b]:at[b] + 1], q[b:b + 1],
                        a[b:b + 1], u[b:b + 1], 0.5, 0.1, 8)
        assert o["decision"][b] == one["decision"][0]
        assert o["score"][b] == one["score"][0]


def test_empty_and_single_entry():
    rng = np.random.default_rng(3)
    keys, emb, tokens, q, a = _random_case(rng, 1, 16, 4, 4)
    u = rng.integers(0, 50, (4, 4), dtype=np.int32)
    o = oracle.lookup(keys[:0], emb[:0], tokens[:0], q, a, u, 0.9, 0.85, 4)
    np.testing.assert_array_equal(o["idx"], -1)
    assert np.all(np.isnan(o["score"])) and np.all(np.isnan(o["resp_score"]))
    np.testing.assert_array_equal(o["decision"], MISS)
    o = oracle.lookup(keys, emb, tokens, q, a, u, -2.0, 0.85, 4)
    np.testing.assert_array_equal(o["idx"], 0)
    assert np.all(np.isinf(o["margin"]))


# --------------------------------------------------------------------------- invariants


def _store(rng, N, d, k_cap=8, vocab=1000):
    keys = oracle.quantise(rng.standard_normal((N, d)).astype(np.float32), oracle.F32)
    emb = oracle.quantise(rng.standard_normal((N, d)).astype(np.float32), oracle.F32)
    tokens = rng.integers(0, vocab, (N, k_cap), dtype=np.int32)
    return keys, emb, tokens


def test_self_query_returns_itself_with_unit_score():
    rng = np.random.default_rng(21)
    raw = rng.standard_normal((3000, 64)).astype(np.float32)
    c = oracle.OracleCache(64, 8, oracle.F32)
    c.insert(raw, rng.standard_normal((3000, 64)).astype(np.float32), rng.integers(0, 9, (3000, 8)))
    sel = rng.integers(0, 3000, 50)
    out = c.lookup(raw[sel], raw[sel], c.tokens[sel], 0.9, 0.85, 8)
    want = [oracle.first_identical(c.keys, i) for i in sel]
    np.testing.assert_array_equal(out["idx"], want)
    assert np.all(out["score"] <= 1.0) and np.all(out["score"] >= (1 - U) ** 2)
    np.testing.assert_array_equal(out["decision"], HIT_EXACT)


def test_first_identical_against_bruteforce():
    """The lowest index whose stored key is bitwise identical to entry i (the exact-tie rule's reference):
    copies planted at known positions -- a later copy names its earliest original, including chains of three
    copies, a copy of the store's first row and a copy that is its last row -- against a brute force over the whole store; a unique row
    names itself; a row differing from another in a single bf16 ulp (in a middle or the last element), or by
    the sign of a zero, is no copy;
    an index outside the store names -1."""
    rng = np.random.default_rng(91)
    N, d = 400, 37
    kq = oracle.quantise(rng.standard_normal((N, d)).astype(np.float32), oracle.F32)
    kq[57] = kq[12]                       # a plain copy
    kq[200] = kq[12]                      # a second copy of the same row
    kq[150] = kq[90]
    kq[N - 1] = kq[3]                     # the last row
    kq[250] = kq[0]                       # a copy of the first row
    kq[301] = kq[300]
    kq[301, 5] ^= 1                       # one bf16 ulp apart: not a copy
    kq[310] = kq[305]
    kq[310, d - 1] ^= 1                   # differs only in the last element
    kq[320] = 0
    kq[321] = 0
    kq[321, 0] = 0x8000                   # -0 against +0 bits: bitwise different
    for i in range(N):
        want = next(j for j in range(i + 1) if np.array_equal(kq[j], kq[i]))
        assert oracle.first_identical(kq, i) == want, i
    assert [oracle.first_identical(kq, i) for i in (57, 200, 150, N - 1, 250)] == [12, 12, 90, 3, 0]
    assert oracle.first_identical(kq, 301) == 301 and oracle.first_identical(kq, 310) == 310
    assert oracle.first_identical(kq, 321) == 321 and oracle.first_identical(kq, 320) == 320
    assert oracle.first_identical(kq, 0) == 0
    assert oracle.first_identical(kq, -1) == -1 and oracle.first_identical(kq, N) == -1


def test_scores_in_unit_interval_and_permutation_invariance():
    rng = np.random.default_rng(22)
    keys, emb, tokens = _store(rng, 2500, 48)
    keys[100] = keys[7]                      # an exact duplicate pair
    q = oracle.quantise(rng.standard_normal((40, 48)).astype(np.float32), oracle.F32)
    q[0] = keys[100]
    q[1] = keys[5]
    a = q.copy()
    u = rng.integers(0, 1000, (40, 8), dtype=np.int32)
    o = oracle.lookup(keys, emb, tokens, q, a, u, 0.2, 0.1, 8)
    assert np.all(np.abs(o["score"]) <= 1)
    rs = o["resp_score"][~np.isnan(o["resp_score"])]
    assert np.all(np.abs(rs) <= 1)
    assert o["idx"][0] == 7
    perm = rng.permutation(2500)
    inv = np.argsort(perm)
    p = oracle.lookup(keys[perm], emb[perm], tokens[perm], q, a, u, 0.2, 0.1, 8)
    # the winner is the same entry, except that the duplicate pair now resolves to whichever copy comes first
    same = inv[o["idx"]] == p["idx"]
    dup_row = np.isin(o["idx"], [7, 100])
    assert np.all(same | dup_row)
    assert p["idx"][0] == min(inv[7], inv[100])
    np.testing.assert_array_equal(p["score"], o["score"])
    # stage 2 reads the winner's own prefix, which differs between the two copies of the duplicate
    np.testing.assert_array_equal(p["decision"][~dup_row], o["decision"][~dup_row])
    np.testing.assert_array_equal(p["resp_score"][~dup_row], o["resp_score"][~dup_row])
    r0 = np.clip(np.float32(bf.widen(a[0]) @ bf.widen(emb[perm][p["idx"][0]])), -1, 1)
    assert p["resp_score"][0] == r0


def test_all_negative_scores():
    rng = np.random.default_rng(23)
    x = rng.standard_normal(32).astype(np.float32)
    c = oracle.OracleCache(32, 2, oracle.F32)
    c.insert(np.stack([x, 2 * x, x]), np.stack([x, x, x]), np.zeros((3, 2)))
    out = c.lookup((-x)[None], x[None], np.zeros((1, 2)), -1.0, 0.0, 2)
    assert out["idx"][0] == 0
    assert -1.0 <= out["score"][0] <= -(1 - U) ** 2


def test_planted_queries_closed_form_and_classes():
    """q = c x + sqrt(1-c^2) v (v orthogonal to x) has cosine c with x: after the bf16 rounding of both
    sides the oracle's score must stay within the rounding bound of c; benign plants are served
    (HIT_EXACT), collisions rejected, misses missed -- the synthetic analogues of BHR = 1, AHR = 0."""
    for name, N in [("tiny", 3000), ("mid", 3000)]:
        w = synth.generate(name, N=N)
        sp = w.spec
        c = oracle.OracleCache(sp.d, sp.k_cap, sp.in_dtype)
        c.insert(w.keys, w.emb, w.tokens)
        o = c.lookup(w.queries, w.la_emb, w.la_tok, sp.tau_q, sp.tau_r, sp.k)
        pl = w.cls != synth.CLS_MISS
        # worst case: every component of both vectors moves by <= u relative, per rounding
        bound = (2 * U + U * U) if sp.in_dtype == oracle.F32 else (4 * U + 6 * U * U)
        err = np.abs(o["s_best"][pl] - w.cos[pl])
        assert np.all(err <= bound), err.max()
        assert err.mean() < 1e-3
        np.testing.assert_array_equal(o["idx"][pl], w.target[pl])
        clear = pl & (w.cos >= sp.tau_q + 2e-3)
        ben = clear & (w.cls == synth.CLS_BENIGN)
        col = clear & (w.cls == synth.CLS_COLLISION)
        assert ben.sum() > 5 and col.sum() > 5
        np.testing.assert_array_equal(o["decision"][ben], HIT_EXACT)
        np.testing.assert_array_equal(o["decision"][col], REJECT)
        np.testing.assert_array_equal(o["decision"][~pl], MISS)
        below = pl & (w.cos < sp.tau_q - 2e-2)
        np.testing.assert_array_equal(o["decision"][below], MISS)


def test_threshold_special_cases():
    rng = np.random.default_rng(24)
    keys, emb, tokens = _store(rng, 500, 40)
    q = oracle.quantise(rng.standard_normal((30, 40)).astype(np.float32), oracle.F32)
    q[:10] = keys[:10]
    a = oracle.quantise(rng.standard_normal((30, 40)).astype(np.float32), oracle.F32)
    u = rng.integers(0, 1000, (30, 8), dtype=np.int32)
    # tau_r <= -1: stage 2 always passes, leaving thresholded top-1 (MIPS) -- pinned by numpy's argmax
    o = oracle.lookup(keys, emb, tokens, q, a, u, 0.1, -1.0, 8)
    S = bf.scores(q, keys)
    np.testing.assert_array_equal(o["idx"], np.argmax(S, axis=1))
    hit = o["score"] >= np.float32(0.1)
    assert np.all(np.isin(o["decision"][hit], [HIT, HIT_EXACT]))
    np.testing.assert_array_equal(o["decision"][~hit], MISS)
    # tau_q > 1: nothing is a hit, stage 2 never runs
    o = oracle.lookup(keys, emb, tokens, q, a, u, 1.0001, 0.0, 8)
    np.testing.assert_array_equal(o["decision"], MISS)
    assert np.all(np.isnan(o["resp_score"]))


def test_stage2_alone():
    """Stage 2 is a dot product of the two quantised prefix embeddings and an equality of k tokens."""
    rng = np.random.default_rng(25)
    keys, emb, tokens = _store(rng, 1, 64, k_cap=16)
    a = oracle.quantise(rng.standard_normal((6, 64)).astype(np.float32), oracle.F32)
    a[0] = emb[0]
    u = np.tile(tokens[0, :5], (6, 1))
    u[2, 4] += 1                              # differs only in the last compared position
    u[3, 0] += 1
    q = np.tile(keys[0], (6, 1))
    o = oracle.lookup(keys, emb, tokens, q, a, u, 0.5, 2.0, 5)   # tau_r > 1: only the token path can pass
    r = np.clip(np.float32(bf.widen(a) @ bf.widen(emb[0])), -1, 1)
    np.testing.assert_array_equal(o["resp_score"], r)
    np.testing.assert_array_equal(o["decision"], [HIT_EXACT, HIT_EXACT, REJECT, REJECT, HIT_EXACT,
                                                  HIT_EXACT])
    # tokens equal but the embedding far: the identical-token rule decides (HIT_EXACT)
    a2 = -emb[[0]]
    o = oracle.lookup(keys, emb, tokens, keys[[0]], a2, tokens[[0], :5], 0.5, 0.9, 5)
    assert o["decision"][0] == HIT_EXACT and o["resp_score"][0] < -0.99
    # k = 1 compares only the first token; k = k_cap compares all of them
    u1 = tokens[[0], :16].copy()
    u1[0, 15] += 1
    assert oracle.lookup(keys, emb, tokens, keys[[0]], -emb[[0]], u1[:, :1], 0.5, 0.9, 1)["decision"][0] == HIT_EXACT
    assert oracle.lookup(keys, emb, tokens, keys[[0]], -emb[[0]], u1, 0.5, 0.9, 16)["decision"][0] == REJECT


def test_paper_thresholds_fixture():
    """The paper-shaped workload uses the thresholds and window the paper calibrates (Appendix A.2)."""
    import json
    import os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_thresholds.json")))
    sp = synth.spec("mid_paper")
    bge = g["tau_c"]["BGE"]
    assert np.float32(sp.tau_q) == np.float32(min(bge["cap"], bge["P5"]))
    qb = g["tau_a"]["Qwen3+BGE"]
    assert np.float32(sp.tau_r) == np.float32(min(qb["cap"], qb["P10"]))
    assert sp.k == g["k"] and sp.d == g["embedding_dim"]["BGE"]
    for name, row in g["tau_a"].items():
        assert abs(min(row["cap"], row["P10"]) - row["used"]) < 1e-9, name


# --------------------------------------------------------------------------- ensemble of lookahead checks


def _ensemble_case(rng, N, d, dms, B, k_cap):
    keys = oracle.quantise(rng.standard_normal((N, d)).astype(np.float32), oracle.F32)
    embs = [oracle.quantise(rng.standard_normal((N, dm)).astype(np.float32), oracle.F32) for dm in dms]
    tokens = rng.integers(0, 20, (N, k_cap), dtype=np.int32)
    q = oracle.quantise(rng.standard_normal((B, d)).astype(np.float32), oracle.F32)
    pick = rng.integers(0, N, B)
    q[: B // 2] = keys[pick[: B // 2]]
    las = []
    for e, dm in zip(embs, dms):
        a = rng.standard_normal((B, dm)).astype(np.float32)
        # some lookaheads close to the candidate's prefix under this model, some far
        # noise scales spread the prefix cosines of the close ones over roughly 0.45 .. 0.98
        scale = rng.uniform(0.2, 2.0, (B // 3, 1)).astype(np.float32)
        a[: B // 3] = bf.widen(e[pick[: B // 3]]) + scale * rng.standard_normal((B // 3, dm)).astype(np.float32) \
            / np.sqrt(dm)
        las.append(oracle.quantise(a, oracle.F32))
    u = rng.integers(0, 20, (B, k_cap), dtype=np.int32)
    u[: B // 6] = tokens[pick[: B // 6]]
    return keys, embs, tokens, q, las, u


def test_ensemble_of_one_is_the_plain_lookup():
    rng = np.random.default_rng(31)
    keys, embs, tokens, q, las, u = _ensemble_case(rng, 400, 48, [48], 60, 6)
    for tq, tr in [(0.5, 0.6), (-1.0, -1.0), (0.9, 0.99)]:
        e = oracle.lookup_ensemble(keys, q, tq, embs, las, [tr], tokens, u, 6)
        o = oracle.lookup(keys, embs[0], tokens, q, las[0], u, tq, tr, 6)
        np.testing.assert_array_equal(e["idx"], o["idx"])
        np.testing.assert_array_equal(e["score"], o["score"])
        np.testing.assert_array_equal(e["decision"], o["decision"])
        np.testing.assert_array_equal(e["resp_score"][:, 0], o["resp_score"])


def test_ensemble_matches_bruteforce_and_rule():
    """Section 4.4: the lookahead passes only if every one of the m checks passes (identical tokens pass all)."""
    rng = np.random.default_rng(32)
    dms = [32, 48, 64]
    keys, embs, tokens, q, las, u = _ensemble_case(rng, 500, 40, dms, 90, 5)
    S = bf.scores(q, keys)
    idx = np.argmax(S, axis=1)
    score = np.clip(S[np.arange(90), idx].astype(np.float32), -1, 1)
    hit = score >= np.float32(0.5)
    R = np.stack([np.clip(np.einsum("bd,bd->b", bf.widen(a), bf.widen(em[idx])).astype(np.float32), -1, 1)
                  for a, em in zip(las, embs)], axis=1)
    tok_eq = np.all(u == tokens[idx], axis=1)
    # fixed thresholds, then per-model thresholds at different quantiles of that model's own prefix scores,
    # so that applying one model's threshold to another changes decisions
    close = R[hit & (R.min(axis=1) > 0.2)]
    assert len(close) >= 10
    quant = [float(np.quantile(close[:, i], qv)) for i, qv in enumerate((0.1, 0.4, 0.25))]
    for taus in ([0.3, 0.5, 0.4], quant, quant[::-1]):
        e = oracle.lookup_ensemble(keys, q, 0.5, embs, las, taus, tokens, u, 5)
        np.testing.assert_array_equal(e["idx"], idx)
        all_pass = np.all(R >= np.array(taus, np.float32)[None, :], axis=1)
        want = np.where(~hit, oracle.MISS, np.where(tok_eq, oracle.HIT_EXACT,
                                                   np.where(all_pass, oracle.HIT, oracle.REJECT)))
        np.testing.assert_array_equal(e["decision"], want)
        np.testing.assert_array_equal(e["resp_score"][hit], R[hit])
        assert np.all(np.isnan(e["resp_score"][~hit]))
        assert (e["decision"] == oracle.HIT).sum() > 3 and (e["decision"] == oracle.REJECT).sum() > 3


def test_ensemble_monotone_and_order_free():
    """More checks can only reject more (never accept a rejected query); the order of the models is irrelevant;
    a model whose threshold is -1 changes nothing."""
    rng = np.random.default_rng(33)
    dms = [32, 64, 48, 40]
    keys, embs, tokens, q, las, u = _ensemble_case(rng, 300, 32, dms, 80, 4)
    taus = [0.35, 0.45, 0.3, 0.5]
    prev = None
    for m in range(1, 5):
        e = oracle.lookup_ensemble(keys, q, 0.4, embs[:m], las[:m], taus[:m], tokens, u, 4)
        if prev is not None:
            was_rejected = prev["decision"] == oracle.REJECT
            assert np.all(e["decision"][was_rejected] == oracle.REJECT)
        prev = e
    perm = [2, 0, 3, 1]
    p = oracle.lookup_ensemble(keys, q, 0.4, [embs[i] for i in perm], [las[i] for i in perm], [taus[i] for i in perm],
                               tokens, u, 4)
    np.testing.assert_array_equal(p["decision"], prev["decision"])
    np.testing.assert_array_equal(p["resp_score"], prev["resp_score"][:, perm])
    two = oracle.lookup_ensemble(keys, q, 0.4, embs[:2], las[:2], taus[:2], tokens, u, 4)
    loose = oracle.lookup_ensemble(keys, q, 0.4, embs[:3], las[:3], taus[:2] + [-1.0], tokens, u, 4)
    np.testing.assert_array_equal(two["decision"], loose["decision"])


# --------------------------------------------------------------------------- threshold calibration (Appendix A.2)


def _pairs(rng, n, d):
    a = rng.standard_normal((n, d)).astype(np.float32)
    # a spread of pair cosines: b = a + noise of a random scale per pair
    scale = rng.uniform(0.05, 3.0, (n, 1)).astype(np.float32)
    b = a + scale * rng.standard_normal((n, d)).astype(np.float32)
    return oracle.quantise(a, oracle.F32), oracle.quantise(b, oracle.F32)


@pytest.mark.parametrize("n,d", [(1, 16), (2, 16), (7, 40), (500, 384), (1001, 64)])
def test_calibration_matches_numpy_percentile(n, d):
    """The pair cosines are dot products of the quantised vectors; the percentile is numpy's default
    (linear between closest ranks); the threshold is min(cap, percentile)."""
    rng = np.random.default_rng(41 + n)
    a, b = _pairs(rng, n, d)
    sims = np.clip(np.einsum("nd,nd->n", bf.widen(a), bf.widen(b)), -1.0, 1.0)
    for p in (0.0, 5.0, 10.0, 37.5, 50.0, 90.0, 99.0, 100.0):
        for cap in (0.8, 0.3, 2.0):
            o = oracle.calibrate(a, b, p, cap)
            np.testing.assert_allclose(o["sims"], sims, rtol=0, atol=1e-12)
            want = float(np.percentile(sims, p))
            assert abs(o["P"] - want) <= 1e-12, (p, o["P"], want)
            assert o["tau"] == min(cap, o["P"])


def test_calibration_closed_forms():
    rng = np.random.default_rng(44)
    x = rng.uniform(-1, 1, 11)
    s = np.sort(x)
    assert oracle.threshold_rule(x, 0.0, 9.0)[0] == s[0]
    assert oracle.threshold_rule(x, 100.0, 9.0)[0] == s[-1]
    assert oracle.threshold_rule(x, 50.0, 9.0)[0] == s[5]            # h = 5 exactly
    assert oracle.threshold_rule(x, 10.0, 9.0)[0] == s[1]            # h = 1 exactly
    h = 10 * 0.25
    assert abs(oracle.threshold_rule(x, 25.0, 9.0)[0] - (s[2] + (h - 2) * (s[3] - s[2]))) <= 1e-15
    for p in (0.0, 33.0, 100.0):
        assert oracle.threshold_rule([0.42], p, 9.0)[0] == 0.42     # one pair: every percentile is it
    assert oracle.threshold_rule(x, 50.0, -5.0)[1] == -5.0           # the cap binds
    # monotone in p, and order-free
    ps = np.linspace(0, 100, 41)
    vals = [oracle.threshold_rule(x, p, 9.0)[0] for p in ps]
    assert all(v1 <= v2 for v1, v2 in zip(vals, vals[1:]))
    assert oracle.threshold_rule(x[::-1], 37.0, 9.0) == oracle.threshold_rule(x, 37.0, 9.0)
    # identical pairs have cosine 1 (up to the bf16 rounding of the normalised vector)
    a, _ = _pairs(rng, 5, 64)
    o = oracle.calibrate(a, a, 50.0, 2.0)
    assert np.all(np.abs(o["sims"] - 1.0) <= 64 * 2.0 ** -8)


def test_calibration_reproduces_the_paper_table():
    """Appendix A.2 prints the natural percentiles and the thresholds used: tau_c = min(0.80, P5) for BGE
    and MiniLM, tau_a = min(0.70, P10) for four (LLM, embedding) pairs.  A similarity set whose percentile
    sits exactly on an order statistic (n = 21 for P5, n = 11 for P10: h = 1) must give the printed
    threshold."""
    import json
    import os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_thresholds.json")))
    rng = np.random.default_rng(45)
    for table, p, n, key in (("tau_c", 5.0, 21, "P5"), ("tau_a", 10.0, 11, "P10")):
        for name, row in g[table].items():
            x = np.concatenate([[row[key]], rng.uniform(row[key] + 1e-3, 1.0, n - 2), [-0.5]])
            rng.shuffle(x)
            P, tau = oracle.threshold_rule(x, p, row["cap"])
            assert P == row[key], (name, P)
            assert abs(tau - row["used"]) <= 1e-12, (name, tau, row["used"])


# --------------------------------------------------------------------------- speculative-decoding acceptance (Section 4.3)


def _softmax_rows(x):
    import scipy.special
    return scipy.special.softmax(np.asarray(x, np.float64), axis=-1)


@pytest.mark.parametrize("dtype", [oracle.F32, oracle.BF16])
def test_accept_length_matches_bruteforce(dtype):
    rng = np.random.default_rng(71 + dtype)
    B, k, V = 6, 9, 1000
    lg = (rng.standard_normal((B, k, V)) * 3.0).astype(np.float32)
    if dtype == oracle.BF16:
        lg_in = synth.to_bf16_bits(lg)
        lg = synth.bf16_bits_to_f64(lg_in).astype(np.float64)
    else:
        lg_in = lg
    tok = rng.integers(0, V, (B, k), dtype=np.int32)
    tok[:, ::2] = np.argmax(lg, axis=-1)[:, ::2]           # some likely tokens
    P = _softmax_rows(lg)
    pt = np.take_along_axis(P, tok[..., None], axis=-1)[..., 0]
    pd = (pt * np.exp(rng.normal(0, 0.7, (B, k)))).astype(np.float32)
    o = oracle.accept_length(lg_in, dtype, tok, pd)
    np.testing.assert_allclose(o["p_target"], pt, rtol=1e-12, atol=0)
    acc = pt >= pd.astype(np.float64)
    want = np.array([np.argmin(np.append(a, False)) for a in acc])      # first rejection (k if none)
    np.testing.assert_array_equal(o["accept_len"], want)
    assert 0 < want.sum() < B * k


def test_accept_length_closed_forms():
    V, k = 4, 6
    zeros = np.zeros((1, k, V), np.float32)              # uniform: P_f = 1/4 exactly
    tok = np.zeros((1, k), np.int32)
    assert np.all(oracle.accept_length(zeros, oracle.F32, tok, np.full((1, k), 0.25, np.float32))["p_target"] == 0.25)
    # equality accepts (the rule is P_f >= P_g)
    assert oracle.accept_length(zeros, oracle.F32, tok, np.full((1, k), 0.25, np.float32))["accept_len"][0] == k
    assert oracle.accept_length(zeros, oracle.F32, tok, np.full((1, k), np.nextafter(np.float32(0.25), 1), np.float32))[
        "accept_len"][0] == 0
    assert oracle.accept_length(zeros, oracle.F32, tok, np.zeros((1, k), np.float32))["accept_len"][0] == k
    assert oracle.accept_length(zeros, oracle.F32, tok, np.full((1, k), 1.5, np.float32))["accept_len"][0] == 0
    # only the leading run counts: accept, accept, reject, accept, ... -> 2
    pd = np.array([[0.1, 0.2, 0.3, 0.1, 0.1, 0.1]], np.float32)
    assert oracle.accept_length(zeros, oracle.F32, tok, pd)["accept_len"][0] == 2
    # one dominant logit: P_f ~ 1 without overflow; an out-of-range token has probability 0
    big = np.zeros((1, 2, 50), np.float32)
    big[0, :, 7] = 1000.0
    o = oracle.accept_length(big, oracle.F32, np.array([[7, 50]], np.int32), np.array([[0.99, 0.0]], np.float32))
    assert abs(o["p_target"][0, 0] - 1.0) < 1e-12 and o["p_target"][0, 1] == 0.0 and o["accept_len"][0] == 2


def test_accept_length_invariances():
    rng = np.random.default_rng(73)
    B, k, V = 4, 8, 300
    # logits on a 2^-10 grid, so that adding 8 is exact in float32
    lg = (np.round(rng.standard_normal((B, k, V)) * 2 * 1024) / 1024).astype(np.float32)
    tok = rng.integers(0, V, (B, k), dtype=np.int32)
    pd = rng.uniform(0, 0.02, (B, k)).astype(np.float32)
    base = oracle.accept_length(lg, oracle.F32, tok, pd)
    assert np.array_equal((lg + np.float32(8.0)).astype(np.float64), lg.astype(np.float64) + 8.0)
    shifted = oracle.accept_length(lg + np.float32(8.0), oracle.F32, tok, pd)
    np.testing.assert_allclose(shifted["p_target"], base["p_target"], rtol=1e-12)
    perm = rng.permutation(V)
    inv = np.argsort(perm)
    permuted = oracle.accept_length(lg[..., perm], oracle.F32, inv[tok].astype(np.int32), pd)
    np.testing.assert_allclose(permuted["p_target"], base["p_target"], rtol=1e-12)
    prev = base["accept_len"]
    for f in (1.5, 3.0, 10.0):                                        # stricter drafts never accept more
        cur = oracle.accept_length(lg, oracle.F32, tok, (pd * f).astype(np.float32))["accept_len"]
        assert np.all(cur <= prev)
        prev = cur


# --------------------------------------------------------------------------- LSH index for stage 1 (Eq. (1))


def test_simhash_is_the_sign_of_the_projections():
    rng = np.random.default_rng(81)
    n, d, bits = 300, 48, 96
    z = oracle.quantise(rng.standard_normal((n, d)).astype(np.float32), oracle.F32)
    z[5] = 0                                                   # zero vector: every projection is 0 -> all bits 1
    r = synth.hyperplanes(bits, d, seed=3)
    sig, proj = oracle.simhash(z, r, bits)
    P = bf.widen(z) @ bf.widen(r).T
    np.testing.assert_allclose(proj, P, rtol=0, atol=1e-12)
    want = np.zeros((n, bits // 32), np.uint32)
    for i in range(bits):
        want[:, i // 32] |= (P[:, i] >= 0).astype(np.uint32) << np.uint32(i % 32)
    np.testing.assert_array_equal(sig, want)
    assert np.all(sig[5] == 0xFFFFFFFF)


def test_simhash_collision_probability_is_one_minus_angle_over_pi():
    """Random hyperplanes: two vectors at angle theta agree on a bit with probability 1 - theta/pi
    (the gapped collision property of Eq. (1) for cosine distance)."""
    rng = np.random.default_rng(82)
    d, bits = 64, 8192
    r = synth.hyperplanes(bits, d, seed=4)
    x = rng.standard_normal(d)
    x /= np.linalg.norm(x)
    v = rng.standard_normal(d)
    v -= (v @ x) * x
    v /= np.linalg.norm(v)
    for theta in (0.1, 0.5, 1.0, np.pi / 2, 2.5):
        y = np.cos(theta) * x + np.sin(theta) * v
        z = oracle.quantise(np.stack([x, y]).astype(np.float32), oracle.F32)
        sig, _ = oracle.simhash(z, r, bits)
        agree = bits - sum(bin(int(w)).count("1") for w in (sig[0] ^ sig[1]))
        ang = np.arccos(np.clip(bf.widen(z[0]) @ bf.widen(z[1]), -1, 1))
        p = 1 - ang / np.pi
        assert abs(agree / bits - p) <= 4 * np.sqrt(p * (1 - p) / bits) + 1e-3, (theta, agree / bits, p)


def _lsh_case(rng, N=600, d=40, bits=64, B=50):
    keys, emb, tok = _store(rng, N, d, k_cap=6, vocab=20)
    q = keys[rng.integers(0, N, B)].copy()
    noise = oracle.quantise(rng.standard_normal((B, d)).astype(np.float32), oracle.F32)
    mix = (0.9 * bf.widen(q) + 0.3 * bf.widen(noise)).astype(np.float32)
    q = oracle.quantise(mix, oracle.F32)
    q[:5] = keys[:5]                                           # self queries
    a = oracle.quantise(rng.standard_normal((B, d)).astype(np.float32), oracle.F32)
    u = rng.integers(0, 20, (B, 6), dtype=np.int32)
    r = synth.hyperplanes(bits, d, seed=int(rng.integers(1 << 30)))
    sk, _ = oracle.simhash(keys, r, bits)
    sq, _ = oracle.simhash(q, r, bits)
    return keys, emb, tok, q, a, u, sk, sq, bits


def test_lsh_lookup_matches_bruteforce_candidates():
    rng = np.random.default_rng(83)
    keys, emb, tok, q, a, u, sk, sq, bits = _lsh_case(rng)
    S = bf.scores(q, keys)
    H = np.array([[sum(bin(int(w)).count("1") for w in (sq[b] ^ sk[i])) for i in range(len(keys))]
                  for b in range(len(q))])
    for radius in (0, 3, 10, 20, bits):
        o = oracle.lookup_lsh(keys, emb, tok, sk, q, sq, a, u, radius, 0.5, 0.6, 6)
        cand = H <= radius
        np.testing.assert_array_equal(o["n_cand"], cand.sum(axis=1))
        masked = np.where(cand, S, -np.inf)
        want = np.where(cand.any(axis=1), np.argmax(masked, axis=1), -1)
        np.testing.assert_array_equal(o["idx"], want)
        full = o["idx"] >= 0
        np.testing.assert_allclose(o["score"][full], np.clip(S[full, want[full]], -1, 1).astype(np.float32),
                                   rtol=0, atol=1e-6)
        assert np.all(np.isnan(o["score"][~full])) and np.all(o["decision"][~full] == oracle.MISS)
        assert np.all(o["idx"][:5] == np.arange(5)) or radius < 0      # a self query is always a candidate
    # radius = bits: every entry is a candidate, so the LSH lookup is the exact lookup
    e = oracle.lookup(keys, emb, tok, q, a, u, 0.5, 0.6, 6)
    o = oracle.lookup_lsh(keys, emb, tok, sk, q, sq, a, u, bits, 0.5, 0.6, 6)
    for f in ("idx", "score", "decision"):
        np.testing.assert_array_equal(o[f], e[f])
    np.testing.assert_array_equal(np.isnan(o["resp_score"]), np.isnan(e["resp_score"]))


def test_lsh_radius_monotone():
    rng = np.random.default_rng(84)
    keys, emb, tok, q, a, u, sk, sq, bits = _lsh_case(rng)
    prev_n, prev_s = None, None
    for radius in range(0, bits + 1, 4):
        o = oracle.lookup_lsh(keys, emb, tok, sk, q, sq, a, u, radius, 0.5, 0.6, 6)
        s = np.where(o["idx"] >= 0, o["score"], -np.inf)
        if prev_n is not None:
            assert np.all(o["n_cand"] >= prev_n) and np.all(s >= prev_s)
        prev_n, prev_s = o["n_cand"], s
