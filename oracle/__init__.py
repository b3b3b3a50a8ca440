"""CPU oracle for the LaCache two-stage cache lookup.

TEST INFRASTRUCTURE ONLY.  The product package never imports this module; only
the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` do.  It wraps ``lacache_oracle.c`` (plain C, IEEE double, OpenMP
over queries) through ctypes and shares nothing with the HIP path.

What it computes, and the passages it follows, is stated in the header of
``lacache_oracle.c``: L2-normalise in double and round once to bfloat16
(cosine similarity, Section 3 and Section 5.1); exact top-1 by dot product,
lowest index on ties, hit when the clamped score >= tau_q (Algorithm 1,
Section 5.1); for hits only, the lookahead check on the matched entry --
identical first-k tokens, or prefix-embedding cosine >= tau_r (Algorithm 1,
Section 4.2 cache structure, Section 5.1); with m lookahead models, all m
checks (Section 4.4); thresholds from benign pairs as capped percentiles of
their cosines (Appendix A.2); the speculative-decoding acceptance length of
the draft tokens (Section 4.3); stage 1 through a random-hyperplane LSH index
with exact re-ranking of the candidates (Eq. (1)).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(_HERE, "lacache_oracle.c")
# LACACHE_ORACLE_LIB points the wrapper at another build of the same source (the mutation tests use it)
LIB = os.environ.get("LACACHE_ORACLE_LIB", os.path.join(_HERE, "liblacache_oracle.so"))

MISS, REJECT, HIT, HIT_EXACT = 0, 1, 2, 3
F32, BF16 = 0, 1


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (plain -O2, OpenMP; no host-specific ISA)."""
    if force or not os.path.exists(LIB):
        tmp = LIB + ".tmp"
        subprocess.run(["gcc", "-O2", "-fopenmp", "-std=c11", "-Wall", "-shared", "-fPIC",
                        "-o", tmp, SRC, "-lm"], check=True)
        os.replace(tmp, LIB)
    return LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build(force=False)
        L = ctypes.CDLL(LIB)
        P = ctypes.c_void_p
        i32, i64, f32 = ctypes.c_int32, ctypes.c_int64, ctypes.c_float
        L.lco_bf16_rne_array.argtypes = [P, i64, P]
        L.lco_quantise.argtypes = [P, i32, i64, i32, P]
        L.lco_dot.argtypes = [P, P, i32]
        L.lco_dot.restype = ctypes.c_double
        L.lco_lookup.argtypes = [P, P, P, i64, i32, i32, P, P, P, i32, f32, f32, i32, P, P, P, P, P, P]
        L.lco_decide.argtypes = [P, P, P, i64, i32, i32, P, P, P, i32, f32, f32, i32, P, P, P, P, P]
        L.lco_first_identical.argtypes = [P, i64, i32, i64]
        f64 = ctypes.c_double
        L.lco_threshold_rule.argtypes = [P, i64, f64, f64, P, P]
        L.lco_calibrate.argtypes = [P, P, i64, i32, f64, f64, P, P, P]
        L.lco_accept_length.argtypes = [P, i32, i32, P, P, i32, i32, P, P]
        L.lco_simhash.argtypes = [P, i64, i32, P, i32, P, P]
        L.lco_lookup_lsh.argtypes = [P, P, P, P, i64, i32, i32, i32, P, P, P, P, i32, i32, f32, f32, i32, P, P, P,
                                     P, P]
        L.lco_first_identical.restype = i64
        L.lco_num_threads.restype = ctypes.c_int
        L.lco_set_num_threads.argtypes = [ctypes.c_int]
        L.lco_lookup_ensemble.argtypes = [P, i64, i32, P, i32, f32, i32, P, P, P, P, P, i32, P, i32, P, P, P, P]
        _lib = L
    return _lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def bf16_rne(x) -> np.ndarray:
    """Round doubles to bfloat16 bit patterns (uint16), one rounding, ties to even."""
    x = _c(x, np.float64)
    out = np.empty(x.shape, np.uint16)
    lib().lco_bf16_rne_array(_ptr(x), x.size, _ptr(out))
    return out


def bf16_to_f64(h) -> np.ndarray:
    """bfloat16 bit patterns -> exact doubles."""
    h = np.asarray(h, dtype=np.uint16)
    return (h.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def quantise(x: np.ndarray, dtype: int | None = None) -> np.ndarray:
    """L2-normalise rows in double, round once to bfloat16. ``x`` is float32, or uint16 bf16 bits."""
    if dtype is None:
        dtype = BF16 if x.dtype == np.uint16 else F32
    x = _c(x, np.uint16 if dtype == BF16 else np.float32)
    x2 = x.reshape(-1, x.shape[-1]) if x.ndim > 1 else x.reshape(1, -1)
    out = np.empty(x2.shape, np.uint16)
    lib().lco_quantise(_ptr(x2), dtype, x2.shape[0], x2.shape[1], _ptr(out))
    return out.reshape(x.shape)


def dot(x: np.ndarray, y: np.ndarray) -> float:
    x = _c(x, np.uint16)
    y = _c(y, np.uint16)
    assert x.shape == y.shape and x.ndim == 1
    return lib().lco_dot(_ptr(x), _ptr(y), x.size)


def _check_store(keys, emb, tokens):
    keys = _c(keys, np.uint16)
    emb = _c(emb, np.uint16)
    tokens = _c(tokens, np.int32)
    N, d = keys.shape
    assert emb.shape == (N, d) and tokens.ndim == 2 and tokens.shape[0] == N
    return keys, emb, tokens, N, d, tokens.shape[1]


def lookup(keys_q, emb_q, tokens, q_q, a_q, u, tau_q: float, tau_r: float, k: int) -> dict:
    """Two-stage lookup over quantised arrays. Returns idx, score, resp_score, decision, s_best, margin."""
    keys_q, emb_q, tokens, N, d, k_cap = _check_store(keys_q, emb_q, tokens)
    q_q = _c(q_q, np.uint16).reshape(-1, d)
    a_q = _c(a_q, np.uint16).reshape(-1, d)
    B = q_q.shape[0]
    u = _c(u, np.int32).reshape(B, -1)
    assert a_q.shape[0] == B and 1 <= k <= k_cap and u.shape[1] == k
    out = dict(idx=np.empty(B, np.int32), score=np.empty(B, np.float32),
               resp_score=np.empty(B, np.float32), decision=np.empty(B, np.int32),
               s_best=np.empty(B, np.float64), margin=np.empty(B, np.float64))
    lib().lco_lookup(_ptr(keys_q), _ptr(emb_q), _ptr(tokens), N, d, k_cap, _ptr(q_q), _ptr(a_q), _ptr(u), B,
                     tau_q, tau_r, k, _ptr(out["idx"]), _ptr(out["score"]), _ptr(out["resp_score"]),
                     _ptr(out["decision"]), _ptr(out["s_best"]), _ptr(out["margin"]))
    return out


def decide(keys_q, emb_q, tokens, q_q, a_q, u, tau_q: float, tau_r: float, k: int, at) -> dict:
    """Post-search steps of the lookup evaluated at entry ``at[b]`` for each query b."""
    keys_q, emb_q, tokens, N, d, k_cap = _check_store(keys_q, emb_q, tokens)
    q_q = _c(q_q, np.uint16).reshape(-1, d)
    a_q = _c(a_q, np.uint16).reshape(-1, d)
    B = q_q.shape[0]
    u = _c(u, np.int32).reshape(B, -1)
    at = _c(at, np.int32).reshape(B)
    assert 1 <= k <= k_cap and u.shape[1] == k
    out = dict(s=np.empty(B, np.float64), score=np.empty(B, np.float32),
               resp_score=np.empty(B, np.float32), decision=np.empty(B, np.int32))
    lib().lco_decide(_ptr(keys_q), _ptr(emb_q), _ptr(tokens), N, d, k_cap, _ptr(q_q), _ptr(a_q), _ptr(u), B,
                     tau_q, tau_r, k, _ptr(at), _ptr(out["s"]), _ptr(out["score"]), _ptr(out["resp_score"]),
                     _ptr(out["decision"]))
    return out


def lookup_ensemble(keys_q, q_q, tau_q: float, embs_q, as_q, tau_r, tokens, u, k: int) -> dict:
    """Two-stage lookup with m lookahead models: embs_q[i] is [N][d_i], as_q[i] is [B][d_i], tau_r[i] a float.

    Returns idx, score, resp_score ([B][m]), decision."""
    keys_q = _c(keys_q, np.uint16)
    N, d = keys_q.shape
    q_q = _c(q_q, np.uint16).reshape(-1, d)
    B = q_q.shape[0]
    m = len(embs_q)
    assert len(as_q) == m and len(tau_r) == m and m >= 1
    embs = [_c(e, np.uint16) for e in embs_q]
    las = [_c(a, np.uint16).reshape(B, -1) for a in as_q]
    dm = np.array([e.shape[1] for e in embs], np.int32)
    for e, a in zip(embs, las):
        assert e.shape[0] == N and a.shape[1] == e.shape[1]
    tokens = _c(tokens, np.int32)
    u = _c(u, np.int32).reshape(B, -1)
    assert u.shape[1] == k and 1 <= k <= tokens.shape[1]
    emb_ptrs = (ctypes.c_void_p * m)(*[e.ctypes.data for e in embs])
    la_ptrs = (ctypes.c_void_p * m)(*[a.ctypes.data for a in las])
    tr = np.ascontiguousarray(tau_r, np.float32)
    out = dict(idx=np.empty(B, np.int32), score=np.empty(B, np.float32), resp_score=np.empty((B, m), np.float32),
               decision=np.empty(B, np.int32))
    lib().lco_lookup_ensemble(_ptr(keys_q), N, d, _ptr(q_q), B, tau_q, m, ctypes.cast(emb_ptrs, ctypes.c_void_p),
                              _ptr(dm), ctypes.cast(la_ptrs, ctypes.c_void_p), _ptr(tr), _ptr(tokens),
                              tokens.shape[1], _ptr(u), k, _ptr(out["idx"]), _ptr(out["score"]),
                              _ptr(out["resp_score"]), _ptr(out["decision"]))
    return out


def threshold_rule(sims, p: float, cap: float):
    """Appendix A.2 rule on given similarities: (P_p with linear interpolation, min(cap, P_p))."""
    x = np.ascontiguousarray(sims, np.float64).ravel()
    assert x.size >= 1 and 0.0 <= p <= 100.0
    P, tau = ctypes.c_double(), ctypes.c_double()
    lib().lco_threshold_rule(_ptr(x), x.size, float(p), float(cap), ctypes.byref(P), ctypes.byref(tau))
    return P.value, tau.value


def calibrate(a_q, b_q, p: float, cap: float) -> dict:
    """Threshold calibration over pairs of quantised vectors a_q[j], b_q[j] ([n][d] bf16 bits).
    Returns sims (float64 [n], clamped cosines), P (the percentile) and tau = min(cap, P)."""
    a_q = _c(a_q, np.uint16)
    b_q = _c(b_q, np.uint16)
    assert a_q.shape == b_q.shape and a_q.ndim == 2 and a_q.shape[0] >= 1
    n, d = a_q.shape
    sims = np.empty(n, np.float64)
    P, tau = ctypes.c_double(), ctypes.c_double()
    lib().lco_calibrate(_ptr(a_q), _ptr(b_q), n, d, float(p), float(cap), _ptr(sims), ctypes.byref(P),
                        ctypes.byref(tau))
    return dict(sims=sims, P=P.value, tau=tau.value)


def accept_length(logits, dtype: int, tokens, p_draft) -> dict:
    """Speculative-decoding acceptance (Section 4.3).  logits: [B][k][V] float32, or bfloat16 bits (uint16)
    with dtype BF16; tokens: [B][k] int32; p_draft: [B][k] float32.  Returns accept_len [B] and p_target
    [B][k] (float64)."""
    logits = np.ascontiguousarray(logits, np.float32 if dtype == F32 else np.uint16)
    B, k, V = logits.shape
    tokens = _c(tokens, np.int32).reshape(B, k)
    p_draft = np.ascontiguousarray(p_draft, np.float32).reshape(B, k)
    out = dict(accept_len=np.empty(B, np.int32), p_target=np.empty((B, k), np.float64))
    lib().lco_accept_length(_ptr(logits), dtype, V, _ptr(tokens), _ptr(p_draft), B, k, _ptr(out["accept_len"]),
                            _ptr(out["p_target"]))
    return out


def simhash(z_q, hyperplanes, bits: int):
    """Random-hyperplane signatures of quantised vectors z_q [n][d] under bf16 hyperplanes [bits][d].
    Returns (sig uint32 [n][bits/32], proj float64 [n][bits])."""
    z_q = _c(z_q, np.uint16)
    n, d = z_q.shape
    r = _c(hyperplanes, np.uint16).reshape(bits, d)
    assert bits % 32 == 0
    sig = np.empty((n, bits // 32), np.uint32)
    proj = np.empty((n, bits), np.float64)
    lib().lco_simhash(_ptr(z_q), n, d, _ptr(r), bits, _ptr(sig), _ptr(proj))
    return sig, proj


def lookup_lsh(keys_q, emb_q, tokens, sig_keys, q_q, sig_q, a_q, u, radius: int, tau_q: float, tau_r: float,
               k: int) -> dict:
    """Two-stage lookup with the LSH index as stage 1 (candidates within `radius` differing bits).
    Returns idx, score, resp_score, decision, n_cand."""
    keys_q, emb_q, tokens, N, d, k_cap = _check_store(keys_q, emb_q, tokens)
    sig_keys = _c(sig_keys, np.uint32)
    words = sig_keys.shape[1]
    q_q = _c(q_q, np.uint16).reshape(-1, d)
    B = q_q.shape[0]
    sig_q = _c(sig_q, np.uint32).reshape(B, words)
    a_q = _c(a_q, np.uint16).reshape(B, d)
    u = _c(u, np.int32).reshape(B, -1)
    out = dict(idx=np.empty(B, np.int32), score=np.empty(B, np.float32), resp_score=np.empty(B, np.float32),
               decision=np.empty(B, np.int32), n_cand=np.empty(B, np.int32))
    lib().lco_lookup_lsh(_ptr(keys_q), _ptr(emb_q), _ptr(tokens), _ptr(sig_keys), N, d, k_cap, words * 32,
                         _ptr(q_q), _ptr(sig_q), _ptr(a_q), _ptr(u), B, int(radius), tau_q, tau_r, k,
                         _ptr(out["idx"]), _ptr(out["score"]), _ptr(out["resp_score"]), _ptr(out["decision"]),
                         _ptr(out["n_cand"]))
    return out


def num_threads() -> int:
    """Threads the oracle's parallel loops use."""
    return int(lib().lco_num_threads())


def set_num_threads(n: int) -> None:
    """Threads the oracle's parallel loops use from now on (n >= 1)."""
    lib().lco_set_num_threads(int(n))


def first_identical(keys_q, i: int) -> int:
    """Lowest index whose quantised key is bitwise identical to key ``i``."""
    keys_q = _c(keys_q, np.uint16)
    N, d = keys_q.shape
    return int(lib().lco_first_identical(_ptr(keys_q), N, d, int(i)))


class OracleCache:
    """The cache as the oracle sees it: quantised rows appended in insertion order."""

    def __init__(self, d: int, k_cap: int, in_dtype: int = BF16):
        self.d, self.k_cap, self.in_dtype = d, k_cap, in_dtype
        self._keys, self._emb, self._tok = [], [], []
        self.keys = np.zeros((0, d), np.uint16)
        self.emb = np.zeros((0, d), np.uint16)
        self.tokens = np.zeros((0, k_cap), np.int32)

    @property
    def size(self) -> int:
        return self.keys.shape[0]

    def insert(self, keys, emb, tokens) -> int:
        """Append entries (Algorithm 1: add the new entry after decoding). Returns the first new index."""
        first = self.size
        kq = quantise(keys, self.in_dtype)
        eq = quantise(emb, self.in_dtype)
        self.keys = np.concatenate([self.keys, kq]) if first else kq
        self.emb = np.concatenate([self.emb, eq]) if first else eq
        t = _c(tokens, np.int32).reshape(-1, self.k_cap)
        self.tokens = np.concatenate([self.tokens, t]) if first else t
        return first

    def lookup(self, queries, lookahead_emb, lookahead_tokens, tau_q, tau_r, k) -> dict:
        qq = quantise(queries, self.in_dtype)
        aq = quantise(lookahead_emb, self.in_dtype)
        out = lookup(self.keys, self.emb, self.tokens, qq, aq, lookahead_tokens, tau_q, tau_r, k)
        out["q_q"], out["a_q"] = qq, aq
        return out
