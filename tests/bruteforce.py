"""Brute-force reference for tiny caches, written independently of the C oracle.

It materialises the whole float64 score matrix of the quantised vectors with
numpy.einsum (no BLAS: every entry is summed by the same loop, so bitwise
identical rows give bitwise identical scores) and takes numpy.argmax, which
returns the first maximum -- the lowest index on ties.
"""
import numpy as np

MISS, REJECT, HIT, HIT_EXACT = 0, 1, 2, 3


def widen(h):
    return (np.asarray(h, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def scores(q_q, keys_q):
    return np.einsum("bd,nd->bn", widen(q_q), widen(keys_q), optimize=False)


def lookup(keys_q, emb_q, tokens, q_q, a_q, u, tau_q, tau_r, k):
    B = q_q.shape[0]
    N = keys_q.shape[0]
    if N == 0:
        nan = np.full(B, np.nan, np.float32)
        return dict(idx=np.full(B, -1, np.int32), score=nan, resp_score=nan.copy(),
                    decision=np.zeros(B, np.int32))
    S = scores(q_q, keys_q)
    idx = np.argmax(S, axis=1)
    score = np.clip(S[np.arange(B), idx].astype(np.float32), np.float32(-1), np.float32(1))
    hit = score >= np.float32(tau_q)
    r = np.einsum("bd,bd->b", widen(a_q), widen(emb_q[idx]), optimize=False)
    r = np.clip(r.astype(np.float32), np.float32(-1), np.float32(1))
    tok_eq = np.all(np.asarray(u)[:, :k] == tokens[idx, :k], axis=1)
    dec = np.where(tok_eq, HIT_EXACT, np.where(r >= np.float32(tau_r), HIT, REJECT))
    dec = np.where(hit, dec, MISS).astype(np.int32)
    resp = np.where(hit, r, np.float32(np.nan)).astype(np.float32)
    return dict(idx=idx.astype(np.int32), score=score, resp_score=resp, decision=dec, S=S)
