"""Helpers of the GPU tests: move a synthetic workload through the C ABI and the oracle."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import synth


def to_dev(a: np.ndarray, dev="cuda:0") -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).to(dev)


def gpu_cache(lc, sp: synth.Spec, keys, emb, tokens, capacity=None, max_batch=4096, insert_chunk=None):
    c = lc.LaCache(capacity or max(1, keys.shape[0]), sp.d, sp.k_cap, sp.in_dtype, max_batch, 0)
    n = keys.shape[0]
    step = insert_chunk or max(1, n)
    for r0 in range(0, n, step):
        r1 = min(n, r0 + step)
        first = c.insert(to_dev(keys[r0:r1]), to_dev(emb[r0:r1]), to_dev(tokens[r0:r1]))
        assert first == r0
    return c


def gpu_lookup(c, queries, la_emb, la_tok, tau_q, tau_r, k, call_b=None) -> dict:
    B = queries.shape[0]
    step = call_b or B
    outs = []
    q, a, t = to_dev(queries), to_dev(la_emb), to_dev(np.ascontiguousarray(la_tok[:, :k]))
    for b0 in range(0, B, step):
        b1 = min(B, b0 + step)
        outs.append(c.lookup(q[b0:b1], a[b0:b1], t[b0:b1], tau_q, tau_r, k))
    torch.cuda.synchronize()
    cat = [torch.cat([o[i] for o in outs]).cpu().numpy() for i in range(4)]
    return dict(idx=cat[0], score=cat[1], resp_score=cat[2], decision=cat[3])


def oracle_store(sp: synth.Spec, keys, emb, tokens):
    return oracle.quantise(keys, sp.in_dtype), oracle.quantise(emb, sp.in_dtype), np.ascontiguousarray(tokens)


def sample_rows(cls: np.ndarray, target: np.ndarray, n: int, seed: int = 0) -> np.ndarray:
    """A stratified sample of query rows: every class, duplicate-aimed queries included."""
    rng = np.random.default_rng(seed)
    rows = []
    for c in np.unique(cls):
        idx = np.nonzero(cls == c)[0]
        rows.append(rng.choice(idx, size=min(len(idx), max(1, n // 3)), replace=False))
    return np.unique(np.concatenate(rows))


def gpu_ensemble_cache(lc, sp: synth.Spec, d_models, keys, embs, tokens, capacity=None, max_batch=4096,
                       insert_chunk=None):
    c = lc.LaCache(capacity or max(1, keys.shape[0]), sp.d, sp.k_cap, sp.in_dtype, max_batch, 0,
                   d_resp=tuple(d_models))
    n = keys.shape[0]
    step = insert_chunk or max(1, n)
    for r0 in range(0, n, step):
        r1 = min(n, r0 + step)
        first = c.insert_ensemble(to_dev(keys[r0:r1]), [to_dev(e[r0:r1]) for e in embs], to_dev(tokens[r0:r1]))
        assert first == r0
    return c


def gpu_lookup_ensemble(c, queries, las, la_tok, tau_q, tau_r, k, call_b=None) -> dict:
    B = queries.shape[0]
    step = call_b or B
    outs = []
    q, t = to_dev(queries), to_dev(np.ascontiguousarray(la_tok[:, :k]))
    a = [to_dev(x) for x in las]
    for b0 in range(0, B, step):
        b1 = min(B, b0 + step)
        outs.append(c.lookup_ensemble(q[b0:b1], [x[b0:b1] for x in a], t[b0:b1], tau_q, tau_r, k))
    torch.cuda.synchronize()
    cat = [torch.cat([o[i] for o in outs]).cpu().numpy() for i in range(4)]
    return dict(idx=cat[0], score=cat[1], resp_score=cat[2], decision=cat[3])
