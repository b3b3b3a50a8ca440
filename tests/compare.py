"""Comparison of a lookup result with the CPU oracle on the same inputs.

Rules (bf16 inputs, float32 accumulation on the GPU vs float64 in the oracle):
  * score      |gpu - oracle| <= 1e-3 for every query;
  * idx        equal to the oracle's argmax, unless the oracle's top-2 margin is
               below 2e-3 -- then the GPU's entry must score within 2e-3 of the
               oracle's maximum (a near tie may legitimately flip);
  * exact ties the GPU's entry must be the lowest index among the entries whose
               stored key is bitwise identical to it (checked separately, so the
               margin exemption never excuses a wrong tie-break);
  * decision   equal to the oracle's decision evaluated at the GPU's entry,
               unless the score is within 2e-3 of tau_q, or stage 2 ran and the
               prefix score is within 2e-3 of tau_r;
  * resp_score within 1e-3 of the oracle's value at the GPU's entry, with NaN
               (stage 2 did not run) in exactly the same places.
"""
from __future__ import annotations

import numpy as np

import oracle

SCORE_TOL = 1e-3
MARGIN = 2e-3


def compare(gpu: dict, orc: dict, keys_q, emb_q, tokens, q_q, a_q, u, tau_q, tau_r, k, rows=None) -> dict:
    """Check GPU outputs against the oracle for the queries `rows` (default all). Returns counters.

    gpu: idx, score, resp_score, decision (numpy, indexed like q_q); orc: the oracle's lookup for the same
    rows (idx, score, decision, s_best, margin).  Raises AssertionError with the offending queries.
    """
    B = q_q.shape[0]
    rows = np.arange(B) if rows is None else np.asarray(rows)
    g = {n: np.asarray(gpu[n])[rows] for n in ("idx", "score", "resp_score", "decision")}
    N = keys_q.shape[0]
    if N == 0:
        assert np.all(g["idx"] == -1), g["idx"]
        assert np.all(np.isnan(g["score"])) and np.all(np.isnan(g["resp_score"]))
        assert np.all(g["decision"] == oracle.MISS)
        return dict(n=len(rows), idx_exact=len(rows), near_tie=0, near_set=0, thr_margin=0)

    at = g["idx"].astype(np.int32)
    assert np.all((at >= 0) & (at < N)), f"index out of range: {at[(at < 0) | (at >= N)]}"
    dec_at = oracle.decide(keys_q, emb_q, tokens, q_q[rows], a_q[rows], np.asarray(u)[rows], tau_q, tau_r, k, at)

    ds = np.abs(g["score"].astype(np.float64) - orc["score"].astype(np.float64))
    bad = np.nonzero(~(ds <= SCORE_TOL))[0]
    assert len(bad) == 0, f"score off by > {SCORE_TOL} at queries {rows[bad][:10]}: {ds[bad][:10]}"

    same = at == orc["idx"]
    near = orc["margin"] < MARGIN
    in_set = dec_at["s"] >= orc["s_best"] - MARGIN
    bad = np.nonzero(~same & ~(near & in_set))[0]
    assert len(bad) == 0, (f"idx differs outside the near-tie exemption at queries {rows[bad][:10]}: gpu "
                           f"{at[bad][:10]} oracle {orc['idx'][bad][:10]} margin {orc['margin'][bad][:10]}")

    ties = np.nonzero(orc["margin"] == 0)[0]
    for t in ties:
        first = oracle.first_identical(keys_q, int(at[t]))
        assert first == at[t], f"query {rows[t]}: exact tie resolved to {at[t]}, lowest identical entry is {first}"
    for t in np.nonzero(~same)[0]:
        first = oracle.first_identical(keys_q, int(at[t]))
        assert first == at[t], f"query {rows[t]}: entry {at[t]} is a later copy of entry {first}"

    ran = ~np.isnan(dec_at["resp_score"])
    thr = (np.abs(g["score"] - np.float32(tau_q)) < MARGIN) | \
          (ran & (np.abs(dec_at["resp_score"] - np.float32(tau_r)) < MARGIN))
    bad = np.nonzero((g["decision"] != dec_at["decision"]) & ~thr)[0]
    assert len(bad) == 0, (f"decision differs at queries {rows[bad][:10]}: gpu {g['decision'][bad][:10]} "
                           f"oracle {dec_at['decision'][bad][:10]}")

    gn = np.isnan(g["resp_score"])
    on = np.isnan(dec_at["resp_score"])
    # a threshold-margin case may legitimately run stage 2 on one side only
    bad = np.nonzero((gn != on) & ~thr)[0]
    assert len(bad) == 0, f"resp_score NaN-ness differs at queries {rows[bad][:10]}"
    both = ~gn & ~on
    dr = np.abs(g["resp_score"][both].astype(np.float64) - dec_at["resp_score"][both])
    assert np.all(dr <= SCORE_TOL), f"resp_score off by {dr.max()}"
    assert np.all(np.abs(g["score"]) <= 1) and np.all(np.abs(g["resp_score"][~gn]) <= 1)
    # near_set: rows whose oracle top-2 margin is below MARGIN (the near-tie set S_b holds more than the top-1, so
    # the idx rule is the set-membership one); near_tie: rows where the GPU's entry differs from the oracle's
    return dict(n=len(rows), idx_exact=int(same.sum()), near_tie=int((~same).sum()), near_set=int(near.sum()),
                thr_margin=int(thr.sum()))


def compare_ensemble(gpu: dict, orc: dict, s1: dict, tau_q, tau_r, rows=None) -> dict:
    """Check an ensemble lookup (resp_score [B][m]) against oracle.lookup_ensemble on the same rows.

    s1 is oracle.lookup on the same keys and queries, used only for its stage-1 s_best and margin.  Same rules
    as compare(): idx equal unless the oracle's top-2 margin is below 2e-3 (such rows are counted and their
    stage 2 is not compared); score within 1e-3; for rows with the oracle's entry, every model's
    resp_score within 1e-3 with NaN in the same places, and the decision equal unless the score is within
    2e-3 of tau_q or some model's prefix score is within 2e-3 of its threshold.
    """
    B = len(orc["idx"])
    rows = np.arange(B) if rows is None else np.asarray(rows)
    g = {n: np.asarray(gpu[n])[rows] for n in ("idx", "score", "resp_score", "decision")}
    tau_r = np.asarray(tau_r, np.float32)
    ds = np.abs(g["score"].astype(np.float64) - orc["score"].astype(np.float64))
    bad = np.nonzero(~(ds <= SCORE_TOL) & ~(np.isnan(g["score"]) & np.isnan(orc["score"])))[0]
    assert len(bad) == 0, f"score off by > {SCORE_TOL} at queries {rows[bad][:10]}: {ds[bad][:10]}"
    same = g["idx"] == orc["idx"]
    bad = np.nonzero(~same & ~(s1["margin"] < MARGIN))[0]
    assert len(bad) == 0, f"idx differs at queries {rows[bad][:10]}: gpu {g['idx'][bad]} oracle {orc['idx'][bad]}"
    gr, orr = g["resp_score"][same], orc["resp_score"][same]
    ran = ~np.isnan(orr).any(axis=1)
    thr = (np.abs(g["score"][same] - np.float32(tau_q)) < MARGIN) | \
          (ran & (np.abs(orr - tau_r[None, :]) < MARGIN).any(axis=1))
    bad = np.nonzero((g["decision"][same] != orc["decision"][same]) & ~thr)[0]
    assert len(bad) == 0, (f"decision differs at queries {rows[same][bad][:10]}: gpu {g['decision'][same][bad][:10]}"
                           f" oracle {orc['decision'][same][bad][:10]}")
    gn, on = np.isnan(gr), np.isnan(orr)
    bad = np.nonzero((gn != on).any(axis=1) & ~thr)[0]
    assert len(bad) == 0, f"resp_score NaN-ness differs at queries {rows[same][bad][:10]}"
    assert np.all(gn.all(axis=1) | ~gn.any(axis=1)), "stage 2 ran for some models only"
    both = ~gn & ~on
    dr = np.abs(gr[both].astype(np.float64) - orr[both])
    assert dr.size == 0 or dr.max() <= SCORE_TOL, f"resp_score off by {dr.max()}"
    assert np.all(np.abs(g["resp_score"][~np.isnan(g["resp_score"])]) <= 1)
    return dict(n=len(rows), idx_exact=int(same.sum()), near_tie=int((~same).sum()), thr_margin=int(thr.sum()),
                decisions=np.bincount(g["decision"], minlength=4).tolist())
