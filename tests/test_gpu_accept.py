"""GPU parity of the speculative-decoding acceptance step (Section 4.3: draft token t_j is accepted while
P_f(t_j) >= P_g(t_j), from the first token on) through the C ABI, against the CPU oracle."""
from __future__ import annotations

import sys

import numpy as np
import pytest

import oracle
import synth
from tests.gpu_util import to_dev

pytestmark = pytest.mark.gpu

P_RTOL = 1e-4  # float32 softmax (max-shifted, tree-summed) against the double oracle


@pytest.fixture(scope="module")
def lc():
    import torch
    assert torch.cuda.is_available()
    import paper_2608_01718_amd as m
    return m


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _valid_lengths(pt, pd):
    """Accepted lengths consistent with the oracle's probabilities: a position whose P_f lies within P_RTOL
    of P_g may go either way; every other position must be decided as the oracle decides it."""
    k = pt.shape[0]
    acc = pt >= pd
    amb = np.abs(pt - pd) <= P_RTOL * np.maximum(pt, pd) + 1e-12
    ok = set()
    for L in range(k + 1):
        lead = np.all(acc[:L] | amb[:L])
        stop = L == k or (not acc[L]) or amb[L]
        if lead and stop:
            ok.add(L)
    return ok


def _run(lc, logits, dtype, tok, pd, rows=None):
    import torch
    acc, pt = lc.lacache_accept_length(to_dev(logits), to_dev(tok), to_dev(pd))
    torch.cuda.synchronize()
    acc, pt = acc.cpu().numpy(), pt.cpu().numpy()
    B = tok.shape[0]
    rows = np.arange(B) if rows is None else rows
    o = oracle.accept_length(logits[rows], dtype, tok[rows], pd[rows])
    err = np.abs(pt[rows].astype(np.float64) - o["p_target"])
    assert np.all(err <= P_RTOL * o["p_target"] + 1e-12), err.max()
    pd64 = pd[rows].astype(np.float64)
    exact = 0
    for i, b in enumerate(rows):
        ok = _valid_lengths(o["p_target"][i], pd64[i])
        assert acc[b] in ok, (b, acc[b], ok)
        exact += acc[b] == o["accept_len"][i]
    return acc, pt, o, exact


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
def test_accept_small_shapes(lc, dtype):
    for B, k, V in [(1, 1, 1), (3, 5, 7), (17, 20, 1000), (5, 70, 3001), (4, 20, 32000), (2, 3, 128256)]:
        say(f"[case] accept B={B} k={k} V={V} dtype={dtype}")
        lg, tok, pd = synth.draft_verification(B, k, V, seed=B * 1000 + V, in_dtype=dtype)
        acc, _, o, exact = _run(lc, lg, dtype, tok, pd)
        assert exact == B


def test_accept_rows_beyond_one_grid(lc):
    """4.3M queries of one draft token over a 3-token vocabulary: more rows than one launch of either kernel
    covers (their workgroups and waves loop); a sample of rows from the whole range, including the last."""
    B, k, V = 4_300_000, 1, 3
    lg, tok, pd = synth.draft_verification(B, k, V, seed=91, in_dtype=synth.F32)
    rng = np.random.default_rng(92)
    rows = np.unique(np.concatenate([rng.integers(0, B, 3000), np.arange(B - 3000, B)]))
    say(f"[case] accept B={B} k={k} V={V}")
    _, _, _, exact = _run(lc, lg, synth.F32, tok, pd, rows=rows)
    assert exact >= rows.size - 10


def test_accept_edges(lc):
    import torch
    B, k, V = 6, 9, 515                                        # odd V: bf16 rows are not 16-byte aligned
    lg, tok, pd = synth.draft_verification(B, k, V, seed=7, in_dtype=synth.F32)
    lg[0, :, 100:400] = -np.inf                                # masked vocabulary entries
    tok[1, 2] = -1                                             # out-of-range tokens: probability 0
    tok[1, 3] = V
    pd[2, :] = 0.0                                             # every token accepted
    pd[3, 0] = 2.0                                             # first token rejected
    lg[4, :, :] = 0.0
    tok[4, :] = 3
    pd[4, :] = np.float32(1.0 / V) * np.float32(0.5)           # uniform logits, P_f = 1/V > P_g
    for dtype, x in ((synth.F32, lg), (synth.BF16, synth.to_bf16_bits(lg))):
        say(f"[case] accept edges dtype={dtype}")
        acc, pt, o, _ = _run(lc, x, dtype, tok, pd)
        assert pt[1, 2] == 0.0 and pt[1, 3] == 0.0
        assert acc[2] == k and acc[3] == 0 and acc[4] == k
        assert abs(pt[4, 0] - 1.0 / V) <= 1e-6 / V
    with pytest.raises(lc.LaCacheError):
        lc.lacache_accept_length(to_dev(lg[:, :, :0].copy()), to_dev(tok), to_dev(pd))       # V = 0
    a0, p0 = lc.lacache_accept_length(torch.zeros((0, 3, 10), device="cuda:0"),
                                      torch.zeros((0, 3), dtype=torch.int32, device="cuda:0"),
                                      torch.zeros((0, 3), device="cuda:0"))
    assert a0.numel() == 0 and p0.numel() == 0


def test_accept_full_size(lc):
    """256 queries x 20 draft tokens over a 128,256-token vocabulary in bf16 (the measured workload), every
    row against the oracle."""
    B, k, V = 256, 20, 128256
    lg, tok, pd = synth.draft_verification(B, k, V, seed=11)
    say(f"[case] accept full size B={B} k={k} V={V}")
    acc, pt, o, exact = _run(lc, lg, synth.BF16, tok, pd)
    say(f"[ok] exact lengths {exact}/{B}, mean accepted {acc.mean():.2f} of {k}")
    assert exact >= B - 2
