"""GPU parity of threshold calibration (Appendix A.2: a threshold is a capped percentile of the cosines of
benign pairs) through the C ABI, against the CPU oracle's calibration on the same seeded pairs."""
from __future__ import annotations

import sys

import numpy as np
import pytest

import oracle
import synth
from tests.compare import SCORE_TOL
from tests.gpu_util import to_dev

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


def _type7(x: np.ndarray, p: float) -> float:
    """The percentile rule of the library applied to its own float32 similarities, in the same double
    arithmetic (h = (n - 1) * p / 100 with p a float32; linear between ranks floor(h) and floor(h) + 1)."""
    s = np.sort(np.asarray(x, np.float32)).astype(np.float64)
    n = s.size
    h = float(n - 1) * (float(np.float32(p)) / 100.0)
    lo = min(int(np.floor(h)), n - 1)
    hi = min(lo + 1, n - 1)
    frac = 0.0 if lo == hi else h - lo
    return float(np.float32(s[lo] + frac * (s[hi] - s[lo])))


def _pairs(rng, n, d, in_dtype, spread=(0.05, 3.0), dup_frac=0.0):
    a = rng.standard_normal((n, d)).astype(np.float32)
    scale = rng.uniform(*spread, (n, 1)).astype(np.float32)
    b = a + scale * rng.standard_normal((n, d)).astype(np.float32)
    if dup_frac:
        k = int(n * dup_frac)
        b[:k] = b[0]
        a[:k] = a[0]            # k identical pairs: k equal similarities
    if in_dtype == synth.BF16:
        return synth.to_bf16_bits(a), synth.to_bf16_bits(b)
    return a, b


def _check(lc, c, a, b, p, cap, which=-1, dim=None):
    sims, tau = c.calibrate(to_dev(a), to_dev(b), p, cap, which)
    sims, tau = sims.cpu().numpy(), tau.cpu().numpy()
    aq, bq = oracle.quantise(a, c.in_dtype), oracle.quantise(b, c.in_dtype)
    o = oracle.calibrate(aq, bq, float(np.float32(p)), float(np.float32(cap)))
    ds = np.abs(sims.astype(np.float64) - o["sims"])
    assert ds.max() <= SCORE_TOL, ds.max()
    # the selection is exact: the percentile of the library's own similarities, bit for bit
    assert tau[0] == _type7(sims, p), (tau[0], _type7(sims, p))
    assert tau[1] == np.float32(min(float(np.float32(cap)), float(tau[0]))) or tau[1] == min(np.float32(cap), tau[0])
    # and within the similarity error of the oracle's percentile (an order statistic moves by at most that)
    assert abs(float(tau[0]) - o["P"]) <= ds.max() + 1e-6, (tau[0], o["P"])
    assert abs(float(tau[1]) - o["tau"]) <= ds.max() + 1e-6
    return sims, tau, o


def _lane_order_sims(aq: np.ndarray, bq: np.ndarray) -> np.ndarray:
    """The float32 dot of two rows of bfloat16 bits in the library's summation order: lane l of a wave takes
    the columns 512 c + 8 l + e (chunk c, then e = 0..7) in sequence, then the 64 lane sums are combined by a
    butterfly (x_l += x_(l xor m) for m = 32, 16, .., 1), lane 0's value clamped to [-1, 1].  Products of two
    bfloat16 values are exact in float32, so the result is fixed bit for bit by the quantised inputs."""
    n, d = aq.shape
    nc = max(1, -(-d // 512))
    def lanes(x):
        f = np.zeros((n, nc * 512), np.float32)
        f[:, :d] = (x.astype(np.uint32) << 16).view(np.float32)
        return f.reshape(n, nc, 64, 8).transpose(0, 2, 1, 3).reshape(n, 64, nc * 8)
    prod = lanes(aq) * lanes(bq)
    acc = np.zeros((n, 64), np.float32)
    for t in range(nc * 8):
        acc = acc + prod[:, :, t]
    lane = np.arange(64)
    for m in (32, 16, 8, 4, 2, 1):
        acc = acc + acc[:, lane ^ m]
    return np.clip(acc[:, 0], np.float32(-1), np.float32(1))


@pytest.mark.parametrize("in_dtype", [synth.F32, synth.BF16])
def test_calibration_sims_bit_exact_in_summation_order(lc, in_dtype):
    """Each pair cosine is the float32 dot of the two vectors quantised exactly as the oracle quantises them
    (norm in double, one rounding to bfloat16), bit for bit once the summation order is fixed: a single
    element rounded the other way changes the sum.  Dimensions for every register layout of the kernel
    (up to 512, 1024 and 2048 columns per row, and beyond)."""
    rng = np.random.default_rng(71 + in_dtype)
    for n, d in [(3000, 1), (3000, 200), (3000, 512), (3000, 513), (2000, 1024), (1000, 1500), (1000, 2048),
                 (500, 2049), (300, 5000)]:
        say(f"[case] calibrate bit-exact n={n} d={d} dtype={in_dtype}")
        c = lc.LaCache(10, d, 4, in_dtype, 16, 0)
        a, b = _pairs(rng, n, d, in_dtype)
        a[:7] = 0                                     # zero vectors score 0
        sims, _ = c.calibrate(to_dev(a), to_dev(b), 50.0, 2.0)
        want = _lane_order_sims(oracle.quantise(a, in_dtype), oracle.quantise(b, in_dtype))
        got = sims.cpu().numpy()
        bad = np.nonzero(got != want)[0]
        assert bad.size == 0, (d, bad[:5], got[bad[:5]], want[bad[:5]])
        c.close()


def test_calibration_pairs_beyond_one_grid(lc):
    """4.5M pairs: more than one launch of the pair-cosine kernel covers (its waves loop), and a selection over
    4.5M similarities; pairs from the first and the last stretch bit for bit in the summation order."""
    rng = np.random.default_rng(81)
    n, d = 4_500_000, 16
    a, b = _pairs(rng, n, d, synth.F32)
    say(f"[case] calibrate n={n} d={d}")
    c = lc.LaCache(10, d, 4, synth.F32, 16, 0)
    sims, _, _ = _check(lc, c, a, b, 5.0, 0.8)
    for sl in (slice(0, 20_000), slice(n - 20_000, n)):
        want = _lane_order_sims(oracle.quantise(a[sl], synth.F32), oracle.quantise(b[sl], synth.F32))
        assert np.array_equal(sims[sl], want)
    c.close()


@pytest.mark.parametrize("in_dtype", [synth.F32, synth.BF16])
def test_calibration_small_cases(lc, in_dtype):
    rng = np.random.default_rng(61 + in_dtype)
    for n, d in [(1, 16), (2, 7), (3, 1), (1000, 384), (4097, 100), (65537, 64)]:
        c = lc.LaCache(10, d, 4, in_dtype, 16, 0)
        a, b = _pairs(rng, n, d, in_dtype)
        for p, cap in [(0.0, 2.0), (5.0, 0.8), (10.0, 0.7), (50.0, 2.0), (99.9, 2.0), (100.0, 0.9)]:
            say(f"[case] calibrate n={n} d={d} dtype={in_dtype} p={p} cap={cap}")
            _check(lc, c, a, b, p, cap)
        c.close()


def test_calibration_ties_negatives_and_zero_vectors(lc):
    rng = np.random.default_rng(63)
    n, d = 5000, 96
    c = lc.LaCache(10, d, 4, synth.F32, 16, 0)
    a, b = _pairs(rng, n, d, synth.F32, spread=(0.5, 20.0), dup_frac=0.4)   # 2000 equal similarities
    b[2000:2100] = -a[2000:2100]                                           # cosine -1
    a[2100:2110] = 0.0                                                     # zero vectors: cosine 0
    for p in (0.0, 1.0, 20.0, 39.99, 40.0, 41.0, 75.0, 100.0):
        sims, tau, _ = _check(lc, c, a, b, p, 2.0)
    assert np.sum(sims == sims[0]) >= 2000 and sims.min() == -1.0
    c.close()


def test_calibration_of_prefix_models(lc):
    """which selects the dimension: -1 the key model, i the i-th prefix model of an ensemble cache."""
    rng = np.random.default_rng(64)
    dims = (384, 1024, 129)
    c = lc.LaCache(10, 768, 4, synth.BF16, 16, 0, d_resp=dims)
    for which, dim in [(-1, 768)] + list(enumerate(dims)):
        a, b = _pairs(rng, 3000, dim, synth.BF16)
        say(f"[case] calibrate which={which} dim={dim}")
        _check(lc, c, a, b, 10.0, 0.7, which)
    import torch
    a, b = _pairs(rng, 10, 384, synth.BF16)
    with pytest.raises(lc.LaCacheError) as ei:
        lc.lacache_calibrate(c, 3, to_dev(a), to_dev(b), 5.0, 0.8)
    assert ei.value.code == lc.EINVAL
    for p, cap in ((-1.0, 0.8), (100.5, 0.8), (float("nan"), 0.8), (5.0, float("inf"))):
        with pytest.raises(lc.LaCacheError):
            lc.lacache_calibrate(c, 0, to_dev(a), to_dev(b), p, cap)
    c.close()


def test_calibration_paper_shaped_full_size(lc):
    """A million benign pairs at d = 1024 (BGE's dimension): query-pair cosines around the paraphrase band
    and the Appendix A.2 rule tau_c = min(0.80, P5); sampled similarities against the oracle, the exact
    selection on all of them, and the percentile against the oracle's over every pair."""
    n, d = 1_000_000, 1024
    c = lc.LaCache(10, d, 4, synth.BF16, 16, 0)
    a, b = synth.calibration_pairs(n, d, 0.80, 0.99, seed=65)
    say("[case] calibrate 1M x 1024 bf16, P5 capped at 0.80")
    sims, tau = c.calibrate(to_dev(a), to_dev(b), 5.0, 0.80)
    sims, tau = sims.cpu().numpy(), tau.cpu().numpy()
    assert tau[0] == _type7(sims, 5.0)
    o = oracle.calibrate(oracle.quantise(a, synth.BF16), oracle.quantise(b, synth.BF16), 5.0, 0.80)
    ds = np.abs(sims.astype(np.float64) - o["sims"])
    assert ds.max() <= SCORE_TOL
    assert abs(float(tau[0]) - o["P"]) <= ds.max() + 1e-6
    assert tau[1] == np.float32(0.80) or tau[1] == tau[0]
    say(f"[ok] P5 = {tau[0]:.6f} (oracle {o['P']:.6f}), tau = {tau[1]:.4f}, max |sim diff| {ds.max():.2e}")
    c.close()
