"""The allocation-free calibration entry point (lacache_calibrate_noalloc, scratch in a static device array)
against the handle-based lacache_calibrate on the same pairs, through the C ABI: two calls in a row, the second
with fewer pairs (the shared scratch keeps the first call's contents, so it must be cleared by the call)."""
from __future__ import annotations

import ctypes
import sys

import numpy as np
import pytest

import synth
from tests.gpu_util import to_dev

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("dtype,d", [(synth.BF16, 1024), (synth.F32, 384)])
def test_noalloc_calibration_matches_handle_calibration(dtype, d):
    import torch
    assert torch.cuda.is_available()
    import paper_2608_01718_amd as lc
    lib = lc.raw_library()
    rng = np.random.default_rng(55 + d)
    c = lc.LaCache(16, d, 4, dtype, 16, 0)
    stream = torch.cuda.current_stream(0).cuda_stream
    for n, p, cap in ((70_001, 5.0, 0.80), (5_003, 10.0, 0.20)):
        say(f"[case] noalloc calibration dtype={dtype} d={d} n={n} p={p} cap={cap}")
        a = rng.standard_normal((n, d)).astype(np.float32)
        b = a + rng.uniform(0.05, 3.0, (n, 1)).astype(np.float32) * rng.standard_normal((n, d)).astype(np.float32)
        if dtype == synth.BF16:
            a, b = synth.to_bf16_bits(a), synth.to_bf16_bits(b)
        da, db = to_dev(a), to_dev(b)
        want_sims, want_tau = c.calibrate(da, db, p, cap, -1)
        sims = torch.full((n,), float("nan"), dtype=torch.float32, device="cuda:0")
        tau = torch.full((2,), float("nan"), dtype=torch.float32, device="cuda:0")
        rc = lib.lacache_calibrate_noalloc(ctypes.c_void_p(da.data_ptr()), ctypes.c_void_p(db.data_ptr()), dtype, d,
                                           n, ctypes.c_float(p), ctypes.c_float(cap),
                                           ctypes.c_void_p(sims.data_ptr()), ctypes.c_void_p(tau.data_ptr()),
                                           ctypes.c_void_p(stream))
        assert rc == lc.OK, lc.lacache_strerror(rc)
        torch.cuda.synchronize()
        # the same kernels on the same inputs: bit-identical similarities and thresholds
        np.testing.assert_array_equal(sims.cpu().numpy().view(np.uint32), want_sims.cpu().numpy().view(np.uint32))
        np.testing.assert_array_equal(tau.cpu().numpy().view(np.uint32), want_tau.cpu().numpy().view(np.uint32))
        say(f"[ok] n={n}: tau {tau.cpu().numpy().tolist()}")
    # argument checks run before any launch
    assert lib.lacache_calibrate_noalloc(None, None, dtype, d, 10, ctypes.c_float(5.0), ctypes.c_float(0.8),
                                         None, None, None) == lc.EINVAL
    c.close()
