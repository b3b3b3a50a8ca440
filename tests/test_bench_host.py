"""Host-side logic of bench.py that needs no GPU: the one-GPU refusal and the HBM-traffic arithmetic of
--pmc-summary (counter readings scaled by what the same counter reads for a copy of known size)."""
from __future__ import annotations

import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")


@pytest.mark.parametrize("argv,env", [(["--gpus", "2"], {}), (["--gpus", "8"], {}), ([], {"WORLD_SIZE": "4"})])
def test_more_than_one_gpu_is_refused(argv, env):
    r = subprocess.run([sys.executable, BENCH] + argv, capture_output=True, text=True, timeout=120,
                       env={**os.environ, **env})
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def _counters(path, counter, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for i, (kernel, value) in enumerate(rows):
            w.writerow({"Dispatch_Id": i, "Kernel_Name": kernel, "Counter_Name": counter, "Counter_Value": value})


def test_pmc_summary_scales_by_the_copy(tmp_path):
    root = tmp_path / "pmc"
    copy_mib = 64
    # the copy reads and writes 64 MiB; say FETCH_SIZE counts half of what it reads, WRITE_SIZE all of it
    _counters(str(root / "fetch_copy" / "run_counter_collection.csv"), "FETCH_SIZE",
              [("copy_kernel", copy_mib * 1024 / 2)])
    _counters(str(root / "write_copy" / "run_counter_collection.csv"), "WRITE_SIZE",
              [("copy_kernel", copy_mib * 1024)])
    gemm, stream = "lacache::k_stage1_gemm(...)", "void lacache::k_stage1_stream<1, true, 2>(...)"
    _counters(str(root / "fetch_bench" / "run_counter_collection.csv"), "FETCH_SIZE",
              [(gemm, 3.0e6), (gemm, 3.2e6), (gemm, 9.9e9), (stream, 750_000.0), (stream, 750_001.0),
               (stream, 10.0), ("other", 1.0)])
    _counters(str(root / "write_bench" / "run_counter_collection.csv"), "WRITE_SIZE",
              [(gemm, 4700.0), (gemm, 4700.0), (gemm, 4700.0), (stream, 128.0), (stream, 128.0), (stream, 128.0)])
    # the 4M x 1024 schedule has counter runs of its own (its GEMM launches, and the streaming leg before it)
    _counters(str(root / "fetch_large" / "run_counter_collection.csv"), "FETCH_SIZE",
              [(stream, 1.0), (gemm, 5.7e6), (gemm, 5.8e6), (gemm, 5.9e6), (gemm, 5.6e6), (gemm, 6.0e6)])
    _counters(str(root / "write_large" / "run_counter_collection.csv"), "WRITE_SIZE",
              [(stream, 1.0), (gemm, 480.0), (gemm, 500.0), (gemm, 490.0), (gemm, 510.0), (gemm, 470.0)])
    out = tmp_path / "traffic.json"
    r = subprocess.run([sys.executable, BENCH, "--pmc-summary", str(root), "--traffic", str(out), "--copy-mib",
                        str(copy_mib)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    d = json.load(open(out))
    assert d["fetch_scale"] == pytest.approx(2.0) and d["write_scale"] == pytest.approx(1.0)
    # medians of the dispatches, in bytes: FETCH x 1024 x 2, WRITE x 1024 x 1
    assert d["serve_large"]["fetch_bytes"] == pytest.approx(3.2e6 * 1024 * 2)
    assert d["serve_large"]["write_bytes"] == pytest.approx(4700.0 * 1024)
    assert d["serve_large"]["traffic_bytes"] == pytest.approx(3.2e6 * 2048 + 4700.0 * 1024)
    assert d["serve_small"]["fetch_bytes"] == pytest.approx(750_000.0 * 1024 * 2)
    assert d["serve_small"]["dispatches"] == 3 and d["serve_large"]["dispatches"] == 3
    assert d["large"]["fetch_bytes"] == pytest.approx(5.8e6 * 1024 * 2)
    assert d["large"]["write_bytes"] == pytest.approx(490.0 * 1024)
    assert d["large"]["dispatches"] == 5
    # each entry carries the digest of the kernel sources it was measured on
    assert len(d["serve_large"]["sources_digest"]) == 16
