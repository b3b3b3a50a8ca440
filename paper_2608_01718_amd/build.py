"""Build liblacache.so (the C-ABI library) for gfx950 with hipcc, in-tree.

    python paper_2608_01718_amd/build.py
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "liblacache.so")
BUILD_DIR = os.path.join(ROOT, "_build")
SOURCES = ["lacache.cpp", "k_store.hip", "k_stage1_stream.hip", "k_stage1_gemm.hip", "k_verify.hip",
           "k_calibrate.hip", "k_accept.hip", "k_lsh.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
    "-I", os.path.join(ROOT, "include"),
    # packed fp32 VALU ops are kept out of every kernel
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *FLAGS, "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the packed-fp32 target feature and says so; that is harmless
    noise = "is not a recognized feature for this target"
    err = "\n".join(line for line in r.stderr.splitlines() if noise not in line)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{err}")
    if err.strip():
        print(err, file=sys.stderr)
    return obj


PROBE_SRC = "roofline_probe.hip"
PROBE = os.path.join(HERE, "roofline_probe")


def _build_probe() -> str:
    """The attainable-ceiling probe bench.py reports beside the datasheet peaks (a separate executable)."""
    obj = _compile(PROBE_SRC)
    tmp = PROBE + ".tmp"
    r = subprocess.run([HIPCC, f"--offload-arch={ARCH}", "-o", tmp, obj], capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link of {PROBE_SRC} failed:\n{r.stderr}")
    os.replace(tmp, PROBE)
    return PROBE


def build() -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    with ThreadPoolExecutor(min(8, len(SOURCES) + 1)) as ex:
        probe = ex.submit(_build_probe)
        objs = list(ex.map(_compile, SOURCES))
        probe.result()
    tmp = OUT + ".tmp"
    r = subprocess.run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs],
                       capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    print(build())
