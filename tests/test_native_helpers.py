"""Host checks of device helpers that are compiled for the host as well (no GPU needed)."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.fixture(scope="module")
def quotient_checker(tmp_path_factory):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    exe = str(tmp_path_factory.mktemp("native") / "quotient_rounding")
    subprocess.run([HIPCC, "-O2", "-std=c++17", "--offload-arch=gfx950",
                    "-I", os.path.join(ROOT, "paper_2608_01718_amd", "csrc"),
                    os.path.join(ROOT, "tests", "native", "quotient_rounding.cpp"), "-o", exe],
                   check=True, capture_output=True)
    return exe


def test_fast_quotient_rounding_is_bit_exact(quotient_checker):
    """bf16 rounding of v * (1/n) with the midpoint fallback equals the rounding of the divided quotient,
    on 2 million random cases, quotients placed on bfloat16 rounding midpoints and 1 to 40 ulps to either side
    of them (40 million cases), powers of two and normalisation-shaped ratios."""
    r = subprocess.run([quotient_checker, "2000000"], capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.startswith("ok ")


@pytest.fixture(scope="module")
def replay_pick_checker(tmp_path_factory):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    exe = str(tmp_path_factory.mktemp("native") / "replay_pick")
    subprocess.run([HIPCC, "-O2", "-std=c++17", "--offload-arch=gfx950",
                    "-I", os.path.join(ROOT, "paper_2608_01718_amd", "csrc"),
                    os.path.join(ROOT, "tests", "native", "replay_pick.cpp"), "-o", exe],
                   check=True, capture_output=True)
    return exe


def test_replay_row_selection(replay_pick_checker):
    """The rule that ends a large-batch group replay picks the lowest row at the stage-1 score, and when no
    replayed score matches it still names a valid row (the lowest at the replay's own maximum) and reports the
    fallback; 200,000 random groups of 1 to 16 rows with many exact ties, merged across lanes in every order."""
    r = subprocess.run([replay_pick_checker], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.startswith("ok ")
