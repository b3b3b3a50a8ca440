"""The pins are strong enough: each plausible mistake planted in a copy of the oracle's C source (a dropped
term, a wrong sign, a flipped comparison, a transposed operand, a wrong rounding rule...) makes
test_oracle_pins.py fail, while the unmodified source passes the same pipeline."""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "lacache_oracle.c")

MUTANTS = {
    "ties go to the highest index": ("return s > best;", "return s >= best;"),
    "dot product drops its last term": ("for (int32_t j = 0; j < d; ++j)\n        s += widen_bf16",
                                        "for (int32_t j = 0; j < d - 1; ++j)\n        s += widen_bf16"),
    "dot product subtracts": ("s += widen_bf16(x[j]) * widen_bf16(y[j]);", "s -= widen_bf16(x[j]) * widen_bf16(y[j]);"),
    "stage 2 reads the key instead of the prefix embedding": ("lco_dot(a, emb + i * (int64_t)d, d)",
                                                              "lco_dot(a, keys + i * (int64_t)d, d)"),
    "stage-1 threshold is strict": ("if (!(score >= tau_q))", "if (!(score > tau_q))"),
    "stage-2 threshold is strict": ("return (r >= tau_r) ? LCO_HIT : LCO_REJECT;",
                                    "return (r > tau_r) ? LCO_HIT : LCO_REJECT;"),
    "rounding ties go up": ("double r = nearbyint(ldexp(v, 7 - lead));", "double r = floor(ldexp(v, 7 - lead) + 0.5);"),
    "norm without square root": ("double n = sqrt(ss);", "double n = ss;"),
    "token compare skips the last token": ("for (int32_t j = 0; j < k; ++j)\n        if (u[j]",
                                           "for (int32_t j = 0; j < k - 1; ++j)\n        if (u[j]"),
    "no clamp at 1": ("    if (f > 1.0f)\n        f = 1.0f;\n", ""),
    "identical tokens also need the embedding": ("    if (tok_eq)\n        return LCO_HIT_EXACT;",
                                                 "    if (tok_eq && r >= tau_r)\n        return LCO_HIT_EXACT;"),
    "second-best never updated": ("} else if (s > second) {", "} else if (s > best) {"),
    "subnormal grid not clamped": ("if (lead < -126)\n        lead = -126;", ""),
    "ensemble checks only the first model": ("if (!(r >= tau_r[i]))", "if (i == 0 && !(r >= tau_r[i]))"),
    "ensemble applies the first threshold to every model": ("if (!(r >= tau_r[i]))", "if (!(r >= tau_r[0]))"),
    "ensemble needs the embeddings even for identical tokens": (
        "decision[b] = tok_eq ? LCO_HIT_EXACT : (all_pass ? LCO_HIT : LCO_REJECT);",
        "decision[b] = all_pass ? (tok_eq ? LCO_HIT_EXACT : LCO_HIT) : LCO_REJECT;"),
    "percentile position uses n instead of n - 1": ("double h = (double)(n - 1) * (p / 100.0);",
                                                    "double h = (double)n * (p / 100.0);"),
    "percentile takes the upper rank without interpolating": (
        "P = x[lo] + (h - (double)lo) * (x[lo + 1] - x[lo]);", "P = x[lo + 1];"),
    "cap applied as a floor": ("*tau_out = fmin(cap, P);", "*tau_out = fmax(cap, P);"),
    "similarities sorted descending": ("return (a > b) - (a < b);", "return (a < b) - (a > b);"),
    "draft accepted only when P_f > P_g": (
        "p_target[(int64_t)b * k + len] >= (double)p_draft", "p_target[(int64_t)b * k + len] > (double)p_draft"),
    "acceptance counts every accepted token, not the leading run": (
        "        while (len < k && p_target[(int64_t)b * k + len] >= (double)p_draft[(int64_t)b * k + len])\n"
        "            ++len;",
        "        for (int32_t j = 0; j < k; ++j)\n"
        "            len += p_target[(int64_t)b * k + j] >= (double)p_draft[(int64_t)b * k + j];"),
    "softmax without the max shift": ("s += exp(read_in(logits, dtype, row, V, v) - m);",
                                      "s += exp(read_in(logits, dtype, row, V, v));"),
    "hyperplane bit set only on a strictly positive projection": ("if (p >= 0.0)\n                sig[j * words",
                                                                   "if (p > 0.0)\n                sig[j * words"),
    "candidates strictly inside the radius": ("words) > radius)", "words) >= radius)"),
    "Hamming distance from OR instead of XOR": ("__builtin_popcount(a[w] ^ b[w])", "__builtin_popcount(a[w] | b[w])"),
    "an exact-tie copy names itself": ("            return j;\n    return i;", "            return i;\n    return i;"),
    "the copy search compares one element too few": (
        "memcmp(keys + j * (int64_t)d, ki, (size_t)d * sizeof(uint16_t))",
        "memcmp(keys + j * (int64_t)d, ki, (size_t)(d - 1) * sizeof(uint16_t))"),
    "the copy search starts after the first row": ("for (int64_t j = 0; j < i; ++j)\n        if (memcmp",
                                                   "for (int64_t j = 1; j < i; ++j)\n        if (memcmp"),
    "probability read at the next vocabulary entry": ("exp(read_in(logits, dtype, row, V, t) - m) / s",
                                                      "exp(read_in(logits, dtype, row, V, (t + 1) % V) - m) / s"),
}


WORKERS = max(1, min(8, os.cpu_count() or 1))


def _run_pins(tmp_path, source: str, tag: str, threads: int) -> int:
    c = tmp_path / f"{tag}.c"
    so = tmp_path / f"{tag}.so"
    c.write_text(source)
    subprocess.run(["gcc", "-O2", "-fopenmp", "-std=c11", "-shared", "-fPIC", "-o", str(so), str(c), "-lm"],
                   check=True)
    env = dict(os.environ, LACACHE_ORACLE_LIB=str(so), OMP_NUM_THREADS=str(threads))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py")], cwd=ROOT, env=env,
                       capture_output=True, text=True)
    return r.returncode


@pytest.fixture(scope="module")
def pin_runs(tmp_path_factory):
    """Exit status of the pin suite on the unmodified source and on every mutant, run side by side (one
    process per source, the host's cores shared among them)."""
    src = open(SRC).read()
    jobs = {"": src}
    for i, (name, (old, new)) in enumerate(sorted(MUTANTS.items())):
        if src.count(old) == 1:
            jobs[name] = src.replace(old, new)
    threads = max(1, (os.cpu_count() or 1) // WORKERS)
    base = tmp_path_factory.mktemp("mutants")
    dirs = {name: base / f"m{i}" for i, name in enumerate(jobs)}
    for p in dirs.values():
        p.mkdir()

    def run(name):
        return name, _run_pins(dirs[name], jobs[name], "oracle", threads)

    with ThreadPoolExecutor(WORKERS) as pool:
        return dict(pool.map(run, jobs))


def test_unmodified_source_passes_the_pins(pin_runs):
    assert pin_runs[""] == 0


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(pin_runs, name):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor not found (or ambiguous): {name}"
    # pytest's status 1: the suite ran and a pin failed (not a crash, a usage error or an interruption)
    assert pin_runs[name] == 1, f"pins did not catch: {name} (status {pin_runs[name]})"
