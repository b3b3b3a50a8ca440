"""Throughput of the two-stage LaCache lookup on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload serve_large|serve_small]

A step is one lookup call through the C ABI -- query normalisation, stage 1
(top-1 over all cached keys) and stage 2 (gather and verify of the hits) -- on
a batch of synthetic queries against a cache of 1,000,000 entries, d = 768,
bfloat16 inputs, k = 16, whose inputs already sit in device memory.

The headline workload (`value`) is serve_large: 4096 queries per call (the
matrix-core-bound regime); serve_small (16 queries per call, the HBM-bound
regime) is measured in the same run and reported under "secondary", and the
same keys with the four-model lookahead ensemble (Section 4.4) under
"ensemble", threshold calibration over a million benign pairs
(Appendix A.2) under "calibration", and the speculative-decoding acceptance
of 256 x 20 draft tokens (Section 4.3) under "accept", and the serve_small
lookup with stage 1 through the LSH index (Eq. (1)) under "lsh".  For
each, "roofline" rates the stage-1 kernel, timed over the timed steps with HIP
events that the library attaches to the kernel's own dispatch on the launch
stream, against the MI355X peak (bf16 dense MFMA 2.5 PFLOP/s, HBM 8 TB/s).
"cpu_baseline" times the CPU oracle on a bounded sample of the same workload
on the host cores.  "attainable" rates the same kernels against what this GPU
sustains, measured at start-up by the roofline_probe executable built beside
the library: bf16 MFMA throughput on random operands (the better of the
16x16x32 and 32x32x16 forms) and a streaming read.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="serve_large", choices=["serve_large", "serve_small"])
    ap.add_argument("--no-secondary", action="store_true", help="measure only the headline workload")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU-oracle baseline")
    ap.add_argument("--no-ensemble", action="store_true", help="skip the lookahead-ensemble measurement")
    ap.add_argument("--no-calibration", action="store_true", help="skip the threshold-calibration measurement")
    ap.add_argument("--no-accept", action="store_true", help="skip the speculative-decoding acceptance measurement")
    ap.add_argument("--no-lsh", action="store_true", help="skip the LSH-indexed lookup measurement")
    ap.add_argument("--no-resident", action="store_true",
                    help="skip the cache-resident workloads (tiny, mid, mid_paper)")
    ap.add_argument("--no-large", action="store_true",
                    help="skip the 4M x 1024 clustered workload with interleaved inserts")
    ap.add_argument("--sweep", action="store_true",
                    help="instead of the bench line, sweep the batch size on the 1M x 768 cache (JSON per size)")
    ap.add_argument("--no-probe", action="store_true",
                    help="skip the attainable-ceiling probe (sustained MFMA rate on random bf16, HBM streaming read)")
    ap.add_argument("--traffic", default=os.path.join(ROOT, "profiles", "traffic.json"),
                    help="per-launch HBM traffic measured with rocprofv3 counters (JSON), if present")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="run one plain device copy of this many MiB (a known-size reference for the HBM "
                         "counters) and exit")
    ap.add_argument("--pmc-summary", default=None,
                    help="directory holding rocprofv3 --pmc runs fetch_bench/, write_bench/, fetch_large/, "
                         "write_large/, fetch_copy/, write_copy/: write the per-launch traffic of the stage-1 "
                         "kernels to --traffic and exit")
    ap.add_argument("--copy-mib", type=int, default=1024, help="size of the copy used by --pmc-summary")
    return ap.parse_args()


STAGE1_KERNELS = {"serve_large": "k_stage1_gemm(", "serve_small": "k_stage1_stream<1, true, 2>",
                  "large": "k_stage1_gemm("}
STAGE1_SOURCES = {"serve_large": ["k_stage1_gemm.hip", "common.hpp"],
                  "serve_small": ["k_stage1_stream.hip", "common.hpp"],
                  "large": ["k_stage1_gemm.hip", "common.hpp"]}
# the counter runs each workload's figures come from: serve_large and serve_small share one bench run,
# the 4M x 1024 schedule has a run of its own (it launches the same GEMM kernel)
PMC_RUNS = {"serve_large": "bench", "serve_small": "bench", "large": "large"}


def sources_digest(name):
    """Digest of the sources of a workload's stage-1 kernel: counters are valid only for that code.  Comments
    and runs of white space are left out, so editing a comment keeps the counters; any change to the code
    voids them."""
    import hashlib
    import re
    h = hashlib.sha256()
    for f in STAGE1_SOURCES[name]:
        text = open(os.path.join(ROOT, "paper_2608_01718_amd", "csrc", f)).read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def calibrate_copy(mib):
    """One plain elementwise pass over a known number of bytes (reads mib MiB, writes mib MiB)."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.int32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    torch.neg(src, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": n * 4}), flush=True)


def pmc_summary(root, out_path, copy_mib):
    """Per-launch HBM traffic of the stage-1 kernels from FETCH_SIZE / WRITE_SIZE (KiB per dispatch), each
    scaled by what the same counter reads for a plain copy of known size."""
    import csv
    import glob

    def per_kernel(sub, counter):
        vals = {}
        for f in glob.glob(os.path.join(root, sub, "**", "*counter_collection.csv"), recursive=True):
            for r in csv.DictReader(open(f)):
                if r["Counter_Name"] == counter:
                    vals.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
        return vals

    copy_bytes = copy_mib * (1 << 20)
    f_copy = max((v for k, vs in per_kernel("fetch_copy", "FETCH_SIZE").items() for v in vs), default=None)
    w_copy = max((v for k, vs in per_kernel("write_copy", "WRITE_SIZE").items() for v in vs), default=None)
    out = {"copy_bytes": copy_bytes, "copy_fetch_kib": f_copy, "copy_write_kib": w_copy,
           "fetch_scale": copy_bytes / (f_copy * 1024), "write_scale": copy_bytes / (w_copy * 1024)}
    for name, kern in STAGE1_KERNELS.items():
        run = PMC_RUNS[name]
        fk, wk = per_kernel("fetch_" + run, "FETCH_SIZE"), per_kernel("write_" + run, "WRITE_SIZE")
        fv = [v for k, vs in fk.items() if kern in k for v in vs]
        wv = [v for k, vs in wk.items() if kern in k for v in vs]
        if not fv or not wv:
            continue
        fetch = sorted(fv)[len(fv) // 2] * 1024 * out["fetch_scale"]
        write = sorted(wv)[len(wv) // 2] * 1024 * out["write_scale"]
        out[name] = {"kernel": kern, "sources_digest": sources_digest(name), "fetch_bytes": fetch,
                     "write_bytes": write, "traffic_bytes": fetch + write, "dispatches": len(fv)}
    json.dump(out, open(out_path, "w"), indent=1)
    print(json.dumps(out), flush=True)


def attainable_ceilings():
    """Run the roofline probe executable built beside the library (a child process) and return its JSON."""
    import subprocess
    exe = os.path.join(ROOT, "paper_2608_01718_amd", "roofline_probe")
    if not os.path.exists(exe):
        log("[bench] roofline_probe not built; attainable ceilings not reported")
        return None
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    if r.returncode != 0:
        log(f"[bench] roofline_probe failed ({r.returncode}): {r.stderr.strip()}")
        return None
    return json.loads(r.stdout.strip().splitlines()[-1])


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def sclk_under_load(torch, step, seconds=1.5):
    """The GPU's shader clock (MHz) while `step` runs back to back: rocm-smi is sampled once, from a separate
    thread, half a second into ~`seconds` of continuous calls.  None when the tool or its reading is missing,
    and under a profiler: its preloaded library would start up, and initialise the GPU, in the sampling
    process too."""
    import re
    import shutil
    import subprocess
    import threading
    if os.environ.get("ROCPROFILER_LIBRARY_CTOR") or "rocprofiler" in os.environ.get("LD_PRELOAD", ""):
        return None
    smi = shutil.which("rocm-smi")
    if smi is None:
        return None
    # the tool is a Python script: run it with this interpreter rather than through its `env` line
    smi = os.path.realpath(smi)
    cmd = [sys.executable, smi] if smi.endswith(".py") else [smi]
    got = {}

    def sample():
        time.sleep(0.5)
        try:
            r = subprocess.run(cmd + ["--showclocks", "--json"], capture_output=True, text=True, timeout=20)
            m = re.search(r"sclk clock speed:\"\s*:\s*\"\((\d+)Mhz\)", r.stdout)
            got["mhz"] = int(m.group(1)) if m else None
        except (OSError, subprocess.SubprocessError):
            got["mhz"] = None

    th = threading.Thread(target=sample)
    t0 = time.time()
    th.start()
    i = 0
    while th.is_alive() or time.time() - t0 < seconds:
        step(i)
        i += 1
        if i % 16 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    th.join()
    return got.get("mhz")


def to_dev(a: np.ndarray, dev="cuda:0"):
    """A host array as a device tensor (bf16 bit patterns travel as int16)."""
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).to(dev)


def build_cache(lc, sp, keys, embs, tokens, capacity=None, max_batch=4096, insert_chunk=1 << 18, d_resp=None):
    """A cache filled with the given entries through lacache_insert (embs: one prefix store, or one per model of
    an ensemble cache when d_resp is given)."""
    c = lc.LaCache(capacity or max(1, keys.shape[0]), sp.d, sp.k_cap, sp.in_dtype, max_batch, 0, d_resp=d_resp)
    n = keys.shape[0]
    for r0 in range(0, n, insert_chunk):
        r1 = min(n, r0 + insert_chunk)
        if d_resp is None:
            first = c.insert(to_dev(keys[r0:r1]), to_dev(embs[r0:r1]), to_dev(tokens[r0:r1]))
        else:
            first = c.insert_ensemble(to_dev(keys[r0:r1]), [to_dev(e[r0:r1]) for e in embs], to_dev(tokens[r0:r1]))
        assert first == r0
    return c


def host_cpu_model() -> str:
    """The host CPU as /proc/cpuinfo names it, with its family / model / stepping numbers (a virtual machine
    may report only a short name)."""
    info = {}
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if not line.strip():
                    break  # the first processor's block is enough
                k, _, v = line.partition(":")
                info[k.strip()] = v.strip()
    except OSError:
        return "unknown"
    name = info.get("model name", "unknown")
    ids = [f"{k} {info[k]}" for k in ("cpu family", "model", "stepping") if k in info]
    return f"{name} ({', '.join(ids)})" if ids else name


def describe(sp, call_b):
    return (f"{sp.name}: N={sp.N:,} cached entries, d={sp.d} bf16 keys and prefix embeddings, k={sp.k} prefix "
            f"tokens, vocab {sp.vocab}, B={call_b} queries per call "
            f"({sp.frac_benign:.0%} benign / {sp.frac_collision:.0%} collision / rest miss"
            + (f", {sp.n_dup} exact-duplicate key pairs" if sp.n_dup else "") + ")")


def run_workload(name, steps, warmup, lc, torch, synth, traffic_db, want_cpu, graph=False):
    sp = synth.spec(name)
    call_b = synth.SERVE_SMALL_CALL_B if name == "serve_small" else sp.B
    t0 = time.time()
    w = synth.generate(sp)
    log(f"[bench] {name}: generated in {time.time() - t0:.1f}s")
    c = build_cache(lc, sp, w.keys, w.emb, w.tokens, max_batch=max(call_b, 16))
    q, a = to_dev(w.queries), to_dev(w.la_emb)
    t = to_dev(np.ascontiguousarray(w.la_tok[:, :sp.k]))
    n_calls = sp.B // call_b
    batches = [(q[i * call_b:(i + 1) * call_b], a[i * call_b:(i + 1) * call_b], t[i * call_b:(i + 1) * call_b])
               for i in range(n_calls)]
    dev = torch.device("cuda", 0)
    outs = [tuple(torch.empty(call_b, dtype=dt, device=dev)
                  for dt in (torch.int32, torch.float32, torch.float32, torch.int32)) for _ in range(n_calls)]

    def step(i):
        bq, ba, bt = batches[i % n_calls]
        c.lookup(bq, ba, bt, sp.tau_q, sp.tau_r, sp.k, out=outs[i % n_calls])

    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    # the timed steps; the library times the stage-1 launches of these very steps with HIP events taken from the
    # kernel's own dispatch on the call's stream (the roofline's kernel time).  Calls of a few hundred
    # microseconds or less time every tenth launch: a timed launch costs the host ~15 us more, which would weigh
    # on the throughput measured in the same loop
    c.profile(1 if call_b >= 1024 else 10)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(steps):
        step(i)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    k_ms, k_n = c.profile_read()
    c.profile(False)
    k_avg = k_ms / max(k_n, 1)
    # per-call times (median and minimum) from a pass with events around every call
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for i in range(steps):
        ev[i][0].record()
        step(i)
        ev[i][1].record()
    torch.cuda.synchronize()
    per_call = sorted(a.elapsed_time(b) for a, b in ev)
    call_ms = dict(median=per_call[len(per_call) // 2], min=per_call[0])
    sclk = sclk_under_load(torch, step)

    graph_res = None
    if graph:
        # the same call captured into a HIP graph and replayed back to back: its kernels' launch cost is paid at
        # capture, not per call (a lookup enqueues only kernels, so the capture holds it whole)
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step(0)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step(0)
        for _ in range(warmup):
            g.replay()
        torch.cuda.synchronize()
        e0.record()
        for _ in range(steps):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        gms = e0.elapsed_time(e1) / steps
        graph_res = dict(value=call_b / (gms * 1e-3), ms_per_step=gms)
        g.reset()

    # one more pass over every call of the pool, then the decisions of all its queries
    # (synthetic analogues of the paper's benign and attack hit rates)
    for i in range(n_calls):
        step(i)
    torch.cuda.synchronize()
    dec = np.concatenate([outs[i][3].cpu().numpy() for i in range(n_calls)])
    ben, col = w.cls == synth.CLS_BENIGN, w.cls == synth.CLS_COLLISION
    served = np.isin(dec, [2, 3])
    rates = dict(benign_hit_rate=float(served[ben].mean()), attack_hit_rate=float(served[col].mean()),
                 miss_rate_of_misses=float((dec[w.cls == synth.CLS_MISS] == 0).mean()))

    flops = 2.0 * call_b * sp.N * sp.d
    key_bytes = float(sp.N) * sp.d * 2
    if call_b >= 1024:
        roof = dict(bound="mfma", achieved=flops / (k_avg * 1e-3) / 1e12, peak=PEAK_BF16_TFLOPS, unit="TFLOP/s")
    else:
        roof = dict(bound="hbm", achieved=key_bytes / (k_avg * 1e-3) / 1e9, peak=PEAK_HBM_GBS, unit="GB/s")
    roof["frac"] = roof["achieved"] / roof["peak"]
    t = traffic_db.get(name)
    # counters describe the code they were taken on: a changed kernel reports no traffic
    roof["traffic"] = t["traffic_bytes"] if t and t.get("sources_digest") == sources_digest(name) else None
    roof["kernel_avg_ms"] = k_avg
    res = dict(workload=name, value=call_b / (ms * 1e-3), unit="lookups/s", ms_per_step=ms, B=call_b, call_ms=call_ms,
               sclk_mhz=sclk, graph=graph_res,
               roofline=roof, rates=rates, config=dict(workload=describe(sp, call_b), N=sp.N, d=sp.d, B=call_b,
                                                       k=sp.k, k_cap=sp.k_cap, tau_q=sp.tau_q, tau_r=sp.tau_r))
    if want_cpu:
        res["cpu_baseline"] = cpu_baseline(sp, w, call_b)
    c.close()
    del w, q, a, t, batches
    torch.cuda.empty_cache()
    return res


def run_resident(steps, warmup, lc, torch, synth):
    """The cache-resident workloads, absolute numbers only: tiny (10,000 x 384 float32 input, 64 queries per
    call) and mid (100,000 x 768 bf16, 256 per call), whose keys (7.7 MB, 154 MB) stay in the 256 MB infinity
    cache across calls, and the paper-shaped mid_paper (100,000 x 1024, k = 20, thresholds 0.80 / 0.70).
    Their calls take tens of microseconds, so each is also timed as one lookup captured into a HIP graph and
    replayed back to back (`graph_value`)."""
    out = []
    for name in ("tiny", "mid", "mid_paper"):
        r = run_workload(name, steps, warmup, lc, torch, synth, {}, False, graph=True)
        k_ms = r["roofline"]["kernel_avg_ms"]
        cfg = r["config"]
        out.append(dict(workload=cfg["workload"], value=r["value"], unit="lookups/s", ms_per_step=r["ms_per_step"],
                        stage1_kernel_avg_ms=k_ms, key_read_gbs=cfg["N"] * cfg["d"] * 2 / (k_ms * 1e-3) / 1e9,
                        graph_value=r["graph"]["value"], graph_ms_per_step=r["graph"]["ms_per_step"],
                        rates=r["rates"]))
    return out


def run_ensemble(steps, warmup, lc, torch, synth):
    """The serve_large workload with the lookahead ensemble of Section 5.4 (four prefix models of dimensions
    1024 / 384 / 768 / 1024, each at the threshold min(0.70, P10) of Appendix A.2, which is 0.70 for the
    synthetic benign prefix cosines U[0.70, 0.98]); half of the benign queries carry one substituted token,
    so the embedding checks decide them."""
    sp = synth.spec("serve_large")
    dims = synth.ENSEMBLE_DIMS
    tau_r = (0.70,) * len(dims)
    call_b = sp.B
    t0 = time.time()
    w = synth.generate(sp)
    embs = synth.ensemble_entries(sp, dims, 0, sp.N)
    las, la_tok = synth.ensemble_lookahead(sp, dims, embs, w.tokens,
                                           dict(cls=w.cls, target=w.target, la_tok=w.la_tok))
    log(f"[bench] ensemble: generated in {time.time() - t0:.1f}s")
    c = build_cache(lc, sp, w.keys, embs, w.tokens, max_batch=call_b, d_resp=tuple(dims))
    del embs
    q = to_dev(w.queries)
    a = [to_dev(x) for x in las]
    t = to_dev(np.ascontiguousarray(la_tok[:, :sp.k]))
    dev = torch.device("cuda", 0)
    out = (torch.empty(call_b, dtype=torch.int32, device=dev), torch.empty(call_b, dtype=torch.float32, device=dev),
           torch.empty((call_b, len(dims)), dtype=torch.float32, device=dev),
           torch.empty(call_b, dtype=torch.int32, device=dev))

    def step():
        c.lookup_ensemble(q, a, t, sp.tau_q, tau_r, sp.k, out=out)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    dec = out[3].cpu().numpy()
    served = np.isin(dec, [2, 3])
    ben, col = w.cls == synth.CLS_BENIGN, w.cls == synth.CLS_COLLISION
    res = dict(workload=f"serve_large keys with {len(dims)} prefix models of dimensions {list(dims)}, "
                        f"tau_r {list(tau_r)}, B={call_b} queries per call",
               m=len(dims), value=call_b / (ms * 1e-3), unit="lookups/s", ms_per_step=ms,
               rates=dict(benign_hit_rate=float(served[ben].mean()), attack_hit_rate=float(served[col].mean())))
    c.close()
    del w, q, a, t
    torch.cuda.empty_cache()
    return res


def run_calibration(steps, warmup, lc, torch, synth):
    """Threshold calibration (Appendix A.2) over a million benign pairs at d = 1024 (BGE's dimension):
    pair cosines as the lookup computes them, then tau_c = min(0.80, P5).  One step is one
    lacache_calibrate call; the pair-cosine pass reads 2 * n * d * 2 bytes."""
    n, d = 1_000_000, 1024
    t0 = time.time()
    a, b = synth.calibration_pairs(n, d, 0.80, 0.99, seed=66)
    log(f"[bench] calibration: generated in {time.time() - t0:.1f}s")
    c = lc.LaCache(16, d, 4, synth.BF16, 16, 0)
    ad, bd = to_dev(a), to_dev(b)
    del a, b
    dev = torch.device("cuda", 0)
    out = (torch.empty(n, dtype=torch.float32, device=dev), torch.empty(2, dtype=torch.float32, device=dev))
    for _ in range(warmup):
        c.calibrate(ad, bd, 5.0, 0.80, out=out)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        c.calibrate(ad, bd, 5.0, 0.80, out=out)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    tau = out[1].cpu().numpy()
    c.close()
    del ad, bd, out
    torch.cuda.empty_cache()
    pair_bytes = 2.0 * n * d * 2
    return dict(workload=f"{n:,} benign pairs, d = {d} bf16, cosines in U[0.80, 0.99], tau_c = min(0.80, P5)",
                value=n / (ms * 1e-3), unit="pairs/s", ms_per_step=ms, P5=float(tau[0]), tau=float(tau[1]),
                pair_read_gbs=pair_bytes / (ms * 1e-3) / 1e9)


def run_accept(steps, warmup, lc, torch, synth):
    """Speculative-decoding acceptance (Section 4.3) for 256 missed or rejected queries with k = 20 draft
    tokens over a 128,256-token vocabulary: the target's bf16 logits at the 20 positions (1.31 GB) are read
    once; one step is one lacache_accept_length call."""
    B, k, V = 256, 20, 128256
    t0 = time.time()
    lg, tok, pd = synth.draft_verification(B, k, V, seed=12)
    log(f"[bench] acceptance: generated in {time.time() - t0:.1f}s")
    lgd, tokd, pdd = to_dev(lg), to_dev(tok), to_dev(pd)
    del lg
    dev = torch.device("cuda", 0)
    out = (torch.empty(B, dtype=torch.int32, device=dev), torch.empty((B, k), dtype=torch.float32, device=dev))
    for _ in range(warmup):
        lc.lacache_accept_length(lgd, tokd, pdd, out=out)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        lc.lacache_accept_length(lgd, tokd, pdd, out=out)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    mean_len = float(out[0].float().mean().item())
    del lgd, tokd, pdd, out
    torch.cuda.empty_cache()
    logit_bytes = 2.0 * B * k * V
    return dict(workload=f"{B} queries x k = {k} draft tokens, vocabulary {V:,}, bf16 target logits",
                value=B / (ms * 1e-3), unit="queries/s", ms_per_step=ms, mean_accepted=mean_len,
                logits_read_gbs=logit_bytes / (ms * 1e-3) / 1e9)


def run_lsh(steps, warmup, lc, torch, synth):
    """The serve_small workload (1M x 768 keys, 16 queries per call) with stage 1 through the LSH index
    (Eq. (1)): 256 random-hyperplane bits per entry, candidates within 64 differing bits, exact re-rank.
    One step is one lacache_lookup_lsh call; recall is measured over the whole 4096-query pool against the
    exact lookup of the same pool."""
    sp = synth.spec("serve_small")
    call_b, bits, radius = synth.SERVE_SMALL_CALL_B, 256, 64
    t0 = time.time()
    w = synth.generate(sp)
    log(f"[bench] lsh: generated in {time.time() - t0:.1f}s")
    c = build_cache(lc, sp, w.keys, w.emb, w.tokens, max_batch=sp.B)
    q, a = to_dev(w.queries), to_dev(w.la_emb)
    t = to_dev(np.ascontiguousarray(w.la_tok[:, :sp.k]))
    exact = c.lookup(q, a, t, sp.tau_q, sp.tau_r, sp.k)
    torch.cuda.synchronize()
    ex_idx, ex_dec = exact[0].cpu().numpy(), exact[3].cpu().numpy()
    t0 = time.time()
    c.enable_lsh(bits, to_dev(synth.hyperplanes(bits, sp.d, seed=sp.seed + 1000)), 256)
    torch.cuda.synchronize()
    t_index = time.time() - t0
    n_calls = sp.B // call_b
    dev = torch.device("cuda", 0)
    outs = [tuple(torch.empty(call_b, dtype=dt, device=dev)
                  for dt in (torch.int32, torch.float32, torch.float32, torch.int32, torch.int32))
            for _ in range(n_calls)]

    def step(i):
        j = i % n_calls
        sl = slice(j * call_b, (j + 1) * call_b)
        c.lookup_lsh(q[sl], a[sl], t[sl], sp.tau_q, sp.tau_r, sp.k, radius, out=outs[j])

    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(steps):
        step(i)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    # the same pool in calls of 256 queries: the per-call launch and host cost spread over more lookups
    big = 256
    outs_big = [tuple(torch.empty(big, dtype=o.dtype, device=dev) for o in outs[0]) for _ in range(sp.B // big)]
    for j in range(len(outs_big)):
        sl = slice(j * big, (j + 1) * big)
        c.lookup_lsh(q[sl], a[sl], t[sl], sp.tau_q, sp.tau_r, sp.k, radius, out=outs_big[j])
    torch.cuda.synchronize()
    e0.record()
    for i in range(steps):
        j = i % len(outs_big)
        sl = slice(j * big, (j + 1) * big)
        c.lookup_lsh(q[sl], a[sl], t[sl], sp.tau_q, sp.tau_r, sp.k, radius, out=outs_big[j])
    e1.record()
    torch.cuda.synchronize()
    ms_big = e0.elapsed_time(e1) / steps
    for i in range(n_calls):
        step(i)
    torch.cuda.synchronize()
    idx = np.concatenate([o[0].cpu().numpy() for o in outs])
    dec = np.concatenate([o[3].cpu().numpy() for o in outs])
    nc = np.concatenate([o[4].cpu().numpy() for o in outs])
    hit = ex_dec >= 1
    c.close()
    del w, q, a, t
    torch.cuda.empty_cache()
    return dict(workload=f"serve_small keys (1M x 768), {call_b} queries per call, {bits}-bit random-hyperplane "
                         f"signatures, Hamming radius {radius}, exact re-rank",
                value=call_b / (ms * 1e-3), unit="lookups/s", ms_per_step=ms,
                value_256_per_call=big / (ms_big * 1e-3), ms_per_256_call=ms_big,
                recall_stage1_hits=float(np.mean((idx == ex_idx) & (dec == ex_dec), where=hit)),
                decisions_equal=float(np.mean(dec == ex_dec)), mean_candidates=float(nc.mean()),
                signature_bytes=float(sp.N) * bits / 8, index_build_s=t_index)


def run_large_interleaved(lc, torch, synth, traffic_db, epochs=8, per_epoch=8, batch=4096):
    """The clustered workload (4,000,000 x 1024 bf16 keys around 10,000 centroids, k = 32, 1024 queries
    per lookup) on its serving schedule: 8 lookups, then an insert of 4096 new clustered entries, repeated
    8 times; from the second round on 10 % of the planted queries aim at the latest insert batch.  Every
    lookup and insert of the schedule is in the timed region (inputs resident in HBM beforehand);
    `value` is queries served per second over the whole cycle.  The stage-1 kernel time is the average over
    the 64 lookups of that timed schedule, measured with events on the library's stream around each launch."""
    sp = synth.spec("large")
    total = sp.N + epochs * batch
    t0 = time.time()
    keys, emb, tok = synth.entries(sp, 0, total)
    c = build_cache(lc, sp, keys[:sp.N], emb[:sp.N], tok[:sp.N], capacity=total, max_batch=sp.B)
    ins, pools = [], []
    for e in range(epochs):
        n = sp.N + e * batch
        ins.append((to_dev(keys[n:n + batch]), to_dev(emb[n:n + batch]), to_dev(tok[n:n + batch])))
        recent = (n - batch, n) if e > 0 else None
        q = synth.queries(sp, keys, emb, tok, np.zeros((0, 2), np.int64), B=per_epoch * sp.B, N=n,
                          stream_chunk=500 + e, recent=recent)
        pools.append(dict(q=to_dev(q["queries"]), a=to_dev(q["la_emb"]),
                          t=to_dev(np.ascontiguousarray(q["la_tok"][:, :sp.k])), cls=q["cls"], target=q["target"],
                          recent=recent))
    del keys, emb, tok
    log(f"[bench] large_interleaved: store, insert batches and query pools ready in {time.time() - t0:.1f}s")
    dev = torch.device("cuda", 0)
    outs = [[tuple(torch.empty(sp.B, dtype=dt, device=dev) for dt in (torch.int32, torch.float32, torch.float32,
                                                                       torch.int32)) for _ in range(per_epoch)]
            for _ in range(epochs)]

    def lookup(e, j):
        p, s_ = pools[e], slice(j * sp.B, (j + 1) * sp.B)
        c.lookup(p["q"][s_], p["a"][s_], p["t"][s_], sp.tau_q, sp.tau_r, sp.k, out=outs[e][j])

    for j in range(2):  # warm-up at the initial size
        lookup(0, j)
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(epochs)]
    c.profile(True)
    for e in range(epochs):
        ev[e][0].record()
        for j in range(per_epoch):
            lookup(e, j)
        ev[e][1].record()
        first = c.insert(*ins[e])
        assert first == sp.N + e * batch
        ev[e][2].record()
    torch.cuda.synchronize()
    k_ms, k_n = c.profile_read()
    c.profile(False)
    total_ms = ev[0][0].elapsed_time(ev[-1][2])
    lookup_ms = sum(ev[e][0].elapsed_time(ev[e][1]) for e in range(epochs))
    insert_ms = sum(ev[e][1].elapsed_time(ev[e][2]) for e in range(epochs))
    n_lookups = epochs * per_epoch

    dec = np.concatenate([np.concatenate([outs[e][j][3].cpu().numpy() for j in range(per_epoch)])
                          for e in range(epochs)])
    idx = np.concatenate([np.concatenate([outs[e][j][0].cpu().numpy() for j in range(per_epoch)])
                          for e in range(epochs)])
    cls = np.concatenate([p["cls"] for p in pools])
    target = np.concatenate([p["target"] for p in pools])
    aimed = np.concatenate([(p["target"] >= p["recent"][0]) if p["recent"] else np.zeros(len(p["cls"]), bool)
                            for p in pools]) & (cls == synth.CLS_BENIGN)
    served = np.isin(dec, [2, 3])
    rates = dict(benign_hit_rate=float(served[cls == synth.CLS_BENIGN].mean()),
                 attack_hit_rate=float(served[cls == synth.CLS_COLLISION].mean()),
                 miss_rate_of_misses=float((dec[cls == synth.CLS_MISS] == 0).mean()),
                 latest_batch_found=float(np.mean(served[aimed] & (idx[aimed] == target[aimed]))),
                 latest_batch_queries=int(aimed.sum()))

    assert k_n == n_lookups
    k_avg = k_ms / k_n
    n_final = sp.N + epochs * batch
    # the lookups of epoch e search sp.N + e * batch entries
    flops = sum(per_epoch * 2.0 * sp.B * (sp.N + e * batch) * sp.d for e in range(epochs))
    achieved = flops / (k_ms * 1e-3) / 1e12
    t = traffic_db.get("large")
    traffic = t["traffic_bytes"] if t and t.get("sources_digest") == sources_digest("large") else None
    c.close()
    del pools, ins, outs
    torch.cuda.empty_cache()
    return dict(workload=(f"large: N={sp.N:,} clustered entries (10,000 centroids) growing by {batch} per insert to "
                          f"{n_final:,}, d={sp.d} bf16, k={sp.k}, B={sp.B} queries per lookup, {per_epoch} lookups "
                          f"then one insert, {epochs} times"),
                value=n_lookups * sp.B / (total_ms * 1e-3), unit="lookups/s",
                ms_per_lookup=lookup_ms / n_lookups, ms_per_insert=insert_ms / epochs,
                insert_entries_per_s=epochs * batch / (insert_ms * 1e-3),
                stage1_kernel_avg_ms=k_avg,
                roofline=dict(bound="mfma", achieved=achieved, peak=PEAK_BF16_TFLOPS, unit="TFLOP/s",
                              frac=achieved / PEAK_BF16_TFLOPS, traffic=traffic),
                rates=rates)


def run_sweep(steps, warmup, lc, torch, synth):
    """Lookup throughput over the batch size on the 1M x 768 serving cache: the exact path at the default
    crossover (the streaming kernel up to three 64-query groups, the GEMM kernel above) and, up to 1024
    queries, the LSH path (256 bits, radius 64); then, for 160-256 queries, the exact path with the
    streaming kernel forced (three and four query groups, `set_small_batch(256)`) and, for 128-256, with the
    GEMM kernel forced (`set_small_batch(0)`): the measurements behind the default crossover.  Prints one JSON line per batch size and path set."""
    sp = synth.spec("serve_large")
    w = synth.generate(sp)
    c = build_cache(lc, sp, w.keys, w.emb, w.tokens, max_batch=sp.B)
    c.enable_lsh(256, to_dev(synth.hyperplanes(256, sp.d, seed=sp.seed + 1000)), 256)
    q, a = to_dev(w.queries), to_dev(w.la_emb)
    t = to_dev(np.ascontiguousarray(w.la_tok[:, :sp.k]))

    def measure(B, path):
        n_calls = max(1, min(16, sp.B // B))
        sl = [slice(i * B, (i + 1) * B) for i in range(n_calls)]
        exact = path != "lsh"

        def call(i):
            s_ = sl[i % n_calls]
            if exact:
                c.lookup(q[s_], a[s_], t[s_], sp.tau_q, sp.tau_r, sp.k)
            else:
                c.lookup_lsh(q[s_], a[s_], t[s_], sp.tau_q, sp.tau_r, sp.k, 64)
        for i in range(warmup):
            call(i)
        torch.cuda.synchronize()
        if exact:
            c.profile(True)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(steps):
            call(i)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        r = {"ms_per_call": ms, "lookups_per_s": B / (ms * 1e-3)}
        if exact:
            k_ms, k_n = c.profile_read()
            c.profile(False)
            k_avg = k_ms / max(k_n, 1)
            r["stage1_ms"] = k_avg
            # both rates: which kernel ran depends on B, d and the crossover
            r["stage1_gbs"] = sp.N * sp.d * 2 / (k_avg * 1e-3) / 1e9
            r["stage1_tflops"] = 2.0 * B * sp.N * sp.d / (k_avg * 1e-3) / 1e12
        return r

    rows = []
    for B in (1, 2, 4, 8, 16, 32, 64, 128, 256, 512, 1024, 2048, 4096):
        res = {"B": B, "exact": measure(B, "exact")}
        if B <= 1024:
            res["lsh"] = measure(B, "lsh")
        print(json.dumps(res), flush=True)
        rows.append(res)
    c.set_small_batch(256)  # the streaming kernel's largest batch at d = 768
    for B in (160, 192, 224, 256):
        res = {"B": B, "exact_stream_forced": measure(B, "exact")}
        print(json.dumps(res), flush=True)
        rows.append(res)
    c.set_small_batch(0)  # every batch on the GEMM kernel
    for B in (128, 160, 192, 224, 256):
        res = {"B": B, "exact_gemm_forced": measure(B, "exact")}
        print(json.dumps(res), flush=True)
        rows.append(res)
    c.close()
    return rows


def cpu_baseline(sp, w, call_b):
    """The CPU oracle, as it is, on a bounded sample: a few queries against the full cache."""
    import oracle
    t0 = time.time()
    kq = oracle.quantise(w.keys, sp.in_dtype)
    eq = oracle.quantise(w.emb, sp.in_dtype)
    t_store = time.time() - t0
    threads = oracle.num_threads()
    n = min(sp.B, 512)  # about 10-30 s of work on a 16-thread host
    qq = oracle.quantise(w.queries[:n], sp.in_dtype)
    aq = oracle.quantise(w.la_emb[:n], sp.in_dtype)
    u = np.ascontiguousarray(w.la_tok[:n, :sp.k])
    t0 = time.perf_counter()
    oracle.lookup(kq, eq, w.tokens, qq, aq, u, sp.tau_q, sp.tau_r, sp.k)
    el = time.perf_counter() - t0
    # the same oracle on one thread, on the first 16 of those queries
    n1 = min(n, 16)
    oracle.set_num_threads(1)
    try:
        t0 = time.perf_counter()
        oracle.lookup(kq, eq, w.tokens, qq[:n1], aq[:n1], u[:n1], sp.tau_q, sp.tau_r, sp.k)
        el1 = time.perf_counter() - t0
    finally:
        oracle.set_num_threads(threads)
    return dict(value=n / el, unit="lookups/s", cores=threads, kind="oracle", cpu_model=host_cpu_model(),
                sample=f"{n} queries of the same pool against all {sp.N:,} entries (queries quantised outside the "
                       f"timed call; store quantisation {t_store:.1f}s not counted), {el:.1f}s",
                single_thread=dict(value=n1 / el1, unit="lookups/s", cores=1,
                                   sample=f"the first {n1} of those queries, {el1:.1f}s"))


def main():
    args = parse()
    if args.pmc_summary:
        pmc_summary(args.pmc_summary, args.traffic, args.copy_mib)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the lookup is built and measured on a single MI355X; "
              "sharding the cache over several GPUs is not implemented.", file=sys.stderr)
        sys.exit(2)
    if args.calibrate_copy_mib:
        calibrate_copy(args.calibrate_copy_mib)
        return
    if args.sweep:
        import torch
        import synth
        import paper_2608_01718_amd as lc
        run_sweep(args.steps, args.warmup, lc, torch, synth)
        return
    probe = None if args.no_probe else attainable_ceilings()
    import torch
    import synth
    import paper_2608_01718_amd as lc  # raises if liblacache.so has not been built
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    traffic_db = {}
    if os.path.exists(args.traffic):
        traffic_db = json.load(open(args.traffic))

    main_res = run_workload(args.workload, args.steps, args.warmup, lc, torch, synth, traffic_db, not args.no_cpu)
    secondary = None
    if not args.no_secondary:
        other = "serve_small" if args.workload == "serve_large" else "serve_large"
        secondary = run_workload(other, args.steps, args.warmup, lc, torch, synth, traffic_db, False)

    ensemble = None if args.no_ensemble else run_ensemble(args.steps, args.warmup, lc, torch, synth)
    calibration = None if args.no_calibration else run_calibration(args.steps, args.warmup, lc, torch, synth)
    accept = None if args.no_accept else run_accept(args.steps, args.warmup, lc, torch, synth)
    lsh = None if args.no_lsh else run_lsh(args.steps, args.warmup, lc, torch, synth)
    large = None if args.no_large else run_large_interleaved(lc, torch, synth, traffic_db)
    resident = None if args.no_resident else run_resident(args.steps, args.warmup, lc, torch, synth)

    line = {
        "metric": "cache lookups/sec (2-stage) at N=1M,d=768; % HBM / MFMA roofline",
        "value": main_res["value"],
        "unit": "lookups/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": main_res["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded Gaussian embeddings with planted benign / collision / miss queries)",
        "config": main_res["config"],
        "roofline": {k: main_res["roofline"][k] for k in ("bound", "achieved", "peak", "unit", "frac", "traffic")},
        "stage1_kernel_avg_ms": main_res["roofline"]["kernel_avg_ms"],
        "call_ms": main_res["call_ms"],
        "sclk_mhz_under_load": main_res["sclk_mhz"],
        "rates": main_res["rates"],
        "cpu_baseline": main_res.get("cpu_baseline"),
    }
    if secondary:
        line["secondary"] = {
            "workload": secondary["config"]["workload"], "value": secondary["value"], "unit": "lookups/s",
            "ms_per_step": secondary["ms_per_step"],
            "roofline": {k: secondary["roofline"][k] for k in ("bound", "achieved", "peak", "unit", "frac",
                                                                  "traffic")},
            "stage1_kernel_avg_ms": secondary["roofline"]["kernel_avg_ms"], "call_ms": secondary["call_ms"],
            "sclk_mhz_under_load": secondary["sclk_mhz"],
            "rates": secondary["rates"]}
    if ensemble:
        line["ensemble"] = ensemble
    if calibration:
        line["calibration"] = calibration
    if accept:
        line["accept"] = accept
    if lsh:
        line["lsh"] = lsh
    if large:
        line["large_interleaved"] = large
    if resident:
        line["resident"] = resident
    if probe:
        # the same kernels rated against what this GPU sustains: MFMA throughput on random bf16 operands
        # (operand-dependent power lowers the clock below the datasheet's) and a plain streaming read
        att = {"mfma_bf16_random_tflops": probe["mfma_random_tflops"],
               "mfma_bf16_random_32x32x16_tflops": probe.get("mfma_random_32x32x16_tflops"),
               "mfma_bf16_random_16x16x32_tflops": probe.get("mfma_random_16x16x32_tflops"),
               "mfma_bf16_constant_tflops": probe["mfma_constant_tflops"], "hbm_read_gbs": probe["hbm_read_gbs"],
               "hbm_read_plain_gbs": probe.get("hbm_read_plain_gbs")}
        for key, res in (("frac", main_res), ("secondary_frac", secondary)):
            if not res:
                continue
            rf = res["roofline"]
            ceil = probe["mfma_random_tflops"] if rf["bound"] == "mfma" else probe["hbm_read_gbs"]
            att[key] = rf["achieved"] / ceil
        line["attainable"] = att
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
