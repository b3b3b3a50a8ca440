"""Python binding of liblacache (the gfx950 LaCache two-stage lookup): argument marshalling only.

Every function mirrors one entry point of ``include/lacache.h`` under the
same name and passes torch device tensors' data pointers and the current HIP
stream straight through; all work runs in the library's kernels.  There is no
fallback: importing this module fails if ``liblacache.so`` has not been built
(``python paper_2608_01718_amd/build.py``).
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblacache.so")

MISS, REJECT, HIT, HIT_EXACT = 0, 1, 2, 3
OK, EINVAL, EFULL, ENOMEM, EHIP = 0, -1, -2, -3, -4
F32, BF16 = 0, 1
MAX_MODELS = 8

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python paper_2608_01718_amd/build.py` "
                      "(there is no non-HIP implementation of the lookup)")

_lib = ctypes.CDLL(LIB_PATH)
_P, _i32, _i64, _f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float
_lib.lacache_create.argtypes = [ctypes.POINTER(_P), _i64, _i32, _i32, ctypes.c_int, _i32, _i32]
_lib.lacache_create_ensemble.argtypes = [ctypes.POINTER(_P), _i64, _i32, _i32, ctypes.c_int, _i32, _i32, _i32,
                                         ctypes.POINTER(_i32)]
_lib.lacache_models.argtypes = [_P]
_lib.lacache_models.restype = _i32
_lib.lacache_insert_ensemble.argtypes = [_P, _P, ctypes.POINTER(_P), _P, _i32, ctypes.POINTER(_i64), _P]
_lib.lacache_lookup_ensemble.argtypes = [_P, _P, ctypes.POINTER(_P), _P, _i32, _f32, ctypes.POINTER(_f32), _i32,
                                         _P, _P, _P, _P, _P]
_lib.lacache_export_prefix.argtypes = [_P, _i32, _i64, _i32, _P, _P]
_lib.lacache_calibrate.argtypes = [_P, _i32, _P, _P, _i64, _f32, _f32, _P, _P, _P]
_lib.lacache_calibrate_noalloc.argtypes = [_P, _P, ctypes.c_int, _i32, _i64, _f32, _f32, _P, _P, _P]
_lib.lacache_accept_length.argtypes = [_P, ctypes.c_int, _i32, _P, _P, _i32, _i32, _P, _P, _P]
_lib.lacache_enable_lsh.argtypes = [_P, _i32, _P, _i32, _P]
_lib.lacache_lookup_lsh.argtypes = [_P, _P, _P, _P, _i32, _f32, _f32, _i32, _i32, _P, _P, _P, _P, _P, _P]
_lib.lacache_export_signatures.argtypes = [_P, _i64, _i32, _P, _P]
_lib.lacache_destroy.argtypes = [_P]
_lib.lacache_insert.argtypes = [_P, _P, _P, _P, _i32, ctypes.POINTER(_i64), _P]
_lib.lacache_lookup.argtypes = [_P, _P, _P, _P, _i32, _f32, _f32, _i32, _P, _P, _P, _P, _P]
_lib.lacache_size.argtypes = [_P]
_lib.lacache_size.restype = _i64
_lib.lacache_export.argtypes = [_P, _i64, _i32, _P, _P, _P, _P]
_lib.lacache_set_small_batch.argtypes = [_P, _i32]
_lib.lacache_profile.argtypes = [_P, _i32]
_lib.lacache_profile_read.argtypes = [_P, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_i64)]
_lib.lacache_replay_fallbacks.argtypes = [_P, ctypes.POINTER(_i64)]
_lib.lacache_strerror.argtypes = [ctypes.c_int]
_lib.lacache_strerror.restype = ctypes.c_char_p

EXPORTED = ("lacache_create", "lacache_create_ensemble", "lacache_models", "lacache_destroy", "lacache_insert",
            "lacache_insert_ensemble", "lacache_lookup", "lacache_lookup_ensemble", "lacache_size",
            "lacache_export", "lacache_export_prefix", "lacache_calibrate", "lacache_calibrate_noalloc",
            "lacache_accept_length",
            "lacache_enable_lsh", "lacache_lookup_lsh", "lacache_export_signatures",
            "lacache_set_small_batch",
            "lacache_profile", "lacache_profile_read", "lacache_replay_fallbacks", "lacache_strerror")


class LaCacheError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__(f"{what}: {lacache_strerror(code)} ({code})")
        self.code = code


def lacache_strerror(code: int) -> str:
    return _lib.lacache_strerror(code).decode()


def _check(code: int, what: str) -> None:
    if code != OK:
        raise LaCacheError(code, what)


def _stream(device: int, stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _vec(t: torch.Tensor, dtype: int, rows: int, d: int, device: int, name: str) -> int:
    want = (torch.float32,) if dtype == F32 else (torch.bfloat16, torch.int16, torch.uint16)
    if t.dtype not in want or t.device.type != "cuda" or t.device.index != device:
        raise ValueError(f"{name}: expected a {want} tensor on cuda:{device}, got {t.dtype} on {t.device}")
    if tuple(t.shape) != (rows, d) or not t.is_contiguous():
        raise ValueError(f"{name}: expected a contiguous [{rows}, {d}] tensor, got {tuple(t.shape)}")
    return t.data_ptr()


def _ints(t: torch.Tensor, shape, device: int, name: str) -> int:
    if t.dtype != torch.int32 or t.device.type != "cuda" or t.device.index != device:
        raise ValueError(f"{name}: expected an int32 tensor on cuda:{device}")
    if tuple(t.shape) != tuple(shape) or not t.is_contiguous():
        raise ValueError(f"{name}: expected a contiguous {list(shape)} tensor, got {tuple(t.shape)}")
    return t.data_ptr()


class LaCache:
    """A handle of the C library plus the sizes it was created with.  ``d_resp`` (one dimension per prefix
    model) makes an ensemble cache through lacache_create_ensemble; without it the cache has one prefix
    model of dimension d."""

    def __init__(self, capacity: int, d: int, k_cap: int, in_dtype: int = BF16, max_batch: int = 4096,
                 device: int = 0, d_resp=None):
        self.capacity, self.d, self.k_cap, self.in_dtype = capacity, d, k_cap, in_dtype
        self.max_batch, self.device = max_batch, device
        h = _P()
        if d_resp is None:
            self.d_resp = (d,)
            _check(_lib.lacache_create(ctypes.byref(h), capacity, d, k_cap, in_dtype, max_batch, device),
                   "lacache_create")
        else:
            self.d_resp = tuple(int(x) for x in d_resp)
            arr = (_i32 * max(1, len(self.d_resp)))(*self.d_resp)
            _check(_lib.lacache_create_ensemble(ctypes.byref(h), capacity, d, k_cap, in_dtype, max_batch, device,
                                                len(self.d_resp), arr), "lacache_create_ensemble")
        self._h = h

    @property
    def m(self) -> int:
        return len(self.d_resp)

    @property
    def handle(self):
        if self._h is None:
            raise ValueError("the cache has been destroyed")
        return self._h

    def insert(self, keys, resp_emb, resp_tokens, stream=None) -> int:
        return lacache_insert(self, keys, resp_emb, resp_tokens, stream)

    def lookup(self, queries, lookahead_emb, lookahead_tokens, tau_q, tau_r, k, out=None, stream=None):
        return lacache_lookup(self, queries, lookahead_emb, lookahead_tokens, tau_q, tau_r, k, out, stream)

    def export(self, first: int, n: int, stream=None):
        return lacache_export(self, first, n, stream)

    def insert_ensemble(self, keys, resp_embs, resp_tokens, stream=None) -> int:
        return lacache_insert_ensemble(self, keys, resp_embs, resp_tokens, stream)

    def lookup_ensemble(self, queries, lookahead_embs, lookahead_tokens, tau_q, tau_r, k, out=None, stream=None):
        return lacache_lookup_ensemble(self, queries, lookahead_embs, lookahead_tokens, tau_q, tau_r, k, out,
                                       stream)

    def export_prefix(self, model: int, first: int, n: int, stream=None):
        return lacache_export_prefix(self, model, first, n, stream)

    def enable_lsh(self, bits: int, hyperplanes, max_candidates: int = 256, stream=None) -> None:
        lacache_enable_lsh(self, bits, hyperplanes, max_candidates, stream)

    def lookup_lsh(self, queries, lookahead_emb, lookahead_tokens, tau_q, tau_r, k, radius, out=None, stream=None):
        return lacache_lookup_lsh(self, queries, lookahead_emb, lookahead_tokens, tau_q, tau_r, k, radius, out,
                                  stream)

    def export_signatures(self, first: int, n: int, stream=None):
        return lacache_export_signatures(self, first, n, stream)

    def calibrate(self, a, b, percentile: float, cap: float, which: int = -1, out=None, stream=None):
        return lacache_calibrate(self, which, a, b, percentile, cap, out, stream)

    def size(self) -> int:
        return lacache_size(self)

    def set_small_batch(self, b_small: int) -> None:
        lacache_set_small_batch(self, b_small)

    def profile(self, every) -> None:
        lacache_profile(self, every)

    def profile_read(self):
        return lacache_profile_read(self)

    def replay_fallbacks(self) -> int:
        return lacache_replay_fallbacks(self)

    def close(self) -> None:
        if getattr(self, "_h", None) is not None:
            lacache_destroy(self)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def lacache_create(capacity: int, d: int, k_cap: int, in_dtype: int = BF16, max_batch: int = 4096,
                   device: int = 0) -> LaCache:
    return LaCache(capacity, d, k_cap, in_dtype, max_batch, device)


def lacache_create_ensemble(capacity: int, d: int, k_cap: int, in_dtype: int, max_batch: int, device: int,
                            d_resp) -> LaCache:
    return LaCache(capacity, d, k_cap, in_dtype, max_batch, device, d_resp=d_resp)


def lacache_models(c: LaCache) -> int:
    return int(_lib.lacache_models(c.handle))


def lacache_destroy(c: LaCache) -> None:
    h, c._h = c._h, None
    _check(_lib.lacache_destroy(h), "lacache_destroy")


def lacache_insert(c: LaCache, keys, resp_emb, resp_tokens, stream=None) -> int:
    n = keys.shape[0]
    first = _i64(-1)
    _check(_lib.lacache_insert(c.handle, _vec(keys, c.in_dtype, n, c.d, c.device, "keys"),
                               _vec(resp_emb, c.in_dtype, n, c.d, c.device, "resp_emb"),
                               _ints(resp_tokens, (n, c.k_cap), c.device, "resp_tokens"), n, ctypes.byref(first),
                               _stream(c.device, stream)), "lacache_insert")
    return first.value


def lacache_insert_ensemble(c: LaCache, keys, resp_embs, resp_tokens, stream=None) -> int:
    """resp_embs: one [n][d_resp[i]] tensor per prefix model."""
    n = keys.shape[0]
    if len(resp_embs) != c.m:
        raise ValueError(f"resp_embs: expected {c.m} tensors, got {len(resp_embs)}")
    ptrs = (_P * c.m)(*[_vec(e, c.in_dtype, n, c.d_resp[i], c.device, f"resp_embs[{i}]")
                         for i, e in enumerate(resp_embs)])
    first = _i64(-1)
    _check(_lib.lacache_insert_ensemble(c.handle, _vec(keys, c.in_dtype, n, c.d, c.device, "keys"), ptrs,
                                        _ints(resp_tokens, (n, c.k_cap), c.device, "resp_tokens"), n,
                                        ctypes.byref(first), _stream(c.device, stream)), "lacache_insert_ensemble")
    return first.value


def lacache_lookup_ensemble(c: LaCache, queries, lookahead_embs, lookahead_tokens, tau_q: float, tau_r, k: int,
                            out=None, stream=None):
    """lookahead_embs: one [B][d_resp[i]] tensor per prefix model; tau_r: one threshold per model.
    Returns (idx int32 [B], score f32 [B], resp_score f32 [B][m], decision int32 [B])."""
    B = queries.shape[0]
    m = c.m
    dev = torch.device("cuda", c.device)
    if len(lookahead_embs) != m or len(tau_r) != m:
        raise ValueError(f"expected {m} lookahead embeddings and {m} thresholds")
    if out is None:
        out = (torch.empty(B, dtype=torch.int32, device=dev), torch.empty(B, dtype=torch.float32, device=dev),
               torch.empty((B, m), dtype=torch.float32, device=dev), torch.empty(B, dtype=torch.int32, device=dev))
    idx, score, resp, dec = out
    for t, dt, n, nm in ((idx, torch.int32, B, "idx"), (score, torch.float32, B, "score"),
                         (resp, torch.float32, B * m, "resp"), (dec, torch.int32, B, "decision")):
        if t.dtype != dt or t.device != dev or t.numel() != n or not t.is_contiguous():
            raise ValueError(f"{nm}: expected a contiguous {dt} tensor of {n} elements on {dev}")
    ptrs = (_P * m)(*[_vec(e, c.in_dtype, B, c.d_resp[i], c.device, f"lookahead_embs[{i}]")
                      for i, e in enumerate(lookahead_embs)])
    taus = (_f32 * m)(*[float(t) for t in tau_r])
    _check(_lib.lacache_lookup_ensemble(c.handle, _vec(queries, c.in_dtype, B, c.d, c.device, "queries"), ptrs,
                                        _ints(lookahead_tokens, (B, k), c.device, "lookahead_tokens"), B,
                                        float(tau_q), taus, int(k), idx.data_ptr(), score.data_ptr(),
                                        resp.data_ptr(), dec.data_ptr(), _stream(c.device, stream)),
           "lacache_lookup_ensemble")
    return out


def lacache_lookup(c: LaCache, queries, lookahead_emb, lookahead_tokens, tau_q: float, tau_r: float, k: int,
                   out=None, stream=None):
    """Returns (idx int32, score f32, resp_score f32, decision int32), each [B], on the cache's device."""
    B = queries.shape[0]
    dev = torch.device("cuda", c.device)
    if out is None:
        out = (torch.empty(B, dtype=torch.int32, device=dev), torch.empty(B, dtype=torch.float32, device=dev),
               torch.empty(B, dtype=torch.float32, device=dev), torch.empty(B, dtype=torch.int32, device=dev))
    idx, score, resp, dec = out
    for t, dt, nm in ((idx, torch.int32, "idx"), (score, torch.float32, "score"), (resp, torch.float32, "resp"),
                      (dec, torch.int32, "decision")):
        if t.dtype != dt or t.device != dev or t.numel() != B or not t.is_contiguous():
            raise ValueError(f"{nm}: expected a contiguous [{B}] {dt} tensor on {dev}")
    _check(_lib.lacache_lookup(c.handle, _vec(queries, c.in_dtype, B, c.d, c.device, "queries"),
                               _vec(lookahead_emb, c.in_dtype, B, c.d, c.device, "lookahead_emb"),
                               _ints(lookahead_tokens, (B, k), c.device, "lookahead_tokens"), B, float(tau_q),
                               float(tau_r), int(k), idx.data_ptr(), score.data_ptr(), resp.data_ptr(),
                               dec.data_ptr(), _stream(c.device, stream)), "lacache_lookup")
    return out


def lacache_size(c: LaCache) -> int:
    return int(_lib.lacache_size(c.handle))


def lacache_export(c: LaCache, first: int, n: int, stream=None):
    """Returns (keys bf16-bits int16 [n][d], emb int16 [n][d], tokens int32 [n][k_cap]) as stored."""
    dev = torch.device("cuda", c.device)
    keys = torch.empty((n, c.d), dtype=torch.int16, device=dev)
    emb = torch.empty((n, c.d_resp[0]), dtype=torch.int16, device=dev)
    tok = torch.empty((n, c.k_cap), dtype=torch.int32, device=dev)
    _check(_lib.lacache_export(c.handle, first, n, keys.data_ptr(), emb.data_ptr(), tok.data_ptr(),
                               _stream(c.device, stream)), "lacache_export")
    return keys, emb, tok


def lacache_export_prefix(c: LaCache, model: int, first: int, n: int, stream=None):
    """The stored prefix embeddings of one model, bf16 bits as int16 [n][d_resp[model]]."""
    if not 0 <= model < c.m:
        raise ValueError(f"model must be in [0, {c.m})")
    emb = torch.empty((n, c.d_resp[model]), dtype=torch.int16, device=torch.device("cuda", c.device))
    _check(_lib.lacache_export_prefix(c.handle, model, first, n, emb.data_ptr(), _stream(c.device, stream)),
           "lacache_export_prefix")
    return emb


def lacache_calibrate(c: LaCache, which: int, a, b, percentile: float, cap: float, out=None, stream=None):
    """Pair cosines and the capped percentile threshold (Appendix A.2).  which = -1: key-model vectors of
    dimension d; else prefix model `which`.  Returns (sims f32 [n], tau f32 [2] = (percentile, min(cap, .)))
    on the cache's device."""
    # an out-of-range `which` is passed through for the library to reject
    dim = c.d_resp[which] if 0 <= which < c.m else (c.d if which == -1 else a.shape[1])
    n = a.shape[0]
    dev = torch.device("cuda", c.device)
    if out is None:
        out = (torch.empty(n, dtype=torch.float32, device=dev), torch.empty(2, dtype=torch.float32, device=dev))
    sims, tau = out
    for t, k, nm in ((sims, n, "sims"), (tau, 2, "tau")):
        if t.dtype != torch.float32 or t.device != dev or t.numel() != k or not t.is_contiguous():
            raise ValueError(f"{nm}: expected a contiguous float32 tensor of {k} elements on {dev}")
    _check(_lib.lacache_calibrate(c.handle, int(which), _vec(a, c.in_dtype, n, dim, c.device, "a"),
                                  _vec(b, c.in_dtype, n, dim, c.device, "b"), n, float(percentile), float(cap),
                                  sims.data_ptr(), tau.data_ptr(), _stream(c.device, stream)), "lacache_calibrate")
    return out


def lacache_calibrate_noalloc(a, b, percentile: float, cap: float, out=None, stream=None):
    """lacache_calibrate without a handle, with the library's static scratch: a, b [n][d] float32 or bfloat16
    (int16/uint16 bits) on the current device.  Returns (sims f32 [n], tau f32 [2]); with `out` given no device
    memory is allocated here either."""
    if a.dim() != 2 or a.shape != b.shape or a.dtype != b.dtype:
        raise ValueError("a, b: expected two [n, d] tensors of one dtype")
    dtype = F32 if a.dtype == torch.float32 else BF16
    n, d = a.shape
    dev = a.device
    if out is None:
        out = (torch.empty(n, dtype=torch.float32, device=dev), torch.empty(2, dtype=torch.float32, device=dev))
    sims, tau = out
    for t, k, nm in ((sims, n, "sims"), (tau, 2, "tau")):
        if t.dtype != torch.float32 or t.device != dev or t.numel() != k or not t.is_contiguous():
            raise ValueError(f"{nm}: expected a contiguous float32 tensor of {k} elements on {dev}")
    _check(_lib.lacache_calibrate_noalloc(_vec(a, dtype, n, d, dev.index, "a"), _vec(b, dtype, n, d, dev.index, "b"),
                                          dtype, d, n, float(percentile), float(cap), sims.data_ptr(),
                                          tau.data_ptr(), _stream(dev.index, stream)),
           "lacache_calibrate_noalloc")
    return out


def lacache_accept_length(logits, draft_tokens, p_draft, out=None, stream=None):
    """Speculative-decoding acceptance (Section 4.3).  logits: [B][k][V] float32 or bfloat16 (int16/uint16
    bits) on a GPU; draft_tokens [B][k] int32; p_draft [B][k] float32.  Returns (accept_len int32 [B],
    p_target float32 [B][k]) on the same device."""
    if logits.dim() != 3 or logits.device.type != "cuda" or not logits.is_contiguous():
        raise ValueError("logits: expected a contiguous [B, k, V] tensor on a GPU")
    B, k, V = logits.shape
    dtype = F32 if logits.dtype == torch.float32 else BF16
    if dtype == BF16 and logits.dtype not in (torch.bfloat16, torch.int16, torch.uint16):
        raise ValueError(f"logits: unsupported dtype {logits.dtype}")
    dev = logits.device
    for t, dt, nm in ((draft_tokens, torch.int32, "draft_tokens"), (p_draft, torch.float32, "p_draft")):
        if t.dtype != dt or t.device != dev or tuple(t.shape) != (B, k) or not t.is_contiguous():
            raise ValueError(f"{nm}: expected a contiguous [{B}, {k}] {dt} tensor on {dev}")
    if out is None:
        out = (torch.empty(B, dtype=torch.int32, device=dev), torch.empty((B, k), dtype=torch.float32, device=dev))
    acc, pt = out
    if acc.dtype != torch.int32 or acc.numel() != B or pt.dtype != torch.float32 or pt.numel() != B * k:
        raise ValueError("out: expected (int32 [B], float32 [B, k])")
    if acc.device != dev or pt.device != dev:
        raise ValueError(f"out: expected tensors on {dev}")
    with torch.cuda.device(dev):  # the entry point runs on the calling thread's current device
        _check(_lib.lacache_accept_length(logits.data_ptr(), dtype, V, draft_tokens.data_ptr(), p_draft.data_ptr(),
                                          B, k, acc.data_ptr(), pt.data_ptr(), _stream(dev.index, stream)),
               "lacache_accept_length")
    return out


def lacache_enable_lsh(c: LaCache, bits: int, hyperplanes, max_candidates: int = 256, stream=None) -> None:
    """hyperplanes: [bits][d] bfloat16 (or int16/uint16 bits) on the cache's device."""
    hp = _vec(hyperplanes, BF16, bits, c.d, c.device, "hyperplanes")
    _check(_lib.lacache_enable_lsh(c.handle, int(bits), hp, int(max_candidates), _stream(c.device, stream)),
           "lacache_enable_lsh")
    c.lsh_bits = int(bits)


def lacache_lookup_lsh(c: LaCache, queries, lookahead_emb, lookahead_tokens, tau_q: float, tau_r: float, k: int,
                       radius: int, out=None, stream=None):
    """Returns (idx int32, score f32, resp_score f32, decision int32, n_cand int32), each [B]."""
    B = queries.shape[0]
    dev = torch.device("cuda", c.device)
    if out is None:
        out = (torch.empty(B, dtype=torch.int32, device=dev), torch.empty(B, dtype=torch.float32, device=dev),
               torch.empty(B, dtype=torch.float32, device=dev), torch.empty(B, dtype=torch.int32, device=dev),
               torch.empty(B, dtype=torch.int32, device=dev))
    for t, dt, nm in zip(out, (torch.int32, torch.float32, torch.float32, torch.int32, torch.int32),
                         ("idx", "score", "resp", "decision", "n_cand")):
        if t.dtype != dt or t.device != dev or t.numel() != B or not t.is_contiguous():
            raise ValueError(f"{nm}: expected a contiguous [{B}] {dt} tensor on {dev}")
    _check(_lib.lacache_lookup_lsh(c.handle, _vec(queries, c.in_dtype, B, c.d, c.device, "queries"),
                                   _vec(lookahead_emb, c.in_dtype, B, c.d, c.device, "lookahead_emb"),
                                   _ints(lookahead_tokens, (B, k), c.device, "lookahead_tokens"), B, float(tau_q),
                                   float(tau_r), int(k), int(radius), *(t.data_ptr() for t in out),
                                   _stream(c.device, stream)), "lacache_lookup_lsh")
    return out


def lacache_export_signatures(c: LaCache, first: int, n: int, stream=None):
    """The stored LSH signatures as int32 bit patterns [n][bits / 32] (view as uint32 on the host)."""
    bits = getattr(c, "lsh_bits", 0)
    if not bits:
        raise ValueError("the LSH index is not enabled")
    sig = torch.empty((n, bits // 32), dtype=torch.int32, device=torch.device("cuda", c.device))
    _check(_lib.lacache_export_signatures(c.handle, first, n, sig.data_ptr(), _stream(c.device, stream)),
           "lacache_export_signatures")
    return sig


def lacache_set_small_batch(c: LaCache, b_small: int) -> None:
    _check(_lib.lacache_set_small_batch(c.handle, b_small), "lacache_set_small_batch")


def lacache_profile(c: LaCache, every) -> None:
    """Time every `every`-th stage-1 launch from now on (True: every launch; False or 0: stop)."""
    n = int(every)  # True -> 1, False -> 0
    _check(_lib.lacache_profile(c.handle, n), "lacache_profile")


def lacache_profile_read(c: LaCache):
    """(total stage-1 milliseconds, number of launches timed) since profiling was enabled or last read."""
    ms, n = ctypes.c_double(0), _i64(0)
    _check(_lib.lacache_profile_read(c.handle, ctypes.byref(ms), ctypes.byref(n)), "lacache_profile_read")
    return ms.value, n.value


def lacache_replay_fallbacks(c: LaCache) -> int:
    """Queries since create whose large-batch group replay did not reproduce their stage-1 score (0 in correct
    operation); synchronises the device."""
    n = _i64(0)
    _check(_lib.lacache_replay_fallbacks(c.handle, ctypes.byref(n)), "lacache_replay_fallbacks")
    return n.value


def raw_library() -> ctypes.CDLL:
    """The loaded C library, for callers that pass raw pointers themselves."""
    return _lib
