"""MI355X (gfx950) range-filtered k-NN search: Python binding of ``libfrog.so``.

Argument marshalling only: every step of the search runs in the library's HIP
kernels (see ``include/frog.h`` for the C ABI and the paper passages each call
follows).  PyTorch supplies device memory and the current stream.  There is no
fallback: if the library is missing, :func:`lib` raises.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libfrog.so")

FROG_OK = 0
ERRORS = {-1: "EINVAL", -2: "ENOMEM", -3: "EHIP", -4: "EBADINDEX", -5: "ENOTUPLOADED",
          -6: "EIO", -7: "EUNSUPPORTED", -8: "ENOTPREPARED"}
(STAT_EXPANSIONS, STAT_EN, STAT_DIST, STAT_SCANNED, STAT_ENTRY, STAT_LSTART, STAT_LEND, STAT_LOADED,
 STAT_SCANROWS, STAT_FALLBACK) = range(10)
STAT_N = 10
STORAGE_F32, STORAGE_F16, STORAGE_BF16 = 0, 1, 2
STORAGE = {"fp32": STORAGE_F32, "fp16": STORAGE_F16, "bf16": STORAGE_BF16}

SYMBOLS = (
    "frog_build_params_default", "frog_search_params_default", "frog_build_index",
    "frog_index_from_arrays", "frog_index_export", "frog_index_info", "frog_index_save",
    "frog_index_load", "frog_index_upload", "frog_index_upload_ex", "frog_index_free",
    "frog_build_index_gpu", "frog_index_build_stats", "frog_rank_bounds", "frog_search",
    "frog_search_ex", "frog_search_noalloc", "frog_index_prepare_sample", "frog_bruteforce_filtered",
    "frog_last_error",
)


class FrogError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"frog error {code} ({ERRORS.get(code, '?')}): {msg}")
        self.code = code


class BuildParams(C.Structure):
    _fields_ = [("m", C.c_int), ("ef_c", C.c_int), ("n_inv", C.c_int), ("patience", C.c_int),
                ("sib_seeds", C.c_int), ("num_threads", C.c_int), ("beta", C.c_double),
                ("gamma", C.c_double), ("seed", C.c_uint64)]


class SearchParams(C.Structure):
    _fields_ = [("epn", C.c_int), ("epn_frac", C.c_double), ("epn_max", C.c_int), ("budget", C.c_int),
                ("seed", C.c_uint64), ("query_base", C.c_int64), ("hash_log2", C.c_int),
                ("phase_events", C.c_void_p), ("entry_mode", C.c_int), ("hotspot_mode", C.c_int),
                ("eager_check", C.c_int)]


_lib = None


def lib() -> C.CDLL:
    """Load libfrog.so (built by ``__graft_entry__.build()``); raises if absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise FileNotFoundError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                                "(python -m paper_2608_16491_amd._build)")
    L = C.CDLL(LIB_PATH)
    P = C.c_void_p
    i64, i32 = C.c_int64, C.c_int
    L.frog_last_error.restype = C.c_char_p
    L.frog_last_error.argtypes = []
    L.frog_build_params_default.restype = None
    L.frog_build_params_default.argtypes = [i32, C.POINTER(BuildParams)]
    L.frog_search_params_default.restype = None
    L.frog_search_params_default.argtypes = [C.POINTER(SearchParams)]
    L.frog_build_index.restype = i32
    L.frog_build_index.argtypes = [P, P, i64, i32, C.POINTER(BuildParams), C.POINTER(P)]
    L.frog_index_from_arrays.restype = i32
    L.frog_index_from_arrays.argtypes = [P, P, P, P, i64, i32, i32, i32, C.POINTER(P)]
    L.frog_index_export.restype = i32
    L.frog_index_export.argtypes = [P, P, P, P, P]
    L.frog_index_info.restype = i32
    L.frog_index_info.argtypes = [P, C.POINTER(i64), C.POINTER(i32), C.POINTER(i32), C.POINTER(i32)]
    L.frog_index_save.restype = i32
    L.frog_index_save.argtypes = [P, C.c_char_p]
    L.frog_index_load.restype = i32
    L.frog_index_load.argtypes = [C.c_char_p, C.POINTER(P)]
    L.frog_index_upload.restype = i32
    L.frog_index_upload.argtypes = [P, i32]
    L.frog_index_upload_ex.restype = i32
    L.frog_build_index_gpu.restype = i32
    L.frog_build_index_gpu.argtypes = [P, P, i64, i32, C.POINTER(BuildParams), i32, C.POINTER(P)]
    L.frog_index_build_stats.restype = i32
    L.frog_index_build_stats.argtypes = [P, C.POINTER(i64), C.POINTER(i64), C.POINTER(C.c_double)]
    L.frog_index_upload_ex.argtypes = [P, i32, i32]
    L.frog_index_free.restype = None
    L.frog_index_free.argtypes = [P]
    L.frog_rank_bounds.restype = i32
    L.frog_rank_bounds.argtypes = [P, P, P, i64, P, P]
    L.frog_search.restype = i32
    L.frog_search.argtypes = [P, P, i64, P, P, i32, i32, P, P, P]
    L.frog_search_ex.restype = i32
    L.frog_search_ex.argtypes = [P, P, i64, P, P, i32, i32, C.POINTER(SearchParams), P, P, P, P]
    L.frog_search_noalloc.restype = i32
    L.frog_search_noalloc.argtypes = [P, P, i64, P, P, i32, i32, C.POINTER(SearchParams), P, P, P, P]
    L.frog_index_prepare_sample.restype = i32
    L.frog_index_prepare_sample.argtypes = [P, C.c_uint64]
    L.frog_bruteforce_filtered.restype = i32
    L.frog_bruteforce_filtered.argtypes = [P, P, i64, P, P, i32, P, P, P, P]
    _lib = L
    return L


def _check(rc: int):
    if rc != FROG_OK:
        raise FrogError(rc, lib().frog_last_error().decode(errors="replace"))


def _np(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(C.c_void_p)


def build_params(d: int, **kw) -> BuildParams:
    p = BuildParams()
    lib().frog_build_params_default(d, C.byref(p))
    for k, v in kw.items():
        if v is not None:
            setattr(p, k, v)
    return p


def search_params(**kw) -> SearchParams:
    p = SearchParams()
    lib().frog_search_params_default(C.byref(p))
    for k, v in kw.items():
        if v is not None:
            setattr(p, k, v)
    return p


class Index:
    """Owns a ``frog_index_t`` (host arrays and, after :meth:`upload`, the
    device copy)."""

    def __init__(self, handle: int):
        self._h = C.c_void_p(handle)

    # -- construction
    @classmethod
    def build(cls, X, attr, device=None, **params) -> "Index":
        """Construct the index (Sec 6) on the host, or with device=k on HIP
        device k (same result; the device copy is then already uploaded)."""
        X = _np(X, np.float32)
        attr = _np(attr, np.float64)
        n, d = X.shape
        assert attr.shape == (n,)
        p = build_params(d, **params)
        h = C.c_void_p()
        if device is None:
            _check(lib().frog_build_index(_ptr(X), _ptr(attr), n, d, C.byref(p), C.byref(h)))
            return cls(h.value)
        _check(lib().frog_build_index_gpu(_ptr(X), _ptr(attr), n, d, C.byref(p), int(device), C.byref(h)))
        ix = cls(h.value)
        ix.storage = "fp32"
        return ix

    def build_stats(self):
        """(distances, sibling-search expansions, kernel milliseconds) of a
        GPU construction."""
        a, b, t = C.c_int64(), C.c_int64(), C.c_double()
        _check(lib().frog_index_build_stats(self._h, C.byref(a), C.byref(b), C.byref(t)))
        return a.value, b.value, t.value

    @classmethod
    def from_arrays(cls, X_rank, attr_sorted, perm, ENC) -> "Index":
        X_rank = _np(X_rank, np.float32)
        attr_sorted = _np(attr_sorted, np.float64)
        perm = _np(perm, np.int32)
        ENC = _np(ENC, np.int32)
        n, d = X_rank.shape
        n2, H, m = ENC.shape
        assert n2 == n and attr_sorted.shape == (n,) and perm.shape == (n,)
        h = C.c_void_p()
        _check(lib().frog_index_from_arrays(_ptr(X_rank), _ptr(attr_sorted), _ptr(perm), _ptr(ENC),
                                            n, d, H, m, C.byref(h)))
        return cls(h.value)

    @classmethod
    def load(cls, path: str) -> "Index":
        h = C.c_void_p()
        _check(lib().frog_index_load(os.fsencode(path), C.byref(h)))
        return cls(h.value)

    def save(self, path: str):
        _check(lib().frog_index_save(self._h, os.fsencode(path)))

    def info(self):
        n, d, H, m = C.c_int64(), C.c_int(), C.c_int(), C.c_int()
        _check(lib().frog_index_info(self._h, C.byref(n), C.byref(d), C.byref(H), C.byref(m)))
        return n.value, d.value, H.value, m.value

    def export(self):
        n, d, H, m = self.info()
        X = np.empty((n, d), np.float32)
        a = np.empty(n, np.float64)
        p = np.empty(n, np.int32)
        E = np.empty((n, H, m), np.int32)
        _check(lib().frog_index_export(self._h, _ptr(X), _ptr(a), _ptr(p), _ptr(E)))
        return dict(X_rank=X, attr_sorted=a, perm=p, ENC=E)

    def upload(self, device: int = 0, storage: str = "fp32") -> "Index":
        """Copy to `device` with rows stored as "fp32", "fp16" or "bf16" (16-bit
        rows rounded to nearest even; the search is then exact over the
        rounded rows)."""
        if storage not in STORAGE:
            raise ValueError(f"storage {storage!r}: one of {sorted(STORAGE)}")
        if storage == "fp32":
            _check(lib().frog_index_upload(self._h, device))
        else:
            _check(lib().frog_index_upload_ex(self._h, device, STORAGE[storage]))
        self.storage = storage
        self._prepared = set()
        return self

    def prepare_sample(self, seed: int = 0) -> "Index":
        """Build the shared entry sample of `seed` on the device (entry_mode 1;
        synchronous, idempotent)."""
        seed = int(seed) & 0xFFFFFFFFFFFFFFFF
        _check(lib().frog_index_prepare_sample(self._h, C.c_uint64(seed)))
        self._prepared = getattr(self, "_prepared", set()) | {seed}
        return self

    def free(self):
        if self._h is not None and self._h.value:
            lib().frog_index_free(self._h)
        self._h = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass

    @property
    def handle(self):
        return self._h


# ------------------------------------------------------------------ device calls

def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return C.c_void_p(s.cuda_stream)


def _dev(t, dtype):
    import torch
    assert t.is_cuda and t.dtype == dtype and t.is_contiguous(), (t.device, t.dtype)
    return C.c_void_p(t.data_ptr())


def rank_bounds(index: Index, lo, hi, stream=None):
    import torch
    nq = lo.shape[0]
    lr = torch.empty((nq, 2), dtype=torch.int32, device=lo.device)
    _check(lib().frog_rank_bounds(index.handle, _dev(lo, torch.float64), _dev(hi, torch.float64), nq,
                                  _dev(lr, torch.int32), _stream(stream)))
    return lr


def search(index: Index, Q, lo, hi, k: int, L: int, *, stats: bool = False, stream=None, out=None,
           **params):
    """FROGSearch for a batch: Q [nq, d] float32, lo/hi [nq] float64, all on
    the index's device.  Returns (ids int32 [nq, k], dists float32 [nq, k]) and,
    with stats=True, the per-query statistics int32 [nq, STAT_N].  Keyword params:
    epn, epn_frac, epn_max, budget, seed, query_base, hash_log2, entry_mode,
    hotspot_mode, eager_check, and events (three torch.cuda.Event recorded before the search kernels,
    after the entry-point kernels and after the last kernel)."""
    import torch
    nq = Q.shape[0]
    if out is None:
        ids = torch.empty((nq, k), dtype=torch.int32, device=Q.device)
        ds = torch.empty((nq, k), dtype=torch.float32, device=Q.device)
    else:
        ids, ds = out
    st = torch.empty((nq, STAT_N), dtype=torch.int32, device=Q.device) if stats else None
    events = params.pop("events", None)
    p = search_params(**params)
    if p.entry_mode == 1 and p.seed not in getattr(index, "_prepared", ()):
        # the sample's level lists are built once per seed, before the search
        index.prepare_sample(p.seed)
    if events is not None:
        # three torch.cuda.Event(enable_timing=True): before the entry-point
        # kernel, between the kernels, after the traversal kernel
        ev_arr = (C.c_void_p * 3)(*[C.c_void_p(e.cuda_event) for e in events])
        p.phase_events = C.cast(ev_arr, C.c_void_p)
    _check(lib().frog_search_ex(index.handle, _dev(Q, torch.float32), nq, _dev(lo, torch.float64),
                                _dev(hi, torch.float64), k, L, C.byref(p), _dev(ids, torch.int32),
                                _dev(ds, torch.float32), None if st is None else _dev(st, torch.int32),
                                _stream(stream)))
    return (ids, ds, st) if stats else (ids, ds)


def bruteforce(index: Index, Q, lo, hi, k: int, stream=None):
    """Exact filtered k-NN on the GPU.  Returns (ids, dists, certified)."""
    import torch
    nq = Q.shape[0]
    ids = torch.empty((nq, k), dtype=torch.int32, device=Q.device)
    ds = torch.empty((nq, k), dtype=torch.float32, device=Q.device)
    cert = torch.empty((nq,), dtype=torch.int32, device=Q.device)
    _check(lib().frog_bruteforce_filtered(index.handle, _dev(Q, torch.float32), nq, _dev(lo, torch.float64),
                                          _dev(hi, torch.float64), k, _dev(ids, torch.int32),
                                          _dev(ds, torch.float32), _dev(cert, torch.int32), _stream(stream)))
    return ids, ds, cert
