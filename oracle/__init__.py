"""CPU oracle for FROG range-filtered k-NN search — TEST INFRASTRUCTURE ONLY.

A plain, slow restatement of the method (arxiv 2608.16491), written in C
(``frog_oracle.c``) and driven from here through ctypes.  Only the tests, the
package's ``smoke()`` and the benchmark's CPU-baseline leg may import this
module.  It shares no code with the HIP library (``paper_2608_16491_amd``) and
never imports it.

Functions and the passages of the paper they follow:

* :func:`dist`           squared L2 distance (Sec 2.1), fp64 accumulation
* :func:`rank_bounds`    attribute range -> rank interval (Sec 4)
* :func:`num_layers`, :func:`segment`   segment-tree geometry (Sec 4, Alg 3)
* :func:`hotspot`        HotspotLocalization (Alg 3, Eq. endcondition)
* :func:`entry_points`   entry-point sampling (Alg 2), stratified per query
* :func:`entry_points_shared`  the same with a rank priority shared by all queries
* :func:`en_ident`       ENIdentification (Alg 4)
* :func:`search`         FROGSearch (Alg 2) with an exact visited set
* :func:`exact`          exhaustive filtered k-NN (Def. 2)
* :func:`build`          index construction (Sec 6, Eq. fusion-distance, Alg 1)
* :func:`closure`        vertices reachable from the entry set through EN(.)

The readings taken where the paper is silent are listed at the top of
``frog_oracle.c``.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "frog_oracle.c")
_LIB = os.path.join(_HERE, "libfrog_oracle.so")

# column meaning of the per-query statistics returned by search()
STAT_EXPANSIONS, STAT_EN, STAT_DIST, STAT_SCANNED, STAT_ENTRY, STAT_LS, STAT_LE = range(7)
NSTAT = 8

_lib = None


def compile_oracle(force: bool = False) -> str:
    """Compile frog_oracle.c into libfrog_oracle.so with gcc (no FMA
    contraction, no fast-math: the arithmetic is exactly as written)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.check_call([
            "gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
            "-ffp-contract=off", "-fno-fast-math", "-Wall", "-Wno-unused-function",
            "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    compile_oracle()
    _lib = configure(C.CDLL(_LIB))
    return _lib


def configure(lib):
    """Declare the C signatures on a loaded oracle library."""
    P = C.c_void_p
    i64, i32, f64, u64 = C.c_int64, C.c_int, C.c_double, C.c_uint64
    lib.fo_dist.restype = C.c_float
    lib.fo_dist.argtypes = [P, P, i32]
    lib.fo_splitmix64.restype = u64
    lib.fo_splitmix64.argtypes = [u64]
    lib.fo_num_layers.restype = i32
    lib.fo_num_layers.argtypes = [i64, i32]
    lib.fo_segment.restype = None
    lib.fo_segment.argtypes = [i64, i32, i64, P, P]
    lib.fo_rank_bounds.restype = None
    lib.fo_rank_bounds.argtypes = [P, i64, f64, f64, P, P]
    lib.fo_hotspot.restype = None
    lib.fo_hotspot.argtypes = [i64, i64, i32, i64, P, P]
    lib.fo_entry_points.restype = i64
    lib.fo_entry_points.argtypes = [i64, i64, i64, u64, u64, P]
    lib.fo_entry_count.restype = i64
    lib.fo_entry_count.argtypes = [i64, i32, f64, i32]
    lib.fo_reduce.restype = u64
    lib.fo_reduce.argtypes = [u64, u64]
    lib.fo_en_ident.restype = i32
    lib.fo_en_ident.argtypes = [P, i32, i32, i64, i64, i64, i32, i32, i32, P, P]
    lib.fo_search_batch.restype = i32
    lib.fo_search_batch.argtypes = [P, P, P, P, i64, i32, i32, i32, P, P, P, i64, P,
                                    i32, i32, i32, f64, i32, i32, u64, i32, i32, i32, P, P, P, i32]
    lib.fo_entry_priority.restype = C.c_uint32
    lib.fo_entry_priority.argtypes = [u64, i64]
    lib.fo_entry_threshold.restype = u64
    lib.fo_entry_threshold.argtypes = [i64, i64]
    lib.fo_entry_points_shared.restype = i64
    lib.fo_entry_points_shared.argtypes = [i64, i64, i64, u64, P]
    lib.fo_exact_batch.restype = i32
    lib.fo_exact_batch.argtypes = [P, P, P, i64, i32, P, P, P, i64, i32, P, P, i32]
    lib.fo_fusion.restype = f64
    lib.fo_fusion.argtypes = [C.c_float, i64, i64, i64, f64, f64]
    lib.fo_rank_order.restype = i32
    lib.fo_rank_order.argtypes = [P, i64, P, P]
    lib.fo_build.restype = i32
    lib.fo_build.argtypes = [P, P, i64, i32, i32, i32, i32, i32, i32, f64, f64, u64, i32,
                             P, P, P, P]
    lib.fo_rng_prune_list.restype = i32
    lib.fo_rng_prune_list.argtypes = [P, i32, P, P, i32, i32, P]
    lib.fo_sibling_search_list.restype = i32
    lib.fo_sibling_search_list.argtypes = [P, i64, i32, P, i32, P, i64, i64, P, i32, i32, i32, P, P, P]
    lib.fo_closure.restype = i64
    lib.fo_closure.argtypes = [P, i32, i32, i64, i64, i64, i32, i32, i32, P, i64, P]
    return lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(C.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def default_threads() -> int:
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        return os.cpu_count() or 1


# ---------------------------------------------------------------- primitives

def dist(a, b) -> np.float32:
    a = _c(a, np.float32)
    b = _c(b, np.float32)
    assert a.shape == b.shape and a.ndim == 1
    return np.float32(_load().fo_dist(_p(a), _p(b), a.shape[0]))


def splitmix64(x: int) -> int:
    return int(_load().fo_splitmix64(C.c_uint64(x & 0xFFFFFFFFFFFFFFFF)))


def num_layers(n: int, n_inv: int) -> int:
    return int(_load().fo_num_layers(n, n_inv))


def segment(n: int, h: int, p: int):
    s = C.c_int64()
    e = C.c_int64()
    _load().fo_segment(n, h, p, C.byref(s), C.byref(e))
    return s.value, e.value


def rank_bounds(attr_sorted, lo: float, hi: float):
    a = _c(attr_sorted, np.float64)
    l = C.c_int64()
    r = C.c_int64()
    _load().fo_rank_bounds(_p(a), a.shape[0], float(lo), float(hi), C.byref(l), C.byref(r))
    return l.value, r.value


def hotspot(l: int, r: int, H: int, n: int):
    Ls = C.c_int()
    Le = C.c_int()
    _load().fo_hotspot(l, r, H, n, C.byref(Ls), C.byref(Le))
    return Ls.value, Le.value


def entry_points(l: int, r: int, epn: int, seed: int, qi: int) -> np.ndarray:
    cnt = max(0, r - l + 1)
    out = np.empty(max(1, min(cnt, epn)), dtype=np.int32)
    k = _load().fo_entry_points(l, r, epn, seed, qi, _p(out))
    return out[:k].copy()


def entry_priority(seed: int, i: int) -> int:
    return int(_load().fo_entry_priority(C.c_uint64(seed & 0xFFFFFFFFFFFFFFFF), i))


def entry_threshold(cnt: int, E: int) -> int:
    return int(_load().fo_entry_threshold(cnt, E))


def entry_points_shared(l: int, r: int, E: int, seed: int) -> np.ndarray:
    """Ranks i of [l, r] whose shared priority is below the threshold for E
    expected entry points."""
    cnt = max(0, r - l + 1)
    out = np.empty(max(1, cnt), dtype=np.int32)
    k = _load().fo_entry_points_shared(l, r, E, C.c_uint64(seed & 0xFFFFFFFFFFFFFFFF), _p(out))
    return out[:k].copy()


def en_ident(ENC: np.ndarray, u: int, l: int, r: int, Ls: int, Le: int, B: int):
    """ENC is [n, H, m] int32.  Returns (EN ids, ENC entries scanned)."""
    E = _c(ENC, np.int32)
    n, H, m = E.shape
    out = np.empty(max(B, 1), dtype=np.int32)
    scanned = C.c_int64(0)
    c = _load().fo_en_ident(_p(E), H, m, u, l, r, Ls, Le, B, _p(out), C.byref(scanned))
    return out[:c].copy(), scanned.value


def fusion(d2: float, ru: int, rv: int, seglen: int, beta: float, gamma: float) -> float:
    return float(_load().fo_fusion(C.c_float(d2), ru, rv, seglen, beta, gamma))


# ---------------------------------------------------------------- index

@dataclass
class OracleIndex:
    perm: np.ndarray         # int32 [n]   rank -> original id
    attr_sorted: np.ndarray  # float64 [n]
    X_rank: np.ndarray       # float32 [n, d] rows in rank order
    ENC: np.ndarray          # int32 [n, H, m]

    @property
    def n(self):
        return self.ENC.shape[0]

    @property
    def H(self):
        return self.ENC.shape[1]

    @property
    def m(self):
        return self.ENC.shape[2]

    @property
    def d(self):
        return self.X_rank.shape[1]


def default_build_params(d: int) -> dict:
    """Paper defaults (Sec 8.1.4): m=16, ef_c=128, n_inv=7 for d <= 300; m=32,
    ef_c=256, n_inv=6 above; beta=0.2, gamma=0.5, patience=30."""
    if d <= 300:
        return dict(m=16, ef_c=128, n_inv=7, patience=30, sib_seeds=16, beta=0.2, gamma=0.5, seed=0)
    return dict(m=32, ef_c=256, n_inv=6, patience=30, sib_seeds=16, beta=0.2, gamma=0.5, seed=0)


def build(X, attr, *, m=None, ef_c=None, n_inv=None, patience=None, sib_seeds=None,
          beta=None, gamma=None, seed=None, threads=None) -> OracleIndex:
    X = _c(X, np.float32)
    attr = _c(attr, np.float64)
    n, d = X.shape
    p = default_build_params(d)
    for key, val in dict(m=m, ef_c=ef_c, n_inv=n_inv, patience=patience, sib_seeds=sib_seeds,
                         beta=beta, gamma=gamma, seed=seed).items():
        if val is not None:
            p[key] = val
    H = num_layers(n, p["n_inv"])
    perm = np.empty(n, np.int32)
    attr_sorted = np.empty(n, np.float64)
    X_rank = np.empty((n, d), np.float32)
    ENC = np.empty((n, H, p["m"]), np.int32)
    rc = _load().fo_build(_p(X), _p(attr), n, d, p["m"], p["ef_c"], p["n_inv"], p["patience"],
                          p["sib_seeds"], p["beta"], p["gamma"], p["seed"],
                          threads or default_threads(), _p(perm), _p(attr_sorted), _p(X_rank), _p(ENC))
    if rc < 0:
        raise RuntimeError(f"oracle build failed ({rc})")
    assert rc == H
    return OracleIndex(perm, attr_sorted, X_rank, ENC)


def rng_prune(X, ids, dists, m: int) -> np.ndarray:
    """The construction's RNG prune (Sec 6.1, alpha = 1) of candidates given
    by rank `ids` (rows of X) with their squared distances to the vertex,
    ascending by (distance, id).  Returns the m-entry temporary-PG row (-1
    padded)."""
    X = _c(X, np.float32)
    ids = _c(ids, np.int32)
    dists = _c(dists, np.float32)
    out = np.full(m, -1, np.int32)
    rc = _load().fo_rng_prune_list(_p(X), X.shape[1], _p(ids), _p(dists), ids.shape[0], m, _p(out))
    if rc < 0:
        raise MemoryError("oracle rng_prune: allocation failed")
    return out


def sibling_search(X, PG, xq, ts: int, te: int, seeds, ef: int, patience: int):
    """The construction's greedy search (Alg 1 with the patience stop of Sec
    6.2.2) for the vector xq over the temporary PG (int32 [n, m], -1 empty)
    restricted to ranks [ts, te], from the given seed ranks.  Returns (the m
    nearest found, their squared distances, expansions)."""
    X = _c(X, np.float32)
    PG = _c(PG, np.int32)
    xq = _c(xq, np.float32)
    seeds = _c(seeds, np.int32)
    n, m = PG.shape
    res = np.full(m, -1, np.int32)
    resd = np.full(m, np.inf, np.float32)
    nexp = C.c_int64(0)
    rc = _load().fo_sibling_search_list(_p(X), n, X.shape[1], _p(PG), m, _p(xq), ts, te, _p(seeds),
                                        seeds.shape[0], ef, patience, _p(res), _p(resd), C.byref(nexp))
    if rc < 0:
        raise MemoryError("oracle sibling_search: allocation failed")
    return res[:rc].copy(), resd[:rc].copy(), nexp.value


# ---------------------------------------------------------------- search

def entry_count(cnt: int, epn: int, epn_frac: float = 0.0, epn_max: int = 0) -> int:
    return int(_load().fo_entry_count(cnt, epn, epn_frac, epn_max))


def search(ix: OracleIndex, Q, lo, hi, k: int, L: int, *, epn: int = 16, epn_frac: float = 0.0,
           epn_max: int = 0, B: int = 16, seed: int = 0, entry_mode: int = 0, hot_mode: int = 0,
           eager: bool = False, qidx=None, threads=None, rank_ids: bool = False):
    """FROGSearch for every query.  Returns (ids int32 [nq,k] original ids or
    ranks, dists float32 [nq,k], stats int64 [nq,8]).  The entry-point count
    is epn, or clamp(ceil(epn_frac * cnt), epn, epn_max) when epn_frac > 0;
    entry_mode 0 draws them stratified per query, 1 from the shared-priority
    sample (that count is then the expected size).  Ablations (Sec 8.2.3):
    hot_mode 1 scans layers L_start..H-1, 2 all layers; eager moves the
    visited check into ENIdentification."""
    Q = _c(Q, np.float32)
    lo = _c(lo, np.float64)
    hi = _c(hi, np.float64)
    nq = Q.shape[0]
    assert Q.shape[1] == ix.d
    ids = np.empty((nq, k), np.int32)
    ds = np.empty((nq, k), np.float32)
    st = np.zeros((nq, NSTAT), np.int64)
    qi = None if qidx is None else _c(qidx, np.int64)
    ENC = _c(ix.ENC, np.int32)
    rc = _load().fo_search_batch(
        _p(ix.X_rank), _p(ENC), _p(ix.attr_sorted), None if rank_ids else _p(ix.perm),
        ix.n, ix.d, ix.H, ix.m, _p(Q), _p(lo), _p(hi), nq,
        None if qi is None else _p(qi), k, L, epn, epn_frac, epn_max, B, seed, entry_mode, hot_mode, int(eager),
        _p(ids), _p(ds), _p(st),
        threads or default_threads())
    if rc:
        raise MemoryError("oracle search: allocation failed")
    return ids, ds, st


def exact(X_rank, attr_sorted, perm, Q, lo, hi, k: int, *, threads=None, rank_ids: bool = False):
    """Exhaustive filtered k-NN.  Returns (ids [nq,k], dists [nq,k])."""
    X_rank = _c(X_rank, np.float32)
    attr_sorted = _c(attr_sorted, np.float64)
    Q = _c(Q, np.float32)
    lo = _c(lo, np.float64)
    hi = _c(hi, np.float64)
    nq = Q.shape[0]
    n, d = X_rank.shape
    ids = np.empty((nq, k), np.int32)
    ds = np.empty((nq, k), np.float32)
    pm = None if (rank_ids or perm is None) else _p(_c(perm, np.int32))
    rc = _load().fo_exact_batch(_p(X_rank), _p(attr_sorted), pm, n, d, _p(Q), _p(lo), _p(hi),
                                nq, k, _p(ids), _p(ds), threads or default_threads())
    if rc:
        raise MemoryError("oracle exact: allocation failed")
    return ids, ds


def closure(ix: OracleIndex, l: int, r: int, Ls: int, Le: int, B: int, entry) -> np.ndarray:
    """Boolean mask of the vertices reachable from `entry` through EN(.)."""
    entry = _c(entry, np.int32)
    reach = np.zeros(ix.n, np.uint8)
    ENC = _c(ix.ENC, np.int32)
    _load().fo_closure(_p(ENC), ix.H, ix.m, ix.n, l, r, Ls, Le, B, _p(entry), entry.shape[0], _p(reach))
    return reach.astype(bool)
