"""Seeded synthetic workloads for range-filtered k-NN search.

This module only draws random inputs: base vectors, one numeric attribute per
vector, query vectors and query ranges.  It holds none of the search method's
arithmetic, so both the CPU oracle (test infrastructure) and the HIP library's
callers may use it.

Every workload draws from ``numpy.random.Generator(PCG64(...))`` seeded by
``SeedSequence(seed).spawn(5)``; the five child streams are used, in order, for
the base vectors, the attribute, the query vectors, the query ranges, and a
reserve stream.  Attribute values of every workload are a permutation of
``0..n-1`` (stored as float64), so a query range ``[lo, hi]`` of integer values
selects exactly ``hi - lo + 1`` objects; its selectivity is that count over n.

Workloads (shapes follow the paper's evaluation datasets, which are not
available here; the synthetic mixtures stand in for them):

* ``tiny``  n=10,000, d=32, i.i.d. N(0,1); 100 N(0,1) queries; selectivity
  cycling through 1%, 10%, 50%, 100%; k=10, L=64.
* ``c2``    n=1,000,000, d=128 Gaussian mixture (1,000 centres ~ N(0,I),
  per-point noise 0.3); 10,000 queries from the mixture; selectivity
  log-uniform on [2^-10, 1]; k=10, L in {32, 64, 128}.
* ``c3``    n=1,000,000, d=960 mixture (500 centres, noise 0.5); 1,000 queries;
  log-uniform [2^-10, 1]; k=10, L=128.
* ``c4``    n=10,000,000, d=96 mixture (2,000 centres, noise 0.3), each vector
  normalised to unit length; attribute = rank of the projection onto a fixed
  random unit direction (ranges select spatially coherent slabs); 10,000
  queries; log-uniform [2^-12, 1]; k=10, L=64.
* ``c5``    the c2 base set; 100,000 queries split evenly over the fixed
  selectivities 0.1%, 1%, 10%, 50%, 100%; k=100, L=256.

``n`` and ``nq`` may be overridden to make a smaller workload of the same
structure (used for parity tests the oracle finishes in seconds).

:func:`more_queries` draws further query batches over the same base set from
the reserve stream: a held-out batch of the workload's own selectivity mix
(to check a setting chosen on the main batch), and batches at one fixed
selectivity.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

__all__ = ["Workload", "make", "NAMES", "ranges_for_selectivity", "more_queries"]

NAMES = ("tiny", "c2", "c3", "c4", "c5")


@dataclass
class Workload:
    name: str
    X: np.ndarray          # float32 [n, d], original object order
    attr: np.ndarray       # float64 [n]
    Q: np.ndarray          # float32 [nq, d]
    lo: np.ndarray         # float64 [nq]
    hi: np.ndarray         # float64 [nq]
    sigma: np.ndarray      # float64 [nq], selectivity the range was drawn for
    k: int
    Ls: tuple
    meta: dict = field(default_factory=dict)

    @property
    def n(self) -> int:
        return int(self.X.shape[0])

    @property
    def d(self) -> int:
        return int(self.X.shape[1])

    @property
    def nq(self) -> int:
        return int(self.Q.shape[0])


def _streams(seed: int):
    ss = np.random.SeedSequence(seed).spawn(5)
    return [np.random.Generator(np.random.PCG64(s)) for s in ss]


def ranges_for_selectivity(rng: np.random.Generator, sigma: np.ndarray, n: int):
    """Integer attribute ranges of count ``clamp(round(sigma*n), 1, n)`` placed
    uniformly at random over the value domain ``0..n-1``."""
    sigma = np.asarray(sigma, dtype=np.float64)
    cnt = np.clip(np.rint(sigma * n), 1, n).astype(np.int64)
    start = rng.integers(0, n - cnt + 1)
    lo = start.astype(np.float64)
    hi = (start + cnt - 1).astype(np.float64)
    return lo, hi


def _mixture(rng_base, rng_q, n, nq, d, centres, noise, unit=False):
    C = rng_base.standard_normal((centres, d), dtype=np.float32)
    a = rng_base.integers(0, centres, n)
    X = rng_base.standard_normal((n, d), dtype=np.float32)
    X *= np.float32(noise)
    X += C[a]
    aq = rng_q.integers(0, centres, nq)
    Q = rng_q.standard_normal((nq, d), dtype=np.float32)
    Q *= np.float32(noise)
    Q += C[aq]
    if unit:
        X /= np.linalg.norm(X, axis=1, keepdims=True).astype(np.float32)
        Q /= np.linalg.norm(Q, axis=1, keepdims=True).astype(np.float32)
    return X, Q


def _log_uniform(rng, nq, lo_exp):
    # selectivity 2^(-lo_exp * U), U ~ U(0,1): log-uniform on [2^-lo_exp, 1]
    return np.exp2(-lo_exp * rng.random(nq))


def make(name: str, *, seed: int = 0, n: int | None = None, nq: int | None = None) -> Workload:
    """Build workload ``name`` (one of NAMES), optionally resized."""
    base, ra, rq, rr, _reserve = _streams(seed)
    if name == "tiny":
        n = 10_000 if n is None else n
        nq = 100 if nq is None else nq
        d = 32
        X = base.standard_normal((n, d), dtype=np.float32)
        attr = ra.permutation(n).astype(np.float64)
        Q = rq.standard_normal((nq, d), dtype=np.float32)
        sigma = np.array([0.01, 0.10, 0.50, 1.00])[np.arange(nq) % 4]
        lo, hi = ranges_for_selectivity(rr, sigma, n)
        return Workload(name, X, attr, Q, lo, hi, sigma, 10, (64,),
                        dict(kind="iid-normal", seed=seed))
    if name in ("c2", "c5"):
        n = 1_000_000 if n is None else n
        nq_default = 10_000 if name == "c2" else 100_000
        nq = nq_default if nq is None else nq
        d = 128
        X, Q = _mixture(base, rq, n, nq, d, 1000, 0.3)
        attr = ra.permutation(n).astype(np.float64)
        if name == "c2":
            sigma = _log_uniform(rr, nq, 10.0)
            k, Ls = 10, (32, 64, 128)
        else:
            bands = np.array([0.001, 0.01, 0.10, 0.50, 1.00])
            sigma = bands[np.arange(nq) * len(bands) // nq]
            k, Ls = 100, (256,)
        lo, hi = ranges_for_selectivity(rr, sigma, n)
        return Workload(name, X, attr, Q, lo, hi, sigma, k, Ls,
                        dict(kind="gaussian-mixture", centres=1000, noise=0.3, seed=seed))
    if name == "c3":
        n = 1_000_000 if n is None else n
        nq = 1_000 if nq is None else nq
        d = 960
        X, Q = _mixture(base, rq, n, nq, d, 500, 0.5)
        attr = ra.permutation(n).astype(np.float64)
        sigma = _log_uniform(rr, nq, 10.0)
        lo, hi = ranges_for_selectivity(rr, sigma, n)
        return Workload(name, X, attr, Q, lo, hi, sigma, 10, (128,),
                        dict(kind="gaussian-mixture", centres=500, noise=0.5, seed=seed))
    if name == "c4":
        n = 10_000_000 if n is None else n
        nq = 10_000 if nq is None else nq
        d = 96
        X, Q = _mixture(base, rq, n, nq, d, 2000, 0.3, unit=True)
        w = ra.standard_normal(d)
        w /= np.linalg.norm(w)
        proj = X.astype(np.float64) @ w
        order = np.argsort(proj, kind="stable")
        attr = np.empty(n, dtype=np.float64)
        attr[order] = np.arange(n, dtype=np.float64)
        sigma = _log_uniform(rr, nq, 12.0)
        lo, hi = ranges_for_selectivity(rr, sigma, n)
        return Workload(name, X, attr, Q, lo, hi, sigma, 10, (64,),
                        dict(kind="gaussian-mixture-unit", centres=2000, noise=0.3,
                             attribute="projection-rank", seed=seed))
    raise ValueError(f"unknown workload {name!r}; expected one of {NAMES}")


# the reserve stream's children, by purpose
_PURPOSE = {"held_out": 0, "fixed": 1}
# mixture parameters of the workloads drawn from one (centres, noise, unit length)
_MIXTURE = {"c2": (1000, 0.3, False), "c5": (1000, 0.3, False), "c3": (500, 0.5, False),
            "c4": (2000, 0.3, True)}


def more_queries(w: Workload, purpose: str, nq: int, *, sigma: float | None = None, seed: int = 0):
    """Queries and ranges over the base set of ``w`` (made by :func:`make`
    with the same seed), drawn from a child of the reserve stream that depends
    on ``purpose`` ("held_out" or "fixed") and, for fixed batches, on sigma.
    ``held_out``: the workload's own selectivity distribution; ``fixed``:
    every range of selectivity ``sigma``.  Query vectors come from the same
    mixture (the centres are the base stream's first draw).  Returns
    (Q, lo, hi, sigma array)."""
    if w.name not in _MIXTURE:
        raise ValueError(f"more_queries: {w.name} is not a mixture workload")
    centres, noise, unit = _MIXTURE[w.name]
    ss = np.random.SeedSequence(seed).spawn(5)
    base = np.random.Generator(np.random.PCG64(ss[0]))
    C = base.standard_normal((centres, w.d), dtype=np.float32)
    key = [_PURPOSE[purpose]] + ([] if sigma is None else [int(round(-np.log2(sigma) * 1000))])
    child = np.random.SeedSequence(entropy=ss[4].entropy, spawn_key=tuple(ss[4].spawn_key) + tuple(key))
    rq, rr = [np.random.Generator(np.random.PCG64(c)) for c in child.spawn(2)]
    aq = rq.integers(0, centres, nq)
    Q = rq.standard_normal((nq, w.d), dtype=np.float32)
    Q *= np.float32(noise)
    Q += C[aq]
    if unit:
        Q /= np.linalg.norm(Q, axis=1, keepdims=True).astype(np.float32)
    if purpose == "fixed":
        sig = np.full(nq, float(sigma))
    elif w.name == "c5":
        bands = np.array([0.001, 0.01, 0.10, 0.50, 1.00])
        sig = bands[np.arange(nq) * len(bands) // nq]
    else:
        sig = _log_uniform(rr, nq, 12.0 if w.name == "c4" else 10.0)
    lo, hi = ranges_for_selectivity(rr, sig, w.n)
    return Q, lo, hi, sig
