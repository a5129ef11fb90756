"""GPU exhaustive filtered k-NN (Def. 2) against the oracle's exhaustive
search, through the C ABI."""
import numpy as np
import pytest

import oracle
import paper_2608_16491_amd as F
import workloads
from tests.parity import assert_parity

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _cuda(a, dtype):
    return torch.as_tensor(np.ascontiguousarray(a)).to(dtype=dtype, device="cuda")


def _run(X, attr, Q, lo, hi, k):
    perm = np.argsort(attr, kind="stable").astype(np.int32)
    srt = attr[perm]
    Xr = X[perm]
    n, d = X.shape
    ENC = -np.ones((n, 1, 1), np.int32)
    ix = F.Index.from_arrays(Xr, srt, perm, ENC).upload(0)
    ids, ds, cert = F.bruteforce(ix, _cuda(Q, torch.float32), _cuda(lo, torch.float64),
                                 _cuda(hi, torch.float64), k)
    torch.cuda.synchronize()
    o_ids, o_d = oracle.exact(Xr, srt, perm, Q, lo, hi, k)
    return ids.cpu().numpy(), ds.cpu().numpy(), cert.cpu().numpy(), o_ids, o_d


def test_bruteforce_tiny():
    print("[gpu] bruteforce tiny", flush=True)
    w = workloads.make("tiny")
    ids, ds, cert, o_ids, o_d = _run(w.X, w.attr, w.Q, w.lo, w.hi, 10)
    assert (cert == 1).all()
    assert_parity(ids, ds, o_ids, o_d, max_residual=0)


@pytest.mark.parametrize("k", [1, 10, 100])
def test_bruteforce_mixture(k):
    print(f"[gpu] bruteforce mixture k={k}", flush=True)
    w = workloads.make("c2", n=40000, nq=200)
    ids, ds, cert, o_ids, o_d = _run(w.X, w.attr, w.Q, w.lo, w.hi, k)
    assert np.isin(cert, (1, 2)).all() and (cert == 1).mean() > 0.99
    assert_parity(ids, ds, o_ids, o_d, max_residual=0)


@pytest.mark.parametrize("d", [200, 1030])
def test_bruteforce_wide_rows(d):
    # rows wider than 128 floats take the chunk loop with the query read per
    # chunk (d = 200: 14 steps of 16 dimensions; d = 1030: 66 steps)
    print(f"[gpu] bruteforce wide rows d={d}", flush=True)
    rng = np.random.default_rng(d)
    n, nq = 3000, 48
    X = rng.standard_normal((n, d)).astype(np.float32)
    attr = rng.permutation(n).astype(np.float64)
    Q = rng.standard_normal((nq, d)).astype(np.float32)
    sig = np.array([0.01, 0.1, 0.5, 1.0])[np.arange(nq) % 4]
    lo, hi = workloads.ranges_for_selectivity(rng, sig, n)
    ids, ds, cert, o_ids, o_d = _run(X, attr, Q, lo, hi, 10)
    assert np.isin(cert, (1, 2)).all()
    assert_parity(ids, ds, o_ids, o_d, max_residual=0)


def test_bruteforce_edges():
    rng = np.random.default_rng(1)
    n, d = 2000, 40
    X = rng.standard_normal((n, d)).astype(np.float32)
    attr = rng.integers(0, 300, n).astype(np.float64)      # duplicate attribute values
    Q = rng.standard_normal((9, d)).astype(np.float32)
    lo = np.array([0, 5, np.nan, 7, 299, 100, 50, -5, 10], np.float64)
    hi = np.array([299, 5, 3, 2, 400, 100.5, 60, 1e9, 10], np.float64)
    ids, ds, cert, o_ids, o_d = _run(X, attr, Q, lo, hi, 25)
    assert (cert == 1).all()
    assert_parity(ids, ds, o_ids, o_d, max_residual=0)
    assert (ids[2] == -1).all() and (ids[3] == -1).all()


@pytest.mark.parametrize("k", [1, 10, 100, 256])
def test_bruteforce_uncertified_rows_are_exact(k):
    # Vectors with large norms close to each other (coordinates 1000 +- 0.01):
    # the fp32 approximation |q|^2 + |x|^2 - 2 q.x errs by ~u |x|^2, far more
    # than the gaps between distances, so the margin test certifies almost
    # nothing and the rows come from the exhaustive exact pass.  A tenth of
    # the vectors are duplicates of others (exact ties, broken by rank).  The
    # coordinates are multiples of the fp32 ulp at 1000, so every fp64 sum is
    # exact and both sides agree bit for bit.
    print(f"[gpu] bruteforce, uncertified rows, k={k}", flush=True)
    rng = np.random.default_rng(3)
    n, d, nq = 20000, 32, 48
    X = (1000.0 + 0.01 * rng.standard_normal((n, d))).astype(np.float32)
    src = rng.choice(n, 2000, replace=False)
    X[src[1000:]] = X[src[:1000]]
    attr = rng.permutation(n).astype(np.float64)
    Q = (1000.0 + 0.01 * rng.standard_normal((nq, d))).astype(np.float32)
    cnt = np.array([n, 1, 7, 300, 4095, 4096, 4097, 9000] * (nq // 8))
    lo = rng.integers(0, n - cnt + 1).astype(np.float64)
    hi = lo + cnt - 1
    ids, ds, cert, o_ids, o_d = _run(X, attr, Q, lo, hi, k)
    assert np.isin(cert, (1, 2)).all() and (cert == 2).sum() >= nq // 2
    assert_parity(ids, ds, o_ids, o_d, max_residual=0)
