"""GPU index construction (Sec 6 on the device) against the oracle's
construction: rank order, rows and the candidate array must be identical,
entry for entry.  The cases mirror the host construction's parity tests
(tests/test_build_parity.py) and add the pool widths of the other kernel
instances (ef_c <= 64 and ef_c = 256)."""
import numpy as np
import pytest

import oracle
import paper_2608_16491_amd as F
import workloads

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _compare(X, attr, **params):
    print(f"[gpu] construction n={X.shape[0]} d={X.shape[1]} {params}", flush=True)
    ix = F.Index.build(X, attr, device=0, **params)
    e = ix.export()
    ox = oracle.build(X, attr, **params)
    assert (e["perm"] == ox.perm).all()
    assert (e["attr_sorted"] == ox.attr_sorted).all()
    assert (e["X_rank"] == ox.X_rank).all()
    assert e["ENC"].shape == ox.ENC.shape
    diff = np.argwhere(e["ENC"] != ox.ENC)
    assert len(diff) == 0, f"{len(diff)} entries differ, first at {diff[:3].tolist()}"
    return ix, ox


def test_gpu_build_iid():
    w = workloads.make("tiny", n=4000, nq=1)
    ix, _ = _compare(w.X, w.attr)
    dists, exps, kms = ix.build_stats()
    assert dists > 0 and exps > 0 and kms > 0


def test_gpu_build_mixture_d128():
    w = workloads.make("c2", n=6000, nq=1)
    _compare(w.X, w.attr)


def test_gpu_build_m32_pool256():
    rng = np.random.default_rng(3)
    X = rng.standard_normal((1500, 320)).astype(np.float32)
    attr = rng.permutation(1500).astype(np.float64)
    _compare(X, attr)          # d > 300: m=32, ef_c=256, n_inv=6


def test_gpu_build_duplicate_attributes_and_odd_sizes():
    rng = np.random.default_rng(4)
    X = rng.standard_normal((777, 20)).astype(np.float32)
    attr = rng.integers(0, 50, 777).astype(np.float64)
    _compare(X, attr, m=8, ef_c=24, n_inv=3, patience=5, sib_seeds=4, beta=0.3, gamma=1.0, seed=9)


def test_gpu_build_beta0_and_long_leaves():
    # beta = 0 (fusion off) and leaves of up to 2^9 ranks (several 64-lane
    # batches in the leaf brute force)
    w = workloads.make("tiny", n=3000, nq=1)
    _compare(w.X, w.attr, n_inv=9, beta=0.0)


def test_gpu_build_tiny_n():
    rng = np.random.default_rng(5)
    for n in (1, 2, 3, 17):
        X = rng.standard_normal((n, 4)).astype(np.float32)
        attr = rng.permutation(n).astype(np.float64)
        _compare(X, attr, m=4, ef_c=8, n_inv=0)


def test_gpu_built_index_is_uploaded_and_searches():
    # the device copy the construction leaves behind serves the search
    w = workloads.make("tiny", n=5000, nq=60)
    ix = F.Index.build(w.X, w.attr, device=0)
    ox = oracle.build(w.X, w.attr)
    dev = torch.device("cuda:0")
    ids, ds = F.search(ix, torch.as_tensor(w.Q, device=dev), torch.as_tensor(w.lo, device=dev),
                       torch.as_tensor(w.hi, device=dev), 10, 64)
    torch.cuda.synchronize()
    o_ids, o_d, _ = oracle.search(ox, w.Q, w.lo, w.hi, 10, 64)
    from tests.parity import assert_parity
    assert_parity(ids.cpu().numpy(), ds.cpu().numpy(), o_ids, o_d)
