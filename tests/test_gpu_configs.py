"""GPU parity on the structures of the other benchmark workloads, at sizes the
oracle finishes in seconds: high-dimensional vectors (d = 960, m = 32, the
64-lanes-per-vector path), a correlated attribute (unit vectors, attribute =
rank of a projection, d = 96 -> three chunks per lane, selectivity down to
2^-12), and the fixed-selectivity sweep at k = 100, L = 256.

The index is built by the library's host construction (the oracle's
construction at these dimensions takes minutes); tests/test_build_parity.py
shows the two constructions are identical entry for entry, including d > 300
with m = 32.  Here the index is only the common input of both searches."""
import numpy as np
import pytest

import oracle
import paper_2608_16491_amd as F
import workloads
from tests.parity import assert_parity

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _run(w, k, L, **p):
    ix = F.Index.build(w.X, w.attr).upload(0)
    arr = ix.export()
    ox = oracle.OracleIndex(arr["perm"], arr["attr_sorted"], arr["X_rank"], arr["ENC"])
    dev = torch.device("cuda:0")
    ids, ds, st = F.search(ix, torch.as_tensor(w.Q, device=dev), torch.as_tensor(w.lo, device=dev),
                           torch.as_tensor(w.hi, device=dev), k, L, stats=True, **p)
    torch.cuda.synchronize()
    o_ids, o_d, o_st = oracle.search(ox, w.Q, w.lo, w.hi, k, L, epn=p.get("epn", 16),
                                     epn_frac=p.get("epn_frac", 0.0), epn_max=p.get("epn_max", 0),
                                     B=p.get("budget", 16))
    ids, ds, st = ids.cpu().numpy(), ds.cpu().numpy(), st.cpu().numpy()
    res = assert_parity(ids, ds, o_ids, o_d)
    ok = np.setdiff1d(np.arange(len(ids)), res)
    assert (st[ok, F.STAT_EXPANSIONS] == o_st[ok, oracle.STAT_EXPANSIONS]).all()
    assert (st[ok, F.STAT_SCANNED] == o_st[ok, oracle.STAT_SCANNED]).all()
    return ix, ids


def test_high_dimensional_structure():
    print("[gpu] c3 structure: n=6000 d=960 m=32", flush=True)
    w = workloads.make("c3", n=6000, nq=120)
    ix, _ = _run(w, 10, 128, epn=16, epn_frac=1.0, epn_max=1024)
    assert ix.info()[3] == 32


def test_correlated_attribute_structure():
    print("[gpu] c4 structure: n=40000 d=96 unit vectors, projection attribute", flush=True)
    w = workloads.make("c4", n=40000, nq=300)
    _run(w, 10, 64, epn=16, epn_frac=1.0, epn_max=1024)


def test_selectivity_sweep_structure_k100():
    print("[gpu] c5 structure: n=30000 d=128, k=100 L=256, fixed bands", flush=True)
    w = workloads.make("c5", n=30000, nq=250)
    _run(w, 100, 256, epn=16, epn_frac=1.0, epn_max=1024)
