"""The correlated-attribute workload at full size: n = 10,000,000 unit vectors,
d = 96, attribute = rank of the projection onto a fixed direction (ranges
select spatially coherent slabs), 10,000 queries with selectivity
log-uniform in [2^-12, 1], k = 10, L = 64.

The index is built on the GPU (the host construction would take minutes at
this size; the two are identical, tests/test_gpu_build.py and the 1M test).
Sampled rows are recomputed by the oracle one by one on the same index
arrays; every row is checked for the properties that hold at any size, and
the exact brute force gives the recall of a sample."""
import time

import numpy as np
import pytest

import oracle
import paper_2608_16491_amd as F
import workloads
from tests.parity import assert_parity

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

K, L = 10, 64


@pytest.fixture(scope="module")
def c4():
    print("[gpu] full-size c4: generating n=10M d=96", flush=True)
    w = workloads.make("c4")
    t0 = time.time()
    ix = F.Index.build(w.X, w.attr, device=0)
    n, d, H, m = ix.info()
    print(f"[gpu] full-size c4: GPU construction {time.time() - t0:.1f}s, H={H} m={m}, "
          f"kernels {ix.build_stats()[2] / 1e3:.1f}s", flush=True)
    arr = ix.export()
    ox = oracle.OracleIndex(arr["perm"], arr["attr_sorted"], arr["X_rank"], arr["ENC"])
    dev = torch.device("cuda:0")
    d = dict(Q=torch.as_tensor(w.Q, device=dev), lo=torch.as_tensor(w.lo, device=dev),
             hi=torch.as_tensor(w.hi, device=dev))
    yield w, ix, ox, d
    ix.free()


@pytest.mark.timeout(900)
@pytest.mark.parametrize("mode", [1, 0])
def test_c4_full_size_sampled_rows_and_properties(c4, mode):
    w, ix, ox, d = c4
    p = dict(epn=16, epn_frac=1.0, epn_max=2048, budget=16, entry_mode=mode, hash_log2=10)
    t0 = time.time()
    ids, ds = F.search(ix, d["Q"], d["lo"], d["hi"], K, L, **p)
    torch.cuda.synchronize()
    print(f"[gpu] c4 search mode {mode}: {time.time() - t0:.3f}s (first call)", flush=True)
    ids, ds = ids.cpu().numpy(), ds.cpu().numpy()
    rng = np.random.default_rng(21)
    sample = np.sort(rng.choice(w.nq, 200, replace=False))
    o_ids, o_d, _ = oracle.search(ox, w.Q[sample], w.lo[sample], w.hi[sample], K, L, qidx=sample,
                                  epn=16, epn_frac=1.0, epn_max=2048, B=16, entry_mode=mode)
    assert_parity(ids[sample], ds[sample], o_ids, o_d, max_residual=1)
    # every row: min(k, cnt) results, in range, distinct, ascending
    cnt = (w.hi - w.lo + 1).astype(np.int64)
    valid = ids >= 0
    assert (valid.sum(1) == np.minimum(K, cnt)).all()
    a = w.attr[np.where(valid, ids, 0)]
    assert ((a >= w.lo[:, None]) & (a <= w.hi[:, None]) | ~valid).all()
    assert (np.diff(np.where(valid, ds, np.inf), axis=1) >= 0).all()
    # recall of the sample against the exact filtered k-NN
    sel = torch.as_tensor(sample, device=d["Q"].device)
    gt, _, cert = F.bruteforce(ix, d["Q"][sel].contiguous(), d["lo"][sel].contiguous(),
                               d["hi"][sel].contiguous(), K)
    torch.cuda.synchronize()
    gt = gt.cpu().numpy()
    assert cert.cpu().numpy().all()
    hits = [len(set(ids[q][ids[q] >= 0]) & set(gt[i][gt[i] >= 0])) / max(1, (gt[i] >= 0).sum())
            for i, q in enumerate(sample)]
    print(f"[gpu] c4 mode {mode}: recall@10 of the sample {np.mean(hits):.4f}", flush=True)
    assert np.mean(hits) > 0.5
