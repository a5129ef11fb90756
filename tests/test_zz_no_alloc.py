"""frog_search_noalloc, the entry point for callers that cannot allocate,
against frog_search_ex through the C ABI: identical ids, bit-identical
distances and identical statistics, on two calls in a row on the shared
scratch array (the second with fewer queries, so the array holds the first
call's leftovers), in both entry modes; a call needing more than the array
holds is refused before anything is enqueued."""
import ctypes as C

import numpy as np
import pytest

import paper_2608_16491_amd as F
import workloads

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

# statistics columns that depend on the tiles the planning forms (bucket
# order follows atomic arrival): the scan's row counts
TILE_COLUMNS = (F.STAT_SCANROWS, F.STAT_FALLBACK)


def _ptr(t):
    return C.c_void_p(t.data_ptr())


def _call(fn, ix, Q, lo, hi, k, L, p):
    nq = Q.shape[0]
    ids = torch.full((nq, k), -7, dtype=torch.int32, device="cuda")
    ds = torch.full((nq, k), -7.0, dtype=torch.float32, device="cuda")
    st = torch.full((nq, F.STAT_N), -7, dtype=torch.int32, device="cuda")
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    rc = fn(ix.handle, _ptr(Q), nq, _ptr(lo), _ptr(hi), k, L, C.byref(p), _ptr(ids), _ptr(ds), _ptr(st), stream)
    torch.cuda.synchronize()
    return rc, ids.cpu().numpy(), ds.cpu().numpy(), st.cpu().numpy()


@pytest.fixture(scope="module")
def case():
    print("[gpu] no-alloc entry point: mixture n=30000 d=128 nq=900", flush=True)
    w = workloads.make("c2", n=30000, nq=900)
    ix = F.Index.build(w.X, w.attr).upload(0)
    ix.prepare_sample(0)
    dev = torch.device("cuda:0")
    return ix, torch.as_tensor(w.Q, device=dev), torch.as_tensor(w.lo, device=dev), torch.as_tensor(w.hi, device=dev)


@pytest.mark.parametrize("mode,L,emax", [(0, 32, 2560), (1, 32, 2560), (1, 100, 1500), (0, 200, 700)])
def test_noalloc_equals_search_ex_two_calls(case, mode, L, emax):
    ix, Q, lo, hi = case
    lib = F.lib()
    p = F.search_params(entry_mode=mode, epn=16, epn_frac=1.0, epn_max=emax, budget=16)
    for nq in (900, 211):   # the second call is smaller
        args = (ix, Q[:nq].contiguous(), lo[:nq].contiguous(), hi[:nq].contiguous(), 10, L, p)
        rc_a, ids_a, ds_a, st_a = _call(lib.frog_search_ex, *args)
        rc_b, ids_b, ds_b, st_b = _call(lib.frog_search_noalloc, *args)
        assert rc_a == 0 and rc_b == 0, lib.frog_last_error()
        assert (ids_a == ids_b).all()
        assert (ds_a.view(np.uint32) == ds_b.view(np.uint32)).all()
        keep = [c for c in range(F.STAT_N) if c not in TILE_COLUMNS]
        assert (st_a[:, keep] == st_b[:, keep]).all()
        assert (ids_b[:, 0] >= 0).mean() > 0.99


def test_noalloc_refuses_oversized_calls(case):
    ix, Q, lo, hi = case
    lib = F.lib()
    # entry mode 1 at L <= 40 takes about 13.5 KB per query: 40,000 queries
    # need about 540 MB, more than the 256 MiB array
    nq = 40000
    rep = (nq + Q.shape[0] - 1) // Q.shape[0]
    Qb = Q.repeat(rep, 1)[:nq].contiguous()
    lob = lo.repeat(rep)[:nq].contiguous()
    hib = hi.repeat(rep)[:nq].contiguous()
    p = F.search_params(entry_mode=1, epn=16, epn_frac=1.0, epn_max=2560, budget=16)
    rc, ids, _, _ = _call(lib.frog_search_noalloc, ix, Qb, lob, hib, 10, 32, p)
    assert rc == -7 and b"scratch" in lib.frog_last_error()
    assert (ids == -7).all()
    # the same call through frog_search_ex allocates and runs
    rc, ids, _, _ = _call(lib.frog_search_ex, ix, Qb, lob, hib, 10, 32, p)
    assert rc == 0 and (ids[:, 0] >= 0).mean() > 0.99


def test_noalloc_needs_a_prepared_seed(case):
    ix, Q, lo, hi = case
    lib = F.lib()
    p = F.search_params(entry_mode=1, seed=31337, epn=16, epn_frac=1.0, epn_max=2560, budget=16)
    rc, ids, _, _ = _call(lib.frog_search_noalloc, ix, Q, lo, hi, 10, 32, p)
    assert rc == -8 and (ids == -7).all()
