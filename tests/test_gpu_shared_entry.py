"""GPU parity of FROGSearch with the shared-priority entry sample
(entry_mode 1: matrix-core scan of the sample, exact re-rank, margin test)
against the CPU oracle's plain reading of the same sampling (every rank of the
range whose priority is below the query's threshold, evaluated one by one).
The index comes from the oracle's construction."""
import numpy as np
import pytest

import oracle
import paper_2608_16491_amd as F
import workloads
from tests.parity import assert_parity
from tests.test_gpu_search import Case

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

SH = dict(entry_mode=1, epn=16, epn_frac=1.0, epn_max=2000)


@pytest.fixture(scope="module")
def tiny():
    print("[gpu] shared entry sample: tiny workload n=10000 d=32 nq=100", flush=True)
    w = workloads.make("tiny")
    return Case(w.X, w.attr, w.Q, w.lo, w.hi)


@pytest.fixture(scope="module")
def mix128():
    print("[gpu] shared entry sample: mixture n=30000 d=128 nq=600", flush=True)
    w = workloads.make("c2", n=30000, nq=600)
    return Case(w.X, w.attr, w.Q, w.lo, w.hi)


@pytest.mark.parametrize("L", [10, 16, 24, 25, 32, 40, 41, 56, 64, 120, 121, 128, 248])
def test_shared_tiny_parity_pool_sizes(tiny, L):
    g_ids, g_d = tiny.gpu(10, L, **SH)
    o_ids, o_d, _ = tiny.cpu(10, L, **SH)
    assert_parity(g_ids, g_d, o_ids, o_d)


@pytest.mark.parametrize("p", [dict(entry_mode=1), dict(entry_mode=1, epn=100),
                               dict(entry_mode=1, epn=4, epn_frac=0.05, epn_max=700),
                               dict(entry_mode=1, epn=16, epn_frac=1.0, epn_max=20000),
                               dict(entry_mode=1, seed=12345, epn=16, epn_frac=0.2, epn_max=3000)])
def test_shared_entry_counts_and_seeds(tiny, p):
    g_ids, g_d = tiny.gpu(10, 64, **p)
    o_ids, o_d, _ = tiny.cpu(10, 64, **p)
    assert_parity(g_ids, g_d, o_ids, o_d)


def test_shared_stats_exact_visited_equal_oracle(tiny):
    # exact visited set: expansions, |EN| sums, distinct evaluations, ENC
    # entries, the sample size and the hotspot all equal the oracle's
    g_ids, g_d, g_st = tiny.gpu(10, 64, stats=True, hash_log2=0, **SH)
    o_ids, o_d, o_st = tiny.cpu(10, 64, **SH)
    res = assert_parity(g_ids, g_d, o_ids, o_d)
    ok = np.setdiff1d(np.arange(len(g_ids)), res)
    cols = [(F.STAT_EXPANSIONS, oracle.STAT_EXPANSIONS), (F.STAT_EN, oracle.STAT_EN),
            (F.STAT_DIST, oracle.STAT_DIST), (F.STAT_SCANNED, oracle.STAT_SCANNED),
            (F.STAT_ENTRY, oracle.STAT_ENTRY), (F.STAT_LSTART, oracle.STAT_LS), (F.STAT_LEND, oracle.STAT_LE)]
    for gc, oc in cols:
        assert (g_st[ok, gc] == o_st[ok, oc]).all(), (gc, g_st[ok, gc][:8], o_st[ok, oc][:8])


@pytest.mark.parametrize("hash_log2", [6, 10])
def test_shared_forgetful_table_does_not_change_results(tiny, hash_log2):
    ref_ids, ref_d, ref_st = tiny.gpu(10, 64, stats=True, hash_log2=0, **SH)
    g_ids, g_d, g_st = tiny.gpu(10, 64, stats=True, hash_log2=hash_log2, **SH)
    assert (g_ids == ref_ids).all() and (g_d.view(np.uint32) == ref_d.view(np.uint32)).all()
    assert (g_st[:, F.STAT_EXPANSIONS] == ref_st[:, F.STAT_EXPANSIONS]).all()
    assert (g_st[:, F.STAT_DIST] >= ref_st[:, F.STAT_DIST]).all()


def test_shared_seeds_keep_their_levels(tiny):
    # seed 0, then 99 (its own levels), then 0 again (the first levels, kept):
    # each run matches the oracle for its seed
    a_ids, a_d = tiny.gpu(10, 64, **SH)
    tiny.gpu(10, 64, **dict(SH, seed=99))
    c_ids, c_d = tiny.gpu(10, 64, **SH)
    assert (a_ids == c_ids).all() and (a_d.view(np.uint32) == c_d.view(np.uint32)).all()
    o2_ids, o2_d, _ = tiny.cpu(10, 64, **dict(SH, seed=99))
    g2_ids, g2_d = tiny.gpu(10, 64, **dict(SH, seed=99))
    assert_parity(g2_ids, g2_d, o2_ids, o2_d)


@pytest.mark.parametrize("L,emax,B", [(32, 2560, 24), (64, 2000, 16), (128, 800, 16)])
def test_shared_mixture_d128_parity(mix128, L, emax, B):
    p = dict(entry_mode=1, epn=16, epn_frac=1.0, epn_max=emax, budget=B)
    g_ids, g_d, g_st = mix128.gpu(10, L, stats=True, **p)
    o_ids, o_d, o_st = mix128.cpu(10, L, **p)
    res = assert_parity(g_ids, g_d, o_ids, o_d)
    ok = np.setdiff1d(np.arange(len(g_ids)), res)
    assert (g_st[ok, F.STAT_ENTRY] == o_st[ok, oracle.STAT_ENTRY]).all()
    assert (g_st[ok, F.STAT_EXPANSIONS] == o_st[ok, oracle.STAT_EXPANSIONS]).all()
    assert g_st[:, F.STAT_FALLBACK].mean() < 0.01


def test_shared_k100_pool248(mix128):
    # the largest pool entry mode 1 takes
    p = dict(entry_mode=1, epn=16, epn_frac=1.0, epn_max=3000)
    g_ids, g_d = mix128.gpu(100, 248, **p)
    o_ids, o_d, _ = mix128.cpu(100, 248, **p)
    assert_parity(g_ids, g_d, o_ids, o_d)


@pytest.mark.parametrize("L", [249, 256])
def test_shared_pools_above_248(tiny, L):
    # pools above 248: 256 candidates per work item, 512 merged
    g_ids, g_d = tiny.gpu(10, L, **SH)
    o_ids, o_d, _ = tiny.cpu(10, L, **SH)
    assert_parity(g_ids, g_d, o_ids, o_d)


def test_shared_k100_pool256(mix128):
    # the 512-entry merged list leaves the margin test room: few queries fall
    # back to evaluating their whole sample
    p = dict(entry_mode=1, epn=16, epn_frac=1.0, epn_max=3000)
    g_ids, g_d, g_st = mix128.gpu(100, 256, stats=True, **p)
    o_ids, o_d, _ = mix128.cpu(100, 256, **p)
    assert_parity(g_ids, g_d, o_ids, o_d)
    assert g_st[:, F.STAT_FALLBACK].mean() < 0.05


def test_unprepared_seed_is_refused(tiny):
    # the C ABI builds nothing inside a search: a seed whose sample was not
    # prepared is an error, reported before anything is enqueued
    import ctypes as C
    L = F.lib()
    p = F.search_params(entry_mode=1, seed=777, epn=16, epn_frac=1.0, epn_max=2000)
    nq = tiny.dQ.shape[0]
    ids = torch.full((nq, 10), -7, dtype=torch.int32, device="cuda")
    ds = torch.empty((nq, 10), dtype=torch.float32, device="cuda")
    rc = L.frog_search_ex(tiny.ix.handle, C.c_void_p(tiny.dQ.data_ptr()), nq, C.c_void_p(tiny.dlo.data_ptr()),
                          C.c_void_p(tiny.dhi.data_ptr()), 10, 64, C.byref(p), C.c_void_p(ids.data_ptr()),
                          C.c_void_p(ds.data_ptr()), None, None)
    assert rc == -8 and b"prepare" in L.frog_last_error()
    torch.cuda.synchronize()
    assert (ids == -7).all()
    assert L.frog_index_prepare_sample(tiny.ix.handle, C.c_uint64(777)) == 0
    # idempotent
    assert L.frog_index_prepare_sample(tiny.ix.handle, C.c_uint64(777)) == 0


def test_concurrent_searches_with_different_seeds(tiny):
    # two host threads, each on its own stream, search one index with
    # different seeds (both prepared first); each result equals the oracle's
    # for its seed on every repetition
    import threading
    seeds = [0, 4242]
    for s in seeds:
        tiny.ix.prepare_sample(s)
    expect = {s: tiny.cpu(10, 64, **dict(SH, seed=s)) for s in seeds}
    results, errors = {}, []

    def work(seed):
        try:
            st = torch.cuda.Stream()
            outs = []
            with torch.cuda.stream(st):
                for _ in range(6):
                    outs.append(F.search(tiny.ix, tiny.dQ, tiny.dlo, tiny.dhi, 10, 64, stream=st,
                                         **dict(SH, seed=seed)))
            st.synchronize()
            results[seed] = [(a.cpu().numpy(), b.cpu().numpy()) for a, b in outs]
        except Exception as ex:   # reported by the main thread
            errors.append(ex)

    threads = [threading.Thread(target=work, args=(s,)) for s in seeds]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    for s in seeds:
        o_ids, o_d, _ = expect[s]
        for g_ids, g_d in results[s]:
            assert_parity(g_ids, g_d, o_ids, o_d)


def test_shared_degenerate_ranges(tiny):
    n = tiny.ox.n
    lo = np.array([5.0, 100.0, np.nan, 3.0, 0.0, -1e9, n - 1.0, 40.0, 10.0, 0.0])
    hi = np.array([5.0, 99.0, 10.0, 3.5, n - 1.0, 1e9, n + 5.0, 39.0, 12.0, 15.0])
    Q = tiny.Q[:10]
    c = Case.__new__(Case)
    c.ox, c.ix = tiny.ox, tiny.ix
    c.Q, c.lo, c.hi = Q, lo, hi
    c.dQ = torch.as_tensor(Q).cuda()
    c.dlo = torch.as_tensor(lo).cuda()
    c.dhi = torch.as_tensor(hi).cuda()
    g_ids, g_d, g_st = c.gpu(10, 32, stats=True, **SH)
    o_ids, o_d, o_st = c.cpu(10, 32, **SH)
    assert_parity(g_ids, g_d, o_ids, o_d, max_residual=0)
    assert (g_st[[1, 2, 7]] == 0).all()


@pytest.mark.parametrize("d", [7, 96, 200])
def test_shared_other_dimensions(d):
    print(f"[gpu] shared entry sample, d={d}", flush=True)
    rng = np.random.default_rng(d)
    n, nq = 4000, 64
    X = rng.standard_normal((n, d)).astype(np.float32)
    attr = rng.permutation(n).astype(np.float64)
    Q = rng.standard_normal((nq, d)).astype(np.float32)
    sig = 2.0 ** (-8 * rng.random(nq))
    cnt = np.maximum(1, np.round(sig * n)).astype(np.int64)
    lo = rng.integers(0, n - cnt + 1)
    hi = lo + cnt - 1
    c = Case(X, attr, Q, lo.astype(np.float64), hi.astype(np.float64), m=8, ef_c=32, n_inv=4)
    p = dict(entry_mode=1, epn=8, epn_frac=0.5, epn_max=300)
    g_ids, g_d = c.gpu(10, 32, **p)
    o_ids, o_d, _ = c.cpu(10, 32, **p)
    assert_parity(g_ids, g_d, o_ids, o_d)


@pytest.mark.parametrize("mode", [0, 1])
def test_duplicate_attribute_values(mode):
    # 8,000 objects on 200 distinct attribute values (40 per value): the rank
    # domain breaks ties by original index, and a range's bounds count
    # attr < lo and attr <= hi, so integer bounds fall on runs of ties and
    # half-integer bounds between them
    print(f"[gpu] duplicate attribute values, entry mode {mode}", flush=True)
    rng = np.random.default_rng(17)
    w = workloads.make("tiny", n=8000, nq=120)
    attr = rng.integers(0, 200, 8000).astype(np.float64)
    a0 = rng.integers(0, 200, 120).astype(np.float64)
    span = rng.integers(0, 60, 120).astype(np.float64)
    lo = np.where(np.arange(120) % 2 == 0, a0, a0 - 0.5)
    hi = np.where(np.arange(120) % 3 == 0, a0 + span, a0 + span + 0.5)
    c = Case(w.X, attr, w.Q, lo, hi)
    p = dict(entry_mode=mode, epn=16, epn_frac=0.5, epn_max=600)
    g_ids, g_d = c.gpu(10, 32, **p)
    o_ids, o_d, _ = c.cpu(10, 32, **p)
    assert_parity(g_ids, g_d, o_ids, o_d)
    # every result lies in its range
    valid = g_ids >= 0
    av = attr[np.where(valid, g_ids, 0)]
    assert ((av >= lo[:, None]) & (av <= hi[:, None]) | ~valid).all()


@pytest.mark.parametrize("kind", ["one", "all_empty", "all_covered", "none_covered"])
def test_shared_query_order_classes(tiny, kind):
    # the pool and traversal take the queries in a planned order (ranges the
    # sample does not cover first, then covered and empty ones): batches made
    # of one class only, and a single query, give the oracle's rows
    n = tiny.ox.n
    rng = np.random.default_rng(11)
    nq = 1 if kind == "one" else 70
    if kind == "all_empty":
        lo = rng.integers(10, n, nq).astype(np.float64)
        hi = lo - 1.0
    elif kind == "all_covered":
        lo = rng.integers(0, n - 500, nq).astype(np.float64)
        hi = lo + rng.integers(0, 400, nq)
    else:
        lo = rng.integers(0, n // 4, nq).astype(np.float64)
        hi = lo + rng.integers(n // 2, 3 * n // 4, nq)
    Q = tiny.Q[np.arange(nq) % tiny.Q.shape[0]]
    c = Case.__new__(Case)
    c.ox, c.ix = tiny.ox, tiny.ix
    c.Q, c.lo, c.hi = Q, lo, hi
    c.dQ = torch.as_tensor(Q).cuda()
    c.dlo = torch.as_tensor(lo).cuda()
    c.dhi = torch.as_tensor(hi).cuda()
    p = dict(entry_mode=1, epn=16, epn_frac=1.0, epn_max=500)
    g_ids, g_d = c.gpu(10, 32, **p)
    o_ids, o_d, _ = c.cpu(10, 32, **p)
    assert_parity(g_ids, g_d, o_ids, o_d, max_residual=0 if kind == "all_empty" else 1)
    if kind == "all_empty":
        assert (g_ids == -1).all()
