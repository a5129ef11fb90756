"""GPU parity of FROGSearch (Alg. 2-4) against the CPU oracle, through the
C ABI.  The index comes from the oracle's own construction and is handed to
the library with frog_index_from_arrays, so every input of the comparison is
produced outside the library."""
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


class Case:
    def __init__(self, X, attr, Q, lo, hi, **build):
        self.ox = oracle.build(X, attr, **build)
        self.ix = F.Index.from_arrays(self.ox.X_rank, self.ox.attr_sorted, self.ox.perm, self.ox.ENC).upload(0)
        self.Q, self.lo, self.hi = Q, np.asarray(lo, np.float64), np.asarray(hi, np.float64)
        self.dQ = _cuda(Q, torch.float32)
        self.dlo = _cuda(self.lo, torch.float64)
        self.dhi = _cuda(self.hi, torch.float64)

    def gpu(self, k, L, stats=False, **p):
        out = F.search(self.ix, self.dQ, self.dlo, self.dhi, k, L, stats=stats, **p)
        torch.cuda.synchronize()
        return tuple(t.cpu().numpy() for t in out)

    def cpu(self, k, L, **p):
        kw = dict(epn=p.get("epn", 16), epn_frac=p.get("epn_frac", 0.0), epn_max=p.get("epn_max", 0),
                  B=p.get("budget", 16), seed=p.get("seed", 0), entry_mode=p.get("entry_mode", 0),
                  hot_mode=p.get("hotspot_mode", 0), eager=bool(p.get("eager_check", 0)))
        qidx = np.arange(self.Q.shape[0]) + p.get("query_base", 0)
        return oracle.search(self.ox, self.Q, self.lo, self.hi, k, L, qidx=qidx, **kw)


@pytest.fixture(scope="module")
def tiny():
    print("[gpu] tiny workload n=10000 d=32 nq=100", flush=True)
    w = workloads.make("tiny")
    return Case(w.X, w.attr, w.Q, w.lo, w.hi)


@pytest.fixture(scope="module")
def mix128():
    print("[gpu] mixture n=30000 d=128 nq=300", flush=True)
    w = workloads.make("c2", n=30000, nq=300)
    return Case(w.X, w.attr, w.Q, w.lo, w.hi)


@pytest.mark.parametrize("L", [32, 64, 128, 256])
def test_tiny_parity_pool_sizes(tiny, L):
    k = 10
    g_ids, g_d = tiny.gpu(k, L)
    o_ids, o_d, _ = tiny.cpu(k, L)
    assert_parity(g_ids, g_d, o_ids, o_d)


def test_tiny_stats_exact_visited_equal_oracle(tiny):
    # with the exact visited set the counts equal the oracle's |visited|,
    # expansions, |EN| sums, ENC entries examined, entry points and hotspot
    g_ids, g_d, g_st = tiny.gpu(10, 64, stats=True, hash_log2=0)
    o_ids, o_d, o_st = tiny.cpu(10, 64)
    res = assert_parity(g_ids, g_d, o_ids, o_d)
    ok = np.setdiff1d(np.arange(len(g_ids)), res)
    cols = [(F.STAT_EXPANSIONS, oracle.STAT_EXPANSIONS), (F.STAT_EN, oracle.STAT_EN),
            (F.STAT_DIST, oracle.STAT_DIST), (F.STAT_SCANNED, oracle.STAT_SCANNED),
            (F.STAT_ENTRY, oracle.STAT_ENTRY), (F.STAT_LSTART, oracle.STAT_LS), (F.STAT_LEND, oracle.STAT_LE)]
    for gc, oc in cols:
        assert (g_st[ok, gc] == o_st[ok, oc]).all(), (gc, g_st[ok, gc][:8], o_st[ok, oc][:8])


@pytest.mark.parametrize("hash_log2", [6, 8, 10, 13])
def test_forgetful_table_does_not_change_results(tiny, hash_log2):
    ref_ids, ref_d, ref_st = tiny.gpu(10, 64, stats=True, hash_log2=0)
    g_ids, g_d, g_st = tiny.gpu(10, 64, stats=True, hash_log2=hash_log2)
    assert (g_ids == ref_ids).all() and (g_d.view(np.uint32) == ref_d.view(np.uint32)).all()
    assert (g_st[:, F.STAT_EXPANSIONS] == ref_st[:, F.STAT_EXPANSIONS]).all()
    assert (g_st[:, F.STAT_DIST] >= ref_st[:, F.STAT_DIST]).all()


@pytest.mark.parametrize("budget", [1, 4, 16, 64])
def test_budget_parity(tiny, budget):
    g_ids, g_d = tiny.gpu(10, 64, budget=budget)
    o_ids, o_d, _ = tiny.cpu(10, 64, budget=budget)
    assert_parity(g_ids, g_d, o_ids, o_d)


@pytest.mark.parametrize("p", [dict(epn=1), dict(epn=100), dict(epn=16, epn_frac=0.05, epn_max=700),
                               dict(epn=4, epn_frac=1.0, epn_max=20000), dict(seed=12345)])
def test_entry_point_parity(tiny, p):
    g_ids, g_d = tiny.gpu(10, 64, **p)
    o_ids, o_d, _ = tiny.cpu(10, 64, **p)
    assert_parity(g_ids, g_d, o_ids, o_d)


def test_query_base_keys_entry_points(tiny):
    # a sub-batch with query_base=i0 reproduces rows i0.. of the full batch
    full_ids, full_d = tiny.gpu(10, 64)
    sub = F.search(tiny.ix, tiny.dQ[37:61].contiguous(), tiny.dlo[37:61].contiguous(),
                   tiny.dhi[37:61].contiguous(), 10, 64, query_base=37)
    torch.cuda.synchronize()
    assert (sub[0].cpu().numpy() == full_ids[37:61]).all()


@pytest.mark.parametrize("k,L", [(1, 32), (10, 10), (64, 64), (100, 256)])
def test_k_and_pool_edges(tiny, k, L):
    g_ids, g_d = tiny.gpu(k, L)
    o_ids, o_d, _ = tiny.cpu(k, L)
    assert_parity(g_ids, g_d, o_ids, o_d)


def test_degenerate_ranges(tiny):
    n = tiny.ox.n
    lo = np.array([5.0, 100.0, np.nan, 3.0, 0.0, -1e9, n - 1.0, 40.0, 10.0, 0.0])
    hi = np.array([5.0, 99.0, 5.0, np.nan, n - 1.0, 1e9, n + 5.0, 47.0, 10.5, 2.0])
    Q = tiny.Q[:10]
    c = Case.__new__(Case)
    c.ox, c.ix, c.Q, c.lo, c.hi = tiny.ox, tiny.ix, Q, lo, hi
    c.dQ, c.dlo, c.dhi = _cuda(Q, torch.float32), _cuda(lo, torch.float64), _cuda(hi, torch.float64)
    g_ids, g_d = c.gpu(10, 64)
    o_ids, o_d, _ = c.cpu(10, 64)
    assert_parity(g_ids, g_d, o_ids, o_d, max_residual=0)
    assert (g_ids[1] == -1).all() and (g_ids[2] == -1).all() and (g_ids[3] == -1).all()
    assert np.isinf(g_d[1]).all()
    assert (g_ids[0, 1:] == -1).all() and g_ids[0, 0] == tiny.ox.perm[5]


def test_rank_bounds_kernel(tiny):
    rng = np.random.default_rng(0)
    lo = np.concatenate([rng.uniform(-10, 10010, 500), [np.nan, 5, 7.5]])
    hi = np.concatenate([lo[:500] + rng.uniform(-5, 3000, 500), [5, np.nan, 7.4]])
    lr = F.rank_bounds(tiny.ix, _cuda(lo, torch.float64), _cuda(hi, torch.float64))
    torch.cuda.synchronize()
    lr = lr.cpu().numpy()
    a = tiny.ox.attr_sorted
    for i in range(500):
        assert lr[i, 0] == np.searchsorted(a, lo[i], "left")
        assert lr[i, 1] == np.searchsorted(a, hi[i], "right") - 1
    assert lr[500, 0] > lr[500, 1] and lr[501, 0] > lr[501, 1] and lr[502, 0] > lr[502, 1]


def test_deterministic(tiny):
    a = tiny.gpu(10, 128)
    b = tiny.gpu(10, 128)
    assert (a[0] == b[0]).all() and (a[1].view(np.uint32) == b[1].view(np.uint32)).all()


@pytest.mark.parametrize("L", [32, 64, 128])
def test_mixture_d128_parity(mix128, L):
    p = dict(epn=16, epn_frac=0.01, epn_max=300)
    g_ids, g_d, g_st = mix128.gpu(10, L, stats=True, **p)
    o_ids, o_d, o_st = mix128.cpu(10, L, **p)
    res = assert_parity(g_ids, g_d, o_ids, o_d)
    ok = np.setdiff1d(np.arange(len(g_ids)), res)
    assert (g_st[ok, F.STAT_EXPANSIONS] == o_st[ok, oracle.STAT_EXPANSIONS]).all()


@pytest.mark.parametrize("entry_mode", [0, 1])
@pytest.mark.parametrize("d", [7, 96, 200, 1021, 1030])
def test_other_dimensions(d, entry_mode):
    # d=7 pads rows to 32 floats; d=96 uses 3 chunks per lane; d=200 the 64-lane
    # path; d=1021 its widest rows with the query in registers (a query length
    # not a multiple of 4); d=1030 its chunk loop (rows past 1024 floats)
    rng = np.random.default_rng(d)
    n, nq = 3000, 64
    X = rng.standard_normal((n, d)).astype(np.float32)
    attr = rng.permutation(n).astype(np.float64)
    Q = rng.standard_normal((nq, d)).astype(np.float32)
    sig = np.array([0.01, 0.1, 0.5, 1.0])[np.arange(nq) % 4]
    lo, hi = workloads.ranges_for_selectivity(rng, sig, n)
    c = Case(X, attr, Q, lo, hi)
    p = {}
    if entry_mode == 1:   # the shared entry sample: matrix-core scan, pool, traversal
        p = dict(entry_mode=1, epn=16, epn_frac=0.2, epn_max=600)
        c.ix.prepare_sample(0)
    g_ids, g_d = c.gpu(10, 64, **p)
    o_ids, o_d, _ = c.cpu(10, 64, **p)
    assert_parity(g_ids, g_d, o_ids, o_d)


@pytest.mark.parametrize("entry_mode", [0, 1])
@pytest.mark.parametrize("hotspot_mode,eager", [(1, 0), (2, 0), (0, 1), (2, 1)])
def test_ablation_switches_match_oracle(tiny, entry_mode, hotspot_mode, eager):
    # Sec 8.2.3 ablations: hotspot without end condition / without localisation,
    # eager visited check (exact visited set); every statistic as the oracle's
    p = dict(entry_mode=entry_mode, epn=16, epn_frac=0.2, epn_max=600, hotspot_mode=hotspot_mode,
             eager_check=eager, hash_log2=0)
    g_ids, g_d, g_st = tiny.gpu(10, 64, stats=True, **p)
    o_ids, o_d, o_st = tiny.cpu(10, 64, **p)
    res = assert_parity(g_ids, g_d, o_ids, o_d)
    ok = np.setdiff1d(np.arange(len(g_ids)), res)
    cols = [(F.STAT_EXPANSIONS, oracle.STAT_EXPANSIONS), (F.STAT_EN, oracle.STAT_EN),
            (F.STAT_DIST, oracle.STAT_DIST), (F.STAT_SCANNED, oracle.STAT_SCANNED),
            (F.STAT_ENTRY, oracle.STAT_ENTRY), (F.STAT_LSTART, oracle.STAT_LS), (F.STAT_LEND, oracle.STAT_LE)]
    for gc, oc in cols:
        assert (g_st[ok, gc] == o_st[ok, oc]).all(), (gc, g_st[ok, gc][:8], o_st[ok, oc][:8])


def test_ablation_hotspot_modes_forgetful_table(tiny):
    # the hotspot ablations also hold with the forgetful LDS table
    for hm in (1, 2):
        g_ids, g_d = tiny.gpu(10, 64, hotspot_mode=hm)
        o_ids, o_d, _ = tiny.cpu(10, 64, hotspot_mode=hm)
        assert_parity(g_ids, g_d, o_ids, o_d)


@pytest.mark.parametrize("mode", [0, 1])
def test_empty_and_single_query_batches(tiny, mode):
    # nq = 0 returns empty outputs without launching; nq = 1 matches the oracle
    p = dict(entry_mode=mode, epn=16, epn_frac=1.0, epn_max=2000)
    d = tiny.dQ.shape[1]
    dev = tiny.dQ.device
    Q0 = torch.empty((0, d), dtype=torch.float32, device=dev)
    lo0 = torch.empty((0,), dtype=torch.float64, device=dev)
    ids, ds = F.search(tiny.ix, Q0, lo0, lo0.clone(), 10, 64, **p)
    torch.cuda.synchronize()
    assert tuple(ids.shape) == (0, 10) and tuple(ds.shape) == (0, 10)
    gt, gd, cert = F.bruteforce(tiny.ix, Q0, lo0, lo0.clone(), 10)
    assert tuple(gt.shape) == (0, 10)
    ids, ds = F.search(tiny.ix, tiny.dQ[3:4].contiguous(), tiny.dlo[3:4].contiguous(), tiny.dhi[3:4].contiguous(),
                       10, 64, **p)
    torch.cuda.synchronize()
    o_ids, o_d, _ = oracle.search(tiny.ox, tiny.Q[3:4], tiny.lo[3:4], tiny.hi[3:4], 10, 64, qidx=np.array([0]),
                                  epn=16, epn_frac=1.0, epn_max=2000, entry_mode=mode)
    assert_parity(ids.cpu().numpy(), ds.cpu().numpy(), o_ids, o_d)
