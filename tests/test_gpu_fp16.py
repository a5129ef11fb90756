"""GPU parity of FROGSearch over an index uploaded with fp16 rows.

The paper keeps the vectors in half precision on the device (Sec 8.1).  The
library rounds each value once to binary16 (nearest even), widens it exactly
in the kernels and accumulates distances as for fp32 rows, so its result is
the exact FROGSearch result over the rounded vectors.  The oracle searches the
same graph with its rows rounded by numpy's float16 conversion (an
independent implementation of the same IEEE rounding) and widened back to
fp32; ids and distances must match under the usual parity rule, in both entry
modes."""
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


def rounded(ox):
    """The oracle index with its rows rounded to binary16 and widened."""
    return oracle.OracleIndex(ox.perm, ox.attr_sorted, ox.X_rank.astype(np.float16).astype(np.float32), ox.ENC)


class HalfCase(Case):
    def __init__(self, X, attr, Q, lo, hi, **build):
        super().__init__(X, attr, Q, lo, hi, **build)
        self.ix.upload(0, storage="fp16")
        self.ox = rounded(self.ox)


@pytest.fixture(scope="module")
def tiny():
    print("[gpu] fp16 rows: tiny workload n=10000 d=32 nq=100", flush=True)
    w = workloads.make("tiny")
    return HalfCase(w.X, w.attr, w.Q, w.lo, w.hi)


@pytest.fixture(scope="module")
def mix128():
    print("[gpu] fp16 rows: mixture n=30000 d=128 nq=400", flush=True)
    w = workloads.make("c2", n=30000, nq=400)
    return HalfCase(w.X, w.attr, w.Q, w.lo, w.hi)


@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("L", [16, 24, 32, 64, 128, 256])
def test_fp16_tiny_parity(tiny, mode, L):
    p = dict(SH, entry_mode=mode)
    g_ids, g_d = tiny.gpu(10, L, **p)
    o_ids, o_d, _ = tiny.cpu(10, L, **p)
    assert_parity(g_ids, g_d, o_ids, o_d)


@pytest.mark.parametrize("p", [dict(entry_mode=0), dict(entry_mode=0, epn=64, hash_log2=0),
                               dict(SH), dict(entry_mode=1, epn=4, epn_frac=0.05, epn_max=700),
                               dict(entry_mode=1, epn=16, epn_frac=1.0, epn_max=3072, budget=24)])
def test_fp16_d128_parity(mix128, p):
    g_ids, g_d = mix128.gpu(10, 64, **p)
    o_ids, o_d, _ = mix128.cpu(10, 64, **p)
    assert_parity(g_ids, g_d, o_ids, o_d)


def test_fp16_stats_exact_visited_equal_oracle(mix128):
    g_ids, g_d, g_st = mix128.gpu(10, 24, stats=True, hash_log2=0, **SH)
    o_ids, o_d, o_st = mix128.cpu(10, 24, **SH)
    res = assert_parity(g_ids, g_d, o_ids, o_d)
    ok = np.setdiff1d(np.arange(len(g_ids)), res)
    cols = [(F.STAT_EXPANSIONS, oracle.STAT_EXPANSIONS), (F.STAT_EN, oracle.STAT_EN),
            (F.STAT_DIST, oracle.STAT_DIST), (F.STAT_ENTRY, oracle.STAT_ENTRY)]
    for gc, oc in cols:
        assert (g_st[ok, gc] == o_st[ok, oc]).all(), (gc, g_st[ok, gc][:8], o_st[ok, oc][:8])


@pytest.mark.parametrize("d", [20, 100])
def test_fp16_padded_rows(d):
    # d not a multiple of 64: rows padded with zeros to 64 / 128 halves
    print(f"[gpu] fp16 rows: padded d={d} n=6000 nq=80", flush=True)
    w = workloads.make("tiny" if d <= 32 else "c2", n=6000, nq=80)
    X = np.ascontiguousarray(w.X[:, :d])
    Q = np.ascontiguousarray(w.Q[:, :d])
    c = HalfCase(X, w.attr, Q, w.lo, w.hi)
    for mode in (0, 1):
        p = dict(SH, entry_mode=mode)
        g_ids, g_d = c.gpu(10, 64, **p)
        o_ids, o_d, _ = c.cpu(10, 64, **p)
        assert_parity(g_ids, g_d, o_ids, o_d)


def test_fp16_then_fp32_upload(tiny):
    # replacing the device copy drops the fp16 norms and sample rows: an fp32
    # upload of the same index matches the fp32 oracle again, and the fp16
    # upload after it the rounded one
    w = workloads.make("tiny")
    ox32 = oracle.build(w.X, w.attr)
    try:
        tiny.ix.upload(0, storage="fp32")
        for mode in (0, 1):
            p = dict(SH, entry_mode=mode)
            g_ids, g_d = tiny.gpu(10, 64, **p)
            o_ids, o_d, _ = oracle.search(ox32, w.Q, w.lo, w.hi, 10, 64, epn=16, epn_frac=1.0, epn_max=2000,
                                          entry_mode=mode)
            assert_parity(g_ids, g_d, o_ids, o_d)
    finally:
        tiny.ix.upload(0, storage="fp16")
    g_ids, g_d = tiny.gpu(10, 64, **SH)
    o_ids, o_d, _ = tiny.cpu(10, 64, **SH)
    assert_parity(g_ids, g_d, o_ids, o_d)


def test_fp16_bruteforce_unsupported(tiny):
    with pytest.raises(F.FrogError) as e:
        F.bruteforce(tiny.ix, tiny.dQ, tiny.dlo, tiny.dhi, 10)
    assert e.value.code == -7


def test_fp16_empty_and_single_ranges(tiny):
    # empty ranges, a single object, and the full domain
    w = workloads.make("tiny")
    a = np.sort(w.attr)
    lo = np.array([a[-1] + 1.0, a[5], a[0] - 1.0, a[100]], np.float64)
    hi = np.array([a[-1] + 2.0, a[5], a[-1] + 1.0, a[99]], np.float64)
    Q = w.Q[:4]
    c = Case.__new__(HalfCase)
    c.ox, c.ix, c.Q, c.lo, c.hi = tiny.ox, tiny.ix, Q, lo, hi
    c.dQ = torch.as_tensor(Q, device="cuda")
    c.dlo = torch.as_tensor(lo, device="cuda")
    c.dhi = torch.as_tensor(hi, device="cuda")
    for mode in (0, 1):
        p = dict(SH, entry_mode=mode)
        g_ids, g_d = c.gpu(10, 64, **p)
        o_ids, o_d, _ = c.cpu(10, 64, **p)
        assert_parity(g_ids, g_d, o_ids, o_d)
        assert (g_ids[0] == -1).all() and (g_ids[3] == -1).all()
        assert (g_ids[1][1:] == -1).all() and g_ids[1][0] >= 0
