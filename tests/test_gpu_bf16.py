"""GPU parity of FROGSearch over an index uploaded with bfloat16 rows.

bfloat16 keeps fp32's exponent range with an 8-bit significand, so unlike
binary16 it cannot overflow on embeddings of any scale.  The library rounds
each value once (nearest, ties to even) and the kernels widen it exactly, so
the result is the exact FROGSearch result over the rounded vectors.  The
oracle searches the same graph with rows rounded here by a different method
(significand and exponent split with frexp, the significand rounded to 8
bits with numpy's ties-to-even rint), widened back to fp32."""
import numpy as np
import pytest

import oracle
import paper_2608_16491_amd as F
import workloads
from tests.parity import assert_parity
from tests.test_gpu_search import Case

torch = pytest.importorskip("torch")

SH = dict(entry_mode=1, epn=16, epn_frac=1.0, epn_max=2000)


def to_bf16(x):
    """x rounded to the nearest bfloat16 (ties to even), as fp32.  Normal
    numbers only: x = m 2^e with 0.5 <= |m| < 1, and bf16 keeps 8 bits of m."""
    m, e = np.frexp(np.asarray(x, np.float64))
    return np.ldexp(np.rint(m * 256.0) / 256.0, e).astype(np.float32)


def test_bf16_rounding_pins():
    # 1 + 2^-8 lies halfway between 1 and 1 + 2^-7: ties to the even 1;
    # 1 + 3 2^-8 lies halfway between 1 + 2^-7 and 1 + 2^-6: the even one
    # is 1 + 2^-6; the largest finite value rounds to 2^128 (overflow)
    v = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8 + 2 ** -12), 3.0, 0.0,
                  np.float32(0.1), 2.0 ** -100 * 1.00390625], np.float64)
    want = np.array([1.0, 1 + 2 ** -6, -(1 + 2 ** -7), 3.0, 0.0, 0.10009765625, 2.0 ** -100], np.float64)
    assert (to_bf16(v).astype(np.float64) == want).all()
    # the result has at most 8 significant bits, and the error is at most
    # half a unit in the last place (2^-9 relative to 2^floor(log2|x|))
    x = np.random.default_rng(0).standard_normal(20000).astype(np.float32)
    r = to_bf16(x).astype(np.float64)
    mm, _ = np.frexp(r)
    assert (np.rint(mm * 256) == mm * 256).all()
    ulp = 2.0 ** (np.floor(np.log2(np.abs(x.astype(np.float64)))) - 7)
    assert (np.abs(r - x) <= ulp / 2).all()


class BCase(Case):
    def __init__(self, X, attr, Q, lo, hi, **build):
        super().__init__(X, attr, Q, lo, hi, **build)
        self.ix.upload(0, storage="bf16")
        ox = self.ox
        self.ox = oracle.OracleIndex(ox.perm, ox.attr_sorted, to_bf16(ox.X_rank), ox.ENC)


@pytest.fixture(scope="module")
def tiny():
    print("[gpu] bf16 rows: tiny workload n=10000 d=32 nq=100", flush=True)
    w = workloads.make("tiny")
    return BCase(w.X, w.attr, w.Q, w.lo, w.hi)


@pytest.fixture(scope="module")
def mix128():
    print("[gpu] bf16 rows: mixture n=30000 d=128 nq=400", flush=True)
    w = workloads.make("c2", n=30000, nq=400)
    return BCase(w.X, w.attr, w.Q, w.lo, w.hi)


@pytest.mark.gpu
@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("L", [16, 32, 64, 128, 256])
def test_bf16_tiny_parity(tiny, mode, L):
    p = dict(SH, entry_mode=mode)
    g_ids, g_d = tiny.gpu(10, L, **p)
    o_ids, o_d, _ = tiny.cpu(10, L, **p)
    assert_parity(g_ids, g_d, o_ids, o_d)


@pytest.mark.gpu
@pytest.mark.parametrize("p", [dict(entry_mode=0), dict(SH), dict(entry_mode=1, epn=4, epn_frac=0.05, epn_max=700),
                               dict(entry_mode=1, epn=16, epn_frac=1.0, epn_max=3072, budget=24)])
def test_bf16_d128_parity(mix128, p):
    g_ids, g_d = mix128.gpu(10, 64, **p)
    o_ids, o_d, _ = mix128.cpu(10, 64, **p)
    assert_parity(g_ids, g_d, o_ids, o_d)


@pytest.mark.gpu
def test_bf16_stats_exact_visited_equal_oracle(mix128):
    g_ids, g_d, g_st = mix128.gpu(10, 24, stats=True, hash_log2=0, **SH)
    o_ids, o_d, o_st = mix128.cpu(10, 24, **SH)
    res = assert_parity(g_ids, g_d, o_ids, o_d)
    ok = np.setdiff1d(np.arange(len(g_ids)), res)
    cols = [(F.STAT_EXPANSIONS, oracle.STAT_EXPANSIONS), (F.STAT_EN, oracle.STAT_EN),
            (F.STAT_DIST, oracle.STAT_DIST), (F.STAT_ENTRY, oracle.STAT_ENTRY)]
    for gc, oc in cols:
        assert (g_st[ok, gc] == o_st[ok, oc]).all(), (gc, g_st[ok, gc][:8], o_st[ok, oc][:8])


@pytest.mark.gpu
def test_bf16_padded_rows_and_large_scale():
    # d = 100 (rows padded to 128 values) with values scaled by 2^40, far
    # beyond binary16's range (squared distances near 2^80 still fit fp32):
    # bf16 keeps the exponent, so the search over the rounded rows matches
    print("[gpu] bf16 rows: padded d=100 n=6000 nq=80, values scaled by 2^40", flush=True)
    w = workloads.make("c2", n=6000, nq=80)
    s = np.float32(2.0 ** 40)
    X = np.ascontiguousarray(w.X[:, :100]) * s
    Q = np.ascontiguousarray(w.Q[:, :100]) * s
    c = BCase(X, w.attr, Q, w.lo, w.hi)
    for mode in (0, 1):
        p = dict(SH, entry_mode=mode)
        g_ids, g_d = c.gpu(10, 64, **p)
        o_ids, o_d, _ = c.cpu(10, 64, **p)
        assert_parity(g_ids, g_d, o_ids, o_d)
