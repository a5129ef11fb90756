"""Pins for the CPU oracle: each test ties one oracle function to something
other than the oracle itself (a library routine, a closed form, brute force on
tiny inputs, a hand-worked example, or an independent textbook algorithm).

Paper passages: squared L2 (Sec 2.1), rank domain (Sec 4), segment tree and
HotspotLocalization (Sec 4, Alg 3, Eq. endcondition), entry points and
FROGSearch (Alg 2), ENIdentification (Alg 4), KANNSearch (Alg 1), RFANNS
(Def. 2), fusion distance (Eq. fusion-distance), boundary effect (Eq.
naive_attr_dist), construction (Sec 6).
"""
import math
import os

import numpy as np
import pytest

import oracle
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ------------------------------------------------------------------ P1 distance

def test_dist_matches_numpy_fp64():
    rng = np.random.default_rng(1)
    for d in (1, 3, 32, 96, 128, 960):
        a = rng.standard_normal(d).astype(np.float32)
        b = rng.standard_normal(d).astype(np.float32)
        ref = np.float32(((a.astype(np.float64) - b.astype(np.float64)) ** 2).sum())
        got = oracle.dist(a, b)
        # fp64 sums of the same terms in two orders agree to ~1e-16 relative;
        # after the single rounding to fp32 they are equal or 1 ulp apart.
        assert abs(float(got) - float(ref)) <= float(np.spacing(ref))


def test_dist_exact_small_integers():
    # integer-valued inputs: every term and the sum are exact
    a = np.array([1, 2, 3, 4], np.float32)
    b = np.array([4, 0, 3, -1], np.float32)
    assert oracle.dist(a, b) == np.float32(9 + 4 + 0 + 25)
    assert oracle.dist(a, a) == 0.0


def test_splitmix64_published_values():
    # SplitMix64 stream from state 0: the first outputs of the published
    # generator (state += golden gamma, then the finaliser).
    # x_1 = mix(0x9E3779B97F4A7C15), x_2 = mix(2*gamma), ...
    expected = [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]
    gamma = 0x9E3779B97F4A7C15
    for i, e in enumerate(expected):
        # fo_splitmix64(x) adds one gamma itself, so feed the state before it
        assert oracle.splitmix64((i * gamma) & 0xFFFFFFFFFFFFFFFF) == e


# ------------------------------------------------------------------ P3 ranks

def test_rank_bounds_match_searchsorted():
    rng = np.random.default_rng(2)
    a = np.sort(rng.integers(0, 50, 200).astype(np.float64))  # many duplicates
    for _ in range(500):
        lo, hi = rng.uniform(-5, 55, 2)
        l, r = oracle.rank_bounds(a, lo, hi)
        assert l == np.searchsorted(a, lo, "left")
        assert r == np.searchsorted(a, hi, "right") - 1
    # exact-value endpoints include all duplicates
    l, r = oracle.rank_bounds(a, 10.0, 10.0)
    assert (a[l:r + 1] == 10.0).all() and (a == 10.0).sum() == r - l + 1


def test_rank_bounds_degenerate():
    a = np.arange(10, dtype=np.float64)
    assert oracle.rank_bounds(a, 5, 3)[0] > oracle.rank_bounds(a, 5, 3)[1]   # lo > hi
    l, r = oracle.rank_bounds(a, np.nan, 3)
    assert l > r
    l, r = oracle.rank_bounds(a, 1, np.nan)
    assert l > r
    assert oracle.rank_bounds(a, -np.inf, np.inf) == (0, 9)
    assert oracle.rank_bounds(a, 100, 200)[0] == 10


def test_rank_order_is_stable_attribute_sort():
    import ctypes as C
    lib = oracle._load()
    rng = np.random.default_rng(3)
    attr = rng.integers(0, 20, 300).astype(np.float64)
    perm = np.empty(300, np.int32)
    srt = np.empty(300, np.float64)
    assert lib.fo_rank_order(oracle._p(attr), 300, oracle._p(perm), oracle._p(srt)) == 0
    assert (perm == np.argsort(attr, kind="stable")).all()
    assert (srt == np.sort(attr)).all()
    attr[7] = np.nan
    assert lib.fo_rank_order(oracle._p(attr), 300, oracle._p(perm), oracle._p(srt)) == -1


# ------------------------------------------------------------------ P5 geometry

def _layers(n, H):
    """Segments per layer by explicit recursive halving (independent of the
    oracle's per-rank descent)."""
    out = [[(0, n - 1)]]
    for _ in range(H - 1):
        nxt = []
        for (L, R) in out[-1]:
            mid = L + (R - L) // 2
            nxt.append((L, mid))
            nxt.append((mid + 1, R))
        out.append(nxt)
    return out


@pytest.mark.parametrize("n", [1, 2, 3, 7, 16, 17, 100, 10_000, 1_000_000])
def test_num_layers_closed_form(n):
    import math
    for n_inv in (0, 6, 7):
        full = (math.ceil(math.log2(n)) if n > 1 else 0) + 1
        assert oracle.num_layers(n, n_inv) == max(1, full - n_inv)
    # the configurations used by the benchmarks
    assert oracle.num_layers(10_000, 7) == 8
    assert oracle.num_layers(1_000_000, 7) == 14
    assert oracle.num_layers(1_000_000, 6) == 15
    assert oracle.num_layers(10_000_000, 7) == 18


@pytest.mark.parametrize("n,H", [(16, 4), (17, 5), (100, 6), (1000, 8)])
def test_segments_partition_each_layer(n, H):
    layers = _layers(n, H)
    for h, segs in enumerate(layers):
        covered = np.zeros(n, int)
        for (L, R) in segs:
            if L <= R:
                covered[L:R + 1] += 1
        assert (covered == 1).all()          # every rank in exactly one segment
        for p in range(n):
            s, e = oracle.segment(n, h, p)
            assert (s, e) in segs and s <= p <= e


# ------------------------------------------------------------------ P4 hotspot

def _hotspot_bruteforce(l, r, H, n):
    layers = _layers(n, H)

    def seg_of(h, p):
        for (L, R) in layers[h]:
            if L <= p <= R:
                return L, R
        raise AssertionError

    Ls = max(h for h in range(H) if seg_of(h, l) == seg_of(h, r))
    Le = Ls
    for h in range(Ls + 1, H):
        _, el = seg_of(h, l)
        sr, _ = seg_of(h, r)
        # overlap with the two boundary segments vs 2^-h (r - l), exactly
        if ((el + 1 - l) + (r - sr)) * 2 ** h >= (r - l):
            Le = h
        else:
            break
    return Ls, Le


def test_hotspot_hand_examples():
    rows = [list(map(int, ln.split())) for ln in open(os.path.join(GOLDEN, "hotspot_n16.txt"))
            if ln.strip() and not ln.startswith("#")]
    assert len(rows) >= 6
    for n, H, l, r, Ls, Le in rows:
        assert oracle.hotspot(l, r, H, n) == (Ls, Le), (l, r)


@pytest.mark.parametrize("n,H", [(16, 4), (37, 5), (100, 6), (1000, 8)])
def test_hotspot_bruteforce(n, H):
    rng = np.random.default_rng(n)
    pairs = [(l, r) for l in range(n) for r in range(l, n)] if n <= 40 else \
        [tuple(sorted(rng.integers(0, n, 2))) for _ in range(400)]
    for l, r in pairs:
        assert oracle.hotspot(l, r, H, n) == _hotspot_bruteforce(l, r, H, n), (l, r)


# ------------------------------------------------------------------ entry points

def test_entry_points_all_when_small():
    assert list(oracle.entry_points(5, 9, 16, 0, 0)) == [5, 6, 7, 8, 9]
    assert len(oracle.entry_points(5, 4, 16, 0, 0)) == 0


def test_entry_points_stratified_distinct_in_range():
    rng = np.random.default_rng(4)
    for _ in range(200):
        l = int(rng.integers(0, 1000))
        cnt = int(rng.integers(17, 5000))
        epn = int(rng.integers(1, 17))
        ep = oracle.entry_points(l, l + cnt - 1, epn, 7, int(rng.integers(0, 1 << 20)))
        assert len(ep) == epn and len(set(ep.tolist())) == epn
        # entry j lies in stratum j of [l, r]
        for j, v in enumerate(ep):
            assert l + (j * cnt) // epn <= v <= l + ((j + 1) * cnt) // epn - 1


def test_entry_points_roughly_uniform():
    # jitter inside each stratum is uniform: over many queries the offset
    # within a stratum of width 10 has a flat histogram
    offs = []
    for qi in range(4000):
        ep = oracle.entry_points(0, 159, 16, 123, qi)
        offs.extend((ep - np.arange(16) * 10).tolist())
    h = np.bincount(offs, minlength=10)
    assert h.min() > 0.85 * h.mean() and h.max() < 1.15 * h.mean()


# ------------------------------------------------------------------ P6 EN(u)

# second sampling reading: a rank priority shared by all queries

def _shared_sample_python(l, r, E, seed):
    """The sample written out with Python integers: priorities from the
    (pinned) SplitMix64, threshold ceil(E * 2^32 / cnt) in exact arithmetic."""
    cnt = r - l + 1
    T = 1 << 32 if cnt <= E else min(1 << 32, -((-E << 32) // cnt))
    key = oracle.splitmix64(seed)
    return [i for i in range(l, r + 1) if (oracle.splitmix64(key ^ i) >> 32) < T]


def test_entry_threshold_closed_form():
    for cnt, E in [(1, 16), (16, 16), (17, 16), (1000, 3), (999_999, 2560), (1_000_000, 2560),
                   (3, 2), (2 ** 31 - 1, 2 ** 30), (123_457, 1)]:
        want = 1 << 32 if cnt <= E else min(1 << 32, -((-E << 32) // cnt))
        assert oracle.entry_threshold(cnt, E) == want, (cnt, E)


def test_entry_priority_is_splitmix_high_word():
    for seed in (0, 1, 0xDEADBEEF, 2 ** 63 + 5):
        for i in (0, 1, 2, 999_999, 2 ** 31 - 1):
            assert oracle.entry_priority(seed, i) == oracle.splitmix64(oracle.splitmix64(seed) ^ i) >> 32


def test_entry_points_shared_membership():
    for (l, r, E, seed) in [(0, 9, 16, 0), (5, 5, 16, 3), (100, 5099, 64, 0), (0, 99_999, 2560, 0),
                            (31_000, 95_000, 700, 7), (10, 400, 390, 1)]:
        got = oracle.entry_points_shared(l, r, E, seed).tolist()
        assert got == _shared_sample_python(l, r, E, seed), (l, r, E, seed)
        if r - l + 1 <= E:
            assert got == list(range(l, r + 1))


def test_entry_points_shared_size_nesting_and_sharing():
    # each rank is included with probability E/cnt, independently: the size is
    # binomial around E and the positions are uniform over the range
    l, r, E = 1000, 200_999, 2560
    sizes, hist = [], np.zeros(10)
    for seed in range(40):
        s = oracle.entry_points_shared(l, r, E, seed)
        sizes.append(len(s))
        hist += np.histogram(s, bins=10, range=(l, r + 1))[0]
    p = E / (r - l + 1)
    sd = np.sqrt(E * (1 - p) / len(sizes))
    assert abs(np.mean(sizes) - E) < 4 * sd
    exp_bin = hist.sum() / 10
    assert (np.abs(hist - exp_bin) < 5 * np.sqrt(exp_bin)).all()
    # a larger E keeps every rank of a smaller one (thresholds are nested)
    a = set(oracle.entry_points_shared(l, r, 500, 3).tolist())
    b = set(oracle.entry_points_shared(l, r, 2000, 3).tolist())
    assert a <= b and len(b) > len(a)
    # two ranges with the same density agree on their overlap
    x = oracle.entry_points_shared(0, 99_999, 1000, 5)
    y = oracle.entry_points_shared(50_000, 149_999, 1000, 5)
    ov = lambda z: z[(z >= 50_000) & (z <= 99_999)].tolist()
    assert ov(x) == ov(y)


def _hand_index():
    # n=12, H=3, m=4; rows handwritten, -1 tails, duplicates across layers
    n, H, m = 12, 3, 4
    E = -np.ones((n, H, m), np.int32)
    E[5, 0] = [11, 0, 6, 3]
    E[5, 1] = [3, 4, 6, -1]
    E[5, 2] = [4, 6, -1, -1]
    E[2, 0] = [9, 10, 11, 1]
    E[2, 1] = [1, 0, 4, 5]
    E[2, 2] = [1, 0, 3, -1]
    return E


def test_en_ident_hand_examples():
    E = _hand_index()
    # range [3,6], layers 0..2, budget 16: in stored order, duplicates kept
    got, sc = oracle.en_ident(E, 5, 3, 6, 0, 2, 16)
    assert got.tolist() == [6, 3, 3, 4, 6, 4, 6] and sc == 12
    # budget 3 stops inside layer 1; entries scanned count whole layers
    got, sc = oracle.en_ident(E, 5, 3, 6, 0, 2, 3)
    assert got.tolist() == [6, 3, 3] and sc == 8
    # hotspot restricted to layers 1..2
    got, sc = oracle.en_ident(E, 5, 0, 11, 1, 2, 16)
    assert got.tolist() == [3, 4, 6, 4, 6] and sc == 8
    # nothing in range
    got, sc = oracle.en_ident(E, 2, 6, 8, 0, 2, 16)
    assert got.tolist() == [] and sc == 12
    # list-comprehension restatement of Alg. 4 on random rows
    rng = np.random.default_rng(5)
    R = rng.integers(-1, 40, (40, 5, 8)).astype(np.int32)
    for _ in range(300):
        u = int(rng.integers(0, 40))
        l, r = sorted(rng.integers(0, 40, 2).tolist())
        Ls = int(rng.integers(0, 5))
        Le = int(rng.integers(Ls, 5))
        B = int(rng.integers(1, 20))
        flat = [v for h in range(Ls, Le + 1) for v in R[u, h] if v != -1 and l <= v <= r]
        got, _ = oracle.en_ident(R, u, l, r, Ls, Le, B)
        assert got.tolist() == flat[:B]


# ------------------------------------------------------------------ P2 exact

def test_exact_matches_numpy_lexsort():
    w = workloads.make("tiny", n=3000, nq=40)
    perm = np.argsort(w.attr, kind="stable").astype(np.int32)
    srt = w.attr[perm]
    Xr = w.X[perm]
    ids, ds = oracle.exact(Xr, srt, perm, w.Q, w.lo, w.hi, 10)
    for i in range(w.nq):
        l = np.searchsorted(srt, w.lo[i], "left")
        r = np.searchsorted(srt, w.hi[i], "right") - 1
        D = ((Xr[l:r + 1].astype(np.float64) - w.Q[i].astype(np.float64)) ** 2).sum(1).astype(np.float32)
        rank = np.arange(l, r + 1)
        o = np.lexsort((rank, D))[:10]
        assert (ids[i, :len(o)] == perm[rank[o]]).all()
        assert np.allclose(ds[i, :len(o)], D[o], rtol=1e-6, atol=0)
        assert (ids[i, len(o):] == -1).all()


def test_exact_breaks_distance_ties_by_rank():
    # integer-valued vectors: many exactly equal distances; order must be
    # (distance, rank), as numpy lexsort gives
    rng = np.random.default_rng(11)
    n, d = 2000, 4
    X = rng.integers(-2, 3, (n, d)).astype(np.float32)
    attr = rng.permutation(n).astype(np.float64)
    perm = np.argsort(attr, kind="stable").astype(np.int32)
    Xr, srt = X[perm], attr[perm]
    Q = rng.integers(-2, 3, (30, d)).astype(np.float32)
    lo = np.zeros(30)
    hi = np.full(30, n - 1.0)
    ids, ds = oracle.exact(Xr, srt, None, Q, lo, hi, 25, rank_ids=True)
    for i in range(30):
        D = ((Xr.astype(np.float64) - Q[i].astype(np.float64)) ** 2).sum(1)
        o = np.lexsort((np.arange(n), D))[:25]
        assert ids[i].tolist() == o.tolist()


def test_exact_empty_and_short_ranges():
    w = workloads.make("tiny", n=500, nq=4)
    perm = np.argsort(w.attr, kind="stable").astype(np.int32)
    srt = w.attr[perm]
    lo = np.array([10.0, 300.0, np.nan, 499.0])
    hi = np.array([12.0, 200.0, 5.0, 1e9])
    ids, ds = oracle.exact(w.X[perm], srt, perm, w.Q, lo, hi, 5)
    assert (ids[0, :3] >= 0).all() and (ids[0, 3:] == -1).all() and np.isinf(ds[0, 3:]).all()
    assert (ids[1] == -1).all() and (ids[2] == -1).all()
    assert ids[3, 0] == perm[499] and (ids[3, 1:] == -1).all()


# ------------------------------------------------------------------ fusion distance

def test_fusion_special_values():
    # beta = 0 reduces to the vector distance
    assert oracle.fusion(9.0, 3, 70, 100, 0.0, 0.5) == 3.0
    # maximal attribute distance (|ru - rv| = len - 1) leaves it unchanged
    assert oracle.fusion(16.0, 0, 99, 100, 0.2, 0.5) == 4.0
    # delta_a = 1/4, gamma = 1/2 -> weight 1 - 0.2 * (1 - 0.5) = 0.9
    assert abs(oracle.fusion(4.0, 10, 35, 101, 0.2, 0.5) - 1.8) < 1e-15
    # the weight only depends on |ru - rv| and grows with it
    a = oracle.fusion(1.0, 10, 15, 101, 0.2, 0.5)
    b = oracle.fusion(1.0, 15, 10, 101, 0.2, 0.5)
    c = oracle.fusion(1.0, 10, 60, 101, 0.2, 0.5)
    assert a == b and a < c < 1.0 and a > 0.8


def test_fusion_shift_constant():
    # Sec 5.2: C_gamma = Cov(Z, Z^gamma) = gamma / (2 (gamma+1)(gamma+2)) for Z ~ U(0,1);
    # checked by quadrature, and 1/15 at gamma = 1/2
    z = (np.arange(2_000_000) + 0.5) / 2_000_000
    for g in (0.25, 0.5, 1.0, 2.0):
        cov = (z * z ** g).mean() - z.mean() * (z ** g).mean()
        assert abs(cov - g / (2 * (g + 1) * (g + 2))) < 1e-6
    assert abs(0.5 / (2 * 1.5 * 2.5) - 1 / 15) < 1e-15


# ------------------------------------------------------------------ build

@pytest.fixture(scope="module")
def tiny_index():
    w = workloads.make("tiny", n=3000, nq=200)
    ix = oracle.build(w.X, w.attr)
    return w, ix


def test_build_structure(tiny_index):
    w, ix = tiny_index
    n, H, m = ix.ENC.shape
    assert H == oracle.num_layers(n, 7) and m == 16
    assert (ix.perm == np.argsort(w.attr, kind="stable")).all()
    assert (ix.X_rank == w.X[ix.perm]).all()
    for h in range(H):
        for u in range(0, n, 7):
            row = ix.ENC[u, h]
            valid = row[row != -1]
            # -1 only at the tail, no self, distinct, inside u's layer-h segment
            assert (row[len(valid):] == -1).all()
            assert u not in valid and len(set(valid.tolist())) == len(valid)
            s, e = oracle.segment(n, h, u)
            assert ((valid >= s) & (valid <= e)).all()
            # ascending fusion distance w.r.t. the segment length
            keys = [oracle.fusion(oracle.dist(ix.X_rank[u], ix.X_rank[v]), u, int(v), e - s + 1, 0.2, 0.5)
                    for v in valid]
            assert all(keys[i] <= keys[i + 1] for i in range(len(keys) - 1))
            if e - s + 1 > m:
                assert len(valid) == m


def test_build_leaf_layer_is_exact_fusion_topm(tiny_index):
    w, ix = tiny_index
    n, H, m = ix.ENC.shape
    h = H - 1
    Xr = ix.X_rank.astype(np.float64)
    for u in range(0, n, 37):
        s, e = oracle.segment(n, h, u)
        cand = [v for v in range(s, e + 1) if v != u]
        D = ((Xr[cand] - Xr[u]) ** 2).sum(1).astype(np.float32)
        keys = np.array([oracle.fusion(float(dv), u, v, e - s + 1, 0.2, 0.5) for dv, v in zip(D, cand)])
        order = np.lexsort((np.array(cand), keys))[:m]
        assert ix.ENC[u, h].tolist() == [cand[i] for i in order]


def test_build_beta0_leaf_is_vector_topm():
    # with beta = 0 the leaf ENC rows are the plain vector top-m (numpy)
    w = workloads.make("tiny", n=700, nq=1)
    ix = oracle.build(w.X, w.attr, beta=0.0)
    n, H, m = ix.ENC.shape
    Xr = ix.X_rank.astype(np.float64)
    for u in range(0, n, 11):
        s, e = oracle.segment(n, H - 1, u)
        cand = np.array([v for v in range(s, e + 1) if v != u])
        D = ((Xr[cand] - Xr[u]) ** 2).sum(1).astype(np.float32)
        assert ix.ENC[u, H - 1].tolist() == cand[np.lexsort((cand, D))[:m]].tolist()


def test_boundary_effect_closed_form():
    # Eq. naive_attr_dist: vector top-m inside a segment with attributes
    # independent of vectors -> mean rank distance (l+1)/3 over positions,
    # l/2 at the boundary.  The beta=0 leaf layer is exactly that method.
    rng = np.random.default_rng(6)
    n, d = 4096, 8
    X = rng.standard_normal((n, d)).astype(np.float32)
    attr = rng.permutation(n).astype(np.float64)
    ix = oracle.build(X, attr, beta=0.0, n_inv=5, m=1)   # leaves of 256, nearest neighbour only
    H = ix.H
    seglen = n >> (H - 1)
    u = np.arange(n)
    v = ix.ENC[:, H - 1, 0]
    dist = np.abs(u - v)
    assert abs(dist.mean() - (seglen + 1) / 3) < 0.05 * seglen / 3
    t = u % seglen
    bd = dist[(t == 0) | (t == seglen - 1)].mean()
    assert abs(bd - seglen / 2) < 0.1 * seglen / 2
    # fusion (beta > 0) pulls candidates closer in rank (Eq. fusion_attr_first_order)
    ix2 = oracle.build(X, attr, beta=0.5, n_inv=5, m=1)
    assert np.abs(u - ix2.ENC[:, H - 1, 0]).mean() < dist.mean()



# ------------------------------------------------------------------ construction: inductive step
#
# Sec 6.1 builds a parent layer from (i) the vertex's m-ANN in its own child
# (the child's temporary PG row), (ii) its m-ANN in the sibling child, found
# by the greedy search of Alg 1 over the sibling's temporary PG with the
# patience stop of Sec 6.2.2; the 2m set is RNG-pruned into the parent's
# temporary PG row and re-ranked by fusion distance into the ENC row.  The
# expected rows below are worked out by hand from the RNG rule (keep a
# candidate c, taken in ascending distance to u, unless an already kept k has
# delta(c, k) < delta(u, c); stop at m kept; top up with the nearest pruned).

def _sq(a, b):
    return oracle.dist(np.asarray(a, np.float32), np.asarray(b, np.float32))


def test_rng_prune_hand_1d():
    # u = 0 on a line; candidates (id: position, squared distance to u):
    # 1: 1 (1), 4: -1.5 (2.25), 2: 2 (4), 3: 3 (9), 5: -4 (16)
    X = np.array([[0.0], [1.0], [2.0], [3.0], [-1.5], [-4.0]], np.float32)
    ids = np.array([1, 4, 2, 3, 5], np.int32)
    dd = np.array([_sq(X[0], X[i]) for i in ids], np.float32)
    assert dd.tolist() == [1.0, 2.25, 4.0, 9.0, 16.0]
    # 1 kept; 4: delta(4,1) = 6.25 >= 2.25 kept; 2: delta(2,1) = 1 < 4 pruned;
    # 3: delta(3,1) = 4 < 9 pruned; 5: delta(5,4) = 6.25 < 16 pruned.
    # kept [1, 4]; the pruned in ascending distance: 2, 3, 5
    assert oracle.rng_prune(X, ids, dd, 1).tolist() == [1]
    assert oracle.rng_prune(X, ids, dd, 2).tolist() == [1, 4]
    assert oracle.rng_prune(X, ids, dd, 3).tolist() == [1, 4, 2]
    assert oracle.rng_prune(X, ids, dd, 4).tolist() == [1, 4, 2, 3]
    assert oracle.rng_prune(X, ids, dd, 5).tolist() == [1, 4, 2, 3, 5]
    assert oracle.rng_prune(X, ids, dd, 7).tolist() == [1, 4, 2, 3, 5, -1, -1]


def test_rng_prune_hand_2d():
    # u = (0,0); a = (1,0) d 1, c = (1.2,0.3) d 1.53, b = (0,1.5) d 2.25,
    # e = (-2,0) d 4, f = (2,2) d 8  (ids 1, 3, 2, 4, 5 in that order)
    X = np.array([[0, 0], [1, 0], [0, 1.5], [1.2, 0.3], [-2, 0], [2, 2]], np.float32)
    ids = np.array([1, 3, 2, 4, 5], np.int32)
    dd = np.array([_sq(X[0], X[i]) for i in ids], np.float32)
    assert (np.diff(dd) > 0).all()
    # a kept; c: delta(c,a) = 0.13 < 1.53 pruned; b: delta(b,a) = 3.25 >= 2.25
    # kept; e: delta(e,a) = 9, delta(e,b) = 6.25, both >= 4, kept;
    # f: delta(f,a) = 5 < 8 pruned.  Kept [a, b, e]; pruned c, f.
    assert oracle.rng_prune(X, ids, dd, 2).tolist() == [1, 2]
    assert oracle.rng_prune(X, ids, dd, 3).tolist() == [1, 2, 4]
    assert oracle.rng_prune(X, ids, dd, 4).tolist() == [1, 2, 4, 3]
    assert oracle.rng_prune(X, ids, dd, 5).tolist() == [1, 2, 4, 3, 5]


def test_rng_prune_tie_keeps_candidate():
    # c2 = (0.5, 1) lies on the bisector of u = (0,0) and c1 = (1,0):
    # delta(c2, c1) = delta(u, c2) = 1.25 exactly.  The rule prunes only on a
    # strictly closer kept neighbour, so c2 stays; c3 = (-3, 0) is kept too
    # (delta(c3,c1) = 16, delta(c3,c2) = 13.25, both >= 9).
    X = np.array([[0, 0], [1, 0], [0.5, 1], [-3, 0]], np.float32)
    ids = np.array([1, 2, 3], np.int32)
    dd = np.array([_sq(X[0], X[i]) for i in ids], np.float32)
    assert dd.tolist() == [1.0, 1.25, 9.0] and _sq(X[2], X[1]) == dd[1]
    assert oracle.rng_prune(X, ids, dd, 3).tolist() == [1, 2, 3]


def _seq_sqdist(A, b):
    """Squared L2 of every row of A to b, summed dimension by dimension in
    float64 (one rounding to float32 at the end)."""
    A = np.asarray(A, np.float64)
    b = np.asarray(b, np.float64)
    s = np.zeros(A.shape[0])
    for i in range(A.shape[1]):
        t = A[:, i] - b[i]
        s = s + t * t
    return s.astype(np.float32)


def test_sibling_search_all_seeded_is_exact_topm():
    # every vertex of the segment seeded: the pool starts with the ef nearest
    # of them, so its top m is the exact top m whatever the graph, and no
    # expansion adds anything (each is non-improving: the search stops after
    # `patience` expansions, or when the pool has none left)
    rng = np.random.default_rng(11)
    n, d, m = 200, 8, 8
    X = rng.standard_normal((n, d)).astype(np.float32)
    ts, te = 50, 149
    PG = rng.integers(ts, te + 1, size=(n, m)).astype(np.int32)
    for trial in range(5):
        xq = rng.standard_normal(d).astype(np.float32)
        seeds = np.arange(ts, te + 1, dtype=np.int32)
        rng.shuffle(seeds)
        res, resd, nexp = oracle.sibling_search(X, PG, xq, ts, te, seeds, ef=32, patience=5)
        cand = np.arange(ts, te + 1)
        D = _seq_sqdist(X[cand], xq)
        order = np.lexsort((cand, D))[:m]
        assert res.tolist() == cand[order].tolist()
        assert resd.tolist() == D[order].tolist()
        assert nexp == 5
    res, _, nexp = oracle.sibling_search(X, PG, xq, ts, te, seeds[:3], ef=32, patience=50)
    assert nexp <= 100


def _chain_pg(n, rows):
    PG = np.full((n, 1), -1, np.int32)
    for u, v in rows.items():
        PG[u, 0] = v
    return PG


@pytest.mark.parametrize("patience", [2, 4, 7])
def test_sibling_search_patience_chain(patience):
    # Points on a line, query at 3.2, m = 1, one seed (vertex 0 at 0).  Chain
    # i -> i+1 with vertex i at position i (0..K), then K -> h, a vertex at
    # 3.25 (nearer to the query than 3).  Best-first follows the chain (each
    # expansion adds exactly one new vertex, the only unexpanded one):
    # expanding 0, 1, 2 adds 1, 2, 3, each a new nearest (improving);
    # expanding 3, 4, ... adds 4, 5, ..., never a new nearest.  After
    # `patience` such expansions in a row (of 3 .. patience+2) the search
    # stops.  So with K = patience + 2 the last of them adds h (improving)
    # and h is found; with K = patience + 3 the search stops after expanding
    # patience + 2 and never reaches h.
    p = patience
    for K, found in ((p + 2, True), (p + 3, False)):
        h = K + 1
        X = np.array([[float(i)] for i in range(K + 1)] + [[3.25]], np.float32)
        PG = _chain_pg(K + 2, {**{i: i + 1 for i in range(K)}, K: h})
        xq = np.array([3.2], np.float32)
        res, _, nexp = oracle.sibling_search(X, PG, xq, 0, K + 1, np.array([0], np.int32), ef=64,
                                            patience=p)
        if found:
            # 0..K expanded, then h (which adds nothing)
            assert res.tolist() == [h] and nexp == K + 2
        else:
            # 0 .. p+2 expanded
            assert res.tolist() == [3] and nexp == p + 3


def test_sibling_search_patience_resets_on_improvement():
    # Query at 0, m = 1, patience 3, seed vertex 0.  Chain v0 -> v1 -> ... ->
    # v7 with positions 5, 4, 4.5, 4.6, 3, 3.5, 3.6, 1 (squared 25, 16,
    # 20.25, 21.16, 9, 12.25, 12.96, 1).  Expansion (adds; new nearest?;
    # patience left): v0 (v1; yes; 3), v1 (v2; no; 2), v2 (v3; no; 1),
    # v3 (v4; yes; 3), v4 (v5; no; 2), v5 (v6; no; 1), v6 (v7; yes; 3),
    # v7 (nothing; no; 2), then no unexpanded vertex is left.  The nearest
    # is v7 after 8 expansions; without the reset the search would stop
    # after expanding v4 with v4 as the nearest.
    pos = [5, 4, 4.5, 4.6, 3, 3.5, 3.6, 1]
    X = np.array([[x] for x in pos], np.float32)
    PG = _chain_pg(8, {i: i + 1 for i in range(7)})
    res, resd, nexp = oracle.sibling_search(X, PG, np.array([0.0], np.float32), 0, 7,
                                            np.array([0], np.int32), ef=64, patience=3)
    assert res.tolist() == [7] and resd.tolist() == [1.0] and nexp == 8


def _restated_build_all_seeded(X, attr, m, H, beta, gamma):
    """The construction of Sec 6 for the case where every sibling vertex is a
    seed of the sibling search, so that search returns the sibling's exact
    m-ANN: leaf rows by brute force, then per layer the child's temporary-PG
    row plus the sibling's exact top m, RNG prune, fusion re-rank."""
    n, d = X.shape
    order = np.argsort(attr, kind="stable")
    Xr = X[order]
    # segments per depth by explicit halving: left [L, mid], right [mid+1, R]
    segs = [[(0, n - 1)]]
    for _ in range(H - 1):
        nxt = []
        for (a, b) in segs[-1]:
            mid = a + (b - a) // 2
            nxt += [(a, mid), (mid + 1, b)]
        segs.append(nxt)
    seg_of = []
    for lay in segs:
        t = np.empty(n, np.int64)
        for i, (a, b) in enumerate(lay):
            t[a:b + 1] = i
        seg_of.append(t)
    D = np.stack([_seq_sqdist(Xr, Xr[u]) for u in range(n)])   # D[u, v]

    def fusion_key(u, v, seglen):
        da = abs(u - v) / (seglen - 1)
        return math.sqrt(float(D[u, v])) * (1.0 - beta * (1.0 - da ** gamma))

    ENC = np.full((n, H, m), -1, np.int32)
    PG = [[] for _ in range(n)]
    h = H - 1
    for u in range(n):
        a, b = segs[h][seg_of[h][u]]
        cand = [v for v in range(a, b + 1) if v != u]
        ENC[u, h, :min(m, len(cand))] = sorted(cand, key=lambda v: (fusion_key(u, v, b - a + 1), v))[:m]
        PG[u] = sorted(cand, key=lambda v: (D[u, v], v))[:m]
    for h in range(H - 2, -1, -1):
        newPG = [None] * n
        for u in range(n):
            a, b = segs[h][seg_of[h][u]]
            mid = a + (b - a) // 2
            sib = range(mid + 1, b + 1) if u <= mid else range(a, mid + 1)
            cand = list(PG[u]) + sorted(sib, key=lambda v: (D[u, v], v))[:m]
            cand.sort(key=lambda v: (D[u, v], v))
            kept = []
            for c in cand:
                if len(kept) == m:
                    break
                if all(not (D[c, k] < D[u, c]) for k in kept):
                    kept.append(c)
            kept += [c for c in cand if c not in kept][:m - len(kept)]
            newPG[u] = kept
            fus = sorted(cand, key=lambda v: (fusion_key(u, v, b - a + 1), v))[:m]
            ENC[u, h, :len(fus)] = fus
        PG = newPG
    return ENC


def test_build_all_seeded_equals_restatement():
    # n = 100: the root's children hold 50 ranks, so 64 seeds cover every
    # sibling at every layer
    rng = np.random.default_rng(12)
    n, d, m = 100, 8, 4
    X = rng.standard_normal((n, d)).astype(np.float32)
    attr = rng.permutation(n).astype(np.float64)
    for beta, gamma in ((0.2, 0.5), (0.0, 0.5), (0.5, 2.0)):
        ix = oracle.build(X, attr, m=m, ef_c=16, n_inv=3, patience=30, sib_seeds=64, beta=beta, gamma=gamma)
        assert ix.H == 5
        ref = _restated_build_all_seeded(X, attr, m, ix.H, beta, gamma)
        assert (ix.ENC == ref).all(), np.argwhere(ix.ENC != ref)[:5]

# ------------------------------------------------------------------ search

def _bruteforce_rank_space(ix, q, l, r, k):
    D = ((ix.X_rank[l:r + 1].astype(np.float64) - q.astype(np.float64)) ** 2).sum(1).astype(np.float32)
    rank = np.arange(l, r + 1)
    o = np.lexsort((rank, D))[:k]
    return rank[o], D[o]


def test_search_equals_bruteforce_when_range_fits_entry_set(tiny_index):
    # P8a: cnt <= epn -> every in-range vertex is an entry point -> exact
    w, ix = tiny_index
    rng = np.random.default_rng(7)
    nq = 60
    start = rng.integers(0, ix.n - 40, nq)
    cnt = rng.integers(1, 40, nq)
    lo = start.astype(np.float64)
    hi = (start + cnt - 1).astype(np.float64)
    Q = w.Q[:nq]
    ids, ds, st = oracle.search(ix, Q, lo, hi, 10, 64, epn=48, rank_ids=True)
    gi, gd = oracle.exact(ix.X_rank, ix.attr_sorted, None, Q, lo, hi, 10, rank_ids=True)
    assert (ids == gi).all() and (ds == gd).all()


def test_search_large_pool_equals_closure_topk(tiny_index):
    # P8b: with L >= n nothing is evicted, so the result is the exact top-k of
    # the closure of the entry set under EN(.)
    w, ix = tiny_index
    n = ix.n
    for i in range(0, 24):
        q, lo, hi = w.Q[i], w.lo[i], w.hi[i]
        l, r = oracle.rank_bounds(ix.attr_sorted, lo, hi)
        Ls, Le = oracle.hotspot(l, r, ix.H, n)
        ep = oracle.entry_points(l, r, 16, 0, i)
        reach = oracle.closure(ix, l, r, Ls, Le, 16, ep)
        ids, ds, st = oracle.search(ix, q[None], [lo], [hi], 10, n, qidx=[i], rank_ids=True)
        vs = np.nonzero(reach)[0]
        D = ((ix.X_rank[vs].astype(np.float64) - q.astype(np.float64)) ** 2).sum(1).astype(np.float32)
        o = np.lexsort((vs, D))[:10]
        kk = len(o)
        assert ids[0, :kk].tolist() == vs[o].tolist()
        assert st[0, oracle.STAT_DIST] == reach.sum()          # every reachable vertex evaluated once
        assert st[0, oracle.STAT_EXPANSIONS] == reach.sum()    # and expanded once
        if reach.sum() == r - l + 1:                            # closure = whole range -> brute force
            bi, _ = _bruteforce_rank_space(ix, q, l, r, 10)
            assert ids[0, :kk].tolist() == bi.tolist()


def _textbook_kann(adj, dist_fn, entries, ef, k):
    """Alg. 1 written independently: pool of (dist, id) kept sorted, expand the
    closest unexpanded, insert every not-yet-computed neighbour, truncate."""
    computed = set()
    pool = []
    for e in entries:
        if e not in computed:
            computed.add(e)
            pool.append((dist_fn(e), e))
    pool = sorted(pool)[:ef]
    expanded = set()
    while True:
        nxt = [p for p in pool if p[1] not in expanded]
        if not nxt:
            break
        u = nxt[0][1]
        expanded.add(u)
        for v in adj(u):
            if v not in computed:
                computed.add(v)
                pool.append((dist_fn(v), v))
        pool = sorted(pool)[:ef]
    return [p[1] for p in pool[:k]], [p[0] for p in pool[:k]]


def test_search_full_range_equals_textbook_greedy(tiny_index):
    # P8c: full range, B <= m, no -1 in layer 0 -> L_start = 0 and EN(u) is the
    # first B entries of u's layer-0 row, so FROGSearch is Alg. 1 over that graph
    w, ix = tiny_index
    assert (ix.ENC[:, 0, :] != -1).all()
    n = ix.n
    B = 12
    for i in range(12):
        q = w.Q[i]
        ep = oracle.entry_points(0, n - 1, 16, 0, i)
        qd = q.astype(np.float64)
        Xr = ix.X_rank.astype(np.float64)
        # the whole pool (k = L), not only the top 10
        ref_ids, ref_d = _textbook_kann(lambda u: ix.ENC[u, 0, :B].tolist(),
                                        lambda v: np.float32(((Xr[v] - qd) ** 2).sum()),
                                        ep.tolist(), 32, 32)
        ids, ds, _ = oracle.search(ix, q[None], [-np.inf], [np.inf], 32, 32, B=B, qidx=[i], rank_ids=True)
        assert ids[0].tolist() == ref_ids


def test_search_invariants_tiny_workload():
    # P9 on the tiny workload: ids in range, distinct, ascending, distances
    # equal to a numpy recomputation, expansions <= distance evaluations
    w = workloads.make("tiny")
    ix = oracle.build(w.X, w.attr)
    ids, ds, st = oracle.search(ix, w.Q, w.lo, w.hi, w.k, 64, rank_ids=True)
    for i in range(w.nq):
        l, r = oracle.rank_bounds(ix.attr_sorted, w.lo[i], w.hi[i])
        row = ids[i][ids[i] >= 0]
        assert ((row >= l) & (row <= r)).all() and len(set(row.tolist())) == len(row)
        assert (np.diff(ds[i][:len(row)]) >= 0).all()
        ref = ((ix.X_rank[row].astype(np.float64) - w.Q[i].astype(np.float64)) ** 2).sum(1)
        assert np.allclose(ds[i][:len(row)], ref.astype(np.float32), rtol=2e-7, atol=0)
        assert st[i, oracle.STAT_EXPANSIONS] <= st[i, oracle.STAT_DIST]
        assert len(row) == min(w.k, r - l + 1)
    # recall against exhaustive search is high on this easy workload
    gi, _ = oracle.exact(ix.X_rank, ix.attr_sorted, None, w.Q, w.lo, w.hi, w.k, rank_ids=True)
    rec = np.mean([len(set(ids[i]) & set(gi[i])) / w.k for i in range(w.nq)])
    assert rec > 0.8


def test_search_degenerate_queries(tiny_index):
    w, ix = tiny_index
    Q = w.Q[:5]
    lo = np.array([100.0, 5.0, np.nan, 0.0, 2999.0])
    hi = np.array([99.0, 5.0, 10.0, 2.0, 5000.0])
    ids, ds, st = oracle.search(ix, Q, lo, hi, 10, 64, rank_ids=True)
    assert (ids[0] == -1).all() and np.isinf(ds[0]).all()
    assert ids[1, 0] == 5 and (ids[1, 1:] == -1).all()
    assert (ids[2] == -1).all()
    assert sorted(ids[3, :3].tolist()) == [0, 1, 2] and (ids[3, 3:] == -1).all()
    assert ids[4, 0] == 2999 and (ids[4, 1:] == -1).all()


def test_search_shared_entries_without_edges_is_entry_topk(tiny_index):
    # an index without edges: the result is the k nearest of the entry sample,
    # which is rebuilt here from its definition
    w, ix = tiny_index
    bare = oracle.OracleIndex(ix.perm, ix.attr_sorted, ix.X_rank, np.full_like(ix.ENC, -1))
    rng = np.random.default_rng(11)
    for i in range(16):
        l = int(rng.integers(0, ix.n - 200))
        r = int(rng.integers(l, min(ix.n, l + 2500)))
        E = 150
        sample = np.array(_shared_sample_python(l, r, E, 9), np.int64)
        q = w.Q[i]
        ids, ds, st = oracle.search(bare, q[None], [float(l)], [float(r)], 10, 32, epn=16, epn_frac=1.0,
                                    epn_max=E, seed=9, entry_mode=1, rank_ids=True)
        D = ((ix.X_rank[sample].astype(np.float64) - q.astype(np.float64)) ** 2).sum(1).astype(np.float32)
        o = np.lexsort((sample, D))[:10]
        assert ids[0, :len(o)].tolist() == sample[o].tolist()
        assert ds[0, :len(o)].tolist() == D[o].tolist()
        assert st[0, oracle.STAT_ENTRY] == len(sample) == st[0, oracle.STAT_DIST]
        assert st[0, oracle.STAT_EXPANSIONS] == min(32, len(sample))


def test_search_shared_full_range_equals_textbook_greedy(tiny_index):
    # P8c with the shared sample as the entry set (entry points are visited)
    w, ix = tiny_index
    n = ix.n
    B = 12
    for i in range(8):
        q = w.Q[i]
        ep = _shared_sample_python(0, n - 1, 40, i)
        qd = q.astype(np.float64)
        Xr = ix.X_rank.astype(np.float64)
        ref_ids, ref_d = _textbook_kann(lambda u: ix.ENC[u, 0, :B].tolist(),
                                        lambda v: np.float32(((Xr[v] - qd) ** 2).sum()),
                                        ep, 32, 32)
        ids, ds, st = oracle.search(ix, q[None], [-np.inf], [np.inf], 32, 32, B=B, epn=16, epn_frac=1.0,
                                    epn_max=40, seed=i, entry_mode=1, rank_ids=True)
        assert ids[0].tolist() == ref_ids
        assert st[0, oracle.STAT_ENTRY] == len(ep)


def test_search_shared_small_range_is_exact(tiny_index):
    # cnt <= E: the shared sample is the whole range, so the result is exact
    w, ix = tiny_index
    rng = np.random.default_rng(12)
    nq = 40
    start = rng.integers(0, ix.n - 60, nq)
    cnt = rng.integers(1, 60, nq)
    lo = start.astype(np.float64)
    hi = (start + cnt - 1).astype(np.float64)
    ids, ds, _ = oracle.search(ix, w.Q[:nq], lo, hi, 10, 32, epn=64, entry_mode=1, rank_ids=True)
    gi, gd = oracle.exact(ix.X_rank, ix.attr_sorted, None, w.Q[:nq], lo, hi, 10, rank_ids=True)
    assert (ids == gi).all() and (ds == gd).all()


# ------------------------------------------------------------------ ablations (Sec 8.2.3)

def _textbook_frog(ix, q, l, r, layers, B, entries, L, eager):
    """Alg. 2 written independently for the ablations: EN(u) = the in-range
    entries of u's rows over `layers` in stored order, at most B of them --
    counted before the visited check (lazy) or skipping visited ones (eager)."""
    qd = q.astype(np.float64)
    dist = lambda v: np.float32(((ix.X_rank[v].astype(np.float64) - qd) ** 2).sum())
    computed = set()
    pool = []
    for e in entries:
        if e not in computed:
            computed.add(e)
            pool.append((dist(e), e))
    pool = sorted(pool)[:L]
    expanded = set()
    while True:
        nxt = [p for p in pool if p[1] not in expanded]
        if not nxt:
            break
        u = nxt[0][1]
        expanded.add(u)
        en = []
        for h in layers:
            for v in ix.ENC[u, h].tolist():
                if v == -1 or not (l <= v <= r):
                    continue
                if eager:
                    if v in computed:
                        continue
                    computed.add(v)
                en.append(v)
                if len(en) == B:
                    break
            if len(en) == B:
                break
        for v in en:
            if eager:
                pool.append((dist(v), v))
            elif v not in computed:
                computed.add(v)
                pool.append((dist(v), v))
        pool = sorted(pool)[:L]
    return [p[1] for p in pool]


@pytest.mark.parametrize("hot_mode,eager", [(0, False), (1, False), (2, False), (0, True), (2, True)])
def test_search_ablations_equal_textbook(tiny_index, hot_mode, eager):
    w, ix = tiny_index
    n, H = ix.n, ix.H
    rng = np.random.default_rng(13)
    for i in range(10):
        cnt = int(rng.integers(60, n // 2))
        l = int(rng.integers(0, n - cnt))
        r = l + cnt - 1
        Ls, Le = oracle.hotspot(l, r, H, n)
        layers = {0: range(Ls, Le + 1), 1: range(Ls, H), 2: range(0, H)}[hot_mode]
        ep = oracle.entry_points(l, r, 16, 0, i)
        ref = _textbook_frog(ix, w.Q[i], l, r, list(layers), 8, ep.tolist(), 24, eager)
        ids, _, st = oracle.search(ix, w.Q[i][None], [float(l)], [float(r)], 24, 24, B=8, qidx=[i],
                                   hot_mode=hot_mode, eager=eager, rank_ids=True)
        assert ids[0][:len(ref)].tolist() == ref, (hot_mode, eager, i)
        assert (st[0, oracle.STAT_LS], st[0, oracle.STAT_LE]) == (min(layers), max(layers))
