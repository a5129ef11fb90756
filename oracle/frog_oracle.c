/*
 * FROG range-filtered k-NN search — CPU ORACLE (test infrastructure only).
 *
 * This file is a plain, slow, deliberately simple restatement of the method of
 * "FROG: Efficient Range-Filtering Approximate Nearest Neighbor Search on GPUs"
 * (arxiv 2608.16491).  It exists to check the HIP library: only the tests, the
 * package's smoke() entry and the benchmark's CPU-baseline leg load it.  It
 * shares no code, header, table or helper with the library; the two meet only
 * through plain arrays.
 *
 * Contents, each following the cited passage of the paper:
 *   fo_dist            squared L2 distance (Sec 2.1, Def. of delta_v; squared
 *                      form and precision are readings, see below)
 *   fo_rank_bounds     attribute range -> contiguous rank interval (Sec 4)
 *   fo_segment         segment of the logical segment tree containing a rank
 *                      at a given depth (Sec 4; split rule of Alg. 3)
 *   fo_num_layers      retained depth H from n and n_inv (Sec 4)
 *   fo_hotspot         HotspotLocalization (Alg. 3, Rules 1-2, Eq. endcondition)
 *   fo_entry_points    entry-point sampling (Alg. 2, uniform sampling from the
 *                      range; deterministic stratified reading)
 *   fo_entry_points_shared  the same sampling with a per-rank random priority
 *                      shared by all queries (second reading, below)
 *   fo_en_ident        ENIdentification (Alg. 4): scan hotspot layers in stored
 *                      order, keep in-range candidates, stop at budget B
 *   fo_search_batch    FROGSearch (Alg. 2) with an exact visited set, and the
 *                      ablation variants of Sec 8.2.3 (hotspot without its end
 *                      condition or without localisation; eager visited check)
 *   fo_exact_batch     exhaustive filtered k-NN (Def. 2, RFANNS), the ground
 *                      truth the search approximates
 *   fo_build           index construction (Sec 6: leaf brute force, then per
 *                      layer child m-ANN + sibling greedy search (Alg. 1 with
 *                      patience), RNG prune -> temporary PG, fusion re-rank
 *                      (Eq. fusion-distance) -> ENC row)
 *   fo_rng_prune_list, fo_sibling_search_list
 *                      the construction's RNG prune (Sec 6.1) and sibling
 *                      search with the patience stop (Sec 6.2.2) on their own,
 *                      so that the tests can pin them on hand-built inputs
 *
 * Readings where the paper is silent (the same readings bind the library):
 *   - distances are SQUARED L2, accumulated in double from float inputs in
 *     index order and rounded once to float; ordering everywhere is by
 *     (distance, id) ascending;
 *   - the invalid candidate marker is -1;
 *   - the boundary terms of Eq. endcondition use segment start positions:
 *     b_l = end of the segment holding l, plus one; b_r = start of the segment
 *     holding r; the test is (b_l-l + r-b_r) * 2^h >= r-l in integers;
 *   - entry points: the count is epn, or, when epn_frac > 0, the per-query
 *     count clamp(ceil(epn_frac * cnt), epn, epn_max) for a range of cnt ranks;
 *     all of [l,r] is used if it holds at most that many ranks, else one rank
 *     per stratum j of [l,r] split into equal strata, at offset
 *     (hi32(splitmix64(seed ^ (query_index << 32) ^ j)) * width) >> 32 inside
 *     the stratum (Lemire's multiply-shift range reduction);
 *   - second entry-point reading (entry_mode 1): every rank i carries the
 *     priority p(i) = hi32(splitmix64(splitmix64(seed) ^ i)) (the seed is
 *     mixed first so that different seeds give unrelated samples); a query whose range holds
 *     cnt ranks and asks for E entry points takes every i in [l,r] with
 *     p(i) < T, T = min(2^32, ceil(E * 2^32 / cnt)), in rank order.  Each
 *     rank of the range is included with probability E/cnt independently of
 *     the others (a uniform random sample of expected size E, all of [l,r]
 *     when cnt <= E); the sample depends on (seed, rank) only, so queries over
 *     overlapping ranges draw from the same random subset;
 *   - duplicates inside EN(u) count against B; the visited set drops them;
 *   - the loop ends when no unexpanded entry is left in the pool;
 *   - empty ranges and fewer than k results pad with (id -1, +inf);
 *   - attribute ranks: stable sort by (value, original id);
 *   - build: normalised attribute distance = |rank difference| / (len - 1)
 *     of the segment the candidates are chosen from; the leaf temporary PG is
 *     the exact vector top-m inside the leaf; the parent temporary PG is the
 *     RNG prune (alpha = 1) of the 2m candidates, topped up to m with the
 *     nearest pruned ones; the sibling search starts from `sib_seeds`
 *     stratified-jittered sibling ranks (splitmix64(seed ^ (u<<32) ^ (h<<24)
 *     ^ j), reduced the same way) and stops early after `patience` consecutive expansions that add
 *     nothing to the current top-m.
 *
 * Nothing here is tuned.  OpenMP only spreads independent queries (or the
 * independent vertices of one layer) over threads; per-item arithmetic is the
 * same sequential code.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define FO_NONE (-1)

/* ------------------------------------------------------------------------ */
/* Basic definitions                                                         */
/* ------------------------------------------------------------------------ */

/* Squared L2 distance: sum over i of (a_i - b_i)^2, each term and the running
 * sum in double, index order, one final rounding to float. */
float fo_dist(const float* a, const float* b, int d) {
    double s = 0.0;
    for (int i = 0; i < d; ++i) {
        double t = (double)a[i] - (double)b[i];
        double t2 = t * t;
        s = s + t2;
    }
    return (float)s;
}

uint64_t fo_splitmix64(uint64_t x) {
    /* SplitMix64 (Steele, Lea, Flood 2014): add the golden-ratio increment,
     * then the variant-13 finaliser of MurmurHash3 as published by Vigna. */
    uint64_t z = x + 0x9E3779B97F4A7C15ULL;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

/* ceil(log2(n)) + 1 layers make a fully expanded tree; n_inv deepest layers
 * are omitted, at least one (the root) is kept. */
int fo_num_layers(int64_t n, int n_inv) {
    int c = 0;
    while (((int64_t)1 << c) < n) ++c;
    int H = c + 1 - n_inv;
    return H < 1 ? 1 : H;
}

/* The segment at depth h holding rank p: split [0, n-1] h times with
 * mid = L + floor((R - L) / 2), left child [L, mid], right child [mid+1, R]. */
void fo_segment(int64_t n, int h, int64_t p, int64_t* s, int64_t* e) {
    int64_t L = 0, R = n - 1;
    for (int i = 0; i < h; ++i) {
        int64_t mid = L + (R - L) / 2;
        if (p <= mid) R = mid; else L = mid + 1;
    }
    *s = L;
    *e = R;
}

/* l = number of attribute values < lo, r = number of values <= hi, minus one.
 * A NaN bound gives the empty interval (l = 0, r = -1). */
void fo_rank_bounds(const double* attr_sorted, int64_t n, double lo, double hi,
                    int64_t* l, int64_t* r) {
    if (isnan(lo) || isnan(hi)) { *l = 0; *r = -1; return; }
    int64_t a = 0, b = n;
    while (a < b) { int64_t mid = a + (b - a) / 2; if (attr_sorted[mid] < lo) a = mid + 1; else b = mid; }
    *l = a;
    a = 0; b = n;
    while (a < b) { int64_t mid = a + (b - a) / 2; if (attr_sorted[mid] <= hi) a = mid + 1; else b = mid; }
    *r = a - 1;
}

/* HotspotLocalization: descend while [l,r] fits in one child (at most to depth
 * H-1); L_start is the depth reached.  Then extend L_end over consecutive
 * deeper layers h while the boundary overlap passes Eq. endcondition. */
void fo_hotspot(int64_t l, int64_t r, int H, int64_t n, int* Ls, int* Le) {
    int64_t L = 0, R = n - 1;
    int d = 0;
    while (d < H - 1) {
        int64_t mid = L + (R - L) / 2;
        if (r <= mid) R = mid;
        else if (l >= mid + 1) L = mid + 1;
        else break;
        d = d + 1;
    }
    *Ls = d;
    *Le = d;
    for (int h = d + 1; h <= H - 1; ++h) {
        int64_t sl, el, sr, er;
        fo_segment(n, h, l, &sl, &el);
        fo_segment(n, h, r, &sr, &er);
        int64_t bl = el + 1, br = sr;
        int64_t lhs = (bl - l) + (r - br);
        if (lhs * ((int64_t)1 << h) >= (r - l)) *Le = h;
        else break;
    }
}

/* An offset in [0, width) from a 64-bit random word: high 32 bits times the
 * width, high half of the product (Lemire, "Fast random integer generation
 * in an interval", 2019).  width < 2^32. */
uint64_t fo_reduce(uint64_t z, uint64_t width) {
    return ((z >> 32) * width) >> 32;
}

/* Number of entry points for a range of cnt ranks. */
int64_t fo_entry_count(int64_t cnt, int epn, double epn_frac, int epn_max) {
    int64_t e = epn;
    if (epn_frac > 0.0) {
        double want = ceil(epn_frac * (double)cnt);
        if (want > (double)epn_max) want = (double)epn_max;
        if (want > (double)e) e = (int64_t)want;
    }
    return e;
}

/* Entry points drawn from [l, r]; returns their number. */
int64_t fo_entry_points(int64_t l, int64_t r, int64_t epn, uint64_t seed, uint64_t qi, int32_t* out) {
    int64_t cnt = r - l + 1;
    if (cnt <= 0) return 0;
    if (cnt <= epn) {
        for (int64_t i = 0; i < cnt; ++i) out[i] = (int32_t)(l + i);
        return cnt;
    }
    for (int64_t j = 0; j < epn; ++j) {
        int64_t s = l + (j * cnt) / epn;
        int64_t t = l + ((j + 1) * cnt) / epn - 1;
        uint64_t z = fo_splitmix64(seed ^ (qi << 32) ^ (uint64_t)j);
        out[j] = (int32_t)(s + (int64_t)fo_reduce(z, (uint64_t)(t - s + 1)));
    }
    return epn;
}

/* Second reading of the sampling: the rank's shared priority, the threshold
 * for E expected entry points out of cnt, and the sample itself. */
uint32_t fo_entry_priority(uint64_t seed, int64_t i) {
    return (uint32_t)(fo_splitmix64(fo_splitmix64(seed) ^ (uint64_t)i) >> 32);
}

uint64_t fo_entry_threshold(int64_t cnt, int64_t E) {
    const uint64_t full = (uint64_t)1 << 32;
    if (cnt <= E) return full;
    /* ceil(E * 2^32 / cnt); E < cnt < 2^31, so E * 2^32 < 2^63 */
    uint64_t t = (((uint64_t)E << 32) + (uint64_t)cnt - 1) / (uint64_t)cnt;
    return t < full ? t : full;
}

int64_t fo_entry_points_shared(int64_t l, int64_t r, int64_t E, uint64_t seed, int32_t* out) {
    int64_t cnt = r - l + 1;
    if (cnt <= 0) return 0;
    uint64_t T = fo_entry_threshold(cnt, E);
    int64_t c = 0;
    for (int64_t i = l; i <= r; ++i)
        if ((uint64_t)fo_entry_priority(seed, i) < T) out[c++] = (int32_t)i;
    return c;
}

/* ENIdentification: layers L_start..L_end of u's ENC block in stored order,
 * keep v != -1 with l <= v <= r, stop once B are kept.  Adds to *scanned the
 * entries of every layer touched (a layer is one chunk when m <= 64). */
int fo_en_ident(const int32_t* ENC, int H, int m, int64_t u, int64_t l, int64_t r,
                int Ls, int Le, int B, int32_t* EN, int64_t* scanned) {
    int cnt = 0;
    for (int h = Ls; h <= Le; ++h) {
        const int32_t* row = ENC + ((int64_t)u * H + h) * m;
        *scanned += m;
        for (int t = 0; t < m; ++t) {
            int32_t v = row[t];
            if (v != FO_NONE && v >= l && v <= r) {
                EN[cnt] = v;
                cnt = cnt + 1;
                if (cnt == B) return cnt;
            }
        }
    }
    return cnt;
}

/* ------------------------------------------------------------------------ */
/* Candidate lists                                                           */
/* ------------------------------------------------------------------------ */

/* forward declarations of the visited set (below) */
typedef struct fo_visited_s fo_visited;
static int fo_visited_insert(fo_visited* s, int32_t v);

typedef struct { float dist; int32_t id; int32_t flag; } fo_cand;

static int fo_cand_cmp(const void* pa, const void* pb) {
    const fo_cand* a = (const fo_cand*)pa;
    const fo_cand* b = (const fo_cand*)pb;
    if (a->dist < b->dist) return -1;
    if (a->dist > b->dist) return 1;
    if (a->id < b->id) return -1;
    if (a->id > b->id) return 1;
    return 0;
}

/* A visited set over 0..n-1: one byte per vertex plus the list of marks, so it
 * can be cleared in time proportional to its content. */
struct fo_visited_s { uint8_t* mark; int32_t* list; int64_t size; };

static int fo_visited_init(fo_visited* v, int64_t n) {
    v->mark = (uint8_t*)calloc((size_t)(n > 0 ? n : 1), 1);
    v->list = (int32_t*)malloc(sizeof(int32_t) * (size_t)(n > 0 ? n : 1));
    v->size = 0;
    return (v->mark && v->list) ? 0 : -1;
}
static void fo_visited_free(fo_visited* v) { free(v->mark); free(v->list); }
static void fo_visited_clear(fo_visited* v) {
    for (int64_t i = 0; i < v->size; ++i) v->mark[v->list[i]] = 0;
    v->size = 0;
}
/* Returns 1 if v was not in the set (and inserts it), 0 otherwise. */
static int fo_visited_insert(fo_visited* s, int32_t v) {
    if (s->mark[v]) return 0;
    s->mark[v] = 1;
    s->list[s->size++] = v;
    return 1;
}

/* ------------------------------------------------------------------------ */
/* FROGSearch (Alg. 2)                                                       */
/* ------------------------------------------------------------------------ */

/* ENIdentification with an eager visited check (the ablation of the lazy
 * check): an in-range candidate already visited is skipped and does not count
 * against B; an admitted one is marked visited at once. */
static int fo_en_ident_eager(const int32_t* ENC, int H, int m, int64_t u, int64_t l, int64_t r,
                             int Ls, int Le, int B, fo_visited* vis, int32_t* EN, int64_t* scanned) {
    int cnt = 0;
    for (int h = Ls; h <= Le; ++h) {
        const int32_t* row = ENC + ((int64_t)u * H + h) * m;
        *scanned += m;
        for (int t = 0; t < m; ++t) {
            int32_t v = row[t];
            if (v != FO_NONE && v >= l && v <= r && fo_visited_insert(vis, v)) {
                EN[cnt] = v;
                cnt = cnt + 1;
                if (cnt == B) return cnt;
            }
        }
    }
    return cnt;
}

/* Per-query statistics written by fo_search_batch (int64 each). */
enum { FO_ST_EXPANSIONS = 0, FO_ST_EN = 1, FO_ST_DIST = 2, FO_ST_SCANNED = 3,
       FO_ST_ENTRY = 4, FO_ST_LS = 5, FO_ST_LE = 6, FO_ST_N = 8 };

typedef struct {
    const float* X;        /* [n][d] vectors in rank order */
    const int32_t* ENC;    /* [n][H][m] */
    const double* attr_sorted;
    const int32_t* perm;   /* rank -> original id, or NULL to report ranks */
    int64_t n;
    int d, H, m;
} fo_index;

static void fo_search_one(const fo_index* ix, const float* q, double lo, double hi,
                          int k, int L, int epn, double epn_frac, int epn_max, int B,
                          uint64_t seed, int entry_mode, int hot_mode, int eager, uint64_t qi,
                          int32_t* out_ids, float* out_d, int64_t* st,
                          fo_visited* vis, fo_cand* pool, fo_cand* work,
                          int32_t* ep, int32_t* EN) {
    for (int i = 0; i < k; ++i) { out_ids[i] = -1; out_d[i] = INFINITY; }
    for (int i = 0; i < FO_ST_N; ++i) st[i] = 0;
    int64_t l, r;
    fo_rank_bounds(ix->attr_sorted, ix->n, lo, hi, &l, &r);
    if (l > r) return;

    int Ls, Le;
    fo_hotspot(l, r, ix->H, ix->n, &Ls, &Le);
    if (hot_mode == 1) Le = ix->H - 1;                  /* no end condition */
    if (hot_mode == 2) { Ls = 0; Le = ix->H - 1; }      /* no localisation */
    st[FO_ST_LS] = Ls;
    st[FO_ST_LE] = Le;

    /* entry points, their distances, pool = the L nearest of them */
    int64_t E = fo_entry_count(r - l + 1, epn, epn_frac, epn_max);
    int64_t ne = entry_mode == 1 ? fo_entry_points_shared(l, r, E, seed, ep)
                                 : fo_entry_points(l, r, E, seed, qi, ep);
    st[FO_ST_ENTRY] = ne;
    fo_visited_clear(vis);
    int64_t nw = 0;
    for (int64_t j = 0; j < ne; ++j) {
        if (fo_visited_insert(vis, ep[j])) {
            work[nw].dist = fo_dist(q, ix->X + (int64_t)ep[j] * ix->d, ix->d);
            work[nw].id = ep[j];
            work[nw].flag = 0;
            nw = nw + 1;
        }
    }
    st[FO_ST_DIST] += nw;
    qsort(work, (size_t)nw, sizeof(fo_cand), fo_cand_cmp);
    int np = (int)(nw < L ? nw : L);
    for (int i = 0; i < np; ++i) pool[i] = work[i];

    for (;;) {
        int i = -1;
        for (int t = 0; t < np; ++t) if (pool[t].flag == 0) { i = t; break; }
        if (i < 0) break;
        pool[i].flag = 1;
        int32_t u = pool[i].id;
        st[FO_ST_EXPANSIONS] += 1;

        int nen = eager ? fo_en_ident_eager(ix->ENC, ix->H, ix->m, u, l, r, Ls, Le, B, vis, EN, &st[FO_ST_SCANNED])
                        : fo_en_ident(ix->ENC, ix->H, ix->m, u, l, r, Ls, Le, B, EN, &st[FO_ST_SCANNED]);
        st[FO_ST_EN] += nen;

        /* lazy visited check just before the distance; new candidates */
        int nnew = 0;
        for (int t = 0; t < np; ++t) work[t] = pool[t];
        for (int t = 0; t < nen; ++t) {
            int32_t v = EN[t];
            if (eager || fo_visited_insert(vis, v)) {
                work[np + nnew].dist = fo_dist(q, ix->X + (int64_t)v * ix->d, ix->d);
                work[np + nnew].id = v;
                work[np + nnew].flag = 0;
                nnew = nnew + 1;
            }
        }
        st[FO_ST_DIST] += nnew;
        /* MergeTopEfS: the L nearest of pool and new */
        qsort(work, (size_t)(np + nnew), sizeof(fo_cand), fo_cand_cmp);
        np = np + nnew < L ? np + nnew : L;
        for (int t = 0; t < np; ++t) pool[t] = work[t];
    }

    int kk = np < k ? np : k;
    for (int i = 0; i < kk; ++i) {
        out_ids[i] = ix->perm ? ix->perm[pool[i].id] : pool[i].id;
        out_d[i] = pool[i].dist;
    }
}

/* Batch driver.  qidx (may be NULL) gives each query's index in its batch,
 * which keys its entry-point jitter (entry_mode 0); NULL means 0..nq-1.
 * entry_mode 0: stratified per-query sample; 1: shared-priority sample.
 * hot_mode 0: HotspotLocalization (Alg. 3); 1: layers L_start..H-1 (no end
 * condition); 2: all layers 0..H-1.  eager: visited check inside
 * ENIdentification instead of after it.
 * Returns 0 or -1 on allocation failure.  stats (may be NULL) is [nq][8]
 * int64. */
int fo_search_batch(const float* X, const int32_t* ENC, const double* attr_sorted,
                    const int32_t* perm, int64_t n, int d, int H, int m,
                    const float* Q, const double* lo, const double* hi, int64_t nq,
                    const int64_t* qidx, int k, int L, int epn, double epn_frac, int epn_max,
                    int B, uint64_t seed, int entry_mode, int hot_mode, int eager, int32_t* out_ids,
                    float* out_d, int64_t* stats, int nthreads) {
    fo_index ix = { X, ENC, attr_sorted, perm, n, d, H, m };
    int fail = 0;
    if (nthreads <= 0) nthreads = 1;
#pragma omp parallel num_threads(nthreads) reduction(|:fail)
    {
        fo_visited vis;
        /* the shared-priority sample has no fixed size: room for a whole range */
        int64_t ep_cap = entry_mode == 1 ? n : fo_entry_count(n, epn, epn_frac, epn_max);
        if (ep_cap < 1) ep_cap = 1;
        fo_cand* pool = (fo_cand*)malloc(sizeof(fo_cand) * (size_t)(L + 1));
        fo_cand* work = (fo_cand*)malloc(sizeof(fo_cand) * (size_t)(L + B + ep_cap + 1));
        int32_t* ep = (int32_t*)malloc(sizeof(int32_t) * (size_t)ep_cap);
        int32_t* EN = (int32_t*)malloc(sizeof(int32_t) * (size_t)(B + 1));
        if (fo_visited_init(&vis, n) || !pool || !work || !ep || !EN) {
            fail = 1;
        } else {
#pragma omp for schedule(dynamic, 4)
            for (int64_t i = 0; i < nq; ++i) {
                int64_t st_local[FO_ST_N];
                fo_search_one(&ix, Q + i * d, lo[i], hi[i], k, L, epn, epn_frac, epn_max, B, seed,
                              entry_mode, hot_mode, eager, (uint64_t)(qidx ? qidx[i] : i),
                              out_ids + i * k, out_d + i * k,
                              stats ? stats + i * FO_ST_N : st_local,
                              &vis, pool, work, ep, EN);
            }
        }
        fo_visited_free(&vis);
        free(pool); free(work); free(ep); free(EN);
    }
    return fail ? -1 : 0;
}

/* ------------------------------------------------------------------------ */
/* Exhaustive filtered k-NN (Def. 2)                                          */
/* ------------------------------------------------------------------------ */

int fo_exact_batch(const float* X, const double* attr_sorted, const int32_t* perm,
                   int64_t n, int d, const float* Q, const double* lo, const double* hi,
                   int64_t nq, int k, int32_t* out_ids, float* out_d, int nthreads) {
    if (nthreads <= 0) nthreads = 1;
    int fail = 0;
#pragma omp parallel num_threads(nthreads) reduction(|:fail)
    {
        fo_cand* best = (fo_cand*)malloc(sizeof(fo_cand) * (size_t)(k + 1));
        if (!best) fail = 1;
        else {
#pragma omp for schedule(dynamic, 1)
            for (int64_t i = 0; i < nq; ++i) {
                int64_t l, r;
                fo_rank_bounds(attr_sorted, n, lo[i], hi[i], &l, &r);
                int nb = 0;
                for (int64_t v = l; v <= r; ++v) {
                    fo_cand c;
                    c.dist = fo_dist(Q + i * d, X + v * d, d);
                    c.id = (int32_t)v;
                    c.flag = 0;
                    /* keep the k smallest (dist, id) in a sorted array */
                    if (nb == k && fo_cand_cmp(&c, &best[k - 1]) >= 0) continue;
                    int pos = nb < k ? nb : k - 1;
                    while (pos > 0 && fo_cand_cmp(&c, &best[pos - 1]) < 0) {
                        best[pos] = best[pos - 1];
                        pos = pos - 1;
                    }
                    best[pos] = c;
                    if (nb < k) nb = nb + 1;
                }
                for (int j = 0; j < k; ++j) {
                    if (j < nb) {
                        out_ids[i * k + j] = perm ? perm[best[j].id] : best[j].id;
                        out_d[i * k + j] = best[j].dist;
                    } else {
                        out_ids[i * k + j] = -1;
                        out_d[i * k + j] = INFINITY;
                    }
                }
            }
        }
        free(best);
    }
    return fail ? -1 : 0;
}

/* ------------------------------------------------------------------------ */
/* Index construction (Sec. 6)                                               */
/* ------------------------------------------------------------------------ */

typedef struct { double key; float dist; int32_t id; } fo_ranked;

static int fo_ranked_cmp(const void* pa, const void* pb) {
    const fo_ranked* a = (const fo_ranked*)pa;
    const fo_ranked* b = (const fo_ranked*)pb;
    if (a->key < b->key) return -1;
    if (a->key > b->key) return 1;
    if (a->id < b->id) return -1;
    if (a->id > b->id) return 1;
    return 0;
}

/* Eq. fusion-distance: delta_v * (1 - beta * (1 - delta_a^gamma)), with
 * delta_v the L2 distance and delta_a = |ru - rv| / (seglen - 1). */
double fo_fusion(float d2, int64_t ru, int64_t rv, int64_t seglen, double beta, double gamma) {
    double dv = sqrt((double)d2);
    int64_t diff = ru > rv ? ru - rv : rv - ru;
    double da = (double)diff / (double)(seglen - 1);
    double w = 1.0 - beta * (1.0 - pow(da, gamma));
    return dv * w;
}

typedef struct { double attr; int32_t id; } fo_attr_id;
static int fo_attr_cmp(const void* pa, const void* pb) {
    const fo_attr_id* a = (const fo_attr_id*)pa;
    const fo_attr_id* b = (const fo_attr_id*)pb;
    if (a->attr < b->attr) return -1;
    if (a->attr > b->attr) return 1;
    return (a->id > b->id) - (a->id < b->id);
}

/* Stable attribute sort: perm[rank] = original id, attr_sorted[rank] = value.
 * Returns -1 if an attribute is NaN. */
int fo_rank_order(const double* attr, int64_t n, int32_t* perm, double* attr_sorted) {
    fo_attr_id* t = (fo_attr_id*)malloc(sizeof(fo_attr_id) * (size_t)(n > 0 ? n : 1));
    if (!t) return -2;
    for (int64_t i = 0; i < n; ++i) {
        if (isnan(attr[i])) { free(t); return -1; }
        t[i].attr = attr[i];
        t[i].id = (int32_t)i;
    }
    qsort(t, (size_t)n, sizeof(fo_attr_id), fo_attr_cmp);
    for (int64_t i = 0; i < n; ++i) { perm[i] = t[i].id; attr_sorted[i] = t[i].attr; }
    free(t);
    return 0;
}

/* Greedy best-first search (Alg. 1) for the vertex xq over the temporary PG
 * restricted to segment [ts, te], pool width ef, several seeds, stopping
 * early after `patience` consecutive expansions that change nothing in the
 * top-m (Sec 6.2.2).  Writes the m nearest found (ascending (dist, id)) to
 * res/resd and returns how many were found; *expansions (may be NULL)
 * receives the number of pool entries expanded. */
static int fo_sibling_search(const float* X, int d, const int32_t* PG, int m,
                             const float* xq, int64_t ts, int64_t te,
                             const int32_t* seeds, int nseeds, int ef, int patience,
                             fo_visited* vis, fo_cand* pool, fo_cand* work,
                             int32_t* res, float* resd, int64_t* expansions) {
    fo_visited_clear(vis);
    int np = 0;
    int nw = 0;
    for (int j = 0; j < nseeds; ++j) {
        if (fo_visited_insert(vis, seeds[j])) {
            work[nw].dist = fo_dist(xq, X + (int64_t)seeds[j] * d, d);
            work[nw].id = seeds[j];
            work[nw].flag = 0;
            nw = nw + 1;
        }
    }
    qsort(work, (size_t)nw, sizeof(fo_cand), fo_cand_cmp);
    np = nw < ef ? nw : ef;
    for (int i = 0; i < np; ++i) pool[i] = work[i];
    int left = patience;
    int64_t nexp = 0;
    for (;;) {
        int i = -1;
        for (int t = 0; t < np; ++t) if (pool[t].flag == 0) { i = t; break; }
        if (i < 0) break;
        pool[i].flag = 1;
        nexp = nexp + 1;
        int32_t w = pool[i].id;
        for (int t = 0; t < np; ++t) work[t] = pool[t];
        int nnew = 0;
        for (int t = 0; t < m; ++t) {
            int32_t v = PG[(int64_t)w * m + t];
            if (v == FO_NONE) continue;
            if (v < ts || v > te) continue; /* temporary PG edges stay inside their segment */
            if (fo_visited_insert(vis, v)) {
                work[np + nnew].dist = fo_dist(xq, X + (int64_t)v * d, d);
                work[np + nnew].id = v;
                work[np + nnew].flag = 0;
                nnew = nnew + 1;
            }
        }
        qsort(work, (size_t)(np + nnew), sizeof(fo_cand), fo_cand_cmp);
        int nnp = np + nnew < ef ? np + nnew : ef;
        /* did any new candidate land in the top-m? */
        int improved = 0;
        int top = nnp < m ? nnp : m;
        for (int t = 0; t < top; ++t) {
            int is_new = 1;
            for (int s = 0; s < np; ++s) if (pool[s].id == work[t].id) { is_new = 0; break; }
            if (is_new) { improved = 1; break; }
        }
        np = nnp;
        for (int t = 0; t < np; ++t) pool[t] = work[t];
        if (improved) left = patience;
        else {
            left = left - 1;
            if (left <= 0) break;
        }
    }
    int nr = np < m ? np : m;
    for (int t = 0; t < nr; ++t) { res[t] = pool[t].id; resd[t] = pool[t].dist; }
    if (expansions) *expansions = nexp;
    return nr;
}

/* RNG prune (alpha = 1) of candidates sorted by distance to u: keep c unless a
 * kept k is closer to c than u is; then top up to m with the nearest pruned. */
static int fo_rng_prune(const float* X, int d, const fo_ranked* cand, int nc, int m, int32_t* out) {
    int nk = 0;
    int* kept = (int*)calloc((size_t)(nc > 0 ? nc : 1), sizeof(int));
    for (int i = 0; i < nc && nk < m; ++i) {
        int ok = 1;
        for (int j = 0; j < nk; ++j) {
            float dck = fo_dist(X + (int64_t)cand[i].id * d, X + (int64_t)out[j] * d, d);
            if (dck < cand[i].dist) { ok = 0; break; }
        }
        if (ok) { out[nk] = cand[i].id; nk = nk + 1; kept[i] = 1; }
    }
    for (int i = 0; i < nc && nk < m; ++i) {
        if (!kept[i]) { out[nk] = cand[i].id; nk = nk + 1; }
    }
    free(kept);
    for (int i = nk; i < m; ++i) out[i] = FO_NONE;
    return nk;
}

/* The two construction steps above on their own, for the tests: the RNG
 * prune of nc candidates given as (id, squared distance to u) ascending by
 * (distance, id); and the sibling search over a temporary PG of n vertices
 * (PG [n][m], -1 for empty slots) with the given seeds.  Each returns what the
 * step returns, or -2 if memory runs out. */
int fo_rng_prune_list(const float* X, int d, const int32_t* ids, const float* dists, int nc, int m,
                      int32_t* out) {
    fo_ranked* cand = (fo_ranked*)malloc(sizeof(fo_ranked) * (size_t)(nc > 0 ? nc : 1));
    if (!cand) return -2;
    for (int i = 0; i < nc; ++i) {
        cand[i].key = (double)dists[i];
        cand[i].dist = dists[i];
        cand[i].id = ids[i];
    }
    int nk = fo_rng_prune(X, d, cand, nc, m, out);
    free(cand);
    return nk;
}

int fo_sibling_search_list(const float* X, int64_t n, int d, const int32_t* PG, int m, const float* xq,
                           int64_t ts, int64_t te, const int32_t* seeds, int nseeds, int ef, int patience,
                           int32_t* res, float* resd, int64_t* expansions) {
    fo_visited vis;
    fo_cand* pool = (fo_cand*)malloc(sizeof(fo_cand) * (size_t)(ef + 1));
    fo_cand* work = (fo_cand*)malloc(sizeof(fo_cand) * (size_t)(ef + m + nseeds + 1));
    int rc = -2;
    if (fo_visited_init(&vis, n) == 0 && pool && work)
        rc = fo_sibling_search(X, d, PG, m, xq, ts, te, seeds, nseeds, ef, patience, &vis, pool, work,
                               res, resd, expansions);
    fo_visited_free(&vis);
    free(pool);
    free(work);
    return rc;
}

/* Build the index.  X is [n][d] in ORIGINAL object order, attr [n].  Outputs:
 * perm [n] (rank -> original id), attr_sorted [n], X_rank [n][d] (vectors in
 * rank order), ENC [n][H][m].  Returns H (>= 1) or a negative error. */
int fo_build(const float* X, const double* attr, int64_t n, int d,
             int m, int ef_c, int n_inv, int patience, int sib_seeds,
             double beta, double gamma, uint64_t seed, int nthreads,
             int32_t* perm, double* attr_sorted, float* X_rank, int32_t* ENC) {
    if (n < 1 || d < 1 || m < 1 || ef_c < m || sib_seeds < 1) return -3;
    if (nthreads <= 0) nthreads = 1;
    int rc = fo_rank_order(attr, n, perm, attr_sorted);
    if (rc) return rc;
    for (int64_t i = 0; i < n; ++i)
        memcpy(X_rank + i * d, X + (int64_t)perm[i] * d, sizeof(float) * (size_t)d);
    int H = fo_num_layers(n, n_inv);
    for (int64_t i = 0; i < n * H * m; ++i) ENC[i] = FO_NONE;

    int32_t* PG = (int32_t*)malloc(sizeof(int32_t) * (size_t)(n * m));
    int32_t* PGn = (int32_t*)malloc(sizeof(int32_t) * (size_t)(n * m));
    if (!PG || !PGn) { free(PG); free(PGn); return -2; }
    for (int64_t i = 0; i < n * m; ++i) { PG[i] = FO_NONE; PGn[i] = FO_NONE; }

    /* Leaf layer: brute force inside each leaf segment. */
    {
        int h = H - 1;
        int fail = 0;
#pragma omp parallel num_threads(nthreads) reduction(|:fail)
        {
            /* the largest leaf holds at most ceil(n / 2^(H-1)) ranks */
            int64_t cap = (n >> h) + 2;
            fo_ranked* fu = (fo_ranked*)malloc(sizeof(fo_ranked) * (size_t)cap);
            fo_ranked* ve = (fo_ranked*)malloc(sizeof(fo_ranked) * (size_t)cap);
            if (!fu || !ve) fail = 1;
            else {
#pragma omp for schedule(dynamic, 16)
                for (int64_t u = 0; u < n; ++u) {
                    int64_t s, e;
                    fo_segment(n, h, u, &s, &e);
                    int64_t len = e - s + 1;
                    int c = 0;
                    for (int64_t v = s; v <= e; ++v) {
                        if (v == u) continue;
                        float d2 = fo_dist(X_rank + u * d, X_rank + v * d, d);
                        fu[c].key = fo_fusion(d2, u, v, len, beta, gamma);
                        fu[c].dist = d2; fu[c].id = (int32_t)v;
                        ve[c].key = (double)d2;
                        ve[c].dist = d2; ve[c].id = (int32_t)v;
                        c = c + 1;
                    }
                    qsort(fu, (size_t)c, sizeof(fo_ranked), fo_ranked_cmp);
                    qsort(ve, (size_t)c, sizeof(fo_ranked), fo_ranked_cmp);
                    for (int t = 0; t < m && t < c; ++t) {
                        ENC[(u * H + h) * m + t] = fu[t].id;
                        PG[u * m + t] = ve[t].id;
                    }
                }
            }
            free(fu); free(ve);
        }
        if (fail) { free(PG); free(PGn); return -2; }
    }

    /* Internal layers, bottom-up. */
    for (int h = H - 2; h >= 0; --h) {
        int fail = 0;
#pragma omp parallel num_threads(nthreads) reduction(|:fail)
        {
            fo_visited vis;
            fo_cand* pool = (fo_cand*)malloc(sizeof(fo_cand) * (size_t)(ef_c + 1));
            fo_cand* work = (fo_cand*)malloc(sizeof(fo_cand) * (size_t)(ef_c + m + sib_seeds + 1));
            int32_t* seeds = (int32_t*)malloc(sizeof(int32_t) * (size_t)sib_seeds);
            int32_t* res = (int32_t*)malloc(sizeof(int32_t) * (size_t)m);
            float* resd = (float*)malloc(sizeof(float) * (size_t)m);
            fo_ranked* cand = (fo_ranked*)malloc(sizeof(fo_ranked) * (size_t)(2 * m));
            fo_ranked* fus = (fo_ranked*)malloc(sizeof(fo_ranked) * (size_t)(2 * m));
            if (fo_visited_init(&vis, n) || !pool || !work || !seeds || !res || !resd || !cand || !fus) {
                fail = 1;
            } else {
#pragma omp for schedule(dynamic, 16)
                for (int64_t u = 0; u < n; ++u) {
                    int64_t s, e;
                    fo_segment(n, h, u, &s, &e);
                    int64_t len = e - s + 1;
                    int64_t mid = s + (e - s) / 2;
                    int64_t ts, te;  /* sibling segment at depth h+1 */
                    if (u <= mid) { ts = mid + 1; te = e; } else { ts = s; te = mid; }
                    const float* xu = X_rank + u * d;
                    int nc = 0;
                    /* m-ANN from the child's temporary PG */
                    for (int t = 0; t < m; ++t) {
                        int32_t v = PG[u * m + t];
                        if (v == FO_NONE) continue;
                        cand[nc].dist = fo_dist(xu, X_rank + (int64_t)v * d, d);
                        cand[nc].key = (double)cand[nc].dist;
                        cand[nc].id = v;
                        nc = nc + 1;
                    }
                    /* m-ANN from a greedy search over the sibling's temporary PG */
                    int64_t tl = te - ts + 1;
                    if (tl > 0) {
                        int ns;
                        if (tl <= sib_seeds) {
                            ns = (int)tl;
                            for (int j = 0; j < ns; ++j) seeds[j] = (int32_t)(ts + j);
                        } else {
                            ns = sib_seeds;
                            for (int j = 0; j < ns; ++j) {
                                int64_t a = ts + ((int64_t)j * tl) / sib_seeds;
                                int64_t b = ts + ((int64_t)(j + 1) * tl) / sib_seeds - 1;
                                uint64_t z = fo_splitmix64(seed ^ ((uint64_t)u << 32) ^ ((uint64_t)h << 24) ^ (uint64_t)j);
                                seeds[j] = (int32_t)(a + (int64_t)fo_reduce(z, (uint64_t)(b - a + 1)));
                            }
                        }
                        int nr = fo_sibling_search(X_rank, d, PG, m, xu, ts, te, seeds, ns, ef_c,
                                                   patience, &vis, pool, work, res, resd, NULL);
                        for (int t = 0; t < nr; ++t) {
                            cand[nc].dist = resd[t];
                            cand[nc].key = (double)resd[t];
                            cand[nc].id = res[t];
                            nc = nc + 1;
                        }
                    }
                    qsort(cand, (size_t)nc, sizeof(fo_ranked), fo_ranked_cmp);
                    /* (i) RNG prune -> parent temporary PG row */
                    fo_rng_prune(X_rank, d, cand, nc, m, PGn + u * m);
                    /* (ii) fusion re-rank -> ENC row of layer h */
                    for (int t = 0; t < nc; ++t) {
                        fus[t].key = fo_fusion(cand[t].dist, u, cand[t].id, len, beta, gamma);
                        fus[t].dist = cand[t].dist;
                        fus[t].id = cand[t].id;
                    }
                    qsort(fus, (size_t)nc, sizeof(fo_ranked), fo_ranked_cmp);
                    for (int t = 0; t < m && t < nc; ++t) ENC[(u * H + h) * m + t] = fus[t].id;
                }
            }
            fo_visited_free(&vis);
            free(pool); free(work); free(seeds); free(res); free(resd); free(cand); free(fus);
        }
        if (fail) { free(PG); free(PGn); return -2; }
        int32_t* t = PG; PG = PGn; PGn = t;
    }
    free(PG);
    free(PGn);
    return H;
}

/* Closure of the entry set under EN(.) (no pool bound): the vertices a search
 * with unbounded pool could ever evaluate.  Marks reach[v] = 1.  Used to check
 * the L >= n special case.  Returns the closure size. */
int64_t fo_closure(const int32_t* ENC, int H, int m, int64_t n, int64_t l, int64_t r,
                   int Ls, int Le, int B, const int32_t* entry, int64_t ne, uint8_t* reach) {
    int32_t* stack = (int32_t*)malloc(sizeof(int32_t) * (size_t)(n > 0 ? n : 1));
    int32_t* EN = (int32_t*)malloc(sizeof(int32_t) * (size_t)(B + 1));
    int64_t top = 0, size = 0, scanned = 0;
    memset(reach, 0, (size_t)n);
    for (int64_t j = 0; j < ne; ++j)
        if (!reach[entry[j]]) { reach[entry[j]] = 1; stack[top++] = entry[j]; size++; }
    while (top > 0) {
        int32_t u = stack[--top];
        int c = fo_en_ident(ENC, H, m, u, l, r, Ls, Le, B, EN, &scanned);
        for (int t = 0; t < c; ++t)
            if (!reach[EN[t]]) { reach[EN[t]] = 1; stack[top++] = EN[t]; size++; }
    }
    free(stack);
    free(EN);
    return size;
}
