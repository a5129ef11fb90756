// Host construction of the FROG index (Sec 6 of the paper).
//
// Input: vectors and one numeric attribute per object.  Output: the
// attribute-rank domain (perm, sorted attributes, vectors in rank order) and
// the dense n x H x m expansion-neighbour-candidate (ENC) array of Sec 4.
//
// Procedure (bottom-up, layers independent inside, Sec 6.1):
//   leaf layer   every vertex ranks the other vertices of its leaf segment by
//                fusion distance (Eq. fusion-distance) and keeps m; the leaf's
//                temporary proximity graph (PG) is the exact vector top-m;
//   layer h      every vertex u of segment S (children A, B) takes the m
//                neighbours of its child's temporary PG plus the m best of a
//                greedy search (Alg. 1, pool ef_c, patience early stop,
//                Sec 6.2.2) over the sibling child's temporary PG; the 2m set
//                is (i) RNG-pruned into u's row of S's temporary PG, and
//                (ii) re-ranked by fusion distance into ENC[u][h].
// Readings where the paper is silent: normalised attribute distance is the
// rank difference over (segment length - 1); the RNG prune keeps a candidate
// unless a kept one is strictly closer to it than u is, then tops the row up
// to m with the nearest pruned candidates; the sibling search starts from
// `sib_seeds` stratified ranks of the sibling, jittered by SplitMix64 keyed on
// (seed, u, h, j) and reduced with Lemire's multiply-shift.
//
// Determinism: every vertex's work depends only on the previous layer, so the
// threads never change a result.  Distances are the library's canonical
// squared L2 (double accumulation in index order, one rounding to float);
// the 4-wide AVX2 kernel below keeps that order per candidate, so results do
// not depend on the vector width.  The translation unit is compiled without
// FMA contraction.

#include <immintrin.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstring>
#include <memory>
#include <thread>

#include "frog_internal.h"

namespace frog {

namespace {

constexpr int32_t kNone = -1;

// ---------------------------------------------------------------- distances

inline float dist1(const float* a, const float* b, int d) {
    double s = 0.0;
    for (int i = 0; i < d; ++i) {
        double t = (double)a[i] - (double)b[i];
        double t2 = t * t;
        s = s + t2;
    }
    return (float)s;
}

// Four distances from q to rows r[0..3]; each lane sums its own candidate's
// terms in index order, like dist1.
inline void dist4(const float* q, const float* const r[4], int d, float out[4]) {
    __m256d s = _mm256_setzero_pd();
    int i = 0;
    for (; i + 4 <= d; i += 4) {
        __m128 a0 = _mm_loadu_ps(r[0] + i), a1 = _mm_loadu_ps(r[1] + i);
        __m128 a2 = _mm_loadu_ps(r[2] + i), a3 = _mm_loadu_ps(r[3] + i);
        _MM_TRANSPOSE4_PS(a0, a1, a2, a3);
        const __m128 cols[4] = {a0, a1, a2, a3};
        for (int c = 0; c < 4; ++c) {
            __m256d qd = _mm256_set1_pd((double)q[i + c]);
            __m256d t = _mm256_sub_pd(qd, _mm256_cvtps_pd(cols[c]));
            s = _mm256_add_pd(s, _mm256_mul_pd(t, t));
        }
    }
    alignas(32) double acc[4];
    _mm256_store_pd(acc, s);
    for (int c = 0; c < 4; ++c) {
        double sc = acc[c];
        for (int j = i; j < d; ++j) {
            double t = (double)q[j] - (double)r[c][j];
            double t2 = t * t;
            sc = sc + t2;
        }
        out[c] = (float)sc;
    }
}

// distances from q to rows ids[0..cnt) of X
inline void dist_many(const float* X, int d, const float* q, const int32_t* ids, int cnt, float* out) {
    int t = 0;
    for (; t + 4 <= cnt; t += 4) {
        const float* r[4] = {X + (int64_t)ids[t] * d, X + (int64_t)ids[t + 1] * d,
                             X + (int64_t)ids[t + 2] * d, X + (int64_t)ids[t + 3] * d};
        dist4(q, r, d, out + t);
    }
    for (; t < cnt; ++t) out[t] = dist1(q, X + (int64_t)ids[t] * d, d);
}

// ---------------------------------------------------------------- helpers

inline uint64_t splitmix64(uint64_t x) {
    uint64_t z = x + 0x9E3779B97F4A7C15ULL;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

inline uint64_t reduce_range(uint64_t z, uint64_t width) { return ((z >> 32) * width) >> 32; }

inline void segment_of(int64_t n, int h, int64_t p, int64_t* s, int64_t* e) {
    int64_t L = 0, R = n - 1;
    for (int i = 0; i < h; ++i) {
        int64_t mid = L + (R - L) / 2;
        if (p <= mid) R = mid; else L = mid + 1;
    }
    *s = L;
    *e = R;
}

inline double fusion(float d2, int64_t ru, int64_t rv, int64_t seglen, double beta, double gamma) {
    double dv = std::sqrt((double)d2);
    int64_t diff = ru > rv ? ru - rv : rv - ru;
    double da = (double)diff / (double)(seglen - 1);
    double w = 1.0 - beta * (1.0 - std::pow(da, gamma));
    return dv * w;
}

struct Ranked {
    double key;
    float dist;
    int32_t id;
};
inline bool ranked_less(const Ranked& a, const Ranked& b) {
    return a.key < b.key || (a.key == b.key && a.id < b.id);
}

struct Cand {
    float dist;
    int32_t id;
    int32_t flag;
};
inline bool cand_less(const Cand& a, const Cand& b) {
    return a.dist < b.dist || (a.dist == b.dist && a.id < b.id);
}

// Run f(i) for i in [0, count) on `threads` threads with dynamic chunks; f
// receives (i, thread_index).
template <class F>
void parallel_for(int64_t count, int threads, int64_t chunk, F&& f) {
    std::atomic<int64_t> next{0};
    auto body = [&](int t) {
        for (;;) {
            int64_t b = next.fetch_add(chunk);
            if (b >= count) break;
            int64_t e = std::min(count, b + chunk);
            for (int64_t i = b; i < e; ++i) f(i, t);
        }
    };
    if (threads <= 1) { body(0); return; }
    std::vector<std::thread> pool;
    pool.reserve(threads);
    for (int t = 0; t < threads; ++t) pool.emplace_back(body, t);
    for (auto& th : pool) th.join();
}

// Per-thread scratch of the sibling search.
struct Scratch {
    std::vector<uint32_t> stamp;  // visited marks, epoch-stamped
    uint32_t epoch = 0;
    std::vector<Cand> pool;
    std::vector<int32_t> newid;
    std::vector<float> newd;
    std::vector<int32_t> seeds;
    std::vector<Ranked> cand, fus;
    std::vector<int32_t> res;
    std::vector<float> resd;
    std::vector<float> dtmp;
    std::vector<char> kept;

    void init(int64_t n, int m, int ef, int ns) {
        stamp.assign((size_t)n, 0);
        pool.resize((size_t)ef + 1);
        newid.resize((size_t)m + ns + 1);
        newd.resize((size_t)m + ns + 1);
        seeds.resize((size_t)ns);
        cand.resize((size_t)2 * m);
        fus.resize((size_t)2 * m);
        res.resize((size_t)m);
        resd.resize((size_t)m);
        dtmp.resize((size_t)2 * m);
        kept.resize((size_t)2 * m);
    }
    void next_epoch() {
        if (++epoch == 0) {
            std::fill(stamp.begin(), stamp.end(), 0u);
            epoch = 1;
        }
    }
    bool visit(int32_t v) {
        if (stamp[(size_t)v] == epoch) return false;
        stamp[(size_t)v] = epoch;
        return true;
    }
};

// Insert c into the sorted pool [0, np) of capacity ef; returns its position
// or -1 when it falls beyond the capacity.
inline int pool_insert(Cand* pool, int& np, int ef, const Cand& c) {
    int pos = (int)(std::lower_bound(pool, pool + np, c, cand_less) - pool);
    if (pos >= ef) return -1;
    int last = np < ef ? np : ef - 1;
    for (int t = last; t > pos; --t) pool[t] = pool[t - 1];
    pool[pos] = c;
    if (np < ef) ++np;
    return pos;
}

// Greedy search of Alg. 1 over the temporary PG restricted to [ts, te].
int sibling_search(const float* X, int d, const int32_t* PG, int m, const float* xq,
                   int64_t ts, int64_t te, const int32_t* seeds, int nseeds, int ef,
                   int patience, Scratch& S, int32_t* res, float* resd) {
    S.next_epoch();
    Cand* pool = S.pool.data();
    int np = 0;
    int nn = 0;
    for (int j = 0; j < nseeds; ++j)
        if (S.visit(seeds[j])) S.newid[(size_t)nn++] = seeds[j];
    dist_many(X, d, xq, S.newid.data(), nn, S.newd.data());
    for (int j = 0; j < nn; ++j) pool_insert(pool, np, ef, Cand{S.newd[(size_t)j], S.newid[(size_t)j], 0});
    int left = patience;
    for (;;) {
        int i = -1;
        for (int t = 0; t < np; ++t)
            if (pool[t].flag == 0) { i = t; break; }
        if (i < 0) break;
        pool[i].flag = 1;
        int32_t w = pool[i].id;
        nn = 0;
        const int32_t* row = PG + (int64_t)w * m;
        for (int t = 0; t < m; ++t) {
            int32_t v = row[t];
            if (v == kNone || v < ts || v > te) continue;
            if (S.visit(v)) S.newid[(size_t)nn++] = v;
        }
        dist_many(X, d, xq, S.newid.data(), nn, S.newd.data());
        bool improved = false;
        for (int j = 0; j < nn; ++j) {
            int pos = pool_insert(pool, np, ef, Cand{S.newd[(size_t)j], S.newid[(size_t)j], 0});
            if (pos >= 0 && pos < m) improved = true;
        }
        if (improved) {
            left = patience;
        } else {
            left = left - 1;
            if (left <= 0) break;
        }
    }
    int nr = np < m ? np : m;
    for (int t = 0; t < nr; ++t) { res[t] = pool[t].id; resd[t] = pool[t].dist; }
    return nr;
}

// RNG prune (alpha = 1) of candidates sorted by distance to u, topped up to m.
void rng_prune(const float* X, int d, const Ranked* cand, int nc, int m, int32_t* out, Scratch& S) {
    int nk = 0;
    char* kept = S.kept.data();
    for (int i = 0; i < nc; ++i) kept[i] = 0;
    for (int i = 0; i < nc && nk < m; ++i) {
        const float* xc = X + (int64_t)cand[i].id * d;
        bool ok = true;
        for (int j = 0; j < nk; ++j) {
            float dck = dist1(xc, X + (int64_t)out[j] * d, d);
            if (dck < cand[i].dist) { ok = false; break; }
        }
        if (ok) { out[nk++] = cand[i].id; kept[i] = 1; }
    }
    for (int i = 0; i < nc && nk < m; ++i)
        if (!kept[i]) out[nk++] = cand[i].id;
    for (int i = nk; i < m; ++i) out[i] = kNone;
}

}  // namespace

int layers_for(int64_t n, int n_inv) {
    int c = 0;
    while (((int64_t)1 << c) < n) ++c;
    int H = c + 1 - n_inv;
    return H < 1 ? 1 : H;
}

int rank_order(const float* X, const double* attr, int64_t n, int d, int m, int n_inv, int threads,
               bool fill_enc, frog_index* out) {
    // attribute-rank domain (Sec 4): sort by (value, original index), a strict
    // order, so chunks sorted apart and merged give the one sorted sequence
    for (int64_t i = 0; i < n; ++i)
        if (std::isnan(attr[i])) return fail(FROG_EINVAL, "attribute %lld is NaN", (long long)i);
    auto less = [&](int32_t a, int32_t b) { return attr[a] < attr[b] || (attr[a] == attr[b] && a < b); };
    std::vector<int32_t> perm((size_t)n), tmp;
    for (int64_t i = 0; i < n; ++i) perm[(size_t)i] = (int32_t)i;
    int parts = 1;
    while (parts * 2 <= threads && (int64_t)parts * 2 * 65536 <= n) parts *= 2;
    if (parts == 1) {
        std::sort(perm.begin(), perm.end(), less);
    } else {
        tmp.resize((size_t)n);
        auto cut = [&](int k) { return (size_t)((int64_t)k * n / parts); };
        parallel_for(parts, parts, 1, [&](int64_t k, int) {
            std::sort(perm.begin() + cut((int)k), perm.begin() + cut((int)k + 1), less);
        });
        for (int w = 1; w < parts; w *= 2) {
            parallel_for(parts / (2 * w), parts / (2 * w), 1, [&](int64_t k, int) {
                const size_t a = cut((int)(2 * w * k)), b = cut((int)(2 * w * k + w)), c = cut((int)(2 * w * k + 2 * w));
                std::merge(perm.begin() + a, perm.begin() + b, perm.begin() + b, perm.begin() + c, tmp.begin() + a, less);
            });
            perm.swap(tmp);
        }
    }
    const int H = layers_for(n, n_inv);
    out->n = n;
    out->d = d;
    out->H = H;
    out->m = m;
    try {
        out->perm = perm;
        out->attr.resize((size_t)n);
        out->X.resize((size_t)n * d);
        out->ENC.resize((size_t)n * H * m);
    } catch (const std::bad_alloc&) {
        return fail(FROG_ENOMEM, "host allocation of the index failed");
    }
    parallel_for(n, threads, 4096, [&](int64_t i, int) {
        out->attr[(size_t)i] = attr[perm[(size_t)i]];
        std::memcpy(&out->X[(size_t)i * d], X + (int64_t)perm[(size_t)i] * d, sizeof(float) * (size_t)d);
    });
    if (fill_enc) {
        const int64_t per = (int64_t)H * m;
        parallel_for(n, threads, 4096, [&](int64_t i, int) {
            std::fill(out->ENC.begin() + i * per, out->ENC.begin() + (i + 1) * per, kNone);
        });
    }
    return FROG_OK;
}

int host_threads(int requested) {
    if (requested > 0) return requested;
    unsigned hw = std::thread::hardware_concurrency();
    return hw ? (int)hw : 1;
}

int fusion_weights(int64_t n, int H, double beta, double gamma, int threads, std::vector<double>& tab,
                   std::vector<int64_t>& meta) {
    // segment lengths at depth h take at most two consecutive values: a
    // segment of length l splits into ceil(l/2) and floor(l/2)
    meta.assign((size_t)4 * H, 0);
    int64_t lo = n, hi = n, total = 0;
    for (int h = 0; h < H; ++h) {
        meta[(size_t)4 * h + 0] = lo;
        meta[(size_t)4 * h + 1] = total;
        total += lo;
        meta[(size_t)4 * h + 2] = hi;
        meta[(size_t)4 * h + 3] = hi == lo ? meta[(size_t)4 * h + 1] : total;
        if (hi != lo) total += hi;
        const int64_t nlo = lo / 2, nhi = (hi + 1) / 2;
        lo = nlo > 0 ? nlo : 1;
        hi = nhi > 0 ? nhi : 1;
    }
    try {
        tab.assign((size_t)std::max<int64_t>(total, 1), 0.0);
    } catch (const std::bad_alloc&) {
        return fail(FROG_ENOMEM, "fusion weight table of %lld entries", (long long)total);
    }
    // the factor fusion() applies to the L2 distance, term by term the same
    // expression, for every offset |ru - rv| of a segment of each length
    std::vector<std::pair<int64_t, int64_t>> lens;
    for (int h = 0; h < H; ++h)
        for (int k = 0; k < 2; ++k) {
            const int64_t len = meta[(size_t)4 * h + 2 * k], off = meta[(size_t)4 * h + 2 * k + 1];
            if (k == 1 && off == meta[(size_t)4 * h + 1]) continue;
            lens.emplace_back(len, off);
        }
    const int64_t chunk = 1 << 16;
    int64_t units = 0;
    std::vector<std::pair<size_t, int64_t>> work;   // (length index, first offset)
    for (size_t i = 0; i < lens.size(); ++i)
        for (int64_t b = 0; b < lens[i].first; b += chunk) { work.emplace_back(i, b); ++units; }
    parallel_for(units, threads, 1, [&](int64_t wi, int) {
        const int64_t len = lens[(size_t)work[(size_t)wi].first].first;
        const int64_t off = lens[(size_t)work[(size_t)wi].first].second;
        const int64_t b = work[(size_t)wi].second, e = std::min(len, b + chunk);
        if (len < 2) return;
        for (int64_t diff = b; diff < e; ++diff) {
            double da = (double)diff / (double)(len - 1);
            double w = 1.0 - beta * (1.0 - std::pow(da, gamma));
            tab[(size_t)(off + diff)] = w;
        }
    });
    return FROG_OK;
}

int build_host(const float* X, const double* attr, int64_t n, int d,
               const frog_build_params_t& p, frog_index* out) {
    const int m = p.m, ef = p.ef_c, ns = p.sib_seeds;
    const int threads = host_threads(p.num_threads);
    int rc = rank_order(X, attr, n, d, m, p.n_inv, threads, true, out);
    if (rc != FROG_OK) return rc;
    const int H = out->H;
    const float* Xr = out->X.data();
    int32_t* ENC = out->ENC.data();
    const double beta = p.beta, gamma = p.gamma;

    std::vector<int32_t> PG((size_t)n * m, kNone), PGn((size_t)n * m, kNone);

    // ---- leaf layer: brute force inside every leaf segment
    {
        const int h = H - 1;
        // enumerate leaf segments in rank order
        std::vector<std::pair<int64_t, int64_t>> segs;
        for (int64_t u = 0; u < n;) {
            int64_t s, e;
            segment_of(n, h, u, &s, &e);
            segs.emplace_back(s, e);
            u = e + 1;
        }
        parallel_for((int64_t)segs.size(), threads, 4, [&](int64_t si, int) {
            const int64_t s = segs[(size_t)si].first, e = segs[(size_t)si].second;
            const int64_t len = e - s + 1;
            std::vector<float> D((size_t)(len * len));
            std::vector<int32_t> ids((size_t)len);
            for (int64_t v = 0; v < len; ++v) ids[(size_t)v] = (int32_t)(s + v);
            for (int64_t a = 0; a < len; ++a)
                dist_many(Xr, d, Xr + (s + a) * d, ids.data(), (int)len, &D[(size_t)(a * len)]);
            std::vector<Ranked> fu, ve;
            fu.reserve((size_t)len);
            ve.reserve((size_t)len);
            for (int64_t a = 0; a < len; ++a) {
                const int64_t u = s + a;
                fu.clear();
                ve.clear();
                for (int64_t b = 0; b < len; ++b) {
                    if (b == a) continue;
                    float d2 = D[(size_t)(a * len + b)];
                    fu.push_back(Ranked{fusion(d2, u, s + b, len, beta, gamma), d2, (int32_t)(s + b)});
                    ve.push_back(Ranked{(double)d2, d2, (int32_t)(s + b)});
                }
                const int c = (int)fu.size();
                const int keep = std::min(m, c);
                std::partial_sort(fu.begin(), fu.begin() + keep, fu.end(), ranked_less);
                std::partial_sort(ve.begin(), ve.begin() + keep, ve.end(), ranked_less);
                for (int t = 0; t < keep; ++t) {
                    ENC[(u * H + h) * m + t] = fu[(size_t)t].id;
                    PG[(size_t)(u * m + t)] = ve[(size_t)t].id;
                }
            }
        });
    }

    // ---- internal layers, bottom-up
    std::vector<Scratch> scratch((size_t)threads);
    for (auto& S : scratch) S.init(n, m, ef, ns);
    for (int h = H - 2; h >= 0; --h) {
        parallel_for(n, threads, 64, [&](int64_t u, int t) {
            Scratch& S = scratch[(size_t)t];
            int64_t s, e;
            segment_of(n, h, u, &s, &e);
            const int64_t len = e - s + 1;
            const int64_t mid = s + (e - s) / 2;
            int64_t ts, te;
            if (u <= mid) { ts = mid + 1; te = e; } else { ts = s; te = mid; }
            const float* xu = Xr + u * d;
            Ranked* cand = S.cand.data();
            int nc = 0;
            // m-ANN from the child's temporary PG
            {
                int32_t ids[256];
                int c = 0;
                for (int j = 0; j < m; ++j) {
                    int32_t v = PG[(size_t)(u * m + j)];
                    if (v != kNone) ids[c++] = v;
                }
                dist_many(Xr, d, xu, ids, c, S.dtmp.data());
                for (int j = 0; j < c; ++j) {
                    cand[nc].dist = S.dtmp[(size_t)j];
                    cand[nc].key = (double)S.dtmp[(size_t)j];
                    cand[nc].id = ids[j];
                    ++nc;
                }
            }
            // m-ANN from the greedy search over the sibling's temporary PG
            const int64_t tl = te - ts + 1;
            if (tl > 0) {
                int nseeds;
                int32_t* seeds = S.seeds.data();
                if (tl <= ns) {
                    nseeds = (int)tl;
                    for (int j = 0; j < nseeds; ++j) seeds[j] = (int32_t)(ts + j);
                } else {
                    nseeds = ns;
                    for (int j = 0; j < ns; ++j) {
                        int64_t a = ts + ((int64_t)j * tl) / ns;
                        int64_t b = ts + ((int64_t)(j + 1) * tl) / ns - 1;
                        uint64_t z = splitmix64(p.seed ^ ((uint64_t)u << 32) ^ ((uint64_t)h << 24) ^ (uint64_t)j);
                        seeds[j] = (int32_t)(a + (int64_t)reduce_range(z, (uint64_t)(b - a + 1)));
                    }
                }
                int nr = sibling_search(Xr, d, PG.data(), m, xu, ts, te, seeds, nseeds, ef,
                                        p.patience, S, S.res.data(), S.resd.data());
                for (int j = 0; j < nr; ++j) {
                    cand[nc].dist = S.resd[(size_t)j];
                    cand[nc].key = (double)S.resd[(size_t)j];
                    cand[nc].id = S.res[(size_t)j];
                    ++nc;
                }
            }
            std::sort(cand, cand + nc, ranked_less);
            // (i) RNG prune -> row of the parent's temporary PG
            rng_prune(Xr, d, cand, nc, m, &PGn[(size_t)(u * m)], S);
            // (ii) fusion re-rank -> ENC row of layer h
            Ranked* fus = S.fus.data();
            for (int j = 0; j < nc; ++j)
                fus[j] = Ranked{fusion(cand[j].dist, u, cand[j].id, len, beta, gamma), cand[j].dist, cand[j].id};
            const int keep = std::min(m, nc);
            std::partial_sort(fus, fus + keep, fus + nc, ranked_less);
            for (int j = 0; j < keep; ++j) ENC[(u * H + h) * m + j] = fus[j].id;
        });
        std::swap(PG, PGn);
    }
    return FROG_OK;
}

}  // namespace frog
