// FROGSearch, entry mode 1 (shared-priority entry sample): the planning
// kernels (rank interval, threshold, level, run, bucket; bucket offsets;
// order; tiles) and the launch of the whole mode-1 pipeline.

#include "ws_pool.h"
#include "search_shared.h"

namespace frog {
namespace {

__global__ void s_init_kernel(uint32_t* meta, uint32_t* qhist, uint32_t* hist, int nbins, int32_t* order,
                              int64_t norder) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < 4) meta[i] = 0u;
    if (i < 2 * kQSub) qhist[i * kQLine] = 0u;
    if (i < nbins) hist[i] = 0u;
    if (i < norder) order[i] = -1;
}

// Half-wave searches over an ascending array a[0, n): each half counts the
// leading entries for which its predicate holds (lanes 0..31 call
// below(v, false), lanes 32..63 below(v, true); each predicate holds on a
// prefix).  A 32-ary search: every round each lane of a half probes one
// position and the half's ballot narrows its interval 32-fold; the two
// halves run in the same rounds (4 for n = 1M).  Every lane returns its
// half's count.
template <typename TA, typename F>
__device__ int64_t half_count(const TA* __restrict__ a, int64_t n, F below) {
    const int lane = lane_id();
    const int hl = lane & 31;
    const bool upper = lane >= 32;
    int64_t lo = 0, hi = n;   // the count lies in [lo, hi]
    for (;;) {
        const bool live = hi > lo;
        if (ballot(live) == 0) break;
        const int64_t step = (hi - lo + 31) / 32;
        const int64_t p = lo + (int64_t)(hl + 1) * step - 1;
        const bool b = live && p < hi && below(a[p], upper);
        const uint64_t m = ballot(b);
        const int c = __popc((uint32_t)(upper ? (m >> 32) : m));
        if (live) {
            const int64_t nhi = lo + (int64_t)(c + 1) * step - 1;
            lo += (int64_t)c * step;
            hi = nhi < hi ? nhi : hi;
        }
    }
    return lo;
}

// One wavefront per query: the rank interval of its range (the two bounds
// searched side by side, one per half-wave), the threshold, the level, the
// run of the level's list (again one bound per half-wave), its windows, and
// a bucket and place per window (lane wi takes window wi).
__global__ __launch_bounds__(kBlock) void s_plan_kernel(SParams P) {
    const int64_t q = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    if (q >= P.a.nq) return;   // wave-uniform
    const SharedLevels& lv = P.a.lv;
    const int64_t n = P.ix.n;
    const int lane = lane_id();
    const double lo_v = P.a.lo[q], hi_v = P.a.hi[q];
    SPlan p{};
    if (isnan(lo_v) || isnan(hi_v)) {
        p.l = 0;
        p.r = -1;
    } else {
        // l = #{attr < lo}, r = #{attr <= hi} - 1
        const int64_t c = half_count(P.ix.attr, n, [&](double v, bool upper) { return upper ? v <= hi_v : v < lo_v; });
        p.l = __builtin_amdgcn_readlane((int32_t)c, 0);
        p.r = __builtin_amdgcn_readlane((int32_t)c, 32) - 1;
    }
    if (p.l <= p.r) {
        const int64_t cnt = (int64_t)p.r - p.l + 1;
        int64_t E = P.a.epn;
        if (P.a.epn_frac > 0.0) {
            double want = ceil(P.a.epn_frac * (double)cnt);
            if (want > (double)P.a.epn_max) want = (double)P.a.epn_max;
            if (want > (double)E) E = (int64_t)want;
        }
        if (cnt <= E) {
            p.all = 1;
            p.T = 0xFFFFFFFFu;
            p.lev = 0;
        } else {
            // ceil(E 2^32 / cnt) < 2^32 since E < cnt < 2^31
            const uint64_t t = (((uint64_t)E << 32) + (uint64_t)cnt - 1) / (uint64_t)cnt;
            p.T = (uint32_t)t;
            const int cl = t <= 1 ? 0 : 64 - __builtin_clzll(t - 1);   // ceil(log2 t)
            p.lev = 32 - cl < lv.nlev ? 32 - cl : lv.nlev;
        }
        if (p.lev == 0) {
            p.a = p.l;
            p.b = p.r + 1;
        } else {
            // first positions of the level's list with rank >= l and >= r + 1
            const int32_t* ar = lv.ranks + lv.off[p.lev];
            const int64_t len = lv.off[p.lev + 1] - lv.off[p.lev];
            const int32_t x0 = p.l, x1 = p.r + 1;
            const int64_t c = half_count(ar, len, [&](int32_t v, bool upper) { return v < (upper ? x1 : x0); });
            p.a = __builtin_amdgcn_readlane((int32_t)c, 0);
            p.b = __builtin_amdgcn_readlane((int32_t)c, 32);
        }
        if (p.b > p.a) {
            p.w0 = p.a >> P.win_log2;
            p.nw = ((p.b - 1) >> P.win_log2) - p.w0 + 1;
        }
    }
    // a place in the bucket of each window (none when the run meets more
    // than kSMaxWin windows: the pool kernel then evaluates the sample exactly)
    if (p.nw <= kSMaxWin && lane < p.nw) {
        const int bin = pair_bin(P, q, p.lev, p.a, p.b, p.w0, lane);
        P.plan[q].pos[lane] = (int32_t)atomicAdd(P.hist + bin, 1u);
    }
    if (lane == 0) {
        SPlan* dst = P.plan + q;
        // the traversal's order: class 0 (the sample is a strict subset of
        // the range: long traversals) before class 1 (covered or empty
        // ranges: short ones), each class spread over kQSub counters
        const int cls = p.l > p.r || p.all ? 1 : 0;
        dst->qpos = (int32_t)atomicAdd(P.qhist + (cls * kQSub + (q & (kQSub - 1))) * kQLine, 1u);
        dst->l = p.l;
        dst->r = p.r;
        dst->T = p.T;
        dst->all = p.all;
        dst->lev = p.lev;
        dst->a = p.a;
        dst->b = p.b;
        dst->w0 = p.w0;
        dst->nw = p.nw;
        if (P.a.stats) {
            P.a.stats[q * FROG_STAT_N + FROG_STAT_SCANROWS] = 0;
            P.a.stats[q * FROG_STAT_N + FROG_STAT_FALLBACK] = 0;
        }
    }
}

// Bucket offsets in two steps.  s_wprefix_kernel, one thread per window:
// the exclusive prefix of the window's kSPer counts (its buckets in order)
// and the window's total padded to a multiple of 16, so that no tile spans
// two windows.  s_wscan_kernel, one workgroup: the windows' starts (levels in
// order, windows in list order), an exclusive scan of the padded totals in
// place; thread t owns windows [kOffPer t, kOffPer t + kOffPer) (the launch
// keeps nwin within 1024 kOffPer).  A pair's place is then its window's
// start + its bucket's prefix + its place in the bucket.
__global__ __launch_bounds__(256) void s_wprefix_kernel(SParams P) {
    constexpr int kV = kSPer / 4;   // 16-byte vectors per window
    static_assert(kSPer % 4 == 0, "16-byte vectors");
    const int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (x >= P.nwin) return;
    const uint4* src = reinterpret_cast<const uint4*>(P.hist + x * kSPer);
    uint4* dst = reinterpret_cast<uint4*>(P.bstart + x * kSPer);
    uint4 h[kV];
#pragma unroll
    for (int i = 0; i < kV; ++i) h[i] = src[i];
    uint32_t run = 0;
#pragma unroll
    for (int i = 0; i < kV; ++i) {
        uint4 o;
        o.x = run;
        run += h[i].x;
        o.y = run;
        run += h[i].y;
        o.z = run;
        run += h[i].z;
        o.w = run;
        run += h[i].w;
        dst[i] = o;
    }
    P.wstart[x] = (run + kSQ - 1) / kSQ * kSQ;
}

__global__ __launch_bounds__(1024) void s_wscan_kernel(SParams P) {
    __shared__ uint32_t wsum[16];
    const int t = threadIdx.x;
    const int lane = t & 63;
    const int w = t >> 6;
    uint32_t v[kOffPer];
    uint32_t tot = 0;
#pragma unroll
    for (int u = 0; u < kOffPer; ++u) {
        const int x = t * kOffPer + u;
        v[u] = x < P.nwin ? P.wstart[x] : 0u;
        tot += v[u];
    }
    // exclusive scan of the threads' totals: within the wavefront, then over
    // the 16 wavefronts
    uint32_t inc = tot;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const uint32_t s = __shfl_up(inc, o);
        if (lane >= o) inc += s;
    }
    if (lane == 63) wsum[w] = inc;
    // the first place of each (class, counter) of the traversal's query
    // order: an exclusive scan of 2 kQSub counts over the first two wavefronts
    static_assert(kQSub == 64, "one wavefront per class");
    __shared__ uint32_t qsum[2];
    uint32_t qc = 0u, qinc = 0u;
    if (t < 2 * kQSub) {
        qc = P.qhist[t * kQLine];
        qinc = qc;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const uint32_t s = __shfl_up(qinc, o);
            if (lane >= o) qinc += s;
        }
        if (lane == 63) qsum[w] = qinc;
    }
    __syncthreads();
    if (t < 2 * kQSub) P.qhist[2 * kQSub * kQLine + t] = qinc - qc + (w == 1 ? qsum[0] : 0u);
    uint32_t run = inc - tot, all = 0;
    for (int i = 0; i < 16; ++i) {
        run += i < w ? wsum[i] : 0u;
        all += wsum[i];
    }
#pragma unroll
    for (int u = 0; u < kOffPer; ++u) {
        const int x = t * kOffPer + u;
        if (x < P.nwin) P.wstart[x] = run;
        run += v[u];
    }
    if (t == 0) {
        P.meta[0] = all;
        P.meta[1] = all / kSQ;
    }
}

// thread per query: the query to its place in the traversal's order, and
// each (query, window) pair to its place
__global__ void s_order_kernel(SParams P) {
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= P.a.nq) return;
    const SPlan* p = P.plan + q;
    const int cls = p->l > p->r || p->all ? 1 : 0;
    P.qorder[P.qhist[2 * kQSub * kQLine + cls * kQSub + (q & (kQSub - 1))] + p->qpos] = (int32_t)q;
    const int nw = p->nw;
    if (nw > kSMaxWin || p->l > p->r) return;
    const int lev = p->lev;
    const int32_t a = p->a, b = p->b, w0 = p->w0;
    for (int wi = 0; wi < nw; ++wi)
        P.order[P.wstart[P.winbase[lev] + w0 + wi] + P.bstart[pair_bin(P, q, lev, a, b, w0, wi)] + p->pos[wi]] =
            (int32_t)(q * kSMaxWin + wi);
}

// one wavefront per tile: lanes 0..15 take its slots, each slot the piece of
// its query's run inside the tile's window
__global__ __launch_bounds__(kBlock) void s_tile_kernel(SParams P) {
    const int lane = lane_id();
    const int64_t t = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    if (t >= P.tmax) return;
    const int64_t places = P.meta[0];
    STile* T = P.tiles + t;
    const int64_t i = t * kSQ + lane;
    int32_t e = -1;
    if (lane < kSQ && i < places) e = P.order[i];
    const int32_t q = e >= 0 ? e / kSMaxWin : -1;
    const int wi = e >= 0 ? e % kSMaxWin : 0;
    SPlan* p = P.plan + (q >= 0 ? q : 0);
    int32_t l = 0, r = -1, lev = 64, all = 0;
    int32_t sa = 0x7FFFFFFF, sb = -1;
    uint32_t thr = 0u;
    if (q >= 0) {
        l = p->l;
        r = p->r;
        thr = p->T;
        lev = p->lev;
        all = p->all;
        const int64_t ws = (int64_t)(p->w0 + wi) << P.win_log2;
        const int64_t we = ws + ((int64_t)1 << P.win_log2);
        sa = (int32_t)(p->a > ws ? p->a : ws);
        sb = (int32_t)(p->b < we ? p->b : we);
    }
    if (lane < kSQ) {
        T->pair[lane] = e;
        T->l[lane] = l;
        T->r[lane] = r;
        T->T[lane] = thr;
    }
    const uint64_t valid = __ballot(q >= 0);
    const uint64_t allm = __ballot(q >= 0 && all);
    int32_t ua = sa, ub = sb, lv = lev;
#pragma unroll
    for (int o = 1; o < kSQ; o <<= 1) {
        ua = min(ua, __shfl_xor(ua, o));
        ub = max(ub, __shfl_xor(ub, o));
        lv = min(lv, __shfl_xor(lv, o));
    }
    ua = uniform(ua);
    ub = uniform(ub);
    lv = uniform(lv);
    const int nq = __popcll(valid);
    // work items: the scan's wavefronts take the tiles' first chunks in tile
    // order; tiles beyond the first scan_slots (a second round) are cut in up
    // to 4 times as many chunks, so that the round that ends the scan is
    // short (with fewer tiles than slots, as many tiles are cut as still fit
    // in one round)
    const int64_t ntiles = P.meta[1];
    const int64_t nfit = (P.scan_slots - ntiles) / 3;   // a tile cut in 4 adds 3 items
    const int64_t nsplit = ntiles > P.scan_slots ? ntiles - P.scan_slots : (nfit < ntiles ? nfit : ntiles);
    const int64_t span = (int64_t)ub - ua;
    int nch = tile_chunks(span, P.nbase, P.chunk_log2);
    if (t >= ntiles - nsplit && span >= 256) nch = 4 * nch < P.nchunk ? 4 * nch : P.nchunk;
    if (q >= 0) p->wchunks[wi] = nch;
    if (lane == 0) {
        T->nch = nch;
        T->allmask = (uint32_t)allm;
        T->lev = nq > 0 ? lv : 0;
        T->ua = nq > 0 ? ua : 0;
        T->ub = nq > 0 ? ub : 0;
        T->nq = nq;
    }
}

}  // namespace

// entry_mode 1: plan, group, scan on the matrix cores, then search
int launch_shared(const DevIndex& ix, const SearchLaunch& a, hipStream_t stream, void* ws, size_t ws_cap) {
    const int kkeep = shared_kkeep(a.L);
    auto sfn = pick_s_search(ix.dp, a.L, ix.storage, lean_launch(a));
    auto pfn = pick_s_pool(ix.dp, a.L, ix.storage);
    // search kernel: pool staging, EN list and visited table per wave
    const int lps = lds_per_wave(a.L, a.hash_log2);
    const int smem = lps * kWavesPerBlock;
    // pool kernel: pool staging and EN list, then the re-rank list
    const int base_lds = lds_per_wave(a.L, 0);
    const int lpw = base_lds + 2 * pool_kkeep(kkeep, a.L) * 8 + 16;
    const int smem_pool = lpw;   // one wavefront (query) per workgroup, as for the scan
    if (smem > 160 * 1024 || smem_pool > 160 * 1024)
        return fail(FROG_EUNSUPPORTED, "LDS per block %d / %d too large", smem, smem_pool);
    if (smem > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void*)sfn, hipFuncAttributeMaxDynamicSharedMemorySize, smem);
        if (e != hipSuccess) return fail(FROG_EHIP, "hipFuncSetAttribute: %s", hipGetErrorString(e));
    }
    if (smem_pool > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void*)pfn, hipFuncAttributeMaxDynamicSharedMemorySize, smem_pool);
        if (e != hipSuccess) return fail(FROG_EHIP, "hipFuncSetAttribute: %s", hipGetErrorString(e));
    }
    auto scan = pick_s_scan(ix.dp, kkeep, ix.storage);
    // one wavefront per scan workgroup: a workgroup's LDS is released only
    // when all its wavefronts have ended, and work items differ in length, so
    // with four per workgroup the LDS of finished items sat idle beside the
    // longest one (C2: 0.407 ms with four, 0.383 ms with one)
    const int scan_waves = 1;
    if (s_scan_lds_per_wave(kkeep) > 160 * 1024)
        return fail(FROG_EUNSUPPORTED, "L=%d needs too much LDS for the entry scan", a.L);
    const int smem_scan = (int)(scan_waves * s_scan_lds_per_wave(kkeep));
    if (smem_scan > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void*)scan, hipFuncAttributeMaxDynamicSharedMemorySize, smem_scan);
        if (e != hipSuccess) return fail(FROG_EHIP, "hipFuncSetAttribute: %s", hipGetErrorString(e));
    }
    const int scan_slots = max_blocks((const void*)scan, smem_scan, 64 * scan_waves) * scan_waves;
    SParams P{};
    P.ix = ix;
    P.a = a;
    // (a pair id, query * kSMaxWin + window index, is an int32)
    if (a.nq > ((int64_t)1 << 28))
        return fail(FROG_EUNSUPPORTED, "entry_mode 1 takes at most 2^28 queries per call (nq=%lld)", (long long)a.nq);
    // windows: W >= 1024 positions, at least 2/5 of the largest sample (a
    // run, about E to 2E positions, then meets at most about 6 windows) and
    // at least n / 1024 (about 2048 windows over all levels); wider while the
    // levels hold more windows than the offsets kernel takes
    {
        const int64_t emax = a.epn_frac > 0.0 && a.epn_max > a.epn ? a.epn_max : a.epn;
        int lg = 10;
        while (((int64_t)1 << lg) < (2 * emax + 4) / 5 || ((int64_t)1 << lg) * 1024 < ix.n) ++lg;
        for (;; ++lg) {
            const int64_t W = (int64_t)1 << lg;
            int64_t nw = 0;
            for (int j = 0; j <= a.lv.nlev; ++j) {
                P.winbase[j] = (int32_t)nw;
                const int64_t len = j == 0 ? ix.n : a.lv.off[j + 1] - a.lv.off[j];
                nw += (len + W - 1) / W;
            }
            P.winbase[a.lv.nlev + 1] = (int32_t)nw;
            P.nwin = (int)nw;
            if (nw <= 1024 * kOffPer) break;   // what s_wscan_kernel takes
        }
        P.win_log2 = lg;
        const int64_t W = (int64_t)1 << lg;
        // work items: a tile of the scan's first round (the first
        // scan_slots tiles) is cut into chunks of W / nbase rows, at least
        // kSChunkRows: one per tile at W = 1024, up to 4 of W / 4 above (2
        // for 256-entry lists, whose cuts and merges cost more per list); a
        // tile of the second round into up to 4 times as many, so that the
        // round that ends the scan is short.  Uniform items fit worse: at C2
        // (3,600 tiles on 3,072 slots) one 1024-row item per tile took
        // 475 us, two 512-row items 492 us, four 256-row items 512 us (each
        // item carries its 16 queries' operands and 16 lists' final cuts and
        // write-out), and cutting only the second round's tiles in four,
        // 426 us.
        const int cmax = kkeep >= 256 ? 2 : kSMaxChunks;
        P.nbase = W / kSChunkRows < cmax ? (int)(W / kSChunkRows) : cmax;
        P.chunk_log2 = lg - (P.nbase == 4 ? 2 : (P.nbase == 2 ? 1 : 0));
        P.nchunk = 4 * P.nbase < cmax ? 4 * P.nbase : cmax;
    }
    // places: at most kSMaxWin pairs per query, plus up to 15 of padding per window
    const int64_t norder = (int64_t)kSMaxWin * a.nq + (int64_t)kSQ * P.nwin;
    P.tmax = (norder + kSQ - 1) / kSQ;
    P.scan_slots = scan_slots;
    P.nbins = P.nwin * kSPer;
    P.kkeep = kkeep;
    P.lds_per_wave = lpw;
    P.lds_list = base_lds;
    P.lds_search = lps;
    int blocks = max_blocks((const void*)sfn, smem);
    const int64_t need = (a.nq + kWavesPerBlock - 1) / kWavesPerBlock;
    if (need < blocks) blocks = (int)need;
    const int64_t items = P.tmax * P.nchunk;
    auto align = [](size_t x) { return (x + 255) / 256 * 256; };
    size_t off = 0;
    auto take = [&](size_t bytes) { const size_t o = off; off += align(bytes); return o; };
    const size_t o_meta = take(16);
    const size_t o_qhist = take((2 * kQSub * kQLine + 2 * kQSub) * 4);
    const size_t o_qorder = take((size_t)a.nq * 4);
    const size_t o_plan = take((size_t)a.nq * sizeof(SPlan));
    const size_t o_hist = take((size_t)P.nbins * 4);
    const size_t o_bstart = take((size_t)P.nbins * 4);
    const size_t o_wstart = take((size_t)P.nwin * 4);
    const size_t o_order = take((size_t)norder * 4);
    const size_t o_tiles = take((size_t)P.tmax * sizeof(STile));
    const int64_t nlists = a.nq * kSMaxWin * P.nchunk;   // (pair, chunk)
    const size_t o_pv = take((size_t)nlists * kkeep * 4);
    const size_t o_pr = take((size_t)nlists * kkeep * 4);
    const size_t o_pthr = take((size_t)nlists * 4);
    const size_t o_pfill = take((size_t)nlists * 4);
    const size_t o_pcnt = take((size_t)nlists * 4);
    const int lp = lp_of(a.L);
    const size_t o_pools = take((size_t)a.nq * 64 * lp * 8);
    const size_t o_pne = take((size_t)a.nq * 4);
    const size_t o_gvis = off;
    if (a.hash_log2 == 0) {
        P.gvis_words = (ix.n + 31) / 32;
        const int64_t cap = ((int64_t)2 << 30) / (P.gvis_words * 4 * kWavesPerBlock);
        if (cap < blocks) blocks = (int)(cap > 0 ? cap : 1);
        off += (size_t)blocks * kWavesPerBlock * P.gvis_words * 4;
    }
    void* wsp = ws;
    hipError_t e = hipSuccess;
    WsLease lease;
    if (ws) {
        if (off > ws_cap)
            return fail(FROG_EUNSUPPORTED,
                        "this call needs %zu bytes of workspace; the scratch array holds %zu (nq=%lld, L=%d, "
                        "entry_mode 1%s)", off, ws_cap, (long long)a.nq, a.L,
                        a.hash_log2 == 0 ? ", exact visited set" : "");
    } else {
        e = lease.acquire(stream, off, &wsp);
        if (e != hipSuccess)
            return fail(e == hipErrorOutOfMemory ? FROG_ENOMEM : FROG_EHIP, "workspace: %s", hipGetErrorString(e));
    }
    char* base = reinterpret_cast<char*>(wsp);
    P.meta = reinterpret_cast<uint32_t*>(base + o_meta);
    P.qhist = reinterpret_cast<uint32_t*>(base + o_qhist);
    P.qorder = reinterpret_cast<int32_t*>(base + o_qorder);
    P.plan = reinterpret_cast<SPlan*>(base + o_plan);
    P.hist = reinterpret_cast<uint32_t*>(base + o_hist);
    P.bstart = reinterpret_cast<uint32_t*>(base + o_bstart);
    P.wstart = reinterpret_cast<uint32_t*>(base + o_wstart);
    P.order = reinterpret_cast<int32_t*>(base + o_order);
    P.tiles = reinterpret_cast<STile*>(base + o_tiles);
    P.pv = reinterpret_cast<float*>(base + o_pv);
    P.pr = reinterpret_cast<int32_t*>(base + o_pr);
    P.pthr = reinterpret_cast<float*>(base + o_pthr);
    P.pfill = reinterpret_cast<int32_t*>(base + o_pfill);
    P.pcnt = reinterpret_cast<int32_t*>(base + o_pcnt);
    P.pools = reinterpret_cast<uint64_t*>(base + o_pools);
    P.pne = reinterpret_cast<int32_t*>(base + o_pne);
    P.gvis = reinterpret_cast<uint32_t*>(base + o_gvis);
    hipEvent_t* ev = reinterpret_cast<hipEvent_t*>(a.events);
    const unsigned qb = (unsigned)((a.nq + 255) / 256);
    // events: before the matrix-core scan, after it, after the search kernel
    // (the planning kernels come before the first, the pool kernel after the
    // second)
    const int64_t ninit = norder > P.nbins ? norder : P.nbins;
    hipLaunchKernelGGL(s_init_kernel, dim3((unsigned)((ninit + 255) / 256)), dim3(256), 0, stream, P.meta, P.qhist,
                       P.hist, P.nbins, P.order, norder);
    const int64_t plan_blocks = (a.nq + kWavesPerBlock - 1) / kWavesPerBlock;
    hipLaunchKernelGGL(s_plan_kernel, dim3((unsigned)plan_blocks), dim3(kBlock), 0, stream, P);
    hipLaunchKernelGGL(s_wprefix_kernel, dim3((unsigned)((P.nwin + 255) / 256)), dim3(256), 0, stream, P);
    hipLaunchKernelGGL(s_wscan_kernel, dim3(1), dim3(1024), 0, stream, P);
    hipLaunchKernelGGL(s_order_kernel, dim3(qb), dim3(256), 0, stream, P);
    hipLaunchKernelGGL(s_tile_kernel, dim3((unsigned)((P.tmax + kWavesPerBlock - 1) / kWavesPerBlock)), dim3(kBlock),
                       0, stream, P);
    if (ev) (void)hipEventRecord(ev[0], stream);
    hipLaunchKernelGGL(scan, dim3((unsigned)((items + scan_waves - 1) / scan_waves)), dim3(64 * scan_waves), smem_scan,
                       stream, P);
    if (ev) (void)hipEventRecord(ev[1], stream);
    hipLaunchKernelGGL(pfn, dim3((unsigned)a.nq), dim3(64), smem_pool,
                       stream, P);
    hipLaunchKernelGGL(sfn, dim3(blocks), dim3(kBlock), smem, stream, P);
    if (ev) (void)hipEventRecord(ev[2], stream);
    e = hipGetLastError();
    lease.release();
    if (e != hipSuccess) return fail(FROG_EHIP, "search launch: %s", hipGetErrorString(e));
    return FROG_OK;
}

}  // namespace frog
