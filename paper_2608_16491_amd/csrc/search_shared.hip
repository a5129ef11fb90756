// FROGSearch, entry mode 1 (shared-priority entry sample): the planning
// kernels (rank interval, threshold, level, run, bucket; bucket offsets;
// order; tiles) and the launch of the whole mode-1 pipeline.

#include "ws_pool.h"
#include "search_shared.h"

namespace frog {
namespace {

__global__ void s_init_kernel(uint32_t* meta, uint32_t* hist, int nbins, int32_t* order, int64_t norder) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < 4) meta[i] = 0u;
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
// run of the level's list (again one bound per half-wave) and a bucket.
__global__ __launch_bounds__(kBlock) void s_plan_kernel(SParams P) {
    const int64_t q = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    if (q >= P.a.nq) return;   // wave-uniform
    const SharedLevels& lv = P.a.lv;
    const int64_t n = P.ix.n;
    const double lo_v = P.a.lo[q], hi_v = P.a.hi[q];
    SPlan p{};
    p.tslot = -1;
    if (isnan(lo_v) || isnan(hi_v)) {
        p.l = 0;
        p.r = -1;
    } else {
        // l = #{attr < lo}, r = #{attr <= hi} - 1
        const int64_t c = half_count(P.ix.attr, n, [&](double v, bool upper) { return upper ? v <= hi_v : v < lo_v; });
        p.l = __builtin_amdgcn_readlane((int32_t)c, 0);
        p.r = __builtin_amdgcn_readlane((int32_t)c, 32) - 1;
    }
    if (p.l > p.r) {
        p.bin = P.nbins - 1;
    } else {
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
        // queries sorted by the midpoint of their range share most of their
        // runs, so a tile's union stays close to one run
        p.bin = p.lev * kSBins + (int)((((int64_t)p.l + p.r) * kSBins) / (2 * n));
    }
    if (lane_id() == 0) {
        p.pos = (int32_t)atomicAdd(P.hist + p.bin, 1u);
        P.plan[q] = p;
        P.lr[2 * q] = p.l;
        P.lr[2 * q + 1] = p.r;
        if (P.a.stats) {
            P.a.stats[q * FROG_STAT_N + FROG_STAT_SCANROWS] = 0;
            P.a.stats[q * FROG_STAT_N + FROG_STAT_FALLBACK] = 0;
        }
    }
}

// Bucket offsets: level by level, each level's run of places padded to a
// multiple of 16; inside a level, buckets in order of the range midpoint.
// The empty ranges' bucket comes last.  Wavefront w owns levels w and w + 16
// (nlev <= 31); lane i owns buckets [32 i, 32 i + 32) of a level, read and
// written as 16-byte vectors.
__global__ __launch_bounds__(1024) void s_offsets_kernel(SParams P) {
    static_assert(kSBins == 64 * 32, "32 buckets per lane");
    constexpr int kWaves = 1024 / 64;
    __shared__ uint32_t start[34];
    const int t = threadIdx.x;
    const int lane = t & 63;
    const int w = t >> 6;
    const int nlev = P.a.lv.nlev;
    uint4 h[2][8];
    uint32_t excl[2] = {0u, 0u};
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        const int j = w + kWaves * s;   // wave-uniform
        uint32_t sum = 0;
#pragma unroll
        for (int i = 0; i < 8; ++i) h[s][i] = make_uint4(0u, 0u, 0u, 0u);
        if (j <= nlev) {
            const uint4* src = reinterpret_cast<const uint4*>(P.hist + (size_t)j * kSBins + lane * 32);
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                h[s][i] = src[i];
                sum += h[s][i].x + h[s][i].y + h[s][i].z + h[s][i].w;
            }
        }
        // exclusive scan of the lanes' sums
        uint32_t inc = sum;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const uint32_t v = __shfl_up(inc, o);
            if (lane >= o) inc += v;
        }
        excl[s] = inc - sum;
        if (lane == 63 && j <= nlev) start[j + 1] = (inc + kSQ - 1) / kSQ * kSQ;
    }
    __syncthreads();
    if (t == 0) {
        start[0] = 0;
        for (int i = 1; i <= nlev + 1; ++i) start[i] += start[i - 1];
        P.bstart[P.nbins - 1] = start[nlev + 1];
        P.meta[0] = start[nlev + 1];
        P.meta[1] = start[nlev + 1] / kSQ;
    }
    __syncthreads();
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        const int j = w + kWaves * s;
        if (j > nlev) continue;
        uint32_t run = start[j] + excl[s];
        uint4* dst = reinterpret_cast<uint4*>(P.bstart + (size_t)j * kSBins + lane * 32);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            uint4 o;
            o.x = run;
            run += h[s][i].x;
            o.y = run;
            run += h[s][i].y;
            o.z = run;
            run += h[s][i].z;
            o.w = run;
            run += h[s][i].w;
            dst[i] = o;
        }
    }
}

__global__ void s_order_kernel(SParams P) {
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= P.a.nq) return;
    const SPlan& p = P.plan[q];
    P.order[P.bstart[p.bin] + p.pos] = (int32_t)q;
}

// one wavefront per tile: lanes 0..15 take its slots
__global__ __launch_bounds__(kBlock) void s_tile_kernel(SParams P) {
    const int lane = lane_id();
    const int64_t t = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    if (t >= P.tmax) return;
    const int64_t places = P.meta[0];
    STile* T = P.tiles + t;
    const int64_t i = t * kSQ + lane;
    int32_t q = -1;
    if (lane < kSQ && i < places) q = P.order[i];
    int32_t l = 0, r = -1, lev = 64, all = 0;
    uint32_t thr = 0u;
    if (q >= 0) {
        SPlan& p = P.plan[q];
        l = p.l;
        r = p.r;
        thr = p.T;
        lev = p.lev;
        all = p.all;
        p.tslot = (int32_t)(t * kSQ + lane);
    }
    if (lane < kSQ) {
        T->q[lane] = q;
        T->l[lane] = l;
        T->r[lane] = r;
        T->T[lane] = thr;
    }
    const uint64_t valid = __ballot(q >= 0);
    const uint64_t allm = __ballot(q >= 0 && all);
    int32_t ul = q >= 0 ? l : 0x7FFFFFFF, ur = q >= 0 ? r : -1, lv = lev;
#pragma unroll
    for (int o = 1; o < kSQ; o <<= 1) {
        ul = min(ul, __shfl_xor(ul, o));
        ur = max(ur, __shfl_xor(ur, o));
        lv = min(lv, __shfl_xor(lv, o));
    }
    ul = uniform(ul);
    ur = uniform(ur);
    lv = uniform(lv);
    const int nq = __popcll(valid);
    // lane 0: the union's first position, lane 1: its end
    int64_t pos = 0;
    if (nq > 0 && lane < 2) pos = level_lower(P.a.lv, P.ix.n, lv, lane == 0 ? (int64_t)ul : (int64_t)ur + 1);
    const int32_t ua = __builtin_amdgcn_readlane((int32_t)pos, 0);
    const int32_t ub = __builtin_amdgcn_readlane((int32_t)pos, 1);
    if (lane == 0) {
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
    const int smem_pool = lpw * kWavesPerBlock;
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
    // wavefronts per scan workgroup: as many as 160 KB of LDS hold (at most 4)
    int scan_waves = (int)((160 * 1024) / s_scan_lds_per_wave(kkeep));
    if (scan_waves > kWavesPerBlock) scan_waves = kWavesPerBlock;
    if (scan_waves < 1) return fail(FROG_EUNSUPPORTED, "L=%d needs too much LDS for the entry scan", a.L);
    const int smem_scan = (int)(scan_waves * s_scan_lds_per_wave(kkeep));
    if (smem_scan > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void*)scan, hipFuncAttributeMaxDynamicSharedMemorySize, smem_scan);
        if (e != hipSuccess) return fail(FROG_EHIP, "hipFuncSetAttribute: %s", hipGetErrorString(e));
    }
    SParams P{};
    P.ix = ix;
    P.a = a;
    const int64_t norder = a.nq + (int64_t)kSQ * (a.lv.nlev + 1);
    P.tmax = (norder + kSQ - 1) / kSQ;
    P.nbins = (a.lv.nlev + 1) * kSBins + 1;
    P.kkeep = kkeep;
    P.lds_per_wave = lpw;
    P.lds_list = base_lds;
    P.lds_search = lps;
    int blocks = max_blocks((const void*)sfn, smem);
    const int64_t need = (a.nq + kWavesPerBlock - 1) / kWavesPerBlock;
    if (need < blocks) blocks = (int)need;
    const int64_t items = P.tmax * kSChunks;
    auto align = [](size_t x) { return (x + 255) / 256 * 256; };
    size_t off = 0;
    auto take = [&](size_t bytes) { const size_t o = off; off += align(bytes); return o; };
    const size_t o_meta = take(16);
    const size_t o_lr = take((size_t)a.nq * 8);
    const size_t o_plan = take((size_t)a.nq * sizeof(SPlan));
    const size_t o_hist = take((size_t)P.nbins * 4);
    const size_t o_bstart = take((size_t)P.nbins * 4);
    const size_t o_order = take((size_t)norder * 4);
    const size_t o_tiles = take((size_t)P.tmax * sizeof(STile));
    const size_t o_pv = take((size_t)items * kSQ * kkeep * 4);
    const size_t o_pr = take((size_t)items * kSQ * kkeep * 4);
    const size_t o_pthr = take((size_t)items * kSQ * 4);
    const size_t o_pfill = take((size_t)items * kSQ * 4);
    const size_t o_pcnt = take((size_t)items * kSQ * 4);
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
    int32_t* lr = reinterpret_cast<int32_t*>(base + o_lr);
    P.lr = lr;
    P.plan = reinterpret_cast<SPlan*>(base + o_plan);
    P.hist = reinterpret_cast<uint32_t*>(base + o_hist);
    P.bstart = reinterpret_cast<uint32_t*>(base + o_bstart);
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
    hipLaunchKernelGGL(s_init_kernel, dim3((unsigned)((ninit + 255) / 256)), dim3(256), 0, stream, P.meta, P.hist,
                       P.nbins, P.order, norder);
    const int64_t plan_blocks = (a.nq + kWavesPerBlock - 1) / kWavesPerBlock;
    hipLaunchKernelGGL(s_plan_kernel, dim3((unsigned)plan_blocks), dim3(kBlock), 0, stream, P);
    hipLaunchKernelGGL(s_offsets_kernel, dim3(1), dim3(1024), 0, stream, P);
    hipLaunchKernelGGL(s_order_kernel, dim3(qb), dim3(256), 0, stream, P);
    hipLaunchKernelGGL(s_tile_kernel, dim3((unsigned)((P.tmax + kWavesPerBlock - 1) / kWavesPerBlock)), dim3(kBlock),
                       0, stream, P);
    if (ev) (void)hipEventRecord(ev[0], stream);
    hipLaunchKernelGGL(scan, dim3((unsigned)((items + scan_waves - 1) / scan_waves)), dim3(64 * scan_waves), smem_scan,
                       stream, P);
    if (ev) (void)hipEventRecord(ev[1], stream);
    hipLaunchKernelGGL(pfn, dim3((unsigned)((a.nq + kWavesPerBlock - 1) / kWavesPerBlock)), dim3(kBlock), smem_pool,
                       stream, P);
    hipLaunchKernelGGL(sfn, dim3(blocks), dim3(kBlock), smem, stream, P);
    if (ev) (void)hipEventRecord(ev[2], stream);
    e = hipGetLastError();
    lease.release();
    if (e != hipSuccess) return fail(FROG_EHIP, "search launch: %s", hipGetErrorString(e));
    return FROG_OK;
}

}  // namespace frog
