// The shared entry sample (entry mode 1): plans, tiles and the parameters
// of its kernels, which four translation units share (planning and launch,
// the matrix-core scan, the pool, the traversal).
#pragma once

#include "search_common.h"

namespace frog {

// ================================================================== shared entry sample
//
// Second reading of the entry-point sampling (entry_mode 1).  Rank i carries
// the priority p(i) = hi32(splitmix64(key ^ i)), key = splitmix64(seed); a
// query asking for E entry points out of cnt ranks takes the ranks of [l, r]
// with p(i) < T, T = ceil(E 2^32 / cnt) (every rank when cnt <= E).  Level
// j >= 1 lists, in rank order, the ranks with p < 2^(32-j); level 0 is every
// rank.  A query's sample lies in the coarsest level whose bound is at least
// T, where it is the run of the list between l and r, filtered by T.
//
// The sample depends on (seed, rank) only, so queries over overlapping ranges
// at the same level draw from the same rows, and their entry distances form
// a dense product (16 queries x a run of rows) for the fp32 matrix cores in
// place of per-query gathers:
//   s_plan_kernel     per query (one wavefront): rank interval, threshold,
//                     level, run in the level's list, and a bucket (level,
//                     range midpoint) for grouping
//   s_offsets_kernel  bucket offsets (one workgroup)
//   s_order_kernel    the queries in bucket order
//   s_tile_kernel     tiles of 16 consecutive queries: the union of their
//                     runs in the finest level among them
//   s_scan_kernel     one wavefront per (tile, eighth of the union): 16 x 16
//                     blocks of q.x on the matrix cores, the approximate
//                     squared distance |q|^2 + |x|^2 - 2 q.x of each query's
//                     sample rows, the kkeep smallest per query kept in LDS
//   s_pool_kernel     one wavefront per query: the kkeep smallest of its
//                     tile's lists, re-ranked with the exact canonical
//                     distance into the pool (the L nearest entry points); a
//                     margin test proves that no row left out could enter the
//                     pool, else the whole sample is evaluated exactly
//   s_search_kernel   one wavefront per query (persistent grid, ~100 VGPRs,
//                     5 wavefronts per SIMD): the traversal from that pool,
//                     where the sample's ranks count as visited by their
//                     priority.
// Bucket order inside a bucket follows atomic arrival, so tiles differ from
// run to run; results do not, since every pool is the exact L nearest of the
// sample.

constexpr int kSQ = 16;        // queries per tile
constexpr int kSChunks = 8;    // work items per tile
constexpr int kSBins = 2048;   // buckets of the range midpoint per level

struct SPlan {
    int32_t l, r;
    uint32_t T;      // threshold
    int32_t all;     // every rank of the range is an entry point
    int32_t lev;     // level whose list holds the sample
    int32_t a, b;    // run [a, b) of [l, r] in that list
    int32_t bin, pos;
    int32_t tslot;   // tile * 16 + slot (-1: empty range)
    int32_t pad[2];
};

struct STile {
    int32_t q[kSQ];
    int32_t l[kSQ];
    int32_t r[kSQ];
    uint32_t T[kSQ];
    uint32_t allmask;
    int32_t lev;      // finest level among the tile's queries
    int32_t ua, ub;   // run of the union of their intervals in that level's list
    int32_t nq;       // 0: unused tile
    int32_t pad[3];
};

struct SParams {
    DevIndex ix;
    SearchLaunch a;
    int32_t* lr;        // [nq][2] rank intervals (written by s_plan_kernel)
    SPlan* plan;
    uint32_t* hist;     // [nbins] queries per bucket
    uint32_t* bstart;   // [nbins] first place of each bucket
    uint32_t* meta;     // [0] places used in `order`, [1] tiles, [2] query counter
    int32_t* order;     // [nq + 16 (nlev + 1)] queries by bucket, each level's run
                        // padded to a multiple of 16 with -1 (no tile spans two levels)
    STile* tiles;       // [tmax]
    int64_t tmax;
    int nbins;
    int kkeep;
    float* pv;          // [tmax * kSChunks][16][kkeep] approximate distances
    int32_t* pr;        // [tmax * kSChunks][16][kkeep] ranks
    float* pthr;        // [tmax * kSChunks][16] threshold of a full list, else +inf
    int32_t* pfill;     // [tmax * kSChunks][16] entries kept
    int32_t* pcnt;      // [tmax * kSChunks][16] sample rows seen
    uint64_t* pools;    // [nq][64 LP] the L nearest sample points per query (sorted keys)
    int32_t* pne;       // [nq] sample size
    uint32_t* gvis;
    int64_t gvis_words;
    int lds_per_wave;   // s_pool_kernel, bytes
    int lds_list;       // offset of the re-rank list inside its wave's LDS
    int lds_search;     // s_search_kernel, bytes per wave
};

using SKernel = void (*)(SParams);
// kernels of the other units, picked by shape
SKernel pick_s_scan(int dp, int kkeep, int storage);   // search_scan.hip
SKernel pick_s_pool(int dp, int L, int storage);       // search_pool.hip
// lean: no statistics, lazy check, LDS visited table (the timed configuration)
SKernel pick_s_search(int dp, int L, int storage, bool lean);   // search_trav.hip
// entry_mode 1: plan, group, scan on the matrix cores, then search (search_shared.hip)
// ws: NULL (stream-ordered allocation) or ws_cap bytes of caller-provided
// device memory
int launch_shared(const DevIndex& ix, const SearchLaunch& a, hipStream_t stream, void* ws, size_t ws_cap);

namespace {

// the timed configuration, which the lean traversal serves
inline bool lean_launch(const SearchLaunch& a) { return !a.stats && !a.eager && a.hash_log2 > 0; }

__device__ __forceinline__ int32_t level_rank(const SharedLevels& lv, int j, int64_t pos) {
    return j == 0 ? (int32_t)pos : lv.ranks[lv.off[j] + pos];
}

// first position of level j's list whose rank is >= x.  One thread: a
// 16-ary search whose 15 probes per round are independent loads (about 5
// dependent rounds at n = 1M instead of 20 binary steps), then a binary
// search over the last 16 positions.
__device__ int64_t level_lower(const SharedLevels& lv, int64_t n, int j, int64_t x) {
    if (j == 0) return x < 0 ? 0 : (x > n ? n : x);
    const int32_t* a = lv.ranks + lv.off[j];
    // the answer lies in [lo, hi]: a[i] < x for i < lo, a[hi] >= x or hi = end
    int64_t lo = 0, hi = lv.off[j + 1] - lv.off[j];
    while (hi - lo > 16) {
        const int64_t step = (hi - lo) / 16;   // probes lo + t step, t = 1..15, all < hi
        int c = 0;
#pragma unroll
        for (int t = 1; t < 16; ++t) c += a[lo + t * step] < x ? 1 : 0;
        // the ranks ascend: probes 1..c are below x, c + 1 .. 15 are not
        const int64_t nlo = c > 0 ? lo + c * step + 1 : lo;
        if (c < 15) hi = lo + (c + 1) * step;
        lo = nlo;
    }
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (a[mid] < x) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

__device__ __forceinline__ uint32_t s_priority(uint64_t key, int32_t i) {
    return (uint32_t)(splitmix64(key ^ (uint64_t)(uint32_t)i) >> 32);
}

// per wave: 16 buffers of 2 kkeep keys, |q|^2 of the 16 queries, 16 list states
__host__ __device__ constexpr size_t s_scan_lds_per_wave(int kkeep) {
    return (size_t)kSQ * 2 * kkeep * 8 + kSQ * 4 + kSQ * 8;
}

// candidates kept per query and work item: K >= L + 8, room for the margin
// (pools above 248 keep 256 per work item and 512 when merged)
inline int shared_kkeep(int L) { return L + 8 <= 48 ? 48 : (L + 8 <= 64 ? 64 : (L + 8 <= 128 ? 128 : 256)); }
// the pool kernel's merged list: at least 64
inline int pool_kkeep(int kkeep, int L) { return L > 248 ? 512 : (kkeep > 64 ? kkeep : 64); }

}  // namespace
}  // namespace frog
