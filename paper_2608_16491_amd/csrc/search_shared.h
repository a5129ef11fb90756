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
// place of per-query gathers.  Each level's list is cut into windows of W
// positions (a power of two); a query's run meets a few consecutive windows,
// and each (query, window) pair is one slot of a tile, so that a tile covers
// at most one window and reads only the rows of that window that its 16
// queries' runs span:
//   s_plan_kernel     per query (one wavefront): rank interval, threshold,
//                     level, run in the level's list, its windows, and per
//                     window a bucket (window, kind and place of the pair's
//                     piece of the run inside it); a place in the query
//                     order of the pool and traversal kernels (queries whose
//                     sample is a strict subset of their range first, the
//                     short covered and empty ones last, to fill the tails)
//   s_wprefix_kernel, s_wscan_kernel
//                     bucket offsets, each window's places padded to a
//                     multiple of 16; the query order's offsets
//   s_order_kernel    the pairs in bucket order, the queries in their order
//   s_tile_kernel     tiles of 16 consecutive places: the span of their
//                     pieces of the window
//   s_scan_kernel     one wavefront per (tile, chunk of its span): 16 x 16
//                     blocks of q.x on the matrix cores, the approximate
//                     squared distance |q|^2 + |x|^2 - 2 q.x of each query's
//                     sample rows, the kkeep smallest per query kept in LDS
//   s_pool_kernel     one wavefront per query: the kkeep smallest of all its
//                     lists (every chunk of every window), re-ranked with the
//                     exact canonical distance into the pool (the L nearest
//                     entry points); a margin test proves that no row left out
//                     could enter the pool, else the whole sample is
//                     evaluated exactly (so is the sample of a query whose run
//                     meets more than kSMaxWin windows)
//   s_search_kernel   one wavefront per query (persistent grid, ~100 VGPRs,
//                     5 wavefronts per SIMD): the traversal from that pool,
//                     where the sample's ranks count as visited by their
//                     priority.
// Bucket order inside a bucket follows atomic arrival, so tiles differ from
// run to run; results do not, since every pool is the exact L nearest of the
// sample.

constexpr int kSQ = 16;          // queries per tile
constexpr int kSMaxChunks = 4;   // work items per tile at most
constexpr int kSChunkRows = 1024;  // rows per work item at least
constexpr int kSMaxWin = 8;      // windows per query at most (more: no tiles, an exact pass)
static_assert(kSMaxWin * kSMaxChunks <= 64, "a query's lists fit one wavefront");
constexpr int kSSub = 16;        // buckets per window for pieces that start at its start / inside it
constexpr int kSFull = 32;       // buckets per window for pieces that cover it (equivalent; spread
                                 // so that their atomic counters do not contend)
constexpr int kSPer = 2 * kSSub + kSFull;   // buckets per window
constexpr int kOffPer = 3;       // windows per thread of s_wscan_kernel (nwin <= 3072)
constexpr int kQSub = 64;        // counters per class of the traversal's query order
constexpr int kQLine = 32;       // their stride (one 128-byte line each: atomics on one line serialise)

struct SPlan {
    int32_t l, r;
    uint32_t T;      // threshold
    int32_t all;     // every rank of the range is an entry point
    int32_t lev;     // level whose list holds the sample
    int32_t a, b;    // run [a, b) of [l, r] in that list
    int32_t w0, nw;  // first window the run meets (in its level) and how many
    int32_t qpos;    // place among the queries of its class and counter (traversal order)
    int32_t pad[6];
    int32_t pos[kSMaxWin];    // per window: place within its bucket
    int32_t wchunks[kSMaxWin];  // per window: work items of the pair's tile (its chunk lists)
};
static_assert(sizeof(SPlan) == 128, "plan layout");

struct STile {
    int32_t pair[kSQ];   // query * kSMaxWin + window index (-1: empty slot)
    int32_t l[kSQ];
    int32_t r[kSQ];
    uint32_t T[kSQ];
    uint32_t allmask;
    int32_t lev;      // level of the tile's window (all its pairs lie in that window)
    int32_t ua, ub;   // span of the slots' pieces of the window, positions in the level's list
    int32_t nq;       // 0: unused tile
    int32_t nch;      // its work items (chunks of its span)
    int32_t pad[2];
};

struct SParams {
    DevIndex ix;
    SearchLaunch a;
    SPlan* plan;
    uint32_t* hist;     // [nbins] pairs per bucket
    uint32_t* bstart;   // [nbins] first place of each bucket within its window
    uint32_t* wstart;   // [nwin] first place of each window
    uint32_t* meta;     // [0] places used in `order`, [1] tiles, [2] query counter
    uint32_t* qhist;    // [2 kQSub] queries per (class, counter) at stride kQLine, then [2 kQSub]
                        // their first places
    int32_t* qorder;    // [nq] the traversal's query order: queries whose sample is a strict
                        // subset of their range, then the others (covered or empty ranges)
    int32_t* order;     // [norder] pairs (query * kSMaxWin + window index) by bucket,
                        // each window's places padded to a multiple of 16 with -1
    STile* tiles;       // [tmax]
    int64_t tmax;
    int nbins;          // nwin * kSPer
    int nwin;           // windows of all levels
    int win_log2;       // W = 2^win_log2 positions per window
    int nchunk;         // work items per tile at most (<= kSMaxChunks): the lists' stride per pair
    int nbase;          // work items of a tile of the scan's first round at most
    int chunk_log2;     // such a tile's span is split into chunks of at least 2^chunk_log2 = W / nbase rows
    int scan_slots;     // scan wavefronts the device holds at once
    int32_t winbase[34];  // first window of level j; winbase[nlev + 1] = nwin
    int kkeep;
    // candidate lists, one per (pair, chunk of the pair's tile): list
    // (query * kSMaxWin + window index) * nchunk + chunk
    float* pv;          // [nq * kSMaxWin * nchunk][kkeep] approximate distances
    int32_t* pr;        // [nq * kSMaxWin * nchunk][kkeep] ranks
    float* pthr;        // [nq * kSMaxWin * nchunk] threshold of a full list, else +inf
    int32_t* pfill;     // [nq * kSMaxWin * nchunk] entries kept
    int32_t* pcnt;      // [nq * kSMaxWin * nchunk] sample rows seen
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

// work items of a tile whose span is `span` rows: chunks of at least
// 2^chunk_log2 rows, at most nchunk
__host__ __device__ __forceinline__ int tile_chunks(int64_t span, int nchunk, int chunk_log2) {
    const int64_t c = (span + ((int64_t)1 << chunk_log2) - 1) >> chunk_log2;
    return c < 1 ? 1 : (c < nchunk ? (int)c : nchunk);
}

// bucket of window wi of query q's run: its window, then the kind of piece
// (pieces that start at the window's start and end inside it, by where they
// end; pieces that cover the window; pieces that start inside it, by where
// they start), so that the pieces of a tile's 16 places lie close
__device__ __forceinline__ int pair_bin(const SParams& P, int64_t q, int lev, int32_t a, int32_t b, int32_t w0,
                                        int wi) {
    const int64_t ws = (int64_t)(w0 + wi) << P.win_log2;
    const int64_t we = ws + ((int64_t)1 << P.win_log2);
    const int64_t sa = a > ws ? a : ws;
    const int64_t sb = b < we ? b : we;
    int sub;
    if (sa > ws) sub = kSSub + kSFull + (int)(((sa - ws) * kSSub) >> P.win_log2);
    else if (sb < we) sub = (int)(((sb - ws - 1) * kSSub) >> P.win_log2);
    else sub = kSSub + (int)(q % kSFull);
    return (P.winbase[lev] + w0 + wi) * kSPer + sub;
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
