// Exhaustive filtered k-NN (Def. 2 of the paper) on gfx950, used as ground
// truth for the approximate search.
//
//   1. Host: each query's rank interval [l, r] (Sec 4) from the index's host
//      copy of the sorted attributes; queries are grouped into tiles of 16
//      with the same octave of range size, ordered by l, so a tile's rows are
//      the union of 16 overlapping intervals.  Each tile's union is cut into
//      row chunks; (tile, chunk) is a work item.
//   2. bf_scan_kernel, one wavefront per work item: the dot products of the
//      tile's 16 queries with 16-row blocks of X run on the fp32 matrix cores
//      (v_mfma_f32_16x16x4_f32, K = 4 per instruction, query operand resident
//      in VGPRs, the next block's rows loaded while the current one is
//      multiplied); the approximate squared distance |q|^2 + |x|^2 - 2 q.x
//      masks rows outside each query's own interval; per query the wavefront
//      keeps the K' smallest approximate distances of its chunk (K' = 2k
//      rounded up to 64, at most 256) and writes them out with its threshold.
//   3. bf_merge_kernel, one wavefront per query: the K' smallest over the
//      tile's chunks, re-ranked with the exact canonical distance (double
//      accumulation, rounded once to float); the k smallest (distance, rank)
//      are the result.  Every row not re-ranked has an approximate distance at
//      or above some kept list's threshold; if the smallest such threshold
//      minus the approximation bound exceeds the k-th exact distance, the
//      result is certified exact (reported per query).
//   4. Queries the margin test leaves uncertified (near-tied distances that
//      the fp32 approximation cannot separate, e.g. vectors with large norms
//      close to each other) are recomputed exhaustively: every rank of the
//      interval with the exact canonical distance (launch_exact_ranges), so
//      every returned row is the exact filtered k-NN.
//
// The approximation bound: with unit roundoff u = 2^-24, fp32 |q|^2 and |x|^2
// (d terms each), the fp32 dot product (d products) and the final two
// operations err by at most (2d + 4) u (|q|^2 + |x|^2); the kernel uses twice
// that with |x|^2 replaced by the largest squared norm in the index.
//
// The host step reads the query ranges back, so this entry point synchronises
// `stream`; it is a ground-truth tool, not the search path.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <vector>

#include "ws_pool.h"
#include "frog_internal.h"
#include "wave_topk.h"

namespace frog {
namespace {

using namespace topk;

constexpr int kQT = 16;       // queries per tile (one MFMA row block)
constexpr int kWaves = 1;     // wavefronts per workgroup: one, so that a finished work item releases its LDS at once
constexpr int kThreads = 64 * kWaves;

typedef float floatx4 __attribute__((ext_vector_type(4)));

struct Tile {
    int32_t q[kQT];   // query index, -1 = unused
    int32_t l[kQT];
    int32_t r[kQT];
    int32_t ul, ur;   // union of the intervals
    int32_t ib, ie;   // its work items
};

struct Item {
    int32_t tile, rb, re;   // rows [rb, re] of the tile's union
};

__host__ __device__ constexpr size_t scan_lds_per_wave(int kkeep) {
    return (size_t)kQT * kkeep * 8 + kQT * 4 + kQT * 16;
}
__host__ __device__ constexpr size_t merge_lds_per_wave(int kkeep) { return (size_t)kkeep * 8 + 16; }

struct BFParams {
    const float* X;       // [n][dp]
    const int32_t* perm;
    int64_t n;
    int d, dp;
    const float* Q;       // [nq][d]
    const Tile* tiles;
    const Item* items;
    int64_t ntiles, nitems;
    int kkeep;            // approximate candidates kept per query and chunk
    int k;
    float maxnorm;        // largest |x|^2 in the index
    float* pv;            // [nitems][16][kkeep] approximate distances
    int32_t* pr;          // [nitems][16][kkeep] rows
    float* pthr;          // [nitems][16] threshold of a full list, else +inf
    int32_t* pfill;       // [nitems][16] entries kept
    int32_t* ids;
    float* dists;
    int32_t* cert;
};

__device__ __forceinline__ int lane_id() { return __lane_id(); }

__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Stage 2.  KT = dp/16 float4 chunks of the query operand kept in registers
// (d <= 128); KT = 0 reloads the operand from global memory for each block.
template <int KT>
__global__ __launch_bounds__(kThreads) void bf_scan_kernel(BFParams P) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int lane = lane_id();
    const int wave = threadIdx.x >> 6;
    const int64_t item = (int64_t)blockIdx.x * kWaves + wave;
    if (item >= P.nitems) return;   // no workgroup barrier follows
    const Item it = P.items[item];
    const Tile& T = P.tiles[it.tile];
    const int dp = P.dp, dp4 = dp >> 2, d = P.d;
    const int kkeep = P.kkeep;
    // per-wave LDS: lists [16][kkeep] (value, row), |q|^2 [16], list state [16][4]
    char* wb = smem + (size_t)wave * scan_lds_per_wave(kkeep);
    float* lv = reinterpret_cast<float*>(wb);
    int32_t* lr = reinterpret_cast<int32_t*>(lv + kQT * kkeep);
    float* qnl = reinterpret_cast<float*>(lr + kQT * kkeep);
    int32_t* lst = reinterpret_cast<int32_t*>(qnl + kQT);

    // MFMA operand mapping (16x16x4 f32): A[i][kk] in lane i + 16 kk, B[kk][j]
    // in lane j + 16 kk, D[4 (lane/16) + e][lane % 16] in element e.  The K
    // loop walks float4 chunks: lane group kk takes dims 16t + 4kk + {0..3}.
    const int ii = lane & 15;
    const int kk = lane >> 4;
    const int qrow = T.q[ii];
    const float* Qr = P.Q + (int64_t)(qrow >= 0 ? qrow : 0) * d;
    auto qchunk = [&](int t) -> float4 {
        const int b = 16 * t + 4 * kk;
        float4 v;
        v.x = (qrow >= 0 && b < d) ? Qr[b] : 0.f;
        v.y = (qrow >= 0 && b + 1 < d) ? Qr[b + 1] : 0.f;
        v.z = (qrow >= 0 && b + 2 < d) ? Qr[b + 2] : 0.f;
        v.w = (qrow >= 0 && b + 3 < d) ? Qr[b + 3] : 0.f;
        return v;
    };
    float4 qa[KT > 0 ? KT : 1];
    float qs = 0.f;
    for (int t = 0; t < dp / 16; ++t) {
        const float4 v = qchunk(t);
        if constexpr (KT > 0) {
#pragma unroll
            for (int u = 0; u < KT; ++u)
                if (u == t) qa[u] = v;
        }
        qs += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
    }
    qs += __shfl_xor(qs, 16);
    qs += __shfl_xor(qs, 32);
    if (kk == 0) {
        qnl[ii] = qs;
        lst[4 * ii + 0] = 0;
        lst[4 * ii + 1] = 0x7f800000;
        lst[4 * ii + 2] = 0;
    }
    wave_sync();
    float qn[4];
    int ql[4], qr[4];
    bool qv[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        qn[e] = qnl[4 * kk + e];
        ql[e] = T.l[4 * kk + e];
        qr[e] = T.r[4 * kk + e];
        qv[e] = T.q[4 * kk + e] >= 0;
    }
    const float4* X4 = reinterpret_cast<const float4*>(P.X);
    const int nblk = (it.re - it.rb + 16) / 16;
    float4 xa[KT > 0 ? KT : 1], xb[KT > 0 ? KT : 1];
    auto load_block = [&](int blk, float4 (&x)[KT > 0 ? KT : 1]) {
        if constexpr (KT > 0) {
            const int row = it.rb + blk * 16 + ii;
            const int rowc = row <= it.re ? row : it.re;
#pragma unroll
            for (int t = 0; t < KT; ++t) x[t] = X4[(int64_t)rowc * dp4 + 4 * t + kk];
        }
    };
    // one block's products and candidates; x holds its rows (d <= 128)
    auto process = [&](int blk, const float4 (&x)[KT > 0 ? KT : 1]) {
        const int row = it.rb + blk * 16 + ii;
        const int rowc = row <= it.re ? row : it.re;
        floatx4 acc = {0.f, 0.f, 0.f, 0.f};
        float xn = 0.f;
        if constexpr (KT > 0) {
#pragma unroll
            for (int t = 0; t < KT; ++t) {
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(qa[t].x, x[t].x, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(qa[t].y, x[t].y, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(qa[t].z, x[t].z, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(qa[t].w, x[t].w, acc, 0, 0, 0);
                xn += x[t].x * x[t].x + x[t].y * x[t].y + x[t].z * x[t].z + x[t].w * x[t].w;
            }
        } else {
            for (int t = 0; t < dp / 16; ++t) {
                const float4 xv = X4[(int64_t)rowc * dp4 + 4 * t + kk];
                const float4 q = qchunk(t);
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(q.x, xv.x, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(q.y, xv.y, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(q.z, xv.z, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(q.w, xv.w, acc, 0, 0, 0);
                xn += xv.x * xv.x + xv.y * xv.y + xv.z * xv.z + xv.w * xv.w;
            }
        }
        xn += __shfl_xor(xn, 16);
        xn += __shfl_xor(xn, 32);
        // lane holds D[4kk + e][ii]: query 4kk + e, row rb + blk*16 + ii
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float ap = qn[e] + xn - 2.f * acc[e];
            const bool cand = qv[e] && row <= it.re && row >= ql[e] && row <= qr[e] &&
                              ap < list_threshold(lst + 4 * (4 * kk + e));
            uint64_t m = __ballot(cand);
            while (m) {
                const int g = __builtin_ctzll(m) >> 4;
                const uint64_t gm = m & (0xFFFFull << (16 * g));
                m &= ~gm;
                const int qi = 4 * g + e;
                offer(TopList{lv + qi * kkeep, lr + qi * kkeep, lst + 4 * qi}, kkeep, gm, ap, rowc);
            }
        }
    };
    // two row buffers in turn: the next block's loads are issued on every
    // step (past the last block they read it again) before the current
    // block is used, so its wait leaves them in flight; a conditional load,
    // or a copy between the buffers, would make the wait drain them
    load_block(0, xa);
    for (int blk = 0; blk < nblk; blk += 2) {
        load_block(blk + 1 < nblk ? blk + 1 : nblk - 1, xb);
        process(blk, xa);
        if (blk + 1 >= nblk) break;
        load_block(blk + 2 < nblk ? blk + 2 : nblk - 1, xa);
        process(blk + 1, xb);
    }
    // write the chunk's lists
    const int64_t base = item * kQT;
    for (int i = 0; i < kQT; ++i) {
        const int fi = lst[4 * i];
        for (int j = lane; j < kkeep; j += 64) {
            P.pv[(base + i) * kkeep + j] = j < fi ? lv[i * kkeep + j] : __int_as_float(0x7f800000);
            P.pr[(base + i) * kkeep + j] = j < fi ? lr[i * kkeep + j] : -1;
        }
        if (lane == 0) {
            P.pthr[base + i] = fi >= kkeep ? list_threshold(lst + 4 * i) : __int_as_float(0x7f800000);
            P.pfill[base + i] = fi;
        }
    }
}

// Stage 3: one wavefront per (tile, query slot).
__global__ __launch_bounds__(kThreads) void bf_merge_kernel(BFParams P) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int lane = lane_id();
    const int wave = threadIdx.x >> 6;
    const int64_t gw = (int64_t)blockIdx.x * kWaves + wave;
    if (gw >= P.ntiles * kQT) return;
    const Tile& T = P.tiles[gw / kQT];
    const int qi = (int)(gw % kQT);
    const int q = T.q[qi];
    if (q < 0) return;
    const int kkeep = P.kkeep, d = P.d, dp = P.dp;
    char* wb = smem + (size_t)wave * merge_lds_per_wave(kkeep);
    const TopList Lst{reinterpret_cast<float*>(wb), reinterpret_cast<int32_t*>(wb) + kkeep,
                      reinterpret_cast<int32_t*>(wb) + 2 * kkeep};
    if (lane == 0) {
        Lst.st[0] = 0;
        Lst.st[1] = 0x7f800000;
        Lst.st[2] = 0;
    }
    wave_sync();
    float texcl = __int_as_float(0x7f800000);   // every row not kept is at or above this
    bool dropped = false;
    for (int item = T.ib; item < T.ie; ++item) {
        const int64_t base = (int64_t)item * kQT + qi;
        texcl = fminf(texcl, P.pthr[base]);
        const int fi = P.pfill[base];
        for (int j0 = 0; j0 < fi; j0 += 64) {
            const int j = j0 + lane;
            const bool have = j < fi;
            const float a = have ? P.pv[base * kkeep + j] : 0.f;
            const int32_t rw = have ? P.pr[base * kkeep + j] : -1;
            const int f = Lst.st[0];
            const uint64_t gm = __ballot(have && (f < kkeep || a < list_threshold(Lst.st)));
            const uint64_t all = __ballot(have);
            if (gm != all) dropped = true;   // candidates at or above a full list's threshold
            if (gm) dropped |= offer(Lst, kkeep, gm, a, rw);
        }
    }
    if (dropped) texcl = fminf(texcl, list_threshold(Lst.st));
    const int f = Lst.st[0];
    // exact re-rank
    const float* Qq = P.Q + (int64_t)q * d;
    uint64_t key[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        key[j] = ~0ull;
        const int slot = lane + 64 * j;
        if (slot < kkeep && slot < f) {
            const int rw = Lst.r[slot];
            const float* xr = P.X + (int64_t)rw * dp;
            double sacc = 0.0;
            for (int c = 0; c < d; ++c) {
                const double t = (double)Qq[c] - (double)xr[c];
                sacc += t * t;
            }
            key[j] = ((uint64_t)__float_as_uint((float)sacc) << 32) | (uint32_t)rw;
        }
    }
    float kth = __int_as_float(0x7f800000);
    int found = 0;
    for (int j = 0; j < P.k; ++j) {
        uint64_t best = key[0];
#pragma unroll
        for (int u = 1; u < 4; ++u) best = key[u] < best ? key[u] : best;
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) {
            const uint64_t other = __shfl_xor(best, o);
            best = other < best ? other : best;
        }
        int32_t oid = -1;
        float od = __int_as_float(0x7f800000);
        if (best != ~0ull) {
            oid = P.perm[(uint32_t)best];
            od = __uint_as_float((uint32_t)(best >> 32));
            kth = od;
            found = j + 1;
#pragma unroll
            for (int u = 0; u < 4; ++u)
                if (key[u] == best) key[u] = ~0ull;
        }
        if (lane == 0) {
            P.ids[(int64_t)q * P.k + j] = oid;
            P.dists[(int64_t)q * P.k + j] = od;
        }
    }
    if (P.cert && lane == 0) {
        double qn = 0.0;
        for (int c = 0; c < d; ++c) qn += (double)Qq[c] * Qq[c];
        const double eps = 2.0 * (2.0 * d + 4.0) * 5.9604644775390625e-08 * (qn + (double)P.maxnorm);
        bool ok;
        if (isinf(texcl)) ok = true;                       // no row was dropped
        else ok = found == P.k && (double)texcl - eps > (double)kth;
        P.cert[q] = ok ? 1 : 0;
    }
}

__global__ void bf_pad_kernel(int64_t nq, int k, const uint8_t* empty, int32_t* ids, float* dists, int32_t* cert) {
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= nq || !empty[q]) return;
    for (int j = 0; j < k; ++j) {
        ids[q * k + j] = -1;
        dists[q * k + j] = __int_as_float(0x7f800000);
    }
    if (cert) cert[q] = 1;
}

}  // namespace

int launch_bruteforce(const frog_index* ix, const float* Q, int64_t nq, const double* lo,
                      const double* hi, int k, int32_t* ids, float* dists, int32_t* cert, void* stream_v) {
    hipStream_t stream = (hipStream_t)stream_v;
    std::vector<double> hlo((size_t)nq), hhi((size_t)nq);
    hipError_t e = hipMemcpyAsync(hlo.data(), lo, sizeof(double) * nq, hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess) e = hipMemcpyAsync(hhi.data(), hi, sizeof(double) * nq, hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return fail(FROG_EHIP, "bruteforce: reading ranges: %s", hipGetErrorString(e));
    const int64_t n = ix->n;
    const double* a = ix->attr.data();
    std::vector<int32_t> L((size_t)nq), R((size_t)nq);
    std::vector<uint8_t> empty((size_t)nq, 0);
    std::vector<int32_t> order;
    order.reserve((size_t)nq);
    for (int64_t q = 0; q < nq; ++q) {
        if (std::isnan(hlo[q]) || std::isnan(hhi[q])) { empty[q] = 1; continue; }
        const int64_t l = std::lower_bound(a, a + n, hlo[q]) - a;
        const int64_t r = (std::upper_bound(a, a + n, hhi[q]) - a) - 1;
        if (l > r) { empty[q] = 1; continue; }
        L[q] = (int32_t)l;
        R[q] = (int32_t)r;
        order.push_back((int32_t)q);
    }
    auto band = [&](int32_t q) { return 63 - __builtin_clzll((uint64_t)(R[q] - L[q] + 1)); };
    std::sort(order.begin(), order.end(), [&](int32_t x, int32_t y) {
        const int bx = band(x), by = band(y);
        if (bx != by) return bx > by;
        if (L[x] != L[y]) return L[x] < L[y];
        return x < y;
    });
    std::vector<Tile> tiles;
    int64_t total_rows = 0;
    for (size_t i = 0; i < order.size();) {
        Tile t;
        const int b = band(order[i]);
        int c = 0;
        t.ul = INT32_MAX;
        t.ur = -1;
        while (c < kQT && i < order.size() && band(order[i]) == b) {
            const int32_t q = order[i++];
            t.q[c] = q;
            t.l[c] = L[q];
            t.r[c] = R[q];
            t.ul = std::min(t.ul, L[q]);
            t.ur = std::max(t.ur, R[q]);
            ++c;
        }
        for (; c < kQT; ++c) { t.q[c] = -1; t.l[c] = 0; t.r[c] = -1; }
        total_rows += (int64_t)t.ur - t.ul + 1;
        tiles.push_back(t);
    }
    // work items: about 8192 row chunks in all (a multiple of 16 rows each)
    int64_t chunk = total_rows / 8192 + 1;
    chunk = std::max<int64_t>(1024, std::min<int64_t>(1 << 18, (chunk + 15) / 16 * 16));
    std::vector<Item> items;
    for (size_t t = 0; t < tiles.size(); ++t) {
        tiles[t].ib = (int32_t)items.size();
        for (int64_t rb = tiles[t].ul; rb <= tiles[t].ur; rb += chunk) {
            const int64_t re = std::min<int64_t>(tiles[t].ur, rb + chunk - 1);
            items.push_back(Item{(int32_t)t, (int32_t)rb, (int32_t)re});
        }
        tiles[t].ie = (int32_t)items.size();
    }
    const float maxnorm = ix->maxnorm;
    int kkeep = 2 * k < 64 ? 64 : (2 * k + 63) / 64 * 64;
    if (kkeep > 256) kkeep = 256;
    auto align = [](size_t x) { return (x + 255) / 256 * 256; };
    const size_t tbytes = align(tiles.size() * sizeof(Tile));
    const size_t ibytes = align(items.size() * sizeof(Item));
    const size_t ebytes = align((size_t)nq);
    const size_t lbytes = align(items.size() * kQT * (size_t)kkeep * 4);
    const size_t sbytes = align(items.size() * kQT * 4);
    const size_t cbytes = align((size_t)nq * 4);
    const size_t ws_bytes = tbytes + ibytes + ebytes + 2 * lbytes + 2 * sbytes + cbytes + 256;
    void* ws = nullptr;
    e = ws_alloc(&ws, ws_bytes, stream);
    if (e != hipSuccess) return fail(FROG_ENOMEM, "bruteforce workspace: %s", hipGetErrorString(e));
    char* base = reinterpret_cast<char*>(ws);
    Tile* dT = reinterpret_cast<Tile*>(base);
    Item* dI = reinterpret_cast<Item*>(base + tbytes);
    uint8_t* dE = reinterpret_cast<uint8_t*>(base + tbytes + ibytes);
    char* lists = base + tbytes + ibytes + ebytes;
    // certification flags: the caller's array, else one in the workspace
    int32_t* dcert = cert ? cert : reinterpret_cast<int32_t*>(lists + 2 * lbytes + 2 * sbytes);
    if (!tiles.empty()) e = hipMemcpyAsync(dT, tiles.data(), tiles.size() * sizeof(Tile), hipMemcpyHostToDevice, stream);
    if (e == hipSuccess && !items.empty())
        e = hipMemcpyAsync(dI, items.data(), items.size() * sizeof(Item), hipMemcpyHostToDevice, stream);
    if (e == hipSuccess) e = hipMemcpyAsync(dE, empty.data(), (size_t)nq, hipMemcpyHostToDevice, stream);
    if (e != hipSuccess) {
        (void)ws_free(ws, stream);
        return fail(FROG_EHIP, "bruteforce upload: %s", hipGetErrorString(e));
    }
    hipLaunchKernelGGL(bf_pad_kernel, dim3((unsigned)((nq + 255) / 256)), dim3(256), 0, stream, nq, k, dE, ids, dists, dcert);
    if (!tiles.empty()) {
        BFParams P{};
        P.X = ix->dX;
        P.perm = ix->dperm;
        P.n = n;
        P.d = ix->d;
        P.dp = ix->dp;
        P.Q = Q;
        P.tiles = dT;
        P.items = dI;
        P.ntiles = (int64_t)tiles.size();
        P.nitems = (int64_t)items.size();
        P.kkeep = kkeep;
        P.k = k;
        P.maxnorm = maxnorm;
        P.pv = reinterpret_cast<float*>(lists);
        P.pr = reinterpret_cast<int32_t*>(lists + lbytes);
        P.pthr = reinterpret_cast<float*>(lists + 2 * lbytes);
        P.pfill = reinterpret_cast<int32_t*>(lists + 2 * lbytes + sbytes);
        P.ids = ids;
        P.dists = dists;
        P.cert = dcert;
        const int smem_scan = (int)(kWaves * scan_lds_per_wave(kkeep));
        void (*scan)(BFParams) = bf_scan_kernel<0>;
        switch (ix->dp) {
            case 32: scan = bf_scan_kernel<2>; break;
            case 64: scan = bf_scan_kernel<4>; break;
            case 96: scan = bf_scan_kernel<6>; break;
            case 128: scan = bf_scan_kernel<8>; break;
            default: break;
        }
        if (smem_scan > 64 * 1024)
            (void)hipFuncSetAttribute((const void*)scan, hipFuncAttributeMaxDynamicSharedMemorySize, smem_scan);
        hipLaunchKernelGGL(scan, dim3((unsigned)((items.size() + kWaves - 1) / kWaves)), dim3(kThreads), smem_scan,
                           stream, P);
        const int smem_merge = (int)(kWaves * merge_lds_per_wave(kkeep));
        hipLaunchKernelGGL(bf_merge_kernel, dim3((unsigned)((tiles.size() * kQT + kWaves - 1) / kWaves)), dim3(kThreads),
                           smem_merge, stream, P);
    }
    e = hipGetLastError();
    // which queries the margin test certified
    std::vector<int32_t> hc((size_t)nq, 1);
    if (e == hipSuccess && !tiles.empty())
        e = hipMemcpyAsync(hc.data(), dcert, (size_t)nq * 4, hipMemcpyDeviceToHost, stream);
    (void)ws_free(ws, stream);
    // keep the host-side arrays alive until the copies have run
    const hipError_t es = hipStreamSynchronize(stream);
    if (e != hipSuccess || es != hipSuccess)
        return fail(FROG_EHIP, "bruteforce launch: %s", hipGetErrorString(e != hipSuccess ? e : es));
    // the rest: every rank of the interval, exactly
    std::vector<int32_t> fq, flr;
    for (int64_t q = 0; q < nq; ++q)
        if (!empty[(size_t)q] && hc[(size_t)q] == 0) {
            fq.push_back((int32_t)q);
            flr.push_back(L[(size_t)q]);
            flr.push_back(R[(size_t)q]);
        }
    if (fq.empty()) return FROG_OK;
    const DevIndex dix{ix->dX, ix->dXh, ix->dENC, ix->dattr, ix->dperm, ix->n, ix->d, ix->dp, ix->H, ix->m,
                       ix->storage};
    return launch_exact_ranges(dix, Q, fq.data(), flr.data(), (int64_t)fq.size(), k, ids, dists, cert, stream);
}

}  // namespace frog
