// Exhaustive filtered k-NN of selected queries with the exact canonical
// distance (the brute force's fallback for queries its margin test cannot
// certify).

#include "ws_pool.h"
#include "search_common.h"

namespace frog {
namespace {

// ------------------------------------------------------------------ exact ranges
//
// Exhaustive filtered k-NN (Def. 2) of selected queries: every rank of each
// query's interval gets the canonical distance (the traversal's gather and
// fp64 code), and the k smallest (distance, rank) are kept.  The brute force
// uses it for the queries its margin test could not certify.  Work items are
// runs of kExactRun ranks, one wavefront each, keeping their k nearest in a
// VGPR pool (merge<LP>); one wavefront per query then merges its items' pools.

constexpr int kExactRun = 4096;

struct XParams {
    DevIndex ix;
    const float* Q;
    const int32_t* fq;    // [nf] query indices
    const int32_t* flr;   // [nf][2] rank intervals (non-empty)
    const int64_t* fo;    // [nf + 1] first work item of each query
    int64_t nf, nitems;
    int k;
    uint64_t* part;       // [nitems][64 LP] each item's k nearest, sorted keys, kEmpty padded
    int32_t* ids;
    float* dists;
    int32_t* cert;        // set to 2 for every query done here
};

template <int C, int LP>
__global__ __launch_bounds__(kBlock) void exact_run_kernel(XParams P) {
    __shared__ __attribute__((aligned(16))) char smem[kWavesPerBlock * 64 * LP * 12];
    const int lane = lane_id();
    const int wave = threadIdx.x >> 6;
    const int64_t item = (int64_t)blockIdx.x * kWavesPerBlock + wave;
    if (item >= P.nitems) return;   // wave-uniform; no workgroup barrier follows
    uint64_t* st_key = reinterpret_cast<uint64_t*>(smem + (size_t)wave * 64 * LP * 12);
    uint32_t* st_flag = reinterpret_cast<uint32_t*>(st_key + 64 * LP);
    // the item's query: the last j with fo[j] <= item
    int64_t a = 0, b = P.nf - 1;
    while (a < b) {
        const int64_t mid = (a + b + 1) >> 1;
        if (P.fo[mid] <= item) a = mid;
        else b = mid - 1;
    }
    const int64_t j = a;
    const int64_t q = P.fq[j];
    const int64_t l = P.flr[2 * j], r = P.flr[2 * j + 1];
    const int64_t b0 = l + (item - P.fo[j]) * kExactRun;
    const int64_t b1 = b0 + kExactRun <= r + 1 ? b0 + kExactRun : r + 1;
    const DevIndex& ix = P.ix;
    const float* qrow = P.Q + q * ix.d;
    float4 qv[C > 0 ? C : 1];
    if constexpr (C > 0) {
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const int bd = chunk_dim<float>(lane & 7, c);
            qv[c].x = bd < ix.d ? qrow[bd] : 0.f;
            qv[c].y = bd + 1 < ix.d ? qrow[bd + 1] : 0.f;
            qv[c].z = bd + 2 < ix.d ? qrow[bd + 2] : 0.f;
            qv[c].w = bd + 3 < ix.d ? qrow[bd + 3] : 0.f;
        }
    }
    Pool<LP> pool;
#pragma unroll
    for (int s = 0; s < LP; ++s) { pool.key[s] = kEmpty; pool.flag[s] = 0u; }
    pool.np = 0;
    for (int64_t p0 = b0; p0 < b1; p0 += 64) {
        const int nb = (int)(b1 - p0 < 64 ? b1 - p0 : 64);
        const int32_t id = lane < nb ? (int32_t)(p0 + lane) : (int32_t)p0;
        float dd;
        if constexpr (C > 0) dd = eval_pipelined<C, float>(ix.X, ix.dp, qv, nb, id);
        else dd = eval_large(ix.X, ix.dp, qrow, ix.d, nb, id);
        merge<LP>(pool, lane < nb ? make_key(dd, id) : kEmpty, nb, P.k, st_key, st_flag);
    }
#pragma unroll
    for (int s = 0; s < LP; ++s) P.part[item * 64 * LP + s * 64 + lane] = pool.key[s];
}

template <int LP>
__global__ __launch_bounds__(kBlock) void exact_merge_kernel(XParams P) {
    __shared__ __attribute__((aligned(16))) char smem[kWavesPerBlock * 64 * LP * 12];
    const int lane = lane_id();
    const int wave = threadIdx.x >> 6;
    const int64_t j = (int64_t)blockIdx.x * kWavesPerBlock + wave;
    if (j >= P.nf) return;   // wave-uniform
    uint64_t* st_key = reinterpret_cast<uint64_t*>(smem + (size_t)wave * 64 * LP * 12);
    uint32_t* st_flag = reinterpret_cast<uint32_t*>(st_key + 64 * LP);
    Pool<LP> pool;
#pragma unroll
    for (int s = 0; s < LP; ++s) { pool.key[s] = kEmpty; pool.flag[s] = 0u; }
    pool.np = 0;
    for (int64_t it = P.fo[j]; it < P.fo[j + 1]; ++it) {
#pragma unroll
        for (int s = 0; s < LP; ++s) {
            const uint64_t key = P.part[it * 64 * LP + s * 64 + lane];
            const int nk = __popcll(ballot(key != kEmpty));   // sorted: a prefix
            if (nk > 0) merge<LP>(pool, key, nk, P.k, st_key, st_flag);
        }
    }
    const int64_t q = P.fq[j];
#pragma unroll
    for (int s = 0; s < LP; ++s) {
        const int p = s * 64 + lane;
        if (p < P.k) {
            const bool have = p < pool.np;
            P.ids[q * P.k + p] = have ? P.ix.perm[(uint32_t)pool.key[s]] : -1;
            P.dists[q * P.k + p] = have ? __uint_as_float((uint32_t)(pool.key[s] >> 32)) : __int_as_float(0x7f800000);
        }
    }
    if (P.cert && lane == 0) P.cert[q] = 2;
}

template <int LP>
void (*pick_exact_run(int dp))(XParams) {
    switch (dp) {
        case 32: return exact_run_kernel<1, LP>;
        case 64: return exact_run_kernel<2, LP>;
        case 96: return exact_run_kernel<3, LP>;
        case 128: return exact_run_kernel<4, LP>;
        default: return exact_run_kernel<0, LP>;
    }
}

}  // namespace

int launch_exact_ranges(const DevIndex& ix, const float* Q, const int32_t* hq, const int32_t* hlr, int64_t nf, int k,
                        int32_t* ids, float* dists, int32_t* cert, void* stream_v) {
    hipStream_t stream = (hipStream_t)stream_v;
    if (nf == 0) return FROG_OK;
    if (ix.storage != FROG_STORAGE_F32 || k < 1 || k > 256)
        return fail(FROG_EINVAL, "exact ranges: fp32 rows and 1 <= k <= 256");
    std::vector<int64_t> fo((size_t)nf + 1, 0);
    for (int64_t j = 0; j < nf; ++j) {
        const int64_t cnt = (int64_t)hlr[2 * j + 1] - hlr[2 * j] + 1;
        if (cnt < 1) return fail(FROG_EINVAL, "exact ranges: empty interval");
        fo[(size_t)j + 1] = fo[(size_t)j] + (cnt + kExactRun - 1) / kExactRun;
    }
    const int64_t nitems = fo[(size_t)nf];
    const int lp = lp_of(k);
    auto align = [](size_t x) { return (x + 255) / 256 * 256; };
    const size_t o_q = 0, o_lr = align((size_t)nf * 4), o_fo = o_lr + align((size_t)nf * 8);
    const size_t o_part = o_fo + align((size_t)(nf + 1) * 8);
    const size_t bytes = o_part + (size_t)nitems * 64 * lp * 8;
    void* ws = nullptr;
    hipError_t e = ws_alloc(&ws, bytes, stream);
    if (e != hipSuccess) return fail(FROG_ENOMEM, "exact ranges workspace: %s", hipGetErrorString(e));
    char* base = reinterpret_cast<char*>(ws);
    XParams P{};
    P.ix = ix;
    P.Q = Q;
    P.fq = reinterpret_cast<const int32_t*>(base + o_q);
    P.flr = reinterpret_cast<const int32_t*>(base + o_lr);
    P.fo = reinterpret_cast<const int64_t*>(base + o_fo);
    P.part = reinterpret_cast<uint64_t*>(base + o_part);
    P.nf = nf;
    P.nitems = nitems;
    P.k = k;
    P.ids = ids;
    P.dists = dists;
    P.cert = cert;
    e = hipMemcpyAsync(base + o_q, hq, (size_t)nf * 4, hipMemcpyHostToDevice, stream);
    if (e == hipSuccess) e = hipMemcpyAsync(base + o_lr, hlr, (size_t)nf * 8, hipMemcpyHostToDevice, stream);
    if (e == hipSuccess) e = hipMemcpyAsync(base + o_fo, fo.data(), (size_t)(nf + 1) * 8, hipMemcpyHostToDevice, stream);
    if (e == hipSuccess) {
        auto run = lp == 1 ? pick_exact_run<1>(ix.dp) : (lp == 2 ? pick_exact_run<2>(ix.dp) : pick_exact_run<4>(ix.dp));
        auto mrg = lp == 1 ? exact_merge_kernel<1> : (lp == 2 ? exact_merge_kernel<2> : exact_merge_kernel<4>);
        hipLaunchKernelGGL(run, dim3((unsigned)((nitems + kWavesPerBlock - 1) / kWavesPerBlock)), dim3(kBlock), 0,
                           stream, P);
        hipLaunchKernelGGL(mrg, dim3((unsigned)((nf + kWavesPerBlock - 1) / kWavesPerBlock)), dim3(kBlock), 0,
                           stream, P);
        e = hipGetLastError();
    }
    (void)ws_free(ws, stream);
    // the host arrays must outlive the copies
    const hipError_t e2 = hipStreamSynchronize(stream);
    if (e != hipSuccess || e2 != hipSuccess)
        return fail(FROG_EHIP, "exact ranges: %s", hipGetErrorString(e != hipSuccess ? e : e2));
    return FROG_OK;
}

}  // namespace frog
