// FROGSearch, entry mode 0 (one stratified sample per query): the
// cooperative search kernel and its launch, the rank-bound kernel, and the
// row gather the shared sample's preparation uses.  The search's design is
// described in search_common.h.

#include "ws_pool.h"
#include "search_common.h"
#include "search_shared.h"

namespace frog {

// Workspace of frog_search_noalloc: a fixed array of device memory, one per
// GPU the library runs on, held until the process ends.  In host code its
// name is only a stand-in: the device address comes from
// hipGetSymbolAddress, taken once per device (scratch_area).
constexpr size_t kScratchBytes = (size_t)256 << 20;
static __device__ __align__(256) char scratch[kScratchBytes];

namespace {

// The whole search in one persistent kernel.  The four wavefronts of a
// workgroup share queries: a 64-bit LDS word holds the workgroup's open query
// and the next unclaimed entry chunk (claimed by compare-and-swap); a wave
// that finds the open query exhausted opens the next one from the global
// counter.  A wave evaluates one chunk (512 entry points) into a pool, writes
// it to global memory and counts the query's finished chunks with a
// workgroup-scope atomic; the wave that finishes the last chunk merges the
// chunk pools (the L nearest entry points) and runs the query's traversal,
// while its siblings go on with the next query's chunks -- so the traversal's
// dependent round trips overlap other queries' bandwidth-bound entry work.
// Only the waves of one workgroup ever touch a query, so workgroup-scope
// release/acquire orders the chunk pools (no cache maintenance on gfx950).
constexpr uint32_t kCtlNone = 0xFFFFFFFFu;       // no open query
constexpr uint32_t kCtlOpening = 0xFFFFFFFEu;    // a wave is opening one
constexpr uint32_t kCtlExhausted = 0xFFFFFFFDu;  // no queries left

__device__ __forceinline__ uint64_t ctl_word(uint32_t q, uint32_t next, uint32_t nch) {
    return ((uint64_t)q << 32) | ((uint64_t)next << 16) | nch;
}

template <int C, int LP, typename XT = float, bool LEAN = false>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(FROG_WAVES_PER_EU)))
void coop_kernel(KParams P) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const DevIndex& ix = P.ix;
    const SearchLaunch& A = P.a;
    const int lane = lane_id();
    uint64_t* ctl = reinterpret_cast<uint64_t*>(smem + (size_t)kWavesPerBlock * P.lds_per_wave);
    if (threadIdx.x == 0) *ctl = ctl_word(kCtlNone, 0, 0);
    __syncthreads();
    WaveLds<LP> W(smem, P.lds_per_wave, A.hash_log2);
    Visited vis;
    vis.tab = W.tab;
    vis.shift = 32 - A.hash_log2;
    const int64_t gwave = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    vis.bits = A.hash_log2 > 0 ? nullptr : P.gvis + gwave * P.gvis_words;
    const uint32_t slots = 64u * LP;

    for (;;) {
        // ---- claim an entry chunk of the workgroup's open query
        uint32_t cq = 0, cc = 0, cn = 0;
        bool done = false;
        for (;;) {
            uint64_t w = 0;
            int state = 0;   // 0 retry, 1 claimed, 2 exhausted
            if (lane == 0) {
                w = __hip_atomic_load(ctl, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
                const uint32_t q = (uint32_t)(w >> 32), nx = (uint32_t)(w >> 16) & 0xFFFFu, nc = (uint32_t)w & 0xFFFFu;
                if (q == kCtlExhausted) {
                    state = 2;
                } else if (q == kCtlOpening) {
                    __builtin_amdgcn_s_sleep(2);
                } else if (q == kCtlNone || nx >= nc) {
                    uint64_t expect = w;
                    if (__hip_atomic_compare_exchange_strong(ctl, &expect, ctl_word(kCtlOpening, 0, 0), __ATOMIC_RELAXED,
                                                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP)) {
                        // open the next non-empty query
                        uint64_t nw = ctl_word(kCtlExhausted, 0, 0);
                        for (;;) {
                            const uint32_t g = atomicAdd(P.counter, 1u);
                            if ((int64_t)g >= A.nq) break;
                            const int64_t l = P.lr[2 * (int64_t)g], r = P.lr[2 * (int64_t)g + 1];
                            const int64_t cnt = r - l + 1;
                            if (cnt <= 0) {
                                // empty range: padding and zero statistics
                                for (int j = 0; j < A.k; ++j) {
                                    A.ids[(int64_t)g * A.k + j] = -1;
                                    A.dists[(int64_t)g * A.k + j] = __int_as_float(0x7f800000);
                                }
                                if (A.stats)
                                    for (int j = 0; j < FROG_STAT_N; ++j) A.stats[(int64_t)g * FROG_STAT_N + j] = 0;
                                continue;
                            }
                            int64_t E = A.epn;
                            if (A.epn_frac > 0.0) {
                                double want = ceil(A.epn_frac * (double)cnt);
                                if (want > (double)A.epn_max) want = (double)A.epn_max;
                                if (want > (double)E) E = (int64_t)want;
                            }
                            const int64_t ne = cnt <= E ? cnt : E;
                            nw = ctl_word(g, 0, (uint32_t)((ne + P.chunk - 1) / P.chunk));
                            break;
                        }
                        __hip_atomic_store(ctl, nw, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
                    }
                } else {
                    uint64_t expect = w;
                    if (__hip_atomic_compare_exchange_strong(ctl, &expect, w + ((uint64_t)1 << 16), __ATOMIC_RELAXED,
                                                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP)) {
                        state = 1;
                        cq = q;
                        cc = nx;
                        cn = nc;
                    }
                }
            }
            state = uniform(__shfl(state, 0));
            if (state == 2) { done = true; break; }
            if (state == 1) {
                cq = (uint32_t)uniform((int)__shfl((int)cq, 0));
                cc = (uint32_t)uniform((int)__shfl((int)cc, 0));
                cn = (uint32_t)uniform((int)__shfl((int)cn, 0));
                break;
            }
        }
        if (done) break;

        // ---- the chunk's entry points
        const int64_t qi = cq;
        const int ci = (int)cc, nch = (int)cn;
        QueryCtx<C, XT> Q;
        Q.load(ix, A, P.lr, qi);
        Q.load_vector(ix);
        Pool<LP> pool;
        const int64_t e0 = (int64_t)ci * P.chunk;
        const int64_t e1 = e0 + P.chunk < Q.ne ? e0 + P.chunk : Q.ne;
        entry_chunk<C, LP, XT>(ix, A, Q, e0, e1, pool, W);

        if (nch > 1) {
            uint64_t* mine = P.part + ((uint64_t)qi * P.cpq + ci) * slots;
#pragma unroll
            for (int s = 0; s < LP; ++s) mine[s * 64 + lane] = pool.key[s];
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
            uint32_t old = 0;
            if (lane == 0)
                old = __hip_atomic_fetch_add(P.done + qi, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            old = (uint32_t)uniform((int)__shfl((int)old, 0));
            if ((int)old != nch - 1) continue;
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
            // the L nearest entry points: merge the other chunks' pools
            for (int c0 = 0; c0 < nch; c0 += 8) {
                uint64_t keys[8][LP];
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const uint64_t* part = P.part + ((uint64_t)qi * P.cpq + c0 + i) * slots;
#pragma unroll
                    for (int s = 0; s < LP; ++s)
                        keys[i][s] = (c0 + i < nch && c0 + i != ci) ? part[s * 64 + lane] : kEmpty;
                }
#pragma unroll
                for (int i = 0; i < 8; ++i) {
#pragma unroll
                    for (int s = 0; s < LP; ++s) {
                        const int nk = __popcll(ballot(keys[i][s] != kEmpty));   // sorted: a prefix
                        if (nk > 0) merge<LP>(pool, keys[i][s], nk, A.L, W.st_key, W.st_flag);
                    }
                }
            }
        }
        traverse<C, LP, XT, LEAN>(P.ix, P.a, P.gvis_words, Q, pool, W, vis);
        if (A.stats && lane == 0) {
            A.stats[qi * FROG_STAT_N + FROG_STAT_SCANROWS] = 0;
            A.stats[qi * FROG_STAT_N + FROG_STAT_FALLBACK] = 0;
        }
    }
}

__global__ void rank_bounds_kernel(DevIndex ix, const double* lo, const double* hi, int64_t nq, int32_t* lr) {
    const int64_t q = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    if (q >= nq) return;
    int64_t l, r;
    rank_interval(ix, lo[q], hi[q], l, r);
    if (lane_id() == 0) {
        lr[2 * q] = (int32_t)l;
        lr[2 * q + 1] = (int32_t)r;
    }
}

__global__ void init_kernel(unsigned int* counter, unsigned int* done, int64_t nq) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i == 0) *counter = 0u;
    if (i < nq) done[i] = 0u;
}

using KernelFn = void (*)(KParams);

template <int C, typename XT, bool LEAN>
KernelFn pick_lp_l(int L) {
    if (L <= 64) return coop_kernel<C, 1, XT, LEAN>;
    if (L <= 128) return coop_kernel<C, 2, XT, LEAN>;
    return coop_kernel<C, 4, XT, LEAN>;
}

template <int C, typename XT = float>
KernelFn pick_lp(int L, bool lean) {
    return lean ? pick_lp_l<C, XT, true>(L) : pick_lp_l<C, XT, false>(L);
}

// fp16 rows come with dp = 64 or 128 (the upload checks it)
KernelFn pick_kernel(int dp, int L, int storage, bool lean) {
    if (storage == FROG_STORAGE_F16) return dp == 64 ? pick_lp<2, __half>(L, lean) : pick_lp<4, __half>(L, lean);
    if (storage == FROG_STORAGE_BF16) return dp == 64 ? pick_lp<2, bf16x>(L, lean) : pick_lp<4, bf16x>(L, lean);
    switch (dp) {
        case 32: return pick_lp<1>(L, lean);
        case 64: return pick_lp<2>(L, lean);
        case 96: return pick_lp<3>(L, lean);
        case 128: return pick_lp<4>(L, lean);
        default: return pick_lp<0>(L, lean);
    }
}

// one 16-byte piece per thread: piece c of row i of out is piece c of row
// ranks[i] of X (w pieces per row)
__global__ void gather_rows_kernel(const uint4* __restrict__ X, int w, const int32_t* __restrict__ ranks,
                                   int64_t count, uint4* __restrict__ out) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t row = i / w;
    if (row >= count) return;
    const int c = (int)(i % w);
    out[i] = X[(int64_t)ranks[row] * w + c];
}

}  // namespace

int launch_gather_rows(const void* X, int row_bytes, const int32_t* ranks, int64_t count, void* out,
                       void* stream_v) {
    hipStream_t stream = (hipStream_t)stream_v;
    if (row_bytes <= 0 || row_bytes % 16 != 0) return fail(FROG_EINVAL, "gather rows: row of %d bytes", row_bytes);
    const int w = row_bytes / 16;
    const int64_t total = count * w;
    hipLaunchKernelGGL(gather_rows_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, stream,
                       reinterpret_cast<const uint4*>(X), w, ranks, count, reinterpret_cast<uint4*>(out));
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(FROG_EHIP, "gather rows: %s", hipGetErrorString(e));
    return FROG_OK;
}

bool search_shape_supported(int dp, int m, int L) {
    return dp >= 32 && dp % 32 == 0 && m >= 1 && m <= 64 && L >= 1 && L <= 256;
}

int launch_search(const DevIndex& ix, const SearchLaunch& a, void* stream_v) {
    return launch_search_ws(ix, a, stream_v, nullptr, 0);
}

int launch_search_ws(const DevIndex& ix, const SearchLaunch& a, void* stream_v, void* wsv, size_t ws_cap) {
    hipStream_t stream = (hipStream_t)stream_v;
    if (a.entry_mode == 1) return launch_shared(ix, a, stream, wsv, ws_cap);
    const KernelFn fn = pick_kernel(ix.dp, a.L, ix.storage, lean_launch(a));
    const int lpw = lds_per_wave(a.L, a.hash_log2);
    const int smem = lpw * kWavesPerBlock + 16;
    if (smem > 160 * 1024) return fail(FROG_EUNSUPPORTED, "LDS per block %d too large", smem);
    if (smem > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void*)fn, hipFuncAttributeMaxDynamicSharedMemorySize, smem);
        if (e != hipSuccess) return fail(FROG_EHIP, "hipFuncSetAttribute: %s", hipGetErrorString(e));
    }
    // entry chunks: FROG_CHUNK entry points per work unit, at most 16 units per query
    const int64_t emax = a.epn_frac > 0.0 ? (a.epn_max > a.epn ? a.epn_max : a.epn) : a.epn;
    int64_t chunk = FROG_CHUNK;
    if ((emax + chunk - 1) / chunk > 16) chunk = ((emax + 15) / 16 + 15) / 16 * 16;
    const int cpq = (int)((emax + chunk - 1) / chunk);
    if (a.nq >= ((int64_t)1 << 31) - 1) return fail(FROG_EINVAL, "nq=%lld too large", (long long)a.nq);
    const int lp = lp_of(a.L);
    int blocks = max_blocks((const void*)fn, smem);
    const int64_t need = (a.nq * cpq + kWavesPerBlock - 1) / kWavesPerBlock;
    if (need < blocks) blocks = (int)need;
    KParams P{};
    P.ix = ix;
    P.a = a;
    P.lds_per_wave = lpw;
    P.cpq = cpq;
    P.chunk = (int)chunk;
    P.gvis_words = 0;
    auto align = [](size_t x) { return (x + 255) / 256 * 256; };
    const size_t off_lr = 256;
    const size_t off_done = off_lr + align((size_t)a.nq * 8);
    const size_t off_part = off_done + align((size_t)a.nq * 4);
    const size_t part_bytes = cpq > 1 ? (size_t)a.nq * cpq * 64 * lp * 8 : 0;
    const size_t off_gvis = off_part + align(part_bytes);
    size_t ws = off_gvis;
    if (a.hash_log2 == 0) {
        P.gvis_words = (ix.n + 31) / 32;
        // bound the bitmap footprint to ~2 GiB
        const int64_t cap = ((int64_t)2 << 30) / (P.gvis_words * 4 * kWavesPerBlock);
        if (cap < blocks) blocks = (int)(cap > 0 ? cap : 1);
        ws += (size_t)blocks * kWavesPerBlock * P.gvis_words * 4;
    }
    void* wsp = wsv;
    hipError_t e = hipSuccess;
    WsLease lease;
    if (wsv) {
        if (ws > ws_cap)
            return fail(FROG_EUNSUPPORTED,
                        "this call needs %zu bytes of workspace; the scratch array holds %zu (nq=%lld, L=%d, "
                        "entry_mode 0%s)", ws, ws_cap, (long long)a.nq, a.L,
                        a.hash_log2 == 0 ? ", exact visited set" : "");
    } else {
        e = lease.acquire(stream, ws, &wsp);
        if (e != hipSuccess)
            return fail(e == hipErrorOutOfMemory ? FROG_ENOMEM : FROG_EHIP, "workspace: %s", hipGetErrorString(e));
    }
    char* base = reinterpret_cast<char*>(wsp);
    P.counter = reinterpret_cast<unsigned int*>(base);
    int32_t* lr = reinterpret_cast<int32_t*>(base + off_lr);
    P.lr = lr;
    P.done = reinterpret_cast<unsigned int*>(base + off_done);
    P.part = reinterpret_cast<uint64_t*>(base + off_part);
    P.gvis = reinterpret_cast<uint32_t*>(base + off_gvis);
    hipLaunchKernelGGL(init_kernel, dim3((unsigned)((a.nq + 255) / 256)), dim3(256), 0, stream, P.counter, P.done, a.nq);
    const int64_t rb_blocks = (a.nq + kWavesPerBlock - 1) / kWavesPerBlock;
    hipLaunchKernelGGL(rank_bounds_kernel, dim3((unsigned)rb_blocks), dim3(kBlock), 0, stream, ix, a.lo, a.hi, a.nq, lr);
    hipEvent_t* ev = reinterpret_cast<hipEvent_t*>(a.events);
    if (ev) (void)hipEventRecord(ev[0], stream);
    hipLaunchKernelGGL(fn, dim3(blocks), dim3(kBlock), smem, stream, P);
    if (ev) {
        (void)hipEventRecord(ev[1], stream);
        (void)hipEventRecord(ev[2], stream);
    }
    e = hipGetLastError();
    lease.release();
    if (e != hipSuccess) return fail(FROG_EHIP, "search launch: %s", hipGetErrorString(e));
    return FROG_OK;
}

int scratch_area(void** ptr, size_t* bytes) {
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static void* addr[kMaxDevices] = {};
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
        return fail(FROG_EHIP, "scratch: no usable current device (%d)", dev);
    std::lock_guard<std::mutex> g(mu);
    if (!addr[dev]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(FROG_EHIP, "scratch: hipGetSymbolAddress: %s", hipGetErrorString(e));
        addr[dev] = p;
    }
    *ptr = addr[dev];
    *bytes = kScratchBytes;
    return FROG_OK;
}

int launch_rank_bounds(const DevIndex& ix, const double* lo, const double* hi, int64_t nq, int32_t* lr,
                       void* stream_v) {
    hipStream_t stream = (hipStream_t)stream_v;
    const int64_t blocks = (nq + kWavesPerBlock - 1) / kWavesPerBlock;
    hipLaunchKernelGGL(rank_bounds_kernel, dim3((unsigned)blocks), dim3(kBlock), 0, stream, ix, lo, hi, nq, lr);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(FROG_EHIP, "rank_bounds launch: %s", hipGetErrorString(e));
    return FROG_OK;
}

}  // namespace frog
