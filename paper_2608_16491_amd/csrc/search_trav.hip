// FROGSearch, entry mode 1: the traversal from each query's pool.

#include "search_shared.h"

namespace frog {
namespace {

// Traversal: persistent, one wavefront per query, from the pool s_pool_kernel
// wrote.  Queries are taken in the planned order: those whose sample is a
// strict subset of their range first, then those whose range the sample
// covers (no candidate is new, the traversal is short) and the empty ones,
// which then fill the kernel's tail (the results do not depend on the order).
template <int C, int LP, typename XT = float, bool LEAN = false>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(FROG_SEARCH_WAVES_PER_EU)))
void s_search_kernel(SParams P) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const DevIndex& ix = P.ix;
    const SearchLaunch& A = P.a;
    const int lane = lane_id();
    const int wave = threadIdx.x >> 6;
    WaveLds<LP> W(smem, P.lds_search, A.hash_log2);
    Visited vis;
    vis.tab = W.tab;
    vis.shift = 32 - A.hash_log2;
    const int64_t gwave = (int64_t)blockIdx.x * kWavesPerBlock + wave;
    vis.bits = A.hash_log2 > 0 ? nullptr : P.gvis + gwave * P.gvis_words;
    for (;;) {
        uint32_t qq = 0;
        if (lane == 0) qq = atomicAdd(P.meta + 2, 1u);
        const int64_t idx = (int64_t)(uint32_t)uniform((int)__shfl((int)qq, 0));
        if (idx >= A.nq) break;
        const int64_t qi = uniform(P.qorder[idx]);
        const SPlan p = P.plan[qi];
        if (p.l > p.r) {
            for (int j = lane; j < A.k; j += 64) {
                A.ids[qi * A.k + j] = -1;
                A.dists[qi * A.k + j] = __int_as_float(0x7f800000);
            }
            if (A.stats && lane < FROG_STAT_N) A.stats[qi * FROG_STAT_N + lane] = 0;
            continue;
        }
        QueryCtx<C, XT> Q;
        Q.set(ix, A, qi, p.l, p.r);   // the plan's rank interval
        Q.load_vector(ix);
        Q.shared = true;
        Q.T = p.T;
        Q.pkey = A.lv.key;
        Q.ne = P.pne[qi];
        Pool<LP> pool;
        int np = 0;
#pragma unroll
        for (int s = 0; s < LP; ++s) {
            pool.key[s] = P.pools[qi * 64 * LP + s * 64 + lane];
            pool.flag[s] = 0u;
            np += __popcll(ballot(pool.key[s] != kEmpty));
        }
        pool.np = np;
        traverse<C, LP, XT, LEAN>(ix, A, P.gvis_words, Q, pool, W, vis);
    }
}

template <int C, typename XT, bool LEAN>
void (*pick_s_search_l(int L))(SParams) {
    if (L <= 64) return s_search_kernel<C, 1, XT, LEAN>;
    if (L <= 128) return s_search_kernel<C, 2, XT, LEAN>;
    return s_search_kernel<C, 4, XT, LEAN>;
}

template <int C, typename XT = float>
void (*pick_s_search_c(int L, bool lean))(SParams) {
    return lean ? pick_s_search_l<C, XT, true>(L) : pick_s_search_l<C, XT, false>(L);
}

}  // namespace

void (*pick_s_search(int dp, int L, int storage, bool lean))(SParams) {
    if (storage == FROG_STORAGE_F16)
        return dp == 64 ? pick_s_search_c<2, __half>(L, lean) : pick_s_search_c<4, __half>(L, lean);
    if (storage == FROG_STORAGE_BF16)
        return dp == 64 ? pick_s_search_c<2, bf16x>(L, lean) : pick_s_search_c<4, bf16x>(L, lean);
    switch (dp) {
        case 32: return pick_s_search_c<1>(L, lean);
        case 64: return pick_s_search_c<2>(L, lean);
        case 96: return pick_s_search_c<3>(L, lean);
        case 128: return pick_s_search_c<4>(L, lean);
        default: return pick_s_search_c<0>(L, lean);
    }
}

}  // namespace frog
