// FROGSearch, entry mode 1: each query's pool from its tile's scan lists
// (exact re-rank, margin test).

#include "search_shared.h"

namespace frog {
namespace {

// The sum of s and the minimum of m over the wavefront, uniform (every lane
// active): data-parallel-primitive moves within each row of 16 lanes, then
// the four rows' results.
__device__ __forceinline__ void wave_sum_min(int& s, float& m) {
    auto step = [&](auto ctrl) {
        constexpr int c = decltype(ctrl)::value;
        s += __builtin_amdgcn_mov_dpp(s, c, 0xF, 0xF, false);
        m = fminf(m, __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(m), c, 0xF, 0xF, false)));
    };
    step(std::integral_constant<int, 0xB1>{});
    step(std::integral_constant<int, 0x4E>{});
    step(std::integral_constant<int, 0x141>{});
    step(std::integral_constant<int, 0x140>{});
    int rs = __builtin_amdgcn_readlane(s, 0);
    float rm = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(m), 0));
#pragma unroll
    for (int r = 16; r < 64; r += 16) {
        rs += __builtin_amdgcn_readlane(s, r);
        rm = fminf(rm, __int_as_float(__builtin_amdgcn_readlane(__float_as_int(m), r)));
    }
    s = rs;
    m = rm;
}

// Exact distances of up to 64 candidates for the pool kernel.  Pools of at
// most 64 gather 16 rows per step, one step at a time: the kernel then fits
// 80 VGPRs and 6 wavefronts per SIMD, so that a 10k-query batch runs in two
// rounds of wavefronts (with two steps in flight it needed 128 VGPRs and
// ran at 4 per SIMD: 67 against 62 us at C2).  Larger pools keep two steps
// in flight at 3 per SIMD.  Both give the same distances (the same
// per-candidate arithmetic).
template <int C, int LP, typename XT, typename QC>
__device__ __forceinline__ float pool_eval(const DevIndex& ix, const QC& Q, int cnt, int32_t myid) {
    if constexpr (C > 0 && LP == 1) {
        float mine = 0.f;
        Gather16<C, XT> g;
        for (int sb0 = 0; sb0 < cnt; sb0 += 16) {
            g.issue(rows_of<XT>(ix), ix.dp, cnt, myid, sb0);
            g.consume(Q.qv, sb0, mine);
        }
        return mine;
    } else {
        return Q.eval_batch(ix, cnt, myid);
    }
}

// The pool of each query: one wavefront per query.  Six wavefronts per
// SIMD for pools of at most 64, three above (no spill either way).
template <int C, int LP, int KK, typename XT = float, int MK = (KK > 64 ? KK : 64)>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(LP == 1 ? 6 : 3))) void s_pool_kernel(SParams P) {
    using namespace topk;
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const DevIndex& ix = P.ix;
    const SearchLaunch& A = P.a;
    const int lane = lane_id();
    const int wave = threadIdx.x >> 6;
    WaveLds<LP> W(smem, P.lds_per_wave, 0);
    char* lbase = smem + (size_t)wave * P.lds_per_wave + P.lds_list;
    // KK: entries of each chunk list the scan left (their stride); the merged
    // list keeps MK >= 64 of them (an offer of 64 fits after a cut), twice
    // the chunk lists' 256 for pools above 248 so that the margin test spans
    // many ranks past the pool's last
    constexpr int kkeep = MK;
    const BufList Lst{reinterpret_cast<uint64_t*>(lbase), reinterpret_cast<int32_t*>(lbase + (size_t)2 * kkeep * 8)};
    const double u_round = 5.9604644775390625e-08;   // 2^-24

    {
        const int64_t idx = (int64_t)blockIdx.x * (blockDim.x >> 6) + wave;
        if (idx >= A.nq) return;   // wave-uniform; no workgroup barrier follows
        const int64_t qi = uniform(P.qorder[idx]);   // the planned order (short queries last)
        const SPlan* pp = P.plan + qi;
        QueryCtx<C, XT> Q;
        Q.qrow = A.Q + qi * ix.d;
        Q.load_vector(ix);   // issued beside the plan's load
        const SPlan p = *pp;
        if (p.l > p.r) return;
        Q.set(ix, A, qi, p.l, p.r);
        Q.shared = true;
        Q.T = p.T;
        Q.pkey = A.lv.key;

        // the kkeep smallest approximate distances over the query's lists:
        // window wi's chunk count in lane wi, its chunks numbered after those
        // of windows 0..wi-1, list i's fill, threshold and sample count in
        // lane i
        buf_init(Lst);
        const bool tiled = p.nw <= kSMaxWin;   // else no lists: the exact pass below
        const int nwq = tiled ? p.nw : 0;
        int wn = 0;   // from the plan already loaded, not a second read
#pragma unroll
        for (int x = 0; x < kSMaxWin; ++x) wn = lane == x && x < nwq ? p.wchunks[x] : wn;
        int wbase = wn;   // inclusive prefix over lanes 0..kSMaxWin-1
#pragma unroll
        for (int o = 1; o < kSMaxWin; o <<= 1) {
            const int v = __shfl_up(wbase, o);
            if (lane >= o) wbase += v;
        }
        const int nl = __builtin_amdgcn_readlane(wbase, kSMaxWin - 1);   // lists, at most kSMaxWin kSMaxChunks
        wbase -= wn;
        int wi = 0;
#pragma unroll
        for (int x = 1; x < kSMaxWin; ++x)
            if (x < nwq && __builtin_amdgcn_readlane(wbase, x) <= lane) wi = x;
        const int lc = lane - __shfl(wbase, wi);
        const int64_t lid = (qi * kSMaxWin + wi) * P.nchunk + lc;   // list `lane`: (pair, chunk)
        int mf = 0, mc = 0;
        float mt = __int_as_float(0x7f800000);
        if (lane < nl) {
            mf = P.pfill[lid];
            mt = P.pthr[lid];
            mc = P.pcnt[lid];
        }
        wave_sum_min(mc, mt);
        int64_t ne = mc;
        float texcl = mt;   // every row left out is at or above this
        // several lists' entries at a time (no round trip between them)
        constexpr int kR = KK > 64 ? KK / 64 : 1;   // entries per lane and list
        constexpr int kG = kR == 1 ? 16 : 4;
        for (int i0 = 0; i0 < nl; i0 += kG) {
            float av[kG][kR];
            int32_t rw[kG][kR];
#pragma unroll
            for (int g = 0; g < kG; ++g) {
                const int i = (i0 + g) & 63;
                const int fi = i0 + g < nl ? __builtin_amdgcn_readlane(mf, i) : 0;
                const int64_t li = ((int64_t)__builtin_amdgcn_readlane((int32_t)(lid >> 32), i) << 32) |
                                   (uint32_t)__builtin_amdgcn_readlane((int32_t)lid, i);
#pragma unroll
                for (int r = 0; r < kR; ++r) {
                    const int j = r * 64 + lane;
                    av[g][r] = j < fi ? P.pv[li * KK + j] : __int_as_float(0x7f800000);
                    rw[g][r] = j < fi ? P.pr[li * KK + j] : -1;
                }
            }
#pragma unroll
            for (int g = 0; g < kG; ++g) {
#pragma unroll
                for (int r = 0; r < kR; ++r) {
                    const uint64_t gm = ballot(rw[g][r] >= 0 && av[g][r] < __int_as_float(Lst.st[1]));
                    if (gm) buf_offer<kkeep>(Lst, gm, av[g][r], rw[g][r]);
                }
            }
        }
        buf_cut<kkeep>(Lst);
        texcl = fminf(texcl, __int_as_float(Lst.st[1]));
        const int f = uniform(Lst.st[0]);

        // exact distances of the kept rows: the pool of the L nearest
        Pool<LP> pool;
#pragma unroll
        for (int s = 0; s < LP; ++s) { pool.key[s] = kEmpty; pool.flag[s] = 0u; }
        pool.np = 0;
        if (f <= 64) {
            // one key per lane: a bitonic sort over the wavefront, the first L are the pool
            const int32_t id = lane < f ? (int32_t)(uint32_t)Lst.key[lane] : 0;
            const float dd = pool_eval<C, LP, XT>(ix, Q, f, id);
            uint64_t key = lane < f ? make_key(dd, id) : kEmpty;
#pragma unroll
            for (int kb = 2; kb <= 64; kb <<= 1) {
#pragma unroll
                for (int jb = kb >> 1; jb > 0; jb >>= 1) {
                    const uint64_t other = (uint64_t)__shfl_xor((long long)key, jb);
                    const bool up = (lane & kb) == 0;
                    const bool low = (lane & jb) == 0;
                    key = (low == up) ? (other < key ? other : key) : (other > key ? other : key);
                }
            }
#pragma unroll
            for (int s = 0; s < LP; ++s) pool.key[s] = (s == 0 && lane < A.L) ? key : kEmpty;
            pool.np = f < A.L ? f : A.L;
        } else {
            for (int j0 = 0; j0 < f; j0 += 64) {
                const int nb = f - j0 < 64 ? f - j0 : 64;
                const int32_t id = lane < nb ? (int32_t)(uint32_t)Lst.key[j0 + lane] : 0;
                const float dd = pool_eval<C, LP, XT>(ix, Q, nb, id);
                merge<LP>(pool, lane < nb ? make_key(dd, id) : kEmpty, nb, A.L, W.st_key, W.st_flag);
            }
        }
        // margin test: a row left out has exact distance >= texcl - eps
        bool certified = tiled;
        if (tiled && !(texcl == __int_as_float(0x7f800000))) {
            certified = false;
            if (pool.np >= A.L) {
                double qsq = 0.0;
                if constexpr (C > 0) {
                    // from the query chunks in registers: each aligned group of
                    // 8 lanes holds the whole query
#pragma unroll
                    for (int c = 0; c < C; ++c)
                        qsq += (double)Q.qv[c].x * Q.qv[c].x + (double)Q.qv[c].y * Q.qv[c].y +
                               (double)Q.qv[c].z * Q.qv[c].z + (double)Q.qv[c].w * Q.qv[c].w;
                    qsq = sum8(qsq);
                } else {
                    for (int cc = lane; cc < ix.d; cc += 64) qsq += (double)Q.qrow[cc] * (double)Q.qrow[cc];
#pragma unroll
                    for (int o = 32; o >= 1; o >>= 1) qsq += __shfl_xor(qsq, o);
                }
                const double eps = 2.0 * (2.0 * ix.d + 4.0) * u_round * (qsq + (double)A.maxnorm);
                uint64_t lk = 0;
#pragma unroll
                for (int s = 0; s < LP; ++s)
                    if (s == ((A.L - 1) >> 6)) lk = readlane64(pool.key[s], (A.L - 1) & 63);
                const double dL = (double)__uint_as_float((uint32_t)(lk >> 32));
                certified = (double)texcl - eps > dL;
            }
        }
        certified = uniform(certified ? 1 : 0) != 0;
        if (!certified) {
            // every sample row, exactly
#pragma unroll
            for (int s = 0; s < LP; ++s) { pool.key[s] = kEmpty; pool.flag[s] = 0u; }
            pool.np = 0;
            ne = 0;
            for (int64_t b0 = p.a; b0 < p.b; b0 += 64) {
                const int64_t pos = b0 + lane;
                const int32_t rk = pos < p.b ? level_rank(A.lv, p.lev, pos) : 0;
                const bool in = pos < p.b && (p.all || s_priority(A.lv.key, rk) < p.T);
                const uint64_t pm = ballot(in);
                const int nb = __popcll(pm);
                ne += nb;
                if (nb == 0) continue;
                if (in) W.enbuf[mbcnt(pm)] = rk;
                wave_sync();
                const int32_t id = lane < nb ? W.enbuf[lane] : 0;
                wave_sync();
                const float dd = pool_eval<C, LP, XT>(ix, Q, nb, id);
                merge<LP>(pool, lane < nb ? make_key(dd, id) : kEmpty, nb, A.L, W.st_key, W.st_flag);
            }
        }
#pragma unroll
        for (int s = 0; s < LP; ++s) P.pools[qi * 64 * LP + s * 64 + lane] = pool.key[s];
        if (lane == 0) {
            P.pne[qi] = (int32_t)ne;
            if (A.stats) A.stats[qi * FROG_STAT_N + FROG_STAT_FALLBACK] = certified ? 0 : 1;
        }
    }
}

template <int C, typename XT = float>
void (*pick_s_pool_c(int L))(SParams) {
    const int kk = shared_kkeep(L);
    if (L <= 64)
        return kk == 48 ? s_pool_kernel<C, 1, 48, XT> : (kk == 64 ? s_pool_kernel<C, 1, 64, XT> : s_pool_kernel<C, 1, 128, XT>);
    if (L <= 128) return kk == 128 ? s_pool_kernel<C, 2, 128, XT> : s_pool_kernel<C, 2, 256, XT>;
    if (L > 248) return s_pool_kernel<C, 4, 256, XT, 512>;
    return s_pool_kernel<C, 4, 256, XT>;
}

}  // namespace

void (*pick_s_pool(int dp, int L, int storage))(SParams) {
    if (storage == FROG_STORAGE_F16) return dp == 64 ? pick_s_pool_c<2, __half>(L) : pick_s_pool_c<4, __half>(L);
    if (storage == FROG_STORAGE_BF16) return dp == 64 ? pick_s_pool_c<2, bf16x>(L) : pick_s_pool_c<4, bf16x>(L);
    switch (dp) {
        case 32: return pick_s_pool_c<1>(L);
        case 64: return pick_s_pool_c<2>(L);
        case 96: return pick_s_pool_c<3>(L);
        case 128: return pick_s_pool_c<4>(L);
        default: return pick_s_pool_c<0>(L);
    }
}

}  // namespace frog
