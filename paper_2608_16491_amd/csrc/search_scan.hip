// FROGSearch, entry mode 1: the matrix-core scan of the shared entry sample.

#include "search_shared.h"

namespace frog {
namespace {


// KT = dp / 16 float4 chunks of the query operand in registers (d <= 128);
// KT = 0 reloads it for every block (fp32 rows only).  XT is the rows'
// storage type: 16-bit rows are widened exactly to fp32 on load.
// Three wavefronts per SIMD: about 160 VGPRs (one row buffer) and, with
// 48-entry lists (L <= 40), 12.5 KB of LDS per wavefront.
template <int KT, int KK, typename XT = float>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(3))) void s_scan_kernel(SParams P) {
    static_assert(sizeof(XT) == 4 || (KT > 0 && KT % 2 == 0), "16-bit rows need dp a multiple of 32 held in registers");
    using namespace topk;
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int lane = lane_id();
    const int wave = threadIdx.x >> 6;
    const int64_t item = (int64_t)blockIdx.x * (blockDim.x >> 6) + wave;
    // when second-round tiles take more chunks than the others, items are
    // chunk-major (every tile's first chunk, then the second chunks, ...):
    // items past a tile's chunk count exit, and they fill whole workgroups
    // (whose LDS is then free again) instead of sitting beside live ones;
    // otherwise tile-major, a tile's chunks side by side in a workgroup
    const bool cmaj = P.nchunk > P.nbase;
    const int c = (int)(cmaj ? item / P.tmax : item % P.nchunk);
    const int64_t t = cmaj ? item % P.tmax : item / P.nchunk;
    if (t >= P.tmax) return;        // wave-uniform; no workgroup barrier follows
    const STile& T = P.tiles[t];
    if (T.nq == 0) return;
    const SharedLevels& lv = P.a.lv;
    const int lev = T.lev;
    const int64_t len = (int64_t)T.ub - T.ua;
    const int nch = T.nch;
    if (c >= nch) return;
    const int64_t c0 = T.ua + len * c / nch;
    const int64_t c1 = T.ua + len * (c + 1) / nch;
    const int dp = P.ix.dp, dp4 = dp >> 2, d = P.ix.d;
    constexpr int kkeep = KK;
    char* wb = smem + (size_t)wave * s_scan_lds_per_wave(kkeep);
    uint64_t* lkey = reinterpret_cast<uint64_t*>(wb);
    float* qnl = reinterpret_cast<float*>(lkey + kSQ * 2 * kkeep);
    int32_t* lst = reinterpret_cast<int32_t*>(qnl + kSQ);
    auto list_of = [&](int sl) { return BufList{lkey + (size_t)sl * 2 * kkeep, lst + 2 * sl}; };

    // MFMA operand mapping (16x16x4 f32): A[i][kk] in lane i + 16 kk, B[kk][j]
    // in lane j + 16 kk, D[4 (lane/16) + e][lane % 16] in element e.  Lane
    // group kk takes dimensions 16 u + 4 kk + {0..3} of K step u (fp32 rows),
    // or 32 (u/2) + 8 kk + 4 (u%2) + {0..3} (fp16 rows: one 16-byte load
    // feeds two K steps).
    const int ii = lane & 15;
    const int kk = lane >> 4;
    const int qrow = T.pair[ii] >= 0 ? T.pair[ii] / kSMaxWin : -1;
    const float* Qr = P.a.Q + (int64_t)(qrow >= 0 ? qrow : 0) * d;
    auto qchunk = [&](int u) -> float4 {
        const int b = sizeof(XT) == 4 ? 16 * u + 4 * kk : 32 * (u >> 1) + 8 * kk + 4 * (u & 1);
        float4 v;
        v.x = (qrow >= 0 && b < d) ? Qr[b] : 0.f;
        v.y = (qrow >= 0 && b + 1 < d) ? Qr[b + 1] : 0.f;
        v.z = (qrow >= 0 && b + 2 < d) ? Qr[b + 2] : 0.f;
        v.w = (qrow >= 0 && b + 3 < d) ? Qr[b + 3] : 0.f;
        return v;
    };
    float4 qa[KT > 0 ? KT : 1];
    float qs = 0.f;
    for (int u = 0; u < dp / 16; ++u) {
        const float4 v = qchunk(u);
        if constexpr (KT > 0) {
#pragma unroll
            for (int w = 0; w < KT; ++w)
                if (w == u) qa[w] = v;
        }
        qs += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
    }
    qs += __shfl_xor(qs, 16);
    qs += __shfl_xor(qs, 32);
    if (kk == 0) {
        qnl[ii] = qs;
        lst[2 * ii + 0] = 0;
        lst[2 * ii + 1] = 0x7f800000;
    }
    wave_sync();
    float qn[4];
    int32_t ql[4], qr[4];
    uint32_t qT[4];
    bool qv[4], qall[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int sl = 4 * kk + e;
        qn[e] = qnl[sl];
        ql[e] = T.l[sl];
        qr[e] = T.r[sl];
        qT[e] = T.T[sl];
        qv[e] = T.pair[sl] >= 0;
        qall[e] = (T.allmask >> sl) & 1u;
    }
    uint32_t scnt[4] = {0u, 0u, 0u, 0u};   // sample rows of slot 4kk + e seen by this lane

    const int64_t nblk = (c1 - c0 + 15) / 16;
    // the level's list and its rows (level 0: every rank, rows of X)
    const int32_t* lranks = lev == 0 ? nullptr : lv.ranks + lv.off[lev];
    const XT* X0 = rows_of<XT>(P.ix);
    const XT* Rl = lev == 0 ? X0 : lev_rows<XT>(lv) + lv.off[lev] * dp;
    const float4* R4 = reinterpret_cast<const float4*>(Rl);
    // the level's priorities and squared row norms, in list order
    const int64_t pbase = lev == 0 ? 0 : P.ix.n + lv.off[lev];
    const uint32_t* lprio = lv.prio + pbase;
    const float* lnorm = lv.norm + pbase;
    auto pos_at = [&](int64_t blk) -> int64_t {
        const int64_t pos = c0 + blk * 16 + ii;
        return pos < c1 ? pos : c1 - 1;   // in bounds past the end
    };
    // the rank load is unconditional (level 0 reads a priority word in its
    // place and discards it): a load under a branch would make the compiler
    // wait, at the first use of any older load, for the loads of the next
    // block issued before it
    const int32_t* rsrc = lranks ? lranks : reinterpret_cast<const int32_t*>(lv.prio);
    auto rank_at = [&](int64_t blk) -> int32_t {
        const int64_t pos = pos_at(blk);
        const int32_t v = rsrc[pos];
        return lranks ? v : (int32_t)pos;
    };
    auto load_rows = [&](int64_t blk, float4 (&x)[KT > 0 ? KT : 1]) {
        if constexpr (KT > 0) {
            const int64_t pos = pos_at(blk);
            if constexpr (sizeof(XT) == 4) {
#pragma unroll
                for (int u = 0; u < KT; ++u) x[u] = R4[pos * dp4 + 4 * u + kk];
            } else {
                // dp halves per row: 16-byte piece 4 v + kk holds K steps 2v, 2v + 1
                const int dp8 = dp >> 3;
#pragma unroll
                for (int v = 0; v < KT / 2; ++v) {
                    const uint4 h = reinterpret_cast<const uint4*>(Rl)[pos * dp8 + 4 * v + kk];
                    x[2 * v] = widen4<XT>(h.x, h.y);
                    x[2 * v + 1] = widen4<XT>(h.z, h.w);
                }
            }
        }
    };
    // list state in registers: entries per slot (uniform) and the threshold
    // of slot 4kk + e in each lane; LDS holds them only around a cut
    int fill[kSQ];
#pragma unroll
    for (int i = 0; i < kSQ; ++i) fill[i] = 0;
    float thr_l[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) thr_l[e] = __int_as_float(0x7f800000);
    // cut every list that the next block (at most 16 entries each) could overflow
    auto make_room = [&]() {
        // fast path: the fullest list has room (a max over the 16 fills)
        int fmax = fill[0];
#pragma unroll
        for (int i = 1; i < kSQ; ++i) fmax = fill[i] > fmax ? fill[i] : fmax;
        if (fmax <= 2 * kkeep - 16) return;
        uint32_t over = 0u;
#pragma unroll
        for (int i = 0; i < kSQ; ++i) over |= (fill[i] > 2 * kkeep - 16 ? 1u : 0u) << i;
        if (over == 0u) return;
        int myfill = 0;
#pragma unroll
        for (int i = 0; i < kSQ; ++i) myfill = lane == i ? fill[i] : myfill;
        if (lane < kSQ) lst[2 * lane] = myfill;
        list_sync();
        while (over) {
            const int sl = __builtin_ctz(over);
            over &= over - 1u;
            buf_cut<kkeep>(list_of(sl), false);
        }
        const int nf = lane < kSQ ? lst[2 * lane] : 0;
#pragma unroll
        for (int i = 0; i < kSQ; ++i) fill[i] = __builtin_amdgcn_readlane(nf, i);
#pragma unroll
        for (int e = 0; e < 4; ++e) thr_l[e] = __int_as_float(lst[2 * (4 * kk + e) + 1]);
    };
    // one 16-row block: q.x on the matrix cores (four independent
    // accumulation chains), then the candidates
    auto products = [&](const float4 (&x)[KT > 0 ? KT : 1], int64_t blk) -> floatx4_t {
        floatx4_t acc;
        if constexpr (KT > 0) {
            floatx4_t a0 = {0.f, 0.f, 0.f, 0.f}, a1 = a0, a2 = a0, a3 = a0;
#pragma unroll
            for (int u = 0; u < KT; ++u) {
                a0 = __builtin_amdgcn_mfma_f32_16x16x4f32(qa[u].x, x[u].x, a0, 0, 0, 0);
                a1 = __builtin_amdgcn_mfma_f32_16x16x4f32(qa[u].y, x[u].y, a1, 0, 0, 0);
                a2 = __builtin_amdgcn_mfma_f32_16x16x4f32(qa[u].z, x[u].z, a2, 0, 0, 0);
                a3 = __builtin_amdgcn_mfma_f32_16x16x4f32(qa[u].w, x[u].w, a3, 0, 0, 0);
            }
            acc = (a0 + a1) + (a2 + a3);
        } else {
            acc = floatx4_t{0.f, 0.f, 0.f, 0.f};
            for (int u = 0; u < dp / 16; ++u) {
                const float4 xv = R4[pos_at(blk) * dp4 + 4 * u + kk];
                const float4 q = qchunk(u);
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(q.x, xv.x, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(q.y, xv.y, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(q.z, xv.z, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(q.w, xv.w, acc, 0, 0, 0);
            }
        }
        return acc;
    };
    auto candidates = [&](const floatx4_t& acc, int32_t rk, uint32_t pri, float xn, int64_t blk) {
        const bool inrun = c0 + blk * 16 + ii < c1;
        const uint64_t below = (1ull << lane) - 1;
        // lane holds D[4kk + e][ii]: query slot 4kk + e, the block's row ii
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            // bitwise: every test evaluated, no branch per term
            const bool insample = inrun & qv[e] & (rk >= ql[e]) & (rk <= qr[e]) & (qall[e] | (pri < qT[e]));
            scnt[e] += insample ? 1u : 0u;
            const float ap = qn[e] + xn - 2.f * acc[e];
            const bool cand = insample && ap < thr_l[e];
            const uint64_t m = __ballot(cand);
            if (m == 0) continue;
            int myfill = fill[e];
#pragma unroll
            for (int g = 1; g < 4; ++g) myfill = kk == g ? fill[4 * g + e] : myfill;
            if (cand) {
                const uint64_t gm = m & (0xFFFFull << (16 * kk));
                lkey[(size_t)(4 * kk + e) * 2 * kkeep + myfill + __popcll(gm & below)] =
                    ((uint64_t)ord_bits(ap) << 32) | (uint32_t)rk;
            }
#pragma unroll
            for (int g = 0; g < 4; ++g) fill[4 * g + e] += __popcll(m & (0xFFFFull << (16 * g)));
        }
    };
    // one row buffer: the loads of block b + 1 are issued as soon as block
    // b's products are issued, and run during b's candidate logic and the
    // other wavefronts' work (positions past the end are clamped to the last
    // one, so the loads are in bounds and unconditional: a load under a branch
    // would make the compiler wait for it, and for every load issued before
    // it, at once)
    if (nblk > 0) {
        float4 x[KT > 0 ? KT : 1];
        load_rows(0, x);
        int32_t rk = rank_at(0);
        uint32_t pr = lprio[pos_at(0)];
        float xn = lnorm[pos_at(0)];
        for (int64_t blk = 0; blk < nblk; ++blk) {
            make_room();
            const floatx4_t acc = products(x, blk);
            load_rows(blk + 1, x);
            const int32_t rk1 = rank_at(blk + 1);
            const uint32_t pr1 = lprio[pos_at(blk + 1)];
            const float xn1 = lnorm[pos_at(blk + 1)];
            candidates(acc, rk, pr, xn, blk);
            rk = rk1;
            pr = pr1;
            xn = xn1;
        }
    }
    // the item's lists: entries kept, threshold, sample rows seen
    if (P.a.stats && lane == 0) {
        int first = 0;
        while (first < kSQ - 1 && T.pair[first] < 0) ++first;
        atomicAdd(P.a.stats + (int64_t)(T.pair[first] / kSMaxWin) * FROG_STAT_N + FROG_STAT_SCANROWS,
                  (int32_t)(nblk * 16));
    }
    // the lists' states to LDS for the last cuts and the write-out
    {
        int myfill = 0;
#pragma unroll
        for (int i = 0; i < kSQ; ++i) myfill = lane == i ? fill[i] : myfill;
        if (lane < kSQ) lst[2 * lane] = myfill;
        list_sync();
    }
    // per-slot sample counts: sum over the 16 lanes of each group
#pragma unroll
    for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) scnt[e] += __shfl_xor(scnt[e], o);
    uint32_t scount[kSQ];
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int e = 0; e < 4; ++e) scount[4 * g + e] = (uint32_t)__shfl((int)scnt[e], 16 * g);
    // slot i's list: (its pair, this chunk).  The slots' pairs are read
    // once, one per lane, before the loop: a load inside it would make each
    // slot wait for the stores of the lists before it (the wait counter
    // counts stores too)
    const int32_t pid_l = lane < kSQ ? T.pair[lane] : -1;
#pragma unroll
    for (int i = 0; i < kSQ; ++i) {
        const int32_t pid = __builtin_amdgcn_readlane(pid_l, i);
        if (pid < 0) continue;   // uniform: an empty slot has no list
        const int64_t lid = (int64_t)pid * P.nchunk + c;
        buf_cut<kkeep>(list_of(i));
        const int fi = __builtin_amdgcn_readfirstlane(lst[2 * i]);
        const uint64_t* kb = lkey + (size_t)i * 2 * kkeep;
        for (int j = lane; j < fi; j += 64) {
            const uint64_t key = kb[j];
            P.pv[lid * kkeep + j] = ord_value((uint32_t)(key >> 32));
            P.pr[lid * kkeep + j] = (int32_t)(uint32_t)key;
        }
        if (lane == 0) {
            P.pthr[lid] = __int_as_float(lst[2 * i + 1]);   // +inf unless a cut dropped rows
            P.pfill[lid] = fi;
            P.pcnt[lid] = (int32_t)scount[i];
        }
    }
}

template <int KK>
void (*pick_s_scan_k(int dp, int storage))(SParams) {
    if (storage == FROG_STORAGE_F16) return dp == 64 ? s_scan_kernel<4, KK, __half> : s_scan_kernel<8, KK, __half>;
    if (storage == FROG_STORAGE_BF16) return dp == 64 ? s_scan_kernel<4, KK, bf16x> : s_scan_kernel<8, KK, bf16x>;
    switch (dp) {
        case 32: return s_scan_kernel<2, KK>;
        case 64: return s_scan_kernel<4, KK>;
        case 96: return s_scan_kernel<6, KK>;
        case 128: return s_scan_kernel<8, KK>;
        default: return s_scan_kernel<0, KK>;
    }
}

}  // namespace

void (*pick_s_scan(int dp, int kkeep, int storage))(SParams) {
    if (kkeep == 48) return pick_s_scan_k<48>(dp, storage);
    if (kkeep == 64) return pick_s_scan_k<64>(dp, storage);
    if (kkeep == 128) return pick_s_scan_k<128>(dp, storage);
    return pick_s_scan_k<256>(dp, storage);
}

}  // namespace frog
