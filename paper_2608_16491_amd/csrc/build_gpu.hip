// Index construction on the GPU (Sec 6), one wavefront per vertex.
//
// The host puts the objects in attribute-rank order (Sec 4) and tabulates the
// fusion-distance factor of Eq. fusion-distance for every offset of every
// segment length; the kernels build the layers bottom-up exactly as the host
// construction does, so the candidate array is the same entry for entry:
//
//   leaf layer    every vertex against the other members of its leaf
//                 segment: the m smallest fusion distances are its ENC row,
//                 the m smallest distances its temporary-graph row;
//   layer h       the vertex's child-layer temporary-graph row (m-ANN inside
//                 its own child), a greedy best-first search with patience
//                 over the sibling child's temporary graph (Alg. 1, pool
//                 ef_c, stratified seeds), the union sorted by distance, RNG
//                 pruned into this layer's temporary-graph row, and re-ranked
//                 by fusion distance into the ENC row of layer h.
//
// Distances are the construction's own: the terms in dimension order, each
// difference, square and partial sum in double, one rounding to float.  A
// lane computes a whole distance, so the order is the same as on the host;
// a wavefront evaluates up to 64 of them at once (the sibling search's new
// candidates, the seeds, the leaf segment, the pairs of the RNG prune).
//
// The sibling search keeps its visited set in a direct-mapped LDS table that
// may forget entries.  That changes no result: a vertex evaluated again is
// either still in the pool (its key is dropped as a duplicate) or was pushed
// out of a full pool, whose largest key only decreases, so it cannot get
// back in; the pool, the expansion order and the patience count are those of
// an exact visited set.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstring>
#include <vector>

#include "frog_internal.h"

namespace frog {

namespace {

constexpr int32_t kNone = -1;
constexpr int kBW = 4;               // wavefronts per workgroup
constexpr int kBBlock = 64 * kBW;
constexpr uint64_t kEmptyKey = ~0ull;

__device__ __forceinline__ int lane_id() { return __lane_id(); }
__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }

__device__ __forceinline__ uint64_t readlane64(uint64_t v, int l) {
    const uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)v, l);
    const uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), l);
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ double readlane_f64(double v, int l) {
    return __longlong_as_double((long long)readlane64((uint64_t)__double_as_longlong(v), l));
}

__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ uint64_t splitmix64(uint64_t x) {
    uint64_t z = x + 0x9E3779B97F4A7C15ULL;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

// (distance, id) as one ordered key; distances are >= 0
__device__ __forceinline__ uint64_t dkey(float d, int32_t id) {
    return ((uint64_t)__float_as_uint(d) << 32) | (uint32_t)id;
}
__device__ __forceinline__ float key_dist(uint64_t k) { return __uint_as_float((uint32_t)(k >> 32)); }
__device__ __forceinline__ int32_t key_id(uint64_t k) { return (int32_t)(uint32_t)k; }

// (a, ia) < (b, ib) for double keys with id ties
__device__ __forceinline__ bool less_fk(double a, int32_t ia, double b, int32_t ib) {
    return a < b || (a == b && ia < ib);
}

// The segment at depth h holding rank p (split rule of Alg. 3: the left
// child [L, mid] with mid = L + floor((R - L) / 2)).
__device__ __forceinline__ void segment_of(int64_t n, int h, int64_t p, int64_t& s, int64_t& e) {
    int64_t L = 0, R = n - 1;
    for (int i = 0; i < h; ++i) {
        const int64_t mid = L + (R - L) / 2;
        if (p <= mid) R = mid; else L = mid + 1;
    }
    s = L;
    e = R;
}

// The construction's squared L2 of two rows (dp floats, zero padded: the
// padding adds +0 and changes nothing).
__device__ __forceinline__ float dist_seq(const float* __restrict__ a, const float* __restrict__ b, int dp) {
    double s = 0.0;
#pragma unroll 8
    for (int i = 0; i < dp; i += 4) {
        const float4 x = *reinterpret_cast<const float4*>(a + i);
        const float4 y = *reinterpret_cast<const float4*>(b + i);
        double t = (double)x.x - (double)y.x;
        s = s + t * t;
        t = (double)x.y - (double)y.y;
        s = s + t * t;
        t = (double)x.z - (double)y.z;
        s = s + t * t;
        t = (double)x.w - (double)y.w;
        s = s + t * t;
    }
    return (float)s;
}

// The same distance with the first row already widened to double (the
// vertex's own row, kept in LDS): t = a_i - (double)b_i as above.
__device__ __forceinline__ float dist_seq_q(const double* __restrict__ a, const float* __restrict__ b, int dp) {
    double s = 0.0;
#pragma unroll 8
    for (int i = 0; i < dp; i += 4) {
        const double2 x0 = *reinterpret_cast<const double2*>(a + i);
        const double2 x1 = *reinterpret_cast<const double2*>(a + i + 2);
        const float4 y = *reinterpret_cast<const float4*>(b + i);
        double t = x0.x - (double)y.x;
        s = s + t * t;
        t = x0.y - (double)y.y;
        s = s + t * t;
        t = x1.x - (double)y.z;
        s = s + t * t;
        t = x1.y - (double)y.w;
        s = s + t * t;
    }
    return (float)s;
}

struct BArgs {
    const float* X;          // n x dp, rank order
    const int32_t* PGc;      // temporary graph of the child layer, n x m
    int32_t* PGn;            // temporary graph of this layer, n x m
    int32_t* ENC;            // n x H x m
    const double* wtab;      // fusion factors (see fusion_weights)
    const int64_t* wmeta;    // 4 per depth
    unsigned long long* stats;  // [0] distances, [1] expansions, [2] length mismatches
    int64_t n;
    int dp, H, m, h, ef, patience, nseed, hash_log2;
    int lds_per_wave;
    uint64_t seed;
};

// the fusion factor of offset diff in a depth-h segment of length len; a
// length the table does not hold is counted and reads offset 0's factor
__device__ __forceinline__ double fusion_factor(const BArgs& A, int h, int64_t len, int64_t diff) {
    const int64_t* mt = A.wmeta + 4 * h;
    int64_t off;
    if (len == mt[0]) off = mt[1];
    else if (len == mt[2]) off = mt[3];
    else {
        atomicAdd(A.stats + 2, 1ull);
        return A.wtab[mt[1]];
    }
    return A.wtab[off + diff];
}

// A sorted list of at most cap <= 64 (double key, id) entries, entry t in
// lane t.  merge() adds the lanes' new entries (unique ids) and keeps the
// cap smallest.
struct FList {
    double k;
    int32_t id;
    int cnt;
    __device__ void init() { k = 0.0; id = kNone; cnt = 0; }
    __device__ void merge(double nk, int32_t nid, bool valid, int cap, double* st_k, int32_t* st_id) {
        const int lane = lane_id();
        const uint64_t vm = ballot(valid);
        if (vm == 0) return;
        int pos_new = 0, shift = 0;
        for (uint64_t mm = vm; mm; mm &= mm - 1) {
            const int j = __builtin_ctzll(mm);
            const double kj = readlane_f64(nk, j);
            const int32_t ij = __builtin_amdgcn_readlane(nid, j);
            pos_new += (valid && less_fk(kj, ij, nk, nid)) ? 1 : 0;
            shift += (lane < cnt && less_fk(kj, ij, k, id)) ? 1 : 0;
        }
        for (int t = 0; t < cnt; ++t) {
            const double kt = readlane_f64(k, t);
            const int32_t it = __builtin_amdgcn_readlane(id, t);
            pos_new += (valid && less_fk(kt, it, nk, nid)) ? 1 : 0;
        }
        if (lane < cnt && lane + shift < cap) { st_k[lane + shift] = k; st_id[lane + shift] = id; }
        if (valid && pos_new < cap) { st_k[pos_new] = nk; st_id[pos_new] = nid; }
        const int nc = cnt + __popcll(vm);
        cnt = nc < cap ? nc : cap;
        wave_sync();
        if (lane < cnt) { k = st_k[lane]; id = st_id[lane]; }
        wave_sync();
    }
};

// ------------------------------------------------------------------ leaf layer

__global__ __launch_bounds__(kBBlock) void leaf_kernel(BArgs A) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int lane = lane_id();
    const int wave = threadIdx.x >> 6;
    const int64_t u = (int64_t)blockIdx.x * kBW + wave;
    if (u >= A.n) return;   // wave-uniform; no workgroup barrier follows
    char* wb = smem + (size_t)wave * A.lds_per_wave;
    float* xu = reinterpret_cast<float*>(wb);
    double* st_k = reinterpret_cast<double*>(wb + (size_t)A.dp * 4);
    int32_t* st_id = reinterpret_cast<int32_t*>(st_k + 64);
    const int h = A.H - 1, m = A.m, dp = A.dp;
    int64_t s, e;
    segment_of(A.n, h, u, s, e);
    const int64_t len = e - s + 1;
    const float4* xr = reinterpret_cast<const float4*>(A.X + u * dp);
    for (int i = lane; i < dp / 4; i += 64) reinterpret_cast<float4*>(xu)[i] = xr[i];
    wave_sync();
    FList F, P;
    F.init();
    P.init();
    unsigned long long nd = 0;
    for (int64_t b0 = s; b0 <= e; b0 += 64) {
        const int64_t v = b0 + lane;
        const bool ok = v <= e && v != u;
        float d2 = 0.f;
        double fk = 0.0;
        if (ok) {
            d2 = dist_seq(xu, A.X + v * dp, dp);
            const int64_t diff = v > u ? v - u : u - v;
            fk = sqrt((double)d2) * fusion_factor(A, h, len, diff);
        }
        nd += __popcll(ballot(ok));
        F.merge(fk, (int32_t)v, ok, m, st_k, st_id);
        P.merge((double)d2, (int32_t)v, ok, m, st_k, st_id);
    }
    if (lane < m) {
        A.ENC[(u * A.H + h) * m + lane] = lane < F.cnt ? F.id : kNone;
        A.PGn[u * m + lane] = lane < P.cnt ? P.id : kNone;
    }
    if (lane == 0 && A.stats) atomicAdd(A.stats, nd);
}

// ------------------------------------------------------------------ internal layers

// The sibling search's pool: up to 64 LP keys sorted ascending, entry
// 64 s + lane in key[s], with an expanded flag.
template <int LP>
struct BPool {
    uint64_t key[LP];
    uint32_t flag[LP];
    int np;
};

// Merge the lanes' new keys into the pool (capacity cap): duplicates of pool
// keys are dropped, the cap smallest kept.  Returns whether a new key landed
// among the first `top` entries.
template <int LP>
__device__ bool bpool_merge(BPool<LP>& P, uint64_t nkey, bool cand, int cap, int top, uint64_t* st_key,
                            uint32_t* st_flag) {
    const int lane = lane_id();
    if (P.np >= cap) {
        const int t = cap - 1;
        uint64_t thr = 0;
#pragma unroll
        for (int s = 0; s < LP; ++s)
            if (s == (t >> 6)) thr = readlane64(P.key[s], t & 63);
        cand = cand && nkey < thr;
    }
    const uint64_t cmask = ballot(cand);
    if (cmask == 0) return false;
    bool keep = cand;
    for (uint64_t mm = cmask; mm; mm &= mm - 1) {
        const int j = __builtin_ctzll(mm);
        const uint64_t kj = readlane64(nkey, j);
        bool eq = false;
#pragma unroll
        for (int s = 0; s < LP; ++s) eq |= P.key[s] == kj;
        if (ballot(eq) != 0 && lane == j) keep = false;
    }
    const uint64_t kmask = ballot(keep);
    if (kmask == 0) return false;
    int ltN = 0, cntP = 0;
    int ltP[LP];
#pragma unroll
    for (int s = 0; s < LP; ++s) ltP[s] = 0;
    for (uint64_t mm = kmask; mm; mm &= mm - 1) {
        const int j = __builtin_ctzll(mm);
        const uint64_t kj = readlane64(nkey, j);
        int c = 0;
#pragma unroll
        for (int s = 0; s < LP; ++s) {
            c += __popcll(ballot(P.key[s] < kj));
            ltP[s] += kj < P.key[s] ? 1 : 0;
        }
        if (lane == j) cntP = c;
        ltN += kj < nkey ? 1 : 0;
    }
#pragma unroll
    for (int s = 0; s < LP; ++s) {
        const int p = s * 64 + lane;
        const int pos = p + ltP[s];
        if (p < P.np && pos < cap) {
            st_key[pos] = P.key[s];
            st_flag[pos] = P.flag[s];
        }
    }
    const int posn = cntP + ltN;
    if (keep && posn < cap) {
        st_key[posn] = nkey;
        st_flag[posn] = 0u;
    }
    const bool improved = ballot(keep && posn < top) != 0;
    const int nk = __popcll(kmask);
    P.np = P.np + nk < cap ? P.np + nk : cap;
    wave_sync();
#pragma unroll
    for (int s = 0; s < LP; ++s) {
        const int p = s * 64 + lane;
        P.key[s] = p < P.np ? st_key[p] : kEmptyKey;
        P.flag[s] = p < P.np ? st_flag[p] : 0u;
    }
    wave_sync();
    return improved;
}

// LDS per wavefront of the layer kernel
__host__ __device__ inline size_t layer_region_bytes(int m, int hash_log2) {
    const size_t tab = (size_t)4 << hash_log2;
    const size_t pairs = (size_t)16 * (m + 3);   // the prune's distances of a round
    return tab > pairs ? tab : pairs;
}
__host__ __device__ inline size_t layer_lds_per_wave(int dp, int m, int hash_log2, int lp) {
    return (size_t)dp * 8 + layer_region_bytes(m, hash_log2) + (size_t)64 * lp * 12 + (size_t)64 * 12;
}

template <int LP>
__global__ __launch_bounds__(kBBlock) void layer_kernel(BArgs A) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int lane = lane_id();
    const int wave = threadIdx.x >> 6;
    const int64_t u = (int64_t)blockIdx.x * kBW + wave;
    if (u >= A.n) return;   // wave-uniform; no workgroup barrier follows
    const int h = A.h, m = A.m, dp = A.dp, ef = A.ef;
    char* wb = smem + (size_t)wave * A.lds_per_wave;
    double* xu = reinterpret_cast<double*>(wb);   // u's row, widened
    char* region = wb + (size_t)dp * 8;
    int32_t* tab = reinterpret_cast<int32_t*>(region);        // visited table, then the prune's distances
    float* gd = reinterpret_cast<float*>(region);
    uint64_t* st_key = reinterpret_cast<uint64_t*>(region + layer_region_bytes(m, A.hash_log2));
    uint32_t* st_flag = reinterpret_cast<uint32_t*>(st_key + 64 * LP);
    int32_t* sid = reinterpret_cast<int32_t*>(st_flag + 64 * LP);  // up to 64 ids in sorted order
    float* sdist = reinterpret_cast<float*>(sid + 64);            // their distances
    int32_t* outp = reinterpret_cast<int32_t*>(sdist + 64);       // pruned row (m <= 32)
    const uint32_t tmask = (1u << A.hash_log2) - 1u;

    int64_t s, e;
    segment_of(A.n, h, u, s, e);
    const int64_t len = e - s + 1;
    const int64_t mid = s + (e - s) / 2;
    int64_t ts, te;
    if (u <= mid) { ts = mid + 1; te = e; } else { ts = s; te = mid; }
    for (int i = lane; i < dp; i += 64) xu[i] = (double)A.X[u * dp + i];
    for (int i = lane; i <= (int)tmask; i += 64) tab[i] = -1;
    wave_sync();
    unsigned long long nd = 0, nexp = 0;

    // the child layer's row: m-ANN of u inside its own child segment
    const int32_t va = lane < m ? A.PGc[u * m + lane] : kNone;
    float da = 0.f;
    if (va != kNone) da = dist_seq_q(xu, A.X + (int64_t)va * dp, dp);
    nd += __popcll(ballot(va != kNone));

    // greedy search of Alg. 1 over the sibling's temporary graph
    BPool<LP> P;
#pragma unroll
    for (int s2 = 0; s2 < LP; ++s2) { P.key[s2] = kEmptyKey; P.flag[s2] = 0u; }
    P.np = 0;
    const int64_t tl = te - ts + 1;
    if (tl > 0) {
        // seeds: the whole sibling when it is small, else one jittered rank
        // per stratum
        int ns;
        int32_t sv = kNone;
        if (tl <= A.nseed) {
            ns = (int)tl;
            if (lane < ns) sv = (int32_t)(ts + lane);
        } else {
            ns = A.nseed;
            if (lane < ns) {
                const int64_t a = ts + ((int64_t)lane * tl) / ns;
                const int64_t b = ts + ((int64_t)(lane + 1) * tl) / ns - 1;
                const uint64_t z = splitmix64(A.seed ^ ((uint64_t)u << 32) ^ ((uint64_t)h << 24) ^ (uint64_t)lane);
                sv = (int32_t)(a + (int64_t)(((z >> 32) * (uint64_t)(b - a + 1)) >> 32));
            }
        }
        const bool isv = lane < ns;
        if (isv) tab[((uint32_t)sv * 0x9E3779B1u) >> (32 - A.hash_log2)] = sv;
        float ds = 0.f;
        if (isv) ds = dist_seq_q(xu, A.X + (int64_t)sv * dp, dp);
        nd += (unsigned long long)ns;
        bpool_merge<LP>(P, isv ? dkey(ds, sv) : kEmptyKey, isv, ef, m, st_key, st_flag);
        int left = A.patience;
        for (int64_t guard = 0; guard <= tl; ++guard) {
            // first unexpanded entry
            int sel = -1;
#pragma unroll
            for (int s2 = 0; s2 < LP; ++s2) {
                const uint64_t fm = ballot(s2 * 64 + lane < P.np && P.flag[s2] == 0u);
                if (sel < 0 && fm != 0) sel = s2 * 64 + __builtin_ctzll(fm);
            }
            if (sel < 0) break;
            uint64_t wk = 0;
#pragma unroll
            for (int s2 = 0; s2 < LP; ++s2)
                if (s2 == (sel >> 6)) {
                    wk = readlane64(P.key[s2], sel & 63);
                    if (lane == (sel & 63)) P.flag[s2] = 1u;
                }
            const int32_t w = key_id(wk);
            ++nexp;
            // the expanded vertex's row, restricted to the sibling segment
            const int32_t v = lane < m ? A.PGc[(int64_t)w * m + lane] : kNone;
            bool fresh = v != kNone && v >= ts && v <= te;
            if (fresh) {
                const uint32_t slot = ((uint32_t)v * 0x9E3779B1u) >> (32 - A.hash_log2);
                if (tab[slot] == v) fresh = false;
                else tab[slot] = v;
            }
            float dv = 0.f;
            if (fresh) dv = dist_seq_q(xu, A.X + (int64_t)v * dp, dp);
            nd += __popcll(ballot(fresh));
            const bool improved = bpool_merge<LP>(P, fresh ? dkey(dv, v) : kEmptyKey, fresh, ef, m, st_key, st_flag);
            if (improved) {
                left = A.patience;
            } else {
                left = left - 1;
                if (left <= 0) break;
            }
        }
    }
    wave_sync();

    // the union sorted by (distance, id): child row in lanes [0, m), the
    // search's m nearest in lanes [m, 2m)
    const int nb = P.np < m ? P.np : m;
    uint64_t ck = kEmptyKey;
    bool cv = false;
    if (lane < m) { cv = va != kNone; ck = cv ? dkey(da, va) : kEmptyKey; }
    const int src = (lane - m) & 63;
    const uint64_t pk = ((uint64_t)(uint32_t)__shfl((int)(uint32_t)(P.key[0] >> 32), src) << 32) |
                        (uint32_t)__shfl((int)(uint32_t)P.key[0], src);
    if (lane >= m && lane < m + nb) { cv = true; ck = pk; }
    const uint64_t vmask = ballot(cv);
    const int nc = __popcll(vmask);
    int rank = 0;
    for (uint64_t mm = vmask; mm; mm &= mm - 1) {
        const int j = __builtin_ctzll(mm);
        rank += readlane64(ck, j) < ck ? 1 : 0;
    }
    if (cv) { sid[rank] = key_id(ck); sdist[rank] = key_dist(ck); }
    wave_sync();

    // RNG prune (alpha = 1) in candidate order, four candidates per round:
    // each is tested against the rows kept before the round and against the
    // round's earlier candidates, and kept unless one of the kept rows is
    // closer to it than u is.  These are the decisions of the one-by-one
    // test (its early exit only skips distances).
    const int G = m + 3;   // member gi's distances at gd[gi G + slot]
    uint64_t kept = 0;
    int nk = 0;
    for (int i0 = 0; i0 < nc && nk < m; i0 += 4) {
        const int g = nc - i0 < 4 ? nc - i0 : 4;
        const int nk0 = nk;
        // member gi: slots [0, nk0) the rows kept so far, then the round's
        // members before it; its pairs start at gi nk0 + gi (gi - 1) / 2
        const int npair = g * nk0 + g * (g - 1) / 2;
        for (int p0 = 0; p0 < npair; p0 += 64) {
            const int p = p0 + lane;
            if (p < npair) {
                int gi = 0;
                while (gi + 1 < g && (gi + 1) * nk0 + (gi + 1) * gi / 2 <= p) ++gi;
                const int slot = p - (gi * nk0 + gi * (gi - 1) / 2);
                const int32_t other = slot < nk0 ? outp[slot] : sid[i0 + slot - nk0];
                gd[gi * G + slot] = dist_seq(A.X + (int64_t)sid[i0 + gi] * dp, A.X + (int64_t)other * dp, dp);
            }
        }
        nd += (unsigned long long)npair;
        wave_sync();
        uint32_t acc = 0;   // members kept in this round
        for (int gi = 0; gi < g && nk < m; ++gi) {
            const float di = sdist[i0 + gi];
            bool viol = false;
            if (lane < nk0 + gi) {
                const bool live = lane < nk0 || ((acc >> (lane - nk0)) & 1u);
                viol = live && gd[gi * G + lane] < di;
            }
            if (ballot(viol) == 0) {
                acc |= 1u << gi;
                kept |= 1ull << (i0 + gi);
                if (lane == 0) outp[nk] = sid[i0 + gi];
                ++nk;
            }
        }
        wave_sync();
    }
    for (int i = 0; i < nc && nk < m; ++i)
        if (!((kept >> i) & 1ull)) {
            if (lane == 0) outp[nk] = sid[i];
            ++nk;
        }
    wave_sync();
    if (lane < m) A.PGn[u * m + lane] = lane < nk ? outp[lane] : kNone;

    // fusion re-rank into the ENC row of layer h
    double fk = 0.0;
    int32_t fid = kNone;
    const bool fv = lane < nc;
    if (fv) {
        fid = sid[lane];
        const int64_t diff = fid > u ? (int64_t)fid - u : u - (int64_t)fid;
        fk = sqrt((double)sdist[lane]) * fusion_factor(A, h, len, diff);
    }
    int fr = 0;
    for (int j = 0; j < nc; ++j) {
        const double kj = readlane_f64(fk, j);
        const int32_t ij = __builtin_amdgcn_readlane(fid, j);
        fr += (fv && less_fk(kj, ij, fk, fid)) ? 1 : 0;
    }
    if (fv && fr < m) A.ENC[(u * A.H + h) * m + fr] = fid;
    if (lane == 0 && A.stats) {
        atomicAdd(A.stats, nd);
        atomicAdd(A.stats + 1, nexp);
    }
}

__global__ void fill_kernel(int32_t* p, int64_t count, int32_t v) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < count) p[i] = v;
}

template <int LP>
int launch_layer(const BArgs& A, hipStream_t stream) {
    const size_t lpw = layer_lds_per_wave(A.dp, A.m, A.hash_log2, LP);
    const size_t smem = lpw * kBW;
    if (smem > 160 * 1024) return fail(FROG_EUNSUPPORTED, "construction needs %zu B of LDS per workgroup", smem);
    if (smem > 64 * 1024) {
        const hipError_t e = hipFuncSetAttribute((const void*)layer_kernel<LP>,
                                                 hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
        if (e != hipSuccess) return fail(FROG_EHIP, "hipFuncSetAttribute: %s", hipGetErrorString(e));
    }
    BArgs B = A;
    B.lds_per_wave = (int)lpw;
    const int64_t blocks = (A.n + kBW - 1) / kBW;
    hipLaunchKernelGGL(layer_kernel<LP>, dim3((unsigned)blocks), dim3(kBBlock), smem, stream, B);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(FROG_EHIP, "layer kernel: %s", hipGetErrorString(e));
    return FROG_OK;
}

}  // namespace

bool device_build_supported(int d, const frog_build_params_t& p) {
    return d >= 1 && d <= 1024 && p.m >= 1 && p.m <= 32 && p.ef_c >= p.m && p.ef_c <= 256 && p.sib_seeds >= 1 &&
           p.sib_seeds <= 64;
}

int build_device(const float* X, const double* attr, int64_t n, int d, const frog_build_params_t& p,
                 int device, frog_index* out) {
    if (!device_build_supported(d, p))
        return fail(FROG_EUNSUPPORTED, "GPU construction needs d <= 1024, m <= 32, ef_c <= 256, sib_seeds <= 64");
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess) return fail(FROG_EHIP, "hipGetDeviceCount failed");
    if (device < 0 || device >= ndev) return fail(FROG_EINVAL, "device %d not in [0, %d)", device, ndev);
    const int m = p.m;
    const int threads = host_threads(p.num_threads);
    // ENC is left unset on the host: the device array is filled with -1 and
    // copied back whole
    int rc = rank_order(X, attr, n, d, m, p.n_inv, threads, false, out);
    if (rc != FROG_OK) return rc;
    const int H = out->H;
    std::vector<double> wtab;
    std::vector<int64_t> wmeta;
    rc = fusion_weights(n, H, p.beta, p.gamma, threads, wtab, wmeta);
    if (rc != FROG_OK) return rc;
    const int dp = (d + 31) / 32 * 32;
    const int lp = p.ef_c <= 64 ? 1 : (p.ef_c <= 128 ? 2 : 4);
    const int hash_log2 = 9;

    int prev = 0;
    if (hipGetDevice(&prev) != hipSuccess) return fail(FROG_EHIP, "hipGetDevice failed");
    if (hipSetDevice(device) != hipSuccess) return fail(FROG_EHIP, "hipSetDevice failed");
    float* dX = nullptr;
    int32_t *dENC = nullptr, *dPG0 = nullptr, *dPG1 = nullptr, *dperm = nullptr;
    double *dW = nullptr, *dattr = nullptr;
    int64_t* dMeta = nullptr;
    unsigned long long* dStats = nullptr;
    const size_t nX = (size_t)n * dp, nE = (size_t)n * H * m, nP = (size_t)n * m;
    auto cleanup = [&]() {
        if (dX) (void)hipFree(dX);
        if (dENC) (void)hipFree(dENC);
        if (dPG0) (void)hipFree(dPG0);
        if (dPG1) (void)hipFree(dPG1);
        if (dW) (void)hipFree(dW);
        if (dMeta) (void)hipFree(dMeta);
        if (dStats) (void)hipFree(dStats);
        if (dattr) (void)hipFree(dattr);
        if (dperm) (void)hipFree(dperm);
        (void)hipSetDevice(prev);
    };
    hipError_t e = hipMalloc(&dX, nX * sizeof(float));
    if (e == hipSuccess) e = hipMalloc(&dENC, nE * sizeof(int32_t));
    if (e == hipSuccess) e = hipMalloc(&dPG0, nP * sizeof(int32_t));
    if (e == hipSuccess) e = hipMalloc(&dPG1, nP * sizeof(int32_t));
    if (e == hipSuccess) e = hipMalloc(&dW, wtab.size() * sizeof(double));
    if (e == hipSuccess) e = hipMalloc(&dMeta, wmeta.size() * sizeof(int64_t));
    if (e == hipSuccess) e = hipMalloc(&dStats, 4 * sizeof(unsigned long long));
    if (e == hipSuccess) e = hipMalloc(&dattr, (size_t)n * sizeof(double));
    if (e == hipSuccess) e = hipMalloc(&dperm, (size_t)n * sizeof(int32_t));
    if (e != hipSuccess) {
        cleanup();
        return fail(e == hipErrorOutOfMemory ? FROG_ENOMEM : FROG_EHIP, "construction buffers: %s",
                    hipGetErrorString(e));
    }
    hipStream_t stream = nullptr;
    if (dp == d) {
        e = hipMemcpy(dX, out->X.data(), nX * sizeof(float), hipMemcpyHostToDevice);
    } else {
        e = hipMemset(dX, 0, nX * sizeof(float));
        if (e == hipSuccess)
            e = hipMemcpy2D(dX, (size_t)dp * sizeof(float), out->X.data(), (size_t)d * sizeof(float),
                            (size_t)d * sizeof(float), (size_t)n, hipMemcpyHostToDevice);
    }
    if (e == hipSuccess) e = hipMemcpy(dW, wtab.data(), wtab.size() * sizeof(double), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(dMeta, wmeta.data(), wmeta.size() * sizeof(int64_t), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemset(dStats, 0, 4 * sizeof(unsigned long long));
    if (e == hipSuccess) e = hipMemcpy(dattr, out->attr.data(), (size_t)n * sizeof(double), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(dperm, out->perm.data(), (size_t)n * sizeof(int32_t), hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        cleanup();
        return fail(FROG_EHIP, "construction upload: %s", hipGetErrorString(e));
    }
    hipEvent_t ev0 = nullptr, ev1 = nullptr;
    if (hipEventCreate(&ev0) != hipSuccess || hipEventCreate(&ev1) != hipSuccess) {
        if (ev0) (void)hipEventDestroy(ev0);
        cleanup();
        return fail(FROG_EHIP, "hipEventCreate failed");
    }
    (void)hipEventRecord(ev0, stream);
    hipLaunchKernelGGL(fill_kernel, dim3((unsigned)((nE + 255) / 256)), dim3(256), 0, stream, dENC, (int64_t)nE, kNone);

    BArgs A{};
    A.X = dX;
    A.ENC = dENC;
    A.wtab = dW;
    A.wmeta = dMeta;
    A.stats = dStats;
    A.n = n;
    A.dp = dp;
    A.H = H;
    A.m = m;
    A.ef = p.ef_c;
    A.patience = p.patience;
    A.nseed = p.sib_seeds;
    A.hash_log2 = hash_log2;
    A.seed = p.seed;
    // leaf layer into the first temporary graph
    A.h = H - 1;
    A.PGc = nullptr;
    A.PGn = dPG0;
    A.lds_per_wave = dp * 4 + 64 * 12;
    const int64_t blocks = (n + kBW - 1) / kBW;
    hipLaunchKernelGGL(leaf_kernel, dim3((unsigned)blocks), dim3(kBBlock), (size_t)A.lds_per_wave * kBW, stream, A);
    e = hipGetLastError();
    if (e != hipSuccess) {
        (void)hipDeviceSynchronize();
        (void)hipEventDestroy(ev0);
        (void)hipEventDestroy(ev1);
        cleanup();
        return fail(FROG_EHIP, "leaf kernel: %s", hipGetErrorString(e));
    }
    int32_t* cur = dPG0;
    int32_t* nxt = dPG1;
    for (int h = H - 2; h >= 0; --h) {
        A.h = h;
        A.PGc = cur;
        A.PGn = nxt;
        rc = lp == 1 ? launch_layer<1>(A, stream) : (lp == 2 ? launch_layer<2>(A, stream) : launch_layer<4>(A, stream));
        if (rc != FROG_OK) {
            (void)hipDeviceSynchronize();
            (void)hipEventDestroy(ev0);
            (void)hipEventDestroy(ev1);
            cleanup();
            return rc;
        }
        std::swap(cur, nxt);
    }
    (void)hipEventRecord(ev1, stream);
    e = hipDeviceSynchronize();
    float kms = 0.f;
    if (e == hipSuccess) (void)hipEventElapsedTime(&kms, ev0, ev1);
    (void)hipEventDestroy(ev0);
    (void)hipEventDestroy(ev1);
    unsigned long long st[4] = {0, 0, 0, 0};
    if (e == hipSuccess) e = hipMemcpy(st, dStats, sizeof(st), hipMemcpyDeviceToHost);
    if (e == hipSuccess) e = hipMemcpy(out->ENC.data(), dENC, nE * sizeof(int32_t), hipMemcpyDeviceToHost);
    if (e != hipSuccess) {
        cleanup();
        return fail(FROG_EHIP, "construction: %s", hipGetErrorString(e));
    }
    if (st[2] != 0) {
        cleanup();
        return fail(FROG_EHIP, "construction: %llu segment lengths outside the fusion table", st[2]);
    }
    out->build_distances = (int64_t)st[0];
    out->build_expansions = (int64_t)st[1];
    out->build_kernel_ms = kms;
    // keep the construction's rows, candidate array, attributes and id map
    // as the device copy
    (void)hipFree(dPG0);
    (void)hipFree(dPG1);
    (void)hipFree(dW);
    (void)hipFree(dMeta);
    (void)hipFree(dStats);
    out->device = device;
    out->dp = dp;
    out->storage = FROG_STORAGE_F32;
    out->dX = dX;
    out->dENC = dENC;
    out->dattr = dattr;
    out->dperm = dperm;
    out->maxnorm = stored_maxnorm(out);
    (void)hipSetDevice(prev);
    return FROG_OK;
}

}  // namespace frog
