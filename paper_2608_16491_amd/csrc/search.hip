// FROGSearch on gfx950: range -> rank interval (Sec 4), HotspotLocalization
// (Alg. 3), entry points (Alg. 2), and the best-first loop of Alg. 2 with
// ENIdentification (Alg. 4), the lazy visited check, distance evaluation and
// MergeTopEfS.
//
// Mapping to CDNA4:
//   - one query per 64-lane wavefront, four independent wavefronts per
//     workgroup, a persistent grid that takes queries from an atomic counter;
//   - the candidate pool (size L <= 64*LP) lives in VGPRs: pool slot p is
//     register s = p / 64 of lane p % 64, holding a 64-bit key
//     (float bits of the squared distance << 32 | rank) -- for non-negative
//     floats the bit pattern orders like the value, so (distance, rank) order
//     is one unsigned compare -- and an expanded flag;
//   - selecting the first unexpanded entry is one ballot per register;
//   - ENIdentification loads up to 64 hotspot candidates per wave load (one
//     per lane, in stored order) and compacts the in-range ones with
//     ballot + mbcnt under the budget B, as Alg. 4 describes for a warp;
//   - the visited check runs after compaction (the paper's lazy check) on a
//     direct-mapped table of 2^hash_log2 ranks in LDS: a lookup is one read,
//     an insert one write.  The table may forget a vertex (a later insert to
//     the same slot overwrites it) but never reports an unseen vertex as
//     seen.  Forgetting cannot change the result: a re-evaluated vertex gets
//     the same key; if it is still in the pool the merge drops the duplicate,
//     and if it is not, it was rejected or evicted when the pool was full, so
//     its key is at or above the pool's current L-th key (which never grows)
//     and the merge rejects it again.  Only the number of evaluations grows.
//     hash_log2 = 0 selects an exact per-wave bitmap in device memory instead
//     (used to count distinct evaluations);
//   - distances: each vector is read by 8 lanes as 16-byte loads (128
//     contiguous bytes per load instruction and vector), differences and
//     squares in double, an 8-lane butterfly sum, one rounding to float --
//     the library's canonical squared L2.  d > 128 uses all 64 lanes per
//     vector.  No matrix cores: every gathered vector is used once;
//   - MergeTopEfS: a new key's position is (# pool keys below it) + (# new
//     keys below it), counted with ballots; a pool key's position is its slot
//     plus (# new keys below it); entries scatter through LDS.  Keys are
//     unique once duplicates are dropped, so this equals sorting the union.

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <cstdint>
#include <map>
#include <mutex>
#include <type_traits>
#include <vector>

#include "frog_internal.h"
#include "wave_topk.h"

namespace frog {
namespace {

constexpr int kWave = 64;
constexpr int kWavesPerBlock = 4;
constexpr int kBlock = kWave * kWavesPerBlock;
constexpr uint64_t kEmpty = ~0ull;
typedef float floatx4_t __attribute__((ext_vector_type(4)));
// Register budget: at least 3 wavefronts per SIMD (168 VGPRs); four would
// make the d = 128 kernel spill, which costs more than the lost wave.
#ifndef FROG_WAVES_PER_EU
#define FROG_WAVES_PER_EU 3
#endif
// The shared-sample traversal kernel needs about 100 VGPRs: 5 wavefronts per SIMD.
#ifndef FROG_SEARCH_WAVES_PER_EU
#define FROG_SEARCH_WAVES_PER_EU 5
#endif
// Entry points per work unit (a chunk of a query's entry phase).
#ifndef FROG_CHUNK
#define FROG_CHUNK 768
#endif

struct KParams {
    DevIndex ix;
    SearchLaunch a;
    unsigned int* counter;   // [2] work counters: entry units, queries
    const int32_t* lr;       // [nq][2] rank intervals, from the prologue kernel
    uint64_t* part;          // [nq][cpq][64 * LP] pools of the entry chunks
    unsigned int* done;      // [nq] finished entry chunks per query
    uint32_t* gvis;          // exact visited bitmaps (hash_log2 == 0)
    int64_t gvis_words;      // words per wave
    int lds_per_wave;        // bytes
    int cpq;                 // work units (entry chunks) per query
    int chunk;               // entry points per chunk, a multiple of 16
};

// ------------------------------------------------------------------ wave helpers

__device__ __forceinline__ int lane_id() { return __lane_id(); }

__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }

__device__ __forceinline__ int mbcnt(uint64_t m) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

__device__ __forceinline__ uint64_t readlane64(uint64_t v, int l) {
    uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)v, l);
    uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), l);
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

__device__ __forceinline__ int64_t uniform64(int64_t v) {
    uint32_t lo = __builtin_amdgcn_readfirstlane((int)(uint32_t)v);
    uint32_t hi = __builtin_amdgcn_readfirstlane((int)(uint32_t)((uint64_t)v >> 32));
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Orders LDS traffic between the lanes of one wavefront.
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

__device__ __forceinline__ uint64_t make_key(float d, int32_t id) {
    return ((uint64_t)__float_as_uint(d) << 32) | (uint32_t)id;
}

// Data-parallel-primitive lane moves of a double (two 32-bit DPP moves).
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
    const uint64_t u = (uint64_t)__double_as_longlong(v);
    const int lo = __builtin_amdgcn_mov_dpp((int)(uint32_t)u, CTRL, 0xF, 0xF, false);
    const int hi = __builtin_amdgcn_mov_dpp((int)(uint32_t)(u >> 32), CTRL, 0xF, 0xF, false);
    return __longlong_as_double((long long)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo));
}

// Sum over each aligned group of 8 lanes, the same value in all 8: quad swaps
// [1,0,3,2] and [2,3,0,1], then the half-row mirror pairs the two quads.
__device__ __forceinline__ double sum8(double s) {
    s += dpp_f64<0xB1>(s);
    s += dpp_f64<0x4E>(s);
    s += dpp_f64<0x141>(s);
    return s;
}

// ------------------------------------------------------------------ a1: ranks

// Number of entries of the ascending array a[0, n) below x (inclusive: <= x),
// by a 64-ary search: each round every lane probes one position and a ballot
// narrows the interval 64-fold.
__device__ int64_t count_below(const double* __restrict__ a, int64_t n, double x, bool inclusive) {
    const int lane = lane_id();
    int64_t lo = 0, hi = n;
    while (hi > lo) {
        const int64_t step = (hi - lo + 63) / 64;
        const int64_t p = lo + (int64_t)(lane + 1) * step - 1;
        bool below = false;
        if (p < hi) {
            const double v = a[p];
            below = inclusive ? (v <= x) : (v < x);
        }
        const int c = __popcll(ballot(below));
        const int64_t nlo = lo + (int64_t)c * step;
        int64_t nhi = lo + (int64_t)(c + 1) * step - 1;
        if (nhi > hi) nhi = hi;
        lo = uniform64(nlo);
        hi = uniform64(nhi);
    }
    return lo;
}

__device__ void rank_interval(const DevIndex& ix, double lo_v, double hi_v, int64_t& l, int64_t& r) {
    if (isnan(lo_v) || isnan(hi_v)) { l = 0; r = -1; return; }
    l = count_below(ix.attr, ix.n, lo_v, false);
    r = count_below(ix.attr, ix.n, hi_v, true) - 1;
}

// ------------------------------------------------------------------ a2: hotspot

__device__ void segment_of(int64_t n, int h, int64_t p, int64_t& s, int64_t& e) {
    int64_t L = 0, R = n - 1;
    for (int i = 0; i < h; ++i) {
        const int64_t mid = L + (R - L) / 2;
        if (p <= mid) R = mid; else L = mid + 1;
    }
    s = L;
    e = R;
}

// Alg. 3: L_start = depth of the deepest segment holding [l, r] (at most H-1);
// L_end extends over consecutive deeper layers while Eq. endcondition holds,
// with the boundary terms b_l = (end of l's segment) + 1, b_r = start of r's.
__device__ void hotspot(int64_t l, int64_t r, int H, int64_t n, int& Ls, int& Le) {
    int64_t L = 0, R = n - 1;
    int d = 0;
    while (d < H - 1) {
        const int64_t mid = L + (R - L) / 2;
        if (r <= mid) R = mid;
        else if (l >= mid + 1) L = mid + 1;
        else break;
        ++d;
    }
    Ls = d;
    Le = d;
    for (int h = d + 1; h <= H - 1; ++h) {
        int64_t sl, el, sr, er;
        segment_of(n, h, l, sl, el);
        segment_of(n, h, r, sr, er);
        const int64_t lhs = (el + 1 - l) + (r - sr);
        if (lhs * ((int64_t)1 << h) >= (r - l)) Le = h;
        else break;
    }
}

// ------------------------------------------------------------------ a8: distances

// Row layout a lane reads (C = dp / 32 float4 chunks per lane, 8 lanes per
// row).  fp32 rows: chunk c of lane `sub` is float4 number sub + 8c of the
// row.  16-bit rows (fp16 or bf16, dp a multiple of 64): the lane's 16-byte
// piece sub + 8(c/2) holds 8 values, of which chunk c is the first or second
// 4, widened exactly to float.

// bfloat16 storage: the upper 16 bits of an fp32 value (a tag type; the
// rows hold the bit patterns).
struct bf16x {
    uint16_t bits;
};

// Four stored 16-bit values (two 32-bit words, first value in the low half)
// widened exactly to float.
template <typename XT>
__device__ __forceinline__ float4 widen4(uint32_t w0, uint32_t w1) {
    if constexpr (std::is_same<XT, __half>::value) {
        const float2 a = __half22float2(__builtin_bit_cast(__half2, w0));
        const float2 b = __half22float2(__builtin_bit_cast(__half2, w1));
        return make_float4(a.x, a.y, b.x, b.y);
    } else {
        static_assert(std::is_same<XT, bf16x>::value, "16-bit storage is fp16 or bf16");
        return make_float4(__uint_as_float(w0 << 16), __uint_as_float(w0 & 0xFFFF0000u), __uint_as_float(w1 << 16),
                           __uint_as_float(w1 & 0xFFFF0000u));
    }
}

// All C chunks of row `id` for lane `sub` (zeros when !v).  fp16 rows take
// one 16-byte load per pair of chunks, so that the 8 lanes of a row read
// 128 contiguous bytes per instruction, as for fp32 rows.
template <int C, typename XT>
__device__ __forceinline__ void load_row(const XT* __restrict__ X, int dp, int64_t id, int sub, bool v,
                                         float4 (&x)[C]) {
    if constexpr (sizeof(XT) == 4) {
#pragma unroll
        for (int c = 0; c < C; ++c)
            x[c] = v ? reinterpret_cast<const float4*>(X)[id * (dp >> 2) + sub + 8 * c]
                     : make_float4(0.f, 0.f, 0.f, 0.f);
    } else {
        static_assert(C % 2 == 0, "fp16 rows come in pairs of chunks");
#pragma unroll
        for (int p = 0; p < C / 2; ++p) {
            const uint4 h = v ? reinterpret_cast<const uint4*>(X)[id * (dp >> 3) + sub + 8 * p]
                              : make_uint4(0u, 0u, 0u, 0u);
            x[2 * p] = widen4<XT>(h.x, h.y);
            x[2 * p + 1] = widen4<XT>(h.z, h.w);
        }
    }
}

// The query dimensions a lane pairs with chunk c (the layout of load_row).
template <typename XT>
__device__ __forceinline__ int chunk_dim(int sub, int c) {
    if constexpr (sizeof(XT) == 4) return 4 * (sub + 8 * c);
    else return 8 * (sub + 8 * (c >> 1)) + 4 * (c & 1);
}

// Squared L2 of up to `cnt` (<= 64) candidates; lane j holds candidate j's
// rank in `myid` and receives its distance in the return value.  The query's
// float4 chunks this lane needs are in qv.
template <int C, typename XT = float>
__device__ float eval_small(const XT* __restrict__ X, int dp, const float4 (&qv)[C], int cnt, int32_t myid) {
    // G = 8 lanes per vector: lane reads float4 chunks (lane % 8) + 8c; one
    // group of 8 vectors per step (an expansion rarely yields more than 8)
    const int lane = lane_id();
    const int sub = lane & 7;
    const int src = (lane & 7) << 3;
    float mine = 0.f;
    for (int sb0 = 0; sb0 < cnt; sb0 += 8) {
        const int j = sb0 + (lane >> 3);
        const int id = __shfl(myid, j & 63);
        const bool v = j < cnt;
        float4 x[C];
        load_row<C, XT>(X, dp, id, sub, v, x);
        double s = 0.0;
#pragma unroll
        for (int c = 0; c < C; ++c) {
            // keep the query in fp32 registers: convert per use, not once
            float4 qf = qv[c];
            asm volatile("" : "+v"(qf.x), "+v"(qf.y), "+v"(qf.z), "+v"(qf.w));
            const double q0 = qf.x, q1 = qf.y, q2 = qf.z, q3 = qf.w;
            double t;
            t = q0 - (double)x[c].x; s += t * t;
            t = q1 - (double)x[c].y; s += t * t;
            t = q2 - (double)x[c].z; s += t * t;
            t = q3 - (double)x[c].w; s += t * t;
        }
        s = sum8(s);
        // vector sb0 + g sits in lanes 8g..8g+7; lane sb0 + g takes it
        const float got = __shfl((float)s, src);
        if ((lane >> 3) == ((sb0 >> 3) & 7)) mine = got;
    }
    return mine;
}

// Same result as eval_small for the entry-point batches (up to 64 candidates),
// with two steps of 16 vectors in flight: the loads of step i+1 are issued
// before step i is reduced, so the arithmetic overlaps the memory latency.
template <int C, typename XT = float>
struct Gather16 {
    float4 x[2][C];
    __device__ __forceinline__ void issue(const XT* __restrict__ X, int dp, int cnt, int32_t myid, int sb0) {
        const int lane = lane_id();
        const int sub = lane & 7;
#pragma unroll
        for (int g = 0; g < 2; ++g) {
            const int j = sb0 + 8 * g + (lane >> 3);
            const int id = __shfl(myid, j & 63);
            const bool v = j < cnt;
            load_row<C, XT>(X, dp, id, sub, v, x[g]);
        }
    }
    __device__ __forceinline__ void consume(const float4 (&qv)[C], int sb0, float& mine) const {
        const int lane = lane_id();
        double s[2] = {0.0, 0.0};
#pragma unroll
        for (int c = 0; c < C; ++c) {
            float4 qf = qv[c];
            asm volatile("" : "+v"(qf.x), "+v"(qf.y), "+v"(qf.z), "+v"(qf.w));
            const double q0 = qf.x, q1 = qf.y, q2 = qf.z, q3 = qf.w;
#pragma unroll
            for (int g = 0; g < 2; ++g) {
                double t;
                t = q0 - (double)x[g][c].x; s[g] += t * t;
                t = q1 - (double)x[g][c].y; s[g] += t * t;
                t = q2 - (double)x[g][c].z; s[g] += t * t;
                t = q3 - (double)x[g][c].w; s[g] += t * t;
            }
        }
        const int src = (lane & 7) << 3;
#pragma unroll
        for (int g = 0; g < 2; ++g) {
            const float f = (float)sum8(s[g]);
            const float got = __shfl(f, src);
            if ((lane >> 3) == (((sb0 >> 3) + g) & 7)) mine = got;
        }
    }
};

template <int C, typename XT = float>
__device__ float eval_pipelined(const XT* __restrict__ X, int dp, const float4 (&qv)[C], int cnt, int32_t myid) {
    float mine = 0.f;
    Gather16<C, XT> a, b;
    a.issue(X, dp, cnt, myid, 0);
    for (int sb0 = 0; sb0 < cnt; sb0 += 32) {
        if (sb0 + 16 < cnt) b.issue(X, dp, cnt, myid, sb0 + 16);
        a.consume(qv, sb0, mine);
        if (sb0 + 32 < cnt) a.issue(X, dp, cnt, myid, sb0 + 32);
        if (sb0 + 16 < cnt) b.consume(qv, sb0 + 16, mine);
    }
    return mine;
}

// d > 128: all 64 lanes read one vector, float4 chunk lane + 64c.
__device__ float eval_large(const float* __restrict__ X, int dp, const float* __restrict__ q, int d, int cnt,
                            int32_t myid) {
    const int lane = lane_id();
    const float4* __restrict__ X4 = reinterpret_cast<const float4*>(X);
    const int dp4 = dp >> 2;
    float mine = 0.f;
    for (int j = 0; j < cnt; ++j) {
        const int id = __builtin_amdgcn_readlane(myid, j);
        double s = 0.0;
        for (int c = lane; c < dp4; c += 64) {
            const float4 x = X4[(int64_t)id * dp4 + c];
            const int b = 4 * c;
            const double q0 = b < d ? q[b] : 0.f, q1 = b + 1 < d ? q[b + 1] : 0.f;
            const double q2 = b + 2 < d ? q[b + 2] : 0.f, q3 = b + 3 < d ? q[b + 3] : 0.f;
            double t;
            t = q0 - (double)x.x; s += t * t;
            t = q1 - (double)x.y; s += t * t;
            t = q2 - (double)x.z; s += t * t;
            t = q3 - (double)x.w; s += t * t;
        }
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) s += __shfl_xor(s, o);
        if (lane == j) mine = (float)s;
    }
    return mine;
}

// ------------------------------------------------------------------ pool

template <int LP>
struct Pool {
    uint64_t key[LP];
    uint32_t flag[LP];
    int np;  // valid entries, wave-uniform
};

// MergeTopEfS: merge new keys (lane j < ns holds one; others kEmpty) into the
// pool, dropping keys already present and keys at or beyond the pool's L-th
// when it is full.  Returns the number of keys that entered.
template <int LP>
__device__ int merge(Pool<LP>& P, uint64_t nkey, int ns, int L, uint64_t* st_key, uint32_t* st_flag) {
    const int lane = lane_id();
    bool cand = lane < ns;
    if (P.np >= L) {
        const int t = L - 1;
        uint64_t thr = 0;
#pragma unroll
        for (int s = 0; s < LP; ++s)
            if (s == (t >> 6)) thr = readlane64(P.key[s], t & 63);
        cand = cand && nkey < thr;
    }
    uint64_t cmask = ballot(cand);
    if (cmask == 0) return 0;
    // drop duplicates: of a pool key, or of an earlier new key
    bool keep = cand;
    for (uint64_t m = cmask; m; m &= m - 1) {
        const int j = __builtin_ctzll(m);
        const uint64_t kj = readlane64(nkey, j);
        bool eq = false;
#pragma unroll
        for (int s = 0; s < LP; ++s) eq |= P.key[s] == kj;
        if (ballot(eq) != 0 && lane == j) keep = false;
        if (lane > j && nkey == kj) keep = false;
    }
    const uint64_t kmask = ballot(keep);
    const int nk = __popcll(kmask);
    if (nk == 0) return 0;
    // positions
    int ltN = 0, cntP = 0;
    int ltP[LP];
#pragma unroll
    for (int s = 0; s < LP; ++s) ltP[s] = 0;
    for (uint64_t m = kmask; m; m &= m - 1) {
        const int j = __builtin_ctzll(m);
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
    // scatter
#pragma unroll
    for (int s = 0; s < LP; ++s) {
        const int p = s * 64 + lane;
        const int pos = p + ltP[s];
        if (p < P.np && pos < L) {
            st_key[pos] = P.key[s];
            st_flag[pos] = P.flag[s];
        }
    }
    if (keep) {
        const int pos = cntP + ltN;
        if (pos < L) {
            st_key[pos] = nkey;
            st_flag[pos] = 0u;
        }
    }
    P.np = P.np + nk < L ? P.np + nk : L;
    wave_sync();
#pragma unroll
    for (int s = 0; s < LP; ++s) {
        const int p = s * 64 + lane;
        P.key[s] = p < P.np ? st_key[p] : kEmpty;
        P.flag[s] = p < P.np ? st_flag[p] : 0u;
    }
    wave_sync();
    return nk;
}

// ------------------------------------------------------------------ visited set

struct Visited {
    int32_t* tab;        // LDS table (forgetful) or nullptr
    uint32_t* bits;      // exact bitmap in device memory
    int shift;           // 32 - hash_log2
    __device__ __forceinline__ uint32_t slot(int32_t v) const { return ((uint32_t)v * 0x9E3779B1u) >> shift; }
    // true if v has not been seen (and records it); never false for an unseen v
    __device__ __forceinline__ bool check_insert(int32_t v) const {
        if (tab) {
            const uint32_t s = slot(v);
            if (tab[s] == v) return false;
            tab[s] = v;
            return true;
        }
        const uint32_t bit = 1u << (v & 31);
        return (atomicOr(bits + (v >> 5), bit) & bit) == 0;
    }
    // membership without inserting (exact set)
    __device__ __forceinline__ bool contains(int32_t v) const {
        if (tab) return tab[slot(v)] == v;
        return (atomicOr(bits + (v >> 5), 0u) >> (v & 31)) & 1u;
    }
    __device__ __forceinline__ void insert(int32_t v) const {
        if (tab) tab[slot(v)] = v;
        else atomicOr(bits + (v >> 5), 1u << (v & 31));
    }
};

// ------------------------------------------------------------------ kernel

// Per-wave LDS: pool staging (64 LP keys + flags), the EN list, the visited
// table.
template <int LP>
struct WaveLds {
    uint64_t* st_key;
    uint32_t* st_flag;
    int32_t* enbuf;
    int32_t* tab;
    __device__ WaveLds(char* smem, int lds_per_wave, int hash_log2) {
        char* wbase = smem + (size_t)(threadIdx.x >> 6) * lds_per_wave;
        st_key = reinterpret_cast<uint64_t*>(wbase);
        st_flag = reinterpret_cast<uint32_t*>(st_key + 64 * LP);
        enbuf = reinterpret_cast<int32_t*>(st_flag + 64 * LP);
        tab = hash_log2 > 0 ? enbuf + 64 : nullptr;
    }
};

// Query context shared by both kernels: the query's float4 chunks this lane
// needs, its rank interval and its entry points (Alg. 2).
// floor(a / b) for 0 <= a < 2^51, b > 0, given rb ~ 1/b: the double estimate is
// off by at most one, which the integer check corrects.
__device__ __forceinline__ int64_t floor_div(int64_t a, int64_t b, double rb) {
    int64_t f = (int64_t)((double)a * rb);
    if (f * b > a) --f;
    else if ((f + 1) * b <= a) ++f;
    return f;
}

// The index's rows, and the shared sample's level rows, in storage type T
// (fp32 or fp16).
template <typename XT>
__device__ __forceinline__ const XT* rows_of(const DevIndex& ix) {
    if constexpr (sizeof(XT) == 4) return ix.X;
    else return reinterpret_cast<const XT*>(ix.Xh);
}
template <typename XT>
__device__ __forceinline__ const XT* lev_rows(const SharedLevels& lv) {
    if constexpr (sizeof(XT) == 4) return lv.xrows;
    else return reinterpret_cast<const XT*>(lv.xrowsh);
}

template <int C, typename XT = float>
struct QueryCtx {
    float4 qv[C > 0 ? C : 1];
    const float* qrow;
    int64_t qi, l, r, cnt, E, ne;
    double rE;
    bool all;
    uint64_t qkey;
    // shared entry sample: rank i of [l, r] is an entry point iff
    // hi32(splitmix64(pkey ^ i)) < T
    bool shared = false;
    uint32_t T = 0;
    uint64_t pkey = 0;

    __device__ void load(const DevIndex& ix, const SearchLaunch& A, const int32_t* lr, int64_t q) {
        qi = q;
        l = uniform(lr[2 * q]);
        r = uniform(lr[2 * q + 1]);
        cnt = r - l + 1;
        E = A.epn;
        if (A.epn_frac > 0.0) {
            double want = ceil(A.epn_frac * (double)cnt);
            if (want > (double)A.epn_max) want = (double)A.epn_max;
            if (want > (double)E) E = (int64_t)want;
        }
        all = cnt <= E;
        ne = cnt <= 0 ? 0 : (all ? cnt : E);
        rE = 1.0 / (double)E;
        qkey = (uint64_t)(A.qbase + q) << 32;
        qrow = A.Q + q * ix.d;
    }
    __device__ void load_vector(const DevIndex& ix) {
        if constexpr (C > 0) {
            const int lane = lane_id();
#pragma unroll
            for (int c = 0; c < C; ++c) {
                const int b = chunk_dim<XT>(lane & 7, c);
                qv[c].x = b < ix.d ? qrow[b] : 0.f;
                qv[c].y = b + 1 < ix.d ? qrow[b + 1] : 0.f;
                qv[c].z = b + 2 < ix.d ? qrow[b + 2] : 0.f;
                qv[c].w = b + 3 < ix.d ? qrow[b + 3] : 0.f;
            }
        }
    }
    // entry point j: every rank when the range holds at most E, else one
    // jittered rank per stratum
    __device__ int32_t entry_id(const SearchLaunch& A, int64_t j) const {
        if (all) return (int32_t)(l + j);
        const int64_t s0 = l + floor_div(j * cnt, E, rE);
        const int64_t t0 = l + floor_div((j + 1) * cnt, E, rE) - 1;
        const uint64_t z = splitmix64(A.seed ^ qkey ^ (uint64_t)j);
        return (int32_t)(s0 + (int64_t)(((z >> 32) * (uint64_t)(t0 - s0 + 1)) >> 32));
    }
    // whether an in-range rank is one of the query's entry points (then it is
    // in the visited set from the start)
    __device__ __forceinline__ bool is_entry(int32_t v) const {
        if (all) return true;
        return shared && (uint32_t)(splitmix64(pkey ^ (uint64_t)(uint32_t)v) >> 32) < T;
    }
    __device__ float eval(const DevIndex& ix, int nb, int32_t myid) const {
        if constexpr (C > 0) return eval_small<C, XT>(rows_of<XT>(ix), ix.dp, qv, nb, myid);
        else return eval_large(ix.X, ix.dp, qrow, ix.d, nb, myid);
    }
    __device__ float eval_batch(const DevIndex& ix, int nb, int32_t myid) const {
        if constexpr (C > 0) return eval_pipelined<C, XT>(rows_of<XT>(ix), ix.dp, qv, nb, myid);
        else return eval_large(ix.X, ix.dp, qrow, ix.d, nb, myid);
    }
};

// a3 (entry points, Alg. 2): evaluate entry points [e0, e1) of a query into
// a pool holding their L nearest.
template <int C, int LP, typename XT>
__device__ void entry_chunk(const DevIndex& ix, const SearchLaunch& A, const QueryCtx<C, XT>& Q, int64_t e0,
                            int64_t e1, Pool<LP>& pool, const WaveLds<LP>& W) {
    const int lane = lane_id();
#pragma unroll
    for (int s = 0; s < LP; ++s) { pool.key[s] = kEmpty; pool.flag[s] = 0u; }
    pool.np = 0;
    // 64 entry points per batch: one id per lane, one merge per batch
    for (int64_t b0 = e0; b0 < e1; b0 += 64) {
        const int nb = (int)(e1 - b0 < 64 ? e1 - b0 : 64);
        const int32_t id = lane < nb ? Q.entry_id(A, b0 + lane) : 0;
        const float dd = Q.eval_batch(ix, nb, id);
        const uint64_t nkey = lane < nb ? make_key(dd, id) : kEmpty;
        merge<LP>(pool, nkey, nb, A.L, W.st_key, W.st_flag);
    }
}

// a2, a4-a11 for one query whose pool holds the L nearest entry points:
// HotspotLocalization, the best-first loop of Alg. 2, output and statistics.
template <int C, int LP, typename XT>
__device__ void traverse(const DevIndex& ix, const SearchLaunch& A, int64_t gvis_words, const QueryCtx<C, XT>& Q,
                         Pool<LP>& pool, const WaveLds<LP>& W, const Visited& vis) {
    const int lane = lane_id();
    const int T = A.hash_log2 > 0 ? (1 << A.hash_log2) : 0;
    const int H = ix.H, m = ix.m, B = A.B, L = A.L, k = A.k;
    const int64_t qi = Q.qi, l = Q.l, r = Q.r;
    int32_t st[FROG_STAT_N];
#pragma unroll
    for (int i = 0; i < FROG_STAT_N; ++i) st[i] = 0;
    if (Q.ne > 0) {
    st[FROG_STAT_ENTRY] = (int32_t)Q.ne;
    st[FROG_STAT_DIST] = (int32_t)Q.ne;

    // a2: hotspot
    int Ls, Le;
    hotspot(l, r, H, ix.n, Ls, Le);
    Ls = uniform(Ls);
    Le = uniform(Le);
    if (A.hotspot_mode == 1) Le = H - 1;                   // ablation: no end condition
    if (A.hotspot_mode == 2) { Ls = 0; Le = H - 1; }       // ablation: no localisation
    st[FROG_STAT_LSTART] = Ls;
    st[FROG_STAT_LEND] = Le;

    // visited set: every entry point (exact bitmap) or the pool's
    // entry points (forgetful table: an entry point outside the pool
    // can never enter it later, its key is above the pool's L-th)
    if (vis.tab) {
        for (int i = lane; i < T; i += 64) vis.tab[i] = -1;
        wave_sync();
#pragma unroll
        for (int s = 0; s < LP; ++s)
            if (s * 64 + lane < pool.np) vis.insert((int32_t)(uint32_t)pool.key[s]);
    } else {
        for (int64_t i = lane; i < gvis_words; i += 64) vis.bits[i] = 0u;
        __threadfence_block();
        // entry points the membership test cannot tell
        if (!Q.shared && !Q.all)
            for (int64_t j = lane; j < Q.ne; j += 64) vis.insert(Q.entry_id(A, j));
        __threadfence_block();
    }
    wave_sync();

    // best-first loop (Alg. 2)
    const int64_t nent = (int64_t)(Le - Ls + 1) * m;
    int32_t* enbuf = W.enbuf;
    // The first 64 hotspot entries of the next unexpanded pool entry
    // are loaded while the current candidates are gathered; they are
    // used only if that entry is the one selected next.
    int32_t pre_u = -1;
    int32_t pre_v = -1;
    for (;;) {
        // a4: first unexpanded entry
        int sel = -1;
#pragma unroll
        for (int s = 0; s < LP; ++s) {
            const uint64_t mk = ballot(pool.flag[s] == 0u && pool.key[s] != kEmpty);
            if (sel < 0 && mk != 0) sel = s * 64 + __builtin_ctzll(mk);
        }
        sel = uniform(sel);
        if (sel < 0) break;
        const int ss = sel >> 6, sl = sel & 63;
        int32_t u = 0;
#pragma unroll
        for (int s = 0; s < LP; ++s) {
            if (s == ss) {
                u = (int32_t)(uint32_t)readlane64(pool.key[s], sl);
                if (lane == sl) pool.flag[s] = 1u;
            }
        }
        u = uniform(u);
        st[FROG_STAT_EXPANSIONS] += 1;

        // a5 + a6: ENC slice of the hotspot, compaction under budget B
        const int32_t* row = ix.ENC + ((int64_t)u * H + Ls) * m;
        const bool hit = u == pre_u;
        // next prefetch: the first unexpanded entry after u
        int nsel = -1;
#pragma unroll
        for (int s = 0; s < LP; ++s) {
            const uint64_t mk = ballot(pool.flag[s] == 0u && pool.key[s] != kEmpty);
            if (nsel < 0 && mk != 0) nsel = s * 64 + __builtin_ctzll(mk);
        }
        nsel = uniform(nsel);
        int32_t nu = -1;
#pragma unroll
        for (int s = 0; s < LP; ++s)
            if (s == (nsel >> 6) && nsel >= 0) nu = (int32_t)(uint32_t)readlane64(pool.key[s], nsel & 63);
        nu = uniform(nu);
        const int32_t cur_pre = pre_v;
        pre_u = nu;
        if (nu >= 0) {
            const int32_t* nrow = ix.ENC + ((int64_t)nu * H + Ls) * m;
            pre_v = lane < nent ? nrow[lane] : -1;
            st[FROG_STAT_LOADED] += (int32_t)(nent < 64 ? nent : 64);
        }
        int nen = 0;
        int64_t scanned = nent;
        for (int64_t off = 0; off < nent && nen < B; off += 64) {
            const int64_t e = off + lane;
            const int32_t v = (off == 0 && hit) ? cur_pre : (e < nent ? row[e] : -1);
            bool pred = v >= l && v <= r;
            if (A.eager) {
                // ablation: visited candidates are skipped here and do not
                // count against the budget; a repeat of an earlier lane's
                // candidate in this load is visited by then (exact set only)
                pred = pred && !Q.is_entry(v) && !vis.contains(v);
                for (uint64_t mm = ballot(pred); mm; mm &= mm - 1) {
                    const int j = __builtin_ctzll(mm);
                    if (lane > j && v == __builtin_amdgcn_readlane(v, j)) pred = false;
                }
            }
            const uint64_t pm = ballot(pred);
            const int rk = mbcnt(pm);
            const int tot = __popcll(pm);
            const int admit = tot < B - nen ? tot : B - nen;
            if (pred && rk < admit) {
                enbuf[nen + rk] = v;
                if (A.eager) vis.insert(v);
            }
            if (!(off == 0 && hit)) st[FROG_STAT_LOADED] += (int32_t)(nent - off < 64 ? nent - off : 64);
            if (admit == B - nen && admit > 0) {
                // budget reached: Alg. 4 examined every layer up to the
                // one holding the last admitted entry
                const int last = uniform(__builtin_ctzll(ballot(pred && rk == admit - 1)));
                scanned = ((off + last) / m + 1) * m;
            }
            nen += admit;
        }
        st[FROG_STAT_SCANNED] += (int32_t)scanned;
        nen = uniform(nen);
        st[FROG_STAT_EN] += nen;
        wave_sync();

        // a7: lazy visited check on the compacted list
        int32_t v = lane < nen ? enbuf[lane] : -1;
        bool fresh = false;
        if (lane < nen) fresh = A.eager || (!Q.is_entry(v) && vis.check_insert(v));
        const uint64_t fm = ballot(fresh);
        const int ns = __popcll(fm);
        wave_sync();
        if (fresh) enbuf[mbcnt(fm)] = v;
        wave_sync();
        const int32_t myid = lane < ns ? enbuf[lane] : 0;
        wave_sync();
        if (ns == 0) continue;

        // a8: gather + distances
        const float dd = Q.eval(ix, ns, myid);
        st[FROG_STAT_DIST] += ns;
        const uint64_t nkey = lane < ns ? make_key(dd, myid) : kEmpty;
        // a9 + a10: MergeTopEfS
        merge<LP>(pool, nkey, ns, L, W.st_key, W.st_flag);
    }
    }

    // a11: output, rank -> original id, padding
#pragma unroll
    for (int s = 0; s < LP; ++s) {
        const int p = s * 64 + lane;
        if (p < k) {
            int32_t oid = -1;
            float od = __int_as_float(0x7f800000);
            if (p < pool.np) {
                oid = ix.perm[(uint32_t)pool.key[s]];
                od = __uint_as_float((uint32_t)(pool.key[s] >> 32));
            }
            A.ids[qi * k + p] = oid;
            A.dists[qi * k + p] = od;
        }
    }
    // the traversal's columns; the shared scan's row count is written by the scan
    if (A.stats && lane < FROG_STAT_SCANROWS) {
        int32_t val = 0;
#pragma unroll
        for (int i = 0; i < FROG_STAT_SCANROWS; ++i)
            if (lane == i) val = st[i];
        A.stats[qi * FROG_STAT_N + lane] = val;
    }
}

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

template <int C, int LP, typename XT = float>
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
        traverse<C, LP, XT>(P.ix, P.a, P.gvis_words, Q, pool, W, vis);
        if (A.stats && lane == 0) A.stats[qi * FROG_STAT_N + FROG_STAT_SCANROWS] = 0;
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
        if (P.a.stats) P.a.stats[q * FROG_STAT_N + FROG_STAT_SCANROWS] = 0;
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

// per wave: 16 buffers of 2 kkeep keys, |q|^2 of the 16 queries, 16 list states
__host__ __device__ constexpr size_t s_scan_lds_per_wave(int kkeep) {
    return (size_t)kSQ * 2 * kkeep * 8 + kSQ * 4 + kSQ * 8;
}

// KT = dp / 16 float4 chunks of the query operand in registers (d <= 128);
// KT = 0 reloads it for every block (fp32 rows only).  XT is the rows'
// storage type: 16-bit rows are widened exactly to fp32 on load.
template <int KT, int KK, typename XT = float>
__global__ __launch_bounds__(kBlock) void s_scan_kernel(SParams P) {
    static_assert(sizeof(XT) == 4 || (KT > 0 && KT % 2 == 0), "16-bit rows need dp a multiple of 32 held in registers");
    using namespace topk;
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int lane = lane_id();
    const int wave = threadIdx.x >> 6;
    const int64_t item = (int64_t)blockIdx.x * (blockDim.x >> 6) + wave;
    const int64_t t = item / kSChunks;
    const int c = (int)(item % kSChunks);
    if (t >= P.tmax) return;        // wave-uniform; no workgroup barrier follows
    const STile& T = P.tiles[t];
    if (T.nq == 0) return;
    const SharedLevels& lv = P.a.lv;
    const int lev = T.lev;
    const int64_t len = (int64_t)T.ub - T.ua;
    const int64_t c0 = T.ua + len * c / kSChunks;
    const int64_t c1 = T.ua + len * (c + 1) / kSChunks;
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
    const int qrow = T.q[ii];
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
        qv[e] = T.q[sl] >= 0;
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
    auto rank_at = [&](int64_t blk) -> int32_t {
        const int64_t pos = pos_at(blk);
        return lranks ? lranks[pos] : (int32_t)pos;
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
    auto process = [&](const float4 (&x)[KT > 0 ? KT : 1], int32_t rk, uint32_t pri, float xn, int64_t blk) {
        const bool inrun = c0 + blk * 16 + ii < c1;
        make_room();
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
        const uint64_t below = (1ull << lane) - 1;
        // lane holds D[4kk + e][ii]: query slot 4kk + e, the block's row ii
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const bool insample = inrun && qv[e] && rk >= ql[e] && rk <= qr[e] && (qall[e] || pri < qT[e]);
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
    // two row buffers in turn: the loads of block b + 2 are issued as soon
    // as block b is multiplied, ranks two blocks ahead of their rows
    // (positions past the end are clamped to the last one, so the loads are
    // in bounds and unconditional: a load under a branch would make the
    // compiler wait for it, and for every load issued before it, at once)
    if (nblk > 0) {
        float4 xa[KT > 0 ? KT : 1], xb[KT > 0 ? KT : 1];
        load_rows(0, xa);
        int32_t ra = rank_at(0);
        uint32_t pa = lprio[pos_at(0)];
        float na = lnorm[pos_at(0)];
        load_rows(1, xb);
        int32_t rb = rank_at(1);
        uint32_t pb = lprio[pos_at(1)];
        float nb = lnorm[pos_at(1)];
        for (int64_t blk = 0; blk < nblk; blk += 2) {
            process(xa, ra, pa, na, blk);
            load_rows(blk + 2, xa);
            ra = rank_at(blk + 2);
            pa = lprio[pos_at(blk + 2)];
            na = lnorm[pos_at(blk + 2)];
            if (blk + 1 < nblk) process(xb, rb, pb, nb, blk + 1);
            load_rows(blk + 3, xb);
            rb = rank_at(blk + 3);
            pb = lprio[pos_at(blk + 3)];
            nb = lnorm[pos_at(blk + 3)];
        }
    }
    // the item's lists: entries kept, threshold, sample rows seen
    if (P.a.stats && lane == 0) {
        int first = 0;
        while (first < kSQ - 1 && T.q[first] < 0) ++first;
        atomicAdd(P.a.stats + (int64_t)T.q[first] * FROG_STAT_N + FROG_STAT_SCANROWS, (int32_t)(nblk * 16));
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
    const int64_t base = item * kSQ;
#pragma unroll
    for (int i = 0; i < kSQ; ++i) {
        buf_cut<kkeep>(list_of(i));
        const int fi = __builtin_amdgcn_readfirstlane(lst[2 * i]);
        const uint64_t* kb = lkey + (size_t)i * 2 * kkeep;
        for (int j = lane; j < fi; j += 64) {
            const uint64_t key = kb[j];
            P.pv[(base + i) * kkeep + j] = ord_value((uint32_t)(key >> 32));
            P.pr[(base + i) * kkeep + j] = (int32_t)(uint32_t)key;
        }
        if (lane == 0) {
            P.pthr[base + i] = __int_as_float(lst[2 * i + 1]);   // +inf unless a cut dropped rows
            P.pfill[base + i] = fi;
            P.pcnt[base + i] = (int32_t)scount[i];
        }
    }
}

// The pool of each query: one wavefront per query.
template <int C, int LP, int KK, typename XT = float>
__global__ __launch_bounds__(kBlock) void s_pool_kernel(SParams P) {
    using namespace topk;
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const DevIndex& ix = P.ix;
    const SearchLaunch& A = P.a;
    const int lane = lane_id();
    const int wave = threadIdx.x >> 6;
    WaveLds<LP> W(smem, P.lds_per_wave, 0);
    char* lbase = smem + (size_t)wave * P.lds_per_wave + P.lds_list;
    // KK: entries of each chunk list the scan left (their stride); the merged
    // list keeps kkeep >= 64 of them (an offer of 64 fits after a cut)
    constexpr int kkeep = KK > 64 ? KK : 64;
    const BufList Lst{reinterpret_cast<uint64_t*>(lbase), reinterpret_cast<int32_t*>(lbase + (size_t)2 * kkeep * 8)};
    const double u_round = 5.9604644775390625e-08;   // 2^-24

    {
        const int64_t qi = (int64_t)blockIdx.x * kWavesPerBlock + wave;
        if (qi >= A.nq) return;   // wave-uniform; no workgroup barrier follows
        const SPlan p = P.plan[qi];
        if (p.l > p.r) return;
        QueryCtx<C, XT> Q;
        Q.load(ix, A, P.lr, qi);
        Q.load_vector(ix);
        Q.shared = true;
        Q.T = p.T;
        Q.pkey = A.lv.key;

        // the kkeep smallest approximate distances over the tile's lists
        buf_init(Lst);
        const int64_t t = p.tslot / kSQ;
        const int slot = p.tslot % kSQ;
        float texcl = __int_as_float(0x7f800000);   // every row left out is at or above this
        // the chunks' fill, threshold and sample count in lanes 0..7, then
        // all their entries at once (no round trip between chunks)
        int mf = 0, mc = 0;
        float mt = __int_as_float(0x7f800000);
        if (lane < kSChunks) {
            const int64_t base = (t * kSChunks + lane) * kSQ + slot;
            mf = P.pfill[base];
            mt = P.pthr[base];
            mc = P.pcnt[base];
        }
        int64_t ne = 0;
#pragma unroll
        for (int o = 1; o < kSChunks; o <<= 1) {
            mc += __shfl_xor(mc, o);
            mt = fminf(mt, __shfl_xor(mt, o));
        }
        ne = uniform(mc);
        texcl = __int_as_float(uniform(__float_as_int(mt)));
        constexpr int kR = KK > 64 ? KK / 64 : 1;   // entries per lane and chunk
        float av[kSChunks][kR];
        int32_t rw[kSChunks][kR];
#pragma unroll
        for (int c = 0; c < kSChunks; ++c) {
            const int fi = __builtin_amdgcn_readlane(mf, c);
            const int64_t base = (t * kSChunks + c) * kSQ + slot;
#pragma unroll
            for (int r = 0; r < kR; ++r) {
                const int j = r * 64 + lane;
                av[c][r] = j < fi ? P.pv[base * KK + j] : __int_as_float(0x7f800000);
                rw[c][r] = j < fi ? P.pr[base * KK + j] : -1;
            }
        }
#pragma unroll
        for (int c = 0; c < kSChunks; ++c) {
#pragma unroll
            for (int r = 0; r < kR; ++r) {
                const uint64_t gm = ballot(rw[c][r] >= 0 && av[c][r] < __int_as_float(Lst.st[1]));
                if (gm) buf_offer<kkeep>(Lst, gm, av[c][r], rw[c][r]);
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
            const float dd = Q.eval_batch(ix, f, id);
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
                const float dd = Q.eval_batch(ix, nb, id);
                merge<LP>(pool, lane < nb ? make_key(dd, id) : kEmpty, nb, A.L, W.st_key, W.st_flag);
            }
        }
        // margin test: a row left out has exact distance >= texcl - eps
        bool certified = true;
        if (!(texcl == __int_as_float(0x7f800000))) {
            certified = false;
            if (pool.np >= A.L) {
                double qsq = 0.0;
                for (int cc = lane; cc < ix.d; cc += 64) qsq += (double)Q.qrow[cc] * (double)Q.qrow[cc];
#pragma unroll
                for (int o = 32; o >= 1; o >>= 1) qsq += __shfl_xor(qsq, o);
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
                const float dd = Q.eval_batch(ix, nb, id);
                merge<LP>(pool, lane < nb ? make_key(dd, id) : kEmpty, nb, A.L, W.st_key, W.st_flag);
            }
        }
#pragma unroll
        for (int s = 0; s < LP; ++s) P.pools[qi * 64 * LP + s * 64 + lane] = pool.key[s];
        if (lane == 0) P.pne[qi] = (int32_t)ne;
    }
}

// Traversal: persistent, one wavefront per query, from the pool s_pool_kernel wrote.
template <int C, int LP, typename XT = float>
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
        const int64_t qi = (int64_t)(uint32_t)uniform((int)__shfl((int)qq, 0));
        if (qi >= A.nq) break;
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
        Q.load(ix, A, P.lr, qi);
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
        traverse<C, LP, XT>(ix, A, P.gvis_words, Q, pool, W, vis);
    }
}


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


// ------------------------------------------------------------------ dispatch

using KernelFn = void (*)(KParams);

template <int C, typename XT = float>
KernelFn pick_lp(int L) {
    if (L <= 64) return coop_kernel<C, 1, XT>;
    if (L <= 128) return coop_kernel<C, 2, XT>;
    return coop_kernel<C, 4, XT>;
}

// fp16 rows come with dp = 64 or 128 (the upload checks it)
KernelFn pick_kernel(int dp, int L, int storage) {
    if (storage == FROG_STORAGE_F16) return dp == 64 ? pick_lp<2, __half>(L) : pick_lp<4, __half>(L);
    if (storage == FROG_STORAGE_BF16) return dp == 64 ? pick_lp<2, bf16x>(L) : pick_lp<4, bf16x>(L);
    switch (dp) {
        case 32: return pick_lp<1>(L);
        case 64: return pick_lp<2>(L);
        case 96: return pick_lp<3>(L);
        case 128: return pick_lp<4>(L);
        default: return pick_lp<0>(L);
    }
}

int lp_of(int L) { return L <= 64 ? 1 : (L <= 128 ? 2 : 4); }

int lds_per_wave(int L, int hash_log2) {
    const int lp = lp_of(L);
    return 64 * lp * 8 + 64 * lp * 4 + 64 * 4 + (hash_log2 > 0 ? (4 << hash_log2) : 0);
}

int max_blocks(KernelFn fn, int smem) {
    static std::mutex mu;
    static std::map<std::pair<void*, int>, int> cache;
    std::lock_guard<std::mutex> g(mu);
    auto key = std::make_pair((void*)fn, smem);
    auto it = cache.find(key);
    if (it != cache.end()) return it->second;
    int dev = 0, per_cu = 0, cus = 0;
    hipGetDevice(&dev);
    hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, (const void*)fn, kBlock, smem) != hipSuccess ||
        per_cu < 1)
        per_cu = 1;
    const int v = per_cu * (cus > 0 ? cus : 1);
    cache[key] = v;
    return v;
}


// candidates kept per query and work item: K >= L + 8, room for the margin
// (the C ABI refuses L > 248 in entry mode 1)
int shared_kkeep(int L) { return L + 8 <= 64 ? 64 : (L + 8 <= 128 ? 128 : 256); }
// the pool kernel's merged list: at least 64
int pool_kkeep(int kkeep) { return kkeep > 64 ? kkeep : 64; }

template <int C, typename XT = float>
void (*pick_s_pool_c(int L))(SParams) {
    const int kk = shared_kkeep(L);
    if (L <= 64) return kk == 64 ? s_pool_kernel<C, 1, 64, XT> : s_pool_kernel<C, 1, 128, XT>;
    if (L <= 128) return kk == 128 ? s_pool_kernel<C, 2, 128, XT> : s_pool_kernel<C, 2, 256, XT>;
    return s_pool_kernel<C, 4, 256, XT>;
}

template <int C, typename XT = float>
void (*pick_s_search_c(int L))(SParams) {
    if (L <= 64) return s_search_kernel<C, 1, XT>;
    if (L <= 128) return s_search_kernel<C, 2, XT>;
    return s_search_kernel<C, 4, XT>;
}

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

void (*pick_s_search(int dp, int L, int storage))(SParams) {
    if (storage == FROG_STORAGE_F16) return dp == 64 ? pick_s_search_c<2, __half>(L) : pick_s_search_c<4, __half>(L);
    if (storage == FROG_STORAGE_BF16) return dp == 64 ? pick_s_search_c<2, bf16x>(L) : pick_s_search_c<4, bf16x>(L);
    switch (dp) {
        case 32: return pick_s_search_c<1>(L);
        case 64: return pick_s_search_c<2>(L);
        case 96: return pick_s_search_c<3>(L);
        case 128: return pick_s_search_c<4>(L);
        default: return pick_s_search_c<0>(L);
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

void (*pick_s_scan(int dp, int kkeep, int storage))(SParams) {
    if (kkeep == 64) return pick_s_scan_k<64>(dp, storage);
    if (kkeep == 128) return pick_s_scan_k<128>(dp, storage);
    return pick_s_scan_k<256>(dp, storage);
}

// entry_mode 1: plan, group, scan on the matrix cores, then search
int launch_shared(const DevIndex& ix, const SearchLaunch& a, hipStream_t stream) {
    const int kkeep = shared_kkeep(a.L);
    auto sfn = pick_s_search(ix.dp, a.L, ix.storage);
    auto pfn = pick_s_pool(ix.dp, a.L, ix.storage);
    // search kernel: pool staging, EN list and visited table per wave
    const int lps = lds_per_wave(a.L, a.hash_log2);
    const int smem = lps * kWavesPerBlock;
    // pool kernel: pool staging and EN list, then the re-rank list
    const int base_lds = lds_per_wave(a.L, 0);
    const int lpw = base_lds + 2 * pool_kkeep(kkeep) * 8 + 16;
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
    int blocks = max_blocks((KernelFn)sfn, smem);
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
    void* wsp = nullptr;
    hipError_t e = hipMallocAsync(&wsp, off, stream);
    if (e != hipSuccess) return fail(e == hipErrorOutOfMemory ? FROG_ENOMEM : FROG_EHIP, "workspace: %s", hipGetErrorString(e));
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
    (void)hipFreeAsync(wsp, stream);
    if (e != hipSuccess) return fail(FROG_EHIP, "search launch: %s", hipGetErrorString(e));
    return FROG_OK;
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
    hipStream_t stream = (hipStream_t)stream_v;
    if (a.entry_mode == 1) return launch_shared(ix, a, stream);
    const KernelFn fn = pick_kernel(ix.dp, a.L, ix.storage);
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
    int blocks = max_blocks(fn, smem);
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
    void* wsp = nullptr;
    hipError_t e = hipMallocAsync(&wsp, ws, stream);
    if (e != hipSuccess) return fail(e == hipErrorOutOfMemory ? FROG_ENOMEM : FROG_EHIP, "workspace: %s", hipGetErrorString(e));
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
    (void)hipFreeAsync(wsp, stream);
    if (e != hipSuccess) return fail(FROG_EHIP, "search launch: %s", hipGetErrorString(e));
    return FROG_OK;
}

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
    hipError_t e = hipMallocAsync(&ws, bytes, stream);
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
    (void)hipFreeAsync(ws, stream);
    // the host arrays must outlive the copies
    const hipError_t e2 = hipStreamSynchronize(stream);
    if (e != hipSuccess || e2 != hipSuccess)
        return fail(FROG_EHIP, "exact ranges: %s", hipGetErrorString(e != hipSuccess ? e : e2));
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
