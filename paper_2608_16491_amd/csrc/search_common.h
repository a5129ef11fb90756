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
//     vector, a per-lane sum over its chunks and a 64-lane sum.  No matrix
//     cores: every gathered vector is used once;
//   - MergeTopEfS: a new key's position is (# pool keys below it) + (# new
//     keys below it), counted with ballots; a pool key's position is its slot
//     plus (# new keys below it); entries scatter through LDS.  Keys are
//     unique once duplicates are dropped, so this equals sorting the union.
//
// This header holds what the search translation units share (wave helpers,
// distances, the pool and its merge, the visited table, the query context and
// the traversal); each kernel family is compiled in its own unit.
#pragma once
#pragma clang diagnostic ignored "-Wunused-function"

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <cstdint>
#include <map>
#include <tuple>
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

// The values of the lanes in `mask`, moved to lanes 0 .. popc(mask) - 1 in
// lane order (a forward permute: every lane sends its value to a distinct
// lane, the others after the selected ones).
__device__ __forceinline__ int32_t compact_lanes(int32_t v, uint64_t mask) {
    const int lane = __lane_id();
    const int below = mbcnt(mask);
    const int dst = ((mask >> lane) & 1ull) ? below : __popcll(mask) + (lane - below);
    return __builtin_amdgcn_ds_permute(dst << 2, v);
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

// Squared L2 of up to `cnt` (1..64) candidates; lane j holds candidate j's
// rank in `myid` and receives its distance in the return value (lanes from
// cnt on receive an unspecified value).  The query's float4 chunks this lane
// needs are in qv.  Lanes of a group past cnt read candidate cnt - 1 again,
// so that every load is issued by every lane: a load under a lane predicate
// is split off into a branch of its own, with a wait of its own.
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
        const int id = __shfl(myid, (j < cnt ? j : cnt - 1) & 63);
        float4 x[C];
        load_row<C, XT>(X, dp, id, sub, true, x);
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

// Same result as eval_small for the entry-point batches (1..64 candidates),
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
            const int id = __shfl(myid, (j < cnt ? j : cnt - 1) & 63);
            load_row<C, XT>(X, dp, id, sub, true, x[g]);
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

// The sum over all 64 lanes, the same value in every lane: each row of 16
// by quad swaps [1,0,3,2], [2,3,0,1] and the half-row and row mirrors, then
// the four rows' sums in a fixed order.
__device__ __forceinline__ double sum64(double s) {
    s = sum8(s);
    s += dpp_f64<0x140>(s);
    const double r0 = __longlong_as_double(((long long)(uint32_t)__builtin_amdgcn_readlane((int)(__double_as_longlong(s) >> 32), 0) << 32) |
                                           (uint32_t)__builtin_amdgcn_readlane((int)__double_as_longlong(s), 0));
    const double r1 = __longlong_as_double(((long long)(uint32_t)__builtin_amdgcn_readlane((int)(__double_as_longlong(s) >> 32), 16) << 32) |
                                           (uint32_t)__builtin_amdgcn_readlane((int)__double_as_longlong(s), 16));
    const double r2 = __longlong_as_double(((long long)(uint32_t)__builtin_amdgcn_readlane((int)(__double_as_longlong(s) >> 32), 32) << 32) |
                                           (uint32_t)__builtin_amdgcn_readlane((int)__double_as_longlong(s), 32));
    const double r3 = __longlong_as_double(((long long)(uint32_t)__builtin_amdgcn_readlane((int)(__double_as_longlong(s) >> 32), 48) << 32) |
                                           (uint32_t)__builtin_amdgcn_readlane((int)__double_as_longlong(s), 48));
    return (r0 + r1) + (r2 + r3);
}

// d > 128: all 64 lanes read one vector, float4 chunk lane + 64c, the
// differences and squares in double, summed over the lane's chunks in order
// and then over the wavefront by sum64.  Rows of up to 1024 padded
// dimensions (4 chunks per lane) keep the query's chunks in registers for
// the call and issue a candidate's four loads together (a chunk past the
// row reads the row's last chunk, its terms zeroed), two candidates in
// flight.
// Wider rows loop over their chunks.  Lane j < cnt receives candidate j's
// distance; lanes from cnt on receive an unspecified value.
__device__ float eval_large(const float* __restrict__ X, int dp, const float* __restrict__ q, int d, int cnt,
                            int32_t myid) {
    const int lane = lane_id();
    const float4* __restrict__ X4 = reinterpret_cast<const float4*>(X);
    const int dp4 = dp >> 2;
    float mine = 0.f;
    if (dp4 <= 4 * 64) {
        // the query's chunks are read per call: hoisted out of a caller's
        // loop they would hold 16 registers across it
        const float* qq = q;
        asm volatile("" : "+v"(qq));
        float4 qc[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int b = 4 * (lane + 64 * i);
            float e[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const float v = qq[b + t < d ? b + t : d - 1];
                e[t] = b + t < d ? v : 0.f;
            }
            qc[i] = make_float4(e[0], e[1], e[2], e[3]);
        }
        auto part = [&](const float4 (&x)[4]) {
            double s = 0.0;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const bool in = lane + 64 * i < dp4;
                // keep the query in fp32 registers: convert per use, not once
                float4 qf = qc[i];
                asm volatile("" : "+v"(qf.x), "+v"(qf.y), "+v"(qf.z), "+v"(qf.w));
                const double q0 = qf.x, q1 = qf.y, q2 = qf.z, q3 = qf.w;
                double t, u = 0.0;
                t = q0 - (double)x[i].x; u += t * t;
                t = q1 - (double)x[i].y; u += t * t;
                t = q2 - (double)x[i].z; u += t * t;
                t = q3 - (double)x[i].w; u += t * t;
                s += in ? u : 0.0;
            }
            return s;
        };
        // two candidates in flight: the next one's loads are issued before
        // the current one's are used (a round past cnt reads candidate
        // cnt - 1 again), so consecutive waits overlap
        auto load = [&](int j, float4 (&x)[4]) {
            const int64_t id = __builtin_amdgcn_readlane(myid, j < cnt ? j : cnt - 1);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int c = lane + 64 * i < dp4 ? lane + 64 * i : dp4 - 1;
                x[i] = X4[id * dp4 + c];
            }
        };
        float4 xa[4], xb[4];
        load(0, xa);
        for (int j = 0; j < cnt; j += 2) {
            load(j + 1, xb);
            const double sa = sum64(part(xa));
            if (lane == j) mine = (float)sa;
            load(j + 2, xa);
            const double sb = sum64(part(xb));
            if (lane == j + 1) mine = (float)sb;
        }
        return mine;
    }
    for (int j = 0; j < cnt; ++j) {
        const int id = __builtin_amdgcn_readlane(myid, j);
        double s = 0.0;
        for (int c = lane; c < dp4; c += 64) {
            const float4 x = X4[(int64_t)id * dp4 + c];
            const int b = 4 * c;
            const double q0 = b < d ? q[b] : 0.f, q1 = b + 1 < d ? q[b + 1] : 0.f;
            const double q2 = b + 2 < d ? q[b + 2] : 0.f, q3 = b + 3 < d ? q[b + 3] : 0.f;
            double t, u = 0.0;
            t = q0 - (double)x.x; u += t * t;
            t = q1 - (double)x.y; u += t * t;
            t = q2 - (double)x.z; u += t * t;
            t = q3 - (double)x.w; u += t * t;
            s += u;
        }
        s = sum64(s);
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
    const uint64_t cmask = ballot(cand);
    if (cmask == 0) return 0;
    // one pass over the candidates in lane order: a candidate equal to a
    // pool key or to an earlier candidate is dropped (so the first of equal
    // candidates is kept unless the pool holds it); a kept one counts the
    // pool keys below it (its place among the pool), and every lane counts
    // the kept candidates below its pool keys (their shift) and below its
    // own candidate (its place among the new keys)
    uint64_t kmask = cmask;
    int ltN = 0, cntP = 0;
    int ltP[LP];
#pragma unroll
    for (int s = 0; s < LP; ++s) ltP[s] = 0;
    for (uint64_t m = cmask; m; m &= m - 1) {
        const int j = __builtin_ctzll(m);
        const uint64_t kj = readlane64(nkey, j);
        bool inpool = false;
        int c = 0;
#pragma unroll
        for (int s = 0; s < LP; ++s) {
            inpool |= ballot(P.key[s] == kj) != 0;
            c += __popcll(ballot(P.key[s] < kj));
        }
        const bool earlier = (ballot(cand && nkey == kj) & ((1ull << j) - 1)) != 0;
        if (inpool || earlier) {
            kmask &= ~(1ull << j);
            continue;
        }
#pragma unroll
        for (int s = 0; s < LP; ++s) ltP[s] += kj < P.key[s] ? 1 : 0;
        if (lane == j) cntP = c;
        ltN += kj < nkey ? 1 : 0;
    }
    const int nk = __popcll(kmask);
    if (nk == 0) return 0;
    const bool keep = (kmask >> lane) & 1ull;
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
        set(ix, A, q, uniform(lr[2 * q]), uniform(lr[2 * q + 1]));
    }
    // the same from a rank interval already at hand
    __device__ void set(const DevIndex& ix, const SearchLaunch& A, int64_t q, int64_t l_, int64_t r_) {
        qi = q;
        l = l_;
        r = r_;
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
// LEAN: the timed configuration (no statistics, lazy check, LDS visited
// table), with the statistics and the ablation branches compiled out and the
// EN list compacted by lane permutes whenever the slice's first 64 entries
// hold it (almost always: the budget fills within about 40 entries at the
// bench settings); the trajectory is the same.
template <int C, int LP, typename XT, bool LEAN = false>
__device__ void traverse(const DevIndex& ix, const SearchLaunch& A, int64_t gvis_words, const QueryCtx<C, XT>& Q,
                         Pool<LP>& pool, const WaveLds<LP>& W, const Visited& vis) {
    const int lane = lane_id();
    const int T = A.hash_log2 > 0 ? (1 << A.hash_log2) : 0;
    const int H = ix.H, m = ix.m, B = A.B, L = A.L, k = A.k;
    const int64_t qi = Q.qi, l = Q.l, r = Q.r;
    const int32_t l32 = (int32_t)l, r32 = (int32_t)r;   // ranks fit int32
    const bool eager = !LEAN && A.eager;
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
        // a4: first unexpanded entry, and the one after it (the prefetch's
        // guess at the next selection), from one ballot per register
        int sel = -1, nsel = -1;
#pragma unroll
        for (int s = 0; s < LP; ++s) {
            uint64_t mk = ballot(pool.flag[s] == 0u && pool.key[s] != kEmpty);
            if (sel < 0 && mk != 0) {
                sel = s * 64 + __builtin_ctzll(mk);
                mk &= mk - 1;
            }
            if (nsel < 0 && sel >= 0 && mk != 0) nsel = s * 64 + __builtin_ctzll(mk);
        }
        sel = uniform(sel);
        if (sel < 0) break;
        nsel = uniform(nsel);
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
        int32_t nu = -1;
#pragma unroll
        for (int s = 0; s < LP; ++s)
            if (s == (nsel >> 6) && nsel >= 0) nu = (int32_t)(uint32_t)readlane64(pool.key[s], nsel & 63);
        nu = uniform(nu);
        // The slice's first 64 entries (loaded on a miss) are issued before
        // the prefetch, and the prefetch is issued on every hop (a valid row
        // when there is no guess) with every lane active, its lanes past the
        // slice masked where it is used: the loads in flight are then the same
        // on every path, and waiting for the slice leaves the prefetch in
        // flight (the wait counter retires loads in order; an optional load
        // makes the wait drain them all).  The previous prefetch is not read
        // after the next one is issued, so the two share a register.
        const int lidx = lane < nent ? lane : 0;
        int32_t x = pre_v;
        if (!hit) x = row[lidx];
        pre_u = nu;
        pre_v = ix.ENC[((int64_t)(nu >= 0 ? nu : u) * H + Ls) * m + lidx];
        if (nu >= 0) st[FROG_STAT_LOADED] += (int32_t)(nent < 64 ? nent : 64);
        const int32_t v0 = lane < nent ? x : -1;
        if (LEAN) {
            // the first 64 entries of the hotspot slice (the prefetched ones
            // on a hit); when they hold the whole slice or at least B
            // in-range entries, the EN list of Alg. 4 (the first B in-range
            // entries in stored order) lies in them: admit those, move them
            // to lanes 0.., check them against the visited table (lazy
            // check) and move the fresh ones down.  Otherwise the general
            // path below scans on.
            const bool inr = v0 >= l32 && v0 <= r32;
            const uint64_t pm = ballot(inr);
            const int tot = __popcll(pm);
            if (nent <= 64 || tot >= B) {
                const int nen = tot < B ? tot : B;
                const uint64_t am = ballot(inr && mbcnt(pm) < nen);
                const int32_t v = compact_lanes(v0, am);
                const bool fresh = lane < nen && !Q.is_entry(v) && vis.check_insert(v);
                const uint64_t fm = ballot(fresh);
                const int ns = __popcll(fm);
                if (ns == 0) continue;
                const int32_t myid = compact_lanes(v, fm);
                const float dd = Q.eval(ix, ns, lane < ns ? myid : 0);
                merge<LP>(pool, lane < ns ? make_key(dd, myid) : kEmpty, ns, L, W.st_key, W.st_flag);
                continue;
            }
        }
        int nen = 0;
        int64_t scanned = nent;
        for (int64_t off = 0; off < nent && nen < B; off += 64) {
            const int64_t e = off + lane;
            const int32_t v = off == 0 ? v0 : (e < nent ? row[e] : -1);
            bool pred = v >= l && v <= r;
            if (eager) {
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
                if (eager) vis.insert(v);
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
        if (lane < nen) fresh = eager || (!Q.is_entry(v) && vis.check_insert(v));
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
    if (!LEAN && A.stats && lane < FROG_STAT_SCANROWS) {
        int32_t val = 0;
#pragma unroll
        for (int i = 0; i < FROG_STAT_SCANROWS; ++i)
            if (lane == i) val = st[i];
        A.stats[qi * FROG_STAT_N + lane] = val;
    }
}

inline int lp_of(int L) { return L <= 64 ? 1 : (L <= 128 ? 2 : 4); }

inline int lds_per_wave(int L, int hash_log2) {
    const int lp = lp_of(L);
    return 64 * lp * 8 + 64 * lp * 4 + 64 * 4 + (hash_log2 > 0 ? (4 << hash_log2) : 0);
}

// workgroups of kernel `fn` (`threads` threads, `smem` bytes of LDS) the
// whole device holds at once
inline int max_blocks(const void* fn, int smem, int threads = kBlock) {
    static std::mutex mu;
    static std::map<std::tuple<const void*, int, int>, int> cache;
    std::lock_guard<std::mutex> g(mu);
    auto key = std::make_tuple(fn, smem, threads);
    auto it = cache.find(key);
    if (it != cache.end()) return it->second;
    int dev = 0, per_cu = 0, cus = 0;
    (void)hipGetDevice(&dev);
    (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, threads, smem) != hipSuccess || per_cu < 1)
        per_cu = 1;
    const int v = per_cu * (cus > 0 ? cus : 1);
    cache[key] = v;
    return v;
}

}  // namespace
}  // namespace frog
