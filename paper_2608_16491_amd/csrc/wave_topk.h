// Per-query lists of the smallest (approximate distance, row) pairs, kept by
// one wavefront in LDS.  The matrix-core scans (the brute force and the
// shared entry sample of the search) offer each query's candidates of a
// 16-row block to its list; a full list holds its largest value as the
// threshold a candidate has to beat.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

namespace frog {
namespace topk {

__device__ __forceinline__ void list_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// The minimum of mn and the maximum of mx over the wavefront, uniform (every
// lane active): data-parallel-primitive moves within each row of 16 lanes
// (quad swaps, half-row and row mirrors), then the four rows' results.
__device__ __forceinline__ void wave_minmax_u32(uint32_t& mn, uint32_t& mx) {
    auto step = [&](auto ctrl) {
        constexpr int c = decltype(ctrl)::value;
        const uint32_t a = (uint32_t)__builtin_amdgcn_mov_dpp((int)mn, c, 0xF, 0xF, false);
        const uint32_t b = (uint32_t)__builtin_amdgcn_mov_dpp((int)mx, c, 0xF, 0xF, false);
        mn = a < mn ? a : mn;
        mx = b > mx ? b : mx;
    };
    step(std::integral_constant<int, 0xB1>{});
    step(std::integral_constant<int, 0x4E>{});
    step(std::integral_constant<int, 0x141>{});
    step(std::integral_constant<int, 0x140>{});
    uint32_t rmn = (uint32_t)__builtin_amdgcn_readlane((int)mn, 0), rmx = (uint32_t)__builtin_amdgcn_readlane((int)mx, 0);
#pragma unroll
    for (int r = 16; r < 64; r += 16) {
        const uint32_t a = (uint32_t)__builtin_amdgcn_readlane((int)mn, r);
        const uint32_t b = (uint32_t)__builtin_amdgcn_readlane((int)mx, r);
        rmn = a < rmn ? a : rmn;
        rmx = b > rmx ? b : rmx;
    }
    mn = rmn;
    mx = rmx;
}

__device__ __forceinline__ float wave_max_pos(float v, int& pos) {
    // max over the wavefront with the lowest position among equals
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const float ov = __shfl_xor(v, o);
        const int op = __shfl_xor(pos, o);
        if (ov > v || (ov == v && op < pos)) { v = ov; pos = op; }
    }
    return v;
}

// A list of at most `cap` (approximate distance, row) pairs in LDS (cap a
// multiple of 64) and its state, also in LDS: the number of entries, and once
// the list is full, the value and slot of its largest entry (the threshold a
// new candidate has to beat).  Every row offered to the list and not kept has
// a value at or above the final threshold.
struct TopList {
    float* v;
    int32_t* r;
    int32_t* st;   // [0] fill, [1] threshold (float bits), [2] slot of the largest
};

__device__ __forceinline__ float list_threshold(const int32_t* st) { return __int_as_float(st[1]); }

// recompute the largest entry of a full list (all lanes)
__device__ __forceinline__ void list_refresh(const TopList& Lst, int cap, float& thr, int& mpos) {
    const int lane = __lane_id();
    float best = Lst.v[lane];
    int pos = lane;
    for (int j = 64 + lane; j < cap; j += 64)
        if (Lst.v[j] > best) { best = Lst.v[j]; pos = j; }
    best = wave_max_pos(best, pos);
    thr = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(best)));
    mpos = __builtin_amdgcn_readfirstlane(pos);
}

// Offer the candidates held by the lanes of `group_mask` (value a, row rw in
// each such lane) to the list.  Returns true if a candidate was dropped or an
// entry evicted.
static __device__ __noinline__ bool offer(TopList Lst, int cap, uint64_t group_mask, float a, int32_t rw) {
    const int lane = __lane_id();
    int f = __builtin_amdgcn_readfirstlane(Lst.st[0]);
    float thr = __int_as_float(__builtin_amdgcn_readfirstlane(Lst.st[1]));
    int mpos = __builtin_amdgcn_readfirstlane(Lst.st[2]);
    bool dropped = false;
    const int c = __popcll(group_mask);
    if (f + c <= cap) {
        // room for all: append in parallel
        if ((group_mask >> lane) & 1) {
            const int pos = f + __popcll(group_mask & ((1ull << lane) - 1));
            Lst.v[pos] = a;
            Lst.r[pos] = rw;
        }
        f += c;
        list_sync();
        if (f == cap) list_refresh(Lst, cap, thr, mpos);
    } else {
        for (uint64_t m = group_mask; m; m &= m - 1) {
            const int src = __builtin_ctzll(m);
            const float av = __shfl(a, src);
            const int32_t rv = __shfl(rw, src);
            if (f < cap) {
                if (lane == 0) { Lst.v[f] = av; Lst.r[f] = rv; }
                ++f;
                list_sync();
                if (f == cap) list_refresh(Lst, cap, thr, mpos);
                continue;
            }
            dropped = true;   // av itself, or the entry it evicts
            if (!(av < thr)) continue;
            if (lane == 0) { Lst.v[mpos] = av; Lst.r[mpos] = rv; }
            list_sync();
            list_refresh(Lst, cap, thr, mpos);
        }
    }
    if (lane == 0) {
        Lst.st[0] = f;
        Lst.st[1] = __float_as_int(thr);
        Lst.st[2] = mpos;
    }
    list_sync();
    return dropped;
}

// Buffered variant for long streams: up to 2K keys (orderable float bits of
// the value << 32 | row) in LDS.  Candidates below the threshold are
// appended; a buffer about to overflow is cut to its K smallest (K-th value
// found by bisection over the value bits, kept entries compacted in place),
// whose largest value becomes the threshold (+inf until the first cut).
// Every candidate offered and not kept has a value at or above the final
// threshold.
struct BufList {
    uint64_t* key;   // [2K]
    int32_t* st;     // [0] fill, [1] threshold (float bits)
};

__device__ __forceinline__ uint32_t ord_bits(float v) {
    const uint32_t b = __float_as_uint(v);
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ float ord_value(uint32_t o) {
    return __uint_as_float((o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o);
}

__device__ __forceinline__ void buf_init(const BufList& B) {
    if (__lane_id() == 0) {
        B.st[0] = 0;
        B.st[1] = 0x7f800000;
    }
    list_sync();
}

// Cut the buffer: with exact = true keep its K smallest entries (all if
// there are at most K); with exact = false keep every entry at or below some
// value x with K <= #kept <= 5K/4 (a cheaper search; the exact cut when ties
// leave no such x).  The bisection over the value bits stops at the first x
// that qualifies (for the exact cut: exactly K entries at or below x), so it
// rarely runs to a single value.  The new threshold is at or below the value
// of every dropped entry.  K is 32, 48, 64, 128 or 256.
template <int K>
__device__ __forceinline__ void buf_cut(const BufList& B, bool exact = true) {
    constexpr int R = (2 * K + 63) / 64;   // entries per lane (the last register partly)
    const int lane = __lane_id();
    const int f = __builtin_amdgcn_readfirstlane(B.st[0]);
    if (f <= K) return;
    uint64_t k[R];
    uint32_t vmin = 0xFFFFFFFFu, vmax = 0u;
#pragma unroll
    for (int i = 0; i < R; ++i) {
        k[i] = i * 64 + lane < f ? B.key[i * 64 + lane] : ~0ull;
        const uint32_t v = (uint32_t)(k[i] >> 32);
        if (i * 64 + lane < f) {
            vmin = v < vmin ? v : vmin;
            vmax = v > vmax ? v : vmax;
        }
    }
    wave_minmax_u32(vmin, vmax);
    // an x in [vmin, vmax] with #(entries <= x) equal to K (exact) or in
    // [K, 5K/4] (loose); failing that, the smallest x with #(entries <= x) >= K
    uint32_t lo = __builtin_amdgcn_readfirstlane(vmin), hi = __builtin_amdgcn_readfirstlane(vmax);
    int cx = f;
    bool loose = false;
    while (lo < hi) {
        const uint32_t mid = lo + ((hi - lo) >> 1);
        int c = 0;
#pragma unroll
        for (int i = 0; i < R; ++i) c += __popcll(__ballot((uint32_t)(k[i] >> 32) <= mid));
        if (c < K) {
            lo = mid + 1;
        } else {
            hi = mid;
            cx = c;
            // keeping every entry <= mid is the cut asked for
            if (c <= (exact ? K : K + K / 4)) {
                loose = true;
                break;
            }
        }
    }
    const uint32_t vk = hi;
    if (!exact && !loose) {
        int c = 0;
#pragma unroll
        for (int i = 0; i < R; ++i) c += __popcll(__ballot((uint32_t)(k[i] >> 32) <= vk));
        cx = c;
        loose = c <= K + K / 4;
    }
    list_sync();
    const uint64_t lt = (1ull << lane) - 1;
    if (loose) {
        // keep every entry <= vk; a dropped entry is above vk
        int wr = 0;
#pragma unroll
        for (int i = 0; i < R; ++i) {
            const bool keep = (uint32_t)(k[i] >> 32) <= vk;
            const uint64_t mk = __ballot(keep);
            if (keep) B.key[wr + __popcll(mk & lt)] = k[i];
            wr += __popcll(mk);
        }
        if (lane == 0) {
            B.st[0] = cx;
            B.st[1] = (int32_t)__float_as_uint(ord_value(vk + 1u));
        }
    } else {
        // entries below vk, then entries equal to vk up to K in all
        int below = 0;
#pragma unroll
        for (int i = 0; i < R; ++i) below += __popcll(__ballot((uint32_t)(k[i] >> 32) < vk));
        int wr = 0, eq = 0;
#pragma unroll
        for (int i = 0; i < R; ++i) {
            const uint32_t v = (uint32_t)(k[i] >> 32);
            const uint64_t mb = __ballot(v < vk);
            const uint64_t me = __ballot(v == vk);
            if (v < vk) B.key[wr + __popcll(mb & lt)] = k[i];
            if (v == vk) {
                const int pos = below + eq + __popcll(me & lt);
                if (pos < K) B.key[pos] = k[i];
            }
            wr += __popcll(mb);
            eq += __popcll(me);
        }
        if (lane == 0) {
            B.st[0] = K;
            B.st[1] = (int32_t)__float_as_uint(ord_value(vk));
        }
    }
    list_sync();
}

// Append the candidates of the lanes in gm (value a, row rw), all of them
// below the current threshold; at most 64 of them, so K >= 64 leaves room
// after a cut.
template <int K>
__device__ __forceinline__ void buf_offer(const BufList& B, uint64_t gm, float a, int32_t rw) {
    const int lane = __lane_id();
    int f = __builtin_amdgcn_readfirstlane(B.st[0]);
    if (f + __popcll(gm) > 2 * K) {
        buf_cut<K>(B, false);
        f = __builtin_amdgcn_readfirstlane(B.st[0]);
        if (f + __popcll(gm) > 2 * K) {   // a loose cut can leave 5K/4: make room for 64
            buf_cut<K>(B, true);
            f = __builtin_amdgcn_readfirstlane(B.st[0]);
        }
        const float thr = __int_as_float(__builtin_amdgcn_readfirstlane(B.st[1]));
        gm &= __ballot(a < thr);
    }
    if ((gm >> lane) & 1) B.key[f + __popcll(gm & ((1ull << lane) - 1))] = ((uint64_t)ord_bits(a) << 32) | (uint32_t)rw;
    if (lane == 0) B.st[0] = f + __popcll(gm);
    list_sync();
}

}  // namespace topk
}  // namespace frog
