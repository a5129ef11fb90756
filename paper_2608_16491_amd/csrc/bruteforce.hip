// Exhaustive filtered k-NN (Def. 2 of the paper) on gfx950, used as ground
// truth for the approximate search.
//
//   1. Host: each query's rank interval [l, r] (Sec 4) from the index's host
//      copy of the sorted attributes; queries are grouped into tiles of 16
//      with the same octave of range size, ordered by l, so a tile's rows are
//      the union of 16 overlapping intervals.
//   2. Device, one workgroup (4 wavefronts) per tile: the dot products of the
//      16 queries with 16-row blocks of X run on the fp32 matrix cores
//      (v_mfma_f32_16x16x4_f32, K = 4 per instruction); the approximate
//      squared distance |q|^2 + |x|^2 - 2 q.x masks rows outside each query's
//      own interval.  Each wavefront keeps, per query, the K' = 64 smallest
//      approximate distances it has seen (threshold test, then replace-max).
//   3. Device, same workgroup: the up-to 4 K' candidates of each query are
//      re-ranked with the exact canonical distance (double accumulation,
//      rounded once to float), and the k smallest (distance, rank) kept.
//      Every row a wavefront did not keep has an approximate distance at or
//      above that wavefront's final threshold; if the smallest such threshold
//      minus the approximation bound exceeds the k-th exact distance, the
//      result is certified exact (reported per query).
//
// The approximation bound: with unit roundoff u = 2^-24, fp32 |q|^2 and |x|^2
// (d terms each), the fp32 dot product (d products) and the final two
// operations err by at most (2d + 4) u (|q|^2 + |x|^2); the kernel uses twice
// that with |x|^2 replaced by the largest squared norm in the index.
//
// The host step reads the query ranges back, so this entry point synchronises
// `stream` once; it is a ground-truth tool, not the search path.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <vector>

#include "frog_internal.h"

namespace frog {
namespace {

constexpr int kQT = 16;       // queries per tile
constexpr int kKeep = 64;     // approximate candidates kept per query per wavefront
constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;

typedef float floatx4 __attribute__((ext_vector_type(4)));

struct Tile {
    int32_t q[kQT];   // query index, -1 = unused
    int32_t l[kQT];
    int32_t r[kQT];
    int32_t ul, ur;   // union of the intervals
};

struct BFParams {
    const float* X;       // [n][dp]
    const int32_t* perm;
    int64_t n;
    int d, dp;
    const float* Q;       // [nq][d]
    const Tile* tiles;
    int k;
    float maxnorm;        // largest |x|^2 in the index
    int32_t* ids;
    float* dists;
    int32_t* cert;
};

__device__ __forceinline__ int lane_id() { return __lane_id(); }

__device__ __forceinline__ float wave_max_pos(float v, int& pos) {
    // max over the wavefront with the lowest lane among equals
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const float ov = __shfl_xor(v, o);
        const int op = __shfl_xor(pos, o);
        if (ov > v || (ov == v && op < pos)) { v = ov; pos = op; }
    }
    return v;
}

__global__ __launch_bounds__(kThreads) void bf_tile_kernel(BFParams P) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const Tile& T = P.tiles[blockIdx.x];
    const int lane = lane_id();
    const int wave = threadIdx.x >> 6;
    const int dp = P.dp;
    // LDS: queries [16][dp] floats, |q|^2 [16], per wave: lists [16][kKeep]
    // (approx float, row int), thresholds [16], fill counts [16], max slot [16]
    float* Qs = reinterpret_cast<float*>(smem);
    float* qn = Qs + kQT * dp;
    char* wb = reinterpret_cast<char*>(qn + kQT) + (size_t)wave * (kQT * kKeep * 8 + kQT * 12);
    float* lv = reinterpret_cast<float*>(wb);
    int32_t* lr = reinterpret_cast<int32_t*>(lv + kQT * kKeep);
    float* thr = reinterpret_cast<float*>(lr + kQT * kKeep);
    int32_t* fill = reinterpret_cast<int32_t*>(thr + kQT);
    int32_t* mpos = fill + kQT;

    for (int i = threadIdx.x; i < kQT * dp; i += kThreads) {
        const int qi = i / dp, c = i % dp;
        const int q = T.q[qi];
        Qs[i] = (q >= 0 && c < P.d) ? P.Q[(int64_t)q * P.d + c] : 0.f;
    }
    if (lane < kQT) {
        thr[lane] = __int_as_float(0x7f800000);
        fill[lane] = 0;
        mpos[lane] = 0;
    }
    __syncthreads();
    if (threadIdx.x < kQT) {
        float s = 0.f;
        for (int c = 0; c < dp; ++c) s += Qs[threadIdx.x * dp + c] * Qs[threadIdx.x * dp + c];
        qn[threadIdx.x] = s;
    }
    __syncthreads();

    // MFMA operand mapping (16x16x4 f32): A[i][kk] in lane i + 16 kk, B[kk][j]
    // in lane j + 16 kk, D[4 (lane/16) + e][lane % 16] in element e.  The K
    // loop walks float4 chunks: lane group kk takes dims 16t + 4kk + {0..3}.
    const int ii = lane & 15;   // query (A) / row (B) index
    const int kk = lane >> 4;
    const int nblk = (T.ur - T.ul + 16) / 16;
    const int ql[4] = {T.l[4 * kk], T.l[4 * kk + 1], T.l[4 * kk + 2], T.l[4 * kk + 3]};
    const int qr[4] = {T.r[4 * kk], T.r[4 * kk + 1], T.r[4 * kk + 2], T.r[4 * kk + 3]};
    const bool qv[4] = {T.q[4 * kk] >= 0, T.q[4 * kk + 1] >= 0, T.q[4 * kk + 2] >= 0, T.q[4 * kk + 3] >= 0};
    const float4* Qs4 = reinterpret_cast<const float4*>(Qs);
    const float4* X4 = reinterpret_cast<const float4*>(P.X);
    const int dp4 = dp >> 2;
    for (int blk = wave; blk < nblk; blk += kWaves) {
        const int row = T.ul + blk * 16 + ii;
        const int rowc = row <= T.ur ? row : T.ur;
        floatx4 acc = {0.f, 0.f, 0.f, 0.f};
        float xn = 0.f;
        for (int t = 0; t < dp / 16; ++t) {
            const float4 x = X4[(int64_t)rowc * dp4 + 4 * t + kk];
            const float4 q = Qs4[ii * dp4 + 4 * t + kk];
            acc = __builtin_amdgcn_mfma_f32_16x16x4f32(q.x, x.x, acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_f32_16x16x4f32(q.y, x.y, acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_f32_16x16x4f32(q.z, x.z, acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_f32_16x16x4f32(q.w, x.w, acc, 0, 0, 0);
            xn += x.x * x.x + x.y * x.y + x.z * x.z + x.w * x.w;
        }
        xn += __shfl_xor(xn, 16);
        xn += __shfl_xor(xn, 32);
        // lane holds D[4kk + e][ii]: query 4kk + e, row ul + blk*16 + ii
        float ap[4];
        bool cand[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int qi = 4 * kk + e;
            ap[e] = qn[qi] + xn - 2.f * acc[e];
            cand[e] = qv[e] && row <= T.ur && row >= ql[e] && row <= qr[e] && ap[e] < thr[qi];
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            uint64_t m = __ballot(cand[e]);
            while (m) {
                const int src = __builtin_ctzll(m);
                m &= m - 1;
                const int qi = 4 * (src >> 4) + e;
                const float a = __shfl(ap[e], src);
                const int rw = T.ul + blk * 16 + (src & 15);
                if (!(a < thr[qi])) continue;
                const int f = fill[qi];
                int slot;
                if (f < kKeep) {
                    slot = f;
                } else {
                    slot = mpos[qi];
                }
                if (lane == 0) {
                    lv[qi * kKeep + slot] = a;
                    lr[qi * kKeep + slot] = rw;
                    if (f < kKeep) fill[qi] = f + 1;
                }
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
                __builtin_amdgcn_wave_barrier();
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
                if (f + 1 >= kKeep) {
                    // list full: the threshold is its largest entry
                    float v = lv[qi * kKeep + lane];
                    int pos = lane;
                    v = wave_max_pos(v, pos);
                    if (lane == 0) {
                        thr[qi] = v;
                        mpos[qi] = pos;
                    }
                    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
                    __builtin_amdgcn_wave_barrier();
                    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
                }
            }
        }
    }
    __syncthreads();

    // exact re-rank: wavefront w finalises queries w, w + 4, w + 8, w + 12
    const int lists_stride = kQT * kKeep * 8 + kQT * 12;
    for (int qi = wave; qi < kQT; qi += kWaves) {
        const int q = T.q[qi];
        if (q < 0) continue;
        uint64_t key[kWaves];
        float tmin = __int_as_float(0x7f800000);
        int total = 0;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            char* b = reinterpret_cast<char*>(qn + kQT) + (size_t)w * lists_stride;
            const float* wlv = reinterpret_cast<const float*>(b);
            const int32_t* wlr = reinterpret_cast<const int32_t*>(wlv + kQT * kKeep);
            const float* wthr = reinterpret_cast<const float*>(wlr + kQT * kKeep);
            const int32_t* wfill = reinterpret_cast<const int32_t*>(wthr + kQT);
            const int f = wfill[qi];
            total += f;
            if (f >= kKeep) tmin = fminf(tmin, wthr[qi]);
            key[w] = ~0ull;
            if (lane < f) {
                const int rw = wlr[qi * kKeep + lane];
                const float* xr = P.X + (int64_t)rw * dp;
                const float* qq = Qs + qi * dp;
                double s = 0.0;
                for (int c = 0; c < P.d; ++c) {
                    const double t = (double)qq[c] - (double)xr[c];
                    s += t * t;
                }
                key[w] = ((uint64_t)__float_as_uint((float)s) << 32) | (uint32_t)rw;
            }
        }
        // k smallest keys by repeated wave minimum
        float kth = __int_as_float(0x7f800000);
        int found = 0;
        for (int j = 0; j < P.k; ++j) {
            uint64_t best = key[0];
#pragma unroll
            for (int w = 1; w < kWaves; ++w) best = key[w] < best ? key[w] : best;
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
                for (int w = 0; w < kWaves; ++w)
                    if (key[w] == best) key[w] = ~0ull;
            }
            if (lane == 0) {
                P.ids[(int64_t)q * P.k + j] = oid;
                P.dists[(int64_t)q * P.k + j] = od;
            }
        }
        if (P.cert && lane == 0) {
            const double eps = 2.0 * (2.0 * P.d + 4.0) * 5.9604644775390625e-08 * ((double)qn[qi] + (double)P.maxnorm);
            bool ok;
            if (isinf(tmin)) ok = true;                       // no wavefront dropped a row
            else ok = found == P.k && (double)tmin - eps > (double)kth;
            P.cert[q] = ok ? 1 : 0;
        }
        (void)total;
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
        tiles.push_back(t);
    }
    if (ix->maxnorm < 0.f) {
        double mx = 0.0;
        for (int64_t i = 0; i < n; ++i) {
            double s = 0.0;
            for (int c = 0; c < ix->d; ++c) s += (double)ix->X[(size_t)(i * ix->d + c)] * ix->X[(size_t)(i * ix->d + c)];
            mx = std::max(mx, s);
        }
        const_cast<frog_index*>(ix)->maxnorm = (float)(mx * (1.0 + 1e-6));
    }
    const size_t tbytes = tiles.size() * sizeof(Tile);
    void* ws = nullptr;
    e = hipMallocAsync(&ws, tbytes + (size_t)nq + 64, stream);
    if (e != hipSuccess) return fail(FROG_ENOMEM, "bruteforce workspace: %s", hipGetErrorString(e));
    Tile* dT = reinterpret_cast<Tile*>(ws);
    uint8_t* dE = reinterpret_cast<uint8_t*>(ws) + tbytes;
    if (tbytes) e = hipMemcpyAsync(dT, tiles.data(), tbytes, hipMemcpyHostToDevice, stream);
    if (e == hipSuccess) e = hipMemcpyAsync(dE, empty.data(), (size_t)nq, hipMemcpyHostToDevice, stream);
    if (e != hipSuccess) { hipFreeAsync(ws, stream); return fail(FROG_EHIP, "bruteforce upload: %s", hipGetErrorString(e)); }
    hipLaunchKernelGGL(bf_pad_kernel, dim3((unsigned)((nq + 255) / 256)), dim3(256), 0, stream, nq, k, dE, ids, dists, cert);
    if (!tiles.empty()) {
        BFParams P{};
        P.X = ix->dX;
        P.perm = ix->dperm;
        P.n = n;
        P.d = ix->d;
        P.dp = ix->dp;
        P.Q = Q;
        P.tiles = dT;
        P.k = k;
        P.maxnorm = ix->maxnorm;
        P.ids = ids;
        P.dists = dists;
        P.cert = cert;
        const int smem = kQT * ix->dp * 4 + kQT * 4 + kWaves * (kQT * kKeep * 8 + kQT * 12);
        if (smem > 160 * 1024) { hipFreeAsync(ws, stream); return fail(FROG_EUNSUPPORTED, "bruteforce: d too large"); }
        if (smem > 64 * 1024) hipFuncSetAttribute((const void*)bf_tile_kernel, hipFuncAttributeMaxDynamicSharedMemorySize, smem);
        hipLaunchKernelGGL(bf_tile_kernel, dim3((unsigned)tiles.size()), dim3(kThreads), smem, stream, P);
    }
    e = hipGetLastError();
    hipFreeAsync(ws, stream);
    // keep the host-side tile array alive until the copy has run
    hipStreamSynchronize(stream);
    if (e != hipSuccess) return fail(FROG_EHIP, "bruteforce launch: %s", hipGetErrorString(e));
    return FROG_OK;
}

}  // namespace frog
