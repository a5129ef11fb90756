// Internal declarations shared by the library's translation units (host C++
// and HIP).  Not part of the public ABI; include/frog.h is.
#pragma once

#include <cstdint>
#include <map>
#include <memory>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "frog.h"

// An allocator whose value-initialisation of a new element is default-
// initialisation: resize() leaves ints and floats unset, so that a large
// array written right after (in parallel, or by a device copy) is not
// cleared first on one thread.
template <class T>
struct uninit_alloc : std::allocator<T> {
    template <class U>
    struct rebind {
        using other = uninit_alloc<U>;
    };
    uninit_alloc() = default;
    template <class U>
    uninit_alloc(const uninit_alloc<U>&) noexcept {}
    template <class U>
    void construct(U* p) noexcept {
        ::new ((void*)p) U;
    }
    template <class U, class... Args>
    void construct(U* p, Args&&... args) {
        ::new ((void*)p) U(std::forward<Args>(args)...);
    }
};

struct frog_index {
    int64_t n = 0;
    int d = 0, H = 0, m = 0;
    // host copy, rank order
    std::vector<float, uninit_alloc<float>> X;        // n * d
    std::vector<double> attr;    // n, ascending
    std::vector<int32_t> perm;   // n, rank -> original index
    std::vector<int32_t, uninit_alloc<int32_t>> ENC;  // n * H * m
    // device copy (HBM): X rows padded to dp values of the storage type
    // (fp32 in dX, or binary16 bit patterns in dXh)
    int device = -1;
    int dp = 0;
    int storage = FROG_STORAGE_F32;
    float* dX = nullptr;
    uint16_t* dXh = nullptr;
    int32_t* dENC = nullptr;
    double* dattr = nullptr;
    int32_t* dperm = nullptr;
    float maxnorm = -1.f;        // largest squared norm of the stored rows, set at upload
    // work of the GPU construction: distances evaluated, sibling-search expansions
    int64_t build_distances = 0, build_expansions = 0;
    double build_kernel_ms = 0.0;   // from the first kernel's start to the last one's end
    // shared entry samples (entry_mode 1), one per prepared seed: built by
    // frog_index_prepare_sample, immutable afterwards, freed only with the
    // device copy (so a pointer taken under the mutex stays valid while the
    // index stays uploaded)
    struct Sample {
        int nlev = 0;
        int64_t off[34] = {};
        int32_t* ranks = nullptr;   // ascending rank lists of levels 1..nlev, concatenated
        void* xrows = nullptr;      // the levels' stored rows, in list order, dp values each
        uint32_t* prio = nullptr;   // priorities: rank order [0, n), then the levels' lists
        float* norm = nullptr;      // squared norms of the stored rows, same layout
    };
    mutable std::mutex shared_mu;
    std::map<uint64_t, std::unique_ptr<Sample>> samples;
};

namespace frog {

// thread-local error message; returns `code` for convenient `return fail(...)`
int fail(int code, const char* fmt, ...);
void clear_error();

// host construction (build_index.cpp)
int build_host(const float* X, const double* attr, int64_t n, int d,
               const frog_build_params_t& p, frog_index* out);
int layers_for(int64_t n, int n_inv);
// the attribute-rank order (Sec 4) of the input on `threads` host threads:
// out's n, d, H, m, perm, attr, X (rank order) and ENC (n x H x m, all -1
// when fill_enc, else left unset for the caller to write)
int rank_order(const float* X, const double* attr, int64_t n, int d, int m, int n_inv, int threads,
               bool fill_enc, frog_index* out);
int host_threads(int requested);
// The fusion-distance factor 1 - beta (1 - (|ru - rv| / (len - 1))^gamma) of
// every offset of every segment length, as the host construction computes
// it: depth h's lengths are meta[4h] and meta[4h + 2], their offsets' factors
// start at tab[meta[4h + 1]] and tab[meta[4h + 3]].
int fusion_weights(int64_t n, int H, double beta, double gamma, int threads, std::vector<double>& tab,
                   std::vector<int64_t>& meta);
// GPU construction (build_gpu.hip): the same index as build_host, with the
// device copy (fp32 rows) left uploaded on `device`
int build_device(const float* X, const double* attr, int64_t n, int d, const frog_build_params_t& p,
                 int device, frog_index* out);
bool device_build_supported(int d, const frog_build_params_t& p);

// device index view passed to the kernels
struct DevIndex {
    const float* X;       // fp32 rows (storage FROG_STORAGE_F32), else NULL
    const uint16_t* Xh;   // binary16 rows (storage FROG_STORAGE_F16), else NULL
    const int32_t* ENC;
    const double* attr;
    const int32_t* perm;
    int64_t n;
    int d, dp, H, m;
    int storage;
};

// Levels of the shared entry sample, as the kernels see them: level j's list
// is ranks[off[j], off[j + 1]) for 1 <= j <= nlev; level 0 is every rank.
struct SharedLevels {
    const int32_t* ranks;
    const float* xrows;  // row p of level j's list at xrows + (off[j] + p) * dp (fp32 storage)
    const uint16_t* xrowsh;  // the same for binary16 storage
    const uint32_t* prio;  // priority of rank i at [i]; of level j's position p at [n + off[j] + p]
    const float* norm;     // squared norm of the row, same indexing (fp32, any order of summation)
    int64_t off[34];
    int nlev;
    uint64_t key;      // splitmix64(seed): priority(i) = hi32(splitmix64(key ^ i))
};

struct SearchLaunch {
    const float* Q;
    int64_t nq;
    const double* lo;
    const double* hi;
    int k, L, epn, epn_max, B, hash_log2;
    double epn_frac;
    uint64_t seed;
    int64_t qbase;
    int32_t* ids;
    float* dists;
    int32_t* stats;
    void** events;   // NULL or 3 hipEvent_t
    int entry_mode;  // 0 stratified per query, 1 shared sample
    int hotspot_mode;  // 0 Alg. 3, 1 no end condition, 2 all layers
    int eager;         // visited check inside ENIdentification (exact set only)
    SharedLevels lv; // entry_mode 1
    float maxnorm;   // entry_mode 1: largest squared row norm of the index
};

// capi.cpp: the prepared shared sample of `seed` (FROG_ENOTPREPARED if
// frog_index_prepare_sample has not built it) and the largest squared norm
// of the stored rows
int find_sample(const frog_index* ix, uint64_t seed, SharedLevels* out, float* maxnorm);
int build_sample(const frog_index* ix, uint64_t seed, frog_index::Sample* S);
// largest squared norm of the device copy's (stored) rows, taken at upload
float stored_maxnorm(const frog_index* ix);

// search.hip
int launch_search(const DevIndex& ix, const SearchLaunch& a, void* stream);
// the same with the per-call workspace in caller-provided device memory of
// ws_cap bytes (no allocation; FROG_EUNSUPPORTED if the call needs more)
int launch_search_ws(const DevIndex& ix, const SearchLaunch& a, void* stream, void* ws, size_t ws_cap);
// the library's fixed workspace array on the current device (its address,
// taken once per device) and its size
int scratch_area(void** ptr, size_t* bytes);
int launch_rank_bounds(const DevIndex& ix, const double* lo, const double* hi, int64_t nq,
                       int32_t* lr, void* stream);
bool search_shape_supported(int dp, int m, int L);
// copy the rows of the listed ranks: out[i] = X[ranks[i]] (row_bytes each, a
// multiple of 16)
int launch_gather_rows(const void* X, int row_bytes, const int32_t* ranks, int64_t count, void* out, void* stream);
// exhaustive filtered k-NN of nf selected queries (host arrays: query
// indices hq, rank intervals hlr [nf][2], non-empty): ids/dists rows of those
// queries are overwritten with the exact result, cert[q] set to 2 (if not
// NULL); synchronises `stream`.  fp32 rows, 1 <= k <= 256.
int launch_exact_ranges(const DevIndex& ix, const float* Q, const int32_t* hq, const int32_t* hlr, int64_t nf, int k,
                        int32_t* ids, float* dists, int32_t* cert, void* stream);
// bruteforce.hip
int launch_bruteforce(const frog_index* ix, const float* Q, int64_t nq, const double* lo,
                      const double* hi, int k, int32_t* ids, float* dists, int32_t* cert,
                      void* stream);

}  // namespace frog
