// Internal declarations shared by the library's translation units (host C++
// and HIP).  Not part of the public ABI; include/frog.h is.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "frog.h"

struct frog_index {
    int64_t n = 0;
    int d = 0, H = 0, m = 0;
    // host copy, rank order
    std::vector<float> X;        // n * d
    std::vector<double> attr;    // n, ascending
    std::vector<int32_t> perm;   // n, rank -> original index
    std::vector<int32_t> ENC;    // n * H * m
    // device copy (HBM): X rows padded to dp floats
    int device = -1;
    int dp = 0;
    float* dX = nullptr;
    int32_t* dENC = nullptr;
    double* dattr = nullptr;
    int32_t* dperm = nullptr;
    float maxnorm = -1.f;        // largest squared row norm, computed on first use
};

namespace frog {

// thread-local error message; returns `code` for convenient `return fail(...)`
int fail(int code, const char* fmt, ...);
void clear_error();

// host construction (build_index.cpp)
int build_host(const float* X, const double* attr, int64_t n, int d,
               const frog_build_params_t& p, frog_index* out);
int layers_for(int64_t n, int n_inv);

// device index view passed to the kernels
struct DevIndex {
    const float* X;
    const int32_t* ENC;
    const double* attr;
    const int32_t* perm;
    int64_t n;
    int d, dp, H, m;
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
};

// search.hip
int launch_search(const DevIndex& ix, const SearchLaunch& a, void* stream);
int launch_rank_bounds(const DevIndex& ix, const double* lo, const double* hi, int64_t nq,
                       int32_t* lr, void* stream);
bool search_shape_supported(int dp, int m, int L);
// bruteforce.hip
int launch_bruteforce(const frog_index* ix, const float* Q, int64_t nq, const double* lo,
                      const double* hi, int k, int32_t* ids, float* dists, int32_t* cert,
                      void* stream);

}  // namespace frog
