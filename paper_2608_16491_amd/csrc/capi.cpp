// extern "C" entry points of include/frog.h: argument validation, the index
// container (host arrays, file format, device upload) and dispatch to the
// host builder and the HIP launchers.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <thread>

#include "frog_internal.h"
#include "ws_pool.h"

namespace frog {

static thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
    char buf[1024];
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

void clear_error() { g_err.clear(); }

}  // namespace frog

using frog::fail;

namespace {

#define HIP_TRY(expr)                                                                   \
    do {                                                                                \
        hipError_t e_ = (expr);                                                         \
        if (e_ != hipSuccess)                                                           \
            return fail(e_ == hipErrorOutOfMemory ? FROG_ENOMEM : FROG_EHIP, "%s: %s", \
                        #expr, hipGetErrorString(e_));                                  \
    } while (0)

void release_device(frog_index* ix) {
    if (ix->device >= 0) {
        int prev = 0;
        hipGetDevice(&prev);
        hipSetDevice(ix->device);
        if (ix->dX) hipFree(ix->dX);
        if (ix->dXh) hipFree(ix->dXh);
        hipFree(ix->dENC);
        hipFree(ix->dattr);
        hipFree(ix->dperm);
        for (auto& kv : ix->samples) {
            frog_index::Sample& s = *kv.second;
            if (s.ranks) hipFree(s.ranks);
            if (s.xrows) hipFree(s.xrows);
            if (s.prio) hipFree(s.prio);
            if (s.norm) hipFree(s.norm);
        }
        hipSetDevice(prev);
    }
    ix->samples.clear();
    ix->dX = nullptr;
    ix->dXh = nullptr;
    ix->maxnorm = -1.f;
    ix->dENC = nullptr;
    ix->dattr = nullptr;
    ix->dperm = nullptr;
    ix->device = -1;
}

// CRC-32 (IEEE 802.3, reflected polynomial 0xEDB88320), slicing by one byte.
struct Crc32 {
    uint32_t table[256];
    Crc32() {
        for (uint32_t i = 0; i < 256; ++i) {
            uint32_t c = i;
            for (int k = 0; k < 8; ++k) c = (c & 1) ? 0xEDB88320u ^ (c >> 1) : c >> 1;
            table[i] = c;
        }
    }
    uint32_t update(uint32_t crc, const void* data, size_t len) const {
        const uint8_t* p = (const uint8_t*)data;
        crc = ~crc;
        for (size_t i = 0; i < len; ++i) crc = table[(crc ^ p[i]) & 0xFF] ^ (crc >> 8);
        return ~crc;
    }
};
const Crc32& crc32() {
    static const Crc32 c;
    return c;
}

constexpr char kMagic[8] = {'F', 'R', 'O', 'G', 'I', 'D', 'X', '1'};
constexpr uint32_t kVersion = 1;

struct FileHeader {
    char magic[8];
    uint32_t version;
    uint32_t reserved;
    int64_t n;
    int32_t d, H, m, pad;
};
static_assert(sizeof(FileHeader) == 40, "file header layout");

int validate_index_arrays(const double* attr, const int32_t* perm, const int32_t* ENC, int64_t n,
                          int H, int m) {
    for (int64_t i = 0; i < n; ++i) {
        if (std::isnan(attr[i])) return fail(FROG_EINVAL, "attr_sorted[%lld] is NaN", (long long)i);
        if (i > 0 && attr[i] < attr[i - 1])
            return fail(FROG_EINVAL, "attr_sorted is not ascending at %lld", (long long)i);
    }
    std::vector<uint8_t> seen((size_t)n, 0);
    for (int64_t i = 0; i < n; ++i) {
        int32_t p = perm[i];
        if (p < 0 || p >= n || seen[(size_t)p])
            return fail(FROG_EINVAL, "perm is not a permutation (entry %lld)", (long long)i);
        seen[(size_t)p] = 1;
    }
    const int64_t tot = n * H * m;
    for (int64_t i = 0; i < tot; ++i) {
        int32_t v = ENC[i];
        if (v < -1 || v >= n) return fail(FROG_EINVAL, "ENC entry %lld out of range", (long long)i);
    }
    return FROG_OK;
}

}  // namespace

extern "C" {

const char* frog_last_error(void) { return frog::g_err.c_str(); }

void frog_build_params_default(int d, frog_build_params_t* p) {
    if (!p) return;
    const bool small = d <= 300;
    p->m = small ? 16 : 32;
    p->ef_c = small ? 128 : 256;
    p->n_inv = small ? 7 : 6;
    p->patience = 30;
    p->sib_seeds = 16;
    p->num_threads = 0;
    p->beta = 0.2;
    p->gamma = 0.5;
    p->seed = 0;
}

void frog_search_params_default(frog_search_params_t* p) {
    if (!p) return;
    p->epn = 16;
    p->epn_frac = 0.0;
    p->epn_max = 0;
    p->budget = 16;
    p->seed = 0;
    p->query_base = 0;
    p->hash_log2 = 10;
    p->phase_events = nullptr;
    p->entry_mode = 0;
    p->hotspot_mode = 0;
    p->eager_check = 0;
}

static int check_build_args(const float* X, const double* attr, int64_t n, int d, const frog_build_params_t* p,
                            frog_index_t** out, frog_build_params_t* q) {
    if (!out) return fail(FROG_EINVAL, "out is NULL");
    *out = nullptr;
    if (!X || !attr) return fail(FROG_EINVAL, "X or attr is NULL");
    if (n < 1 || n > INT32_MAX - 1) return fail(FROG_EINVAL, "n=%lld outside [1, 2^31-2]", (long long)n);
    if (d < 1 || d > 65536) return fail(FROG_EINVAL, "d=%d outside [1, 65536]", d);
    if (p) *q = *p; else frog_build_params_default(d, q);
    if (q->m < 1 || q->m > 64) return fail(FROG_EINVAL, "m=%d outside [1, 64]", q->m);
    if (q->ef_c < q->m || q->ef_c > 4096) return fail(FROG_EINVAL, "ef_c=%d outside [m, 4096]", q->ef_c);
    if (q->n_inv < 0 || q->n_inv > 40) return fail(FROG_EINVAL, "n_inv=%d outside [0, 40]", q->n_inv);
    if (q->patience < 1) return fail(FROG_EINVAL, "patience=%d < 1", q->patience);
    if (q->sib_seeds < 1 || q->sib_seeds > 4096)
        return fail(FROG_EINVAL, "sib_seeds=%d outside [1, 4096]", q->sib_seeds);
    if (!(q->beta >= 0.0 && q->beta < 1.0) || !(q->gamma > 0.0))
        return fail(FROG_EINVAL, "beta=%g must be in [0,1), gamma=%g > 0", q->beta, q->gamma);
    return FROG_OK;
}

int frog_build_index_gpu(const float* X, const double* attr, int64_t n, int d, const frog_build_params_t* p,
                         int device, frog_index_t** out) {
    frog::clear_error();
    frog_build_params_t q;
    int rc = check_build_args(X, attr, n, d, p, out, &q);
    if (rc) return rc;
    if (!frog::device_build_supported(d, q))
        return fail(FROG_EUNSUPPORTED, "GPU construction needs d <= 1024, m <= 32, ef_c <= 256, sib_seeds <= 64");
    frog_index* ix = new (std::nothrow) frog_index;
    if (!ix) return fail(FROG_ENOMEM, "allocation failed");
    rc = frog::build_device(X, attr, n, d, q, device, ix);
    if (rc != FROG_OK) { delete ix; return rc; }
    *out = ix;
    return FROG_OK;
}

int frog_index_build_stats(const frog_index_t* ix, int64_t* distances, int64_t* expansions, double* kernel_ms) {
    frog::clear_error();
    if (!ix) return fail(FROG_EINVAL, "index is NULL");
    if (distances) *distances = ix->build_distances;
    if (expansions) *expansions = ix->build_expansions;
    if (kernel_ms) *kernel_ms = ix->build_kernel_ms;
    return FROG_OK;
}

int frog_build_index(const float* X, const double* attr, int64_t n, int d,
                     const frog_build_params_t* p, frog_index_t** out) {
    frog::clear_error();
    if (!out) return fail(FROG_EINVAL, "out is NULL");
    *out = nullptr;
    if (!X || !attr) return fail(FROG_EINVAL, "X or attr is NULL");
    if (n < 1 || n > INT32_MAX - 1) return fail(FROG_EINVAL, "n=%lld outside [1, 2^31-2]", (long long)n);
    if (d < 1 || d > 65536) return fail(FROG_EINVAL, "d=%d outside [1, 65536]", d);
    frog_build_params_t q;
    if (p) q = *p; else frog_build_params_default(d, &q);
    if (q.m < 1 || q.m > 64) return fail(FROG_EINVAL, "m=%d outside [1, 64]", q.m);
    if (q.ef_c < q.m || q.ef_c > 4096) return fail(FROG_EINVAL, "ef_c=%d outside [m, 4096]", q.ef_c);
    if (q.n_inv < 0 || q.n_inv > 40) return fail(FROG_EINVAL, "n_inv=%d outside [0, 40]", q.n_inv);
    if (q.patience < 1) return fail(FROG_EINVAL, "patience=%d < 1", q.patience);
    if (q.sib_seeds < 1 || q.sib_seeds > 4096) return fail(FROG_EINVAL, "sib_seeds=%d outside [1, 4096]", q.sib_seeds);
    if (!(q.beta >= 0.0 && q.beta < 1.0) || !(q.gamma > 0.0))
        return fail(FROG_EINVAL, "beta=%g must be in [0,1), gamma=%g > 0", q.beta, q.gamma);
    frog_index* ix = new (std::nothrow) frog_index;
    if (!ix) return fail(FROG_ENOMEM, "allocation failed");
    int rc = frog::build_host(X, attr, n, d, q, ix);
    if (rc != FROG_OK) { delete ix; return rc; }
    *out = ix;
    return FROG_OK;
}

int frog_index_from_arrays(const float* X_rank, const double* attr_sorted, const int32_t* perm,
                           const int32_t* ENC, int64_t n, int d, int H, int m, frog_index_t** out) {
    frog::clear_error();
    if (!out) return fail(FROG_EINVAL, "out is NULL");
    *out = nullptr;
    if (!X_rank || !attr_sorted || !perm || !ENC) return fail(FROG_EINVAL, "NULL array");
    if (n < 1 || n > INT32_MAX - 1 || d < 1 || d > 65536 || H < 1 || H > 40 || m < 1 || m > 64)
        return fail(FROG_EINVAL, "bad shape n=%lld d=%d H=%d m=%d", (long long)n, d, H, m);
    int rc = validate_index_arrays(attr_sorted, perm, ENC, n, H, m);
    if (rc) return rc;
    frog_index* ix = new (std::nothrow) frog_index;
    if (!ix) return fail(FROG_ENOMEM, "allocation failed");
    try {
        ix->n = n; ix->d = d; ix->H = H; ix->m = m;
        ix->X.assign(X_rank, X_rank + n * d);
        ix->attr.assign(attr_sorted, attr_sorted + n);
        ix->perm.assign(perm, perm + n);
        ix->ENC.assign(ENC, ENC + n * H * m);
    } catch (const std::bad_alloc&) {
        delete ix;
        return fail(FROG_ENOMEM, "host allocation failed");
    }
    *out = ix;
    return FROG_OK;
}

int frog_index_export(const frog_index_t* ix, float* X_rank, double* attr_sorted, int32_t* perm,
                      int32_t* ENC) {
    frog::clear_error();
    if (!ix) return fail(FROG_EINVAL, "index is NULL");
    if (X_rank) std::memcpy(X_rank, ix->X.data(), ix->X.size() * sizeof(float));
    if (attr_sorted) std::memcpy(attr_sorted, ix->attr.data(), ix->attr.size() * sizeof(double));
    if (perm) std::memcpy(perm, ix->perm.data(), ix->perm.size() * sizeof(int32_t));
    if (ENC) std::memcpy(ENC, ix->ENC.data(), ix->ENC.size() * sizeof(int32_t));
    return FROG_OK;
}

int frog_index_info(const frog_index_t* ix, int64_t* n, int* d, int* H, int* m) {
    frog::clear_error();
    if (!ix) return fail(FROG_EINVAL, "index is NULL");
    if (n) *n = ix->n;
    if (d) *d = ix->d;
    if (H) *H = ix->H;
    if (m) *m = ix->m;
    return FROG_OK;
}

int frog_index_save(const frog_index_t* ix, const char* path) {
    frog::clear_error();
    if (!ix || !path) return fail(FROG_EINVAL, "NULL argument");
    FILE* f = std::fopen(path, "wb");
    if (!f) return fail(FROG_EIO, "cannot open %s for writing", path);
    FileHeader h{};
    std::memcpy(h.magic, kMagic, 8);
    h.version = kVersion;
    h.n = ix->n; h.d = ix->d; h.H = ix->H; h.m = ix->m;
    uint32_t crc = 0;
    struct Part { const void* p; size_t len; } parts[5] = {
        {&h, sizeof(h)},
        {ix->X.data(), ix->X.size() * sizeof(float)},
        {ix->attr.data(), ix->attr.size() * sizeof(double)},
        {ix->perm.data(), ix->perm.size() * sizeof(int32_t)},
        {ix->ENC.data(), ix->ENC.size() * sizeof(int32_t)}};
    bool ok = true;
    for (auto& part : parts) {
        crc = crc32().update(crc, part.p, part.len);
        ok = ok && std::fwrite(part.p, 1, part.len, f) == part.len;
    }
    ok = ok && std::fwrite(&crc, 4, 1, f) == 1;
    ok = (std::fclose(f) == 0) && ok;
    return ok ? FROG_OK : fail(FROG_EIO, "write to %s failed", path);
}

int frog_index_load(const char* path, frog_index_t** out) {
    frog::clear_error();
    if (!path || !out) return fail(FROG_EINVAL, "NULL argument");
    *out = nullptr;
    FILE* f = std::fopen(path, "rb");
    if (!f) return fail(FROG_EIO, "cannot open %s", path);
    FileHeader h{};
    if (std::fread(&h, sizeof(h), 1, f) != 1) { std::fclose(f); return fail(FROG_EBADINDEX, "short header"); }
    if (std::memcmp(h.magic, kMagic, 8) != 0 || h.version != kVersion) {
        std::fclose(f);
        return fail(FROG_EBADINDEX, "bad magic or version in %s", path);
    }
    if (h.n < 1 || h.n > INT32_MAX - 1 || h.d < 1 || h.d > 65536 || h.H < 1 || h.H > 40 || h.m < 1 || h.m > 64) {
        std::fclose(f);
        return fail(FROG_EBADINDEX, "bad shape in header");
    }
    frog_index* ix = new (std::nothrow) frog_index;
    if (!ix) { std::fclose(f); return fail(FROG_ENOMEM, "allocation failed"); }
    try {
        ix->n = h.n; ix->d = h.d; ix->H = h.H; ix->m = h.m;
        ix->X.resize((size_t)h.n * h.d);
        ix->attr.resize((size_t)h.n);
        ix->perm.resize((size_t)h.n);
        ix->ENC.resize((size_t)h.n * h.H * h.m);
    } catch (const std::bad_alloc&) {
        delete ix;
        std::fclose(f);
        return fail(FROG_ENOMEM, "host allocation failed");
    }
    uint32_t crc = crc32().update(0, &h, sizeof(h));
    struct Part { void* p; size_t len; } parts[4] = {
        {ix->X.data(), ix->X.size() * sizeof(float)},
        {ix->attr.data(), ix->attr.size() * sizeof(double)},
        {ix->perm.data(), ix->perm.size() * sizeof(int32_t)},
        {ix->ENC.data(), ix->ENC.size() * sizeof(int32_t)}};
    bool ok = true;
    for (auto& part : parts) {
        ok = ok && std::fread(part.p, 1, part.len, f) == part.len;
        if (ok) crc = crc32().update(crc, part.p, part.len);
    }
    uint32_t stored = 0;
    ok = ok && std::fread(&stored, 4, 1, f) == 1;
    std::fclose(f);
    if (!ok || stored != crc) {
        delete ix;
        return fail(FROG_EBADINDEX, "truncated file or checksum mismatch in %s", path);
    }
    int rc = validate_index_arrays(ix->attr.data(), ix->perm.data(), ix->ENC.data(), ix->n, ix->H, ix->m);
    if (rc) { delete ix; return fail(FROG_EBADINDEX, "%s", frog_last_error()); }
    *out = ix;
    return FROG_OK;
}

int frog_index_upload(frog_index_t* ix, int device) {
    return frog_index_upload_ex(ix, device, FROG_STORAGE_F32);
}

}  // extern "C"

namespace frog {

// The 16-bit pattern of v rounded to nearest even in `storage` (fp16: the
// compiler's binary16 conversion; bf16: the upper half of the fp32 bits after
// adding half an ulp, ties to even); false if v or its rounding is not
// finite.
bool half_bits(float v, int storage, uint16_t* out) {
    if (!std::isfinite(v)) return false;
    if (storage == FROG_STORAGE_F16) {
        const _Float16 h = (_Float16)v;
        if (!(h == h) || h > (_Float16)65504.f || h < (_Float16)-65504.f) return false;
        std::memcpy(out, &h, 2);
        return true;
    }
    uint32_t b;
    std::memcpy(&b, &v, 4);
    const uint32_t r = b + 0x7FFFu + ((b >> 16) & 1u);
    const uint16_t h = (uint16_t)(r >> 16);
    if ((h & 0x7F80u) == 0x7F80u) return false;   // rounded to infinity
    *out = h;
    return true;
}

// value c of row i as the device stores it
float stored_value(const frog_index* ix, int64_t i, int c) {
    const float v = ix->X[(size_t)i * ix->d + c];
    if (ix->storage == FROG_STORAGE_F16) return (float)(_Float16)v;
    if (ix->storage == FROG_STORAGE_BF16) {
        uint16_t h = 0;
        half_bits(v, FROG_STORAGE_BF16, &h);
        const uint32_t w = (uint32_t)h << 16;
        float f;
        std::memcpy(&f, &w, 4);
        return f;
    }
    return v;
}

// the largest squared norm of the stored rows (in double, then widened by
// a relative 1e-6 so that it bounds the fp32 value), on all host threads
float stored_maxnorm(const frog_index* ix) {
    const int T = host_threads(0);
    std::vector<double> part((size_t)T, 0.0);
    std::vector<std::thread> th;
    for (int t = 0; t < T; ++t)
        th.emplace_back([&, t]() {
            double mx = 0.0;
            for (int64_t i = ix->n * t / T; i < ix->n * (t + 1) / T; ++i) {
                double s = 0.0;
                for (int c = 0; c < ix->d; ++c) {
                    const double v = stored_value(ix, i, c);
                    s += v * v;
                }
                mx = std::max(mx, s);
            }
            part[(size_t)t] = mx;
        });
    for (auto& x : th) x.join();
    double mx = 0.0;
    for (double v : part) mx = std::max(mx, v);
    return (float)(mx * (1.0 + 1e-6));
}

}  // namespace frog

extern "C" {

int frog_index_upload_ex(frog_index_t* ix, int device, int storage) {
    frog::clear_error();
    if (!ix) return fail(FROG_EINVAL, "index is NULL");
    if (storage != FROG_STORAGE_F32 && storage != FROG_STORAGE_F16 && storage != FROG_STORAGE_BF16)
        return fail(FROG_EINVAL, "storage=%d: FROG_STORAGE_F32, FROG_STORAGE_F16 or FROG_STORAGE_BF16", storage);
    const bool half = storage != FROG_STORAGE_F32;
    if (half && ix->d > 128) return fail(FROG_EUNSUPPORTED, "16-bit storage needs d <= 128 (d=%d)", ix->d);
    // 16-bit rows: round every value once (nearest even) and pad to dp values
    const int dp = half ? (ix->d + 63) / 64 * 64 : (ix->d + 31) / 32 * 32;
    std::vector<uint16_t> hx;
    if (half) {
        hx.assign((size_t)ix->n * dp, 0);
        for (int64_t i = 0; i < ix->n; ++i)
            for (int c = 0; c < ix->d; ++c) {
                const float v = ix->X[(size_t)i * ix->d + c];
                uint16_t bits;
                if (!frog::half_bits(v, storage, &bits))
                    return fail(FROG_EUNSUPPORTED, "row %lld: value %g outside the %s range", (long long)i, (double)v,
                                storage == FROG_STORAGE_F16 ? "fp16" : "bf16");
                hx[(size_t)i * dp + c] = bits;
            }
    }
    int ndev = 0;
    HIP_TRY(hipGetDeviceCount(&ndev));
    if (device < 0 || device >= ndev) return fail(FROG_EINVAL, "device %d not in [0, %d)", device, ndev);
    release_device(ix);
    int prev = 0;
    HIP_TRY(hipGetDevice(&prev));
    HIP_TRY(hipSetDevice(device));
    const size_t nX = (size_t)ix->n * dp, nE = (size_t)ix->n * ix->H * ix->m;
    ix->device = device;
    ix->dp = dp;
    ix->storage = storage;
    auto bail = [&](int rc) { release_device(ix); hipSetDevice(prev); return rc; };
    hipError_t e = half ? hipMalloc(&ix->dXh, nX * sizeof(uint16_t)) : hipMalloc(&ix->dX, nX * sizeof(float));
    if (e == hipSuccess) e = hipMalloc(&ix->dENC, nE * sizeof(int32_t));
    if (e == hipSuccess) e = hipMalloc(&ix->dattr, (size_t)ix->n * sizeof(double));
    if (e == hipSuccess) e = hipMalloc(&ix->dperm, (size_t)ix->n * sizeof(int32_t));
    if (e != hipSuccess)
        return bail(fail(e == hipErrorOutOfMemory ? FROG_ENOMEM : FROG_EHIP, "device allocation: %s",
                         hipGetErrorString(e)));
    if (half) {
        e = hipMemcpy(ix->dXh, hx.data(), nX * sizeof(uint16_t), hipMemcpyHostToDevice);
    } else if (dp == ix->d) {
        e = hipMemcpy(ix->dX, ix->X.data(), nX * sizeof(float), hipMemcpyHostToDevice);
    } else {
        e = hipMemset(ix->dX, 0, nX * sizeof(float));
        if (e == hipSuccess)
            e = hipMemcpy2D(ix->dX, (size_t)dp * sizeof(float), ix->X.data(), (size_t)ix->d * sizeof(float),
                            (size_t)ix->d * sizeof(float), (size_t)ix->n, hipMemcpyHostToDevice);
    }
    if (e == hipSuccess) e = hipMemcpy(ix->dENC, ix->ENC.data(), nE * sizeof(int32_t), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(ix->dattr, ix->attr.data(), (size_t)ix->n * sizeof(double), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(ix->dperm, ix->perm.data(), (size_t)ix->n * sizeof(int32_t), hipMemcpyHostToDevice);
    if (e != hipSuccess) return bail(fail(FROG_EHIP, "upload: %s", hipGetErrorString(e)));
    ix->maxnorm = frog::stored_maxnorm(ix);
    hipSetDevice(prev);
    return FROG_OK;
}

void frog_index_free(frog_index_t* ix) {
    if (!ix) return;
    release_device(ix);
    delete ix;
}

}  // extern "C"

namespace {

frog::DevIndex view(const frog_index* ix) {
    return frog::DevIndex{ix->dX, ix->dXh, ix->dENC, ix->dattr, ix->dperm, ix->n, ix->d, ix->dp, ix->H, ix->m,
                          ix->storage};
}

// Device entry points run on the index's device; the caller's stream must
// belong to it.
int check_device_index(const frog_index_t* ix) {
    if (!ix) return fail(FROG_EINVAL, "index is NULL");
    if (ix->device < 0 || (!ix->dX && !ix->dXh)) return fail(FROG_ENOTUPLOADED, "index has not been uploaded");
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return fail(FROG_EHIP, "hipGetDevice failed");
    if (cur != ix->device)
        return fail(FROG_EINVAL, "current device %d differs from the index's device %d", cur, ix->device);
    return FROG_OK;
}

}  // namespace

extern "C" {

int frog_rank_bounds(const frog_index_t* ix, const double* d_lo, const double* d_hi, int64_t nq,
                     int32_t* d_lr, void* stream) {
    frog::clear_error();
    int rc = check_device_index(ix);
    if (rc) return rc;
    if (nq < 0) return fail(FROG_EINVAL, "nq < 0");
    if (nq == 0) return FROG_OK;
    if (!d_lo || !d_hi || !d_lr) return fail(FROG_EINVAL, "NULL device pointer");
    return frog::launch_rank_bounds(view(ix), d_lo, d_hi, nq, d_lr, stream);
}

}  // extern "C"

namespace {

// Validation and argument marshalling shared by frog_search_ex and
// the other search entry points; on FROG_OK with *empty == false, *a is ready to launch.
int search_args(const frog_index_t* ix, const float* d_queries, int64_t nq, const double* d_lo, const double* d_hi,
                int k, int L, const frog_search_params_t* p, int32_t* d_ids, float* d_dists, int32_t* d_stats,
                frog::SearchLaunch* out, bool* empty) {
    *empty = true;
    int rc = check_device_index(ix);
    if (rc) return rc;
    frog_search_params_t q;
    if (p) q = *p; else frog_search_params_default(&q);
    if (nq < 0) return fail(FROG_EINVAL, "nq < 0");
    if (k < 1 || L < k || L > 256) return fail(FROG_EINVAL, "need 1 <= k <= L <= 256 (k=%d, L=%d)", k, L);
    if (q.budget < 1 || q.budget > 64) return fail(FROG_EINVAL, "budget=%d outside [1, 64]", q.budget);
    if (q.epn < 1 || q.epn > (1 << 20)) return fail(FROG_EINVAL, "epn=%d outside [1, 2^20]", q.epn);
    if (!(q.epn_frac >= 0.0) || q.epn_frac > 1.0) return fail(FROG_EINVAL, "epn_frac=%g outside [0, 1]", q.epn_frac);
    if (q.epn_frac > 0.0 && (q.epn_max < q.epn || q.epn_max > (1 << 20)))
        return fail(FROG_EINVAL, "epn_max=%d outside [epn, 2^20]", q.epn_max);
    if (q.hash_log2 != 0 && (q.hash_log2 < 6 || q.hash_log2 > 13))
        return fail(FROG_EINVAL, "hash_log2=%d: 0 or 6..13", q.hash_log2);
    if (q.query_base < 0) return fail(FROG_EINVAL, "query_base < 0");
    if (q.entry_mode != 0 && q.entry_mode != 1) return fail(FROG_EINVAL, "entry_mode=%d: 0 or 1", q.entry_mode);
    if (q.hotspot_mode < 0 || q.hotspot_mode > 2) return fail(FROG_EINVAL, "hotspot_mode=%d: 0, 1 or 2", q.hotspot_mode);
    if (q.eager_check != 0 && q.eager_check != 1) return fail(FROG_EINVAL, "eager_check=%d: 0 or 1", q.eager_check);
    if (q.eager_check && q.hash_log2 != 0)
        return fail(FROG_EINVAL, "eager_check needs the exact visited set (hash_log2 = 0)");
    if (!frog::search_shape_supported(ix->dp, ix->m, L))
        return fail(FROG_EUNSUPPORTED, "no search kernel for padded d=%d, m=%d, L=%d", ix->dp, ix->m, L);
    if (nq == 0) return FROG_OK;
    if (!d_queries || !d_lo || !d_hi || !d_ids || !d_dists) return fail(FROG_EINVAL, "NULL device pointer");
    frog::SearchLaunch& a = *out;
    a = frog::SearchLaunch{};
    a.Q = d_queries; a.nq = nq; a.lo = d_lo; a.hi = d_hi; a.k = k; a.L = L;
    a.epn = q.epn; a.epn_max = q.epn_frac > 0.0 ? q.epn_max : q.epn; a.epn_frac = q.epn_frac;
    a.B = q.budget; a.hash_log2 = q.hash_log2; a.seed = q.seed; a.qbase = q.query_base;
    a.ids = d_ids; a.dists = d_dists; a.stats = d_stats; a.events = q.phase_events;
    a.entry_mode = q.entry_mode;
    a.hotspot_mode = q.hotspot_mode;
    a.eager = q.eager_check;
    if (q.entry_mode == 1) {
        rc = frog::find_sample(ix, q.seed, &a.lv, &a.maxnorm);
        if (rc) return rc;
    }
    *empty = false;
    return FROG_OK;
}

}  // namespace

extern "C" {

int frog_search_ex(const frog_index_t* ix, const float* d_queries, int64_t nq, const double* d_lo,
                   const double* d_hi, int k, int L, const frog_search_params_t* p, int32_t* d_ids,
                   float* d_dists, int32_t* d_stats, void* stream) {
    frog::clear_error();
    frog::SearchLaunch a;
    bool empty = true;
    const int rc = search_args(ix, d_queries, nq, d_lo, d_hi, k, L, p, d_ids, d_dists, d_stats, &a, &empty);
    if (rc || empty) return rc;
    return frog::launch_search(view(ix), a, stream);
}

int frog_search_noalloc(const frog_index_t* ix, const float* d_queries, int64_t nq, const double* d_lo,
                        const double* d_hi, int k, int L, const frog_search_params_t* p, int32_t* d_ids,
                        float* d_dists, int32_t* d_stats, void* stream) {
    frog::clear_error();
    frog::SearchLaunch a;
    bool empty = true;
    int rc = search_args(ix, d_queries, nq, d_lo, d_hi, k, L, p, d_ids, d_dists, d_stats, &a, &empty);
    if (rc || empty) return rc;
    void* ws = nullptr;
    size_t cap = 0;
    rc = frog::scratch_area(&ws, &cap);
    if (rc) return rc;
    return frog::launch_search_ws(view(ix), a, stream, ws, cap);
}

int frog_search(const frog_index_t* ix, const float* d_queries, int64_t nq, const double* d_lo,
                const double* d_hi, int k, int L, int32_t* d_ids, float* d_dists, void* stream) {
    return frog_search_ex(ix, d_queries, nq, d_lo, d_hi, k, L, nullptr, d_ids, d_dists, nullptr, stream);
}

int frog_bruteforce_filtered(const frog_index_t* ix, const float* d_queries, int64_t nq,
                             const double* d_lo, const double* d_hi, int k, int32_t* d_ids,
                             float* d_dists, int32_t* d_certified, void* stream) {
    frog::clear_error();
    int rc = check_device_index(ix);
    if (rc) return rc;
    if (nq < 0) return fail(FROG_EINVAL, "nq < 0");
    if (k < 1 || k > 256) return fail(FROG_EINVAL, "k=%d outside [1, 256]", k);
    if (ix->storage != FROG_STORAGE_F32)
        return fail(FROG_EUNSUPPORTED, "exhaustive search needs an index uploaded with fp32 rows");
    if (nq == 0) return FROG_OK;
    if (!d_queries || !d_lo || !d_hi || !d_ids || !d_dists) return fail(FROG_EINVAL, "NULL device pointer");
    return frog::launch_bruteforce(ix, d_queries, nq, d_lo, d_hi, k, d_ids, d_dists, d_certified, stream);
}

}  // extern "C"

namespace frog {

static uint64_t mix64(uint64_t x) {
    uint64_t z = x + 0x9E3779B97F4A7C15ULL;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

// Level j (1 <= j <= nlev) holds the ranks whose priority p has at least j
// leading zero bits (p < 2^(32-j)); nlev covers the smallest threshold any
// query can ask for (one entry point out of n).  Builds one seed's lists, row
// copies, priorities and norms on the index's device (synchronously).
int build_sample(const frog_index* ix, uint64_t seed, frog_index::Sample* S) {
    const int64_t n = ix->n;
    const uint64_t key = mix64(seed);
    const uint64_t tmin = ((uint64_t)1 << 32) / (uint64_t)n + 1;   // >= ceil(2^32 / n)
    int cl = 0;
    while (((uint64_t)1 << cl) < tmin) ++cl;
    const int nlev = std::max(1, std::min(31, 32 - cl + 1));
    std::vector<uint8_t> depth((size_t)n);
    std::vector<int64_t> cnt((size_t)nlev + 2, 0);
    std::vector<uint32_t> prio_rank((size_t)n);
    for (int64_t i = 0; i < n; ++i) {
        const uint32_t p = (uint32_t)(mix64(key ^ (uint64_t)i) >> 32);
        prio_rank[(size_t)i] = p;
        const int z = p == 0 ? 32 : __builtin_clz(p);
        depth[(size_t)i] = (uint8_t)std::min(z, nlev);
        for (int j = 1; j <= depth[(size_t)i]; ++j) ++cnt[(size_t)j];
    }
    int64_t off[34] = {};
    for (int j = 1; j <= nlev; ++j) off[j + 1] = off[j] + cnt[(size_t)j];
    std::vector<int32_t> ranks((size_t)std::max<int64_t>(off[nlev + 1], 1));
    std::vector<int64_t> fill(off, off + nlev + 2);
    for (int64_t i = 0; i < n; ++i)
        for (int j = 1; j <= depth[(size_t)i]; ++j) ranks[(size_t)fill[(size_t)j]++] = (int32_t)i;
    // priorities and squared norms, by rank and then in list order
    const int64_t total = off[nlev + 1];
    std::vector<uint32_t> prio((size_t)(n + total));
    std::vector<float> nrm((size_t)(n + total));
    for (int64_t i = 0; i < n; ++i) {
        float sq = 0.f;
        for (int c = 0; c < ix->d; ++c) {
            const float v = stored_value(ix, i, c);
            sq += v * v;
        }
        prio[(size_t)i] = prio_rank[(size_t)i];
        nrm[(size_t)i] = sq;
    }
    for (int64_t p = 0; p < total; ++p) {
        prio[(size_t)(n + p)] = prio_rank[(size_t)ranks[(size_t)p]];
        nrm[(size_t)(n + p)] = nrm[(size_t)ranks[(size_t)p]];
    }
    auto drop = [&]() {
        if (S->ranks) (void)hipFree(S->ranks);
        if (S->xrows) (void)hipFree(S->xrows);
        if (S->prio) (void)hipFree(S->prio);
        if (S->norm) (void)hipFree(S->norm);
        S->ranks = nullptr; S->xrows = nullptr; S->prio = nullptr; S->norm = nullptr;
    };
    hipError_t e = hipMalloc(&S->ranks, ranks.size() * sizeof(int32_t));
    if (e == hipSuccess)
        e = hipMemcpy(S->ranks, ranks.data(), ranks.size() * sizeof(int32_t), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMalloc(&S->prio, prio.size() * sizeof(uint32_t));
    if (e == hipSuccess) e = hipMemcpy(S->prio, prio.data(), prio.size() * sizeof(uint32_t), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMalloc(&S->norm, nrm.size() * sizeof(float));
    if (e == hipSuccess) e = hipMemcpy(S->norm, nrm.data(), nrm.size() * sizeof(float), hipMemcpyHostToDevice);
    // the listed stored rows, so that a scan over a list reads contiguous rows
    const int row_bytes = ix->dp * (ix->storage == FROG_STORAGE_F32 ? 4 : 2);
    if (e == hipSuccess) e = hipMalloc(&S->xrows, (size_t)std::max<int64_t>(total, 1) * row_bytes);
    int rc = FROG_OK;
    if (e == hipSuccess && total > 0) {
        const void* rows = ix->storage == FROG_STORAGE_F32 ? (const void*)ix->dX : (const void*)ix->dXh;
        rc = launch_gather_rows(rows, row_bytes, S->ranks, total, S->xrows, nullptr);
        if (rc == FROG_OK) e = hipDeviceSynchronize();
    }
    if (e != hipSuccess || rc != FROG_OK) {
        drop();
        if (rc != FROG_OK) return rc;
        return fail(e == hipErrorOutOfMemory ? FROG_ENOMEM : FROG_EHIP, "shared sample levels: %s",
                    hipGetErrorString(e));
    }
    std::copy(off, off + 34, S->off);
    S->nlev = nlev;
    return FROG_OK;
}

int find_sample(const frog_index* ix, uint64_t seed, SharedLevels* out, float* maxnorm) {
    std::lock_guard<std::mutex> g(ix->shared_mu);
    auto it = ix->samples.find(seed);
    if (it == ix->samples.end())
        return fail(FROG_ENOTPREPARED, "entry_mode 1 with seed %llu: call frog_index_prepare_sample first",
                    (unsigned long long)seed);
    const frog_index::Sample& S = *it->second;
    out->ranks = S.ranks;
    out->xrows = ix->storage == FROG_STORAGE_F32 ? static_cast<const float*>(S.xrows) : nullptr;
    out->xrowsh = ix->storage != FROG_STORAGE_F32 ? static_cast<const uint16_t*>(S.xrows) : nullptr;
    out->prio = S.prio;
    out->norm = S.norm;
    std::copy(S.off, S.off + 34, out->off);
    out->nlev = S.nlev;
    out->key = mix64(seed);
    *maxnorm = ix->maxnorm;
    return FROG_OK;
}

}  // namespace frog

extern "C" {

int frog_index_prepare_sample(frog_index_t* ix, uint64_t seed) {
    frog::clear_error();
    int rc = check_device_index(ix);
    if (rc) return rc;
    {
        std::lock_guard<std::mutex> g(ix->shared_mu);
        if (ix->samples.count(seed)) return FROG_OK;
    }
    // built outside the lock, so searches with other seeds are not held up
    std::unique_ptr<frog_index::Sample> S(new (std::nothrow) frog_index::Sample);
    if (!S) return fail(FROG_ENOMEM, "allocation failed");
    rc = frog::build_sample(ix, seed, S.get());
    if (rc) return rc;
    std::lock_guard<std::mutex> g(ix->shared_mu);
    if (ix->samples.count(seed)) {
        // another thread prepared the same seed meanwhile: keep its copy
        (void)hipFree(S->ranks);
        (void)hipFree(S->xrows);
        (void)hipFree(S->prio);
        (void)hipFree(S->norm);
        return FROG_OK;
    }
    ix->samples.emplace(seed, std::move(S));
    return FROG_OK;
}

}  // extern "C"

namespace frog {

namespace {

hipMemPool_t device_pool(hipError_t* err) {
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static hipMemPool_t pools[kMaxDevices] = {};
    int dev = -1;
    *err = hipGetDevice(&dev);
    if (*err != hipSuccess) return nullptr;
    if (dev < 0 || dev >= kMaxDevices) {
        *err = hipErrorInvalidDevice;
        return nullptr;
    }
    std::lock_guard<std::mutex> g(mu);
    if (!pools[dev]) {
        hipMemPoolProps props{};
        props.allocType = hipMemAllocationTypePinned;
        props.handleTypes = hipMemHandleTypeNone;
        props.location.type = hipMemLocationTypeDevice;
        props.location.id = dev;
        hipMemPool_t pool = nullptr;
        *err = hipMemPoolCreate(&pool, &props);
        if (*err != hipSuccess) return nullptr;
        uint64_t keep = ~0ull;
        *err = hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &keep);
        if (*err != hipSuccess) {
            (void)hipMemPoolDestroy(pool);
            return nullptr;
        }
        pools[dev] = pool;
    }
    return pools[dev];
}

}  // namespace

hipError_t ws_alloc(void** ptr, size_t bytes, hipStream_t stream) {
    hipError_t e = hipSuccess;
    hipMemPool_t pool = device_pool(&e);
    if (!pool) return e;
    return hipMallocFromPoolAsync(ptr, bytes, pool, stream);
}

hipError_t ws_free(void* ptr, hipStream_t stream) { return hipFreeAsync(ptr, stream); }

struct Slot {
    std::mutex mu;          // held by the lease while a call enqueues
    void* ptr = nullptr;
    size_t cap = 0;
};

namespace {

Slot* slot_for(hipStream_t stream, hipError_t* err) {
    static std::mutex mu;
    static std::map<std::pair<int, hipStream_t>, std::unique_ptr<Slot>> slots;
    int dev = -1;
    *err = hipGetDevice(&dev);
    if (*err != hipSuccess) return nullptr;
    std::lock_guard<std::mutex> g(mu);
    std::unique_ptr<Slot>& sl = slots[std::make_pair(dev, stream)];
    if (!sl) {
        sl.reset(new (std::nothrow) Slot);
        if (!sl) {
            *err = hipErrorOutOfMemory;
            return nullptr;
        }
    }
    return sl.get();
}

}  // namespace

hipError_t WsLease::acquire(hipStream_t stream, size_t bytes, void** ptr) {
    release();
    hipError_t e = hipSuccess;
    Slot* sl = slot_for(stream, &e);
    if (!sl) return e;
    sl->mu.lock();
    slot_ = sl;
    // The buffer's earlier uses were enqueued on this stream handle, so they
    // run before this call's work.  (A handle is only recycled once the
    // destroyed stream's work has completed and its object is released.)
    if (sl->cap < bytes) {
        if (sl->ptr) (void)ws_free(sl->ptr, stream);
        sl->ptr = nullptr;
        sl->cap = 0;
        // a little headroom, so that batches of slowly growing size do not
        // reallocate every time
        const size_t want = bytes + bytes / 8;
        e = ws_alloc(&sl->ptr, want, stream);
        if (e != hipSuccess) {
            sl->ptr = nullptr;
            return e;
        }
        sl->cap = want;
    }
    *ptr = sl->ptr;
    return hipSuccess;
}

void WsLease::release() {
    if (!slot_) return;
    slot_->mu.unlock();
    slot_ = nullptr;
}

}  // namespace frog
