/*
 * frog.h — C ABI of the MI355X (gfx950) range-filtered k-NN search library.
 *
 * The library implements the query-time path of FROG ("FROG: Efficient
 * Range-Filtering Approximate Nearest Neighbor Search on GPUs", arxiv
 * 2608.16491) on one AMD GPU, plus the host-side index construction that
 * produces its input and an exhaustive filtered search used as ground truth.
 *
 * Conventions for every entry point:
 *   - Return value: FROG_OK (0) or a negative FROG_E* code.  frog_last_error()
 *     returns a thread-local message for the last failure on the calling
 *     thread.  No C++ exception crosses this ABI and the library never exits
 *     the process.
 *   - Host pointers are read during the call only.  Device pointers ("d_")
 *     are caller-owned HIP device memory; they must stay valid until `stream`
 *     has executed the enqueued work.  `stream` is a hipStream_t passed as
 *     void* (NULL = the null stream).  Device entry points only ENQUEUE work
 *     and return; every argument error detectable on the host is reported
 *     before anything is enqueued.
 *   - Ranks: objects are renumbered by ascending attribute (ties by original
 *     index), so an attribute range [lo, hi] is the rank interval
 *     [#{a < lo}, #{a <= hi} - 1] (Sec 4).  Results report ORIGINAL object
 *     indices.  A NaN bound or lo > hi gives an empty range: not an error, the
 *     output row is padding.
 *   - Distances are SQUARED L2, accumulated in double from float inputs and
 *     rounded once to float; rows of results are ascending by (distance,
 *     rank).  Missing results (empty range, fewer than k reachable) are padded
 *     with id -1 and distance +inf.  Inputs must be finite.
 */
#ifndef FROG_H
#define FROG_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    FROG_OK = 0,
    FROG_EINVAL = -1,        /* bad argument (null pointer, size, parameter) */
    FROG_ENOMEM = -2,        /* host or device allocation failed */
    FROG_EHIP = -3,          /* a HIP runtime call failed; message has its text */
    FROG_EBADINDEX = -4,     /* index file: bad magic, version, size or checksum */
    FROG_ENOTUPLOADED = -5,  /* device entry point called before frog_index_upload */
    FROG_EIO = -6,           /* file could not be opened, read or written */
    FROG_EUNSUPPORTED = -7,  /* shape outside what the kernels are built for */
    FROG_ENOTPREPARED = -8   /* entry_mode 1 with a seed frog_index_prepare_sample has not built */
};

typedef struct frog_index frog_index_t; /* opaque; owns host and device copies */

/* Index construction parameters (Sec 6; defaults of Sec 8.1.4). */
typedef struct {
    int m;            /* expansion-neighbour candidates per vertex per layer: 16 (d<=300), 32 */
    int ef_c;         /* pool width of the construction-time greedy search: 128 (d<=300), 256 */
    int n_inv;        /* deepest segment-tree layers omitted: 7 (d<=300), 6 */
    int patience;     /* early-termination patience of the sibling search: 30 */
    int sib_seeds;    /* seeds of each sibling search (stratified over the sibling): 16 */
    int num_threads;  /* host threads; <= 0 means all available */
    double beta;      /* fusion-distance shrink, Eq. fusion-distance: 0.2 */
    double gamma;     /* fusion-distance decay: 0.5 */
    uint64_t seed;    /* seed of the sibling-search seed jitter: 0 */
} frog_build_params_t;

/* Query-time parameters of FROGSearch (Alg. 2). */
typedef struct {
    int epn;            /* entry points; minimum count when epn_frac > 0: 16 */
    double epn_frac;    /* 0: fixed epn; > 0: per-query count clamp(ceil(epn_frac*cnt), epn, epn_max) */
    int epn_max;        /* upper bound of the per-query count (ignored when epn_frac == 0) */
    int budget;         /* expansion budget B of ENIdentification (Alg. 4), 1..64: 16 */
    uint64_t seed;      /* entry-point jitter seed: 0 */
    int64_t query_base; /* batch index of query 0; keys the entry-point jitter: 0 */
    int hash_log2;      /* visited table of 2^hash_log2 slots in LDS (6..13): 10;
                           0 selects an exact visited set in device memory (slow;
                           used to count distinct evaluations) */
    void** phase_events;/* NULL, or 3 caller-created hipEvent_t recorded on `stream`:
                           entry_mode 0: before and after the search kernel (the
                           second and third together); entry_mode 1: before and
                           after the matrix-core entry scan, and after the
                           search kernels (pool and traversal) */
    int entry_mode;     /* how the entry points of Alg. 2 are drawn uniformly from
                           the range: 0 (default) one per stratum, jittered per
                           query; 1 every rank whose priority, a hash of (seed,
                           rank) shared by all queries, is below count/cnt of
                           its range: a sample of expected size count that
                           overlapping queries share, evaluated on matrix
                           cores in tiles of 16 queries.  Mode 1 reads the
                           seed's level lists, which frog_index_prepare_sample
                           must have built (else FROG_ENOTPREPARED) */
    int hotspot_mode;   /* ablation of HotspotLocalization (Sec 8.2.3): 0 (default)
                           layers L_start..L_end of Alg. 3; 1 layers
                           L_start..H-1 (no end condition); 2 all layers */
    int eager_check;    /* ablation of the lazy visited check: 1 checks (and
                           marks) visited candidates inside ENIdentification,
                           so visited ones do not count against the budget;
                           needs the exact visited set (hash_log2 = 0) */
} frog_search_params_t;

/* Per-query statistics written by frog_search_ex (int32, FROG_STAT_N per query). */
enum {
    FROG_STAT_EXPANSIONS = 0, /* pool entries expanded */
    FROG_STAT_EN = 1,         /* sum over expansions of |EN(u)| */
    FROG_STAT_DIST = 2,       /* distance evaluations performed (entry points included) */
    FROG_STAT_SCANNED = 3,    /* ENC entries of the hotspot layers Alg. 4 examined */
    FROG_STAT_ENTRY = 4,      /* entry points */
    FROG_STAT_LSTART = 5,     /* hotspot first layer (Alg. 3) */
    FROG_STAT_LEND = 6,       /* hotspot last layer */
    FROG_STAT_LOADED = 7,     /* ENC entries actually loaded by the kernel */
    FROG_STAT_SCANROWS = 8,   /* entry_mode 1: rows the shared entry scan read, each
                                 tile's rows credited to the query of its first slot
                                 (a query has a tile per window its run meets), so the
                                 column sums to the scan's rows; 0 in entry_mode 0 */
    FROG_STAT_FALLBACK = 9,   /* entry_mode 1: 1 if the margin test could not prove the
                                 scan's candidates hold the L nearest sample points, so
                                 the whole sample was evaluated exactly (0 otherwise) */
    FROG_STAT_N = 10
};

/* Fill *p with the paper's defaults for dimension d. */
void frog_build_params_default(int d, frog_build_params_t* p);
void frog_search_params_default(frog_search_params_t* p);

/* Build the index on the host (Sec 6: attribute-rank domain, leaf brute force,
 * bottom-up layers with child m-ANN + sibling greedy search (Alg. 1 with
 * patience), RNG-pruned temporary graphs, fusion re-rank into the n x H x m
 * candidate array of Sec 4).  X: n x d floats, row-major, original order;
 * attr: n doubles (no NaN).  p = NULL uses frog_build_params_default(d).  On
 * success *out owns a host index (not yet on a device). */
int frog_build_index(const float* X, const double* attr, int64_t n, int d,
                     const frog_build_params_t* p, frog_index_t** out);

/* The same construction on HIP device `device`: the host sorts by attribute
 * and tabulates the fusion-distance factors; the leaf brute force and every
 * layer (child m-ANN, sibling greedy search with patience, RNG prune, fusion
 * re-rank; Sec 6, Alg. 1) run as kernels, one wavefront per vertex, with the
 * construction's distances (dimension order, double accumulation, one
 * rounding), so the candidate array equals frog_build_index's entry for
 * entry.  X, attr: host arrays as for frog_build_index.  On success *out owns
 * a host index whose device copy (fp32 rows) is already uploaded on `device`.
 * Errors: as frog_build_index; FROG_EUNSUPPORTED unless d <= 1024, m <= 32,
 * ef_c <= 256 and sib_seeds <= 64; FROG_EHIP / FROG_ENOMEM from the device.
 * p->num_threads only sizes the host part. */
int frog_build_index_gpu(const float* X, const double* attr, int64_t n, int d,
                         const frog_build_params_t* p, int device, frog_index_t** out);

/* Work of the GPU construction that made idx: distances evaluated,
 * sibling-search expansions, and the time from its first kernel's start to
 * its last one's end in milliseconds (all 0 for a host-built index; any
 * pointer may be NULL). */
int frog_index_build_stats(const frog_index_t* idx, int64_t* distances, int64_t* expansions,
                           double* kernel_ms);

/* Wrap already-built arrays (copied): X_rank n x d floats in rank order,
 * attr_sorted n ascending doubles, perm n ints (rank -> original index, a
 * permutation), ENC n x H x m ints (each entry -1 or a rank).  Validates sizes,
 * the permutation, the ordering of attr_sorted and the entry range. */
int frog_index_from_arrays(const float* X_rank, const double* attr_sorted,
                           const int32_t* perm, const int32_t* ENC,
                           int64_t n, int d, int H, int m, frog_index_t** out);

/* Copy the host arrays out (any pointer may be NULL to skip it). */
int frog_index_export(const frog_index_t* idx, float* X_rank, double* attr_sorted,
                      int32_t* perm, int32_t* ENC);
int frog_index_info(const frog_index_t* idx, int64_t* n, int* d, int* H, int* m);

/* Index file: header (magic, version, n, d, H, m), the four arrays, CRC-32 of
 * everything before it.  Load reports FROG_EBADINDEX on any mismatch. */
int frog_index_save(const frog_index_t* idx, const char* path);
int frog_index_load(const char* path, frog_index_t** out);

/* Copy the index to HIP device `device` (the HBM layout: X rows in rank order,
 * padded to a multiple of 32 floats; ENC n x H x m; attr_sorted; perm).  The
 * device copy is read-only afterwards, so concurrent searches on different
 * streams are safe.  Calling it again replaces the previous device copy and
 * drops every prepared sample (no search may be running then). */
int frog_index_upload(frog_index_t* idx, int device);

/* The shared entry sample of `seed` for entry_mode 1 (the second reading of
 * Alg. 2's uniform sampling: rank i is drawn when its priority
 * hi32(splitmix64(splitmix64(seed) ^ i)) is below the query's threshold).
 * Builds, on the index's device, for levels j = 1..~log2(n) the ascending
 * ranks whose priority is below 2^(32-j), a copy of their stored rows in the
 * same order, and every rank's priority and squared row norm: about
 * n * (4 dp + 20) bytes of device memory for fp32 rows (n * (2 dp + 20) for
 * 16-bit rows), 0.53 GB at n = 1M, d = 128.  Synchronous (it waits for the
 * device); idempotent (a prepared seed returns at once); safe to call while
 * other threads search with other seeds.  The lists are immutable once built
 * and freed with the device copy (frog_index_upload again, or
 * frog_index_free).  Errors: FROG_ENOTUPLOADED, FROG_ENOMEM, FROG_EHIP. */
int frog_index_prepare_sample(frog_index_t* idx, uint64_t seed);

/* Storage type of the device copy's rows. */
enum {
    FROG_STORAGE_F32 = 0,  /* fp32 rows, dp = d rounded up to a multiple of 32 */
    FROG_STORAGE_F16 = 1,  /* IEEE binary16 rows (round to nearest even), dp = d
                              rounded up to a multiple of 64, d <= 128 */
    FROG_STORAGE_BF16 = 2  /* bfloat16 rows (the upper half of the fp32 value,
                              round to nearest even), same padding and limit */
};

/* As frog_index_upload, with the rows stored as `storage` (FROG_STORAGE_*).
 * The paper keeps the vectors in half precision on the device (Sec 8.1); with
 * fp16 or bf16 rows the search returns the exact FROGSearch result over the
 * rounded vectors:
 * each row is rounded once on the host, converted exactly to fp32 in the
 * kernels, and distances are accumulated as for fp32 rows.  Queries stay
 * fp32.  The host copy keeps the fp32 rows (export and save are unchanged).
 * Errors: FROG_EINVAL for an unknown storage value, FROG_EUNSUPPORTED for
 * 16-bit rows with d > 128 or a value whose rounding overflows the format
 * (or is not finite).  A 16-bit device copy serves frog_search /
 * frog_search_ex (both entry modes) and frog_rank_bounds;
 * frog_bruteforce_filtered needs fp32 rows and returns FROG_EUNSUPPORTED. */
int frog_index_upload_ex(frog_index_t* idx, int device, int storage);
/* Release host and device memory.  NULL is a no-op. */
void frog_index_free(frog_index_t* idx);

/* Range -> rank interval (Sec 4) for nq queries: d_lr[2i] = l, d_lr[2i+1] = r
 * (int32; l > r when empty). */
int frog_rank_bounds(const frog_index_t* idx, const double* d_lo, const double* d_hi,
                     int64_t nq, int32_t* d_lr, void* stream);

/* FROGSearch (Alg. 2 with HotspotLocalization, Alg. 3, and ENIdentification,
 * Alg. 4) for nq queries with default parameters.  d_queries: nq x d floats
 * row-major; d_lo/d_hi: nq doubles; k >= 1, L in [k, 256] (pool size ef_s);
 * outputs d_ids (int32) and d_dists (float), nq x k each. */
int frog_search(const frog_index_t* idx, const float* d_queries, int64_t nq,
                const double* d_lo, const double* d_hi, int k, int L,
                int32_t* d_ids, float* d_dists, void* stream);

/* As frog_search with explicit parameters (p = NULL: defaults) and optional
 * per-query statistics d_stats (NULL or nq x FROG_STAT_N int32).  With
 * p->entry_mode == 1 the seed's sample must be prepared
 * (frog_index_prepare_sample), else FROG_ENOTPREPARED; nothing is built or
 * freed here, so searches on several streams or threads may share an index
 * whatever their seeds.  The per-call workspace (counters, rank intervals,
 * chunk pools; in entry_mode 1 plans, tiles, candidate lists and pools: about
 * 13.5 KB per query at L <= 40, sized for the worst case) is a device buffer the library
 * keeps per (device, stream) for the life of the process, grown
 * stream-ordered when a call needs more, so repeated calls allocate nothing;
 * threads enqueueing on one stream take turns, other streams have their own
 * buffer. */
int frog_search_ex(const frog_index_t* idx, const float* d_queries, int64_t nq,
                   const double* d_lo, const double* d_hi, int k, int L,
                   const frog_search_params_t* p, int32_t* d_ids, float* d_dists,
                   int32_t* d_stats, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): exactly
 * frog_search_ex (same arguments, same results, same errors), except that the
 * per-call workspace (work counters, rank intervals, chunk pools; in
 * entry_mode 1 the plans, tiles, candidate lists and pools) lives in a fixed
 * 256 MiB array of device memory inside the library instead of coming from
 * hipMallocAsync.  Nothing is allocated or freed by this call.
 *   - Each GPU the library runs on holds its own array until the process
 *     ends; its address is looked up once per device, on the first call there.
 *   - Every call on a GPU shares that GPU's array, and the array keeps the
 *     last call's contents (the kernels clear what must start at zero):
 *     calls that overlap on one GPU (other streams, other threads) race and
 *     must be serialised by the caller.
 *   - A call whose workspace exceeds 256 MiB is refused with FROG_EUNSUPPORTED
 *     before anything is enqueued.  Roughly: entry_mode 0 needs 12 bytes per
 *     query plus, when the entry count exceeds one 768-point chunk,
 *     512 * ceil(L/64) bytes per chunk (about 2 KB per query at 2,560 entry
 *     points and L <= 64); entry_mode 1 at n = 1M about 13.5 KB per query at
 *     L <= 40 (about 19,700 queries per call), 17.6 KB up to L = 56, 34.5 KB
 *     up to L = 120 and 35 KB up to L = 256, plus about 2 MB; the exact
 *     visited set (hash_log2 = 0) adds n/8 bytes per resident wavefront and
 *     is refused at realistic n.
 *   - entry_mode 1 needs the seed prepared (frog_index_prepare_sample). */
int frog_search_noalloc(const frog_index_t* idx, const float* d_queries, int64_t nq,
                        const double* d_lo, const double* d_hi, int k, int L,
                        const frog_search_params_t* p, int32_t* d_ids, float* d_dists,
                        int32_t* d_stats, void* stream);

/* Exhaustive filtered k-NN (Def. 2, RFANNS): the exact k nearest objects whose
 * attribute lies in [lo, hi], by (distance, rank), padded with (-1, +inf).
 * The dot products q.x run on fp32 matrix cores; a per-query margin test
 * proves that the candidates re-ranked with the exact squared distance hold
 * the result; a query the test cannot certify is recomputed over every rank
 * of its range with the exact distance.  Every row is exact.  1 <= k <= 256.
 * d_certified (NULL or nq int32) tells how each row was obtained: 1 = by the
 * margin test (or an empty range), 2 = by the exhaustive exact pass.  The
 * ranges and the certification are read back to the host, so this call
 * synchronises `stream`; it is a ground-truth tool, not the search path. */
int frog_bruteforce_filtered(const frog_index_t* idx, const float* d_queries, int64_t nq,
                             const double* d_lo, const double* d_hi, int k,
                             int32_t* d_ids, float* d_dists, int32_t* d_certified,
                             void* stream);

/* Message of the last failure on this thread ("" if none). */
const char* frog_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* FROG_H */
