/*
 * rsc.h - C ABI of the MI355X (gfx950) implementation of the RSC
 * aggregation hot path: the GCN aggregation SpMM Y = A_hat * H and its
 * top-k column-row approximation (score pairs, keep the top k, slice the
 * kept columns out of the CSR matrix, cache the slice, run SpMM on it);
 * also the unbiased randomized column-row sampler, the MEAN-aggregator
 * operand, the layer-wise budget allocation and a CSR validity check.
 *
 * Paper: Liu et al., "RSC: Accelerate Graph Neural Networks Training via
 * Randomized Sparse Computations", ICML 2023 (arXiv 2210.10737).
 *
 * Conventions
 *   - Pointers are DEVICE pointers unless the name ends in _host.
 *   - Every call that takes a stream enqueues its work on that stream and
 *     returns without synchronising, unless it is marked [sync].
 *   - Arguments are validated on the host before anything is enqueued; a
 *     call that returns an error has enqueued nothing and changed no output
 *     or cache state, except where stated.
 *   - The caller owns every buffer it passes. Buffers returned by
 *     rsc_cache_get are borrowed from the cache.
 *   - Dense matrices are row-major fp32 with a leading dimension (in floats)
 *     ld >= d, ld % 4 == 0, and a 16-byte-aligned base pointer. Columns
 *     d .. ld-1 of an output are never written.
 *   - CSR matrices: int32 row pointers and column indices, fp32 values,
 *     nnz < 2^31, columns strictly increasing within each row.
 *   - No C++ exception crosses this interface. Asynchronous device faults
 *     surface at the caller's next synchronisation.
 *   - Stateless calls are reentrant; a cache handle must not be used from
 *     two host threads at once, and two calls that share a workspace must
 *     not overlap on the device. The calls on one cache share its internal
 *     buffers and workspaces, so they must be ordered on the device (one
 *     stream, or events between streams).
 *   - A plan or cache lives on the device that was current when it was
 *     made; a call that launches work for it with another device current
 *     returns RSC_ERR_INVALID_ARGUMENT.
 */
#ifndef RSC_H
#define RSC_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RSC_ABI_VERSION 5

typedef enum {
    RSC_OK = 0,
    RSC_ERR_INVALID_ARGUMENT = 1, /* null pointer, d < 1, k < 0, k > n, ld < d ... */
    RSC_ERR_UNSUPPORTED = 2,      /* nnz >= 2^31, ld % 4 != 0, misaligned base pointer */
    RSC_ERR_OUT_OF_MEMORY = 3,    /* a device allocation by the cache failed */
    RSC_ERR_CAPACITY = 4,         /* caller-provided buffer or workspace too small */
    RSC_ERR_NO_DEVICE = 5,        /* no HIP device visible */
    RSC_ERR_HIP = 6,              /* a HIP runtime call failed; see rsc_last_error() */
    RSC_ERR_INTERNAL = 7
} rsc_status_t;

/* A CSR matrix in device memory (section 3.3.1: the entries of row i are
 * Col/Val[Rowptr[i] .. Rowptr[i+1]-1]). rowptr has n_rows + 1 entries with
 * rowptr[0] = 0 and rowptr[n_rows] = nnz. */
typedef struct {
    int32_t n_rows;
    int32_t n_cols;
    int64_t nnz;
    const int32_t *rowptr;
    const int32_t *col;
    const float *val;
} rsc_csr_t;

/* Human-readable name of a status code (static storage). */
const char *rsc_status_string(rsc_status_t status);
/* Detail of the last error raised on the calling host thread (thread-local;
 * empty string if none). */
const char *rsc_last_error(void);
/* RSC_ABI_VERSION of the loaded library. */
int32_t rsc_abi_version(void);

/* CSR well-formedness (the form section 3.3.1's Rowptr/Col/Val describe,
 * with sorted unique columns so that column norms are well defined):
 * rowptr[0] = 0, rowptr[n_rows] = nnz, rowptr non-decreasing, every col in
 * [0, n_cols), columns strictly increasing within each row. [sync] Checked
 * on the device in O(nnz); a row's entries are read only once its bounds are
 * in range. Returns RSC_OK (and *bad_row_host = -1 if given) or
 * RSC_ERR_INVALID_ARGUMENT with *bad_row_host = the first offending row.
 * With the environment variable RSC_VALIDATE=1, every entry point that takes
 * a caller's CSR (rsc_spmm, rsc_col_sqnorms, rsc_degree_scale,
 * rsc_slice_csr, rsc_cache_create) runs this check first and returns its
 * error without launching anything else. */
rsc_status_t rsc_csr_validate(const rsc_csr_t *A, int64_t *bad_row_host, hipStream_t stream);

/* ---------------------------------------------------------------- A1 --- */
/* Exact sparse-dense product Y = A * B (the SpMM of Eq. 1's implementation
 * form, section 2.1; the forward aggregation of section 3.1).
 *   A: n_rows x n_cols CSR.  B: n_cols x d, leading dimension ldb.
 *   Y: n_rows x d, leading dimension ldy; every row is written (empty rows
 *      get zeros).
 * Accumulation: fp32 over runs of at most 64 consecutive entries, folded
 * into fp64; one rounding to fp32 per output. Features up to 128 wide take
 * a lane layout that gathers several entries per load, and the features may
 * be processed in several passes of 32/64 columns of B (both chosen from
 * n_rows, nnz, n_cols and d only, with the environment variable
 * RSC_SPMM_SLICE = 16/32/64/128/256 as an override); the layout sets the
 * summation order. Rows may be
 * taken longest first (when rows are long on average; RSC_SPMM_ORDER = 0/1
 * overrides), which never changes a result. Column-blocked mode: the
 * features are taken in passes of 16, 32 or 64 floats (the narrowest that
 * holds d; wider d in 64-float passes); when that slice of the referenced B
 * rows spans 2..16 ranges of about 4.5 MiB and rows hold at least 56, 112 or
 * 224 entries per range on average (64-, 32-, 16-float passes), the columns
 * are cut into P = min(8, ranges) equal index ranges processed one after
 * another (the gathered B rows then stay in L2, or mostly so for ranges of
 * up to two L2 sizes); each row's entries in one range are summed as above and rounded
 * to an fp32 partial, and the P partials are added in fp64 in range order
 * and rounded once (RSC_SPMM_BLOCKED = 0 switches it off, 2..8 forces that
 * P). Deterministic: equal arguments give bitwise equal Y, and
 * rsc_spmm_sampled with every column kept reproduces rsc_spmm bitwise.
 * ws / ws_bytes: scratch of at least rsc_spmm_workspace_bytes(A) bytes,
 * 256-byte aligned, private to this call until it completes on `stream`. */
size_t rsc_spmm_workspace_bytes(const rsc_csr_t *A);
rsc_status_t rsc_spmm(const rsc_csr_t *A, const float *B, int32_t d, int64_t ldb, float *Y,
                      int64_t ldy, void *ws, size_t ws_bytes, hipStream_t stream);

/* rsc_spmm for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation): the
 * same product with no workspace argument and no allocation. Its scratch is
 * a static 32 MiB device array inside the library, one per GPU, held until
 * the process ends; a product needs 512 bytes plus 4 max(n_rows,
 * min(8 n_rows, nnz / 1025)) bytes of it (about 8.3M rows at most), beyond
 * which the call returns RSC_ERR_CAPACITY without launching. A product whose
 * column-blocked buffers do not also fit runs unblocked (then Y may differ
 * from rsc_spmm's within rounding; otherwise it is bitwise equal). Every
 * call on one GPU uses that GPU's scratch, which keeps the last call's
 * contents (the call clears what it needs): calls that overlap on one GPU
 * (two streams, or two host threads) race and give wrong results, so order
 * them on the device. RSC_VALIDATE does not apply (the check allocates). */
rsc_status_t rsc_spmm_noalloc(const rsc_csr_t *A, const float *B, int32_t d, int64_t ldb, float *Y,
                              int64_t ldy, hipStream_t stream);

/* Plan for repeated exact products with one sparse operand (a training
 * run's static A_hat). Same product, same kernels, same summation order as
 * rsc_spmm: rsc_spmm_plan_run gives Y bitwise equal to rsc_spmm on the same
 * arguments (with the RSC_SPMM_* switches as they were when the plan was
 * made; a plan whose workspace cannot hold a later switch's column-blocked
 * buffers runs unblocked). What the plan adds is per-matrix preparation,
 * done once:
 *   - its own workspace, so runs need none;
 *   - when the product runs column-blocked, the split bounds of the rows
 *     (for the range count of feature widths above 32; a run at a width
 *     whose range count differs builds its own, as rsc_spmm does, and so
 *     does every later run of the plan);
 *   - the long-row list (or the length-class row order) and its length,
 *     which every rsc_spmm call builds first;
 *   - for operands with more than 262,144 columns, a copy of col whose bit
 *     31 marks the "hub" columns, the columns of highest entry count that
 *     together hold just under half of the entries (entry-weighted median of
 *     the column counts, on a scale of 8 steps per octave). When one feature
 *     pass gathers from more than 512 MiB of B rows (far beyond the on-chip
 *     caches), the other columns' rows are gathered non-temporally, so the
 *     hubs' rows stay in L2. This changes cache allocation only, never a
 *     value; RSC_SPMM_HINT=0 switches the policy off.
 * rsc_spmm_plan_create [sync] borrows A's arrays (they must outlive the plan
 * and not change) and allocates 4 nnz bytes for the copy, 4 (P+1) n_rows
 * bytes for the split bounds and the workspace (stream-ordered, on `stream`);
 * RSC_ERR_OUT_OF_MEMORY if that fails. Runs of one plan share its workspace, so they must be
 * ordered on the device. The sampled-matrix cache prepares each new slice's
 * row list the same way at refresh time; its sampled products do not take
 * the column hint (on the cached slices it measured slower). */
typedef struct rsc_spmm_plan rsc_spmm_plan_t;
rsc_status_t rsc_spmm_plan_create(const rsc_csr_t *A, hipStream_t stream, rsc_spmm_plan_t **out);
rsc_status_t rsc_spmm_plan_run(rsc_spmm_plan_t *plan, const float *B, int32_t d, int64_t ldb, float *Y,
                               int64_t ldy, hipStream_t stream);
/* rsc_spmm_plan_destroy waits (on the host) for the plan's own runs on
 * every stream they used (runs captured into a HIP graph excepted: the
 * caller synchronises those launches), then frees the plan's memory,
 * stream-ordered; work on other streams is not waited for. NULL is a no-op. */
rsc_status_t rsc_spmm_plan_destroy(rsc_spmm_plan_t *plan);

/* Measurement helper, not a step of the method: the gather-only pass of the
 * plan's exact product. Streams the plan's column indices (its hinted copy
 * when it has one) in stored order, 64 entries per wave, and loads each
 * referenced row of B with the lane layout, feature passes and cache policy
 * an unblocked run of the plan takes for this d (rows are not walked, no
 * values are read); the loaded values are summed and one float per 64
 * entries is written to sink (sink_count >= ceil(nnz / 64)), only so that no
 * load is dropped. inflight (4, 8 or 16): loads each wave issues before
 * consuming any. Its duration bounds how fast the product's own gather
 * pattern can run, the "gather ceiling" of the product.
 * Y (nullable; n_rows x d, ldy, checked like rsc_spmm's Y): also write an
 * output of the product's size with the product's store pattern, the rows
 * shared evenly over the waves, each wave's after its gathers. Y's contents
 * afterwards are unspecified (not the product); nothing is written when A
 * has no entries. The duration then bounds the gathers plus the output
 * stream. *slice_out (nullable) receives the feature-pass width used. Runs
 * are tracked for rsc_spmm_plan_destroy like rsc_spmm_plan_run. */
rsc_status_t rsc_spmm_plan_gather_probe(rsc_spmm_plan_t *plan, const float *B, int32_t d, int64_t ldb,
                                        int32_t inflight, float *sink, int64_t sink_count, float *Y,
                                        int64_t ldy, int32_t *slice_out, hipStream_t stream);

/* MEAN aggregator operand (appendix A.3: SpMM_MEAN(A, H) = D^-1 A H, D the
 * degree matrix of A, D_ii = stored entries of row i). Writes A's values
 * divided by a degree into val_out (nnz entries, same structure as A), each
 * fp32(val / deg) computed in fp64 and rounded once; a zero degree gives 0.
 *   by_column = 0: deg = the length of the entry's own row -> D^-1 A, the
 *     forward operand (deg_rowptr unused, may be NULL);
 *   by_column = 1: deg = deg_rowptr[c+1] - deg_rowptr[c] for the entry's
 *     column c -> pass the CSR of A^T as A and A's rowptr as deg_rowptr to
 *     get A^T D^-1 = (D^-1 A)^T, the backward operand.
 * rsc_spmm on the result is SpMM_MEAN; the cache and sampled SpMM apply to it
 * unchanged (its column norms come from the CSR of its transpose). */
rsc_status_t rsc_degree_scale(const rsc_csr_t *A, const int32_t *deg_rowptr, int32_t by_column,
                              float *val_out, hipStream_t stream);

/* ---------------------------------------------------------------- A2 --- */
/* Column square-norms of a sparse operand X (Eq. 3's ||X[:, i]||^2; the
 * ||A_hat^T[:, i]||^2 of Eq. 4a). Pass the CSR of X^T: column i of X is
 * row i of X^T. cn2[i] = sum of val^2 over row i of XT, fp64, in stored
 * order. colnnz (nullable) receives the entry count of each column of X
 * (Eq. 4b's #nnz_i). Both have XT->n_rows entries. */
rsc_status_t rsc_col_sqnorms(const rsc_csr_t *XT, double *cn2, int32_t *colnnz,
                             hipStream_t stream);

/* ---------------------------------------------------------------- A3 --- */
/* Pair keys (Eq. 3 and the top-k rule of section 2.2.1). For i < n:
 *   rn2[i] = sum_{j<d} B[i, j]^2 (fp64, ascending j)
 *   q[i]   = cn2[i] * rn2[i]       (fp64)
 *   key[i] = isnan(q) ? 0 : bits(q) + 1   (unsigned order == order of q,
 *            NaN last)
 *   score[i] = fl32(sqrt(q[i]))    (nullable output)
 *   rn2 (nullable output, fp64[n]) receives rn2[i]; its sum is ||B||_F^2,
 *   the normaliser of Eq. 4a.
 * q is the squared pair score ||X[:, i]||^2 ||B[i, :]||^2 without the
 * common normaliser, which changes no ranking. B is n x d with leading
 * dimension ldb. */
rsc_status_t rsc_pair_scores(const double *cn2, const float *B, int32_t n, int32_t d,
                             int64_t ldb, uint64_t *key, float *score, double *rn2,
                             hipStream_t stream);

/* ---------------------------------------------------------------- A4 --- */
/* Top-k selection (section 2.2.1): the k indices with the largest keys,
 * ties broken by the lower index. idx receives them in ascending order
 * (k entries); mask receives ceil(n/32) words, bit (i & 31) of word i >> 5
 * set iff i is selected. 0 <= k <= n. Any uint64 keys are accepted.
 * ws: at least rsc_topk_workspace_bytes(n) bytes, 256-byte aligned. */
size_t rsc_topk_workspace_bytes(int32_t n);
rsc_status_t rsc_topk_select(const uint64_t *key, int32_t n, int32_t k, int32_t *idx,
                             uint32_t *mask, void *ws, size_t ws_bytes, hipStream_t stream);

/* ---------------------------------------------------------------- A5 --- */
/* Column slice A' = A[:, S] (section 3.3.1, Fig. 5's rebuild of Rowptr and
 * Col; appendix C: whole columns dropped, every row kept). Entries whose
 * column has its mask bit set are kept in their original order; column ids
 * stay global; rowptr_out (n_rows + 1 entries) is the running count of kept
 * entries; rows may become empty.
 * colw (nullable, fp64[n_cols]): per-column scale; when given, each kept
 * value becomes fl32(val * colw[col]) (fp64 product, one rounding), as the
 * randomized sampler's 1/(k p) weighting needs.
 * nnz_out: device int64 receiving nnz'. The slice runs as a stream
 * compaction in four launches (a tile-to-row table, count, scan, emit;
 * RSC_SLICE_PAIRED=0 turns off the count's block pairing for masks of
 * 1.28M to 2.56M columns, which changes only its speed);
 * with the environment variable RSC_SLICE_FUSED=1 it runs as one fused
 * kernel instead (count, a decoupled look-back scan over tiles taken in
 * ticket order, compaction). Both give the same bytes. The fused kernel's
 * waits are bounded: if one ever ran out, *nnz_out would be -1 and
 * rsc_slice_csr's synchronous form and rsc_cache_get would return
 * RSC_ERR_INTERNAL.
 * capacity: entries available in col_out / val_out. If capacity >= A->nnz
 * the call is asynchronous. Otherwise it is [sync]: entries beyond capacity
 * are not written, and RSC_ERR_CAPACITY is returned when nnz' > capacity
 * (rowptr_out and *nnz_out are still complete).
 * ws: at least rsc_slice_workspace_bytes(A) bytes, 256-byte aligned. */
size_t rsc_slice_workspace_bytes(const rsc_csr_t *A);
rsc_status_t rsc_slice_csr(const rsc_csr_t *A, const uint32_t *mask, const double *colw,
                           int32_t *rowptr_out, int32_t *col_out, float *val_out, int64_t capacity,
                           int64_t *nnz_out, void *ws, size_t ws_bytes, hipStream_t stream);

/* -------------------------------------------- randomized sampling --- */
/* Unbiased column-row sampling (section 2.2, Eq. 2 with the probabilities
 * of Eq. 3), the alternative to top-k: k i.i.d. draws i_t ~ p over the n
 * pairs, p_i proportional to ||X[:, i]|| ||B[i, :]|| = sqrt(q_i) (q decoded
 * from the rsc_pair_scores key; NaN -> 0), each drawn pair scaled by
 * 1/(k p_{i_t}), so E[approx] = X B. Exactly:
 *   w_i = floor(sqrt(q_i) * 2^S / max_j sqrt(q_j)) (int64; S = 38 for
 *         n <= 2^24, else 62 - ceil(log2 n), so total <= 2^62; if some score
 *         is +Inf the infinite ones get 2^S and the rest 0), W = inclusive
 *         prefix sum of w, total = W[n-1];
 *   draw t (0 <= t < k): z = t-th output of SplitMix64 seeded with `seed`
 *         (Steele, Lea & Flood 2014), u = floor(z * total / 2^64),
 *         i_t = smallest i with W[i] > u;
 *   count[i] = draws of i; colw[i] = count[i] * total / (k * w_i) (fp64,
 *         0 if not drawn); mask bit i set iff count[i] > 0.
 * All decisions are integer, so results are bitwise reproducible. If every
 * weight is 0 nothing is drawn. ws: rsc_sample_workspace_bytes(n) bytes,
 * 256-byte aligned. */
size_t rsc_sample_workspace_bytes(int32_t n);
rsc_status_t rsc_sample_columns(const uint64_t *key, int32_t n, int32_t k, uint64_t seed,
                                int32_t *count, double *colw, uint32_t *mask, void *ws,
                                size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------ A6 / A7 --- */
/* Sampled-matrix cache (section 3.3.1): keeps the sliced operand and reuses
 * it across nearby steps; refreshed every `refresh_interval` steps (10 in
 * section 5.1). The cache owns its device buffers (sized for the full
 * operand, so refreshes never reallocate) until rsc_cache_destroy.
 *   rsc_cache_create [sync]: X is the sparse operand to be sliced, XT the
 *     CSR of its transpose (for the column norms; pass X again for a
 *     symmetric operand). Computes cn2 and colnnz once (the operand is
 *     fixed across steps). X and XT must stay valid for the cache's life.
 *   rsc_cache_refresh: scores the pairs against B (n_cols x d, ldb), keeps
 *     the top k columns and slices X; records `step` as the refresh step.
 *     It is rsc_cache_score followed by rsc_cache_select.
 *   rsc_cache_score: only computes the pair keys and the rows' square-norms
 *     against B into the cache (readable through rsc_cache_buffers), leaving
 *     the current slice in place; used when k comes from the keys of several
 *     operands, as in the layer-wise allocation of section 3.2.
 *   rsc_cache_select: top k of the keys last scored, then the slice; records
 *     `step` as the refresh step (RSC_ERR_INVALID_ARGUMENT if nothing was
 *     scored yet).
 *   rsc_cache_refresh_random: scores against B, then the randomized sampler
 *     (rsc_sample_columns: k_draws draws with `seed`) instead of top-k, and
 *     the slice with each kept column scaled by its colw; rsc_cache_get then
 *     reports k = k_draws and no index list (idx_out = NULL).
 *   rsc_cache_get (host only): returns the current slice (its nnz is read
 *     from the device once per refresh, waiting for the refresh if needed),
 *     the ascending kept indices, k, the slice version (0 = never
 *     refreshed, +1 per refresh) and needs_refresh = (never refreshed) or
 *     (step - last_refresh_step >= refresh_interval). The returned pointers
 *     stay valid until the next refresh or destroy.
 *   rsc_spmm_sampled: Y' = X[:, S] * B on the cached slice (Eq. 2 with the
 *     top-k rule: kept pairs summed with scale 1), the same kernels as
 *     rsc_spmm; every row of Y' is written. Needs a refreshed cache. Each
 *     selection prepares the products for the feature width of the operand
 *     last scored (row list, or split bounds when column-blocked); a
 *     product of another width whose preparation differs builds its own,
 *     and so does every later product until the next selection. */
typedef struct rsc_cache rsc_cache_t;
rsc_status_t rsc_cache_create(const rsc_csr_t *X, const rsc_csr_t *XT, int32_t refresh_interval,
                              hipStream_t stream, rsc_cache_t **out);
/* Device memory provider for a cache (for example a framework's caching
 * allocator): alloc returns device memory of at least `bytes` bytes,
 * 256-byte aligned, usable on `stream`, or NULL; free releases it. Both are
 * called on the calling host thread, only inside rsc_cache_create_ex (and its
 * failure path) and rsc_cache_destroy, with the create call's stream. */
typedef struct {
    void *(*alloc)(size_t bytes, hipStream_t stream, void *ctx);
    void (*free)(void *ptr, hipStream_t stream, void *ctx);
    void *ctx;
} rsc_allocator_t;
/* rsc_cache_create with the cache's device buffers taken from `allocator`
 * (NULL: the stream-ordered hipMallocAsync on `stream`, freed with
 * hipFreeAsync once the cache's work is done, so neither waits for other
 * streams; memory freed this way returns to the device's default pool and
 * is released at a later synchronisation). A pointer from alloc that is NULL gives
 * RSC_ERR_OUT_OF_MEMORY; one that is not 256-byte aligned gives
 * RSC_ERR_UNSUPPORTED (both after freeing what was taken). The allocator
 * struct is copied; ctx must stay valid until rsc_cache_destroy. */
rsc_status_t rsc_cache_create_ex(const rsc_csr_t *X, const rsc_csr_t *XT, int32_t refresh_interval,
                                 const rsc_allocator_t *allocator, hipStream_t stream, rsc_cache_t **out);
rsc_status_t rsc_cache_refresh(rsc_cache_t *cache, const float *B, int32_t d, int64_t ldb,
                               int32_t k, int64_t step, hipStream_t stream);
rsc_status_t rsc_cache_score(rsc_cache_t *cache, const float *B, int32_t d, int64_t ldb,
                             hipStream_t stream);
rsc_status_t rsc_cache_select(rsc_cache_t *cache, int32_t k, int64_t step, hipStream_t stream);
rsc_status_t rsc_cache_refresh_random(rsc_cache_t *cache, const float *B, int32_t d, int64_t ldb,
                                      int32_t k_draws, uint64_t seed, int64_t step,
                                      hipStream_t stream);
rsc_status_t rsc_cache_get(rsc_cache_t *cache, int64_t step, rsc_csr_t *slice_out,
                           const int32_t **idx_out, int32_t *k_out, int32_t *needs_refresh_out,
                           uint64_t *version_out);
rsc_status_t rsc_spmm_sampled(rsc_cache_t *cache, const float *B, int32_t d, int64_t ldb,
                              float *Y, int64_t ldy, hipStream_t stream);
/* Measurement helper, not a step of the method: the gather-only pass of
 * rsc_spmm_sampled on the cached slice, as rsc_spmm_plan_gather_probe is for
 * a plan (the slice's column stream, the feature passes the sampled product
 * takes, no hint; rows not walked, no values; one float per 64 kept
 * entries into sink, sink_count >= ceil(nnz' / 64); Y nullable, the
 * product's n_rows x d output stream as for a plan). Needs a refreshed
 * cache; reads nnz' like rsc_cache_get. */
rsc_status_t rsc_cache_gather_probe(rsc_cache_t *cache, const float *B, int32_t d, int64_t ldb,
                                    int32_t inflight, float *sink, int64_t sink_count, float *Y,
                                    int64_t ldy, int32_t *slice_out, hipStream_t stream);
/* Device arrays owned by the cache: cn2 (fp64) and colnnz (int32), n_cols
 * entries each; keys (uint64) and row square-norms rn2 (fp64) of the last
 * scored operand; mask (ceil(n_cols/32) words) of the last selection. Any
 * output pointer may be NULL. */
rsc_status_t rsc_cache_buffers(rsc_cache_t *cache, const double **cn2, const int32_t **colnnz,
                               const uint64_t **key, const double **rn2, const uint32_t **mask);
/* The Frobenius normalisers of Eq. 4a: *fro_x2_host = ||X||_F^2 = the sum of
 * the column square-norms cn2 (computed at create), *fro_b2_host =
 * ||B||_F^2 = the sum of the row square-norms rn2 of the operand last scored
 * (rsc_cache_score / refresh; RSC_ERR_INVALID_ARGUMENT before any score).
 * Both are fp64 sums computed on the device in one fixed order (blocks of
 * 8,192 consecutive terms, each thread summing 32 terms 256 apart in turn,
 * then fixed binary trees over the threads and over the blocks), so they are
 * bitwise reproducible; for these non-negative terms they lie within
 * (n - 1) units of roundoff of the sequential sum. [sync]: waits for
 * `stream`, on which the scores were enqueued. Either pointer may be NULL. */
rsc_status_t rsc_cache_norms(rsc_cache_t *cache, double *fro_x2_host, double *fro_b2_host,
                             hipStream_t stream);
/* Staleness of a cached selection (section 3.3.1 and Fig. 4: how well the
 * columns chosen at one refresh still match the top pairs of a later
 * gradient). The cache keeps the selection that its latest select, refresh
 * or randomized refresh replaced ("previous", S_prev; its k_prev pairs) and
 * the current one (S_new). `order` (device, int32[n], n = columns of X)
 * ranks the n pairs best first, e.g. the ranking rsc_greedy_profile writes
 * for the newly scored keys. Writes, each pointer nullable:
 *   *auc_host     = the share of (selected, unselected) pairs of S_prev that
 *                   `order` ranks selected-first: the count of such ordered
 *                   pairs over k_prev (n - k_prev), in fp64; NaN when S_prev
 *                   is empty or holds all n pairs (an exact integer count
 *                   and one division, so equal bit for bit to any exact
 *                   evaluation of that definition);
 *   *overlap_host = |S_prev & S_new|;  *prev_k_host = k_prev.
 * RSC_ERR_INVALID_ARGUMENT before the second selection or when `order` is
 * not a ranking of 0..n-1 (an entry outside [0, n), or a selected pair
 * ranked other than once). [sync]: waits for `stream`, on which the
 * selections and the ranking were enqueued. */
rsc_status_t rsc_cache_staleness(rsc_cache_t *cache, const int32_t *order, double *auc_host,
                                 int64_t *overlap_host, int64_t *prev_k_host, hipStream_t stream);
/* Waits (on the host) for the work this cache's own calls enqueued, on
 * every stream they used, then frees its buffers (stream-ordered, on a
 * library-owned stream of the cache's device; through the allocator for a
 * cache made by rsc_cache_create_ex). Work on other streams is not waited
 * for. Calls captured into a HIP graph are not tracked: synchronise the
 * graph's launches before destroying the cache. NULL is a no-op. */
rsc_status_t rsc_cache_destroy(rsc_cache_t *cache);

/* ---------------------------------------------------------------- A8 --- */
/* Column budget (uniform allocation of section 5.2.2, k = C |V|) with C as
 * the rational num/den: floor(n * num / den). Returns -1 if n < 0, num < 0,
 * den <= 0 or num > den. Host only. */
int32_t rsc_k_from_fraction(int32_t n, int32_t num, int32_t den);

/* Layer-wise allocation of k_l under a FLOPs budget (Eq. 4a/4b, solved by
 * the greedy of section 3.2.1 / Algorithm 1). Host compute.
 *   key_host[l]: the n pair keys of layer l (rsc_pair_scores encoding).
 *   colnnz_host: the n column entry counts of the operand; nnz = |E|.
 *   d_host[l]: width of layer l's dense operand; fro_a2 = ||A||_F^2;
 *   fro_b2_host[l] = ||grad H^(l+1)||_F^2.
 *   Budget C = C_num / C_den; step = max(1, floor(n * alpha_num / alpha_den)).
 *   RSC_ERR_INVALID_ARGUMENT unless C >= 0, 0 <= alpha <= 1 (alpha is a
 *   fraction of the n columns) and sum_l nnz d_l fits int64.
 * Pairs rank by (key desc, index asc). Starting from k_l = n, while
 * Bud * C_den > C_num * sum_l nnz d_l, the eligible layer (k_l > 0) whose
 * shrink to max(0, k_l - step) loses the least normalised score mass
 * (sum of sqrt(q) over the dropped ranks in rank order, fp64, divided by
 * sqrt(fro_a2) * sqrt(fro_b2[l]); NaN keys count 0; lowest layer on ties)
 * is shrunk, and Bud drops by d_l times the dropped columns' entry counts.
 * Writes k_out_host[0..L) and, if budget_out_host is not NULL, the final
 * Bud. */
rsc_status_t rsc_greedy_allocate(int32_t L, int32_t n, int64_t nnz,
                                 const uint64_t *const *key_host, const int32_t *colnnz_host,
                                 const int32_t *d_host, double fro_a2, const double *fro_b2_host,
                                 int32_t C_num, int32_t C_den, int32_t alpha_num,
                                 int32_t alpha_den, int32_t *k_out_host,
                                 int64_t *budget_out_host);

/* Device-assisted form of the same allocation, for large n. The greedy
 * shrinks a layer by step = max(1, floor(n * alpha_num / alpha_den)) ranks
 * at a time from the bottom of its ranking, so per layer it only needs the
 * profile over blocks of `step` ranks counted from the lowest rank: block j
 * covers ranks [max(0, n - (j+1) step), n - j step) of the ranking
 * (key desc, index asc), and
 *   mass[j]  = sum of sqrt(q) over the block in ascending rank order (fp64;
 *              NaN keys count 0), q decoded from the key;
 *   count[j] = sum of colnnz over the block.
 * rsc_greedy_profile computes it on the device (stable radix sort of the
 * keys); order (nullable, int32[n]) receives the ranking itself. mass and
 * count hold rsc_greedy_blocks(n, alpha_num, alpha_den) entries (-1 for
 * n < 0 or alpha outside [0, 1], where both calls fail). ws: at
 * least rsc_greedy_profile_workspace_bytes(n) bytes, 256-byte aligned.
 * rsc_greedy_allocate_profiles runs the greedy loop on the host from the
 * layers' profiles (copied to the host); given the same keys it returns the
 * same k_l and budget as rsc_greedy_allocate. */
size_t rsc_greedy_profile_workspace_bytes(int32_t n);
int32_t rsc_greedy_blocks(int32_t n, int32_t alpha_num, int32_t alpha_den);
rsc_status_t rsc_greedy_profile(const uint64_t *key, const int32_t *colnnz, int32_t n,
                                int32_t alpha_num, int32_t alpha_den, double *mass,
                                int64_t *count, int32_t *order, void *ws, size_t ws_bytes,
                                hipStream_t stream);
rsc_status_t rsc_greedy_allocate_profiles(int32_t L, int32_t n, int64_t nnz, int32_t alpha_num,
                                          int32_t alpha_den, const double *const *mass_host,
                                          const int64_t *const *count_host, const int32_t *d_host,
                                          double fro_a2, const double *fro_b2_host, int32_t C_num,
                                          int32_t C_den, int32_t *k_out_host,
                                          int64_t *budget_out_host);

#ifdef __cplusplus
}
#endif

#endif /* RSC_H */
