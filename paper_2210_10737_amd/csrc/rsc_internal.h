// Internal declarations shared by the library's HIP translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <algorithm>

namespace rsc {

constexpr int kWave = 64;

// ---- SpMM --------------------------------------------------------------
size_t spmm_ws_bytes(int32_t n_rows, int64_t nnz, int32_t n_cols);
// nnz_bound sizes the long-row list; nnz_hint (expected entries) and
// n_src_hint (distinct B rows the entries reference) choose the feature slice
// and the column-blocked mode, which runs only if ws_bytes holds its buffers.
// hint_cols: col carries the hub hint in bit 31 (a plan's own copy only);
// kernels always mask that bit off.
int32_t spmm_slice_width(int32_t n_rows, int64_t nnz, int64_t n_src, int32_t d);
// What an SpMM plan prepared once for its operand: the column-blocked split
// bounds (split, P; P = 1 for an unblocked product) and, in the plan's own
// workspace, the long-row (or long-piece) list or the length-class order,
// with long_rows their count (-1: not known on the host, the launch uses the
// bound) and ordered the row-order decision taken.
// A launch uses them only while its own decisions match (ready); one that
// did not (*used_prep false) rebuilt the list in that workspace.
struct SpmmPrepared {
    const int32_t *split = nullptr;
    int32_t P = 1;
    bool ordered = false;
    bool ready = false;
    int32_t long_rows = 0;
};
hipError_t spmm_launch(int32_t n_rows, int32_t n_cols, int64_t nnz_bound, const int32_t *rowptr,
                       const int32_t *col, const float *val, const float *B, int32_t d, int64_t ldb, float *Y,
                       int64_t ldy, void *ws, size_t ws_bytes, hipStream_t stream, int64_t nnz_hint,
                       int64_t n_src_hint, bool hint_cols = false, const SpmmPrepared *prep = nullptr,
                       bool *used_prep = nullptr);
// The column-blocked mode's range count for a product (1 = not blocked) and
// its split bounds S[(P + 1) * n_rows]; the row-order decision; and the
// preparation a launch would do, run once into a plan's workspace (then
// *spmm_long_count_of(ws) holds the list's length on the device).
int32_t spmm_column_blocks(int32_t n_rows, int64_t nnz, int64_t n_src, int32_t d);
hipError_t spmm_split_launch(int32_t n_rows, int32_t n_cols, const int32_t *rowptr, const int32_t *col, int32_t P,
                             int32_t *S, hipStream_t stream);
bool spmm_use_order(int32_t n_rows, int64_t nnz);
// whether a pass `slice` floats wide over n_src B rows takes the hub hint
// (on a column copy that carries it)
bool spmm_hint_taken(int64_t n_src, int32_t d, int32_t slice);
hipError_t spmm_rows_prepare(int32_t n_rows, int64_t nnz_bound, const int32_t *rowptr, void *ws,
                             hipStream_t stream);
hipError_t spmm_blocked_prepare(int32_t n_rows, int64_t nnz_bound, const int32_t *S, int32_t P, void *ws,
                                hipStream_t stream);
size_t spmm_blocked_fits(int32_t n_rows, int64_t nnz_bound, int32_t P);  // workspace bytes the blocked mode needs
// workspace bytes an unblocked product needs (header and row list); with at
// least this much a launch runs, blocked only if the blocked buffers also fit
size_t spmm_core_ws_bytes(int32_t n_rows, int64_t nnz_bound);
const int32_t *spmm_long_count_of(const void *ws);

// ---- gather-ceiling probe (measurement helper) ---------------------------
int64_t gather_probe_sink_count(int64_t nnz);
// Y (nullable, n_rows x d, ldy): also write an output of the product's size
hipError_t gather_probe_launch(const int32_t *col, int64_t nnz, const float *B, int64_t ldb, int32_t d, int32_t slice,
                               bool hint, int32_t inflight, float *sink, float *Y, int64_t ldy, int32_t n_rows,
                               hipStream_t stream);

// ---- scores ------------------------------------------------------------
hipError_t col_sqnorms_launch(int32_t n, const int32_t *rowptr_t, const float *val_t, double *cn2,
                              int32_t *colnnz, hipStream_t stream);
// out = sum of x[0..n) in one fixed order (fp64; 0 for n = 0); ws holds
// sum_ws_bytes(n) bytes of block sums
size_t sum_ws_bytes(int64_t n);
hipError_t sum_fixed_order_launch(const double *x, int64_t n, double *ws, double *out, hipStream_t stream);
hipError_t pair_scores_launch(const double *cn2, const float *B, int32_t n, int32_t d, int64_t ldb,
                              uint64_t *key, float *score, double *rn2, hipStream_t stream);

// ---- top-k -------------------------------------------------------------
size_t topk_ws_bytes(int32_t n);
hipError_t topk_launch(const uint64_t *key, int32_t n, int32_t k, int32_t *idx, uint32_t *mask,
                       void *ws, hipStream_t stream);

// ---- slice -------------------------------------------------------------
size_t slice_ws_bytes(int64_t nnz);
hipError_t slice_launch(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr, const int32_t *col,
                        const float *val, const uint32_t *mask, int32_t *rowptr_out,
                        int32_t *col_out, float *val_out, int64_t capacity, int64_t *nnz_out,
                        void *ws, hipStream_t stream, const double *colw = nullptr);

// ---- column hub hint for the SpMM gathers --------------------------------
// hub_bits_launch: from per-column degrees (optionally only the columns kept
// by mask), the entry-weighted median split; writes the n-bit hub set into
// the workspace (hub_bits_of). flag_cols_launch: col with bit 31 = hub bit.
// Used by SpMM plans; the sampled products do not take the hint (measured
// slower on the cached slices).
size_t hub_ws_bytes(int32_t n);
uint32_t *hub_bits_of(void *ws);
hipError_t hub_bits_launch(const int32_t *deg, const uint32_t *mask, int32_t n, void *ws, hipStream_t stream);
hipError_t degree_count_launch(const int32_t *col, int64_t nnz, int32_t n_cols, int32_t *deg, hipStream_t stream);
hipError_t flag_cols_launch(const int32_t *col, int64_t nnz, const uint32_t *bits, int32_t *colf,
                            hipStream_t stream);

// ---- randomized column-row sampling ------------------------------------
size_t sample_ws_bytes(int32_t n);
hipError_t sample_launch(const uint64_t *key, int32_t n, int32_t k, uint64_t seed, int32_t *count,
                         double *colw, uint32_t *mask, void *ws, hipStream_t stream);

// ---- CSR validation ----------------------------------------------------
hipError_t csr_validate_launch(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr,
                               const int32_t *col, unsigned long long *first_bad, hipStream_t stream);

// ---- MEAN aggregator operand -------------------------------------------
hipError_t degree_scale_launch(int32_t n_rows, const int32_t *rowptr, const int32_t *col, const float *val,
                               const int32_t *deg_rowptr, int32_t by_column, float *out, hipStream_t stream);

// ---- layer-wise allocation ---------------------------------------------
int32_t greedy_step(int32_t n, int32_t alpha_num, int32_t alpha_den);
int32_t greedy_blocks(int32_t n, int32_t step);
size_t greedy_profile_ws_bytes(int32_t n);
// staleness counts of a previous selection under a ranking (acc: device,
// staleness_acc_count() entries, cleared by the launch)
int32_t staleness_acc_count();
hipError_t staleness_launch(const int32_t *order, int32_t n, const uint32_t *prev, const uint32_t *cur,
                            unsigned long long *acc, hipStream_t stream);
hipError_t greedy_profile_launch(const uint64_t *key, const int32_t *colnnz, int32_t n, int32_t step,
                                 double *mass, int64_t *count, int32_t *order_out, void *ws,
                                 hipStream_t stream);

// ---- helpers -----------------------------------------------------------
inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace rsc
