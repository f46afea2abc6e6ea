// CSR well-formedness on the device: rowptr[0] = 0, rowptr[n_rows] = nnz,
// rowptr non-decreasing, 0 <= col < n_cols, and columns strictly increasing
// within each row (the form every step assumes; a duplicate entry would
// change a column norm). A row's entries are read only after its bounds are
// known to lie in [0, nnz], so a malformed rowptr cannot send the check out
// of bounds. The first offending row is kept with an integer atomic min.
#include "rsc_internal.h"

namespace rsc {
namespace {

__global__ void validate_init_kernel(unsigned long long *first_bad) { *first_bad = ~0ull; }

__global__ __launch_bounds__(256) void csr_validate_kernel(const int32_t *__restrict__ rowptr,
                                                           const int32_t *__restrict__ col, int32_t n_rows,
                                                           int32_t n_cols, int64_t nnz,
                                                           unsigned long long *first_bad) {
    const int lane = threadIdx.x & 63;
    const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (r >= n_rows) return;
    const int64_t s = rowptr[r], e = rowptr[r + 1];
    bool bad = s < 0 || e > nnz || s > e || (r == 0 && s != 0) || (r == n_rows - 1 && e != nnz);
    if (!bad) {
        for (int64_t t = s + lane; t < e; t += 64) {
            const int32_t c = col[t];
            if (c < 0 || c >= n_cols) bad = true;
            if (t + 1 < e && col[t + 1] <= c) bad = true;
        }
    }
    if (__ballot(bad) != 0 && lane == 0) atomicMin(first_bad, (unsigned long long)r);
}

}  // namespace

hipError_t csr_validate_launch(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr,
                               const int32_t *col, unsigned long long *first_bad, hipStream_t stream) {
    validate_init_kernel<<<1, 1, 0, stream>>>(first_bad);
    if (n_rows > 0)
        csr_validate_kernel<<<(unsigned)ceil_div((int64_t)n_rows, 4), 256, 0, stream>>>(rowptr, col, n_rows, n_cols,
                                                                                     nnz, first_bad);
    return hipGetLastError();
}

}  // namespace rsc
