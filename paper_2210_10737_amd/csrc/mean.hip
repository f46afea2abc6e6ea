// Operand of the MEAN aggregator (appendix A.3): SpMM_MEAN(A, H) = D^-1 A H,
// D the degree matrix of A (D_ii = stored entries of row i). The row-scaled
// values of D^-1 A feed the forward SpMM unchanged; its transpose A^T D^-1,
// the backward operand, scales each entry of A^T's CSR by the degree of its
// column. Both are one pass over the entries: one wave per row, each value
// divided in fp64 and rounded once to fp32.
#include "rsc_internal.h"

namespace rsc {
namespace {

__global__ __launch_bounds__(256) void degree_scale_kernel(int32_t n_rows, const int32_t *__restrict__ rowptr,
                                                           const int32_t *__restrict__ col,
                                                           const float *__restrict__ val,
                                                           const int32_t *__restrict__ deg_rowptr,
                                                           int32_t by_column, float *__restrict__ out) {
    const int lane = threadIdx.x & 63;
    const int32_t r = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (r >= n_rows) return;
    const int32_t s = rowptr[r], e = rowptr[r + 1];
    const int32_t row_len = e - s;
    for (int64_t t = (int64_t)s + lane; t < e; t += 64) {  // int64: t + 64 may pass 2^31 - 1
        int32_t deg = row_len;
        if (by_column) {
            const int32_t c = col[t];
            deg = deg_rowptr[c + 1] - deg_rowptr[c];
        }
        out[t] = deg > 0 ? (float)((double)val[t] / (double)deg) : 0.0f;
    }
}

}  // namespace

hipError_t degree_scale_launch(int32_t n_rows, const int32_t *rowptr, const int32_t *col, const float *val,
                               const int32_t *deg_rowptr, int32_t by_column, float *out, hipStream_t stream) {
    if (n_rows == 0) return hipSuccess;
    degree_scale_kernel<<<(unsigned)ceil_div(n_rows, 4), 256, 0, stream>>>(n_rows, rowptr, col, val, deg_rowptr,
                                                                           by_column, out);
    return hipGetLastError();
}

}  // namespace rsc
