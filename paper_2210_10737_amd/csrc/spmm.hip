// Sparse-dense product Y = A * B for CSR A (the aggregation SpMM of the
// GCN layer, section 2.1; the same kernel runs on the column slice for the
// top-k approximation of section 2.2.1).
//
// Work mapping (gfx950, wave64):
//   * one wave per row; the feature dimension is spread over the lanes,
//     4 consecutive fp32 features per lane (one 128-bit load), 256 features
//     per wave, two such vectors per lane for widths up to 512;
//   * the row's (col, val) pairs are fetched 64 at a time with one
//     coalesced, non-temporal load and broadcast from the owning lane with
//     v_readlane into scalar registers, so each gathered B row is addressed
//     by a scalar base plus the lane offset;
//   * 8 gathers are issued before their FMAs for memory-level parallelism;
//   * products are accumulated in fp32 over each run of <= 64 entries and the
//     run sum is folded into an fp64 accumulator; one fp32 rounding per output;
//   * rows with more than kLongRow entries are taken by persistent 4-wave
//     blocks: the waves take interleaved runs of 64 entries and their fp64
//     sums are combined in LDS in fixed wave order. No float atomics, so the
//     result is bitwise reproducible.
#include "rsc_internal.h"

namespace rsc {
namespace {

constexpr int kUnroll = 8;
typedef float vf4 __attribute__((ext_vector_type(4)));

__global__ void fill_i32_kernel(int32_t *p, int32_t v) { *p = v; }

__global__ __launch_bounds__(256) void collect_long_rows_kernel(const int32_t *__restrict__ rowptr,
                                                                int32_t n_rows, int32_t *count,
                                                                int32_t *list) {
    const int32_t r = blockIdx.x * blockDim.x + threadIdx.x;
    if (r < n_rows && rowptr[r + 1] - rowptr[r] > kLongRow) list[atomicAdd(count, 1)] = r;
}

// Accumulates runs of 64 entries starting at beg, beg + stride, ... (< end)
// into acc. `act[q]` says whether this lane's q-th float4 lies inside d.
template <int NV>
__device__ __forceinline__ void accumulate_runs(const int32_t *__restrict__ col,
                                                const float *__restrict__ val,
                                                const float *__restrict__ B, int64_t ldb,
                                                int32_t beg, int32_t end, int32_t stride,
                                                const bool (&act)[NV], int lane,
                                                double (&acc)[NV][4]) {
    for (int32_t base = beg; base < end; base += stride) {
        const int32_t cnt = __builtin_amdgcn_readfirstlane(min(kWave, end - base));
        int32_t my_c = 0;
        float my_v = 0.f;
        if (lane < cnt) {
            my_c = __builtin_nontemporal_load(col + base + lane);
            my_v = __builtin_nontemporal_load(val + base + lane);
        }
        float a[NV][4];
#pragma unroll
        for (int q = 0; q < NV; ++q) a[q][0] = a[q][1] = a[q][2] = a[q][3] = 0.f;

        for (int32_t t = 0; t < cnt; t += kUnroll) {
            float4 b[kUnroll][NV];
            float v[kUnroll];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
#pragma unroll
                for (int q = 0; q < NV; ++q) b[u][q] = make_float4(0.f, 0.f, 0.f, 0.f);
                v[u] = 0.f;
                if (t + u < cnt) {  // wave-uniform
                    const int32_t c = __builtin_amdgcn_readlane(my_c, t + u);
                    v[u] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(my_v), t + u));
                    const float4 *brow = reinterpret_cast<const float4 *>(B + (int64_t)c * ldb) + lane;
#pragma unroll
                    for (int q = 0; q < NV; ++q)
                        if (act[q]) b[u][q] = brow[q * kWave];
                }
            }
#pragma unroll
            for (int u = 0; u < kUnroll; ++u)
#pragma unroll
                for (int q = 0; q < NV; ++q) {
                    a[q][0] = fmaf(v[u], b[u][q].x, a[q][0]);
                    a[q][1] = fmaf(v[u], b[u][q].y, a[q][1]);
                    a[q][2] = fmaf(v[u], b[u][q].z, a[q][2]);
                    a[q][3] = fmaf(v[u], b[u][q].w, a[q][3]);
                }
        }
#pragma unroll
        for (int q = 0; q < NV; ++q)
#pragma unroll
            for (int x = 0; x < 4; ++x) acc[q][x] += (double)a[q][x];
    }
}

template <int NV>
__device__ __forceinline__ void store_row(float *__restrict__ yrow, int32_t d, int lane,
                                          const double (&acc)[NV][4]) {
#pragma unroll
    for (int q = 0; q < NV; ++q) {
        const int32_t f = 4 * lane + 4 * kWave * q;
        if (f + 4 <= d) {
            vf4 o = {(float)acc[q][0], (float)acc[q][1], (float)acc[q][2], (float)acc[q][3]};
            __builtin_nontemporal_store(o, reinterpret_cast<vf4 *>(yrow + f));
        } else if (f < d) {
            for (int x = 0; x < d - f; ++x) yrow[f + x] = (float)acc[q][x];
        }
    }
}

// Blocks [0, n_long_blocks) walk the long-row list; the remaining blocks take
// 4 consecutive rows each (one per wave) and skip long rows.
template <int NV>
__global__ __launch_bounds__(256) void spmm_kernel(const int32_t *__restrict__ rowptr,
                                                   const int32_t *__restrict__ col,
                                                   const float *__restrict__ val,
                                                   const float *__restrict__ B, int64_t ldb,
                                                   float *__restrict__ Y, int64_t ldy, int32_t n_rows,
                                                   int32_t d, const int32_t *__restrict__ long_count,
                                                   const int32_t *__restrict__ long_rows,
                                                   int32_t n_long_blocks) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    bool act[NV];
#pragma unroll
    for (int q = 0; q < NV; ++q) act[q] = 4 * lane + 4 * kWave * q < d;

    if ((int32_t)blockIdx.x < n_long_blocks) {
        __shared__ double red[kSpmmBlockWaves][NV * 4][kWave];
        const int32_t nl = __builtin_amdgcn_readfirstlane(*long_count);
        for (int32_t j = blockIdx.x; j < nl; j += n_long_blocks) {
            const int32_t r = __builtin_amdgcn_readfirstlane(long_rows[j]);
            const int32_t s = __builtin_amdgcn_readfirstlane(rowptr[r]);
            const int32_t e = __builtin_amdgcn_readfirstlane(rowptr[r + 1]);
            double acc[NV][4];
#pragma unroll
            for (int q = 0; q < NV; ++q) acc[q][0] = acc[q][1] = acc[q][2] = acc[q][3] = 0.0;
            accumulate_runs<NV>(col, val, B, ldb, s + kWave * wave, e, kWave * kSpmmBlockWaves, act,
                                lane, acc);
#pragma unroll
            for (int q = 0; q < NV; ++q)
#pragma unroll
                for (int x = 0; x < 4; ++x) red[wave][q * 4 + x][lane] = acc[q][x];
            __syncthreads();
            if (wave == 0) {
#pragma unroll
                for (int q = 0; q < NV; ++q)
#pragma unroll
                    for (int x = 0; x < 4; ++x) {
                        double t = red[0][q * 4 + x][lane];
#pragma unroll
                        for (int w = 1; w < kSpmmBlockWaves; ++w) t += red[w][q * 4 + x][lane];
                        acc[q][x] = t;
                    }
                store_row<NV>(Y + (int64_t)r * ldy, d, lane, acc);
            }
            __syncthreads();
        }
        return;
    }

    const int32_t r = (blockIdx.x - n_long_blocks) * kSpmmBlockWaves + wave;
    if (r >= n_rows) return;
    const int32_t s = __builtin_amdgcn_readfirstlane(rowptr[r]);
    const int32_t e = __builtin_amdgcn_readfirstlane(rowptr[r + 1]);
    if (n_long_blocks > 0 && e - s > kLongRow) return;
    double acc[NV][4];
#pragma unroll
    for (int q = 0; q < NV; ++q) acc[q][0] = acc[q][1] = acc[q][2] = acc[q][3] = 0.0;
    accumulate_runs<NV>(col, val, B, ldb, s, e, kWave, act, lane, acc);
    store_row<NV>(Y + (int64_t)r * ldy, d, lane, acc);
}

struct SpmmWs {
    int32_t long_count;
    int32_t pad[63];
};

inline int64_t long_rows_bound(int32_t n_rows, int64_t nnz) {
    return std::min<int64_t>(n_rows, nnz / (kLongRow + 1));
}

}  // namespace

size_t spmm_ws_bytes(int32_t n_rows, int64_t nnz) {
    return sizeof(SpmmWs) + align_up(sizeof(int32_t) * (size_t)std::max<int64_t>(1, long_rows_bound(n_rows, nnz)), 256);
}

hipError_t spmm_launch(int32_t n_rows, int64_t nnz_bound, const int32_t *rowptr, const int32_t *col,
                       const float *val, const float *B, int32_t d, int64_t ldb, float *Y,
                       int64_t ldy, void *ws, hipStream_t stream) {
    if (n_rows == 0) return hipSuccess;
    SpmmWs *h = static_cast<SpmmWs *>(ws);
    int32_t *list = reinterpret_cast<int32_t *>(h + 1);
    const int64_t lbound = long_rows_bound(n_rows, nnz_bound);
    const int32_t n_long_blocks = (int32_t)std::min<int64_t>(lbound, kSpmmLongBlocks);
    if (n_long_blocks > 0) {
        fill_i32_kernel<<<1, 1, 0, stream>>>(&h->long_count, 0);
        collect_long_rows_kernel<<<(unsigned)ceil_div(n_rows, 256), 256, 0, stream>>>(
            rowptr, n_rows, &h->long_count, list);
    }
    const unsigned grid = (unsigned)(n_long_blocks + ceil_div(n_rows, kSpmmBlockWaves));
    // features are processed 512 at a time (two float4 per lane)
    for (int32_t f0 = 0; f0 < d; f0 += 8 * kWave) {
        const int32_t dl = std::min<int32_t>(d - f0, 8 * kWave);
        if (dl <= 4 * kWave)
            spmm_kernel<1><<<grid, 256, 0, stream>>>(rowptr, col, val, B + f0, ldb, Y + f0, ldy, n_rows,
                                                     dl, &h->long_count, list, n_long_blocks);
        else
            spmm_kernel<2><<<grid, 256, 0, stream>>>(rowptr, col, val, B + f0, ldb, Y + f0, ldy, n_rows,
                                                     dl, &h->long_count, list, n_long_blocks);
    }
    return hipGetLastError();
}

}  // namespace rsc
