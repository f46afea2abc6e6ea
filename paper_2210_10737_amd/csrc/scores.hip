// Pair scores of the column-row pairs (Eq. 3; the top-k rule of section
// 2.2.1; the ||A^T[:, i]|| ||grad H[i, :]|| terms of Eq. 4a).
//
// Both reductions follow one canonical order so that the keys, and hence the
// selection, are bitwise reproducible: an fp64 sum of exact fp32 squares in
// plain index order.
#include "rsc_internal.h"

namespace rsc {
namespace {

// cn2[i] = sum of val^2 over row i of X^T, in stored order. One wave per
// row: the wave loads 64 values at a time (coalesced) and adds their squares
// one after another in stored order, each value broadcast with readlane, so
// the sum is the sequential one while the loads stay wide. Products of fp32
// values are exact in fp64, so fma(v, v, acc) equals acc + v * v.
__global__ __launch_bounds__(256) void col_sqnorms_kernel(int32_t n, const int32_t *__restrict__ rowptr,
                                                          const float *__restrict__ val,
                                                          double *__restrict__ cn2,
                                                          int32_t *__restrict__ colnnz) {
    const int lane = threadIdx.x & 63;
    const int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (i >= n) return;
    const int32_t s = __builtin_amdgcn_readfirstlane(rowptr[i]);
    const int32_t e = __builtin_amdgcn_readfirstlane(rowptr[i + 1]);
    double acc = 0.0;
    for (int64_t base = s; base < e; base += 64) {
        const int32_t cnt = (int32_t)min<int64_t>(64, e - base);
        const int vb = lane < cnt ? __float_as_int(__builtin_nontemporal_load(val + base + lane)) : 0;
        if (cnt == 64) {
#pragma unroll
            for (int t = 0; t < 64; ++t) {
                const double v = (double)__int_as_float(__builtin_amdgcn_readlane(vb, t));
                acc = fma(v, v, acc);
            }
        } else {
            for (int t = 0; t < cnt; ++t) {
                const double v = (double)__int_as_float(__builtin_amdgcn_readlane(vb, t));
                acc = fma(v, v, acc);
            }
        }
    }
    if (lane == 0) {
        cn2[i] = acc;
        if (colnnz) colnnz[i] = e - s;
    }
}

// 256 rows per block, one row per thread. B is streamed through LDS in tiles
// of 256 rows x 32 features (each row segment is one 128-byte line, read by
// 8 lanes with 128-bit loads); each thread then sums its own row of the tile
// in ascending feature order.
constexpr int kRows = 256;
constexpr int kTileF = 32;

__global__ __launch_bounds__(256) void pair_scores_kernel(const double *__restrict__ cn2,
                                                          const float *__restrict__ B, int32_t n,
                                                          int32_t d, int64_t ldb,
                                                          uint64_t *__restrict__ key,
                                                          float *__restrict__ score,
                                                          double *__restrict__ rn2) {
    constexpr int kLoads = kRows * kTileF / 4 / 256;  // float4 loads per thread per tile
    __shared__ float tile[kRows][kTileF + 1];
    const int t = threadIdx.x;
    const int64_t row0 = (int64_t)blockIdx.x * kRows;
    float4 v[kLoads];
    // the next tile's loads are issued before the current tile is summed
    auto load = [&](int32_t f0) {
#pragma unroll
        for (int it = 0; it < kLoads; ++it) {
            const int idx = t + 256 * it;
            const int rl = idx >> 3, fq = idx & 7;
            const int64_t row = row0 + rl;
            const int32_t f = f0 + 4 * fq;
            v[it] = make_float4(0.f, 0.f, 0.f, 0.f);
            // ld % 4 == 0 and ld >= d, so a float4 starting below d stays in the row
            if (row < n && f < d) v[it] = *reinterpret_cast<const float4 *>(B + row * ldb + f);
        }
    };
    double acc = 0.0;
    load(0);
    for (int32_t f0 = 0; f0 < d; f0 += kTileF) {
#pragma unroll
        for (int it = 0; it < kLoads; ++it) {
            const int idx = t + 256 * it;
            const int rl = idx >> 3, fq = idx & 7;
            tile[rl][4 * fq + 0] = v[it].x;
            tile[rl][4 * fq + 1] = v[it].y;
            tile[rl][4 * fq + 2] = v[it].z;
            tile[rl][4 * fq + 3] = v[it].w;
        }
        __syncthreads();
        if (f0 + kTileF < d) load(f0 + kTileF);
        const int lim = min(kTileF, d - f0);
        for (int j = 0; j < lim; ++j) {
            const double b = (double)tile[t][j];
            acc = fma(b, b, acc);
        }
        __syncthreads();
    }
    const int64_t row = row0 + t;
    if (row < n) {
        const double q = cn2[row] * acc;
        const uint64_t bits = (uint64_t)__double_as_longlong(q);
        key[row] = isnan(q) ? 0ull : bits + 1ull;
        if (score) score[row] = (float)sqrt(q);
        if (rn2) rn2[row] = acc;
    }
}

// Frobenius normalisers of Eq. 4a (||X||_F^2 = sum of cn2, ||B||_F^2 = sum
// of rn2) as fp64 sums in one fixed order, so the greedy's cross-layer
// comparison is bitwise reproducible: block b sums elements
// [b * kSumChunk, (b + 1) * kSumChunk), each thread its 32 elements t, t + 256,
// ... one after another, then the 256 thread sums in a fixed binary tree;
// one block adds the block sums the same way. Summing non-negative terms in
// any order stays within (n - 1) units of roundoff of the sequential sum.
constexpr int kSumThreads = 256;
constexpr int kSumPer = 32;
constexpr int kSumChunk = kSumThreads * kSumPer;

__device__ __forceinline__ double block_tree_sum(double v, double *lds) {
    const int t = threadIdx.x;
    lds[t] = v;
    __syncthreads();
    for (int h = kSumThreads / 2; h > 0; h >>= 1) {
        if (t < h) lds[t] = lds[t] + lds[t + h];
        __syncthreads();
    }
    return lds[0];
}

__global__ __launch_bounds__(kSumThreads) void sum_chunks_kernel(const double *__restrict__ x, int64_t n,
                                                                 double *__restrict__ part) {
    __shared__ double lds[kSumThreads];
    const int64_t base = (int64_t)blockIdx.x * kSumChunk + threadIdx.x;
    double acc = 0.0;
#pragma unroll
    for (int j = 0; j < kSumPer; ++j) {
        const int64_t i = base + (int64_t)kSumThreads * j;
        if (i < n) acc += x[i];
    }
    const double s = block_tree_sum(acc, lds);
    if (threadIdx.x == 0) part[blockIdx.x] = s;
}

__global__ __launch_bounds__(kSumThreads) void sum_parts_kernel(const double *__restrict__ part, int64_t np,
                                                                double *__restrict__ out) {
    __shared__ double lds[kSumThreads];
    double acc = 0.0;
    for (int64_t i = threadIdx.x; i < np; i += kSumThreads) acc += part[i];
    const double s = block_tree_sum(acc, lds);
    if (threadIdx.x == 0) *out = s;
}

}  // namespace

size_t sum_ws_bytes(int64_t n) { return sizeof(double) * (size_t)std::max<int64_t>(1, ceil_div(n, kSumChunk)); }

hipError_t sum_fixed_order_launch(const double *x, int64_t n, double *ws, double *out, hipStream_t stream) {
    const int64_t np = ceil_div(n, kSumChunk);
    if (np > 0) sum_chunks_kernel<<<(unsigned)np, kSumThreads, 0, stream>>>(x, n, ws);
    sum_parts_kernel<<<1, kSumThreads, 0, stream>>>(ws, np, out);
    return hipGetLastError();
}

hipError_t col_sqnorms_launch(int32_t n, const int32_t *rowptr_t, const float *val_t, double *cn2,
                              int32_t *colnnz, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    col_sqnorms_kernel<<<(unsigned)ceil_div(n, 4), 256, 0, stream>>>(n, rowptr_t, val_t, cn2, colnnz);
    return hipGetLastError();
}

hipError_t pair_scores_launch(const double *cn2, const float *B, int32_t n, int32_t d, int64_t ldb,
                              uint64_t *key, float *score, double *rn2, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    pair_scores_kernel<<<(unsigned)ceil_div(n, kRows), 256, 0, stream>>>(cn2, B, n, d, ldb, key, score, rn2);
    return hipGetLastError();
}

}  // namespace rsc
