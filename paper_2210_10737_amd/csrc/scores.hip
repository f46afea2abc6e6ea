// Pair scores of the column-row pairs (Eq. 3; the top-k rule of section
// 2.2.1; the ||A^T[:, i]|| ||grad H[i, :]|| terms of Eq. 4a).
//
// Both reductions follow one canonical order so that the keys, and hence the
// selection, are bitwise reproducible: an fp64 sum of exact fp32 squares in
// plain index order.
#include "rsc_internal.h"

namespace rsc {
namespace {

// cn2[i] = sum of val^2 over row i of X^T, in stored order: a sequential
// fp64 chain per row. Products of fp32 values are exact in fp64, so
// fma(v, v, acc) equals acc + v * v.
//
// One wave per 64 consecutive rows. Rows of at most kNormThreadMax entries
// are walked by their own lane, 16 values per step through four aligned
// float4 loads (the next step's loads in flight), so the chain costs no
// memory operation or broadcast per value and the 64 lanes' chains advance
// together. The wave then takes its longer rows one at a time: 64 values per
// coalesced load (four more loads in flight), squared by the lanes and read
// back by the chain from LDS. A wave-per-row form for every row kept 63 of 64 lanes
// idle in the chain and took 3-5x longer on graphs of short rows.
constexpr int32_t kNormThreadMax = 2048;

__device__ __forceinline__ double sq_chain_thread(const float *__restrict__ val, int64_t s, int64_t e) {
    double acc = 0.0;
    int64_t p = s;
    while (p < e && (reinterpret_cast<uintptr_t>(val + p) & 15)) {  // up to 3 values to a 16-byte boundary
        const double v = (double)val[p++];
        acc = fma(v, v, acc);
    }
    if (p + 16 <= e) {
        const float4 *q = reinterpret_cast<const float4 *>(val + p);
        float4 a = q[0], b = q[1], c = q[2], d = q[3];
        for (; p + 16 <= e; p += 16) {
            float4 na = a, nb = b, nc = c, nd = d;
            if (p + 32 <= e) {
                const float4 *qn = reinterpret_cast<const float4 *>(val + p + 16);
                na = qn[0];
                nb = qn[1];
                nc = qn[2];
                nd = qn[3];
            }
            const float w[16] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w, c.x, c.y, c.z, c.w, d.x, d.y, d.z, d.w};
#pragma unroll
            for (int t = 0; t < 16; ++t) {
                const double v = (double)w[t];
                acc = fma(v, v, acc);
            }
            a = na;
            b = nb;
            c = nc;
            d = nd;
        }
    }
    for (; p < e; ++p) {
        const double v = (double)val[p];
        acc = fma(v, v, acc);
    }
    return acc;
}

// Adds, in order, the squares of the first cnt values of a 64-value batch
// (lane t holds value t): each lane squares its value exactly in fp64 and
// stores it in LDS, and the chain reads the squares back at one address for
// all lanes (a broadcast read into a vector register), so nothing but the
// adds sits on the chain. buf alternates between two 64-entry halves so the
// next batch can be stored while this one is read.
__device__ __forceinline__ void chain64(float x, int32_t cnt, int lane, double *buf, double &acc) {
    buf[lane] = (double)x * (double)x;  // exact: fma(v, v, acc) == acc + v * v
    __syncthreads();                    // one-wave block
    if (cnt >= 64) {
#pragma unroll
        for (int t0 = 0; t0 < 64; t0 += 8) {
            double w[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) w[u] = buf[t0 + u];
#pragma unroll
            for (int u = 0; u < 8; ++u) acc += w[u];
        }
    } else {
        for (int t = 0; t < cnt; ++t) acc += buf[t];
    }
}

__device__ __forceinline__ double sq_chain_wave(const float *__restrict__ val, int64_t s, int64_t e, int lane,
                                                double (*buf)[64]) {
    double acc = 0.0;
    auto ld = [&](int64_t base) -> float {
        return base + lane < e ? __builtin_nontemporal_load(val + base + lane) : 0.f;
    };
    float c0 = ld(s), c1 = ld(s + 64), c2 = ld(s + 128), c3 = ld(s + 192);
    for (int64_t base = s; base < e; base += 256) {
        const float n0 = ld(base + 256), n1 = ld(base + 320), n2 = ld(base + 384), n3 = ld(base + 448);
        const int64_t left = e - base;
        chain64(c0, (int32_t)min<int64_t>(64, left), lane, buf[0], acc);
        if (left > 64) chain64(c1, (int32_t)min<int64_t>(64, left - 64), lane, buf[1], acc);
        if (left > 128) chain64(c2, (int32_t)min<int64_t>(64, left - 128), lane, buf[0], acc);
        if (left > 192) chain64(c3, (int32_t)min<int64_t>(64, left - 192), lane, buf[1], acc);
        c0 = n0;
        c1 = n1;
        c2 = n2;
        c3 = n3;
    }
    return acc;
}

__global__ __launch_bounds__(64) void col_sqnorms_kernel(int32_t n, const int32_t *__restrict__ rowptr,
                                                         const float *__restrict__ val, double *__restrict__ cn2,
                                                         int32_t *__restrict__ colnnz) {
    __shared__ double buf[2][64];
    const int lane = threadIdx.x;
    const int64_t r = (int64_t)blockIdx.x * kWave + lane;
    int32_t s = 0, e = 0;
    if (r < n) {
        s = rowptr[r];
        e = rowptr[r + 1];
        if (colnnz) colnnz[r] = e - s;
    }
    const bool is_long = r < n && e - s > kNormThreadMax;
    if (r < n && !is_long) cn2[r] = sq_chain_thread(val, s, e);
    uint64_t longs = __ballot(is_long);
    while (longs) {  // wave-uniform
        const int j = __builtin_ctzll(longs);
        longs &= longs - 1;
        const int32_t sj = __builtin_amdgcn_readlane(s, j), ej = __builtin_amdgcn_readlane(e, j);
        const double acc = sq_chain_wave(val, sj, ej, lane, buf);
        if (lane == 0) cn2[r - lane + j] = acc;  // row r0 + j
    }
}

// 256 rows per block, one row per thread. B is streamed through LDS in tiles
// of 256 rows x 32 features (each row segment is one 128-byte line, read by
// 8 lanes with 128-bit loads); each thread then sums its own row of the tile
// in ascending feature order.
constexpr int kRows = 256;
constexpr int kTileF = 32;
typedef float vf4 __attribute__((ext_vector_type(4)));

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
            // ld % 4 == 0 and ld >= d, so a float4 starting below d stays in the row;
            // B is read once, so its lines are streamed past the caches
            if (row < n && f < d) {
                const vf4 x = __builtin_nontemporal_load(reinterpret_cast<const vf4 *>(B + row * ldb + f));
                v[it] = make_float4(x.x, x.y, x.z, x.w);
            }
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
    col_sqnorms_kernel<<<(unsigned)ceil_div(n, kWave), kWave, 0, stream>>>(n, rowptr_t, val_t, cn2, colnnz);
    return hipGetLastError();
}

hipError_t pair_scores_launch(const double *cn2, const float *B, int32_t n, int32_t d, int64_t ldb,
                              uint64_t *key, float *score, double *rn2, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    pair_scores_kernel<<<(unsigned)ceil_div(n, kRows), 256, 0, stream>>>(cn2, B, n, d, ldb, key, score, rn2);
    return hipGetLastError();
}

}  // namespace rsc
