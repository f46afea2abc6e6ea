// Column hub hint for the SpMM gathers (a cache policy; no effect on values).
//
// When the gathered B rows far outgrow the on-chip caches, a row fetched for
// a low-degree column is rarely reused before it is evicted, and it evicts
// rows of high-degree columns that would have been. So the columns are split
// at the entry-weighted median of their degree: the columns above it (which
// hold just under half of the entries) keep the default load policy, the
// rest are gathered non-temporally. The split is marked in bit 31 of the
// column index, in a copy of col that an SpMM plan owns.
//
// Degrees are bucketed on a log scale (8 buckets per octave); the weighted
// median is found on the device from a histogram of entries per bucket. (The
// cached slices of the sampled product do not use the hint: their kept
// columns are mostly of low degree, and it measured slower there.)
#include "rsc_internal.h"

namespace rsc {
namespace {

constexpr int kHubBuckets = 256;  // 8 per octave over 32 octaves

// Bucket of a degree >= 1: 8 * floor(log2 deg) + the next three bits.
__device__ __forceinline__ int hub_bucket(int32_t deg) {
    const int e = 31 - __clz(deg);
    const int sub = e >= 3 ? (deg >> (e - 3)) & 7 : (deg << (3 - e)) & 7;
    return 8 * e + sub;
}

__global__ __launch_bounds__(256) void fill_i32_kernel(int32_t *p, int64_t count) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = 0;
}

// deg[c] = entries in column c (integer atomics; order-independent).
__global__ __launch_bounds__(256) void degree_count_kernel(const int32_t *__restrict__ col, int64_t nnz,
                                                           int32_t *__restrict__ deg) {
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < nnz;
         t += (int64_t)gridDim.x * blockDim.x)
        atomicAdd(&deg[col[t]], 1);
}

// hist[b] += sum of deg over the columns (kept by mask, if given) in bucket
// b; hist starts cleared.
__global__ __launch_bounds__(256) void hub_hist_kernel(const int32_t *__restrict__ deg,
                                                       const uint32_t *__restrict__ mask, int32_t n,
                                                       unsigned long long *__restrict__ hist) {
    __shared__ unsigned long long lh[kHubBuckets];
    lh[threadIdx.x] = 0;
    __syncthreads();
    for (int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c < n;
         c += (int64_t)gridDim.x * blockDim.x) {
        const int32_t g = deg[c];
        const bool kept = !mask || ((mask[c >> 5] >> (c & 31)) & 1u);
        if (kept && g > 0) atomicAdd(&lh[hub_bucket(g)], (unsigned long long)g);
    }
    __syncthreads();
    if (lh[threadIdx.x]) atomicAdd(&hist[threadIdx.x], lh[threadIdx.x]);
}

// *bstar = the largest bucket b with (entries in buckets >= b) >= half of
// all entries; the hub columns are the buckets above it (255: none).
__global__ __launch_bounds__(64) void hub_pick_kernel(const unsigned long long *__restrict__ hist,
                                                      int32_t *__restrict__ bstar) {
    if (threadIdx.x != 0) return;
    unsigned long long total = 0;
    for (int b = 0; b < kHubBuckets; ++b) total += hist[b];
    int32_t pick = kHubBuckets - 1;
    unsigned long long cum = 0;
    for (int b = kHubBuckets - 1; b >= 0; --b) {
        cum += hist[b];
        if (total > 0 && 2 * cum >= total) {
            pick = b;
            break;
        }
    }
    *bstar = pick;
}

// bits: bit c set iff column c is a hub (one wave ballot per 64 columns).
__global__ __launch_bounds__(256) void hub_bits_kernel(const int32_t *__restrict__ deg, int32_t n,
                                                       const int32_t *__restrict__ bstar,
                                                       uint32_t *__restrict__ bits) {
    const int32_t b = *bstar;
    const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int32_t g = c < n ? deg[c] : 0;
    const uint64_t ball = __ballot(g > 0 && hub_bucket(g) > b);
    const int lane = threadIdx.x & 63;
    const int64_t w = (c - lane) / 32;  // first word of this wave's 64 columns
    const int64_t words = ((int64_t)n + 31) / 32;
    if (lane == 0 && w < words) bits[w] = (uint32_t)ball;
    if (lane == 32 && w + 1 < words) bits[w + 1] = (uint32_t)(ball >> 32);
}

// colf[t] = col[t] with bit 31 set iff col[t] is a hub column.
__global__ __launch_bounds__(256) void flag_cols_kernel(const int32_t *__restrict__ col, int64_t nnz,
                                                        const uint32_t *__restrict__ bits,
                                                        int32_t *__restrict__ colf) {
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < nnz;
         t += (int64_t)gridDim.x * blockDim.x) {
        const int32_t c = col[t];
        colf[t] = (int32_t)((uint32_t)c | (((bits[c >> 5] >> (c & 31)) & 1u) << 31));
    }
}

inline unsigned grid_for(int64_t items, int64_t per_block, int64_t cap) {
    return (unsigned)std::max<int64_t>(1, std::min<int64_t>(ceil_div(std::max<int64_t>(items, 1), per_block), cap));
}

}  // namespace

size_t hub_ws_bytes(int32_t n) {
    return align_up(sizeof(unsigned long long) * kHubBuckets, 256) + 256 +
           align_up(sizeof(uint32_t) * (size_t)ceil_div(std::max<int32_t>(n, 1), 32), 256);
}

uint32_t *hub_bits_of(void *ws) {
    return reinterpret_cast<uint32_t *>(static_cast<char *>(ws) +
                                        align_up(sizeof(unsigned long long) * kHubBuckets, 256) + 256);
}

hipError_t hub_bits_launch(const int32_t *deg, const uint32_t *mask, int32_t n, void *ws, hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    auto *hist = static_cast<unsigned long long *>(ws);
    auto *bstar = reinterpret_cast<int32_t *>(static_cast<char *>(ws) +
                                              align_up(sizeof(unsigned long long) * kHubBuckets, 256));
    fill_i32_kernel<<<1, 256, 0, stream>>>(reinterpret_cast<int32_t *>(hist), 2 * kHubBuckets);
    hub_hist_kernel<<<grid_for(n, 256, 1024), 256, 0, stream>>>(deg, mask, n, hist);
    hub_pick_kernel<<<1, 64, 0, stream>>>(hist, bstar);
    hub_bits_kernel<<<(unsigned)ceil_div(n, 256), 256, 0, stream>>>(deg, n, bstar, hub_bits_of(ws));
    return hipGetLastError();
}

hipError_t degree_count_launch(const int32_t *col, int64_t nnz, int32_t n_cols, int32_t *deg, hipStream_t stream) {
    fill_i32_kernel<<<grid_for(n_cols, 256, 1024), 256, 0, stream>>>(deg, n_cols);
    if (nnz > 0) degree_count_kernel<<<grid_for(nnz, 256, 8192), 256, 0, stream>>>(col, nnz, deg);
    return hipGetLastError();
}

hipError_t flag_cols_launch(const int32_t *col, int64_t nnz, const uint32_t *bits, int32_t *colf,
                            hipStream_t stream) {
    if (nnz > 0) flag_cols_kernel<<<grid_for(nnz, 256, 8192), 256, 0, stream>>>(col, nnz, bits, colf);
    return hipGetLastError();
}

}  // namespace rsc
