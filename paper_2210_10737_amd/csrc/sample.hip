// Randomized column-row sampling (section 2.2, Eq. 2 with the probabilities
// of Eq. 3): k i.i.d. draws i_t ~ p, p_i proportional to sqrt(q_i), each
// drawn pair scaled by 1/(k p_{i_t}).
//
// Every decision is integer, so the draws are reproducible bit for bit:
//   * p is held as integer weights w_i = floor(sqrt(q_i) * 2^S / m),
//     m = max_j sqrt(q_j) (a max over the keys, order-free), with S = 38 up
//     to 2^24 pairs and 62 - ceil(log2 n) above, so the total stays <= 2^62;
//   * the CDF W_i = w_0 + ... + w_i is an exact int64 inclusive scan;
//   * draw t takes the t-th output z_t of the SplitMix64 generator seeded
//     with `seed`, u_t = floor(z_t * total / 2^64), and i_t = the smallest i
//     with W_i > u_t (binary search); counts are integer atomics;
//   * if some score is +Inf, the infinite ones share the mass uniformly;
//   * a column drawn c_i times enters once with scale
//     colw_i = c_i * total / (k * w_i) (fp64), i.e. c_i / (k p_i).
#include "rsc_internal.h"

namespace rsc {
namespace {

constexpr int kScanTile = 4096;  // 256 threads x 16

__device__ __forceinline__ double key_sqrt(uint64_t u) {
    return u == 0 ? 0.0 : sqrt(__longlong_as_double((long long)(u - 1)));
}

__device__ __forceinline__ uint64_t splitmix64(uint64_t seed, uint64_t t) {
    uint64_t z = seed + (t + 1) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

struct SampleWs {
    unsigned long long max_key;
    int64_t pad[31];
};

__global__ void sample_init_kernel(SampleWs *h) { h->max_key = 0ull; }

// max over the keys: a block-wide max, then one atomic per block (the grid
// is kept small: every atomic hits the same address)
__global__ __launch_bounds__(256) void max_key_kernel(const uint64_t *__restrict__ key, int32_t n, SampleWs *h) {
    __shared__ unsigned long long s[4];
    unsigned long long m = 0ull;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        m = max(m, (unsigned long long)key[i]);
    for (int off = 32; off > 0; off >>= 1) m = max(m, (unsigned long long)__shfl_down(m, off));
    if ((threadIdx.x & 63) == 0) s[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        m = max(max(s[0], s[1]), max(s[2], s[3]));
        if (m) atomicMax(&h->max_key, m);
    }
}

// w_i and the per-tile sums of w
__global__ __launch_bounds__(256) void weights_kernel(const uint64_t *__restrict__ key, int32_t n, int bits,
                                                      const SampleWs *__restrict__ h, int64_t *__restrict__ w,
                                                      int64_t *__restrict__ tile_sum) {
    __shared__ int64_t s[4];
    const double m = key_sqrt(h->max_key);
    const double scale = m > 0.0 ? ldexp(1.0, bits) / m : 0.0;  // 2^S / m
    const int64_t ts = (int64_t)blockIdx.x * kScanTile;
    int64_t acc = 0;
    for (int j = 0; j < kScanTile / 256; ++j) {
        const int64_t i = ts + threadIdx.x + 256 * j;
        if (i < n) {
            const double r = key_sqrt(key[i]);
            // infinite scores share the mass uniformly
            const int64_t wi = isinf(m) ? (isinf(r) ? ((int64_t)1 << bits) : 0) : (int64_t)(r * scale);
            w[i] = wi;
            acc += wi;
        }
    }
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_down(acc, off);
    if ((threadIdx.x & 63) == 0) s[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) tile_sum[blockIdx.x] = s[0] + s[1] + s[2] + s[3];
}

// exclusive scan of the tile sums, in place (one block of 1024 threads)
__global__ __launch_bounds__(1024) void tile_scan_kernel(int64_t *__restrict__ tile_sum, int32_t nt) {
    __shared__ int64_t sh[1024];
    const int t = threadIdx.x;
    const int32_t per = (nt + 1023) / 1024;
    const int32_t lo = min(nt, t * per), hi = min(nt, lo + per);
    int64_t s = 0;
    for (int32_t i = lo; i < hi; ++i) s += tile_sum[i];
    sh[t] = s;
    __syncthreads();
    for (int off = 1; off < 1024; off <<= 1) {
        const int64_t x = t >= off ? sh[t - off] : 0;
        __syncthreads();
        sh[t] += x;
        __syncthreads();
    }
    int64_t run = sh[t] - s;
    for (int32_t i = lo; i < hi; ++i) {
        const int64_t c = tile_sum[i];
        tile_sum[i] = run;
        run += c;
    }
}

// inclusive prefix W within each tile: each thread scans 16 consecutive
// entries, then a block scan over the threads' sums
__global__ __launch_bounds__(256) void prefix_kernel(const int64_t *__restrict__ w, int32_t n,
                                                     const int64_t *__restrict__ tile_off,
                                                     int64_t *__restrict__ W) {
    __shared__ int64_t sh[256];
    constexpr int kPer = kScanTile / 256;
    const int t = threadIdx.x;
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)t * kPer;
    int64_t v[kPer];
    int64_t s = 0;
    for (int j = 0; j < kPer; ++j) {
        v[j] = base + j < n ? w[base + j] : 0;
        s += v[j];
    }
    sh[t] = s;
    __syncthreads();
    for (int off = 1; off < 256; off <<= 1) {
        const int64_t x = t >= off ? sh[t - off] : 0;
        __syncthreads();
        sh[t] += x;
        __syncthreads();
    }
    int64_t run = tile_off[blockIdx.x] + sh[t] - s;
    for (int j = 0; j < kPer; ++j) {
        run += v[j];
        if (base + j < n) W[base + j] = run;
    }
}

__global__ __launch_bounds__(256) void draw_kernel(const int64_t *__restrict__ W, int32_t n, int32_t k,
                                                   uint64_t seed, int32_t *__restrict__ count) {
    const int32_t t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= k) return;
    const uint64_t total = (uint64_t)W[n - 1];
    if (total == 0) return;
    const uint64_t u = __umul64hi(splitmix64(seed, (uint64_t)t), total);
    int32_t lo = 0, hi = n - 1;  // smallest i with W[i] > u
    while (lo < hi) {
        const int32_t mid = lo + (hi - lo) / 2;
        if ((uint64_t)W[mid] > u) hi = mid; else lo = mid + 1;
    }
    atomicAdd(&count[lo], 1);
}

__global__ __launch_bounds__(256) void colw_kernel(const int32_t *__restrict__ count, const int64_t *__restrict__ w,
                                                   const int64_t *__restrict__ W, int32_t n, int32_t k,
                                                   double *__restrict__ colw, uint32_t *__restrict__ mask) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int lane = threadIdx.x & 63;
    const bool in = i < n;
    const int32_t c = in ? count[i] : 0;
    if (in) {
        const double total = (double)W[n - 1];
        colw[i] = c ? (double)c * total / ((double)k * (double)w[i]) : 0.0;
    }
    const uint64_t bal = __ballot(c > 0);
    const int64_t word = (i - lane) / 32;
    const int64_t nwords = ((int64_t)n + 31) / 32;
    if (lane == 0 && word < nwords) mask[word] = (uint32_t)bal;
    if (lane == 32 && word + 1 < nwords) mask[word + 1] = (uint32_t)(bal >> 32);
}

__global__ __launch_bounds__(256) void zero_i32_kernel(int32_t *p, int64_t count) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = 0;
}

}  // namespace

size_t sample_ws_bytes(int32_t n) {
    const size_t nn = (size_t)std::max<int32_t>(n, 1);
    const size_t nt = (size_t)ceil_div((int64_t)nn, kScanTile);
    return align_up(sizeof(SampleWs), 256) + 2 * align_up(nn * 8, 256) + align_up(nt * 8, 256);
}

hipError_t sample_launch(const uint64_t *key, int32_t n, int32_t k, uint64_t seed, int32_t *count,
                         double *colw, uint32_t *mask, void *ws, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    const size_t nn = (size_t)n;
    const int32_t nt = (int32_t)ceil_div(n, kScanTile);
    char *p = static_cast<char *>(ws);
    SampleWs *h = reinterpret_cast<SampleWs *>(p);
    p += align_up(sizeof(SampleWs), 256);
    int64_t *w = reinterpret_cast<int64_t *>(p);
    p += align_up(nn * 8, 256);
    int64_t *W = reinterpret_cast<int64_t *>(p);
    p += align_up(nn * 8, 256);
    int64_t *tile = reinterpret_cast<int64_t *>(p);
    const unsigned g = (unsigned)std::min<int64_t>(ceil_div(n, 256), 4096);
    sample_init_kernel<<<1, 1, 0, stream>>>(h);
    zero_i32_kernel<<<g, 256, 0, stream>>>(count, n);
    max_key_kernel<<<std::min<unsigned>(g, 256), 256, 0, stream>>>(key, n, h);
    int bits = 38;  // weight resolution S
    if (n > (1 << 24)) {
        int lg = 0;
        while ((int64_t{1} << lg) < (int64_t)n) ++lg;
        bits = 62 - lg;
    }
    weights_kernel<<<nt, 256, 0, stream>>>(key, n, bits, h, w, tile);
    tile_scan_kernel<<<1, 1024, 0, stream>>>(tile, nt);
    prefix_kernel<<<nt, 256, 0, stream>>>(w, n, tile, W);
    if (k > 0) draw_kernel<<<(unsigned)ceil_div(k, 256), 256, 0, stream>>>(W, n, k, seed, count);
    colw_kernel<<<(unsigned)ceil_div(n, 256), 256, 0, stream>>>(count, w, W, n, k, colw, mask);
    return hipGetLastError();
}

}  // namespace rsc
