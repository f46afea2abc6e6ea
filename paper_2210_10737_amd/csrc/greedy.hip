// Device part of the layer-wise allocation (Eq. 4a/4b, the greedy of
// section 3.2.1 / Algorithm 1): the per-layer score-mass and entry-count
// profile over the pair ranking.
//
// The greedy shrinks a layer's k by `step` ranks at a time from the bottom of
// its ranking, so all it needs per layer are, for every block of `step`
// ranks counted from the lowest rank, the fp64 sum of sqrt(q) over the block
// (ascending rank order) and the sum of the blocks' column entry counts.
// 1. The ranking (key descending, index ascending) is a stable LSD radix sort
//    of (~key, index) pairs: 8 passes of 8 bits; per pass a per-tile digit
//    histogram, one scan over (digit, tile), and a stable scatter that ranks
//    each element among equal digits with wave ballots.
// 2. One lane per block sums its ranks in order (the order the reference
//    sums them in), so the profile is bit-identical to the sequential one.
#include "rsc_internal.h"

namespace rsc {
namespace {

constexpr int kSortTile = 4096;          // elements per tile: 256 threads x 16
constexpr int kSortChunks = kSortTile / 256;
constexpr int kDigits = 256;

__global__ __launch_bounds__(256) void sort_init_kernel(const uint64_t *__restrict__ key, int32_t n,
                                                        uint64_t *__restrict__ k_out,
                                                        int32_t *__restrict__ v_out) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        k_out[i] = ~key[i];  // ascending ~key == descending key
        v_out[i] = (int32_t)i;
    }
}

// counts[digit * n_tiles + tile]
__global__ __launch_bounds__(256) void sort_hist_kernel(const uint64_t *__restrict__ k, int32_t n, int shift,
                                                        uint32_t *__restrict__ counts, int32_t n_tiles) {
    __shared__ uint32_t h[kDigits];
    h[threadIdx.x] = 0;
    __syncthreads();
    const int64_t ts = (int64_t)blockIdx.x * kSortTile;
    for (int c = 0; c < kSortChunks; ++c) {
        const int64_t i = ts + c * 256 + threadIdx.x;
        if (i < n) atomicAdd(&h[(k[i] >> shift) & 0xFF], 1u);
    }
    __syncthreads();
    counts[(int64_t)threadIdx.x * n_tiles + blockIdx.x] = h[threadIdx.x];
}

// Exclusive scan of counts (length m) in place; one block of 1024 threads,
// each owning a contiguous range.
__global__ __launch_bounds__(1024) void sort_scan_kernel(uint32_t *__restrict__ counts, int64_t m) {
    __shared__ uint32_t sh[1024];
    const int t = threadIdx.x;
    const int64_t per = (m + 1023) / 1024;
    const int64_t lo = std::min<int64_t>(m, t * per), hi = std::min<int64_t>(m, lo + per);
    uint32_t s = 0;
    for (int64_t i = lo; i < hi; ++i) s += counts[i];
    sh[t] = s;
    __syncthreads();
    for (int off = 1; off < 1024; off <<= 1) {
        const uint32_t x = t >= off ? sh[t - off] : 0;
        __syncthreads();
        sh[t] += x;
        __syncthreads();
    }
    uint32_t run = sh[t] - s;
    for (int64_t i = lo; i < hi; ++i) {
        const uint32_t c = counts[i];
        counts[i] = run;
        run += c;
    }
}

// Stable scatter: elements are taken in index order, 256 per chunk; an
// element's destination is its digit's tile offset + the number of earlier
// elements of the tile with the same digit.
__global__ __launch_bounds__(256) void sort_scatter_kernel(const uint64_t *__restrict__ k_in,
                                                           const int32_t *__restrict__ v_in, int32_t n,
                                                           int shift, const uint32_t *__restrict__ offsets,
                                                           int32_t n_tiles, uint64_t *__restrict__ k_out,
                                                           int32_t *__restrict__ v_out) {
    __shared__ uint32_t base[kDigits];            // running position per digit in this tile
    __shared__ uint32_t wcnt[4][kDigits];         // per-wave digit counts of the current chunk
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    const uint64_t lt = (1ull << lane) - 1ull;
    base[t] = offsets[(int64_t)t * n_tiles + blockIdx.x];
    const int64_t ts = (int64_t)blockIdx.x * kSortTile;
    for (int c = 0; c < kSortChunks; ++c) {
        const int64_t i = ts + c * 256 + t;
        const bool in = i < n;
        const uint64_t kv = in ? k_in[i] : 0ull;
        const int32_t vv = in ? v_in[i] : 0;
        const uint32_t dg = (uint32_t)((kv >> shift) & 0xFF);
        // lanes of this wave with the same digit (and in range)
        uint64_t peers = __ballot(in);
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            const uint64_t bb = __ballot((dg >> b) & 1u);
            peers &= ((dg >> b) & 1u) ? bb : ~bb;
        }
        const uint32_t rank_w = __popcll(peers & lt);
        wcnt[0][t] = wcnt[1][t] = wcnt[2][t] = wcnt[3][t] = 0;
        __syncthreads();
        // the lowest lane of each peer group publishes the group's count
        if (in && (peers & lt) == 0) wcnt[w][dg] = __popcll(peers);
        __syncthreads();
        if (in) {
            uint32_t before = base[dg] + rank_w;
            for (int v = 0; v < w; ++v) before += wcnt[v][dg];
            k_out[before] = kv;
            v_out[before] = vv;
        }
        __syncthreads();
        base[t] += wcnt[0][t] + wcnt[1][t] + wcnt[2][t] + wcnt[3][t];
        __syncthreads();
    }
}

// Block j (counted from the lowest rank) covers ranks
// [max(0, n - (j+1) step), n - j step). One lane per block.
__global__ __launch_bounds__(256) void greedy_profile_kernel(const uint64_t *__restrict__ sorted_notkey,
                                                             const int32_t *__restrict__ order,
                                                             const int32_t *__restrict__ colnnz, int32_t n,
                                                             int32_t step, int32_t n_blocks,
                                                             double *__restrict__ mass,
                                                             int64_t *__restrict__ count) {
    const int32_t j = blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= n_blocks) return;
    const int64_t hi = (int64_t)n - (int64_t)j * step;
    const int64_t lo = std::max<int64_t>(0, hi - step);
    double s = 0.0;
    int64_t c = 0;
    for (int64_t p = lo; p < hi; ++p) {
        const uint64_t u = ~sorted_notkey[p];
        if (u != 0) s += sqrt(__longlong_as_double((long long)(u - 1)));
        c += colnnz[order[p]];
    }
    mass[j] = s;
    count[j] = c;
}

}  // namespace

int32_t greedy_step(int32_t n, int32_t alpha_num, int32_t alpha_den) {
    const int64_t s = ((int64_t)n * alpha_num) / alpha_den;
    return (int32_t)std::max<int64_t>(1, s);
}

int32_t greedy_blocks(int32_t n, int32_t step) { return n <= 0 ? 0 : (int32_t)ceil_div(n, step); }

size_t greedy_profile_ws_bytes(int32_t n) {
    const size_t nn = (size_t)std::max<int32_t>(n, 1);
    const size_t tiles = (size_t)ceil_div((int64_t)nn, kSortTile);
    return 2 * align_up(nn * 8, 256) + 2 * align_up(nn * 4, 256) + align_up(tiles * kDigits * 4, 256);
}

hipError_t greedy_profile_launch(const uint64_t *key, const int32_t *colnnz, int32_t n, int32_t step,
                                 double *mass, int64_t *count, int32_t *order_out, void *ws,
                                 hipStream_t stream) {
    if (n == 0) return hipSuccess;
    const size_t nn = (size_t)n;
    const int32_t n_tiles = (int32_t)ceil_div(n, kSortTile);
    char *p = static_cast<char *>(ws);
    uint64_t *ka = reinterpret_cast<uint64_t *>(p);
    p += align_up(nn * 8, 256);
    uint64_t *kb = reinterpret_cast<uint64_t *>(p);
    p += align_up(nn * 8, 256);
    int32_t *va = reinterpret_cast<int32_t *>(p);
    p += align_up(nn * 4, 256);
    int32_t *vb = reinterpret_cast<int32_t *>(p);
    p += align_up(nn * 4, 256);
    uint32_t *counts = reinterpret_cast<uint32_t *>(p);
    const unsigned g = (unsigned)std::min<int64_t>(ceil_div(n, 256), 4096);
    sort_init_kernel<<<g, 256, 0, stream>>>(key, n, ka, va);
    for (int pass = 0; pass < 8; ++pass) {
        const int shift = 8 * pass;
        sort_hist_kernel<<<n_tiles, 256, 0, stream>>>(ka, n, shift, counts, n_tiles);
        sort_scan_kernel<<<1, 1024, 0, stream>>>(counts, (int64_t)kDigits * n_tiles);
        sort_scatter_kernel<<<n_tiles, 256, 0, stream>>>(ka, va, n, shift, counts, n_tiles, kb, vb);
        std::swap(ka, kb);
        std::swap(va, vb);
    }
    const int32_t nb = greedy_blocks(n, step);
    greedy_profile_kernel<<<(unsigned)ceil_div(nb, 256), 256, 0, stream>>>(ka, va, colnnz, n, step, nb,
                                                                          mass, count);
    if (order_out) {
        const hipError_t e = hipMemcpyAsync(order_out, va, nn * 4, hipMemcpyDeviceToDevice, stream);
        if (e != hipSuccess) return e;
    }
    return hipGetLastError();
}

}  // namespace rsc
