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
//    histogram, a scan of each digit's tile counts (one wave per digit), and
//    a stable scatter that places each digit after the smaller digits' totals
//    and ranks each element among equal digits with wave ballots.
// 2. sqrt(q) and the column entry count are gathered per rank in parallel;
//    then one wave per block adds its ranks' sqrt(q) one after another in
//    rank order (the order that defines the sum), so the profile is
//    bit-identical to the sequential one.
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

// Per digit: exclusive scan of its tile counts in place (counts are stored
// digit-major, counts[digit * n_tiles + tile]) and the digit's total. One
// wave per digit, 64 tiles per step.
__global__ __launch_bounds__(256) void sort_digit_scan_kernel(uint32_t *__restrict__ counts, int32_t n_tiles,
                                                              uint32_t *__restrict__ dtot) {
    const int lane = threadIdx.x & 63;
    const int dg = blockIdx.x * 4 + (threadIdx.x >> 6);
    uint32_t *row = counts + (int64_t)dg * n_tiles;
    uint32_t carry = 0;
    for (int32_t t0 = 0; t0 < n_tiles; t0 += 64) {
        const int32_t t = t0 + lane;
        const uint32_t v = t < n_tiles ? row[t] : 0u;
        uint32_t incl = v;
        for (int off = 1; off < 64; off <<= 1) {
            const uint32_t x = __shfl_up(incl, off);
            if (lane >= off) incl += x;
        }
        if (t < n_tiles) row[t] = carry + incl - v;
        carry += __shfl(incl, 63);
    }
    if (lane == 0) dtot[dg] = carry;
}

// Stable scatter: elements are taken in index order, 256 per chunk; an
// element's destination is its digit's tile offset + the number of earlier
// elements of the tile with the same digit.
__global__ __launch_bounds__(256) void sort_scatter_kernel(const uint64_t *__restrict__ k_in,
                                                           const int32_t *__restrict__ v_in, int32_t n,
                                                           int shift, const uint32_t *__restrict__ offsets,
                                                           const uint32_t *__restrict__ dtot, int32_t n_tiles,
                                                           uint64_t *__restrict__ k_out,
                                                           int32_t *__restrict__ v_out) {
    __shared__ uint32_t base[kDigits];            // running position per digit in this tile
    __shared__ uint32_t wcnt[4][kDigits];         // per-wave digit counts of the current chunk
    __shared__ uint32_t wsum[4];
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    const uint64_t lt = (1ull << lane) - 1ull;
    // start of digit t in the output: exclusive scan of the digit totals
    const uint32_t tot = dtot[t];
    uint32_t incl = tot;
    for (int off = 1; off < 64; off <<= 1) {
        const uint32_t x = __shfl_up(incl, off);
        if (lane >= off) incl += x;
    }
    if (lane == 63) wsum[w] = incl;
    __syncthreads();
    uint32_t before = incl - tot;
    for (int v = 0; v < w; ++v) before += wsum[v];
    base[t] = before + offsets[(int64_t)t * n_tiles + blockIdx.x];
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
            uint32_t pos = base[dg] + rank_w;
            for (int v = 0; v < w; ++v) pos += wcnt[v][dg];
            k_out[pos] = kv;
            v_out[pos] = vv;
        }
        __syncthreads();
        base[t] += wcnt[0][t] + wcnt[1][t] + wcnt[2][t] + wcnt[3][t];
        __syncthreads();
    }
}

// Per rank p (ascending = best first): sqrt(q) of the pair at that rank in
// fp64 and the entry count of its column, gathered in parallel so the
// in-order sums below read contiguous arrays.
__global__ __launch_bounds__(256) void rank_values_kernel(const uint64_t *__restrict__ sorted_notkey,
                                                          const int32_t *__restrict__ order,
                                                          const int32_t *__restrict__ colnnz, int32_t n,
                                                          double *__restrict__ rv, int32_t *__restrict__ rc) {
    for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < n;
         p += (int64_t)gridDim.x * blockDim.x) {
        const uint64_t u = ~sorted_notkey[p];
        rv[p] = u != 0 ? sqrt(__longlong_as_double((long long)(u - 1))) : 0.0;
        rc[p] = colnnz[order[p]];
    }
}

// Block j (counted from the lowest rank) covers ranks
// [max(0, n - (j+1) step), n - j step); one wave per block. The wave loads 64
// ranks at a time (the next 64 in flight meanwhile); the fp64 mass is added
// one rank after another in ascending rank order (the order that defines
// it), the integer count by a wave reduction (exact in any order).
__global__ __launch_bounds__(64) void greedy_profile_kernel(const double *__restrict__ rv,
                                                            const int32_t *__restrict__ rc, int32_t n,
                                                            int32_t step, int32_t n_blocks,
                                                            double *__restrict__ mass,
                                                            int64_t *__restrict__ count) {
    const int32_t j = blockIdx.x;
    if (j >= n_blocks) return;
    const int lane = threadIdx.x;
    const int64_t hi = (int64_t)n - (int64_t)j * step;
    const int64_t lo = std::max<int64_t>(0, hi - step);
    int64_t c = 0;
    for (int64_t b = lo + lane; b < hi; b += 64) c += rc[b];
    for (int off = 32; off > 0; off >>= 1) c += __shfl_xor(c, off);
    // the chain reads its values from LDS at one address for all lanes (a
    // broadcast read into a vector register), so no broadcast instruction
    // sits between two adds; two 64-value buffers, the next one filled
    // while the current one is summed
    __shared__ double buf[2][64];
    double s = 0.0;
    double x = lo + lane < hi ? rv[lo + lane] : 0.0;
    int cur = 0;
    for (int64_t base = lo; base < hi; base += 64) {
        const int32_t cnt = (int32_t)std::min<int64_t>(64, hi - base);
        buf[cur][lane] = x;
        const double xn = base + 64 + lane < hi ? rv[base + 64 + lane] : 0.0;  // the next 64, in flight
        __syncthreads();  // one-wave block: the buffer is written
        const double *bp = buf[cur];
        if (cnt == 64) {
#pragma unroll
            for (int t0 = 0; t0 < 64; t0 += 8) {
                double w[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) w[u] = bp[t0 + u];
#pragma unroll
                for (int u = 0; u < 8; ++u) s += w[u];
            }
        } else {
            for (int t = 0; t < cnt; ++t) s += bp[t];
        }
        cur ^= 1;
        x = xn;
    }
    if (lane == 0) {
        mass[j] = s;
        count[j] = c;
    }
}

// ---- staleness of a selection (section 3.3.1, Fig. 4) ---------------------
// For a previous selection S (mask prev) and a new ranking `order` (pairs
// best first): the matching score of S under the new ranking is the share of
// (selected, unselected) pairs that the ranking puts in that order. With the
// selected pairs at ranks r_1 < ... < r_k, the unselected pairs after rank
// r_j number (n - 1 - r_j) - (k - j), so the count of ordered pairs is
// sum_j (n - 1 - r_j) - k (k - 1) / 2: one pass over the ranks adds
// n - 1 - r for every selected pair. Integer sums with integer atomics, so
// the result does not depend on the order of the blocks.
//   acc[0] = sum of (n - 1 - r) over ranks r whose pair is in prev
//   acc[1] = number of those ranks
//   acc[2] = ranks whose entry lies outside [0, n) (not a ranking)
//   acc[3] = |prev| from the mask words, acc[4] = |prev & cur|
constexpr int kStaleAcc = 5;

__global__ __launch_bounds__(64) void stale_zero_kernel(unsigned long long *__restrict__ acc) {
    if (threadIdx.x < kStaleAcc) acc[threadIdx.x] = 0;
}

__device__ __forceinline__ unsigned long long wave_sum_u64(unsigned long long v) {
#pragma unroll
    for (int m = 1; m < kWave; m <<= 1) v += __shfl_xor(v, m);
    return v;
}

__global__ __launch_bounds__(256) void stale_count_kernel(const int32_t *__restrict__ order, int32_t n,
                                                          const uint32_t *__restrict__ prev,
                                                          const uint32_t *__restrict__ cur,
                                                          unsigned long long *__restrict__ acc) {
    unsigned long long v[kStaleAcc] = {0, 0, 0, 0, 0};
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < n; r += stride) {
        const int32_t i = order[r];
        if ((uint32_t)i >= (uint32_t)n) {
            v[2] += 1;
        } else if ((prev[i >> 5] >> (i & 31)) & 1u) {
            v[0] += (unsigned long long)(n - 1 - r);
            v[1] += 1;
        }
    }
    const int64_t words = ((int64_t)n + 31) / 32;
    for (int64_t w = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; w < words; w += stride) {
        uint32_t p = prev[w];
        if (w == words - 1 && (n & 31)) p &= (1u << (n & 31)) - 1u;  // bits past n are not pairs
        v[3] += __popc(p);
        v[4] += __popc(p & cur[w]);
    }
    __shared__ unsigned long long part[256 / kWave][kStaleAcc];
    const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
#pragma unroll
    for (int j = 0; j < kStaleAcc; ++j) {
        const unsigned long long t = wave_sum_u64(v[j]);
        if (lane == 0) part[wv][j] = t;
    }
    __syncthreads();
    if (threadIdx.x < kStaleAcc) {
        unsigned long long t = 0;
        for (int q = 0; q < 256 / kWave; ++q) t += part[q][threadIdx.x];
        if (t) atomicAdd(&acc[threadIdx.x], t);
    }
}

}  // namespace

int32_t staleness_acc_count() { return kStaleAcc; }

hipError_t staleness_launch(const int32_t *order, int32_t n, const uint32_t *prev, const uint32_t *cur,
                            unsigned long long *acc, hipStream_t stream) {
    stale_zero_kernel<<<1, 64, 0, stream>>>(acc);
    if (n > 0) {
        const int64_t work = std::max<int64_t>(n, ceil_div(n, 32));
        const unsigned g = (unsigned)std::min<int64_t>(ceil_div(work, 256), 1024);
        stale_count_kernel<<<g, 256, 0, stream>>>(order, n, prev, cur, acc);
    }
    return hipGetLastError();
}

int32_t greedy_step(int32_t n, int32_t alpha_num, int32_t alpha_den) {
    // callers pass 0 <= alpha_num <= alpha_den, so 0 <= s <= n fits int32
    const int64_t s = ((int64_t)n * alpha_num) / alpha_den;
    return (int32_t)std::max<int64_t>(1, s);
}

int32_t greedy_blocks(int32_t n, int32_t step) { return n <= 0 ? 0 : (int32_t)ceil_div(n, step); }

size_t greedy_profile_ws_bytes(int32_t n) {
    const size_t nn = (size_t)std::max<int32_t>(n, 1);
    const size_t tiles = (size_t)ceil_div((int64_t)nn, kSortTile);
    return 2 * align_up(nn * 8, 256) + 2 * align_up(nn * 4, 256) + align_up(tiles * kDigits * 4, 256) +
           align_up(kDigits * 4, 256);
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
    p += align_up((size_t)n_tiles * kDigits * 4, 256);
    uint32_t *dtot = reinterpret_cast<uint32_t *>(p);
    const unsigned g = (unsigned)std::min<int64_t>(ceil_div(n, 256), 4096);
    sort_init_kernel<<<g, 256, 0, stream>>>(key, n, ka, va);
    for (int pass = 0; pass < 8; ++pass) {
        const int shift = 8 * pass;
        sort_hist_kernel<<<n_tiles, 256, 0, stream>>>(ka, n, shift, counts, n_tiles);
        sort_digit_scan_kernel<<<kDigits / 4, 256, 0, stream>>>(counts, n_tiles, dtot);
        sort_scatter_kernel<<<n_tiles, 256, 0, stream>>>(ka, va, n, shift, counts, dtot, n_tiles, kb, vb);
        std::swap(ka, kb);
        std::swap(va, vb);
    }
    // after an even number of passes the ranking is back in (ka, va); kb and vb are free
    double *rv = reinterpret_cast<double *>(kb);
    int32_t *rc = vb;
    rank_values_kernel<<<g, 256, 0, stream>>>(ka, va, colnnz, n, rv, rc);
    const int32_t nb = greedy_blocks(n, step);
    greedy_profile_kernel<<<(unsigned)nb, 64, 0, stream>>>(rv, rc, n, step, nb, mass, count);
    if (order_out) {
        const hipError_t e = hipMemcpyAsync(order_out, va, nn * 4, hipMemcpyDeviceToDevice, stream);
        if (e != hipSuccess) return e;
    }
    return hipGetLastError();
}

}  // namespace rsc
