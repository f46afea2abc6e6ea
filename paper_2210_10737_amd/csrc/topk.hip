// Top-k selection (section 2.2.1): the k largest uint64 keys, ties broken by
// the lower index, returned as ascending indices and an n-bit mask.
//
// 1. Radix select of the threshold T = the k-th largest key, most significant
//    digit first: 6 passes of 11/11/11/11/10/10 bits. Each pass builds a
//    grid-wide histogram of the digit over the keys that match the prefix
//    chosen so far (LDS histograms, then integer atomics into global bins).
//    The digit that holds the k-th key is picked at the start of the next
//    kernel: every block reads the finished histogram and makes the same
//    pick (a wave-shuffle scan over the bins), and its first block records
//    the state after it, one slot per pass, so no kernel of its own is
//    needed. After the last pass T is known, and r = the number of keys
//    equal to T that must be kept (G = k - r keys are strictly above T).
// 2. Tiles of 4096 keys count (== T) and (> T) (their kernel makes the last
//    pick); one block scans the tile counts; a third kernel keeps key i iff
//    key > T, or key == T and fewer than r equal keys precede it, writing
//    mask words from wave ballots and idx at the running count of kept keys.
//    Everything is integer, so the result is exact and deterministic.
// Up to 16,384 keys the whole selection runs in one block with the keys in
// LDS (one launch; the small graphs are launch-bound).
#include "rsc_internal.h"

namespace rsc {
namespace {

constexpr int kBins = 2048;
constexpr int kTile = 4096;     // keys per tile: 4 waves x 16 groups of 64
constexpr int kPasses = 6;

// Of eq keys equal to the threshold, how many are taken when want more are
// still wanted: want clamped to [0, eq], in integers.
__device__ __forceinline__ int64_t clamp_take(int64_t want, int64_t eq) {
    return want < 0 ? 0 : (want < eq ? want : eq);
}

__constant__ const int kShift[kPasses] = {53, 42, 31, 20, 10, 0};
__constant__ const int kWidth[kPasses] = {11, 11, 11, 11, 10, 10};

struct TopkState {
    uint64_t prefix;  // digits of T fixed so far
    uint64_t pmask;   // which bits of prefix are fixed
    int64_t k_rem;    // how many keys among those matching prefix remain to be taken
    int64_t pad;
};

// st[p] = the state after p picks (st[0] initial, st[kPasses] final: prefix
// = T, k_rem = r); the histogram of pass p is hist[p % 3] (pass p reads
// pass p - 1's and clears pass p + 1's, three distinct buffers).
struct TopkWs {
    TopkState st[kPasses + 1];
    uint32_t hist[3][kBins];
};

struct PickOut {
    uint64_t prefix, pmask;
    int64_t k_rem, count;
};

// One block of 256 threads picks the digit of `pass` from histogram h,
// starting from state *sp: thread t owns the bins nb-1-t*per .. nb-per-t*per
// (descending), and an exclusive scan over threads (within each wave by
// shuffles, then over the four wave totals) gives the count of keys in
// higher bins. Every thread gets the new state.
__device__ void block_pick_256(const TopkState *sp, const uint32_t *h, int pass, uint64_t &prefix, uint64_t &pmask,
                               int64_t &k_rem, int64_t *wsum, PickOut *s_out) {
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    const int shift = kShift[pass];
    const int nb = 1 << kWidth[pass];
    const int per = nb / 256;  // 8 or 4
    uint32_t hv[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) hv[j] = j < per ? h[nb - 1 - (t * per + j)] : 0u;
    prefix = sp->prefix;
    pmask = sp->pmask;
    k_rem = sp->k_rem;
    int64_t s = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) s += hv[j];
    int64_t incl = s;
    for (int off = 1; off < 64; off <<= 1) {
        const int64_t x = __shfl_up(incl, off);
        if (lane >= off) incl += x;
    }
    if (lane == 63) wsum[w] = incl;
    __syncthreads();
    int64_t run = incl - s;  // keys in bins above this thread's range
    for (int u = 0; u < w; ++u) run += wsum[u];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int64_t c = hv[j];
        if (j < per && run < k_rem && run + c >= k_rem) {  // exactly one (thread, bin) satisfies this
            const int b = nb - 1 - (t * per + j);
            s_out->prefix = prefix | ((uint64_t)b << shift);
            s_out->pmask = pmask | ((uint64_t)(nb - 1) << shift);
            s_out->k_rem = k_rem - run;
        }
        run += c;
    }
    __syncthreads();
    prefix = s_out->prefix;
    pmask = s_out->pmask;
    k_rem = s_out->k_rem;
}

__global__ __launch_bounds__(256) void topk_init_kernel(TopkWs *h, int64_t k) {
    for (int b = threadIdx.x; b < kBins; b += blockDim.x) h->hist[0][b] = 0;
    if (threadIdx.x == 0) {
        h->st[0].prefix = 0;
        h->st[0].pmask = 0;
        h->st[0].k_rem = k;
    }
}

// Pass p: the pick of pass p - 1 (from its finished histogram; the first
// block records the state in st[p]), the clearing of pass p + 1's histogram,
// then this pass's histogram over the keys that match the prefix.
__global__ __launch_bounds__(256) void topk_hist_kernel(const uint64_t *__restrict__ key, int32_t n, TopkWs *ws,
                                                        int pass) {
    __shared__ uint32_t lh[kBins];
    __shared__ int64_t wsum[4];
    __shared__ PickOut s_out;
    const int shift = kShift[pass];
    const uint64_t dmask = (1ull << kWidth[pass]) - 1ull;
    for (int b = threadIdx.x; b < kBins; b += blockDim.x) lh[b] = 0;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    // eight keys per thread loaded before any is counted (the first eight
    // before the pick, so the two waits overlap), then the rest one at a time
    uint64_t k[8];
    bool more = i + 7 * stride < n;
    if (more) {
#pragma unroll
        for (int u = 0; u < 8; ++u) k[u] = key[i + u * stride];
    }
    uint64_t prefix = ws->st[0].prefix, pmask = ws->st[0].pmask;
    if (pass > 0) {
        int64_t k_rem;
        block_pick_256(&ws->st[pass - 1], ws->hist[(pass - 1) % 3], pass - 1, prefix, pmask, k_rem, wsum, &s_out);
        if (blockIdx.x == 0 && threadIdx.x == 0) {
            ws->st[pass].prefix = prefix;
            ws->st[pass].pmask = pmask;
            ws->st[pass].k_rem = k_rem;
        }
    }
    if (blockIdx.x == 0)
        for (int b = threadIdx.x; b < kBins; b += blockDim.x) ws->hist[(pass + 1) % 3][b] = 0;
    __syncthreads();  // lh cleared
    uint32_t *hist = ws->hist[pass % 3];
    while (more) {
        if (pass == 0) {  // block-uniform
            // the top digit is nearly constant over the keys: a wave whose
            // keys all share one digit adds them with one LDS atomic
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const uint32_t dg = (uint32_t)((k[u] >> shift) & dmask);
                const uint32_t d0 = __shfl(dg, 0);
                if (__ballot(dg == d0) == ~0ull) {
                    if ((threadIdx.x & 63) == 0) atomicAdd(&lh[d0], 64u);
                } else {
                    atomicAdd(&lh[dg], 1u);
                }
            }
        } else {
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if ((k[u] & pmask) == prefix) atomicAdd(&lh[(k[u] >> shift) & dmask], 1u);
        }
        i += 8 * stride;
        more = i + 7 * stride < n;
        if (more) {
#pragma unroll
            for (int u = 0; u < 8; ++u) k[u] = key[i + u * stride];
        }
    }
    for (; i < n; i += stride) {
        const uint64_t kv = key[i];
        if ((kv & pmask) == prefix) atomicAdd(&lh[(kv >> shift) & dmask], 1u);
    }
    __syncthreads();
    for (int b = threadIdx.x; b < (1 << kWidth[pass]); b += blockDim.x)
        if (lh[b]) atomicAdd(&hist[b], lh[b]);
}

// Also makes the last pass's pick (every block; the first records the final
// state, T and r, for the scan and the emit).
__global__ __launch_bounds__(256) void topk_tile_count_kernel(const uint64_t *__restrict__ key,
                                                              int32_t n, TopkWs *ws,
                                                              uint32_t *__restrict__ tile_eq,
                                                              uint32_t *__restrict__ tile_gt) {
    __shared__ uint32_t s_eq[4], s_gt[4];
    __shared__ int64_t wsum[4];
    __shared__ PickOut s_out;
    // the tile's keys are loaded before the pick, so the two waits overlap
    const int64_t ts = (int64_t)blockIdx.x * kTile;
    uint64_t kv[kTile / 256];
#pragma unroll
    for (int j = 0; j < kTile / 256; ++j) {
        const int64_t i = ts + threadIdx.x + 256 * j;
        kv[j] = i < n ? key[i] : 0ull;
    }
    uint64_t T, pmask;
    int64_t r;
    block_pick_256(&ws->st[kPasses - 1], ws->hist[(kPasses - 1) % 3], kPasses - 1, T, pmask, r, wsum, &s_out);
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        ws->st[kPasses].prefix = T;
        ws->st[kPasses].pmask = pmask;
        ws->st[kPasses].k_rem = r;
    }
    uint32_t eq = 0, gt = 0;
#pragma unroll
    for (int j = 0; j < kTile / 256; ++j) {
        const bool in = ts + threadIdx.x + 256 * j < n;
        eq += in && kv[j] == T;
        gt += in && kv[j] > T;
    }
    for (int off = 32; off > 0; off >>= 1) {
        eq += __shfl_down(eq, off);
        gt += __shfl_down(gt, off);
    }
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    if (lane == 0) { s_eq[w] = eq; s_gt[w] = gt; }
    __syncthreads();
    if (threadIdx.x == 0) {
        tile_eq[blockIdx.x] = s_eq[0] + s_eq[1] + s_eq[2] + s_eq[3];
        tile_gt[blockIdx.x] = s_gt[0] + s_gt[1] + s_gt[2] + s_gt[3];
    }
}

// Block-wide exclusive scan (1024 threads, values int64): within each wave
// by shuffles, then over the 16 wave totals (sh holds at least 16 entries).
__device__ int64_t block_exclusive_scan_1024(int64_t v, int64_t *sh, int64_t *total) {
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    int64_t incl = v;
    for (int off = 1; off < 64; off <<= 1) {
        const int64_t x = __shfl_up(incl, off);
        if (lane >= off) incl += x;
    }
    if (lane == 63) sh[w] = incl;
    __syncthreads();
    int64_t before = 0, tot = 0;
    for (int u = 0; u < 16; ++u) {
        const int64_t x = sh[u];
        before += u < w ? x : 0;
        tot += x;
    }
    *total = tot;
    __syncthreads();  // sh may be rewritten by the next call
    return before + incl - v;
}

// One block of 1024 threads picks the digit of `pass` from histogram h
// (nb bins; LDS or global): thread t owns bins nb-1-(t*per+j), descending,
// and the exclusive scan gives the keys in all higher bins. Updates
// prefix/pmask/k_rem for every thread and returns the picked bin's count.
__device__ int64_t block_pick_1024(const uint32_t *h, int pass, uint64_t &prefix, uint64_t &pmask, int64_t &k_rem,
                                   int64_t *s_scan, PickOut *s_out) {
    const int t = threadIdx.x;
    const int shift = kShift[pass];
    const int nb = 1 << kWidth[pass];
    const uint64_t dmask = (uint64_t)(nb - 1);
    const int per = nb / 1024;  // 2 or 1
    int64_t sum = 0;
    for (int j = 0; j < per; ++j) sum += h[nb - 1 - (t * per + j)];
    int64_t total;
    int64_t run = block_exclusive_scan_1024(sum, s_scan, &total);
    for (int j = 0; j < per; ++j) {
        const int b = nb - 1 - (t * per + j);
        const int64_t c = h[b];
        if (run < k_rem && run + c >= k_rem) {  // exactly one (thread, bin)
            s_out->prefix = prefix | ((uint64_t)b << shift);
            s_out->pmask = pmask | (dmask << shift);
            s_out->k_rem = k_rem - run;
            s_out->count = c;
        }
        run += c;
    }
    __syncthreads();
    prefix = s_out->prefix;
    pmask = s_out->pmask;
    k_rem = s_out->k_rem;
    const int64_t count = s_out->count;
    __syncthreads();  // every thread has read s_out before it is written again
    return count;
}

// One block of 1024 threads; thread t owns a contiguous range of tiles.
__global__ __launch_bounds__(1024) void topk_tile_scan_kernel(int32_t nt, const TopkState *__restrict__ st,
                                                              const uint32_t *__restrict__ tile_eq,
                                                              const uint32_t *__restrict__ tile_gt,
                                                              uint32_t *__restrict__ eq_before,
                                                              uint32_t *__restrict__ sel_before) {
    __shared__ int64_t sh[16];
    const int t = threadIdx.x;
    const int32_t per = (nt + 1023) / 1024;
    const int32_t lo = min(nt, t * per), hi = min(nt, lo + per);
    const int64_t r = st->k_rem;
    int64_t tot;
    int64_t s = 0;
    for (int32_t i = lo; i < hi; ++i) s += tile_eq[i];
    int64_t run = block_exclusive_scan_1024(s, sh, &tot);
    int64_t sel_local = 0;
    for (int32_t i = lo; i < hi; ++i) {
        eq_before[i] = (uint32_t)run;
        const int64_t take = clamp_take(r - run, tile_eq[i]);
        sel_local += tile_gt[i] + take;
        run += tile_eq[i];
    }
    int64_t srun = block_exclusive_scan_1024(sel_local, sh, &tot);
    for (int32_t i = lo; i < hi; ++i) {
        sel_before[i] = (uint32_t)srun;
        const int64_t eb = eq_before[i];
        const int64_t take = clamp_take(r - eb, tile_eq[i]);
        srun += tile_gt[i] + take;
    }
}

__global__ __launch_bounds__(256) void topk_emit_kernel(const uint64_t *__restrict__ key, int32_t n,
                                                        const TopkState *__restrict__ st,
                                                        const uint32_t *__restrict__ eq_before,
                                                        const uint32_t *__restrict__ sel_before,
                                                        int32_t *__restrict__ idx,
                                                        uint32_t *__restrict__ mask, int32_t k) {
    __shared__ uint32_t s_eq[4], s_gt[4];
    const uint64_t T = st->prefix;
    const int64_t r = st->k_rem;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const uint64_t lt_mask = (1ull << lane) - 1ull;
    const int64_t wbase = (int64_t)blockIdx.x * kTile + (int64_t)w * (kTile / 4);
    const int64_t nwords = ((int64_t)n + 31) / 32;
    uint32_t eq = 0, gt = 0;
    for (int g = 0; g < kTile / 4 / 64; ++g) {
        const int64_t i = wbase + 64 * g + lane;
        const bool in = i < n;
        const uint64_t kv = in ? key[i] : 0ull;
        eq += __popcll(__ballot(in && kv == T));
        gt += __popcll(__ballot(in && kv > T));
    }
    if (lane == 0) { s_eq[w] = eq; s_gt[w] = gt; }
    __syncthreads();
    int64_t eq_base = eq_before[blockIdx.x], sel_base = sel_before[blockIdx.x];
    for (int v = 0; v < w; ++v) {
        const int64_t take = clamp_take(r - eq_base, s_eq[v]);
        sel_base += s_gt[v] + take;
        eq_base += s_eq[v];
    }
    for (int g = 0; g < kTile / 4 / 64; ++g) {
        const int64_t base = wbase + 64 * g;
        const int64_t i = base + lane;
        const bool in = i < n;
        const uint64_t kv = in ? key[i] : 0ull;
        const bool is_eq = in && kv == T;
        const uint64_t eqbal = __ballot(is_eq);
        const bool sel = (in && kv > T) || (is_eq && eq_base + __popcll(eqbal & lt_mask) < r);
        const uint64_t selbal = __ballot(sel);
        const int64_t pos = sel_base + __popcll(selbal & lt_mask);
        if (sel && pos < k) idx[pos] = (int32_t)i;
        const int64_t word = base / 32;
        if (lane == 0 && word < nwords) mask[word] = (uint32_t)selbal;
        if (lane == 32 && word + 1 < nwords) mask[word + 1] = (uint32_t)(selbal >> 32);
        eq_base += __popcll(eqbal);
        sel_base += __popcll(selbal);
    }
}

// Small inputs (n <= kSmallN) in one block of 1024 threads, the keys held in
// LDS: the same six radix passes (LDS histogram, a block scan picks the
// digit), then thread t takes keys [16 t, 16 t + 16): block scans of its
// (== T) count and of its kept count give the ranks, idx is written at the
// running kept count and each 16-bit piece of the mask is paired with its
// neighbour's into a word. One launch instead of fifteen; same result.
constexpr int kSmallN = 16384;
constexpr int kSmallThreads = 1024;
constexpr int kSmallPer = kSmallN / kSmallThreads;  // 16 keys per thread in the emit
static_assert(kSmallPer == 16, "two threads' 16-bit pieces make one mask word");

__global__ __launch_bounds__(kSmallThreads) void topk_small_kernel(const uint64_t *__restrict__ key, int32_t n,
                                                                   int32_t k, int32_t *__restrict__ idx,
                                                                   uint32_t *__restrict__ mask) {
    __shared__ uint64_t s_key[kSmallN];
    __shared__ uint32_t s_hist[kBins];
    __shared__ int64_t s_scan[kSmallThreads / 64];
    __shared__ PickOut s_out;
    const int t = threadIdx.x;
    for (int i = t; i < n; i += kSmallThreads) s_key[i] = key[i];
    uint64_t prefix = 0, pmask = 0;
    int64_t k_rem = k;
    for (int pass = 0; pass < kPasses; ++pass) {
        const int shift = kShift[pass];
        const uint64_t dmask = (1ull << kWidth[pass]) - 1ull;
        for (int b = t; b < kBins; b += kSmallThreads) s_hist[b] = 0;
        __syncthreads();  // keys loaded (first pass), histogram cleared
        for (int i = t; i < n; i += kSmallThreads) {
            const uint64_t kv = s_key[i];
            if ((kv & pmask) == prefix) atomicAdd(&s_hist[(kv >> shift) & dmask], 1u);
        }
        __syncthreads();
        block_pick_1024(s_hist, pass, prefix, pmask, k_rem, s_scan, &s_out);
    }
    const uint64_t T = prefix;
    const int64_t r = k_rem;  // keys equal to T that are kept (the lowest indices)
    const int lo = min(n, t * kSmallPer), hi = min(n, lo + kSmallPer);
    int64_t eq = 0;
    for (int i = lo; i < hi; ++i) eq += s_key[i] == T;
    int64_t total;
    int64_t eq_before = block_exclusive_scan_1024(eq, s_scan, &total);
    uint32_t bits = 0;
    int64_t kept = 0;
    for (int i = lo; i < hi; ++i) {
        const uint64_t kv = s_key[i];
        bool sel = kv > T;
        if (kv == T) sel = eq_before++ < r;
        if (sel) {
            bits |= 1u << (i - lo);
            ++kept;
        }
    }
    int64_t pos = block_exclusive_scan_1024(kept, s_scan, &total);
    for (int i = lo; i < hi; ++i)
        if ((bits >> (i - lo)) & 1u) idx[pos++] = i;
    const uint32_t hi16 = __shfl_down(bits, 1);  // the odd neighbour's piece
    const int64_t word = t / 2;
    if ((t & 1) == 0 && word < ((int64_t)n + 31) / 32) mask[word] = bits | (hi16 << 16);
}

__global__ __launch_bounds__(256) void fill_u32_kernel(uint32_t *p, int64_t count, uint32_t v) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

}  // namespace

size_t topk_ws_bytes(int32_t n) {
    const size_t nt = (size_t)ceil_div(std::max<int32_t>(n, 1), kTile);
    return align_up(sizeof(TopkWs), 256) + 4 * align_up(nt * sizeof(uint32_t), 256);
}

hipError_t topk_launch(const uint64_t *key, int32_t n, int32_t k, int32_t *idx, uint32_t *mask,
                       void *ws, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    const int64_t nwords = ceil_div(n, 32);
    if (k == 0) {
        fill_u32_kernel<<<(unsigned)std::min<int64_t>(ceil_div(nwords, 256), 1024), 256, 0, stream>>>(
            mask, nwords, 0u);
        return hipGetLastError();
    }
    if (n <= kSmallN) {
        topk_small_kernel<<<1, kSmallThreads, 0, stream>>>(key, n, k, idx, mask);
        return hipGetLastError();
    }
    TopkWs *h = static_cast<TopkWs *>(ws);
    const int32_t nt = (int32_t)ceil_div(n, kTile);
    char *p = static_cast<char *>(ws) + align_up(sizeof(TopkWs), 256);
    const size_t tb = align_up((size_t)nt * sizeof(uint32_t), 256);
    uint32_t *tile_eq = reinterpret_cast<uint32_t *>(p);
    uint32_t *tile_gt = reinterpret_cast<uint32_t *>(p + tb);
    uint32_t *eq_before = reinterpret_cast<uint32_t *>(p + 2 * tb);
    uint32_t *sel_before = reinterpret_cast<uint32_t *>(p + 3 * tb);

    topk_init_kernel<<<1, 256, 0, stream>>>(h, k);
    // Each block flushes its non-empty bins with one global atomic each. The
    // first two passes count every key, into a few bins (pass 0) or into
    // most of them (pass 1), so they run on 256 and 128 blocks to keep those
    // atomics few (measured on 2.45M keys: 12.4 and 9.5 us, against 18.9 and
    // 29.6 with eight keys per thread); later passes count only the keys
    // under the chosen prefix and take eight keys per thread, for more loads
    // in flight.
    const unsigned hgrid_wide = (unsigned)std::min<int64_t>(ceil_div(n, 256 * 8), 2048);
    const unsigned hgrid_pass[2] = {std::min(hgrid_wide, 256u), std::min(hgrid_wide, 128u)};
    for (int pass = 0; pass < kPasses; ++pass)
        topk_hist_kernel<<<pass < 2 ? hgrid_pass[pass] : hgrid_wide, 256, 0, stream>>>(key, n, h, pass);
    topk_tile_count_kernel<<<nt, 256, 0, stream>>>(key, n, h, tile_eq, tile_gt);
    topk_tile_scan_kernel<<<1, 1024, 0, stream>>>(nt, &h->st[kPasses], tile_eq, tile_gt, eq_before, sel_before);
    topk_emit_kernel<<<nt, 256, 0, stream>>>(key, n, &h->st[kPasses], eq_before, sel_before, idx, mask, k);
    return hipGetLastError();
}

}  // namespace rsc
