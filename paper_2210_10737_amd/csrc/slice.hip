// Column slice of a CSR matrix, A' = A[:, S] (section 3.3.1 and Fig. 5's
// rebuild of Rowptr and Col; appendix C: whole columns are dropped, every row
// is kept, so rows may become empty).
//
// Entry t is kept iff bit col[t] of the mask is set. Because kept entries
// stay in their original order, the output position of a kept entry is the
// number of kept entries before it, and Rowptr'[i] is that count at position
// Rowptr[i]. So the slice is one stream compaction over the nnz entries:
//   0. per tile of 4096 entries: the first row whose Rowptr lies in it (a
//      table built from Rowptr; it also clears the tile counts);
//   1. per tile: the kept flags as 64 wave ballots (reads col; the n-bit mask
//      is tested from LDS, loaded piece by piece), stored for step 3, and
//      their count;
//   2. one block scans the tile counts (and stores nnz');
//   3. per tile: load col/val into registers, scan the tile's ballot counts,
//      compact the kept entries in LDS and write them out coalesced at their
//      global positions, and write Rowptr'[i] for every row whose Rowptr[i]
//      falls in the tile.
// A single-pass form (count, decoupled look-back scan over ticketed tiles,
// compaction in one kernel; below) gives the same bytes and is available on
// request; the launches above measured faster.
// Integer-only and deterministic. With a per-column scale (the randomized
// sampler's 1/(k p)), each kept value becomes fl32(val * colw[col]).
#include <cstdlib>

#include "rsc_internal.h"

namespace rsc {
namespace {

constexpr int kTile = 4096;          // entries per tile
constexpr int kPer = kTile / 256;    // 256-entry chunks per tile

// Entry o of a tile (0 <= o < kTile) is position o & 255 of chunk o >> 8;
// within a chunk, wave (o >> 6) & 3, lane o & 63. The kept flags of one
// (chunk, wave) are one 64-bit ballot, stored per tile in that order
// (tile_bits[tile * kGroups + chunk * 4 + wave]) for the emit kernel.
constexpr int kGroups = kPer * 4;
static_assert(kGroups == 64, "one wave scans the (chunk, wave) ballots of a tile");

// Count pass with the mask in LDS: random 4-byte lookups into a large bit
// set would each touch an L2 line (the set outgrows L1); in LDS they cost a
// few cycles. Persistent blocks of 1024 threads (one per CU, 156 KB of LDS
// each) walk the column range in pieces of 1,277,952 columns: load that
// piece of the mask, then test every tile's entries against it, taking
// kTilesPerIter tiles per step with the next step's column loads already in
// flight. Each wave publishes its ballots and its kept count without waiting
// for anything: the first piece stores the ballots, later pieces OR theirs in
// (an entry is kept by at most one piece; the same lane wrote the stored
// value), and every piece adds the wave's count of each tile to tile_cnt
// (cleared beforehand) with an integer atomic. No result depends on the order
// of the atomics, and the steps need no barrier.
constexpr int kMaskLdsWords = 39936;  // 156 KB of LDS: 1,277,952 columns per piece
constexpr int kCountThreads = 1024;
constexpr int kTilesPerIterSingle = 4;  // tiles per step, one block per CU
constexpr int kTilesPerIterPaired = 4;  // tiles per step, paired blocks (8 measured the same)
constexpr int kCountWaves = kCountThreads / 64;
static_assert(kTile == kCountThreads * 4, "four entries per thread per tile");

// kPaired (a mask of exactly two pieces): blocks 16 g + x and 16 g + 8 + x
// (x < 8) form pair 8 g + x; the first holds piece 0, the second piece 1,
// and both walk the pair's tiles at the same time. Blocks are dispatched to
// the 8 XCDs round-robin, so the two share an L2 and col is mostly fetched
// from HBM once; both OR their ballots into tile_bits, which starts cleared.
template <bool kPaired, int kTilesPerIter>
__global__ __launch_bounds__(kCountThreads) void slice_count_kernel(const int32_t *__restrict__ col, int64_t nnz,
                                                                    const uint32_t *__restrict__ mask,
                                                                    int32_t n_words, int32_t nt,
                                                                    uint32_t *__restrict__ tile_cnt,
                                                                    uint64_t *__restrict__ tile_bits) {
    __shared__ uint32_t s_mask[kMaskLdsWords];
    const int T = threadIdx.x, lane = T & 63, wv = T >> 6;
    const int32_t piece = kPaired ? (int32_t)((blockIdx.x >> 3) & 1) : 0;
    const int32_t group = kPaired ? (int32_t)((blockIdx.x >> 4) * 8 + (blockIdx.x & 7)) : (int32_t)blockIdx.x;
    const int32_t groups = kPaired ? (int32_t)(gridDim.x / 2) : (int32_t)gridDim.x;
    for (int32_t w0 = piece * kMaskLdsWords; w0 == piece * kMaskLdsWords || (!kPaired && w0 < n_words);
         w0 += kMaskLdsWords) {
        const int32_t words = max(0, min(kMaskLdsWords, n_words - w0));
        __syncthreads();  // the previous piece's lookups are done
        for (int i = T; i < words; i += kCountThreads) s_mask[i] = mask[w0 + i];
        __syncthreads();
        // column v is in this piece iff 0 <= v - lo < span (32-bit: both are
        // below 2^31, and the padding value -1 falls outside)
        const int32_t lo = w0 * 32;
        const uint32_t span = (uint32_t)words * 32u;
        const int32_t stride = groups * kTilesPerIter;
        // the next step's column loads are issued before this step's tests
        // (a step's tiles are consecutive: value (u, i) is entry
        // T + kCountThreads * (4 u + i) from the step's first entry)
        int32_t nx[kTilesPerIter][4];
        auto load = [&](int32_t t0) {
            const int64_t base = (int64_t)t0 * kTile;
            const int64_t left = nnz - base;
            const int32_t rem = left < (int64_t)kTilesPerIter * kTile ? (int32_t)left : kTilesPerIter * kTile;
            const int32_t *src = col + base;
#pragma unroll
            for (int u = 0; u < kTilesPerIter; ++u)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int32_t q = T + kCountThreads * (4 * u + i);
                    // paired: the partner block reads the same lines from L2
                    nx[u][i] = q < rem ? (kPaired ? src[q] : __builtin_nontemporal_load(src + q)) : -1;
                }
        };
        load(group * kTilesPerIter);
        for (int32_t t0 = group * kTilesPerIter; t0 < nt; t0 += stride) {
            int32_t cv[kTilesPerIter][4];
#pragma unroll
            for (int u = 0; u < kTilesPerIter; ++u)
#pragma unroll
                for (int i = 0; i < 4; ++i) cv[u][i] = nx[u][i];
            if (t0 + stride < nt) load(t0 + stride);
            // lane 4 u + i keeps ballot (u, i) and lane u the wave's count of
            // tile u, so the step's 16 ballots and 4 counts leave in one store
            // (or atomic) instruction each. A tile's four lookups read LDS
            // unconditionally (an index outside the piece is clamped and its
            // word ignored), so they issue together and share one wait
            // instead of each one branching and waiting on its own.
            uint64_t my_ball = 0;
            uint32_t my_cnt = 0;
#pragma unroll
            for (int u = 0; u < kTilesPerIter; ++u) {
                uint32_t off[4], word[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    off[i] = (uint32_t)(cv[u][i] - lo);
                    word[i] = s_mask[min(off[i] >> 5, (uint32_t)(kMaskLdsWords - 1))];
                }
                uint32_t c = 0;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const bool k = off[i] < span && ((word[i] >> (off[i] & 31)) & 1u);
                    const uint64_t b = __ballot(k);
                    c += __popcll(b);
                    if (lane == 4 * u + i) my_ball = b;
                }
                if (lane == u) my_cnt = c;
            }
            if (lane < 4 * kTilesPerIter && t0 + (lane >> 2) < nt) {
                // group (o >> 6) of tile t0 + u for entries T + kCountThreads * i
                uint64_t *g = tile_bits + (int64_t)(t0 + (lane >> 2)) * 64 + wv + kCountWaves * (lane & 3);
                if (w0 == 0 && !kPaired)
                    *g = my_ball;
                else if (my_ball)
                    atomicOr(reinterpret_cast<unsigned long long *>(g), (unsigned long long)my_ball);
            }
            if (lane < kTilesPerIter && my_cnt && t0 + lane < nt) atomicAdd(&tile_cnt[t0 + lane], my_cnt);
        }
    }
}

// tile_row[t] = the first row i with rowptr[i] >= t * kTile, for every tile
// t < nt: row i takes the tiles whose first entry lies in
// (rowptr[i - 1], rowptr[i]] (rowptr[-1] read as -1), so for a well-formed
// row pointer each tile is written exactly once. The emit reads its rows'
// range from here instead of two binary searches per tile. The same launch
// clears the tile counts the count pass adds into (and, for the paired count
// pass, the ballots).
__global__ __launch_bounds__(256) void slice_tile_rows_kernel(const int32_t *__restrict__ rowptr, int32_t n_rows,
                                                              int32_t nt, int32_t *__restrict__ tile_row,
                                                              uint32_t *__restrict__ tile_cnt,
                                                              uint64_t *__restrict__ tile_bits_to_clear) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t first = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    for (int64_t t = first; t < nt; t += stride) tile_cnt[t] = 0;
    if (tile_bits_to_clear)
        for (int64_t t = first; t < (int64_t)nt * kGroups; t += stride) tile_bits_to_clear[t] = 0;
    for (int64_t i = first; i <= n_rows; i += stride) {
        const int64_t a = i == 0 ? -1 : (int64_t)rowptr[i - 1];
        const int64_t b = rowptr[i];
        const int64_t t0 = a < 0 ? 0 : a / kTile + 1;  // first tile starting above a
        const int64_t t1 = min<int64_t>(b / kTile, (int64_t)nt - 1);
        for (int64_t t = t0; t <= t1; ++t) tile_row[t] = (int32_t)i;
    }
}

__global__ __launch_bounds__(1024) void slice_scan_kernel(int32_t nt, const uint32_t *__restrict__ tile_cnt,
                                                          uint32_t *__restrict__ tile_off,
                                                          int64_t *__restrict__ nnz_out) {
    __shared__ int64_t sh[1024];
    const int t = threadIdx.x;
    const int32_t per = (nt + 1023) / 1024;
    const int32_t lo = min(nt, t * per), hi = min(nt, lo + per);
    int64_t s = 0;
#pragma unroll 8
    for (int32_t i = lo; i < hi; ++i) s += tile_cnt[i];  // unrolled: 8 loads in flight, not 1
    sh[t] = s;
    __syncthreads();
    for (int off = 1; off < 1024; off <<= 1) {
        const int64_t x = t >= off ? sh[t - off] : 0;
        __syncthreads();
        sh[t] += x;
        __syncthreads();
    }
    int64_t run = sh[t] - s;
#pragma unroll 8
    for (int32_t i = lo; i < hi; ++i) {
        tile_off[i] = (uint32_t)run;
        run += tile_cnt[i];
    }
    if (t == 1023) *nnz_out = sh[1023];
}

// First index i in [0, n] with rowptr[i] >= x (rowptr has n + 1 entries).
__device__ int32_t lower_bound_rowptr(const int32_t *__restrict__ rowptr, int32_t n, int64_t x) {
    int32_t lo = 0, hi = n + 1;
    while (lo < hi) {
        const int32_t mid = lo + (hi - lo) / 2;
        if (rowptr[mid] < x) lo = mid + 1; else hi = mid;
    }
    return lo;
}

// The kept entries before entry o of a tile are the counts of the earlier
// (chunk, wave) ballots plus the ballot's bits below o's lane.
__global__ __launch_bounds__(256) void slice_emit_kernel(const int32_t *__restrict__ rowptr, int32_t n_rows,
                                                         const int32_t *__restrict__ col,
                                                         const float *__restrict__ val, int64_t nnz,
                                                         const uint64_t *__restrict__ tile_bits,
                                                         const uint32_t *__restrict__ tile_off,
                                                         const int32_t *__restrict__ tile_row,
                                                         int32_t *__restrict__ rowptr_out,
                                                         int32_t *__restrict__ col_out,
                                                         float *__restrict__ val_out, int64_t capacity,
                                                         const double *__restrict__ colw) {
    __shared__ int32_t s_col[kTile];   // kept entries of the tile, compacted
    __shared__ float s_val[kTile];
    __shared__ uint64_t s_ball[kGroups];
    __shared__ uint32_t s_pre[kGroups + 1];  // kept entries before each ballot; [kGroups] = tile total
    __shared__ int32_t s_rows[2];
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    const int64_t ts = (int64_t)blockIdx.x * kTile;
    const int64_t te = min<int64_t>(ts + kTile, nnz);
    const bool last = blockIdx.x == gridDim.x - 1;
    // the rows whose Rowptr[i] lies in the tile (clamped to [0, n_rows + 1],
    // so a malformed row pointer cannot send the stores below out of range)
    if (t == 0) s_rows[0] = min(max(tile_row[blockIdx.x], 0), n_rows + 1);
    if (t == 1) s_rows[1] = last ? n_rows + 1 : min(max(tile_row[blockIdx.x + 1], 0), n_rows + 1);
    int32_t rc[kPer];
    float rv[kPer];
    uint64_t ball[kPer];
#pragma unroll
    for (int j = 0; j < kPer; ++j) {  // coalesced loads
        const int64_t p = ts + 256 * j + t;
        rc[j] = p < te ? __builtin_nontemporal_load(col + p) : -1;
        rv[j] = p < te ? __builtin_nontemporal_load(val + p) : 0.f;
    }
    if (t < kGroups) s_ball[t] = tile_bits[(int64_t)blockIdx.x * kGroups + t];
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kPer; ++j) ball[j] = s_ball[j * 4 + w];
    if (w == 0) {  // exclusive scan of the kGroups ballot counts (kGroups == 64)
        const uint32_t cnt = __popcll(s_ball[lane]);
        uint32_t incl = cnt;
        for (int off = 1; off < 64; off <<= 1) {
            const uint32_t x = __shfl_up(incl, off);
            if (lane >= off) incl += x;
        }
        s_pre[lane] = incl - cnt;
        if (lane == 63) s_pre[kGroups] = incl;
    }
    __syncthreads();
    const uint64_t below = (1ull << lane) - 1ull;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
        if ((ball[j] >> lane) & 1ull) {
            const uint32_t q = s_pre[j * 4 + w] + __popcll(ball[j] & below);
            s_col[q] = rc[j];
            s_val[q] = rv[j];
        }
    }
    __syncthreads();
    const int64_t base = (int64_t)tile_off[blockIdx.x];
    const uint32_t total = s_pre[kGroups];
    for (uint32_t i = t; i < total; i += 256) {
        const int64_t pos = base + i;
        if (pos < capacity) {
            const int32_t c = s_col[i];
            col_out[pos] = c;
            val_out[pos] = colw ? (float)((double)s_val[i] * colw[c]) : s_val[i];
        }
    }
    // Rowptr'[i] for the rows whose Rowptr[i] lies in [ts, te) (and, in the
    // last tile, also those equal to nnz).
    const int32_t r0 = s_rows[0], r1 = s_rows[1];
    for (int64_t i = (int64_t)r0 + t; i < r1; i += 256) {
        const int64_t off = (int64_t)rowptr[i] - ts;
        uint32_t c;
        if (off < 0) {  // only for a malformed row pointer
            c = 0;
        } else if (off >= kTile || ts + off >= te) {
            c = total;
        } else {
            const int g = (int)(off >> 6), l = (int)(off & 63);  // g = chunk * 4 + wave
            c = s_pre[g] + __popcll(s_ball[g] & ((1ull << l) - 1ull));
        }
        rowptr_out[i] = (int32_t)(base + c);
    }
}

// ---- single pass: count, decoupled look-back scan and compaction fused ----
// Persistent blocks of 256 threads take kSub consecutive 4096-entry tiles at
// a time in ticket order (an atomic counter), so a ticket's predecessors were
// all taken by blocks that are already running. Per ticket: load col/val
// (16 kSub entries per thread, coalesced; entry o = 256 i + thread, ballot
// group o >> 6), test the mask bits (from LDS when the mask is small enough
// for several blocks per CU, else from global memory, where the n-bit set
// stays in L2), one ballot per 64 entries; publish the ticket's kept count,
// then the first wave looks back over the predecessors' published counts
// (64 at a time) until it meets an inclusive prefix, and publishes this
// ticket's inclusive prefix. The kept entries are then written at their
// global positions straight from registers: the kept entries of one ballot
// are consecutive in the output, so each wave's stores cover one contiguous
// range. Several blocks per CU keep several tickets' loads and look-backs in
// flight at once; three tiles per ticket cut the look-backs and ticket
// atomics to a third.
// Status word of a ticket: bits 63..62 = 1 (count published) or 2 (inclusive
// prefix published), bits 61..0 the value; 0 = nothing yet.
// Every wait is bounded: after kSpinLimit polls without progress the kernel
// records a failure (*nnz_out = -1), takes the missing counts as 0 and
// finishes, so no wave can wait forever.
constexpr int kFusedThreads = 256;
constexpr int kFusedSub = 3;           // 4096-entry tiles per ticket (one look-back for 12,288 entries)
constexpr int kFusedBlocksPerCu = 8;
constexpr int kLdsPerCu = 160 * 1024;
constexpr uint64_t kFlagAgg = 1ull << 62, kFlagIncl = 2ull << 62, kValMask = (1ull << 62) - 1;
constexpr int64_t kSpinLimit = 1ll << 22;
static_assert(kTile == kFusedThreads * kPer, "kPer entries per thread per tile");

// A status word carries its own value, so relaxed device-scope atomics
// suffice (no other data is published through it); acquire loads would also
// invalidate the CU's vector L1 on every poll.
__device__ __forceinline__ uint64_t load_status(const uint64_t *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_status(uint64_t *p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <bool kLdsMask, int kSub>
__global__ __launch_bounds__(kFusedThreads) void slice_fused_kernel(
    const int32_t *__restrict__ rowptr, int32_t n_rows, const int32_t *__restrict__ col,
    const float *__restrict__ val, int64_t nnz, const uint32_t *__restrict__ mask, int32_t n_words, int32_t nt,
    uint64_t *__restrict__ status, int32_t *__restrict__ ticket, int32_t *__restrict__ rowptr_out,
    int32_t *__restrict__ col_out, float *__restrict__ val_out, int64_t capacity, int64_t *__restrict__ nnz_out,
    int32_t *__restrict__ failed, const double *__restrict__ colw) {
    extern __shared__ uint32_t s_mask[];  // n_words words with kLdsMask, else empty
    __shared__ uint64_t s_ball[kGroups * kSub];
    __shared__ uint32_t s_pre[kGroups * kSub + 1];
    __shared__ int32_t s_tile, s_rows[2];
    __shared__ int64_t s_base;
    const int T = threadIdx.x, lane = T & 63, wv = T >> 6;
    if constexpr (kLdsMask) {
        for (int i = T; i < n_words; i += kFusedThreads) s_mask[i] = mask[i];
    }
    for (;;) {
        if (T == 0) s_tile = atomicAdd(ticket, 1);
        __syncthreads();  // s_tile visible; the previous tile's shared state is no longer read
        const int32_t tile = s_tile;
        if (tile >= nt) break;  // block-uniform
        const int64_t ts = (int64_t)tile * kTile * kSub;
        const int64_t te = min<int64_t>(ts + (int64_t)kTile * kSub, nnz);
        const bool last = tile == nt - 1;
        if (T == 0) s_rows[0] = lower_bound_rowptr(rowptr, n_rows, ts);
        if (T == 1) s_rows[1] = last ? n_rows + 1 : lower_bound_rowptr(rowptr, n_rows, te);
        int32_t rc[kPer * kSub];
        float rv[kPer * kSub];
#pragma unroll
        for (int i = 0; i < kPer * kSub; ++i) {
            const int64_t p = ts + T + kFusedThreads * i;
            rc[i] = p < te ? __builtin_nontemporal_load(col + p) : -1;
            rv[i] = p < te ? __builtin_nontemporal_load(val + p) : 0.f;
        }
#pragma unroll
        for (int i = 0; i < kPer * kSub; ++i) {
            const int32_t c = rc[i];
            bool k = false;
            if (c >= 0 && (c >> 5) < n_words) {
                const uint32_t wd = kLdsMask ? s_mask[c >> 5] : mask[c >> 5];
                k = (wd >> (c & 31)) & 1u;
            }
            const uint64_t b = __ballot(k);
            if (lane == 0) s_ball[4 * i + wv] = b;
        }
        __syncthreads();
        if (wv == 0) {
            // exclusive scan of the ballot counts (kSub per lane), then publish and look back
            uint32_t cnt[kSub], own = 0;
#pragma unroll
            for (int u = 0; u < kSub; ++u) {
                cnt[u] = __popcll(s_ball[kSub * lane + u]);
                own += cnt[u];
            }
            uint32_t incl = own;
            for (int off = 1; off < 64; off <<= 1) {
                const uint32_t x = __shfl_up(incl, off);
                if (lane >= off) incl += x;
            }
            uint32_t run = incl - own;
#pragma unroll
            for (int u = 0; u < kSub; ++u) {
                s_pre[kSub * lane + u] = run;
                run += cnt[u];
            }
            const uint32_t total = __shfl(incl, 63);
            if (lane == 63) s_pre[kGroups * kSub] = incl;
            int64_t excl = 0;
            if (tile == 0) {
                if (lane == 0) store_status(status, kFlagIncl | total);
            } else {
                if (lane == 0) store_status(status + tile, kFlagAgg | total);
                int32_t q0 = tile - 1;  // nearest predecessor of the current window
                int64_t polls = 0;
                for (;;) {
                    const int32_t q = q0 - lane;
                    const uint64_t st = q >= 0 ? load_status(status + q) : kFlagIncl;  // before tile 0: prefix 0
                    const uint64_t flag = st >> 62;
                    const uint64_t incl_lanes = __ballot(flag == 2);
                    const uint64_t empty_lanes = __ballot(flag == 0);
                    const int first = incl_lanes ? __ffsll((long long)incl_lanes) - 1 : 64;
                    const uint64_t need = first == 64 ? ~0ull : (2ull << first) - 1ull;  // lanes 0..first
                    if (empty_lanes & need) {
                        if (++polls < kSpinLimit) continue;  // a predecessor has not published yet
                        if (lane == 0) atomicExch(failed, 1);
                    }
                    uint64_t v = (lane <= first && flag != 0) ? (st & kValMask) : 0;
                    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
                    excl += (int64_t)v;
                    if (first < 64 || (empty_lanes & need)) break;
                    q0 -= 64;
                }
                if (lane == 0) store_status(status + tile, kFlagIncl | (uint64_t)(excl + total));
            }
            if (lane == 0) {
                s_base = excl;
                if (last) *nnz_out = atomicAdd(failed, 0) ? -1 : excl + total;
            }
        }
        __syncthreads();
        const int64_t base = s_base;
        const uint64_t below = (1ull << lane) - 1ull;
#pragma unroll
        for (int i = 0; i < kPer * kSub; ++i) {
            const uint64_t b = s_ball[4 * i + wv];
            if ((b >> lane) & 1ull) {
                const int64_t pos = base + s_pre[4 * i + wv] + __popcll(b & below);
                if (pos < capacity) {
                    col_out[pos] = rc[i];
                    val_out[pos] = colw ? (float)((double)rv[i] * colw[rc[i]]) : rv[i];
                }
            }
        }
        const uint32_t total = s_pre[kGroups * kSub];
        const int32_t r0 = s_rows[0], r1 = s_rows[1];
        for (int64_t i = (int64_t)r0 + T; i < r1; i += kFusedThreads) {
            const int64_t off = (int64_t)rowptr[i] - ts;
            uint32_t c;
            if (off >= (int64_t)kTile * kSub || ts + off >= te) {
                c = total;
            } else {
                const int g = (int)(off >> 6), l = (int)(off & 63);
                c = s_pre[g] + __popcll(s_ball[g] & ((1ull << l) - 1ull));
            }
            rowptr_out[i] = (int32_t)(base + c);
        }
    }
}

__global__ __launch_bounds__(256) void zero_words_kernel(uint64_t *__restrict__ p, int64_t count) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = 0;
}

__global__ __launch_bounds__(256) void zero_rows_kernel(int32_t *__restrict__ p, int64_t count,
                                                        int64_t *__restrict__ nnz_out) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = 0;
    if (blockIdx.x == 0 && threadIdx.x == 0) *nnz_out = 0;
}

// Whether the fused kernel keeps the mask in LDS: a copy per block, when at
// least three blocks' copies (plus their small shared state) fit a CU.
bool mask_in_lds(int32_t n_words) {
    return sizeof(uint32_t) * (size_t)n_words + 2048 <= (size_t)kLdsPerCu / 3;
}

// The three launches are the default: with the count's ballots and counts
// published by atomics and the emit's row ranges read from a table, they
// measured faster than the single pass on every workload (slice kernels,
// three launches against single pass: tiny 21 / 26 us, social 344-393 /
// 372-403 us, protein 250 / 281 us, gcn2 72 / 114 us, copurchase 503 /
// 787 us). RSC_SLICE_FUSED = 1 / 0 forces the single-pass / three-launch form.
// RSC_SLICE_PAIRED = 0 makes a two-piece mask walk col twice with one block
// per CU instead of in pairs.
bool paired_count() {
    if (const char *env = getenv("RSC_SLICE_PAIRED")) return atoi(env) != 0;
    return true;
}

bool use_fused() {
    if (const char *env = getenv("RSC_SLICE_FUSED")) return atoi(env) != 0;
    return false;
}

}  // namespace

size_t slice_ws_bytes(int64_t nnz) {
    const size_t nt = (size_t)ceil_div(std::max<int64_t>(nnz, 1), kTile);
    return 2 * align_up(nt * sizeof(uint32_t), 256) + align_up(nt * kGroups * sizeof(uint64_t), 256) +
           align_up((nt + 1) * sizeof(int32_t), 256);
}

hipError_t slice_launch(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr, const int32_t *col,
                        const float *val, const uint32_t *mask, int32_t *rowptr_out,
                        int32_t *col_out, float *val_out, int64_t capacity, int64_t *nnz_out,
                        void *ws, hipStream_t stream, const double *colw) {
    if (nnz == 0) {
        zero_rows_kernel<<<(unsigned)std::min<int64_t>(ceil_div((int64_t)n_rows + 1, 256), 1024), 256, 0,
                           stream>>>(rowptr_out, (int64_t)n_rows + 1, nnz_out);
        return hipGetLastError();
    }
    const int32_t nt = (int32_t)ceil_div(nnz, kTile);
    const size_t tb = align_up((size_t)nt * sizeof(uint32_t), 256);
    uint32_t *tile_cnt = static_cast<uint32_t *>(ws);
    uint32_t *tile_off = reinterpret_cast<uint32_t *>(static_cast<char *>(ws) + tb);
    uint64_t *tile_bits = reinterpret_cast<uint64_t *>(static_cast<char *>(ws) + 2 * tb);
    int32_t *tile_row = reinterpret_cast<int32_t *>(static_cast<char *>(ws) + 2 * tb +
                                                    align_up((size_t)nt * kGroups * sizeof(uint64_t), 256));
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) == hipSuccess)
        (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    const int32_t n_words = (int32_t)ceil_div((int64_t)n_cols, 32);
    if (use_fused()) {
        // ws: [ticket, failure flag | pad to 256 B][status word per tile]
        int32_t *ticket = static_cast<int32_t *>(ws);
        uint64_t *status = reinterpret_cast<uint64_t *>(static_cast<char *>(ws) + 256);
        const int32_t nt2 = (int32_t)ceil_div(nt, kFusedSub);
        const int64_t words = 32 + (int64_t)nt2;  // the 256-byte head and the status words
        zero_words_kernel<<<(unsigned)std::min<int64_t>(ceil_div(words, 256), 1024), 256, 0, stream>>>(
            static_cast<uint64_t *>(ws), words);
        const size_t mask_bytes = sizeof(uint32_t) * (size_t)n_words;
        const bool lds = mask_in_lds(n_words);
        const int per_cu = lds ? (int)std::min<size_t>(kFusedBlocksPerCu, kLdsPerCu / (mask_bytes + 2048))
                               : kFusedBlocksPerCu;
        const unsigned grid = (unsigned)std::max<int64_t>(1, std::min<int64_t>((int64_t)cus * per_cu, nt2));
        if (lds)
            slice_fused_kernel<true, kFusedSub><<<grid, kFusedThreads, mask_bytes, stream>>>(
                rowptr, n_rows, col, val, nnz, mask, n_words, nt2, status, ticket, rowptr_out, col_out, val_out,
                capacity, nnz_out, ticket + 1, colw);
        else
            slice_fused_kernel<false, kFusedSub><<<grid, kFusedThreads, 0, stream>>>(
                rowptr, n_rows, col, val, nnz, mask, n_words, nt2, status, ticket, rowptr_out, col_out, val_out,
                capacity, nnz_out, ticket + 1, colw);
        return hipGetLastError();
    }
    // a mask of two LDS pieces is tested by pairs of blocks (one piece each,
    // the same tiles at the same time), given whole groups of 16 blocks
    const int32_t n_pieces = (int32_t)ceil_div(std::max<int32_t>(n_words, 1), kMaskLdsWords);
    const int64_t pair_grid = std::min<int64_t>(cus, 2 * ceil_div(nt, kTilesPerIterPaired)) / 16 * 16;
    const bool paired = n_pieces == 2 && pair_grid >= 16 && paired_count();
    slice_tile_rows_kernel<<<(unsigned)std::min<int64_t>(ceil_div(std::max<int64_t>((int64_t)n_rows + 1, nt), 256),
                                                         4096),
                             256, 0, stream>>>(rowptr, n_rows, nt, tile_row, tile_cnt, paired ? tile_bits : nullptr);
    if (paired) {
        slice_count_kernel<true, kTilesPerIterPaired><<<(unsigned)pair_grid, kCountThreads, 0, stream>>>(
            col, nnz, mask, n_words, nt, tile_cnt, tile_bits);
    } else {
        const unsigned cgrid =
            (unsigned)std::max<int64_t>(1, std::min<int64_t>(cus, ceil_div(nt, kTilesPerIterSingle)));
        slice_count_kernel<false, kTilesPerIterSingle><<<cgrid, kCountThreads, 0, stream>>>(
            col, nnz, mask, n_words, nt, tile_cnt, tile_bits);
    }
    slice_scan_kernel<<<1, 1024, 0, stream>>>(nt, tile_cnt, tile_off, nnz_out);
    slice_emit_kernel<<<nt, 256, 0, stream>>>(rowptr, n_rows, col, val, nnz, tile_bits, tile_off, tile_row,
                                              rowptr_out, col_out, val_out, capacity, colw);
    return hipGetLastError();
}

}  // namespace rsc
