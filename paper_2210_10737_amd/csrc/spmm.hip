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
//   * 8 gather instructions (4 in the layouts that take 8 or 16 entries per
//     instruction) are issued before their FMAs for memory-level parallelism;
//   * products are accumulated in fp32 over each run of <= 64 entries and the
//     run sum is folded into an fp64 accumulator; one fp32 rounding per output;
//   * rows with more than kLongRow entries are taken by persistent 8-wave
//     blocks: the waves take interleaved runs of 64 entries and their fp64
//     sums are combined in LDS in fixed wave order. No float atomics, so the
//     result is bitwise reproducible;
//   * features up to 128 wide take a layout of 16..128 floats (several
//     entries per load instruction), and B may be processed in several such
//     feature slices when the slice of the referenced B rows gets close to
//     cache size;
//   * on graphs with long rows on average, rows are taken longest length
//     class first (a scheduling order only);
//   * when the referenced B rows span a few L2-sized ranges, the columns are
//     cut into those ranges and processed one range at a time, with fp32
//     partial rows combined in fixed range order (column-blocked mode);
//   * bit 31 of a column index (set only in a plan's own copy of col) marks
//     hub columns; when the gathered rows far outgrow the caches, the other
//     columns' rows are loaded non-temporally so the hubs' stay in L2;
//   * the per-call preparation (long-row list or row order, split bounds)
//     can be done once by a plan or at a cache refresh and reused.
#include <cstdlib>

#include "rsc_internal.h"

namespace rsc {

// Rows with more than kLongRow entries are processed by a whole 8-wave
// block (waves take interleaved runs of 64 entries, then a fixed-order LDS
// reduction); shorter rows by one wave. Long rows are handed out to
// persistent blocks through an atomic counter.
constexpr int kLongRow = 1024;
constexpr int kSpmmRowWaves = 4;      // rows (waves) per block of the row kernel
constexpr int kSpmmLongWaves = 8;     // waves per block of the long-row kernel
constexpr int kSpmmLongBlocks = 1024;  // persistent blocks that walk the long-row list

namespace {

constexpr int kUnroll = 8;
typedef float vf4 __attribute__((ext_vector_type(4)));
constexpr int32_t kColMask = 0x7FFFFFFF;  // bit 31 of a column index: cache hint

__device__ __forceinline__ float4 load_nt(const float4 *p) {
    const vf4 x = __builtin_nontemporal_load(reinterpret_cast<const vf4 *>(p));
    return make_float4(x.x, x.y, x.z, x.w);
}

__global__ void zero_counters_kernel(int32_t *p) { p[0] = 0; p[1] = 0; }
__global__ void zero_next_kernel(int32_t *p) { *p = 0; }

// Appends every row longer than kLongRow to `list`; row r spans
// [ptr[r], ptr[r + end_off]) (end_off = 1 for a CSR row pointer). Each thread checks
// kCollectPerThread rows (coalesced reads); a block-wide scan gives each long
// row its place, and one atomic per block reserves the block's range, so the
// list costs a few hundred atomics rather than one per row. The list order
// only decides which block takes which row.
constexpr int kCollectThreads = 1024;
constexpr int kCollectPerThread = 4;

__global__ __launch_bounds__(kCollectThreads) void collect_long_rows_kernel(
    const int32_t *__restrict__ ptr, int64_t end_off, int32_t n_rows, int32_t *count, int32_t *list) {
    __shared__ int32_t s_wave[kCollectThreads / 64];
    __shared__ int32_t s_base;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int64_t base = (int64_t)blockIdx.x * kCollectThreads * kCollectPerThread;
    bool is_long[kCollectPerThread];
    int32_t mine = 0;
#pragma unroll
    for (int i = 0; i < kCollectPerThread; ++i) {
        const int64_t r = base + t + (int64_t)kCollectThreads * i;
        is_long[i] = r < n_rows && ptr[r + end_off] - ptr[r] > kLongRow;
        mine += is_long[i];
    }
    // exclusive scan of `mine` over the block: within the wave, then across waves
    int32_t incl = mine;
    for (int off = 1; off < 64; off <<= 1) {
        const int32_t x = __shfl_up(incl, off);
        if (lane >= off) incl += x;
    }
    if (lane == 63) s_wave[wave] = incl;
    __syncthreads();
    int32_t before = incl - mine, total = 0;
    for (int w = 0; w < kCollectThreads / 64; ++w) {
        before += w < wave ? s_wave[w] : 0;
        total += s_wave[w];
    }
    if (total == 0) return;  // block-uniform
    if (t == 0) s_base = atomicAdd(count, total);
    __syncthreads();
    int32_t pos = s_base + before;
#pragma unroll
    for (int i = 0; i < kCollectPerThread; ++i)
        if (is_long[i]) list[pos++] = (int32_t)(base + t + (int64_t)kCollectThreads * i);
}

// Lane layout: LPE lanes per gathered entry, G = 64 / LPE entries per load
// instruction. Lane L belongs to entry-group g = L / LPE and owns features
// 4 * (L % LPE) .. +3 of the current feature slice (plus +256 for NV = 2,
// which is only used with LPE = 64).
template <int LPE>
struct Layout {
    static constexpr int G = kWave / LPE;
    static_assert(kWave % LPE == 0, "LPE must divide the wave");
};

// Accumulates runs of 64 entries starting at beg, beg + stride, ... (< end)
// into acc. `act[q]` says whether this lane's q-th float4 lies inside d.
// Within a run, entry-group g takes entries g, g + G, g + 2G, ...; the group
// partials are combined by a butterfly over the groups (fixed order, every
// lane ends with the same sum) before the run is folded into fp64.
// Bit 31 of a column index is a cache hint (set by a plan or a cache on
// their own copies; a caller's indices are < 2^31): with kHint, gathers of
// columns without it bypass cache allocation (non-temporal), so the rows of
// the columns that carry half the entries stay in L2. Values are unchanged.
template <int LPE, int NV, bool kHint>
__device__ __forceinline__ void accumulate_runs(const int32_t *__restrict__ col,
                                                const float *__restrict__ val,
                                                const float *__restrict__ B, int64_t ldb,
                                                int64_t beg, int64_t end, int32_t stride,
                                                const bool (&act)[NV], int lane,
                                                double (&acc)[NV][4]) {
    constexpr int G = Layout<LPE>::G;
    const int g = lane / LPE, sl = lane % LPE;
    for (int64_t base = beg; base < end; base += stride) {  // int64: base + stride may pass 2^31 - 1
        const int32_t cnt = __builtin_amdgcn_readfirstlane((int32_t)min<int64_t>(kWave, end - base));
        int32_t my_c = 0;
        float my_v = 0.f;
        if (lane < cnt) {
            my_c = __builtin_nontemporal_load(col + base + lane);
            my_v = __builtin_nontemporal_load(val + base + lane);
        }
        float a[NV][4];
#pragma unroll
        for (int q = 0; q < NV; ++q) a[q][0] = a[q][1] = a[q][2] = a[q][3] = 0.f;

        if constexpr (G == 1) {
            // one entry per instruction: broadcast (col, val) into SGPRs
            for (int32_t t = 0; t < cnt; t += kUnroll) {
                float4 b[kUnroll][NV];
                float v[kUnroll];
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) {
#pragma unroll
                    for (int q = 0; q < NV; ++q) b[u][q] = make_float4(0.f, 0.f, 0.f, 0.f);
                    v[u] = 0.f;
                    if (t + u < cnt) {  // wave-uniform
                        const int32_t cf = __builtin_amdgcn_readlane(my_c, t + u);
                        const int32_t c = cf & kColMask;
                        v[u] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(my_v), t + u));
                        const float4 *brow = reinterpret_cast<const float4 *>(B + (int64_t)c * ldb) + lane;
                        if (kHint && cf >= 0) {  // not a hub column: stream it past the caches
#pragma unroll
                            for (int q = 0; q < NV; ++q)
                                if (act[q]) b[u][q] = load_nt(brow + q * kWave);
                        } else {
#pragma unroll
                            for (int q = 0; q < NV; ++q)
                                if (act[q]) b[u][q] = brow[q * kWave];
                        }
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
        } else {
            static_assert(NV == 1, "sliced layouts hold one float4 per lane");
            constexpr int kSteps = kWave / G;  // steps that cover the 64-entry run
            constexpr int kWin = G >= 8 ? 4 : kUnroll;  // steps per window (gathers in flight)
            // one window of kUnroll steps at a time: unrolling the step loop
            // too keeps every window's (col, val) live at once (130 VGPRs for
            // G = 2) and costs occupancy
#pragma unroll 1
            for (int t0 = 0; t0 < kSteps; t0 += kWin) {
                if (t0 * G >= cnt) break;  // wave-uniform
                float4 b[kWin];
                float v[kWin];
#pragma unroll
                for (int u = 0; u < kWin; ++u) {
                    const int j = (t0 + u) * G + g;  // entry of this group within the run
                    const int32_t cf = __shfl(my_c, j & (kWave - 1));
                    const int32_t c = cf & kColMask;
                    const float vv = __shfl(my_v, j & (kWave - 1));
                    b[u] = make_float4(0.f, 0.f, 0.f, 0.f);
                    v[u] = 0.f;
                    if (t0 + u < kSteps && j < cnt && act[0]) {
                        const float4 *brow = reinterpret_cast<const float4 *>(B + (int64_t)c * ldb) + sl;
                        b[u] = (kHint && cf >= 0) ? load_nt(brow) : *brow;
                        v[u] = vv;
                    }
                }
#pragma unroll
                for (int u = 0; u < kWin; ++u) {
                    a[0][0] = fmaf(v[u], b[u].x, a[0][0]);
                    a[0][1] = fmaf(v[u], b[u].y, a[0][1]);
                    a[0][2] = fmaf(v[u], b[u].z, a[0][2]);
                    a[0][3] = fmaf(v[u], b[u].w, a[0][3]);
                }
            }
#pragma unroll
            for (int m = LPE; m < kWave; m <<= 1)
#pragma unroll
                for (int x = 0; x < 4; ++x) a[0][x] += __shfl_xor(a[0][x], m);
        }
#pragma unroll
        for (int q = 0; q < NV; ++q)
#pragma unroll
            for (int x = 0; x < 4; ++x) acc[q][x] += (double)a[q][x];
    }
}

template <int LPE, int NV>
__device__ __forceinline__ void store_row(float *__restrict__ yrow, int32_t d, int lane,
                                          const double (&acc)[NV][4]) {
    if (lane >= LPE) return;  // every entry-group holds the same sums; group 0 stores
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

// Long rows: persistent blocks of kSpmmLongWaves waves take rows from the list
// through an atomic counter; within a row the waves take interleaved runs of
// 64 entries and their fp64 sums are added in LDS in fixed wave order.
// Row r spans [ptr[r], ptr[r + off]) and is written to row r of Y.
// B and Y point at the first feature of the current slice; d is its width.
template <int LPE, int NV, bool kHint>
__global__ __launch_bounds__(kSpmmLongWaves * 64) void spmm_long_kernel(
    const int32_t *__restrict__ ptr, int64_t off, const int32_t *__restrict__ col, const float *__restrict__ val,
    const float *__restrict__ B, int64_t ldb, float *__restrict__ Y, int64_t ldy, int32_t d,
    const int32_t *__restrict__ long_count, int32_t *__restrict__ long_next,
    const int32_t *__restrict__ long_rows) {
    __shared__ double red[kSpmmLongWaves][NV * 4][kWave];
    __shared__ int32_t s_job;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int sl = lane % LPE;
    bool act[NV];
#pragma unroll
    for (int q = 0; q < NV; ++q) act[q] = 4 * sl + 4 * kWave * q < d;
    const int32_t nl = __builtin_amdgcn_readfirstlane(*long_count);
    for (;;) {
        if (threadIdx.x == 0) s_job = atomicAdd(long_next, 1);
        __syncthreads();
        const int32_t j = __builtin_amdgcn_readfirstlane(s_job);
        if (j >= nl) break;  // block-uniform: every wave read the same s_job
        const int32_t r = __builtin_amdgcn_readfirstlane(long_rows[j]);
        const int32_t s = __builtin_amdgcn_readfirstlane(ptr[r]);
        const int32_t e = __builtin_amdgcn_readfirstlane(ptr[r + off]);
        double acc[NV][4];
#pragma unroll
        for (int q = 0; q < NV; ++q) acc[q][0] = acc[q][1] = acc[q][2] = acc[q][3] = 0.0;
        accumulate_runs<LPE, NV, kHint>(col, val, B, ldb, (int64_t)s + kWave * wave, e, kWave * kSpmmLongWaves, act,
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
                    for (int w = 1; w < kSpmmLongWaves; ++w) t += red[w][q * 4 + x][lane];
                    acc[q][x] = t;
                }
            store_row<LPE, NV>(Y + (int64_t)r * ldy, d, lane, acc);
        }
        __syncthreads();  // red and s_job are reused by the next row
    }
}

// Short rows: one wave per row, kSpmmRowWaves rows per block; rows longer
// than kLongRow are left to spmm_long_kernel when skip_long. With `order`,
// the rows are taken in that order after its first *long_count entries (the
// long rows): a processing order only, each row's sum is unchanged. Row r
// spans [ptr[r], ptr[r + off]); kCsr says off == 1 (a CSR row pointer, both
// bounds then come from one 8-byte scalar load).
template <int LPE, int NV, bool kCsr, bool kHint>
__global__ __launch_bounds__(kSpmmRowWaves * 64) void spmm_rows_kernel(
    const int32_t *__restrict__ ptr, int64_t off, const int32_t *__restrict__ col, const float *__restrict__ val,
    const float *__restrict__ B, int64_t ldb, float *__restrict__ Y, int64_t ldy, int32_t n_rows,
    int32_t d, int32_t skip_long, const int32_t *__restrict__ order, const int32_t *__restrict__ long_count) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int sl = lane % LPE;
    bool act[NV];
#pragma unroll
    for (int q = 0; q < NV; ++q) act[q] = 4 * sl + 4 * kWave * q < d;
    int32_t r = blockIdx.x * kSpmmRowWaves + wave;
    if (order) {
        const int64_t i = (int64_t)__builtin_amdgcn_readfirstlane(*long_count) + r;
        if (i >= n_rows) return;
        r = __builtin_amdgcn_readfirstlane(order[i]);
    } else if (r >= n_rows) {
        return;
    }
    const int32_t s = __builtin_amdgcn_readfirstlane(ptr[r]);
    const int32_t e = __builtin_amdgcn_readfirstlane(kCsr ? ptr[r + 1] : ptr[(int64_t)r + off]);
    if (skip_long && e - s > kLongRow) return;
    double acc[NV][4];
#pragma unroll
    for (int q = 0; q < NV; ++q) acc[q][0] = acc[q][1] = acc[q][2] = acc[q][3] = 0.0;
    accumulate_runs<LPE, NV, kHint>(col, val, B, ldb, s, e, kWave, act, lane, acc);
    store_row<LPE, NV>(Y + (int64_t)r * ldy, d, lane, acc);
}

constexpr int kClasses = 32;

struct SpmmWs {
    int32_t long_count;  // rows in the long-row list
    int32_t long_next;   // next long row to hand out (one counter per feature pass)
    int32_t pad[30];
    int32_t cls_count[kClasses];   // rows per length class (ordered mode)
    int32_t cls_cursor[kClasses];  // next free slot of each class in the order
    int32_t pad2[32];
};

inline int64_t long_rows_bound(int32_t n_rows, int64_t nnz) {
    return std::min<int64_t>(n_rows, nnz / (kLongRow + 1));
}

// Pieces longer than kLongRow in the column-blocked mode with P ranges: up to
// P per row, and no more than nnz / (kLongRow + 1) in all.
inline int64_t long_pieces_bound(int32_t n_rows, int64_t nnz, int32_t P) {
    return std::min<int64_t>((int64_t)P * n_rows, nnz / (kLongRow + 1));
}

// Length class of a row: 0 for at most one entry, else ceil(log2(len)), so
// rows longer than kLongRow = 1024 are exactly the classes >= 11.
__device__ __forceinline__ int row_class(int32_t len) { return len <= 1 ? 0 : 32 - __clz(len - 1); }
constexpr int kLongClass = 11;
static_assert(kLongRow == 1024, "class boundary of the long rows");

__global__ __launch_bounds__(128) void zero_header_kernel(SpmmWs *h) {
    reinterpret_cast<int32_t *>(h)[threadIdx.x] = 0;
}

// Rows per length class: an LDS histogram per block, one atomic per class.
__global__ __launch_bounds__(kCollectThreads) void class_hist_kernel(const int32_t *__restrict__ rowptr,
                                                                    int32_t n_rows, SpmmWs *h) {
    __shared__ int32_t hist[kClasses];
    if (threadIdx.x < kClasses) hist[threadIdx.x] = 0;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * kCollectThreads * kCollectPerThread;
#pragma unroll
    for (int i = 0; i < kCollectPerThread; ++i) {
        const int64_t r = base + threadIdx.x + (int64_t)kCollectThreads * i;
        if (r < n_rows) atomicAdd(&hist[row_class(rowptr[r + 1] - rowptr[r])], 1);
    }
    __syncthreads();
    if (threadIdx.x < kClasses && hist[threadIdx.x]) atomicAdd(&h->cls_count[threadIdx.x], hist[threadIdx.x]);
}

// Class start offsets with the longest class first; the long rows (classes
// >= kLongClass) come out as the first long_count entries of the order.
__global__ __launch_bounds__(64) void class_scan_kernel(SpmmWs *h) {
    const int c = threadIdx.x;
    if (c >= kClasses) return;
    int32_t start = 0, lng = 0;
    for (int k = c + 1; k < kClasses; ++k) start += h->cls_count[k];
    for (int k = kLongClass; k < kClasses; ++k) lng += h->cls_count[k];
    h->cls_cursor[c] = start;
    if (c == 0) {
        h->long_count = lng;
        h->long_next = 0;
    }
}

// Places every row in its class's range (the order within a class follows
// the atomics and does not matter: it only decides which wave takes a row).
__global__ __launch_bounds__(kCollectThreads) void class_scatter_kernel(const int32_t *__restrict__ rowptr,
                                                                       int32_t n_rows, SpmmWs *h,
                                                                       int32_t *__restrict__ order) {
    __shared__ int32_t hist[kClasses];
    __shared__ int32_t slot[kClasses];
    if (threadIdx.x < kClasses) hist[threadIdx.x] = 0;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * kCollectThreads * kCollectPerThread;
    int cls[kCollectPerThread];
#pragma unroll
    for (int i = 0; i < kCollectPerThread; ++i) {
        const int64_t r = base + threadIdx.x + (int64_t)kCollectThreads * i;
        cls[i] = r < n_rows ? row_class(rowptr[r + 1] - rowptr[r]) : -1;
        if (cls[i] >= 0) atomicAdd(&hist[cls[i]], 1);
    }
    __syncthreads();
    if (threadIdx.x < kClasses)
        slot[threadIdx.x] = hist[threadIdx.x] ? atomicAdd(&h->cls_cursor[threadIdx.x], hist[threadIdx.x]) : 0;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kCollectPerThread; ++i)
        if (cls[i] >= 0)
            order[atomicAdd(&slot[cls[i]], 1)] = (int32_t)(base + threadIdx.x + (int64_t)kCollectThreads * i);
}

// Rows are taken longest class first when rows are long on average: the
// heavy rows then start first and the kernels end on short rows. Results do
// not depend on it. RSC_SPMM_ORDER=0/1 overrides.
// Gathered rows beyond this many bytes per feature pass take the column
// cache hint (twice the 256 MB MALL).
constexpr double kHintBytes = 512.0 * 1024 * 1024;

inline bool use_hint() {
    if (const char *env = getenv("RSC_SPMM_HINT")) return atoi(env) != 0;
    return true;
}

inline bool use_order(int32_t n_rows, int64_t nnz) {
    if (const char *env = getenv("RSC_SPMM_ORDER")) return atoi(env) != 0;
    return n_rows > 0 && nnz >= 128LL * n_rows;
}

// ---- column-blocked mode ------------------------------------------------
// When the columns of B fit L2 in a few pieces, the product is taken one
// piece at a time: the columns are cut into P equal ranges, and "virtual row"
// (b, r) = the entries of row r whose column lies in range b (contiguous in
// the row, since columns are sorted). The virtual rows are processed
// block-major, so at any moment the whole GPU gathers from one range of B
// rows (a few MB, resident in each XCD's L2) instead of from all of them.
// Each virtual row writes a partial row; a combine pass adds the P partials
// of row r in fixed order b = 0..P-1 in fp64 and rounds once.
constexpr int kBlockW = 64;                         // features per blocked pass, the widest layout
constexpr double kBlockBytes = 4.5 * 1024 * 1024;   // B bytes per column range (~ one XCD's L2)
constexpr int kMaxBlocks = 8;                       // partial outputs at most 8 x Y per pass
constexpr int kPieceMin = 56;                       // mean entries per piece of a row for blocking

// Features per blocked pass for feature width d: the narrowest of the 16-,
// 32- and 64-float layouts that holds d (wider d in several 64-float
// passes), so no lane of a narrow product idles.
inline int32_t blocked_width(int32_t d) { return d <= 16 ? 16 : d <= 32 ? 32 : kBlockW; }

// Number of column ranges P for a product with n_rows rows, about nnz
// entries, n_src distinct B rows referenced and d features; 1 = not blocked.
// Blocked when the referenced slice of B one pass gathers from (the
// blocked_width(d) floats of each row) spans 2..16 L2-sized ranges and rows
// are long enough that each piece still fills about 14 load instructions on
// average: kPieceMin entries in the 64-float layout (4 entries per
// instruction), twice and four times that in the 32- and 16-float layouts
// (8 and 16 per instruction; shorter pieces made a power-law graph with
// 489 entries per row slower at d = 16 and 32, while a uniform one with
// 600 per row gained 16-33 %). Beyond 8 ranges P stays 8: ranges of up to
// two L2 sizes still keep most gathers on chip (on a 233K-node graph with
// 489 entries per row, 8 ranges of 7.5 MB measured 5 % faster than
// unblocked passes at d = 256, while 32-float passes over ranges that do
// fit L2 were slower: twice the passes over the row structure).
// RSC_SPMM_BLOCKED=0 switches the mode off, =2..8 forces that P.
inline int32_t column_blocks(int32_t n_rows, int64_t nnz, int64_t n_src, int32_t d) {
    if (n_rows <= 0 || (int64_t)(kMaxBlocks + 1) * n_rows > INT32_MAX) return 1;  // virtual rows are int32
    if (const char *env = getenv("RSC_SPMM_BLOCKED")) {
        const int v = atoi(env);
        if (v == 0) return 1;
        if (v >= 2 && v <= kMaxBlocks) return v;
    }
    const int32_t W = blocked_width(d);
    int64_t P = (int64_t)std::ceil((double)n_src * W * 4 / kBlockBytes);
    if (P < 2 || P > 2 * kMaxBlocks) return 1;
    P = std::min<int64_t>(P, kMaxBlocks);
    if (nnz < (int64_t)kPieceMin * (kBlockW / W) * P * n_rows) return 1;
    return (int32_t)P;
}

// S[b * n_rows + r] = first entry of row r with column >= b * n_cols / P
// (b = 0: rowptr[r]; b = P: rowptr[r + 1]); binary search in the sorted row.
// Piece b of row r ("virtual row" v = b * n_rows + r) is then
// [S[v], S[v + n_rows]): the row kernels take S with offset n_rows as their
// row pointer, and consecutive virtual rows run through one column range.
__global__ __launch_bounds__(256) void split_rows_kernel(const int32_t *__restrict__ rowptr,
                                                         const int32_t *__restrict__ col, int32_t n_rows,
                                                         int32_t n_cols, int32_t P, int32_t *__restrict__ S) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (int64_t)n_rows * (P + 1)) return;
    const int32_t b = (int32_t)(t / n_rows);
    const int64_t r = t - (int64_t)b * n_rows;
    const int32_t s = rowptr[r], e = rowptr[r + 1];
    int32_t pos;
    if (b == 0) {
        pos = s;
    } else if (b == P) {
        pos = e;
    } else {
        const int64_t bound = (int64_t)b * n_cols / P;
        int32_t lo = s, hi = e;
        while (lo < hi) {
            const int32_t mid = lo + (hi - lo) / 2;
            if ((col[mid] & kColMask) < bound) lo = mid + 1; else hi = mid;
        }
        pos = lo;
    }
    S[t] = pos;
}

// Y[r][f] = fl32(sum over b = 0..P-1 of part[b * n_rows + r][f]) in fp64;
// one thread per 4 features of a row.
__global__ __launch_bounds__(256) void combine_blocks_kernel(const float *__restrict__ part, int64_t ldp,
                                                             int32_t n_rows, int32_t P, int32_t d,
                                                             float *__restrict__ Y, int64_t ldy) {
    const int32_t q = (d + 3) / 4;
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (int64_t)n_rows * q) return;
    const int64_t r = t / q;
    const int32_t f = 4 * (int32_t)(t - r * q);
    const int32_t m = min(4, d - f);
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
    for (int32_t b = 0; b < P; ++b) {
        const float *p = part + ((int64_t)b * n_rows + r) * ldp + f;
        if (m == 4) {
            const vf4 x = __builtin_nontemporal_load(reinterpret_cast<const vf4 *>(p));
            acc[0] += (double)x.x;
            acc[1] += (double)x.y;
            acc[2] += (double)x.z;
            acc[3] += (double)x.w;
        } else {
            for (int i = 0; i < m; ++i) acc[i] += (double)p[i];
        }
    }
    float *y = Y + r * ldy + f;
    if (m == 4) {
        const vf4 o = {(float)acc[0], (float)acc[1], (float)acc[2], (float)acc[3]};
        __builtin_nontemporal_store(o, reinterpret_cast<vf4 *>(y));
    } else {
        for (int i = 0; i < m; ++i) y[i] = (float)acc[i];
    }
}

}  // namespace

namespace {
// entries of the row list: the whole processing order (n_rows), or the long
// rows, or the long pieces of a column-blocked product with up to kMaxBlocks
// ranges (one layout for every P, so a workspace never depends on the range
// count an environment switch picks)
int64_t list_entries(int32_t n_rows, int64_t nnz) {
    return std::max<int64_t>({1, (int64_t)n_rows, long_pieces_bound(n_rows, nnz, kMaxBlocks)});
}
size_t list_bytes(int32_t n_rows, int64_t nnz) {
    return align_up(sizeof(int32_t) * (size_t)list_entries(n_rows, nnz), 256);
}
// bytes of the blocked mode's split points and partial rows for P ranges
size_t blocked_bytes(int32_t n_rows, int32_t P) {
    if (P <= 1) return 0;
    return align_up(sizeof(int32_t) * (size_t)n_rows * (P + 1), 256) +
           align_up(sizeof(float) * (size_t)P * n_rows * kBlockW, 256);
}
}  // namespace

int32_t spmm_column_blocks(int32_t n_rows, int64_t nnz, int64_t n_src, int32_t d) {
    return column_blocks(n_rows, nnz, n_src, d);
}

hipError_t spmm_split_launch(int32_t n_rows, int32_t n_cols, const int32_t *rowptr, const int32_t *col, int32_t P,
                             int32_t *S, hipStream_t stream) {
    const int64_t ns = (int64_t)n_rows * (P + 1);
    if (ns > 0) split_rows_kernel<<<(unsigned)ceil_div(ns, 256), 256, 0, stream>>>(rowptr, col, n_rows, n_cols, P, S);
    return hipGetLastError();
}

size_t spmm_ws_bytes(int32_t n_rows, int64_t nnz, int32_t n_cols) {
    // header, the row list, then the blocked mode's buffers when the full
    // product would be blocked (a slice of it never needs more ranges)
    size_t blocked = 0;
    for (const int32_t d : {16, 32, kBlockW})  // the three blocked layouts' range counts
        blocked = std::max(blocked, blocked_bytes(n_rows, column_blocks(n_rows, nnz, n_cols, d)));
    return sizeof(SpmmWs) + list_bytes(n_rows, nnz) + blocked;
}

int32_t spmm_slice_width(int32_t n_rows, int64_t nnz, int64_t n_src, int32_t d) {
    // Feature-slice width (floats) of one pass. Slices of 16/32/64/128 use
    // 4/8/16/32 lanes per gathered entry; 256 (512 for d > 256) is one pass.
    // Features up to 128 wide take the narrowest layout that holds them in one
    // pass (several entries per load instruction instead of idle lanes).
    // Gathers are limited by the rate of L2-miss requests, so several narrower
    // passes pay off when the slice of the referenced B rows comes close to L2
    // size and rows are long enough to amortise the extra passes over
    // rowptr/col/val; only for widths of whole 128-byte lines (d % 32 == 0),
    // since a slice that straddles lines doubles the requests.
    if (const char *env = getenv("RSC_SPMM_SLICE")) {
        const int v = atoi(env);
        if (v == 16 || v == 32 || v == 64 || v == 128) return v;
        if (v == 256 || v == 512) return d > 256 ? 512 : 256;
    }
    const int32_t fit = d <= 16 ? 16 : d <= 32 ? 32 : d <= 64 ? 64 : d <= 128 ? 128 : d <= 256 ? 256 : 512;
    if (d <= 32 || d % 32 != 0 || n_rows <= 0 || nnz < 128LL * n_rows) return fit;
    const double mib = 1024.0 * 1024.0;
    const double ws32 = (double)n_src * 32 * 4 / mib, ws64 = 2 * ws32;
    if (ws32 > 64.0) return fit;
    if (ws64 <= 30.0 && ws32 > 8.0) return std::min(64, fit);
    return 32;
}

bool spmm_use_order(int32_t n_rows, int64_t nnz) { return use_order(n_rows, nnz); }

bool spmm_hint_taken(int64_t n_src, int32_t d, int32_t slice) {
    return use_hint() && (double)n_src * std::min(d, slice) * sizeof(float) > kHintBytes;
}

hipError_t spmm_rows_prepare(int32_t n_rows, int64_t nnz_bound, const int32_t *rowptr, void *ws,
                             hipStream_t stream) {
    if (n_rows == 0) return hipSuccess;
    SpmmWs *h = static_cast<SpmmWs *>(ws);
    int32_t *list = reinterpret_cast<int32_t *>(h + 1);
    const int64_t lbound = long_rows_bound(n_rows, nnz_bound);
    const unsigned cgrid = (unsigned)ceil_div(n_rows, kCollectThreads * kCollectPerThread);
    if (use_order(n_rows, nnz_bound)) {
        zero_header_kernel<<<1, 128, 0, stream>>>(h);
        class_hist_kernel<<<cgrid, kCollectThreads, 0, stream>>>(rowptr, n_rows, h);
        class_scan_kernel<<<1, 64, 0, stream>>>(h);
        class_scatter_kernel<<<cgrid, kCollectThreads, 0, stream>>>(rowptr, n_rows, h, list);
    } else if (lbound > 0) {
        zero_counters_kernel<<<1, 1, 0, stream>>>(&h->long_count);
        collect_long_rows_kernel<<<cgrid, kCollectThreads, 0, stream>>>(rowptr, 1, n_rows, &h->long_count, list);
    }
    return hipGetLastError();
}

hipError_t spmm_blocked_prepare(int32_t n_rows, int64_t nnz_bound, const int32_t *S, int32_t P, void *ws,
                                hipStream_t stream) {
    SpmmWs *h = static_cast<SpmmWs *>(ws);
    int32_t *list = reinterpret_cast<int32_t *>(h + 1);
    const int32_t nv = P * n_rows;
    if (P > kMaxBlocks || long_pieces_bound(n_rows, nnz_bound, P) > list_entries(n_rows, nnz_bound))
        return hipErrorInvalidValue;
    zero_counters_kernel<<<1, 1, 0, stream>>>(&h->long_count);
    if (long_rows_bound(n_rows, nnz_bound) > 0 && nv > 0)
        collect_long_rows_kernel<<<(unsigned)ceil_div(nv, kCollectThreads * kCollectPerThread), kCollectThreads, 0,
                                   stream>>>(S, n_rows, nv, &h->long_count, list);
    return hipGetLastError();
}

size_t spmm_core_ws_bytes(int32_t n_rows, int64_t nnz_bound) { return sizeof(SpmmWs) + list_bytes(n_rows, nnz_bound); }

size_t spmm_blocked_fits(int32_t n_rows, int64_t nnz_bound, int32_t P) {
    return sizeof(SpmmWs) + list_bytes(n_rows, nnz_bound) + blocked_bytes(n_rows, P);
}

const int32_t *spmm_long_count_of(const void *ws) { return &static_cast<const SpmmWs *>(ws)->long_count; }

hipError_t spmm_launch(int32_t n_rows, int32_t n_cols, int64_t nnz_bound, const int32_t *rowptr,
                       const int32_t *col, const float *val, const float *B, int32_t d, int64_t ldb, float *Y,
                       int64_t ldy, void *ws, size_t ws_bytes, hipStream_t stream, int64_t nnz_hint,
                       int64_t n_src_hint, bool hint_cols, const SpmmPrepared *prep, bool *used_prep) {
    if (used_prep) *used_prep = false;
    if (n_rows == 0) return hipSuccess;
    SpmmWs *h = static_cast<SpmmWs *>(ws);
    int32_t *list = reinterpret_cast<int32_t *>(h + 1);  // long-row list, or the whole processing order
    // The blocked mode is chosen from the expected entries and referenced B
    // rows (the same for the exact product and a full-budget slice of it);
    // it runs only when the workspace holds its buffers.
    const int32_t P = column_blocks(n_rows, nnz_hint, n_src_hint, d);
    const size_t head = sizeof(SpmmWs) + list_bytes(n_rows, nnz_bound);
    if (P > 1 && head + blocked_bytes(n_rows, P) <= ws_bytes) {
        // the long-piece list must hold every piece the collect pass can find
        if (P > kMaxBlocks || long_pieces_bound(n_rows, nnz_bound, P) > list_entries(n_rows, nnz_bound))
            return hipErrorInvalidValue;
        char *p = static_cast<char *>(ws) + head;
        float *part = reinterpret_cast<float *>(p + align_up(sizeof(int32_t) * (size_t)n_rows * (P + 1), 256));
        const int32_t nv = P * n_rows;  // virtual rows, block-major
        // split bounds and the long-piece list: a plan's, prepared once (the
        // list then already sits in this workspace), or this call's
        const bool pre = prep && prep->ready && prep->P == P && prep->split;
        if (used_prep) *used_prep = pre;
        const int32_t *S = pre ? prep->split : reinterpret_cast<const int32_t *>(p);
        int32_t n_long;
        if (pre) {
            n_long = (int32_t)std::min<int64_t>(
                prep->long_rows >= 0 ? prep->long_rows : long_rows_bound(n_rows, nnz_bound), kSpmmLongBlocks);
        } else {
            const hipError_t e = spmm_split_launch(n_rows, n_cols, rowptr, col, P, reinterpret_cast<int32_t *>(p),
                                                   stream);
            if (e != hipSuccess) return e;
            // long pieces (a piece of a row longer than kLongRow) go to the
            // persistent 8-wave blocks as in the unblocked mode
            n_long = (int32_t)std::min<int64_t>(long_rows_bound(n_rows, nnz_bound), kSpmmLongBlocks);
            if (n_long > 0) {
                zero_counters_kernel<<<1, 1, 0, stream>>>(&h->long_count);
                collect_long_rows_kernel<<<(unsigned)ceil_div(nv, kCollectThreads * kCollectPerThread),
                                           kCollectThreads, 0, stream>>>(S, n_rows, nv, &h->long_count, list);
            }
        }
        const unsigned vgrid = (unsigned)ceil_div(nv, kSpmmRowWaves);
        // partial rows are W floats apart (the workspace holds kBlockW)
        const int32_t W = blocked_width(d);
        for (int32_t f0 = 0; f0 < d; f0 += W) {
            const int32_t dl = std::min<int32_t>(d - f0, W);
#define RSC_SPMM_BLOCKED_LAUNCH(LPE_)                                                                         \
    do {                                                                                                      \
        if (n_long > 0) {                                                                                     \
            if (f0 > 0 || pre) zero_next_kernel<<<1, 1, 0, stream>>>(&h->long_next);                          \
            spmm_long_kernel<LPE_, 1, false><<<n_long, kSpmmLongWaves * 64, 0, stream>>>(                     \
                S, n_rows, col, val, B + f0, ldb, part, W, dl, &h->long_count, &h->long_next, list);          \
        }                                                                                                     \
        spmm_rows_kernel<LPE_, 1, false, false><<<vgrid, kSpmmRowWaves * 64, 0, stream>>>(                    \
            S, n_rows, col, val, B + f0, ldb, part, W, nv, dl, n_long > 0 ? 1 : 0, nullptr, &h->long_count);  \
    } while (0)
            if (W == 16)
                RSC_SPMM_BLOCKED_LAUNCH(4);
            else if (W == 32)
                RSC_SPMM_BLOCKED_LAUNCH(8);
            else
                RSC_SPMM_BLOCKED_LAUNCH(16);
#undef RSC_SPMM_BLOCKED_LAUNCH
            const int64_t nc = (int64_t)n_rows * ((dl + 3) / 4);
            combine_blocks_kernel<<<(unsigned)ceil_div(nc, 256), 256, 0, stream>>>(part, W, n_rows, P, dl,
                                                                                  Y + f0, ldy);
        }
        return hipGetLastError();
    }
    const bool ordered = use_order(n_rows, nnz_bound);
    // a plan's row list (long rows, or the whole order) prepared once sits in
    // this workspace already; else this call builds it
    const bool pre = prep && prep->ready && prep->P == 1 && prep->ordered == ordered;
    if (used_prep) *used_prep = pre;
    int32_t n_long_blocks;
    if (pre) {
        n_long_blocks = (int32_t)std::min<int64_t>(
            prep->long_rows >= 0 ? prep->long_rows : long_rows_bound(n_rows, nnz_bound), kSpmmLongBlocks);
    } else {
        n_long_blocks = (int32_t)std::min<int64_t>(long_rows_bound(n_rows, nnz_bound), kSpmmLongBlocks);
        const hipError_t e = spmm_rows_prepare(n_rows, nnz_bound, rowptr, ws, stream);
        if (e != hipSuccess) return e;
    }
    const int32_t *order = ordered ? list : nullptr;
    const unsigned grid = (unsigned)ceil_div(n_rows, kSpmmRowWaves);
    const int32_t slice = spmm_slice_width(n_rows, nnz_hint, n_src_hint, d);
    // the hint pays off only when the gathered rows far outgrow the on-chip
    // caches (MALL included); below that, bypassing them loses reuse
    const bool hint = hint_cols && spmm_hint_taken(n_src_hint, d, slice);
    for (int32_t f0 = 0; f0 < d;) {
        const int32_t dl = std::min<int32_t>(d - f0, slice);
#define RSC_SPMM_LAUNCH_H(LPE_, NV_, H_)                                                               \
    do {                                                                                               \
        if (n_long_blocks > 0) {                                                                       \
            if (f0 > 0 || pre) zero_next_kernel<<<1, 1, 0, stream>>>(&h->long_next);                   \
            spmm_long_kernel<LPE_, NV_, H_><<<n_long_blocks, kSpmmLongWaves * 64, 0, stream>>>(         \
                rowptr, 1, col, val, B + f0, ldb, Y + f0, ldy, dl, &h->long_count, &h->long_next, list);  \
        }                                                                                              \
        spmm_rows_kernel<LPE_, NV_, true, H_><<<grid, kSpmmRowWaves * 64, 0, stream>>>(                \
            rowptr, 1, col, val, B + f0, ldb, Y + f0, ldy, n_rows, dl, n_long_blocks > 0 ? 1 : 0, order,  \
            &h->long_count);                                                                           \
    } while (0)
#define RSC_SPMM_LAUNCH(LPE_, NV_)                   \
    do {                                             \
        if (hint)                                    \
            RSC_SPMM_LAUNCH_H(LPE_, NV_, true);      \
        else                                         \
            RSC_SPMM_LAUNCH_H(LPE_, NV_, false);     \
    } while (0)
        switch (slice) {
            case 16: RSC_SPMM_LAUNCH(4, 1); break;
            case 32: RSC_SPMM_LAUNCH(8, 1); break;
            case 64: RSC_SPMM_LAUNCH(16, 1); break;
            case 128: RSC_SPMM_LAUNCH(32, 1); break;
            default:
                if (dl <= 4 * kWave) RSC_SPMM_LAUNCH(64, 1); else RSC_SPMM_LAUNCH(64, 2);
        }
#undef RSC_SPMM_LAUNCH
#undef RSC_SPMM_LAUNCH_H
        f0 += dl;
    }
    return hipGetLastError();
}

}  // namespace rsc
