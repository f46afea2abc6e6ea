// C ABI of the library (declared in include/rsc.h): argument validation,
// status codes, the sampled-matrix cache and the host-side budget helpers.
// Every device step is a kernel of spmm.hip, scores.hip, topk.hip,
// slice.hip, sample.hip, mean.hip, greedy.hip or validate.hip.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "rsc.h"
#include "rsc_internal.h"

namespace {

thread_local std::string g_err;

rsc_status_t fail(rsc_status_t s, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return s;
}

rsc_status_t hip_fail(hipError_t e, const char *what) {
    return fail(RSC_ERR_HIP, "%s: %s (%s)", what, hipGetErrorName(e), hipGetErrorString(e));
}

#define RSC_TRY(expr)                     \
    do {                                  \
        rsc_status_t _s = (expr);         \
        if (_s != RSC_OK) return _s;      \
    } while (0)

#define RSC_HIP(expr, what)                         \
    do {                                            \
        hipError_t _e = (expr);                     \
        if (_e != hipSuccess) return hip_fail(_e, what); \
    } while (0)

bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

rsc_status_t check_device() {
    static const int count = [] {  // counted once, thread-safe initialisation
        int c = 0;
        if (hipGetDeviceCount(&c) != hipSuccess) c = 0;
        return c;
    }();
    if (count <= 0) return fail(RSC_ERR_NO_DEVICE, "no HIP device visible");
    return RSC_OK;
}

// bud / total > C_num / C_den without overflow (both sides can pass 2^63)
bool over_budget(int64_t bud, int64_t total, int32_t C_num, int32_t C_den) {
    return (__int128)bud * C_den > (__int128)C_num * total;
}

rsc_status_t check_csr(const rsc_csr_t *A, const char *name) {
    if (!A) return fail(RSC_ERR_INVALID_ARGUMENT, "%s is NULL", name);
    if (A->n_rows < 0 || A->n_cols < 0 || A->nnz < 0)
        return fail(RSC_ERR_INVALID_ARGUMENT, "%s has negative dimensions", name);
    if (A->nnz >= (int64_t(1) << 31)) return fail(RSC_ERR_UNSUPPORTED, "%s: nnz >= 2^31", name);
    if (!A->rowptr) return fail(RSC_ERR_INVALID_ARGUMENT, "%s->rowptr is NULL", name);
    if (A->nnz > 0 && (!A->col || !A->val))
        return fail(RSC_ERR_INVALID_ARGUMENT, "%s->col/val is NULL", name);
    if (!aligned(A->rowptr, 4) || !aligned(A->col, 4) || !aligned(A->val, 4))
        return fail(RSC_ERR_UNSUPPORTED, "%s arrays must be 4-byte aligned", name);
    return RSC_OK;
}

rsc_status_t check_dense(const void *p, int64_t rows, int32_t d, int64_t ld, const char *name) {
    if (d < 1) return fail(RSC_ERR_INVALID_ARGUMENT, "d = %d < 1", d);
    if (ld < d) return fail(RSC_ERR_INVALID_ARGUMENT, "%s: ld %lld < d %d", name, (long long)ld, d);
    if (ld % 4 != 0) return fail(RSC_ERR_UNSUPPORTED, "%s: ld %lld is not a multiple of 4", name, (long long)ld);
    if (rows > 0 && !p) return fail(RSC_ERR_INVALID_ARGUMENT, "%s is NULL", name);
    if (!aligned(p, 16)) return fail(RSC_ERR_UNSUPPORTED, "%s is not 16-byte aligned", name);
    return RSC_OK;
}

rsc_status_t check_ws(const void *ws, size_t ws_bytes, size_t need, const char *what) {
    if (ws_bytes < need)
        return fail(RSC_ERR_CAPACITY, "%s workspace: %zu bytes given, %zu needed", what, ws_bytes, need);
    if (need > 0 && !ws) return fail(RSC_ERR_INVALID_ARGUMENT, "%s workspace is NULL", what);
    if (!aligned(ws, 256)) return fail(RSC_ERR_UNSUPPORTED, "%s workspace is not 256-byte aligned", what);
    return RSC_OK;
}

bool validate_env() {
    const char *v = getenv("RSC_VALIDATE");
    return v && v[0] == '1';
}

rsc_status_t validate(const rsc_csr_t *A, const char *name, int64_t *bad_row, hipStream_t stream) {
    if (bad_row) *bad_row = -1;
    if (A->n_rows == 0) {
        if (A->nnz != 0) {
            if (bad_row) *bad_row = 0;
            return fail(RSC_ERR_INVALID_ARGUMENT, "%s: no rows but nnz = %lld", name, (long long)A->nnz);
        }
        return RSC_OK;
    }
    unsigned long long *d_bad = nullptr, h_bad = 0;
    RSC_HIP(hipMallocAsync((void **)&d_bad, sizeof(unsigned long long), stream), "validate alloc");
    hipError_t e = rsc::csr_validate_launch(A->n_rows, A->n_cols, A->nnz, A->rowptr, A->col, d_bad, stream);
    if (e == hipSuccess) e = hipMemcpyAsync(&h_bad, d_bad, sizeof h_bad, hipMemcpyDeviceToHost, stream);
    (void)hipFreeAsync(d_bad, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return hip_fail(e, "validate");
    if (h_bad != ~0ull) {
        if (bad_row) *bad_row = (int64_t)h_bad;
        return fail(RSC_ERR_INVALID_ARGUMENT, "%s: malformed CSR at row %llu", name, h_bad);
    }
    return RSC_OK;
}

// Whether a product with this many B rows can ever take the column cache hint
// (the SpMM uses it when one feature pass gathers from more than 512 MiB of
// B rows, and a pass is at most 512 floats wide).
bool hint_worthwhile(int32_t n_src) { return (double)n_src * 512 * sizeof(float) > 512.0 * 1024 * 1024; }

// The greedy's shared argument checks: alpha is a fraction of the n columns
// (0 <= alpha <= 1) and the full budget sum_l nnz d_l fits int64 (*total).
rsc_status_t check_greedy(int32_t L, int32_t n, int64_t nnz, const int32_t *d_host, int32_t C_num, int32_t C_den,
                          int32_t alpha_num, int32_t alpha_den, int64_t *total) {
    if (L < 1 || n < 0 || nnz < 0) return fail(RSC_ERR_INVALID_ARGUMENT, "L < 1, n < 0 or nnz < 0");
    if (C_num < 0 || C_den <= 0 || alpha_num < 0 || alpha_den <= 0 || alpha_num > alpha_den)
        return fail(RSC_ERR_INVALID_ARGUMENT, "bad budget or step fraction (need C >= 0, 0 <= alpha <= 1)");
    __int128 t = 0;
    for (int32_t l = 0; l < L; ++l) {
        if (d_host[l] < 1) return fail(RSC_ERR_INVALID_ARGUMENT, "d[%d] < 1", l);
        t += (__int128)nnz * d_host[l];
    }
    if (t > (__int128)INT64_MAX) return fail(RSC_ERR_INVALID_ARGUMENT, "budget sum_l nnz * d_l exceeds int64");
    *total = (int64_t)t;
    return RSC_OK;
}

// The device a plan or cache was made on must be the current one when it is used.
rsc_status_t check_same_device(int made_on, const char *what) {
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return fail(RSC_ERR_NO_DEVICE, "no current HIP device");
    if (cur != made_on)
        return fail(RSC_ERR_INVALID_ARGUMENT, "%s was made on device %d, current device is %d", what, made_on, cur);
    return RSC_OK;
}

// Completion markers of the work a plan or cache has enqueued: one event per
// stream it was used on, recorded after each call (not while the stream is
// being captured into a graph: a captured call runs when the caller launches
// the graph, which the caller synchronises). Destroying the handle waits for
// these events only, so work on other streams is never waited for.
struct StreamFence {
    std::vector<std::pair<hipStream_t, hipEvent_t>> ev;

    hipError_t record(hipStream_t s) {
        hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
        hipError_t e = hipStreamIsCapturing(s, &cs);
        if (e != hipSuccess) return e;
        if (cs != hipStreamCaptureStatusNone) return hipSuccess;
        for (auto &p : ev)
            if (p.first == s) return hipEventRecord(p.second, s);
        hipEvent_t x = nullptr;
        e = hipEventCreateWithFlags(&x, hipEventDisableTiming);
        if (e != hipSuccess) return e;
        ev.emplace_back(s, x);
        return hipEventRecord(x, s);
    }

    // waits for every recorded event and releases them; the first error
    hipError_t wait_and_release() {
        hipError_t first = hipSuccess;
        for (auto &p : ev) {
            const hipError_t e = hipEventSynchronize(p.second);
            if (first == hipSuccess) first = e;
            (void)hipEventDestroy(p.second);
        }
        ev.clear();
        return first;
    }
};

// Device memory of plans and caches (and the validation flag) comes from the
// stream-ordered allocator: hipFree would wait for every stream on the
// device, hipFreeAsync only orders the free on one stream. After a handle's
// own work has completed, its memory is freed on a library-owned stream of
// its device (non-blocking, default priority), so destroying it never waits
// for work on other streams; on a failed create, on the creation stream.
constexpr int kMaxDevices = 64;
std::mutex g_stream_mu;
hipStream_t g_free_stream[kMaxDevices] = {};

hipError_t free_stream_of_current_device(hipStream_t *out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_stream_mu);
    if (!g_free_stream[dev]) {
        e = hipStreamCreateWithFlags(&g_free_stream[dev], hipStreamNonBlocking);
        if (e != hipSuccess) return e;
    }
    *out = g_free_stream[dev];
    return hipSuccess;
}

// Pinned host words for the caches' slice-size readback, taken from chunks
// that are never released (hipHostFree would also wait for the whole device).
std::mutex g_pin_mu;
std::vector<int64_t *> g_pin_free;

hipError_t take_pinned_word(int64_t **out) {
    std::lock_guard<std::mutex> lock(g_pin_mu);
    if (g_pin_free.empty()) {
        constexpr int kChunk = 64;
        int64_t *chunk = nullptr;
        const hipError_t e = hipHostMalloc((void **)&chunk, kChunk * sizeof(int64_t), hipHostMallocPortable);
        if (e != hipSuccess) return e;
        for (int i = kChunk - 1; i >= 0; --i) g_pin_free.push_back(chunk + i);
    }
    *out = g_pin_free.back();
    g_pin_free.pop_back();
    return hipSuccess;
}

void return_pinned_word(int64_t *p) {
    if (!p) return;
    std::lock_guard<std::mutex> lock(g_pin_mu);
    g_pin_free.push_back(p);
}

// with RSC_VALIDATE=1, the device check of a caller's CSR before any launch
rsc_status_t maybe_validate(const rsc_csr_t *A, const char *name, hipStream_t stream) {
    return validate_env() ? validate(A, name, nullptr, stream) : RSC_OK;
}

}  // namespace

struct rsc_cache {
    rsc_allocator_t alloc{};   // alloc.alloc == NULL: hipMallocAsync / hipFreeAsync
    hipStream_t alloc_stream = nullptr;
    rsc_csr_t X{}, XT{};
    int32_t interval = 10;
    int32_t n = 0;  // pairs = columns of X
    int device = 0;
    double *cn2 = nullptr;
    int32_t *colnnz = nullptr;
    uint64_t *key = nullptr;
    double *rn2 = nullptr;  // row square-norms of the last scored dense operand
    double *norms = nullptr;   // [0] = sum of cn2 (||X||_F^2), [1] = sum of rn2 of the last scored operand
    double *sum_ws = nullptr;  // block sums of the fixed-order reductions
    int32_t *count = nullptr;  // randomized refresh: draws per column
    double *colw = nullptr;    // randomized refresh: per-column scale
    void *ws_sample = nullptr;
    size_t ws_sample_bytes = 0;
    bool random = false;       // the current slice comes from rsc_cache_refresh_random
    bool scored = false;       // keys have been computed at least once
    int32_t score_d = 64;      // feature width of the last scored operand
    int32_t *idx = nullptr;
    uint32_t *mask = nullptr;
    uint32_t *prev_mask = nullptr;          // the selection the latest one replaced
    bool has_prev = false;                  // at least two selections were made
    unsigned long long *stale_acc = nullptr;  // staleness counts
    int32_t *s_rowptr = nullptr;
    int32_t *s_col = nullptr;
    float *s_val = nullptr;
    int64_t *d_nnz = nullptr;
    int64_t *h_nnz = nullptr;  // pinned
    void *ws_topk = nullptr, *ws_slice = nullptr, *ws_spmm = nullptr;
    size_t ws_topk_bytes = 0, ws_slice_bytes = 0, ws_spmm_bytes = 0;
    hipEvent_t ev = nullptr;
    int32_t *s_split = nullptr;  // the slice's column-blocked split bounds (when its product is blocked)
    int32_t split_P = 0;          // ranges s_split has room for
    rsc::SpmmPrepared prep;       // the slice product's row list, prepared at each refresh (in ws_spmm)
    int32_t x_long_rows = -1;     // rows of X longer than the long-row threshold (0: no slice has any)
    int32_t k = 0;
    int64_t last_step = 0;
    uint64_t version = 0;
    bool nnz_known = false;
    int64_t nnz_slice = 0;
    StreamFence fence;            // completion of the calls' work, per stream
    hipStream_t free_stream = nullptr;  // the library's stream for this device's frees
};

extern "C" {

const char *rsc_status_string(rsc_status_t s) {
    switch (s) {
        case RSC_OK: return "RSC_OK";
        case RSC_ERR_INVALID_ARGUMENT: return "RSC_ERR_INVALID_ARGUMENT";
        case RSC_ERR_UNSUPPORTED: return "RSC_ERR_UNSUPPORTED";
        case RSC_ERR_OUT_OF_MEMORY: return "RSC_ERR_OUT_OF_MEMORY";
        case RSC_ERR_CAPACITY: return "RSC_ERR_CAPACITY";
        case RSC_ERR_NO_DEVICE: return "RSC_ERR_NO_DEVICE";
        case RSC_ERR_HIP: return "RSC_ERR_HIP";
        case RSC_ERR_INTERNAL: return "RSC_ERR_INTERNAL";
    }
    return "RSC_ERR_UNKNOWN";
}

const char *rsc_last_error(void) { return g_err.c_str(); }

int32_t rsc_abi_version(void) { return RSC_ABI_VERSION; }

rsc_status_t rsc_csr_validate(const rsc_csr_t *A, int64_t *bad_row_host, hipStream_t stream) {
    if (bad_row_host) *bad_row_host = -1;
    RSC_TRY(check_csr(A, "A"));
    RSC_TRY(check_device());
    return validate(A, "A", bad_row_host, stream);
}

// ------------------------------------------------------------------- A1
size_t rsc_spmm_workspace_bytes(const rsc_csr_t *A) {
    if (!A || A->n_rows < 0 || A->nnz < 0) return 0;
    return rsc::spmm_ws_bytes(A->n_rows, A->nnz, A->n_cols);
}

rsc_status_t rsc_spmm(const rsc_csr_t *A, const float *B, int32_t d, int64_t ldb, float *Y,
                      int64_t ldy, void *ws, size_t ws_bytes, hipStream_t stream) {
    RSC_TRY(check_csr(A, "A"));
    RSC_TRY(check_dense(B, A->n_cols, d, ldb, "B"));
    RSC_TRY(check_dense(Y, A->n_rows, d, ldy, "Y"));
    RSC_TRY(check_ws(ws, ws_bytes, rsc::spmm_ws_bytes(A->n_rows, A->nnz, A->n_cols), "spmm"));
    RSC_TRY(check_device());
    RSC_TRY(maybe_validate(A, "A", stream));
    RSC_HIP(rsc::spmm_launch(A->n_rows, A->n_cols, A->nnz, A->rowptr, A->col, A->val, B, d, ldb, Y, ldy, ws,
                             ws_bytes, stream, A->nnz, A->n_cols),
            "spmm launch");
    return RSC_OK;
}

// ------------------------------------------------------------------- A1 without allocation
// Scratch of rsc_spmm_noalloc: a static device array, one copy per GPU the
// library runs on, held until the process ends. Its name is a host-side
// stand-in in host code; the device address of the current GPU's copy comes
// from hipGetSymbolAddress (looked up once per device, with that device
// current) and only that address is passed to kernels.
constexpr size_t kNoallocScratchBytes = size_t(32) << 20;
static __device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

namespace {
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxScratchDevices] = {};

rsc_status_t scratch_of_current_device(void **out) {
    int dev = -1;
    RSC_HIP(hipGetDevice(&dev), "current device");
    if (dev < 0 || dev >= kMaxScratchDevices)
        return fail(RSC_ERR_UNSUPPORTED, "device %d: the no-allocation SpMM supports devices 0..%d", dev,
                    kMaxScratchDevices - 1);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        RSC_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "no-allocation SpMM scratch address");
        if (!p || !aligned(p, 256)) return fail(RSC_ERR_INTERNAL, "scratch address is not 256-byte aligned");
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return RSC_OK;
}
}  // namespace

struct rsc_spmm_plan {
    rsc_csr_t A{};
    int32_t *colf = nullptr;   // A's columns with the hub hint in bit 31 (large graphs only)
    int32_t *split = nullptr;  // column-blocked mode's split bounds (when the product is blocked)
    rsc::SpmmPrepared prep;    // what the runs skip: split bounds, row list (in ws) and its length
    void *ws = nullptr;
    size_t ws_bytes = 0;
    int device = 0;
    StreamFence fence;         // completion of the runs, per stream
    hipStream_t free_stream = nullptr;  // the library's stream for this device's frees
};

// frees the plan's memory, ordered on `s` (stream-ordered frees)
static void plan_free(rsc_spmm_plan_t *p, hipStream_t s) {
    if (!p) return;
    if (p->colf) (void)hipFreeAsync(p->colf, s);
    if (p->split) (void)hipFreeAsync(p->split, s);
    if (p->ws) (void)hipFreeAsync(p->ws, s);
    delete p;
}

rsc_status_t rsc_spmm_plan_create(const rsc_csr_t *A, hipStream_t stream, rsc_spmm_plan_t **out) {
    if (!out) return fail(RSC_ERR_INVALID_ARGUMENT, "out is NULL");
    *out = nullptr;
    RSC_TRY(check_csr(A, "A"));
    RSC_TRY(check_device());
    RSC_TRY(maybe_validate(A, "A", stream));
    rsc_spmm_plan_t *p = new rsc_spmm_plan_t();
    p->A = *A;
    (void)hipGetDevice(&p->device);
    p->ws_bytes = std::max<size_t>(rsc::spmm_ws_bytes(A->n_rows, A->nnz, A->n_cols), 256);
    if (hipMallocAsync(&p->ws, p->ws_bytes, stream) != hipSuccess) {
        (void)hipGetLastError();
        plan_free(p, stream);
        return fail(RSC_ERR_OUT_OF_MEMORY, "plan workspace of %zu bytes", p->ws_bytes);
    }
    // the per-call preparation of the product, done once: split bounds and
    // long-piece list (column-blocked), or the long-row list / row order
    // (prepared for feature widths of 33 and more; a narrower product whose
    // range count differs prepares for itself on every run)
    const int32_t P = std::max(1, rsc::spmm_column_blocks(A->n_rows, A->nnz, A->n_cols, 64));
    {
        hipError_t e = hipSuccess;
        if (P > 1) {
            e = hipMallocAsync((void **)&p->split, sizeof(int32_t) * (size_t)A->n_rows * (P + 1), stream);
            if (e == hipSuccess) e = rsc::spmm_split_launch(A->n_rows, A->n_cols, A->rowptr, A->col, P, p->split, stream);
            if (e == hipSuccess) e = rsc::spmm_blocked_prepare(A->n_rows, A->nnz, p->split, P, p->ws, stream);
        } else {
            p->prep.ordered = rsc::spmm_use_order(A->n_rows, A->nnz);
            e = rsc::spmm_rows_prepare(A->n_rows, A->nnz, A->rowptr, p->ws, stream);
        }
        int32_t long_rows = 0;
        const bool has_list = P > 1 || p->prep.ordered || std::min<int64_t>(A->n_rows, A->nnz / 1025) > 0;
        if (e == hipSuccess && has_list && A->n_rows > 0)
            e = hipMemcpyAsync(&long_rows, rsc::spmm_long_count_of(p->ws), sizeof long_rows, hipMemcpyDeviceToHost,
                               stream);
        if (e == hipSuccess) e = hipStreamSynchronize(stream);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            plan_free(p, stream);
            return e == hipErrorOutOfMemory ? fail(RSC_ERR_OUT_OF_MEMORY, "plan preparation")
                                            : hip_fail(e, "plan preparation");
        }
        p->prep.split = p->split;
        p->prep.P = P;
        p->prep.long_rows = long_rows;
        p->prep.ready = true;
    }
    if (hint_worthwhile(A->n_cols) && A->nnz > 0) {
        int32_t *deg = nullptr;
        void *ws_hub = nullptr;
        hipError_t e = hipMallocAsync((void **)&p->colf, sizeof(int32_t) * (size_t)A->nnz, stream);
        if (e == hipSuccess) e = hipMallocAsync((void **)&deg, sizeof(int32_t) * (size_t)A->n_cols, stream);
        if (e == hipSuccess) e = hipMallocAsync(&ws_hub, rsc::hub_ws_bytes(A->n_cols), stream);
        if (e == hipSuccess) e = rsc::degree_count_launch(A->col, A->nnz, A->n_cols, deg, stream);
        if (e == hipSuccess) e = rsc::hub_bits_launch(deg, nullptr, A->n_cols, ws_hub, stream);
        if (e == hipSuccess) e = rsc::flag_cols_launch(A->col, A->nnz, rsc::hub_bits_of(ws_hub), p->colf, stream);
        if (deg) (void)hipFreeAsync(deg, stream);
        if (ws_hub) (void)hipFreeAsync(ws_hub, stream);
        if (e == hipSuccess) e = hipStreamSynchronize(stream);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            plan_free(p, stream);
            return e == hipErrorOutOfMemory ? fail(RSC_ERR_OUT_OF_MEMORY, "plan allocation failed")
                                            : hip_fail(e, "plan create");
        }
    }
    {
        hipError_t e = free_stream_of_current_device(&p->free_stream);
        if (e == hipSuccess) e = hipStreamSynchronize(stream);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            plan_free(p, stream);
            return hip_fail(e, "plan create");
        }
    }
    *out = p;
    return RSC_OK;
}

rsc_status_t rsc_spmm_plan_run(rsc_spmm_plan_t *p, const float *B, int32_t d, int64_t ldb, float *Y, int64_t ldy,
                               hipStream_t stream) {
    if (!p) return fail(RSC_ERR_INVALID_ARGUMENT, "plan is NULL");
    const rsc_csr_t *A = &p->A;
    RSC_TRY(check_dense(B, A->n_cols, d, ldb, "B"));
    RSC_TRY(check_dense(Y, A->n_rows, d, ldy, "Y"));
    RSC_TRY(check_same_device(p->device, "plan"));
    bool used = false;
    const hipError_t e = rsc::spmm_launch(A->n_rows, A->n_cols, A->nnz, A->rowptr, p->colf ? p->colf : A->col,
                                          A->val, B, d, ldb, Y, ldy, p->ws, p->ws_bytes, stream, A->nnz, A->n_cols,
                                          p->colf != nullptr, &p->prep, &used);
    // a run whose decisions differed (an environment switch changed since the
    // plan was made) rebuilt its own row list in the plan's workspace: from
    // then on every run prepares for itself
    if (!used && A->n_rows > 0) p->prep.ready = false;
    RSC_HIP(e, "plan run");
    RSC_HIP(p->fence.record(stream), "plan run event");
    return RSC_OK;
}

rsc_status_t rsc_spmm_plan_gather_probe(rsc_spmm_plan_t *p, const float *B, int32_t d, int64_t ldb, int32_t inflight,
                                       float *sink, int64_t sink_count, float *Y, int64_t ldy, int32_t *slice_out,
                                       hipStream_t stream) {
    if (!p) return fail(RSC_ERR_INVALID_ARGUMENT, "plan is NULL");
    const rsc_csr_t *A = &p->A;
    RSC_TRY(check_dense(B, A->n_cols, d, ldb, "B"));
    if (Y) RSC_TRY(check_dense(Y, A->n_rows, d, ldy, "Y"));
    if (inflight != 4 && inflight != 8 && inflight != 16)
        return fail(RSC_ERR_INVALID_ARGUMENT, "inflight = %d (4, 8 or 16)", inflight);
    const int64_t need = rsc::gather_probe_sink_count(A->nnz);
    if (sink_count < need) return fail(RSC_ERR_CAPACITY, "sink holds %lld floats, %lld needed", (long long)sink_count,
                                       (long long)need);
    if (need > 0 && !sink) return fail(RSC_ERR_INVALID_ARGUMENT, "sink is NULL");
    RSC_TRY(check_same_device(p->device, "plan"));
    // the feature passes and cache policy an unblocked run of the plan takes
    const int32_t slice = rsc::spmm_slice_width(A->n_rows, A->nnz, A->n_cols, d);
    const bool hint = p->colf != nullptr && rsc::spmm_hint_taken(A->n_cols, d, slice);
    if (slice_out) *slice_out = slice;
    RSC_HIP(rsc::gather_probe_launch(p->colf ? p->colf : A->col, A->nnz, B, ldb, d, slice, hint, inflight, sink, Y,
                                     ldy, A->n_rows, stream),
            "gather probe launch");
    RSC_HIP(p->fence.record(stream), "gather probe event");
    return RSC_OK;
}

rsc_status_t rsc_spmm_noalloc(const rsc_csr_t *A, const float *B, int32_t d, int64_t ldb, float *Y, int64_t ldy,
                              hipStream_t stream) {
    RSC_TRY(check_csr(A, "A"));
    RSC_TRY(check_dense(B, A->n_cols, d, ldb, "B"));
    RSC_TRY(check_dense(Y, A->n_rows, d, ldy, "Y"));
    const size_t need = rsc::spmm_core_ws_bytes(A->n_rows, A->nnz);
    if (need > kNoallocScratchBytes)
        return fail(RSC_ERR_CAPACITY,
                    "rsc_spmm_noalloc: %d rows and %lld entries need %zu bytes of scratch; the static scratch "
                    "holds %zu",
                    A->n_rows, (long long)A->nnz, need, kNoallocScratchBytes);
    RSC_TRY(check_device());
    void *ws = nullptr;
    RSC_TRY(scratch_of_current_device(&ws));
    RSC_HIP(rsc::spmm_launch(A->n_rows, A->n_cols, A->nnz, A->rowptr, A->col, A->val, B, d, ldb, Y, ldy, ws,
                             kNoallocScratchBytes, stream, A->nnz, A->n_cols),
            "spmm_noalloc launch");
    return RSC_OK;
}

rsc_status_t rsc_spmm_plan_destroy(rsc_spmm_plan_t *p) {
    if (!p) return RSC_OK;
    const hipError_t e = p->fence.wait_and_release();  // the plan's own runs only
    plan_free(p, p->free_stream);
    if (e != hipSuccess) return hip_fail(e, "plan destroy");
    return RSC_OK;
}

rsc_status_t rsc_degree_scale(const rsc_csr_t *A, const int32_t *deg_rowptr, int32_t by_column, float *val_out,
                              hipStream_t stream) {
    RSC_TRY(check_csr(A, "A"));
    if (A->nnz > 0 && !val_out) return fail(RSC_ERR_INVALID_ARGUMENT, "val_out is NULL");
    if (by_column && !deg_rowptr) return fail(RSC_ERR_INVALID_ARGUMENT, "deg_rowptr is NULL");
    if (!aligned(val_out, 4) || !aligned(deg_rowptr, 4)) return fail(RSC_ERR_UNSUPPORTED, "misaligned argument");
    RSC_TRY(check_device());
    RSC_TRY(maybe_validate(A, "A", stream));
    RSC_HIP(rsc::degree_scale_launch(A->n_rows, A->rowptr, A->col, A->val, deg_rowptr, by_column ? 1 : 0, val_out,
                                     stream),
            "degree scale launch");
    return RSC_OK;
}

// ------------------------------------------------------------------- A2
rsc_status_t rsc_col_sqnorms(const rsc_csr_t *XT, double *cn2, int32_t *colnnz, hipStream_t stream) {
    RSC_TRY(check_csr(XT, "XT"));
    if (XT->n_rows > 0 && !cn2) return fail(RSC_ERR_INVALID_ARGUMENT, "cn2 is NULL");
    if (!aligned(cn2, 8)) return fail(RSC_ERR_UNSUPPORTED, "cn2 is not 8-byte aligned");
    RSC_TRY(check_device());
    RSC_TRY(maybe_validate(XT, "XT", stream));
    RSC_HIP(rsc::col_sqnorms_launch(XT->n_rows, XT->rowptr, XT->val, cn2, colnnz, stream),
            "col_sqnorms launch");
    return RSC_OK;
}

// ------------------------------------------------------------------- A3
rsc_status_t rsc_pair_scores(const double *cn2, const float *B, int32_t n, int32_t d, int64_t ldb,
                             uint64_t *key, float *score, double *rn2, hipStream_t stream) {
    if (n < 0) return fail(RSC_ERR_INVALID_ARGUMENT, "n = %d < 0", n);
    RSC_TRY(check_dense(B, n, d, ldb, "B"));
    if (n > 0 && (!cn2 || !key)) return fail(RSC_ERR_INVALID_ARGUMENT, "cn2/key is NULL");
    if (!aligned(cn2, 8) || !aligned(key, 8) || !aligned(rn2, 8))
        return fail(RSC_ERR_UNSUPPORTED, "cn2/key/rn2 not 8-byte aligned");
    RSC_TRY(check_device());
    RSC_HIP(rsc::pair_scores_launch(cn2, B, n, d, ldb, key, score, rn2, stream), "pair_scores launch");
    return RSC_OK;
}

// ------------------------------------------------------------------- A4
size_t rsc_topk_workspace_bytes(int32_t n) { return n < 0 ? 0 : rsc::topk_ws_bytes(n); }

rsc_status_t rsc_topk_select(const uint64_t *key, int32_t n, int32_t k, int32_t *idx, uint32_t *mask,
                             void *ws, size_t ws_bytes, hipStream_t stream) {
    if (n < 0) return fail(RSC_ERR_INVALID_ARGUMENT, "n = %d < 0", n);
    if (k < 0 || k > n) return fail(RSC_ERR_INVALID_ARGUMENT, "k = %d outside [0, n = %d]", k, n);
    if (n > 0 && (!key || !mask)) return fail(RSC_ERR_INVALID_ARGUMENT, "key/mask is NULL");
    if (k > 0 && !idx) return fail(RSC_ERR_INVALID_ARGUMENT, "idx is NULL");
    if (!aligned(key, 8) || !aligned(idx, 4) || !aligned(mask, 4))
        return fail(RSC_ERR_UNSUPPORTED, "key/idx/mask misaligned");
    RSC_TRY(check_ws(ws, ws_bytes, rsc::topk_ws_bytes(n), "topk"));
    RSC_TRY(check_device());
    RSC_HIP(rsc::topk_launch(key, n, k, idx, mask, ws, stream), "topk launch");
    return RSC_OK;
}

// ------------------------------------------------------------------- randomized sampling
size_t rsc_sample_workspace_bytes(int32_t n) { return n < 0 ? 0 : rsc::sample_ws_bytes(n); }

rsc_status_t rsc_sample_columns(const uint64_t *key, int32_t n, int32_t k, uint64_t seed, int32_t *count,
                                double *colw, uint32_t *mask, void *ws, size_t ws_bytes, hipStream_t stream) {
    if (n < 0 || k < 0) return fail(RSC_ERR_INVALID_ARGUMENT, "n < 0 or k < 0");
    if (n > 0 && (!key || !count || !colw || !mask))
        return fail(RSC_ERR_INVALID_ARGUMENT, "key/count/colw/mask is NULL");
    if (!aligned(key, 8) || !aligned(colw, 8) || !aligned(count, 4) || !aligned(mask, 4))
        return fail(RSC_ERR_UNSUPPORTED, "misaligned sampler argument");
    RSC_TRY(check_ws(ws, ws_bytes, rsc::sample_ws_bytes(n), "sample"));
    RSC_TRY(check_device());
    RSC_HIP(rsc::sample_launch(key, n, k, seed, count, colw, mask, ws, stream), "sample launch");
    return RSC_OK;
}

// ------------------------------------------------------------------- A5
size_t rsc_slice_workspace_bytes(const rsc_csr_t *A) {
    if (!A || A->nnz < 0) return 0;
    return rsc::slice_ws_bytes(A->nnz);
}

rsc_status_t rsc_slice_csr(const rsc_csr_t *A, const uint32_t *mask, const double *colw, int32_t *rowptr_out,
                           int32_t *col_out, float *val_out, int64_t capacity, int64_t *nnz_out, void *ws,
                           size_t ws_bytes, hipStream_t stream) {
    RSC_TRY(check_csr(A, "A"));
    if (capacity < 0) return fail(RSC_ERR_INVALID_ARGUMENT, "capacity < 0");
    if (!rowptr_out || !nnz_out) return fail(RSC_ERR_INVALID_ARGUMENT, "rowptr_out/nnz_out is NULL");
    if (A->nnz > 0 && !mask) return fail(RSC_ERR_INVALID_ARGUMENT, "mask is NULL");
    if (capacity > 0 && (!col_out || !val_out)) return fail(RSC_ERR_INVALID_ARGUMENT, "col_out/val_out is NULL");
    if (!aligned(nnz_out, 8)) return fail(RSC_ERR_UNSUPPORTED, "nnz_out is not 8-byte aligned");
    if (!aligned(colw, 8)) return fail(RSC_ERR_UNSUPPORTED, "colw is not 8-byte aligned");
    RSC_TRY(check_ws(ws, ws_bytes, rsc::slice_ws_bytes(A->nnz), "slice"));
    RSC_TRY(check_device());
    RSC_TRY(maybe_validate(A, "A", stream));
    RSC_HIP(rsc::slice_launch(A->n_rows, A->n_cols, A->nnz, A->rowptr, A->col, A->val, mask, rowptr_out, col_out, val_out,
                              capacity, nnz_out, ws, stream, colw),
            "slice launch");
    if (capacity < A->nnz) {
        int64_t got = 0;
        RSC_HIP(hipMemcpyAsync(&got, nnz_out, sizeof got, hipMemcpyDeviceToHost, stream), "slice nnz read");
        RSC_HIP(hipStreamSynchronize(stream), "slice sync");
        if (got < 0) return fail(RSC_ERR_INTERNAL, "slice: the single-pass scan did not complete");
        if (got > capacity)
            return fail(RSC_ERR_CAPACITY, "slice has %lld entries, capacity %lld", (long long)got,
                        (long long)capacity);
    }
    return RSC_OK;
}

// ------------------------------------------------------------------- A6 / A7
// frees the cache's memory: through its allocator, or ordered on `s`
static void cache_free(rsc_cache_t *c, hipStream_t s) {
    if (!c) return;
    void *dev[] = {c->cn2, c->colnnz, c->key, c->rn2, c->norms, c->sum_ws, c->count, c->colw, c->idx, c->mask,
                   c->prev_mask, c->stale_acc, c->s_rowptr, c->s_col, c->s_val, c->d_nnz, c->ws_topk, c->ws_slice, c->ws_spmm, c->ws_sample,
                   c->s_split};
    for (void *p : dev) {
        if (!p) continue;
        if (c->alloc.alloc)
            c->alloc.free(p, c->alloc_stream, c->alloc.ctx);
        else
            (void)hipFreeAsync(p, s);
    }
    return_pinned_word(c->h_nnz);
    if (c->ev) (void)hipEventDestroy(c->ev);
    delete c;
}

rsc_status_t rsc_cache_create(const rsc_csr_t *X, const rsc_csr_t *XT, int32_t refresh_interval,
                              hipStream_t stream, rsc_cache_t **out) {
    return rsc_cache_create_ex(X, XT, refresh_interval, nullptr, stream, out);
}

rsc_status_t rsc_cache_create_ex(const rsc_csr_t *X, const rsc_csr_t *XT, int32_t refresh_interval,
                                 const rsc_allocator_t *allocator, hipStream_t stream, rsc_cache_t **out) {
    if (!out) return fail(RSC_ERR_INVALID_ARGUMENT, "out is NULL");
    RSC_TRY(check_csr(X, "X"));
    RSC_TRY(check_csr(XT, "XT"));
    if (XT->n_rows != X->n_cols || XT->n_cols != X->n_rows || XT->nnz != X->nnz)
        return fail(RSC_ERR_INVALID_ARGUMENT, "XT is not shaped like the transpose of X");
    if (refresh_interval < 1) return fail(RSC_ERR_INVALID_ARGUMENT, "refresh_interval < 1");
    if (allocator && (!allocator->alloc || !allocator->free))
        return fail(RSC_ERR_INVALID_ARGUMENT, "allocator without alloc or free");
    RSC_TRY(check_device());
    RSC_TRY(maybe_validate(X, "X", stream));
    if (XT != X) RSC_TRY(maybe_validate(XT, "XT", stream));
    rsc_cache_t *c = new rsc_cache_t();
    if (allocator) c->alloc = *allocator;
    c->alloc_stream = stream;
    c->X = *X;
    c->XT = *XT;
    c->interval = refresh_interval;
    c->n = X->n_cols;
    (void)hipGetDevice(&c->device);
    const int64_t n = std::max<int32_t>(c->n, 1), m = std::max<int64_t>(X->nnz, 1);
    c->ws_topk_bytes = rsc::topk_ws_bytes(c->n);
    c->ws_slice_bytes = rsc::slice_ws_bytes(X->nnz);
    c->ws_spmm_bytes = rsc::spmm_ws_bytes(X->n_rows, X->nnz, X->n_cols);
    c->ws_sample_bytes = rsc::sample_ws_bytes(c->n);
    // split bounds for as many ranges as the full product takes at any of
    // the blocked layouts' widths; a slice's product that would take more
    // runs unblocked
    c->split_P = 1;
    for (const int32_t w : {16, 32, 64})
        c->split_P = std::max(c->split_P, rsc::spmm_column_blocks(X->n_rows, X->nnz, X->n_cols, w));
    struct {
        void **p;
        size_t bytes;
    } allocs[] = {
        {(void **)&c->cn2, sizeof(double) * n},
        {(void **)&c->colnnz, sizeof(int32_t) * n},
        {(void **)&c->key, sizeof(uint64_t) * n},
        {(void **)&c->rn2, sizeof(double) * n},
        {(void **)&c->norms, sizeof(double) * 2},
        {(void **)&c->sum_ws, rsc::sum_ws_bytes(n)},
        {(void **)&c->count, sizeof(int32_t) * n},
        {(void **)&c->colw, sizeof(double) * n},
        {(void **)&c->idx, sizeof(int32_t) * n},
        {(void **)&c->mask, sizeof(uint32_t) * (size_t)rsc::ceil_div(n, 32)},
        {(void **)&c->prev_mask, sizeof(uint32_t) * (size_t)rsc::ceil_div(n, 32)},
        {(void **)&c->stale_acc, sizeof(unsigned long long) * (size_t)rsc::staleness_acc_count()},
        {(void **)&c->s_rowptr, sizeof(int32_t) * ((size_t)X->n_rows + 1)},
        {(void **)&c->s_col, sizeof(int32_t) * m},
        {(void **)&c->s_val, sizeof(float) * m},
        {(void **)&c->d_nnz, sizeof(int64_t)},
        {&c->ws_topk, c->ws_topk_bytes},
        {&c->ws_slice, c->ws_slice_bytes},
        {&c->ws_spmm, c->ws_spmm_bytes},
        {&c->ws_sample, c->ws_sample_bytes},
        {(void **)&c->s_split, sizeof(int32_t) * ((size_t)X->n_rows + 1) * (c->split_P + 1)},
    };
    for (auto &a : allocs) {
        const size_t bytes = std::max<size_t>(a.bytes, 256);
        if (c->alloc.alloc) {
            *a.p = c->alloc.alloc(bytes, stream, c->alloc.ctx);
            if (!*a.p) {
                cache_free(c, stream);
                return fail(RSC_ERR_OUT_OF_MEMORY, "allocator returned NULL for %zu bytes", bytes);
            }
            if (!aligned(*a.p, 256)) {
                cache_free(c, stream);
                return fail(RSC_ERR_UNSUPPORTED, "allocator returned memory that is not 256-byte aligned");
            }
        } else if (hipMallocAsync(a.p, bytes, stream) != hipSuccess) {
            (void)hipGetLastError();
            cache_free(c, stream);
            return fail(RSC_ERR_OUT_OF_MEMORY, "cache allocation of %zu bytes failed", a.bytes);
        }
    }
    hipError_t e = take_pinned_word(&c->h_nnz);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&c->ev, hipEventDisableTiming);
    if (e == hipSuccess) e = free_stream_of_current_device(&c->free_stream);
    if (e == hipSuccess) e = rsc::col_sqnorms_launch(XT->n_rows, XT->rowptr, XT->val, c->cn2, c->colnnz, stream);
    if (e == hipSuccess) e = rsc::sum_fixed_order_launch(c->cn2, c->n, c->sum_ws, c->norms, stream);
    // whether X has long rows at all: a slice's rows are parts of X's, so if
    // none is long, the sampled products need no long-row pass
    int32_t x_long = 0;
    const bool any_long_possible =
        rsc::spmm_use_order(X->n_rows, X->nnz) || std::min<int64_t>(X->n_rows, X->nnz / 1025) > 0;
    if (e == hipSuccess && any_long_possible && X->n_rows > 0) {
        e = rsc::spmm_rows_prepare(X->n_rows, X->nnz, X->rowptr, c->ws_spmm, stream);
        if (e == hipSuccess)
            e = hipMemcpyAsync(&x_long, rsc::spmm_long_count_of(c->ws_spmm), sizeof x_long, hipMemcpyDeviceToHost,
                               stream);
    }
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) {
        cache_free(c, stream);
        return hip_fail(e, "cache create");
    }
    c->x_long_rows = x_long;
    *out = c;
    return RSC_OK;
}

// Before a new selection overwrites the mask: keep the current one (if any)
// as the previous selection, for rsc_cache_staleness.
static rsc_status_t keep_previous_selection(rsc_cache_t *c, hipStream_t stream) {
    if (c->version == 0) return RSC_OK;
    RSC_HIP(hipMemcpyAsync(c->prev_mask, c->mask, sizeof(uint32_t) * (size_t)rsc::ceil_div(c->n, 32),
                           hipMemcpyDeviceToDevice, stream),
            "cache previous selection");
    c->has_prev = true;
    return RSC_OK;
}

// After a new slice: what every sampled product of feature width d (the
// last scored operand's) would build first (split bounds and long-piece list
// when blocked, else the long-row list or the row order), built once into
// ws_spmm. Asynchronous (the list's length stays on the device; launches use
// its bound).
static hipError_t cache_prepare(rsc_cache_t *c, int32_t d, hipStream_t stream) {
    c->prep = rsc::SpmmPrepared{};
    const rsc_csr_t &X = c->X;
    if (X.n_rows == 0) return hipSuccess;
    const int64_t kk = std::min<int64_t>(c->k, c->n);
    const int64_t nnz_hint = c->n > 0 ? X.nnz * kk / c->n : 0;
    const int32_t P = std::max(1, rsc::spmm_column_blocks(X.n_rows, nnz_hint, kk, d));
    hipError_t e;
    if (P > 1) {
        if (P > c->split_P || rsc::spmm_blocked_fits(X.n_rows, X.nnz, P) > c->ws_spmm_bytes) return hipSuccess;
        e = rsc::spmm_split_launch(X.n_rows, X.n_cols, c->s_rowptr, c->s_col, P, c->s_split, stream);
        if (e == hipSuccess) e = rsc::spmm_blocked_prepare(X.n_rows, X.nnz, c->s_split, P, c->ws_spmm, stream);
        c->prep.split = c->s_split;
    } else {
        c->prep.ordered = rsc::spmm_use_order(X.n_rows, X.nnz);
        e = rsc::spmm_rows_prepare(X.n_rows, X.nnz, c->s_rowptr, c->ws_spmm, stream);
    }
    c->prep.P = P;
    c->prep.long_rows = c->x_long_rows == 0 ? 0 : -1;  // else the length stays on the device
    c->prep.ready = e == hipSuccess;
    return e;
}

rsc_status_t rsc_cache_score(rsc_cache_t *c, const float *B, int32_t d, int64_t ldb, hipStream_t stream) {
    if (!c) return fail(RSC_ERR_INVALID_ARGUMENT, "cache is NULL");
    RSC_TRY(check_dense(B, c->n, d, ldb, "B"));
    RSC_TRY(check_same_device(c->device, "cache"));
    RSC_HIP(rsc::pair_scores_launch(c->cn2, B, c->n, d, ldb, c->key, nullptr, c->rn2, stream), "cache scores");
    RSC_HIP(rsc::sum_fixed_order_launch(c->rn2, c->n, c->sum_ws, c->norms + 1, stream), "cache norm sum");
    c->scored = true;
    c->score_d = d;
    RSC_HIP(c->fence.record(stream), "cache event");
    return RSC_OK;
}

rsc_status_t rsc_cache_select(rsc_cache_t *c, int32_t k, int64_t step, hipStream_t stream) {
    if (!c) return fail(RSC_ERR_INVALID_ARGUMENT, "cache is NULL");
    if (k < 0 || k > c->n) return fail(RSC_ERR_INVALID_ARGUMENT, "k = %d outside [0, %d]", k, c->n);
    if (!c->scored) return fail(RSC_ERR_INVALID_ARGUMENT, "cache select before any score");
    RSC_TRY(check_same_device(c->device, "cache"));
    RSC_TRY(keep_previous_selection(c, stream));
    RSC_HIP(rsc::topk_launch(c->key, c->n, k, c->idx, c->mask, c->ws_topk, stream), "cache topk");
    RSC_HIP(rsc::slice_launch(c->X.n_rows, c->X.n_cols, c->X.nnz, c->X.rowptr, c->X.col, c->X.val, c->mask, c->s_rowptr,
                              c->s_col, c->s_val, c->X.nnz, c->d_nnz, c->ws_slice, stream),
            "cache slice");
    RSC_HIP(hipMemcpyAsync(c->h_nnz, c->d_nnz, sizeof(int64_t), hipMemcpyDeviceToHost, stream), "cache nnz");
    RSC_HIP(hipEventRecord(c->ev, stream), "cache event");
    c->k = k;
    c->last_step = step;
    c->version += 1;
    c->nnz_known = false;
    c->random = false;
    RSC_HIP(cache_prepare(c, c->score_d, stream), "cache slice preparation");
    RSC_HIP(c->fence.record(stream), "cache event");
    return RSC_OK;
}

rsc_status_t rsc_cache_refresh_random(rsc_cache_t *c, const float *B, int32_t d, int64_t ldb, int32_t k_draws,
                                      uint64_t seed, int64_t step, hipStream_t stream) {
    if (!c) return fail(RSC_ERR_INVALID_ARGUMENT, "cache is NULL");
    RSC_TRY(check_dense(B, c->n, d, ldb, "B"));
    if (k_draws < 0) return fail(RSC_ERR_INVALID_ARGUMENT, "k_draws < 0");
    RSC_TRY(check_same_device(c->device, "cache"));
    RSC_TRY(rsc_cache_score(c, B, d, ldb, stream));
    RSC_TRY(keep_previous_selection(c, stream));
    RSC_HIP(rsc::sample_launch(c->key, c->n, k_draws, seed, c->count, c->colw, c->mask, c->ws_sample, stream),
            "cache sample");
    RSC_HIP(rsc::slice_launch(c->X.n_rows, c->X.n_cols, c->X.nnz, c->X.rowptr, c->X.col, c->X.val, c->mask, c->s_rowptr,
                              c->s_col, c->s_val, c->X.nnz, c->d_nnz, c->ws_slice, stream, c->colw),
            "cache weighted slice");
    RSC_HIP(hipMemcpyAsync(c->h_nnz, c->d_nnz, sizeof(int64_t), hipMemcpyDeviceToHost, stream), "cache nnz");
    RSC_HIP(hipEventRecord(c->ev, stream), "cache event");
    c->k = k_draws;
    c->last_step = step;
    c->version += 1;
    c->nnz_known = false;
    c->random = true;
    RSC_HIP(cache_prepare(c, c->score_d, stream), "cache slice preparation");
    RSC_HIP(c->fence.record(stream), "cache event");
    return RSC_OK;
}

rsc_status_t rsc_cache_refresh(rsc_cache_t *c, const float *B, int32_t d, int64_t ldb, int32_t k, int64_t step,
                               hipStream_t stream) {
    if (!c) return fail(RSC_ERR_INVALID_ARGUMENT, "cache is NULL");
    RSC_TRY(check_dense(B, c->n, d, ldb, "B"));
    if (k < 0 || k > c->n) return fail(RSC_ERR_INVALID_ARGUMENT, "k = %d outside [0, %d]", k, c->n);
    RSC_TRY(rsc_cache_score(c, B, d, ldb, stream));
    return rsc_cache_select(c, k, step, stream);
}

rsc_status_t rsc_cache_get(rsc_cache_t *c, int64_t step, rsc_csr_t *slice_out, const int32_t **idx_out,
                           int32_t *k_out, int32_t *needs_refresh_out, uint64_t *version_out) {
    if (!c) return fail(RSC_ERR_INVALID_ARGUMENT, "cache is NULL");
    if (needs_refresh_out) *needs_refresh_out = (c->version == 0 || step - c->last_step >= c->interval) ? 1 : 0;
    if (version_out) *version_out = c->version;
    if (k_out) *k_out = c->version ? c->k : 0;
    if (idx_out) *idx_out = (c->version && !c->random) ? c->idx : nullptr;
    if (slice_out) {
        rsc_csr_t s{};
        s.n_rows = c->X.n_rows;
        s.n_cols = c->X.n_cols;
        if (c->version) {
            if (!c->nnz_known) {
                RSC_HIP(hipEventSynchronize(c->ev), "cache get wait");
                if (*c->h_nnz < 0) return fail(RSC_ERR_INTERNAL, "cache slice: the single-pass scan did not complete");
                c->nnz_slice = *c->h_nnz;
                c->nnz_known = true;
            }
            s.nnz = c->nnz_slice;
            s.rowptr = c->s_rowptr;
            s.col = c->s_col;
            s.val = c->s_val;
        }
        *slice_out = s;
    }
    return RSC_OK;
}

rsc_status_t rsc_spmm_sampled(rsc_cache_t *c, const float *B, int32_t d, int64_t ldb, float *Y, int64_t ldy,
                              hipStream_t stream) {
    if (!c) return fail(RSC_ERR_INVALID_ARGUMENT, "cache is NULL");
    if (c->version == 0) return fail(RSC_ERR_INVALID_ARGUMENT, "cache was never refreshed");
    RSC_TRY(check_dense(B, c->X.n_cols, d, ldb, "B"));
    RSC_TRY(check_dense(Y, c->X.n_rows, d, ldy, "Y"));
    RSC_TRY(check_same_device(c->device, "cache"));
    // nnz of the full operand bounds the slice's and sizes the long-row list;
    // the expected kept share k/n of the entries and the k kept source rows
    // choose the feature slice (a function of the arguments only, so results
    // never depend on which calls came before).
    const int64_t kk = std::min<int64_t>(c->k, c->n);
    const int64_t nnz_hint = c->n > 0 ? c->X.nnz * kk / c->n : 0;
    bool used = false;
    const hipError_t e = rsc::spmm_launch(c->X.n_rows, c->X.n_cols, c->X.nnz, c->s_rowptr, c->s_col, c->s_val, B, d,
                                          ldb, Y, ldy, c->ws_spmm, c->ws_spmm_bytes, stream, nnz_hint, kk, false,
                                          &c->prep, &used);
    if (!used) c->prep.ready = false;  // the launch rebuilt its own list in ws_spmm
    RSC_HIP(e, "spmm_sampled launch");
    RSC_HIP(c->fence.record(stream), "cache event");
    return RSC_OK;
}

rsc_status_t rsc_cache_gather_probe(rsc_cache_t *c, const float *B, int32_t d, int64_t ldb, int32_t inflight,
                                    float *sink, int64_t sink_count, float *Y, int64_t ldy, int32_t *slice_out,
                                    hipStream_t stream) {
    if (!c) return fail(RSC_ERR_INVALID_ARGUMENT, "cache is NULL");
    if (c->version == 0) return fail(RSC_ERR_INVALID_ARGUMENT, "cache was never refreshed");
    RSC_TRY(check_dense(B, c->X.n_cols, d, ldb, "B"));
    if (Y) RSC_TRY(check_dense(Y, c->X.n_rows, d, ldy, "Y"));
    if (inflight != 4 && inflight != 8 && inflight != 16)
        return fail(RSC_ERR_INVALID_ARGUMENT, "inflight = %d (4, 8 or 16)", inflight);
    RSC_TRY(check_same_device(c->device, "cache"));
    rsc_csr_t s{};
    RSC_TRY(rsc_cache_get(c, c->last_step, &s, nullptr, nullptr, nullptr, nullptr));  // nnz' (waits once per refresh)
    const int64_t need = rsc::gather_probe_sink_count(s.nnz);
    if (sink_count < need) return fail(RSC_ERR_CAPACITY, "sink holds %lld floats, %lld needed", (long long)sink_count,
                                       (long long)need);
    if (need > 0 && !sink) return fail(RSC_ERR_INVALID_ARGUMENT, "sink is NULL");
    // the feature passes rsc_spmm_sampled takes (decided from the call's shape)
    const int64_t kk = std::min<int64_t>(c->k, c->n);
    const int64_t nnz_hint = c->n > 0 ? c->X.nnz * kk / c->n : 0;
    const int32_t slice = rsc::spmm_slice_width(c->X.n_rows, nnz_hint, kk, d);
    if (slice_out) *slice_out = slice;
    RSC_HIP(rsc::gather_probe_launch(s.col, s.nnz, B, ldb, d, slice, false, inflight, sink, Y, ldy, s.n_rows, stream),
            "gather probe launch");
    RSC_HIP(c->fence.record(stream), "gather probe event");
    return RSC_OK;
}

rsc_status_t rsc_cache_buffers(rsc_cache_t *c, const double **cn2, const int32_t **colnnz, const uint64_t **key,
                               const double **rn2, const uint32_t **mask) {
    if (!c) return fail(RSC_ERR_INVALID_ARGUMENT, "cache is NULL");
    if (cn2) *cn2 = c->cn2;
    if (colnnz) *colnnz = c->colnnz;
    if (key) *key = c->key;
    if (rn2) *rn2 = c->rn2;
    if (mask) *mask = c->mask;
    return RSC_OK;
}

rsc_status_t rsc_cache_norms(rsc_cache_t *c, double *fro_x2_host, double *fro_b2_host, hipStream_t stream) {
    if (!c) return fail(RSC_ERR_INVALID_ARGUMENT, "cache is NULL");
    if (fro_b2_host && !c->scored) return fail(RSC_ERR_INVALID_ARGUMENT, "cache norms before any score");
    RSC_TRY(check_same_device(c->device, "cache"));
    double h[2] = {0.0, 0.0};
    RSC_HIP(hipMemcpyAsync(h, c->norms, sizeof h, hipMemcpyDeviceToHost, stream), "cache norms read");
    RSC_HIP(hipStreamSynchronize(stream), "cache norms wait");
    if (fro_x2_host) *fro_x2_host = h[0];
    if (fro_b2_host) *fro_b2_host = h[1];
    return RSC_OK;
}

rsc_status_t rsc_cache_staleness(rsc_cache_t *c, const int32_t *order, double *auc_host, int64_t *overlap_host,
                                 int64_t *prev_k_host, hipStream_t stream) {
    if (!c) return fail(RSC_ERR_INVALID_ARGUMENT, "cache is NULL");
    if (!c->has_prev) return fail(RSC_ERR_INVALID_ARGUMENT, "cache staleness needs two selections");
    if (c->n > 0 && !order) return fail(RSC_ERR_INVALID_ARGUMENT, "order is NULL");
    if (!aligned(order, 4)) return fail(RSC_ERR_UNSUPPORTED, "order is not 4-byte aligned");
    RSC_TRY(check_same_device(c->device, "cache"));
    const int32_t n = c->n;
    unsigned long long h[8] = {0};
    RSC_HIP(rsc::staleness_launch(order, n, c->prev_mask, c->mask, c->stale_acc, stream), "staleness launch");
    RSC_HIP(hipMemcpyAsync(h, c->stale_acc, sizeof(unsigned long long) * (size_t)rsc::staleness_acc_count(),
                           hipMemcpyDeviceToHost, stream),
            "staleness read");
    RSC_HIP(hipStreamSynchronize(stream), "staleness wait");
    const unsigned long long ranks_sum = h[0], k = h[1], bad = h[2], k_mask = h[3], both = h[4];
    if (bad != 0 || k != k_mask)
        return fail(RSC_ERR_INVALID_ARGUMENT, "order is not a ranking of the %d pairs", n);
    // ordered (selected, unselected) pairs over all such pairs
    const double auc = (k == 0 || k == (unsigned long long)n)
                           ? NAN
                           : (double)(ranks_sum - k * (k - 1) / 2) / ((double)k * (double)(n - (int64_t)k));
    if (auc_host) *auc_host = auc;
    if (overlap_host) *overlap_host = (int64_t)both;
    if (prev_k_host) *prev_k_host = (int64_t)k;
    return RSC_OK;
}

rsc_status_t rsc_cache_destroy(rsc_cache_t *c) {
    if (!c) return RSC_OK;
    const hipError_t e = c->fence.wait_and_release();  // the cache's own work only
    cache_free(c, c->free_stream);
    if (e != hipSuccess) return hip_fail(e, "cache destroy");
    return RSC_OK;
}

// ------------------------------------------------------------------- A8
int32_t rsc_k_from_fraction(int32_t n, int32_t num, int32_t den) {
    if (n < 0 || num < 0 || den <= 0 || num > den) return -1;
    return (int32_t)(((int64_t)n * (int64_t)num) / (int64_t)den);
}

rsc_status_t rsc_greedy_allocate(int32_t L, int32_t n, int64_t nnz, const uint64_t *const *key_host,
                                 const int32_t *colnnz_host, const int32_t *d_host, double fro_a2,
                                 const double *fro_b2_host, int32_t C_num, int32_t C_den, int32_t alpha_num,
                                 int32_t alpha_den, int32_t *k_out_host, int64_t *budget_out_host) {
    if (!key_host || !colnnz_host || !d_host || !fro_b2_host || !k_out_host)
        return fail(RSC_ERR_INVALID_ARGUMENT, "NULL host array");
    int64_t total = 0;
    RSC_TRY(check_greedy(L, n, nnz, d_host, C_num, C_den, alpha_num, alpha_den, &total));
    for (int32_t l = 0; l < L; ++l)
        if (!key_host[l]) return fail(RSC_ERR_INVALID_ARGUMENT, "key_host[%d] is NULL", l);
    // rank order per layer: (key desc, index asc); contribution sqrt(q) with
    // NaN keys (0) counting 0
    std::vector<std::vector<int32_t>> order(L);
    std::vector<std::vector<double>> contrib(L);
    for (int32_t l = 0; l < L; ++l) {
        const uint64_t *key = key_host[l];
        auto &o = order[l];
        o.resize(n);
        for (int32_t i = 0; i < n; ++i) o[i] = i;
        std::sort(o.begin(), o.end(), [key](int32_t a, int32_t b) {
            return key[a] != key[b] ? key[a] > key[b] : a < b;
        });
        auto &c = contrib[l];
        c.resize(n);
        for (int32_t p = 0; p < n; ++p) {
            const uint64_t u = key[o[p]];
            if (u == 0) {
                c[p] = 0.0;
            } else {
                const uint64_t bits = u - 1;
                double q;
                std::memcpy(&q, &bits, sizeof q);
                c[p] = std::sqrt(q);
            }
        }
        k_out_host[l] = n;
    }
    const int32_t step = rsc::greedy_step(n, alpha_num, alpha_den);
    int64_t bud = total;
    while (over_budget(bud, total, C_num, C_den)) {
        int32_t best = -1;
        double best_inc = 0.0;
        for (int32_t l = 0; l < L; ++l) {
            const int32_t k = k_out_host[l];
            if (k <= 0) continue;
            const int32_t k2 = std::max(0, k - step);
            double s = 0.0;
            for (int32_t p = k2; p < k; ++p) s += contrib[l][p];
            const double inc = s / (std::sqrt(fro_a2) * std::sqrt(fro_b2_host[l]));
            if (best < 0 || inc < best_inc) {
                best = l;
                best_inc = inc;
            }
        }
        if (best < 0) break;
        const int32_t k = k_out_host[best], k2 = std::max(0, k - step);
        int64_t drop = 0;
        for (int32_t p = k2; p < k; ++p) drop += colnnz_host[order[best][p]];
        bud -= (int64_t)d_host[best] * drop;
        k_out_host[best] = k2;
    }
    if (budget_out_host) *budget_out_host = bud;
    return RSC_OK;
}

size_t rsc_greedy_profile_workspace_bytes(int32_t n) { return n < 0 ? 0 : rsc::greedy_profile_ws_bytes(n); }

int32_t rsc_greedy_blocks(int32_t n, int32_t alpha_num, int32_t alpha_den) {
    if (n < 0 || alpha_num < 0 || alpha_den <= 0 || alpha_num > alpha_den) return -1;
    return rsc::greedy_blocks(n, rsc::greedy_step(n, alpha_num, alpha_den));
}

rsc_status_t rsc_greedy_profile(const uint64_t *key, const int32_t *colnnz, int32_t n, int32_t alpha_num,
                                int32_t alpha_den, double *mass, int64_t *count, int32_t *order, void *ws,
                                size_t ws_bytes, hipStream_t stream) {
    if (n < 0 || alpha_num < 0 || alpha_den <= 0 || alpha_num > alpha_den)
        return fail(RSC_ERR_INVALID_ARGUMENT, "n < 0 or bad step fraction (need 0 <= alpha <= 1)");
    if (n > 0 && (!key || !colnnz || !mass || !count))
        return fail(RSC_ERR_INVALID_ARGUMENT, "key/colnnz/mass/count is NULL");
    if (!aligned(key, 8) || !aligned(mass, 8) || !aligned(count, 8) || !aligned(colnnz, 4) || !aligned(order, 4))
        return fail(RSC_ERR_UNSUPPORTED, "misaligned profile argument");
    RSC_TRY(check_ws(ws, ws_bytes, rsc::greedy_profile_ws_bytes(n), "greedy profile"));
    RSC_TRY(check_device());
    RSC_HIP(rsc::greedy_profile_launch(key, colnnz, n, rsc::greedy_step(n, alpha_num, alpha_den), mass, count,
                                       order, ws, stream),
            "greedy profile launch");
    return RSC_OK;
}

rsc_status_t rsc_greedy_allocate_profiles(int32_t L, int32_t n, int64_t nnz, int32_t alpha_num,
                                          int32_t alpha_den, const double *const *mass_host,
                                          const int64_t *const *count_host, const int32_t *d_host,
                                          double fro_a2, const double *fro_b2_host, int32_t C_num,
                                          int32_t C_den, int32_t *k_out_host, int64_t *budget_out_host) {
    if (!mass_host || !count_host || !d_host || !fro_b2_host || !k_out_host)
        return fail(RSC_ERR_INVALID_ARGUMENT, "NULL host array");
    int64_t total = 0;
    RSC_TRY(check_greedy(L, n, nnz, d_host, C_num, C_den, alpha_num, alpha_den, &total));
    for (int32_t l = 0; l < L; ++l)
        if (!mass_host[l] || !count_host[l]) return fail(RSC_ERR_INVALID_ARGUMENT, "profile %d is NULL", l);
    const int32_t step = rsc::greedy_step(n, alpha_num, alpha_den);
    for (int32_t l = 0; l < L; ++l) k_out_host[l] = n;
    int64_t bud = total;
    while (over_budget(bud, total, C_num, C_den)) {
        int32_t best = -1;
        double best_inc = 0.0;
        for (int32_t l = 0; l < L; ++l) {
            if (k_out_host[l] <= 0) continue;
            const int32_t j = (n - k_out_host[l]) / step;  // next block from the bottom of the ranking
            const double inc = mass_host[l][j] / (std::sqrt(fro_a2) * std::sqrt(fro_b2_host[l]));
            if (best < 0 || inc < best_inc) {
                best = l;
                best_inc = inc;
            }
        }
        if (best < 0) break;
        const int32_t j = (n - k_out_host[best]) / step;
        bud -= (int64_t)d_host[best] * count_host[best][j];
        k_out_host[best] = std::max(0, k_out_host[best] - step);
    }
    if (budget_out_host) *budget_out_host = bud;
    return RSC_OK;
}

}  // extern "C"
