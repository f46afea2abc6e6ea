// Gather-ceiling probe: the B-row gathers of an exact SpMM and nothing else.
// A measurement helper, not a step of the method: it tells how fast the
// memory system serves the product's own access pattern (the same column
// stream, the same row-slice width per pass, the same cache policy), so the
// SpMM's time can be set against what that pattern allows rather than
// against the HBM peak alone.
//
// Each wave takes 64 consecutive entries of the column stream (row
// boundaries play no part: rows are consecutive runs of it), loads their
// columns with one coalesced load and gathers each referenced B row slice
// with the SpMM's lane layout (LPE lanes per entry, one float4 per lane, two
// for 512-wide rows), `kInflight` loads issued before any is consumed. The
// loaded values are added into a register sum; one float per wave goes to
// `sink`, so no load can be dropped. No values and no row pointers: only the
// col stream (4 bytes per entry) besides the gathers.
//
// With Y, the probe also writes an output of the product's size (n_rows rows
// of the pass's slice, the same non-temporal float4 stores as the SpMM's row
// store), shared evenly over the waves: wave w writes rows
// [w n_rows / W, (w + 1) n_rows / W) of W waves after its gathers, each
// element its wave's sum. That is the gather pattern plus the output stream,
// the product's whole compulsory traffic bar values and row pointers; where
// the output is a large share of it (sampled products of sparse slices)
// it bounds the product more tightly than the gathers alone.
#include "rsc_internal.h"

namespace rsc {
namespace {

typedef float vf4 __attribute__((ext_vector_type(4)));
constexpr int32_t kColMask = 0x7FFFFFFF;  // bit 31: a plan's hub-column hint
constexpr int kProbeWaves = 4;            // waves per block

__device__ __forceinline__ vf4 load_nt(const vf4 *p) { return __builtin_nontemporal_load(p); }

template <int LPE, int NV, int kInflight, bool kHint>
__global__ __launch_bounds__(kProbeWaves * 64) void gather_probe_kernel(const int32_t *__restrict__ col, int64_t nnz,
                                                                       const float *__restrict__ B, int64_t ldb,
                                                                       int32_t d, float *__restrict__ sink,
                                                                       float *__restrict__ Y, int64_t ldy,
                                                                       int32_t n_rows) {
    constexpr int G = kWave / LPE;  // entries per load instruction
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t w = (int64_t)blockIdx.x * kProbeWaves + (threadIdx.x >> 6);
    const int64_t base = w * kWave;
    if (base >= nnz) return;  // wave-uniform
    const int32_t cnt = __builtin_amdgcn_readfirstlane((int32_t)min<int64_t>(kWave, nnz - base));
    const int32_t my_c = lane < cnt ? __builtin_nontemporal_load(col + base + lane) : 0;
    const int g = lane / LPE, sl = lane % LPE;
    bool act[NV];
#pragma unroll
    for (int q = 0; q < NV; ++q) act[q] = 4 * sl + 4 * kWave * q < d;
    vf4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int32_t t = 0; t < cnt; t += kInflight * G) {
        vf4 b[kInflight][NV];
#pragma unroll
        for (int u = 0; u < kInflight; ++u) {
            const int32_t j = t + u * G + g;  // entry of this lane's group
            int32_t cf;
            if constexpr (G == 1)
                cf = __builtin_amdgcn_readlane(my_c, (t + u) & (kWave - 1));
            else
                cf = __shfl(my_c, j & (kWave - 1));
            const int32_t c = cf & kColMask;
            const vf4 *brow = reinterpret_cast<const vf4 *>(B + (int64_t)c * ldb) + sl;
#pragma unroll
            for (int q = 0; q < NV; ++q) {
                b[u][q] = vf4{0.f, 0.f, 0.f, 0.f};
                if (j < cnt && act[q]) b[u][q] = (kHint && cf >= 0) ? load_nt(brow + q * kWave) : brow[q * kWave];
            }
        }
#pragma unroll
        for (int u = 0; u < kInflight; ++u)
#pragma unroll
            for (int q = 0; q < NV; ++q) acc += b[u][q];
    }
    float s = acc.x + acc.y + acc.z + acc.w;
#pragma unroll
    for (int m = 1; m < kWave; m <<= 1) s += __shfl_xor(s, m);
    if (lane == 0) sink[w] = s;
    if (Y == nullptr) return;  // kernel-uniform
    const int64_t n_waves = (nnz + kWave - 1) / kWave;
    const int64_t r1 = (w + 1) * n_rows / n_waves;  // <= n_rows since w < n_waves
    const vf4 o = {s, s, s, s};
    for (int64_t r = w * n_rows / n_waves + g; r < r1; r += G) {
        float *yrow = Y + r * ldy;
#pragma unroll
        for (int q = 0; q < NV; ++q) {
            const int32_t f = 4 * sl + 4 * kWave * q;
            if (f + 4 <= d) {
                __builtin_nontemporal_store(o, reinterpret_cast<vf4 *>(yrow + f));
            } else if (f < d) {
                for (int32_t x = f; x < d; ++x) yrow[x] = s;
            }
        }
    }
}

struct ProbeOut {
    float *Y;  // nullptr: no output stream
    int64_t ldy;
    int32_t n_rows;
};

template <int LPE, int NV, int U>
void launch_one(const int32_t *col, int64_t nnz, const float *B, int64_t ldb, int32_t dl, bool hint, float *sink,
                ProbeOut out, hipStream_t stream) {
    const unsigned grid = (unsigned)ceil_div(ceil_div(nnz, kWave), kProbeWaves);
    if (hint)
        gather_probe_kernel<LPE, NV, U, true>
            <<<grid, kProbeWaves * 64, 0, stream>>>(col, nnz, B, ldb, dl, sink, out.Y, out.ldy, out.n_rows);
    else
        gather_probe_kernel<LPE, NV, U, false>
            <<<grid, kProbeWaves * 64, 0, stream>>>(col, nnz, B, ldb, dl, sink, out.Y, out.ldy, out.n_rows);
}

template <int U>
void launch_width(const int32_t *col, int64_t nnz, const float *B, int64_t ldb, int32_t dl, int32_t slice, bool hint,
                  float *sink, ProbeOut out, hipStream_t stream) {
    switch (slice) {
        case 16: launch_one<4, 1, U>(col, nnz, B, ldb, dl, hint, sink, out, stream); break;
        case 32: launch_one<8, 1, U>(col, nnz, B, ldb, dl, hint, sink, out, stream); break;
        case 64: launch_one<16, 1, U>(col, nnz, B, ldb, dl, hint, sink, out, stream); break;
        case 128: launch_one<32, 1, U>(col, nnz, B, ldb, dl, hint, sink, out, stream); break;
        default:
            if (dl <= 4 * kWave)
                launch_one<64, 1, U>(col, nnz, B, ldb, dl, hint, sink, out, stream);
            else
                launch_one<64, 2, U>(col, nnz, B, ldb, dl, hint, sink, out, stream);
    }
}

}  // namespace

int64_t gather_probe_sink_count(int64_t nnz) { return ceil_div(nnz, kWave); }

hipError_t gather_probe_launch(const int32_t *col, int64_t nnz, const float *B, int64_t ldb, int32_t d, int32_t slice,
                               bool hint, int32_t inflight, float *sink, float *Y, int64_t ldy, int32_t n_rows,
                               hipStream_t stream) {
    if (nnz <= 0) return hipSuccess;
    for (int32_t f0 = 0; f0 < d; f0 += slice) {
        const int32_t dl = std::min<int32_t>(d - f0, slice);
        const ProbeOut out{Y ? Y + f0 : nullptr, ldy, n_rows};
        switch (inflight) {
            case 4: launch_width<4>(col, nnz, B + f0, ldb, dl, slice, hint, sink, out, stream); break;
            case 16: launch_width<16>(col, nnz, B + f0, ldb, dl, slice, hint, sink, out, stream); break;
            default: launch_width<8>(col, nnz, B + f0, ldb, dl, slice, hint, sink, out, stream);
        }
    }
    return hipGetLastError();
}

}  // namespace rsc
