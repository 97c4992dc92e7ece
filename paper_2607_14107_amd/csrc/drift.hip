// polestar_drift: per-token KL drift between current and previous hidden
// states (Sec. 3, eq. "drift"; the distribution of a token is the softmax of
// its hidden state over the d channels).
//
// A row is spread over 64-256 threads (4 waves at d = 4096, two 16-byte
// chunks of each row per lane): the two rows of the token are loaded once
// with coalesced 16-byte loads into registers (an HBM-bound stream of 2*d
// elements), the common max is reduced (shuffles, then LDS across the
// row's waves), then the thread accumulates in fp32
//   Zb  = sum e_c,              e_c = exp(b_c - m)
//   Sqe = sum e_c * expm1(dlt_c),   dlt = a - b
//   Spd = sum e_c * (1 + expm1(dlt_c)) * dlt_c
// so that sum exp(a_c - m) = Zb + Sqe and
//   KL(softmax(a) || softmax(b)) = Spd / (Zb + Sqe) - log1p(Sqe / Zb).
// Only one exponential per element is needed besides expm1, and identical
// rows give exactly 0.
#include "common.hpp"
#include "host_common.hpp"

namespace ps {
namespace {

constexpr int kDriftBlock = 256;
constexpr float kSmall = 0.0625f;              // |dlt| below this: series for expm1

// expm1 for |x| < 1/16 from its Taylor series; the first omitted term
// x^6/720 is below 1.4e-9 relative there.
__device__ __forceinline__ float expm1_small(float x) {
    float p = fmaf(x, 1.0f / 120.0f, 1.0f / 24.0f);
    p = fmaf(x, p, 1.0f / 6.0f);
    p = fmaf(x, p, 0.5f);
    p = fmaf(x, p, 1.0f);
    return x * p;
}

// expm1 on either branch, chosen by a bitwise select so that the code stays
// straight-line (no per-element exec-mask branches); both sides are cheap.
__device__ __forceinline__ float expm1_any(float x) {
    const float series = expm1_small(x);
    const float direct = fast_exp2(x * kLog2e) - 1.0f;
    const uint32_t pick = 0u - static_cast<uint32_t>(fabsf(x) < kSmall);
    return __uint_as_float((__float_as_uint(series) & pick) | (__float_as_uint(direct) & ~pick));
}

// Reduce NV values at once over the TPR threads of a row: wave shuffles,
// then one LDS round across the row's waves.  `red` holds NV floats per wave.
template <int TPR, int NV, bool MAX>
__device__ __forceinline__ void row_reduce(float (&v)[NV], float* red) {
#pragma unroll
    for (int i = 0; i < NV; ++i) v[i] = MAX ? wave_max(v[i]) : wave_sum(v[i]);
    if constexpr (TPR > kWave) {
        const int w = threadIdx.x >> 6;
        const int lane = threadIdx.x & 63;
        constexpr int W = TPR / kWave;        // waves per row
        if (lane == 0) {
#pragma unroll
            for (int i = 0; i < NV; ++i) red[w * NV + i] = v[i];
        }
        __syncthreads();
        const int first = (w / W) * W;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            float x = red[first * NV + i];
#pragma unroll
            for (int q = 1; q < W; ++q) x = MAX ? fmaxf(x, red[(first + q) * NV + i]) : x + red[(first + q) * NV + i];
            v[i] = x;
        }
        __syncthreads();
    }
}

// One row of d elements per TPR threads (TPR = 64, 128 or 256); each thread
// keeps NCH 16-byte chunks of both rows in registers.  Rows of a workgroup:
// kDriftBlock / TPR.
template <bool BF16, int TPR, int NCH>
__global__ __launch_bounds__(kDriftBlock) void drift_kernel(const char* __restrict__ hc,
                                                            const char* __restrict__ hp,
                                                            float* __restrict__ out,
                                                            int rows, int d) {
    using T = Elem<BF16>;
    __shared__ float red[3 * (kDriftBlock / kWave)];
    const int tr = threadIdx.x % TPR;             // thread within the row
    const int row_raw = blockIdx.x * (kDriftBlock / TPR) + threadIdx.x / TPR;
    const bool live = row_raw < rows;
    const int row = live ? row_raw : rows - 1;    // keep every thread in the reductions
    const size_t base = static_cast<size_t>(row) * d * T::kBytes;
    const int chunks = d / T::E;

    // Unconditional loads: chunks past the row end re-read chunk 0 and are
    // masked out of the arithmetic.
    uint4 ra[NCH], rb[NCH];
    bool ok[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        const int ch = c * TPR + tr;
        ok[c] = ch < chunks;
        const size_t off = base + static_cast<size_t>(ok[c] ? ch : 0) * 16;
        ra[c] = ld16(hc + off);
        rb[c] = ld16(hp + off);
    }
    __builtin_amdgcn_sched_barrier(0);    // every load in flight before any use

    // Pass 1: common maximum of the row.
    float m = -INFINITY;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        float a[T::E], b[T::E];
        T::unpack(ra[c], a);
        T::unpack(rb[c], b);
#pragma unroll
        for (int j = 0; j < T::E; ++j) m = fmaxf(m, ok[c] ? fmaxf(a[j], b[j]) : -INFINITY);
    }
    {
        float mx[1] = {m};
        row_reduce<TPR, 1, true>(mx, red);
        m = mx[0];
    }
    const float mlog = m * kLog2e;

    // Pass 2: the three sums (masked chunks contribute nothing).
    float zb = 0.0f, sqe = 0.0f, spd = 0.0f;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        float a[T::E], b[T::E];
        T::unpack(ra[c], a);
        T::unpack(rb[c], b);
        const float keep = ok[c] ? 1.0f : 0.0f;
#pragma unroll
        for (int j = 0; j < T::E; ++j) {
            const float dl = a[j] - b[j];
            const float e = keep * fast_exp2(fmaf(b[j], kLog2e, -mlog));
            const float em = expm1_any(dl);
            zb += e;
            sqe = fmaf(e, em, sqe);
            spd = fmaf(fmaf(e, em, e), dl, spd);
        }
    }
    {
        float sums[3] = {zb, sqe, spd};
        row_reduce<TPR, 3, false>(sums, red);
        zb = sums[0];
        sqe = sums[1];
        spd = sums[2];
    }
    if (live && tr == 0) out[row] = spd / (zb + sqe) - log1pf(sqe / zb);
}

template <bool BF16, int TPR, int NCH>
void launch(const void* hc, const void* hp, float* out, int rows, int d, hipStream_t s) {
    dim3 grid(ceil_div(rows, kDriftBlock / TPR));
    hipLaunchKernelGGL((drift_kernel<BF16, TPR, NCH>), grid, dim3(kDriftBlock), 0, s,
                       static_cast<const char*>(hc), static_cast<const char*>(hp), out, rows, d);
}

// chunks per row -> (threads per row, chunks per thread)
template <bool BF16>
bool dispatch(int chunks, const void* hc, const void* hp, float* out, int rows, int d,
              hipStream_t s) {
    if (chunks <= 64) { launch<BF16, 64, 1>(hc, hp, out, rows, d, s); return true; }
    if (chunks <= 128) { launch<BF16, 64, 2>(hc, hp, out, rows, d, s); return true; }
    if (chunks <= 256) { launch<BF16, 128, 2>(hc, hp, out, rows, d, s); return true; }
    if (chunks <= 512) { launch<BF16, 256, 2>(hc, hp, out, rows, d, s); return true; }
    if (chunks <= 1024) { launch<BF16, 256, 4>(hc, hp, out, rows, d, s); return true; }
    if (chunks <= 2048) { launch<BF16, 256, 8>(hc, hp, out, rows, d, s); return true; }
    return false;
}

}  // namespace
}  // namespace ps

extern "C" polestar_status polestar_drift(polestar_dtype dtype, int batch, int seq, int d,
                                          const void* h_cur, const void* h_prev, float* drift,
                                          hipStream_t stream) {
    using namespace ps;
    if (!dtype_ok(dtype) || batch <= 0 || seq <= 0 || d <= 0 || !h_cur || !h_prev || !drift)
        return POLESTAR_ERR_INVALID_ARGUMENT;
    if (!row_ok(dtype, d) || !aligned16(h_cur) || !aligned16(h_prev) || !aligned16(drift))
        return POLESTAR_ERR_UNSUPPORTED;
    const bool bf16 = dtype == POLESTAR_BF16;
    const long rows = static_cast<long>(batch) * seq;
    if (rows > 0x7fffffffL) return POLESTAR_ERR_UNSUPPORTED;
    const int chunks = d / (bf16 ? 8 : 4);
    const bool ok = bf16 ? dispatch<true>(chunks, h_cur, h_prev, drift, static_cast<int>(rows), d, stream)
                         : dispatch<false>(chunks, h_cur, h_prev, drift, static_cast<int>(rows), d, stream);
    if (!ok) return POLESTAR_ERR_UNSUPPORTED;   // d above 16384 (bf16) / 8192 (fp32)
    return launch_status();
}
