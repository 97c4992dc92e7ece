// polestar_drift: per-token KL drift between current and previous hidden
// states (Sec. 3, eq. "drift"; the distribution of a token is the softmax of
// its hidden state over the d channels).
//
// One wavefront owns one row: it loads the two rows of the token once with
// coalesced 16-byte loads into registers (an HBM-bound stream of 2*d
// elements), reduces the common max, then accumulates in fp32
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

constexpr int kDriftBlock = 256;               // 4 waves, one row each
constexpr int kRowsPerBlock = kDriftBlock / kWave;
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

__device__ __forceinline__ float expm1_any(float x) {
    return fabsf(x) < kSmall ? expm1_small(x) : fast_exp2(x * kLog2e) - 1.0f;
}

template <bool BF16, int NCH>
__global__ __launch_bounds__(kDriftBlock) void drift_kernel(const char* __restrict__ hc,
                                                            const char* __restrict__ hp,
                                                            float* __restrict__ out,
                                                            int rows, int d) {
    using T = Elem<BF16>;
    const int lane = threadIdx.x & 63;
    const int row = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
    if (row >= rows) return;
    const size_t base = static_cast<size_t>(row) * d * T::kBytes;

    uint4 ra[NCH], rb[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        const int e0 = (c * kWave + lane) * T::E;
        if (e0 < d) {
            ra[c] = ld16(hc + base + static_cast<size_t>(e0) * T::kBytes);
            rb[c] = ld16(hp + base + static_cast<size_t>(e0) * T::kBytes);
        }
    }

    // Pass 1: common maximum and the largest |dlt| of the row.
    float m = -INFINITY, big = 0.0f;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        const int e0 = (c * kWave + lane) * T::E;
        if (e0 < d) {
            float a[T::E], b[T::E];
            T::unpack(ra[c], a);
            T::unpack(rb[c], b);
#pragma unroll
            for (int j = 0; j < T::E; ++j) {
                m = fmaxf(m, fmaxf(a[j], b[j]));
                big = fmaxf(big, fabsf(a[j] - b[j]));
            }
        }
    }
    m = wave_max(m);
    big = wave_max(big);
    const float mlog = m * kLog2e;

    // Pass 2: the three sums.
    float zb = 0.0f, sqe = 0.0f, spd = 0.0f;
    if (big < kSmall) {
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const int e0 = (c * kWave + lane) * T::E;
            if (e0 < d) {
                float a[T::E], b[T::E];
                T::unpack(ra[c], a);
                T::unpack(rb[c], b);
#pragma unroll
                for (int j = 0; j < T::E; ++j) {
                    const float dl = a[j] - b[j];
                    const float e = fast_exp2(fmaf(b[j], kLog2e, -mlog));
                    const float em = expm1_small(dl);
                    zb += e;
                    sqe = fmaf(e, em, sqe);
                    spd = fmaf(fmaf(e, em, e), dl, spd);
                }
            }
        }
    } else {
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const int e0 = (c * kWave + lane) * T::E;
            if (e0 < d) {
                float a[T::E], b[T::E];
                T::unpack(ra[c], a);
                T::unpack(rb[c], b);
#pragma unroll
                for (int j = 0; j < T::E; ++j) {
                    const float dl = a[j] - b[j];
                    const float e = fast_exp2(fmaf(b[j], kLog2e, -mlog));
                    const float em = expm1_any(dl);
                    zb += e;
                    sqe = fmaf(e, em, sqe);
                    spd = fmaf(fmaf(e, em, e), dl, spd);
                }
            }
        }
    }
    zb = wave_sum(zb);
    sqe = wave_sum(sqe);
    spd = wave_sum(spd);
    if (lane == 0) out[row] = spd / (zb + sqe) - log1pf(sqe / zb);
}

template <bool BF16, int NCH>
void launch(const void* hc, const void* hp, float* out, int rows, int d, hipStream_t s) {
    dim3 grid(ceil_div(rows, kRowsPerBlock));
    hipLaunchKernelGGL((drift_kernel<BF16, NCH>), grid, dim3(kDriftBlock), 0, s,
                       static_cast<const char*>(hc), static_cast<const char*>(hp), out, rows, d);
}

template <bool BF16>
bool dispatch(int nch, const void* hc, const void* hp, float* out, int rows, int d,
              hipStream_t s) {
    switch (nch) {
        case 1: launch<BF16, 1>(hc, hp, out, rows, d, s); return true;
        case 2: launch<BF16, 2>(hc, hp, out, rows, d, s); return true;
        case 3: launch<BF16, 3>(hc, hp, out, rows, d, s); return true;
        case 4: launch<BF16, 4>(hc, hp, out, rows, d, s); return true;
        case 5: launch<BF16, 5>(hc, hp, out, rows, d, s); return true;
        case 6: launch<BF16, 6>(hc, hp, out, rows, d, s); return true;
        case 7: launch<BF16, 7>(hc, hp, out, rows, d, s); return true;
        case 8: launch<BF16, 8>(hc, hp, out, rows, d, s); return true;
        case 10: launch<BF16, 10>(hc, hp, out, rows, d, s); return true;
        case 12: launch<BF16, 12>(hc, hp, out, rows, d, s); return true;
        case 16: launch<BF16, 16>(hc, hp, out, rows, d, s); return true;
        default: return false;
    }
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
    const int per_chunk = kWave * (bf16 ? 8 : 4);
    int nch = ceil_div(d, per_chunk);
    // round the register budget up to an instantiated size
    static const int sizes[] = {1, 2, 3, 4, 5, 6, 7, 8, 10, 12, 16};
    int pick = 0;
    for (int s : sizes)
        if (s >= nch) { pick = s; break; }
    if (pick == 0) return POLESTAR_ERR_UNSUPPORTED;   // d above 8192 (bf16) / 4096 (fp32)
    const long rows = static_cast<long>(batch) * seq;
    if (rows > 0x7fffffffL) return POLESTAR_ERR_UNSUPPORTED;
    bool ok = bf16 ? dispatch<true>(pick, h_cur, h_prev, drift, static_cast<int>(rows), d, stream)
                   : dispatch<false>(pick, h_cur, h_prev, drift, static_cast<int>(rows), d, stream);
    if (!ok) return POLESTAR_ERR_UNSUPPORTED;
    return launch_status();
}
