// polestar_drift: per-token KL drift between current and previous hidden
// states (Sec. 3, eq. "drift"; the distribution of a token is the softmax of
// its hidden state over the d channels).
//
// A row is spread over one wave (batches of 2048 rows and more, d up to 4096
// in bf16: eight 16-byte chunks of each row per lane) or 128-256 threads:
// the two rows of the token are loaded once
// with coalesced 16-byte loads into registers (an HBM-bound stream of 2*d
// elements), both row maxima ma, mb are reduced (shuffles, then LDS across
// the row's waves), then the thread accumulates in fp32, with reference
// points ra = rb = max(ma, mb) when |ma - mb| <= 16, else ra = ma, rb = mb,
// eb_c = exp(b_c - rb), ea_c = exp(a_c - ra) and dl_c = (a_c - b_c) - (ra - rb),
//   Zb  = sum eb_c,   Za = sum ea_c,
//   Sqe = sum (ea_c - eb_c)   (as eb_c * expm1(dl_c) when |dl_c| < 1/8),
//   Spd = sum ea_c * dl_c
// so that KL(softmax(a) || softmax(b)) = Spd / Za - log(Za / Zb), with
// Za = Zb + Sqe and log(Za / Zb) = log1p(Sqe / Zb) while the two sums are
// within a factor of two.  Every term lies in [0, 1] (no overflow or 0 * inf
// for rows that differ by any amount), nearly equal rows keep their small
// drift accurate, and identical rows give exactly 0.
#include "drift_dev.hpp"

namespace ps {
namespace {

template <bool BF16, int TPR, int NCH>
__global__ __launch_bounds__(kDriftBlock) void drift_kernel(const char* __restrict__ hc,
                                                            const char* __restrict__ hp,
                                                            float* __restrict__ out,
                                                            int rows, int d) {
    drift_body<BF16, TPR, NCH>(hc, hp, out, rows, d, blockIdx.x);
}

template <bool BF16, int TPR, int NCH>
void launch(const void* hc, const void* hp, float* out, int rows, int d, hipStream_t s) {
    dim3 grid(ceil_div(rows, kDriftBlock / TPR));
    hipLaunchKernelGGL((drift_kernel<BF16, TPR, NCH>), grid, dim3(kDriftBlock), 0, s,
                       static_cast<const char*>(hc), static_cast<const char*>(hp), out, rows, d);
}

// Launch shape from drift_config (the table the fused step uses too).
template <bool BF16>
bool dispatch(int chunks, const void* hc, const void* hp, float* out, int rows, int d,
              hipStream_t s) {
    int tpr = 0, nch = 0;
    if (!drift_config(chunks, rows, tpr, nch)) return false;
    switch (tpr * 16 + nch) {
#define PS_CASE(TPR, NCH) \
        case TPR * 16 + NCH: launch<BF16, TPR, NCH>(hc, hp, out, rows, d, s); return true;
        PS_DRIFT_SHAPES(PS_CASE)
#undef PS_CASE
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
    const long rows = static_cast<long>(batch) * seq;
    if (rows > 0x7fffffffL) return POLESTAR_ERR_UNSUPPORTED;
    const int chunks = d / (bf16 ? 8 : 4);
    const bool ok = bf16 ? dispatch<true>(chunks, h_cur, h_prev, drift, static_cast<int>(rows), d, stream)
                         : dispatch<false>(chunks, h_cur, h_prev, drift, static_cast<int>(rows), d, stream);
    if (!ok) return POLESTAR_ERR_UNSUPPORTED;   // d above 16384 (bf16) / 8192 (fp32)
    return launch_status();
}
