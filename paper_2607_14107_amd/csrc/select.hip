// polestar_select: TopK of the drift over the cached positions of each
// sequence (Alg. 1, TopK; cached set I = J \ J_b of Sec. 2).
//
// One 1024-thread workgroup per sequence.  Each thread keeps IPT consecutive
// positions in registers as order-preserving 32-bit keys of the fp32 drift
// (+0.0 and -0.0 share one key).  A most-significant-digit-first radix
// select (4 passes of 8 bits, histograms in LDS) finds the key T of the k-th
// largest candidate and how many candidates equal to T are still needed;
// those are taken lowest position first.  Two block prefix sums in position
// order then rank the ties and write the chosen positions ascending.  The
// work is integer-only and latency-bound (tens of KB per step).
#include "common.hpp"
#include "host_common.hpp"

namespace ps {
namespace {

constexpr int kSelBlock = 1024;

__device__ __forceinline__ uint32_t order_key(float f) {
    uint32_t u = __float_as_uint(f);
    if (u == 0x80000000u) u = 0u;                       // -0.0 -> +0.0
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

template <int IPT>
__global__ __launch_bounds__(kSelBlock) void select_kernel(const float* __restrict__ drift,
                                                           const uint8_t* __restrict__ elig,
                                                           int seq, int bs, int bl, int k,
                                                           int32_t* __restrict__ idx,
                                                           int32_t* __restrict__ cnt) {
    __shared__ int hist[256];
    __shared__ int scan_tmp[17];
    __shared__ uint32_t sh_prefix;
    __shared__ int sh_remaining;

    const int b = blockIdx.x;
    const int t = threadIdx.x;
    const int p0 = t * IPT;
    if (k == 0) {                       // uniform over the block
        if (t == 0) cnt[b] = 0;
        return;
    }
    const float* dr = drift + static_cast<size_t>(b) * seq;
    const uint8_t* el = elig ? elig + static_cast<size_t>(b) * seq : nullptr;

    uint32_t key[IPT];
    bool valid[IPT];
    int nv = 0;
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
        const int p = p0 + j;
        bool v = p < seq && !(p >= bs && p < bs + bl);
        if (v && el) v = el[p] != 0;
        valid[j] = v;
        key[j] = v ? order_key(dr[p]) : 0u;
        nv += v ? 1 : 0;
    }
    int n_cand;
    (void)block_excl_scan(nv, scan_tmp, &n_cand);

    bool sel[IPT];
    if (k >= n_cand) {
#pragma unroll
        for (int j = 0; j < IPT; ++j) sel[j] = valid[j];
    } else {
        uint32_t prefix = 0u, pmask = 0u;
        int remaining = k;   // >= 1 here
        for (int shift = 24; shift >= 0; shift -= 8) {
            if (t < 256) hist[t] = 0;
            __syncthreads();
#pragma unroll
            for (int j = 0; j < IPT; ++j)
                if (valid[j] && (key[j] & pmask) == prefix)
                    atomicAdd(&hist[(key[j] >> shift) & 255u], 1);
            __syncthreads();
            if (t < kWave) {
                // lane t owns bins 4t..4t+3; suffix sums from the top bin down
                const int h0 = hist[4 * t], h1 = hist[4 * t + 1];
                const int h2 = hist[4 * t + 2], h3 = hist[4 * t + 3];
                const int own = h0 + h1 + h2 + h3;
                int suf = own;   // inclusive suffix over lanes >= t
#pragma unroll
                for (int o = 1; o < kWave; o <<= 1) {
                    int v = __shfl_down(suf, o);
                    if (t + o < kWave) suf += v;
                }
                int run = suf - own;   // count in bins above 4t+3
                const int hv[4] = {h0, h1, h2, h3};
#pragma unroll
                for (int q = 3; q >= 0; --q) {
                    const int above = run;
                    run += hv[q];
                    if (run >= remaining && above < remaining) {
                        sh_prefix = prefix | (static_cast<uint32_t>(4 * t + q) << shift);
                        sh_remaining = remaining - above;
                    }
                }
            }
            __syncthreads();
            prefix = sh_prefix;
            remaining = sh_remaining;
            pmask |= 255u << shift;
            __syncthreads();
        }
        // prefix is the key T of the k-th largest; take `remaining` keys equal
        // to T, lowest position first.
        int neq = 0;
#pragma unroll
        for (int j = 0; j < IPT; ++j) neq += (valid[j] && key[j] == prefix) ? 1 : 0;
        int eq_total;
        int eq_rank = block_excl_scan(neq, scan_tmp, &eq_total);
#pragma unroll
        for (int j = 0; j < IPT; ++j) {
            const bool eq = valid[j] && key[j] == prefix;
            sel[j] = (valid[j] && key[j] > prefix) || (eq && eq_rank < remaining);
            eq_rank += eq ? 1 : 0;
        }
    }

    int ns = 0;
#pragma unroll
    for (int j = 0; j < IPT; ++j) ns += sel[j] ? 1 : 0;
    int total;
    int pos = block_excl_scan(ns, scan_tmp, &total);
    int32_t* out = idx + static_cast<size_t>(b) * k;
#pragma unroll
    for (int j = 0; j < IPT; ++j)
        if (sel[j]) out[pos++] = p0 + j;
    for (int i = total + t; i < k; i += kSelBlock) out[i] = -1;
    if (t == 0) cnt[b] = total;
}

template <int IPT>
void launch(int batch, int seq, const float* drift, const uint8_t* elig, int bs, int bl, int k,
            int32_t* idx, int32_t* cnt, hipStream_t s) {
    hipLaunchKernelGGL((select_kernel<IPT>), dim3(batch), dim3(kSelBlock), 0, s, drift, elig, seq,
                       bs, bl, k, idx, cnt);
}

}  // namespace
}  // namespace ps

extern "C" polestar_status polestar_select(int batch, int seq, const float* drift,
                                           const uint8_t* eligible, int block_start,
                                           int block_len, int k, int32_t* stale_idx,
                                           int32_t* stale_count, hipStream_t stream) {
    using namespace ps;
    if (batch <= 0 || seq <= 0 || !drift || !stale_count || block_start < 0 || block_len < 0 ||
        block_start > seq - block_len || k < 0 || k > seq || (k > 0 && !stale_idx))
        return POLESTAR_ERR_INVALID_ARGUMENT;
    const int ipt = ceil_div(seq, kSelBlock);
    int32_t* idx = stale_idx;
    switch (ipt <= 1 ? 1 : ipt <= 2 ? 2 : ipt <= 4 ? 4 : ipt <= 8 ? 8 : ipt <= 16 ? 16 : ipt <= 32 ? 32 : 0) {
        case 1: launch<1>(batch, seq, drift, eligible, block_start, block_len, k, idx, stale_count, stream); break;
        case 2: launch<2>(batch, seq, drift, eligible, block_start, block_len, k, idx, stale_count, stream); break;
        case 4: launch<4>(batch, seq, drift, eligible, block_start, block_len, k, idx, stale_count, stream); break;
        case 8: launch<8>(batch, seq, drift, eligible, block_start, block_len, k, idx, stale_count, stream); break;
        case 16: launch<16>(batch, seq, drift, eligible, block_start, block_len, k, idx, stale_count, stream); break;
        case 32: launch<32>(batch, seq, drift, eligible, block_start, block_len, k, idx, stale_count, stream); break;
        default: return POLESTAR_ERR_UNSUPPORTED;   // seq above 32768
    }
    return launch_status();
}
