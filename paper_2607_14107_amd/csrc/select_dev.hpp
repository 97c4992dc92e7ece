// Device side of polestar_select (Alg. 1, TopK of the drift over the cached
// positions I = J \ J_b of Sec. 2), shared by the stand-alone kernel and the
// fused step kernel.
//
// One 256-thread workgroup (4 waves) per sequence.  Each thread keeps IPT
// consecutive positions in registers as order-preserving 32-bit keys of the
// fp32 drift (+0.0 and -0.0 share one key).  A most-significant-digit-first
// radix select (4 passes of 8 bits, double-buffered histograms in LDS, two
// barriers per pass) finds the key T of the k-th largest candidate and how
// many candidates equal to T are still needed; those are taken lowest
// position first.  Two prefix sums in position order then rank the ties and
// write the chosen positions ascending.  The work is integer-only and
// latency-bound (tens of KB per step), so the barrier count is what matters.
#pragma once

#include "common.hpp"

namespace ps {
namespace {


constexpr int kSelBlock = 256;                 // 4 waves per sequence
constexpr int kSelWaves = kSelBlock / kWave;

__device__ __forceinline__ uint32_t order_key(float f) {
    uint32_t u = __float_as_uint(f);
    if (u == 0x80000000u) u = 0u;                       // -0.0 -> +0.0
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Exclusive prefix sum over the 4 waves of the workgroup in thread order.
// `tot` holds kSelWaves ints of LDS owned by this call site.  One barrier.
__device__ __forceinline__ int scan4(int v, int* tot, int* total) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int incl = wave_incl_scan(v, lane);
    if (lane == 63) tot[w] = incl;
    __syncthreads();
    int before = 0, all = 0;
#pragma unroll
    for (int i = 0; i < kSelWaves; ++i) {
        const int x = tot[i];
        before += i < w ? x : 0;
        all += x;
    }
    *total = all;
    return before + incl - v;
}

// The selection for sequence b by one 256-thread workgroup.
template <int IPT>
__device__ __forceinline__ void select_body(const float* __restrict__ drift,
                                            const uint8_t* __restrict__ elig, int seq, int bs,
                                            int bl, int k, int32_t* __restrict__ idx,
                                            int32_t* __restrict__ cnt, int b) {
    __shared__ int hist[2][256];
    __shared__ int tot[4][kSelWaves];
    __shared__ uint32_t sh_prefix[4];
    __shared__ int sh_remaining[4];

    const int t = threadIdx.x;
    const int p0 = t * IPT;
    if (k == 0) {                       // uniform over the block
        if (t == 0) cnt[b] = 0;
        return;
    }
    const float* dr = drift + static_cast<size_t>(b) * seq;
    const uint8_t* el = elig ? elig + static_cast<size_t>(b) * seq : nullptr;

    // keys in registers; positions p0 .. p0 + IPT - 1 of this thread.  Every
    // load is issued before any is used (positions past seq re-read 0).
    float dv[IPT];
    uint8_t ev[IPT];
#pragma unroll
    for (int j = 0; j < IPT; ++j) dv[j] = dr[min(p0 + j, seq - 1)];
    if (el) {                           // uniform branch, outside the element loop
#pragma unroll
        for (int j = 0; j < IPT; ++j) ev[j] = el[min(p0 + j, seq - 1)];
    } else {
#pragma unroll
        for (int j = 0; j < IPT; ++j) ev[j] = 1;
    }
    __builtin_amdgcn_sched_barrier(0);
    uint32_t key[IPT];
    bool valid[IPT];
    int nv = 0;
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
        const int p = p0 + j;
        const bool v = (p < seq) & !((p >= bs) & (p < bs + bl)) & (ev[j] != 0);
        valid[j] = v;
        key[j] = v ? order_key(dv[j]) : 0u;
        nv += v ? 1 : 0;
    }
    hist[0][t] = 0;                     // first histogram buffer (one bin per thread)
    int n_cand;
    (void)scan4(nv, tot[0], &n_cand);   // its barrier also publishes the cleared bins

    bool sel[IPT];
    if (k >= n_cand) {
#pragma unroll
        for (int j = 0; j < IPT; ++j) sel[j] = valid[j];
    } else {
        // Radix select, most significant byte first: find the key T of the
        // k-th largest candidate and how many candidates equal to T to take.
        uint32_t prefix = 0u, pmask = 0u;
        int remaining = k;   // >= 1 here
#pragma unroll
        for (int pass = 0; pass < 4; ++pass) {
            const int shift = 24 - 8 * pass;
            int* h = hist[pass & 1];
            hist[(pass + 1) & 1][t] = 0;        // next pass's buffer, idle since the last pass
#pragma unroll
            for (int j = 0; j < IPT; ++j)
                if (valid[j] && (key[j] & pmask) == prefix)
                    atomicAdd(&h[(key[j] >> shift) & 255u], 1);
            __syncthreads();
            if (t < kWave) {
                // lane t owns bins 4t..4t+3; suffix sums from the top bin down
                const int h0 = h[4 * t], h1 = h[4 * t + 1], h2 = h[4 * t + 2], h3 = h[4 * t + 3];
                const int own = h0 + h1 + h2 + h3;
                int suf = own;   // inclusive suffix over lanes >= t
#pragma unroll
                for (int o = 1; o < kWave; o <<= 1) {
                    const int v = __shfl_down(suf, o);
                    if (t + o < kWave) suf += v;
                }
                int run = suf - own;   // count in bins above 4t+3
                const int hv[4] = {h0, h1, h2, h3};
#pragma unroll
                for (int q = 3; q >= 0; --q) {
                    const int above = run;
                    run += hv[q];
                    if (run >= remaining && above < remaining) {
                        sh_prefix[pass] = prefix | (static_cast<uint32_t>(4 * t + q) << shift);
                        sh_remaining[pass] = remaining - above;
                    }
                }
            }
            __syncthreads();
            prefix = sh_prefix[pass];
            remaining = sh_remaining[pass];
            pmask |= 255u << shift;
        }
        // prefix is the key T of the k-th largest; take `remaining` keys equal
        // to T, lowest position first.
        int neq = 0;
#pragma unroll
        for (int j = 0; j < IPT; ++j) neq += (valid[j] && key[j] == prefix) ? 1 : 0;
        int eq_total;
        int eq_rank = scan4(neq, tot[1], &eq_total);
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
    int pos = scan4(ns, tot[2], &total);
    int32_t* out = idx + static_cast<size_t>(b) * k;
#pragma unroll
    for (int j = 0; j < IPT; ++j)
        if (sel[j]) out[pos++] = p0 + j;
    for (int i = total + t; i < k; i += kSelBlock) out[i] = -1;
    if (t == 0) cnt[b] = total;
}

// Keys per thread for a sequence of `seq` positions: the instantiated
// buckets 1, 2, 3, 4, 6, 8, 16, 32, 64 (0: above 16384 positions).
inline int select_ipt(int seq) {
    const int need = (seq + kSelBlock - 1) / kSelBlock;
    const int buckets[] = {1, 2, 3, 4, 6, 8, 16, 32, 64};
    for (int v : buckets)
        if (need <= v) return v;
    return 0;
}

}  // namespace
}  // namespace ps
