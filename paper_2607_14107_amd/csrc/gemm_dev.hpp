// Device side of the skinny "gather rows -> MFMA GEMM -> scatter rows": row
// bookkeeping, output addressing and the small-M kernel body, shared by the
// GEMM kernels and the fused step kernel.  Internal to the library.
#pragma once

#include "common.hpp"
#include "gemm.hpp"

namespace ps {
namespace {

constexpr int kGemmBlock = 256;
constexpr int kSmallWaves = 4;    // gemm_small_kernel: waves per workgroup
constexpr int kSmallBlock = kSmallWaves * 64;

// Row bookkeeping --------------------------------------------------------------
// Refresh mode: sequence b contributes count_b stale rows followed by its
// block_len active-block rows; rows of all sequences are numbered
// consecutively.  pre[b] is the first row of sequence b, pre[batch] the total.
__device__ int build_prefix(const GemmArgs& g, int* pre, int* scan_tmp) {
    int carry = 0;
    for (int base = 0; base < g.batch; base += blockDim.x) {
        const int b = base + threadIdx.x;
        int v = 0;
        if (b < g.batch) {
            int c = g.stale_count ? g.stale_count[b] : 0;
            c = c < 0 ? 0 : (c > g.k_max ? g.k_max : c);
            v = c + g.block_len;
        }
        int tot;
        const int ex = block_excl_scan(v, scan_tmp, &tot);
        if (b < g.batch) pre[b] = carry + ex;
        carry += tot;
    }
    if (threadIdx.x == 0) pre[g.batch] = carry;
    __syncthreads();
    return carry;
}

// Row m -> (sequence, position); b = -1 when the row maps to nothing.
__device__ void map_row(const GemmArgs& g, const int* pre, int total, int m, int& b, int& pos) {
    b = -1;
    pos = 0;
    if (m < 0 || m >= total) return;
    if (g.mode == kGemmBlockRows) {
        b = m / g.block_len;
        pos = g.block_start + (m - b * g.block_len);
        return;
    }
    int lo = 0, hi = g.batch - 1;       // last b with pre[b] <= m
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (pre[mid] <= m) lo = mid; else hi = mid - 1;
    }
    const int local = m - pre[lo];
    const int cnt = pre[lo + 1] - pre[lo] - g.block_len;
    if (local < cnt) {
        const int p = g.stale_idx[static_cast<size_t>(lo) * g.k_max + local];
        if (p < 0 || p >= g.seq) return;          // out-of-range entries refresh nothing
        pos = p;
    } else {
        pos = g.block_start + (local - cnt);
    }
    b = lo;
}

template <bool BF16>
__device__ __forceinline__ void store_elem(char* p, float v) {
    if constexpr (BF16) *reinterpret_cast<uint16_t*>(p) = static_cast<uint16_t>(f32_to_bf16_bits(v));
    else *reinterpret_cast<float*>(p) = v;
}

// Destination of output element (row with sequence b / position pos / row
// number m, column n).
template <bool BF16>
__device__ __forceinline__ char* out_ptr(const GemmArgs& g, int b, int pos, int m, int n) {
    constexpr size_t es = Elem<BF16>::kBytes;
    if (g.mode == kGemmBlockRows)
        return g.out0 + (static_cast<size_t>(m) * g.N + n) * es;
    const size_t row = static_cast<size_t>(b) * g.seq + pos;
    if (n < g.n0) return g.out0 + (row * g.n0 + n) * es;
    return g.out1 + (row * (g.N - g.n0) + (n - g.n0)) * es;
}

// 8 consecutive fp32 values -> destination (16-byte bf16 or 2x16-byte fp32 store).
template <bool BF16>
__device__ __forceinline__ void store8(char* dst, const float* v) {
    if constexpr (BF16) {
        st16(dst, make_uint4(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                             pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7])));
    } else {
        st16(dst, make_uint4(__float_as_uint(v[0]), __float_as_uint(v[1]),
                             __float_as_uint(v[2]), __float_as_uint(v[3])));
        st16(dst + 16, make_uint4(__float_as_uint(v[4]), __float_as_uint(v[5]),
                                  __float_as_uint(v[6]), __float_as_uint(v[7])));
    }
}

// Weight row of output column n (nullptr past N).
__device__ __forceinline__ const char* weight_row(const GemmArgs& g, int n, int es) {
    if (n >= g.N) return nullptr;
    return n < g.n0 ? g.w0 + static_cast<size_t>(n) * g.K * es
                    : g.w1 + static_cast<size_t>(n - g.n0) * g.K * es;
}

// ---------------------------------------------------------------------------
// gemm_small_kernel: at most 16*MT rows, 16 columns per workgroup, the 4
// waves take super-steps w, w+4, w+8, ... of K and are summed in LDS.
// ---------------------------------------------------------------------------

template <bool BF16, int MT>
__device__ __forceinline__ void small_body(const GemmArgs& g, int bx, int by) {
    using T = Elem<BF16>;
    constexpr int ES = T::kBytes;
    constexpr int BM = MT * 16;
    __shared__ int rowb[BM], rowp[BM];
    __shared__ int scan_tmp[17];
    __shared__ float red[kSmallWaves][BM][17];
    extern __shared__ int pre[];

    const int t = threadIdx.x;
    const int lane = t & 63;
    const int w = t >> 6;
    const int col0 = bx * 16;
    const int m0 = by * BM;
    const int kcol = (lane >> 4) * 64;
    const int nsteps = g.K / (256 / ES);
    // wave w: super-steps w, w+W, ...; the last one it owns is slast
    // (prefetches past it re-read slast and are ignored).
    constexpr int W = kSmallWaves;
    const int nmine = w < nsteps ? (nsteps - 1 - w) / W + 1 : 0;
    const int slast = w < nsteps ? w + W * (nmine - 1) : 0;

    // Weight row of column col0 + lane%16 (past N: row 0, never stored); its
    // first two super-steps are requested before the row bookkeeping.
    const char* brow = weight_row(g, col0 + (lane & 15), ES);
    if (!brow) brow = g.w0;
    auto load_b = [&](int step, uint4 (&rb)[4]) {
#pragma unroll
        for (int s = 0; s < 4; ++s) rb[s] = ld16(brow + step * 256 + kcol + 16 * s);
    };
    uint4 q0[4], q1[4], q2[4];
    load_b(min(w, slast), q0);
    load_b(min(w + W, slast), q1);

    const int total = g.mode == kGemmRefresh ? build_prefix(g, pre, scan_tmp)
                                             : g.batch * g.block_len;
    if (m0 >= total) return;
    if (t < BM) {
        int b, pos;
        map_row(g, pre, total, m0 + t, b, pos);
        rowb[t] = b;
        rowp[t] = pos;
    }
    __syncthreads();

    // Rows past the end read row 0 and are never stored.
    const char* arow[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const int r = mt * 16 + (lane & 15);
        const int b = rowb[r];
        arow[mt] = b >= 0 ? g.x + (static_cast<size_t>(b) * g.seq + rowp[r]) * g.K * ES : g.x;
    }
    auto load_a = [&](int step, uint4 (&ra)[MT][4]) {
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) ra[mt][s] = ld16(arow[mt] + step * 256 + kcol + 16 * s);
    };
    floatx4 acc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[mt] = floatx4{0.f, 0.f, 0.f, 0.f};
    auto compute = [&](const uint4 (&ra)[MT][4], const uint4 (&rb)[4]) {
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) acc[mt] = Mma<BF16>::step(ra[mt][s], rb[s], acc[mt]);
    };

    uint4 a0[MT][4], a1[MT][4], a2[MT][4];
    load_a(min(w, slast), a0);
    load_a(min(w + W, slast), a1);
#define PS_SMALL_STEP(I, A_USE, B_USE, A_LOAD, B_LOAD)                      \
    {                                                                       \
        __builtin_amdgcn_sched_barrier(0);                                  \
        load_a(min(w + W * ((I) + 2), slast), A_LOAD);                      \
        load_b(min(w + W * ((I) + 2), slast), B_LOAD);                      \
        __builtin_amdgcn_sched_barrier(0);                                  \
        compute(A_USE, B_USE);                                              \
    }
    int ic = 0;
    for (; ic + 3 <= nmine; ic += 3) {
        PS_SMALL_STEP(ic, a0, q0, a2, q2)
        PS_SMALL_STEP(ic + 1, a1, q1, a0, q0)
        PS_SMALL_STEP(ic + 2, a2, q2, a1, q1)
    }
    if (ic < nmine) PS_SMALL_STEP(ic, a0, q0, a2, q2)
    if (ic + 1 < nmine) PS_SMALL_STEP(ic + 1, a1, q1, a0, q0)
#undef PS_SMALL_STEP

    // sum the waves in order: lane holds rows mt*16 + 4*(lane/16) + i, column lane%16
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) red[w][mt * 16 + 4 * (lane >> 4) + i][lane & 15] = acc[mt][i];
    __syncthreads();
    // thread -> (row r, 8 columns c)
    for (int idx = t; idx < BM * 2; idx += kSmallBlock) {
        const int r = idx >> 1, c = (idx & 1) * 8;
        const int b = rowb[r];
        const int n = col0 + c;
        if (b < 0 || n >= g.N) continue;
        float v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            float acc_j = red[0][r][c + j];
#pragma unroll
            for (int q = 1; q < kSmallWaves; ++q) acc_j += red[q][r][c + j];
            v[j] = acc_j;
        }
        store8<BF16>(out_ptr<BF16>(g, b, rowp[r], m0 + r, n), v);
    }
}

}  // namespace
}  // namespace ps
