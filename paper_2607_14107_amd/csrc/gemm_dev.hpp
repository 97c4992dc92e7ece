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
// Refresh mode: sequence b owns rows [b*R, (b+1)*R), R = k_max + block_len:
// its first count_b rows are its stale positions, the last block_len rows
// its active block; rows in between (count_b < k_max) map to nothing.  A
// fixed stride costs no prefix over the counts, so a row's position is one
// load away.  Block-rows mode: row m is position block_start + m % block_len
// of sequence m / block_len.
__device__ __forceinline__ int gemm_rows_total(const GemmArgs& g) {
    return g.batch * (g.mode == kGemmRefresh ? g.k_max + g.block_len : g.block_len);
}

// Row m -> (sequence, position); b = -1 when the row maps to nothing.
__device__ __forceinline__ void map_row(const GemmArgs& g, int m, int& b, int& pos) {
    b = -1;
    pos = 0;
    if (m < 0 || m >= gemm_rows_total(g)) return;
    if (g.mode == kGemmBlockRows) {
        b = m / g.block_len;
        pos = g.block_start + (m - b * g.block_len);
        return;
    }
    const int R = g.k_max + g.block_len;
    const int sb = m / R;
    const int local = m - sb * R;
    if (local >= g.k_max) {
        b = sb;
        pos = g.block_start + (local - g.k_max);
        return;
    }
    int c = g.stale_count[sb];
    const int p = g.stale_idx[static_cast<size_t>(sb) * g.k_max + local];
    c = c < 0 ? 0 : (c > g.k_max ? g.k_max : c);
    if (local >= c || p < 0 || p >= g.seq) return;   // unused slot or out-of-range entry: refresh nothing
    b = sb;
    pos = p;
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
    __shared__ float red[kSmallWaves][BM][17];

    const int t = threadIdx.x;
    const int lane = t & 63;
    const int w = t >> 6;
    const int col0 = bx * 16;
    const int m0 = by * BM;
    const int kcol = (lane >> 4) * 16;   // lane group g reads bytes 16g + 64s: 64 contiguous bytes of a row per load
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
        for (int s = 0; s < 4; ++s) rb[s] = ld16(brow + step * 256 + 64 * s + kcol);
    };
    uint4 q0[4], q1[4], q2[4];
    load_b(min(w, slast), q0);
    load_b(min(w + W, slast), q1);

    if (m0 >= gemm_rows_total(g)) return;
    if (t < BM) {
        int b, pos;
        map_row(g, m0 + t, b, pos);
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
            for (int mt = 0; mt < MT; ++mt) ra[mt][s] = ld16(arow[mt] + step * 256 + 64 * s + kcol);
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
