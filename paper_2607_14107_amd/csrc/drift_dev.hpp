// Device side of polestar_drift (drift.hip) and of the fused step's first
// launch: the per-token KL drift between current and previous hidden states
// (Sec. 3, eq. "drift"; the distribution of a token is the softmax of its
// hidden state over the d channels).  The arithmetic is described in
// drift.hip.
#pragma once

#include "common.hpp"
#include "host_common.hpp"

namespace ps {
namespace {

constexpr int kDriftBlock = 256;
constexpr float kSmall = 0.0625f;              // |dl| below this: series for expm1
constexpr float kNear = 16.0f;                 // row maxima closer than this: one reference

// expm1 for |x| < 1/16 from its Taylor series; the first omitted term
// x^6/720 is below 1.4e-9 relative there.
__device__ __forceinline__ float expm1_small(float x) {
#pragma clang fp contract(off)
    float p = fmaf(x, 1.0f / 120.0f, 1.0f / 24.0f);
    p = fmaf(x, p, 1.0f / 6.0f);
    p = fmaf(x, p, 0.5f);
    p = fmaf(x, p, 1.0f);
    return x * p;
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

// The row's KL from its four sums (za and zb lie in [exp(-16), d]).  While
// the two sums stay within a factor of two of each other, za is taken as
// zb + sqe, consistent with log1p(sqe / zb), which keeps the small drift of
// nearly equal rows accurate (and exactly 0 for equal rows); beyond that the
// direct sum za and log(za / zb) carry no cancellation.
__device__ __forceinline__ float drift_finish(float zb, float za, float sqe, float spd) {
#pragma clang fp contract(off)
    const float r = sqe / zb;
    if (fabsf(r) <= 0.5f) return spd / (zb + sqe) - log1pf(r);
    return spd / za - logf(za / zb);
}

// One row of d elements per TPR threads (TPR = 64, 128 or 256); each thread
// keeps NCH 16-byte chunks of both rows in registers.  Rows of a workgroup:
// kDriftBlock / TPR.
template <bool BF16, int TPR, int NCH>
__device__ __forceinline__ void drift_body(const char* __restrict__ hc, const char* __restrict__ hp,
                                           float* __restrict__ out, int rows, int d, int blk) {
    // Every multiply-add below is an explicit fmaf: no other contraction, so
    // the stand-alone kernel and the fused step's launch (different inline
    // contexts) round identically.
#pragma clang fp contract(off)
    using T = Elem<BF16>;
    __shared__ float red[4 * (kDriftBlock / kWave)];
    const int tr = threadIdx.x % TPR;             // thread within the row
    const int row_raw = blk * (kDriftBlock / TPR) + threadIdx.x / TPR;
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

    // Pass 1: the maximum of each row (ma of the current, mb of the previous).
    float mx[2] = {-INFINITY, -INFINITY};
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        float a[T::E], b[T::E];
        T::unpack(ra[c], a);
        T::unpack(rb[c], b);
#pragma unroll
        for (int j = 0; j < T::E; ++j) {
            mx[0] = fmaxf(mx[0], ok[c] ? a[j] : -INFINITY);
            mx[1] = fmaxf(mx[1], ok[c] ? b[j] : -INFINITY);
        }
    }
    row_reduce<TPR, 2, true>(mx, red);
    // Reference points of the exponentials: the common maximum while the two
    // maxima are within kNear of each other (the terms of the KL then cancel
    // from their natural size), else each row's own maximum, the difference
    // of the two moving into dl.  Either way each term lies in [0, 1] and
    // both sums hold a term of at least exp(-kNear).
    const bool near = fabsf(mx[0] - mx[1]) <= kNear;
    const float m = fmaxf(mx[0], mx[1]);
    const float shift = near ? 0.0f : mx[0] - mx[1];
    const float mal = (near ? m : mx[0]) * kLog2e, mbl = (near ? m : mx[1]) * kLog2e;

    // Pass 2: the four sums (masked chunks contribute nothing).
    float zb = 0.0f, za = 0.0f, sqe = 0.0f, spd = 0.0f;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        float a[T::E], b[T::E];
        T::unpack(ra[c], a);
        T::unpack(rb[c], b);
        const float keep = ok[c] ? 1.0f : 0.0f;
#pragma unroll
        for (int j = 0; j < T::E; ++j) {
            const float dl = (a[j] - b[j]) - shift;
            const float eb = keep * fast_exp2(fmaf(b[j], kLog2e, -mbl));
            const float ead = keep * fast_exp2(fmaf(a[j], kLog2e, -mal));
            const float em = expm1_small(dl);
            const bool small = fabsf(dl) < kSmall;
            const float qe = small ? eb * em : ead - eb;
            const float ea = small ? fmaf(eb, em, eb) : ead;
            zb += eb;
            za += ea;
            sqe += qe;
            spd = fmaf(ea, dl, spd);
        }
    }
    float sums[4] = {zb, za, sqe, spd};
    row_reduce<TPR, 4, false>(sums, red);
    if (live && tr == 0) out[row] = drift_finish(sums[0], sums[1], sums[2], sums[3]);
}

// chunks per row -> (threads per row, chunks per thread); false above 2048
// chunks (d above 16384 in bf16 / 8192 in fp32)
inline bool drift_config(int chunks, int& tpr, int& nch) {
    static const int cfg[6][3] = {{64, 64, 1}, {128, 64, 2}, {256, 128, 2}, {512, 256, 2}, {1024, 256, 4}, {2048, 256, 8}};
    for (const auto& c : cfg)
        if (chunks <= c[0]) {
            tpr = c[1];
            nch = c[2];
            return true;
        }
    return false;
}

}  // namespace
}  // namespace ps
