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
constexpr float kSmall = 0.125f;               // |dl| below this: expm1 from its series
constexpr float kNear = 16.0f;                 // row maxima closer than this: one reference
constexpr uint32_t kNeutral = 0xF149F149u;     // -1e30 in both bf16 halves (and as fp32): masked chunks

// expm1 for |x| < 1/8 from its Taylor series to x^5/120; the first omitted
// term x^6/720 is below 4.3e-8 relative there.
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

// One row of d elements per TPR threads (64, 128 or 256); each thread keeps
// NCH 16-byte chunks of both rows in registers.
// Rows of a workgroup: kDriftBlock / TPR.
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
    // then set to -1e30 in both rows (no share of either maximum, zero
    // exponentials, dl = 0 or the row shift: nothing added to any sum).
    uint4 ra[NCH], rb[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        const int ch = c * TPR + tr;
        const size_t off = base + static_cast<size_t>(ch < chunks ? ch : 0) * 16;
        ra[c] = ld16_nt(hc + off);   // both rows are read once per call
        rb[c] = ld16_nt(hp + off);
    }
    __builtin_amdgcn_sched_barrier(0);    // every load in flight before any use
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        if (c * TPR + tr >= chunks) {
            ra[c] = make_uint4(kNeutral, kNeutral, kNeutral, kNeutral);
            rb[c] = ra[c];
        }
    }

    // Pass 1: the maximum of each row (ma of the current, mb of the previous).
    float mx[2] = {-INFINITY, -INFINITY};
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        float a[T::E], b[T::E];
        T::unpack(ra[c], a);
        T::unpack(rb[c], b);
#pragma unroll
        for (int j = 0; j < T::E; ++j) {
            mx[0] = fmaxf(mx[0], a[j]);
            mx[1] = fmaxf(mx[1], b[j]);
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

    // Pass 2: the four sums.  A chunk whose elements all move by less than
    // 1/8 (every chunk of a lightly perturbed row) takes one exponential per
    // element, ea = eb (1 + expm1(dl)); otherwise both exponentials are
    // taken directly, and ea - eb still comes from the series where |dl| is
    // small.
    float zb = 0.0f, za = 0.0f, sqe = 0.0f, spd = 0.0f;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        float a[T::E], b[T::E], dl[T::E], eb[T::E];
        T::unpack(ra[c], a);
        T::unpack(rb[c], b);
        bool big = false;
#pragma unroll
        for (int j = 0; j < T::E; ++j) {
            dl[j] = (a[j] - b[j]) - shift;
            big |= !(fabsf(dl[j]) < kSmall);
            eb[j] = fast_exp2(fmaf(b[j], kLog2e, -mbl));
        }
        if (!big) {
#pragma unroll
            for (int j = 0; j < T::E; ++j) {
                const float em = expm1_small(dl[j]);
                const float ea = fmaf(eb[j], em, eb[j]);
                sqe = fmaf(eb[j], em, sqe);
                zb += eb[j];
                za += ea;
                spd = fmaf(ea, dl[j], spd);
            }
        } else {
#pragma unroll
            for (int j = 0; j < T::E; ++j) {
                const float ead = fast_exp2(fmaf(a[j], kLog2e, -mal));
                const float qs = eb[j] * expm1_small(dl[j]);
                const float qe = fabsf(dl[j]) < kSmall ? qs : ead - eb[j];
                sqe += qe;
                zb += eb[j];
                za += ead;
                spd = fmaf(ead, dl[j], spd);
            }
        }
    }
    float sums[4] = {zb, za, sqe, spd};
    row_reduce<TPR, 4, false>(sums, red);
    if (live && tr == 0) out[row] = drift_finish(sums[0], sums[1], sums[2], sums[3]);
}

// (chunks per row, rows) -> (threads per row, chunks per thread).  With at
// least 2048 rows: 128 threads per row of up to 8 chunks each (two rows per
// workgroup) up to 1024 chunks (d = 8192 bf16); one wave per row with as many
// chunks per lane as d needs ran 2-7 us slower on the batch-8 and Dream-7B
// layer steps, because the fused launch that also runs the vocabulary scan
// takes the register count of its largest role (149 registers for 7 chunks
// per lane against 87 for 4).  Fewer rows (or longer ones): 256 threads per
// row, so that a batch-1 layer still spreads over every compute unit.
// False above 2048 chunks (d above 16384 in bf16 / 8192 in fp32).
// PS_DRIFT_SHAPES lists the shapes this can return, for the launch tables.
inline bool drift_config(int chunks, long rows, int& tpr, int& nch) {
    if (chunks <= 0 || chunks > 2048) return false;
    if (rows >= 2048 && chunks <= 1024) {
        tpr = 128;
        const int need = (chunks + 127) / 128;
        nch = need <= 4 ? need : 8;
    } else {
        tpr = 256;
        const int need = (chunks + 255) / 256;
        nch = need <= 1 ? 1 : need <= 2 ? 2 : need <= 4 ? 4 : 8;
    }
    return true;
}
#define PS_DRIFT_SHAPES(X) X(128, 1) X(128, 2) X(128, 3) X(128, 4) X(128, 8) \
    X(256, 1) X(256, 2) X(256, 4) X(256, 8)

}  // namespace
}  // namespace ps
