// The cached hidden-state residual codec (Sec. 4.1 "Cluster and Quantize
// Hidden States"; App. C quantization format; App. D format ablation), in the
// OCP microscaling formats MI355X supports: MXFP4 (E2M1 values) and MXFP8
// (E4M3 values), one E8M0 power-of-two scale per 32 channels.
//
//   polestar_cluster_means  per cluster, the mean of its window members' rows
//   polestar_codec_encode   rows -> residual to their cluster's mean -> codes
//   polestar_codec_gather   codes of listed rows -> mean + decoded residual
//                           (fp32) and, fused, the rows' RMSNorm (dtype): the
//                           dequantisation folded into the gather that starts
//                           a packet's forward
//
// Rounding is done in software from the format definitions (exponent from the
// float's bits, rintf for ties-to-even, explicit saturation), so the codes
// are exactly those of the definition.
#include "common.hpp"
#include "host_common.hpp"

namespace ps {
namespace {

constexpr int kCodecBlock = 32;                 // channels per scale
constexpr int kCbThreads = 256;

// Element formats: exponent bits, mantissa bits, bias, scale emax, largest code.
template <int FMT> struct Fmt;
template <> struct Fmt<POLESTAR_MXFP4> {
    static constexpr int EB = 2, MB = 1, BIAS = 1, EMAX = 2, MAXCODE = 0x7, BITS = 4;
    static constexpr float VMAX = 6.0f;
};
template <> struct Fmt<POLESTAR_MXFP8> {
    static constexpr int EB = 4, MB = 3, BIAS = 7, EMAX = 8, MAXCODE = 0x7E, BITS = 8;
    static constexpr float VMAX = 448.0f;
};

// floor(log2 a) of a positive finite float, from its bits (subnormals too).
__device__ __forceinline__ int floor_log2(float a) {
    int e;
    (void)frexpf(a, &e);                        // a = f 2^e, 0.5 <= f < 1
    return e - 1;
}

// |v| rounded to the element grid, ties to even, saturated; returns the code
// with the sign bit (no negative zero).
template <int FMT>
__device__ __forceinline__ uint32_t quantize(float v) {
    using F = Fmt<FMT>;
    const float a = fabsf(v);
    uint32_t code;
    if (a >= F::VMAX) {
        code = F::MAXCODE;
    } else {
        const int emin = 1 - F::BIAS;                         // exponent of the smallest normal
        const int e = a > 0.f ? floor_log2(a) : emin - 1;     // zero takes the subnormal path (code 0)
        if (e < emin) {                                       // subnormal: multiples of 2^(emin - MB)
            code = static_cast<uint32_t>(rintf(ldexpf(a, F::MB - emin)));   // q = 2^MB is the smallest normal
        } else {
            const float m = ldexpf(a, -e);                    // [1, 2)
            uint32_t q = static_cast<uint32_t>(rintf((m - 1.f) * (1 << F::MB)));
            int ee = e;
            if (q == (1u << F::MB)) { q = 0; ++ee; }
            code = (static_cast<uint32_t>(ee + F::BIAS) << F::MB) | q;
            code = code > F::MAXCODE ? F::MAXCODE : code;
        }
    }
    const uint32_t sign = (v < 0.f && code != 0) ? (1u << (F::EB + F::MB)) : 0u;
    return code | sign;
}

template <int FMT>
__device__ __forceinline__ float dequantize(uint32_t code) {
    using F = Fmt<FMT>;
    const uint32_t mag = code & ((1u << (F::EB + F::MB)) - 1);
    const int e = static_cast<int>(mag >> F::MB);
    const int m = static_cast<int>(mag & ((1u << F::MB) - 1));
    const float v = e == 0 ? ldexpf(static_cast<float>(m), 1 - F::BIAS - F::MB)
                           : ldexpf(1.f + static_cast<float>(m) / (1 << F::MB), e - F::BIAS);
    return (code >> (F::EB + F::MB)) & 1 ? -v : v;
}

// means[b][k] = mean over the window members of cluster k of x rows; thread
// per channel quad, members summed in window order.  grid (quads / 256, b)
__global__ __launch_bounds__(kCbThreads) void cluster_means_kernel(const float* __restrict__ x, int seq, int d,
                                                                   const int32_t* __restrict__ win, int n_win,
                                                                   const int32_t* __restrict__ labels, int K,
                                                                   float* __restrict__ means) {
    constexpr int kMaxK = 16;
    const int b = blockIdx.y;
    const int c = 4 * (blockIdx.x * kCbThreads + threadIdx.x);
    if (c >= d) return;
    float4 acc[kMaxK];
    int cnt[kMaxK];
#pragma unroll
    for (int k = 0; k < kMaxK; ++k) { acc[k] = make_float4(0.f, 0.f, 0.f, 0.f); cnt[k] = 0; }
    const int32_t* wb = win + static_cast<size_t>(b) * n_win;
    for (int i0 = 0; i0 < n_win; i0 += 8) {
        float4 v[8];
        int lab[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int p = min(max(wb[min(i0 + u, n_win - 1)], 0), seq - 1);
            lab[u] = i0 + u < n_win ? labels[static_cast<size_t>(b) * seq + p] : -1;
            v[u] = *reinterpret_cast<const float4*>(x + (static_cast<size_t>(b) * seq + p) * d + c);
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
#pragma unroll
            for (int k = 0; k < kMaxK; ++k) {
                const float f = lab[u] == k ? 1.f : 0.f;
                acc[k].x = fmaf(v[u].x, f, acc[k].x);
                acc[k].y = fmaf(v[u].y, f, acc[k].y);
                acc[k].z = fmaf(v[u].z, f, acc[k].z);
                acc[k].w = fmaf(v[u].w, f, acc[k].w);
                cnt[k] += lab[u] == k;
            }
        }
    }
#pragma unroll
    for (int k = 0; k < kMaxK; ++k) {
        if (k < K) {
            const float inv = cnt[k] > 0 ? 1.f / static_cast<float>(cnt[k]) : 0.f;
            *reinterpret_cast<float4*>(means + (static_cast<size_t>(b) * K + k) * d + c) =
                make_float4(acc[k].x * inv, acc[k].y * inv, acc[k].z * inv, acc[k].w * inv);
        }
    }
}

// One thread per 32-channel block of a listed row: residual to the row's
// cluster mean (fp32), block exponent, codes.  grid (k_max, b)
template <int FMT>
__global__ __launch_bounds__(kCbThreads) void encode_kernel(const float* __restrict__ x, int seq, int d,
                                                            const int32_t* __restrict__ idx,
                                                            const int32_t* __restrict__ count, int k_max,
                                                            const int32_t* __restrict__ labels, int K,
                                                            const float* __restrict__ means,
                                                            uint8_t* __restrict__ codes, uint8_t* __restrict__ scales) {
    using F = Fmt<FMT>;
    const int r = blockIdx.x, b = blockIdx.y;
    const int cnt = min(max(count[b], 0), k_max);
    if (r >= cnt) return;
    const int p = idx[static_cast<size_t>(b) * k_max + r];
    if (p < 0 || p >= seq) return;
    const int lab = labels[static_cast<size_t>(b) * seq + p];
    const float* xr = x + (static_cast<size_t>(b) * seq + p) * d;
    const float* mr = (lab >= 0 && lab < K) ? means + (static_cast<size_t>(b) * K + lab) * d : nullptr;
    const size_t row_code_bytes = static_cast<size_t>(d) * F::BITS / 8;
    uint8_t* cr = codes + (static_cast<size_t>(b) * seq + p) * row_code_bytes;
    uint8_t* sr = scales + (static_cast<size_t>(b) * seq + p) * (d / kCodecBlock);
    for (int blk = threadIdx.x; blk < d / kCodecBlock; blk += kCbThreads) {
        float rv[kCodecBlock];
        float amax = 0.f;
#pragma unroll
        for (int q = 0; q < kCodecBlock / 4; ++q) {
            const float4 xv = *reinterpret_cast<const float4*>(xr + blk * kCodecBlock + 4 * q);
            const float4 mv = mr ? *reinterpret_cast<const float4*>(mr + blk * kCodecBlock + 4 * q)
                                 : make_float4(0.f, 0.f, 0.f, 0.f);
            rv[4 * q] = xv.x - mv.x;
            rv[4 * q + 1] = xv.y - mv.y;
            rv[4 * q + 2] = xv.z - mv.z;
            rv[4 * q + 3] = xv.w - mv.w;
        }
#pragma unroll
        for (int i = 0; i < kCodecBlock; ++i) amax = fmaxf(amax, fabsf(rv[i]));
        const int e = amax > 0.f ? max(floor_log2(amax) - F::EMAX, -127) : -127;
        sr[blk] = static_cast<uint8_t>(e + 127);
        uint32_t c[kCodecBlock];
#pragma unroll
        for (int i = 0; i < kCodecBlock; ++i) c[i] = quantize<FMT>(ldexpf(rv[i], -e));
        if constexpr (F::BITS == 4) {
            uint32_t w[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                w[j] = 0;
#pragma unroll
                for (int i = 0; i < 8; ++i) w[j] |= (c[8 * j + i] & 0xFu) << (4 * i);
            }
            *reinterpret_cast<uint4*>(cr + blk * 16) = make_uint4(w[0], w[1], w[2], w[3]);
        } else {
            uint32_t w[8];
#pragma unroll
            for (int j = 0; j < 8; ++j)
                w[j] = c[4 * j] | (c[4 * j + 1] << 8) | (c[4 * j + 2] << 16) | (c[4 * j + 3] << 24);
            *reinterpret_cast<uint4*>(cr + blk * 32) = make_uint4(w[0], w[1], w[2], w[3]);
            *reinterpret_cast<uint4*>(cr + blk * 32 + 16) = make_uint4(w[4], w[5], w[6], w[7]);
        }
    }
}

// Row r < count[b] of the list: x_out = mean + decoded residual (fp32) and,
// if h_out, RMSNorm of it in dtype; rows past the count: zeros.  One
// workgroup per row, 4 channels per thread and pass, PER passes.
template <int FMT, bool BF16, int PER>
__global__ __launch_bounds__(kCbThreads) void gather_kernel(const uint8_t* __restrict__ codes,
                                                            const uint8_t* __restrict__ scales, int seq, int d,
                                                            const int32_t* __restrict__ idx,
                                                            const int32_t* __restrict__ count, int k_max,
                                                            const int32_t* __restrict__ labels, int K,
                                                            const float* __restrict__ means, float eps,
                                                            float* __restrict__ x_out, char* __restrict__ h_out) {
    using F = Fmt<FMT>;
    constexpr int ES = Elem<BF16>::kBytes;
    __shared__ float red[kCbThreads / kWave];
    const int r = blockIdx.x, b = blockIdx.y;
    const int cnt = min(max(count[b], 0), k_max);
    const int p0 = r < cnt ? idx[static_cast<size_t>(b) * k_max + r] : -1;
    const bool ok = p0 >= 0 && p0 < seq;
    const int p = ok ? p0 : 0;
    const int lab = ok ? labels[static_cast<size_t>(b) * seq + p] : -1;
    const float* mr = (lab >= 0 && lab < K) ? means + (static_cast<size_t>(b) * K + lab) * d : nullptr;
    const size_t row_code_bytes = static_cast<size_t>(d) * F::BITS / 8;
    const uint8_t* cr = codes + (static_cast<size_t>(b) * seq + p) * row_code_bytes;
    const uint8_t* sr = scales + (static_cast<size_t>(b) * seq + p) * (d / kCodecBlock);
    float4 v[PER];
    float ss = 0.f;
#pragma unroll
    for (int u = 0; u < PER; ++u) {
        const int c = 4 * (threadIdx.x + u * kCbThreads);
        float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
        if (ok && c < d) {
            const float sc = ldexpf(1.f, static_cast<int>(sr[c / kCodecBlock]) - 127);
            uint32_t q[4];
            if constexpr (F::BITS == 4) {
                const uint32_t w = *reinterpret_cast<const uint16_t*>(cr + c / 2);
#pragma unroll
                for (int i = 0; i < 4; ++i) q[i] = (w >> (4 * i)) & 0xFu;
            } else {
                const uint32_t w = *reinterpret_cast<const uint32_t*>(cr + c);
#pragma unroll
                for (int i = 0; i < 4; ++i) q[i] = (w >> (8 * i)) & 0xFFu;
            }
            const float4 mv = mr ? *reinterpret_cast<const float4*>(mr + c) : make_float4(0.f, 0.f, 0.f, 0.f);
            o = make_float4(mv.x + dequantize<FMT>(q[0]) * sc, mv.y + dequantize<FMT>(q[1]) * sc,
                            mv.z + dequantize<FMT>(q[2]) * sc, mv.w + dequantize<FMT>(q[3]) * sc);
        }
        v[u] = o;
        ss = fmaf(o.x, o.x, fmaf(o.y, o.y, fmaf(o.z, o.z, fmaf(o.w, o.w, ss))));
        if (c < d) *reinterpret_cast<float4*>(x_out + (static_cast<size_t>(b) * k_max + r) * d + c) = o;
    }
    if (h_out == nullptr) return;                       // uniform
    ss = wave_sum(ss);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
    __syncthreads();
    float tot = 0.f;
#pragma unroll
    for (int w = 0; w < kCbThreads / kWave; ++w) tot += red[w];
    const float s = 1.0f / sqrtf(tot / static_cast<float>(d) + eps);
    char* hr = h_out + (static_cast<size_t>(b) * k_max + r) * d * ES;
#pragma unroll
    for (int u = 0; u < PER; ++u) {
        const int c = 4 * (threadIdx.x + u * kCbThreads);
        if (c < d) {
            const float4 o = make_float4(v[u].x * s, v[u].y * s, v[u].z * s, v[u].w * s);
            if constexpr (BF16)
                *reinterpret_cast<uint2*>(hr + 2 * c) = make_uint2(pack_bf16x2(o.x, o.y), pack_bf16x2(o.z, o.w));
            else
                *reinterpret_cast<float4*>(hr + 4 * c) = o;
        }
    }
}

bool fmt_ok(int fmt) { return fmt == POLESTAR_MXFP4 || fmt == POLESTAR_MXFP8; }

}  // namespace
}  // namespace ps

extern "C" size_t polestar_codec_row_bytes(int fmt, int d) {
    using namespace ps;
    if (!fmt_ok(fmt) || d <= 0 || d % kCodecBlock) return 0;
    return static_cast<size_t>(d) * (fmt == POLESTAR_MXFP4 ? 4 : 8) / 8;
}

extern "C" polestar_status polestar_cluster_means(int batch, int seq, int d, const float* x, const int32_t* win_idx,
                                                  int n_win, const int32_t* labels, int n_clusters, float* means,
                                                  hipStream_t stream) {
    using namespace ps;
    if (batch <= 0 || seq <= 0 || d <= 0 || n_win <= 0 || n_clusters <= 0 || !x || !win_idx || !labels || !means)
        return POLESTAR_ERR_INVALID_ARGUMENT;
    if (n_clusters > 16 || d % 4 || !aligned16(x) || !aligned16(means) || batch > 65535)
        return POLESTAR_ERR_UNSUPPORTED;
    hipLaunchKernelGGL(cluster_means_kernel, dim3(ceil_div(d / 4, kCbThreads), batch), dim3(kCbThreads), 0, stream,
                       x, seq, d, win_idx, n_win, labels, n_clusters, means);
    return launch_status();
}

extern "C" polestar_status polestar_codec_encode(int fmt, int batch, int seq, int d, const float* x,
                                                 const int32_t* idx, const int32_t* count, int k_max,
                                                 const int32_t* labels, int n_clusters, const float* means,
                                                 uint8_t* codes, uint8_t* scales, hipStream_t stream) {
    using namespace ps;
    if (!fmt_ok(fmt) || batch <= 0 || seq <= 0 || d <= 0 || k_max < 0 || n_clusters <= 0 || !x || !labels ||
        !means || !codes || !scales || (k_max > 0 && (!idx || !count)))
        return POLESTAR_ERR_INVALID_ARGUMENT;
    if (d % kCodecBlock || !aligned16(x) || !aligned16(means) || !aligned16(codes) || batch > 65535)
        return POLESTAR_ERR_UNSUPPORTED;
    if (k_max == 0) return POLESTAR_OK;
    const dim3 grid(k_max, batch);
    if (fmt == POLESTAR_MXFP4)
        hipLaunchKernelGGL((encode_kernel<POLESTAR_MXFP4>), grid, dim3(kCbThreads), 0, stream, x, seq, d, idx, count,
                           k_max, labels, n_clusters, means, codes, scales);
    else
        hipLaunchKernelGGL((encode_kernel<POLESTAR_MXFP8>), grid, dim3(kCbThreads), 0, stream, x, seq, d, idx, count,
                           k_max, labels, n_clusters, means, codes, scales);
    return launch_status();
}

extern "C" polestar_status polestar_codec_gather(int fmt, polestar_dtype dtype, int batch, int seq, int d,
                                                 const uint8_t* codes, const uint8_t* scales, const int32_t* idx,
                                                 const int32_t* count, int k_max, const int32_t* labels,
                                                 int n_clusters, const float* means, float eps, float* x_out,
                                                 void* h_out, hipStream_t stream) {
    using namespace ps;
    if (!fmt_ok(fmt) || !dtype_ok(dtype) || batch <= 0 || seq <= 0 || d <= 0 || k_max < 0 || n_clusters <= 0 ||
        !(eps >= 0.f) || (k_max > 0 && (!codes || !scales || !idx || !count || !labels || !means || !x_out)))
        return POLESTAR_ERR_INVALID_ARGUMENT;
    if (d % kCodecBlock || d > 4 * kCbThreads * 16 || !aligned16(means) || !aligned16(x_out) || !aligned16(h_out) ||
        !aligned16(codes) || batch > 65535)
        return POLESTAR_ERR_UNSUPPORTED;
    if (k_max == 0) return POLESTAR_OK;
    const dim3 grid(k_max, batch);
    const int per = ceil_div(d, 4 * kCbThreads);
    char* h = static_cast<char*>(h_out);
#define PS_GATHER(F, BF, P)                                                                                        \
    hipLaunchKernelGGL((gather_kernel<F, BF, P>), grid, dim3(kCbThreads), 0, stream, codes, scales, seq, d, idx,   \
                       count, k_max, labels, n_clusters, means, eps, x_out, h)
#define PS_GATHER_P(F, BF) \
    if (per <= 4) PS_GATHER(F, BF, 4); else if (per <= 8) PS_GATHER(F, BF, 8); else PS_GATHER(F, BF, 16)
    const bool bf16 = dtype == POLESTAR_BF16;
    if (fmt == POLESTAR_MXFP4) { if (bf16) { PS_GATHER_P(POLESTAR_MXFP4, true); } else { PS_GATHER_P(POLESTAR_MXFP4, false); } }
    else { if (bf16) { PS_GATHER_P(POLESTAR_MXFP8, true); } else { PS_GATHER_P(POLESTAR_MXFP8, false); } }
#undef PS_GATHER_P
#undef PS_GATHER
    return launch_status();
}
