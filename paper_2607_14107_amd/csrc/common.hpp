// Shared device helpers of the Polestar gfx950 kernels: element types,
// bf16 conversion, 16-byte memory access, wavefront (64-lane) reductions and
// MFMA wrappers.  Host-side argument checks live in host_common.hpp.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ps {

constexpr int kWave = 64;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

// --- element types ---------------------------------------------------------

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// fp32 -> bf16, round to nearest, ties to even (NaN -> quiet NaN).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0u;
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return f32_to_bf16_bits(lo) | (f32_to_bf16_bits(hi) << 16);
}

// Two finite floats to packed bf16 in one v_cvt_pk_bf16_f32 (round to nearest
// even, the same bits as pack_bf16x2 for every non-NaN input; NaN keeps its
// sign and payload instead of becoming 0x7fc0).
typedef __bf16 bf16x2_hw __attribute__((ext_vector_type(2)));
typedef float float2_hw __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t cvt_pk_bf16(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((float2_hw){lo, hi}, bf16x2_hw));
}

// Storage traits: E = element count of one 16-byte chunk.
template <bool BF16> struct Elem;
template <> struct Elem<true> {
    static constexpr int kBytes = 2;
    static constexpr int E = 8;
    __device__ __forceinline__ static void unpack(const uint4& v, float* f) {
        f[0] = bf16_lo(v.x); f[1] = bf16_hi(v.x);
        f[2] = bf16_lo(v.y); f[3] = bf16_hi(v.y);
        f[4] = bf16_lo(v.z); f[5] = bf16_hi(v.z);
        f[6] = bf16_lo(v.w); f[7] = bf16_hi(v.w);
    }
};
template <> struct Elem<false> {
    static constexpr int kBytes = 4;
    static constexpr int E = 4;
    __device__ __forceinline__ static void unpack(const uint4& v, float* f) {
        f[0] = __uint_as_float(v.x); f[1] = __uint_as_float(v.y);
        f[2] = __uint_as_float(v.z); f[3] = __uint_as_float(v.w);
    }
};

// --- 16-byte memory access ---------------------------------------------------

__device__ __forceinline__ uint4 ld16(const void* p) {
    return *reinterpret_cast<const uint4*>(p);
}
// A 16-byte load of data read once per call (weights of a single row tile,
// previous hidden states, logits): marked non-temporal so that the stream
// does not push the caches and the rows the step reuses out of L2 and the
// Infinity Cache.
typedef unsigned int u32x4_nt __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ld16_nt(const void* p) {
    return __builtin_bit_cast(uint4, __builtin_nontemporal_load(reinterpret_cast<const u32x4_nt*>(p)));
}
__device__ __forceinline__ void st16(void* p, const uint4& v) {
    *reinterpret_cast<uint4*>(p) = v;
}
__device__ __forceinline__ uint4 zero16() { return make_uint4(0u, 0u, 0u, 0u); }

// --- wavefront reductions (all 64 lanes take part) ---------------------------

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
    return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}
__device__ __forceinline__ int wave_sum_i(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

// Inclusive prefix sum over the 64 lanes.
__device__ __forceinline__ int wave_incl_scan(int v, int lane) {
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        int t = __shfl_up(v, o);
        if (lane >= o) v += t;
    }
    return v;
}

// Exclusive prefix sum over the whole block (blockDim.x a multiple of 64,
// at most 1024 threads).  `scratch` holds >= 17 ints of shared memory.
// Returns the exclusive prefix; *total receives the block sum.
__device__ __forceinline__ int block_excl_scan(int v, int* scratch, int* total) {
    const int lane = threadIdx.x & 63;
    const int wid = threadIdx.x >> 6;
    const int nw = blockDim.x >> 6;
    int incl = wave_incl_scan(v, lane);
    if (lane == 63) scratch[wid] = incl;
    __syncthreads();
    if (wid == 0) {
        int w = lane < nw ? scratch[lane] : 0;
        int wi = wave_incl_scan(w, lane);
        if (lane < nw) scratch[lane] = wi - w;
        if (lane == nw - 1) scratch[16] = wi;
    }
    __syncthreads();
    int res = scratch[wid] + incl - v;
    *total = scratch[16];
    __syncthreads();
    return res;
}

// --- MFMA ------------------------------------------------------------------
// 16x16 output tiles.  For both operands lane l carries index (l % 16) of the
// non-reduced dimension and k-group (l / 16); the result lane l holds
// C[4*(l/16) + i][l % 16], i = 0..3.  Callers only rely on A and B using the
// same lane -> k assignment, so the order of k inside an instruction is free.

__device__ __forceinline__ floatx4 mfma_bf16(const uint4& a, const uint4& b, floatx4 c) {
    bf16x8 av = __builtin_bit_cast(bf16x8, a);
    bf16x8 bv = __builtin_bit_cast(bf16x8, b);
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, c, 0, 0, 0);
}

__device__ __forceinline__ floatx4 mfma_f32(float a, float b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// One 16-byte slice of A and of B per lane: 32 bf16 k-values (one MFMA) or
// 4 fp32 k-values (four MFMAs), accumulated into c.
template <bool BF16> struct Mma;
template <> struct Mma<true> {
    __device__ __forceinline__ static floatx4 step(const uint4& a, const uint4& b, floatx4 c) {
        return mfma_bf16(a, b, c);
    }
};
template <> struct Mma<false> {
    __device__ __forceinline__ static floatx4 step(const uint4& a, const uint4& b, floatx4 c) {
        c = mfma_f32(__uint_as_float(a.x), __uint_as_float(b.x), c);
        c = mfma_f32(__uint_as_float(a.y), __uint_as_float(b.y), c);
        c = mfma_f32(__uint_as_float(a.z), __uint_as_float(b.z), c);
        c = mfma_f32(__uint_as_float(a.w), __uint_as_float(b.w), c);
        return c;
    }
};

// 32x32 output tiles (twice the flops per issue slot of 16x16x32 on gfx950).
// Lane l carries index (l % 32) of the non-reduced dimension and k-group
// (l / 32); result register j of lane l holds
// C[8*(j/4) + 4*(l/32) + (j%4)][l % 32].
typedef float floatx16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ int mfma32_row(int lane, int j) { return 8 * (j >> 2) + 4 * (lane >> 5) + (j & 3); }

template <bool BF16> struct Mma32;
template <> struct Mma32<true> {
    __device__ __forceinline__ static floatx16 step(const uint4& a, const uint4& b, floatx16 c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                      __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    }
};
template <> struct Mma32<false> {
    __device__ __forceinline__ static floatx16 step(const uint4& a, const uint4& b, floatx16 c) {
        c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
        return c;
    }
};

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

}  // namespace ps
