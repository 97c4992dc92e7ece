// The rest of a pre-norm layer stack around the hot path, so that the
// denoising loop of Alg. 1 can run on a whole model: token + position
// embedding, RMSNorm, dense row projections (the shared MFMA GEMM), the SwiGLU
// product, the fp32 residual add, and the copy of refreshed rows into the
// cached hidden states.  All are HBM-bound row kernels except the projection.
#include "common.hpp"
#include "gemm.hpp"
#include "host_common.hpp"

namespace ps {
namespace {

constexpr int kRowBlock = 256;

// Four consecutive elements of a dtype row as fp32 (8-byte bf16 / 16-byte fp32).
template <bool BF16>
__device__ __forceinline__ float4 ld4(const char* row, long c) {
    if constexpr (BF16) {
        const uint2 v = *reinterpret_cast<const uint2*>(row + 2 * c);
        return make_float4(bf16_lo(v.x), bf16_hi(v.x), bf16_lo(v.y), bf16_hi(v.y));
    } else {
        return *reinterpret_cast<const float4*>(row + 4 * c);
    }
}

template <bool BF16>
__device__ __forceinline__ void st4(char* row, long c, float4 v) {
    if constexpr (BF16) {
        *reinterpret_cast<uint2*>(row + 2 * c) = make_uint2(pack_bf16x2(v.x, v.y), pack_bf16x2(v.z, v.w));
    } else {
        *reinterpret_cast<float4*>(row + 4 * c) = v;
    }
}

// x[b][r][:] = tok[ids[b][lo + r]][:] + pos[lo + r][:]   (fp32 out); grid (n_rows, batch)
template <bool BF16>
__global__ __launch_bounds__(kRowBlock) void embed_kernel(const int32_t* __restrict__ ids, int seq, int lo,
                                                          int n_rows, int d, const char* __restrict__ tok,
                                                          int vocab, const char* __restrict__ pos,
                                                          float* __restrict__ x) {
    constexpr int ES = Elem<BF16>::kBytes;
    const int r = blockIdx.x, b = blockIdx.y;
    const int p = lo + r;
    const int id = min(max(ids[static_cast<size_t>(b) * seq + p], 0), vocab - 1);
    const char* tr = tok + static_cast<size_t>(id) * d * ES;
    const char* pr = pos + static_cast<size_t>(p) * d * ES;
    float* xr = x + (static_cast<size_t>(b) * n_rows + r) * d;
    for (int c = 4 * threadIdx.x; c < d; c += 4 * kRowBlock) {
        const float4 a = ld4<BF16>(tr, c), e = ld4<BF16>(pr, c);
        *reinterpret_cast<float4*>(xr + c) = make_float4(a.x + e.x, a.y + e.y, a.z + e.z, a.w + e.w);
    }
}

// out[b][out_start + r] = x[b][x_start + r] / sqrt(mean(x^2) + eps), rounded
// to dtype; the row is read once into registers.  grid (n_rows, batch)
template <bool BF16, int PER>
__global__ __launch_bounds__(kRowBlock) void rmsnorm_kernel(const float* __restrict__ x, int x_seq, int x_start,
                                                            int d, float eps, char* __restrict__ out,
                                                            int out_seq, int out_start) {
    constexpr int ES = Elem<BF16>::kBytes;
    __shared__ float red[kRowBlock / kWave];
    const int r = blockIdx.x, b = blockIdx.y;
    const float* xr = x + (static_cast<size_t>(b) * x_seq + x_start + r) * d;
    char* orow = out + (static_cast<size_t>(b) * out_seq + out_start + r) * d * ES;
    float4 v[PER];
    float s = 0.f;
#pragma unroll
    for (int u = 0; u < PER; ++u) {
        const int c = 4 * (threadIdx.x + u * kRowBlock);
        v[u] = c < d ? *reinterpret_cast<const float4*>(xr + c) : make_float4(0.f, 0.f, 0.f, 0.f);
        s = fmaf(v[u].x, v[u].x, s);
        s = fmaf(v[u].y, v[u].y, s);
        s = fmaf(v[u].z, v[u].z, s);
        s = fmaf(v[u].w, v[u].w, s);
    }
    s = wave_sum(s);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
    __syncthreads();
    float tot = 0.f;
#pragma unroll
    for (int w = 0; w < kRowBlock / kWave; ++w) tot += red[w];
    const float sc = 1.0f / sqrtf(tot / static_cast<float>(d) + eps);
#pragma unroll
    for (int u = 0; u < PER; ++u) {
        const int c = 4 * (threadIdx.x + u * kRowBlock);
        if (c < d) st4<BF16>(orow, c, make_float4(v[u].x * sc, v[u].y * sc, v[u].z * sc, v[u].w * sc));
    }
}

// x[i] += y[i] (fp32 += dtype), four elements per thread
template <bool BF16>
__global__ __launch_bounds__(kRowBlock) void residual_add_kernel(float* __restrict__ x, const char* __restrict__ y,
                                                                 long n4) {
    for (long i = static_cast<long>(blockIdx.x) * kRowBlock + threadIdx.x; i < n4;
         i += static_cast<long>(gridDim.x) * kRowBlock) {
        float4 a = reinterpret_cast<float4*>(x)[i];
        const float4 e = ld4<BF16>(y, 4 * i);
        a.x += e.x; a.y += e.y; a.z += e.z; a.w += e.w;
        reinterpret_cast<float4*>(x)[i] = a;
    }
}

// a[r][f] = silu(gu[r][f]) * gu[r][F + f], rounded to dtype
template <bool BF16>
__global__ __launch_bounds__(kRowBlock) void swiglu_kernel(const char* __restrict__ gu, int F,
                                                           char* __restrict__ out, long rows) {
    constexpr int ES = Elem<BF16>::kBytes;
    const long n4 = rows * (F / 4);
    for (long i = static_cast<long>(blockIdx.x) * kRowBlock + threadIdx.x; i < n4;
         i += static_cast<long>(gridDim.x) * kRowBlock) {
        const long r = i / (F / 4);
        const long c = 4 * (i - r * (F / 4));
        const char* row = gu + r * 2 * F * ES;
        const float4 g = ld4<BF16>(row, c), u = ld4<BF16>(row, F + c);
        const float4 o = make_float4(g.x / (1.f + expf(-g.x)) * u.x, g.y / (1.f + expf(-g.y)) * u.y,
                                     g.z / (1.f + expf(-g.z)) * u.z, g.w / (1.f + expf(-g.w)) * u.w);
        st4<BF16>(out + r * F * ES, c, o);
    }
}

// dst[b][p] = src[b][p] for the first stale_count[b] entries p of
// stale_idx[b] and for p in the block; grid (k_max + block_len, batch)
__global__ __launch_bounds__(kRowBlock) void copy_rows_kernel(const char* __restrict__ src, char* __restrict__ dst,
                                                              int seq, int row_bytes,
                                                              const int32_t* __restrict__ stale_idx,
                                                              const int32_t* __restrict__ stale_count, int k_max,
                                                              int block_start, int block_len) {
    const int r = blockIdx.x, b = blockIdx.y;
    const int cnt = stale_count ? min(max(stale_count[b], 0), k_max) : 0;
    int p;
    if (r < cnt) p = stale_idx[static_cast<size_t>(b) * k_max + r];
    else if (r - cnt < block_len) p = block_start + (r - cnt);
    else return;
    if (p < 0 || p >= seq) return;
    const size_t off = (static_cast<size_t>(b) * seq + p) * row_bytes;
    for (int c = 16 * threadIdx.x; c < row_bytes; c += 16 * kRowBlock)
        st16(dst + off + c, ld16(src + off + c));
}

// dst[b][r] = src[b][idx[b][r]] for r < count[b] (entries outside [0, seq)
// give zero rows), zero rows for r in [count[b], k_max); grid (k_max, batch)
__global__ __launch_bounds__(kRowBlock) void gather_rows_kernel(const char* __restrict__ src, char* __restrict__ dst,
                                                                int seq, int row_bytes, const int32_t* __restrict__ idx,
                                                                const int32_t* __restrict__ count, int k_max) {
    const int r = blockIdx.x, b = blockIdx.y;
    const int cnt = min(max(count[b], 0), k_max);
    const int p = r < cnt ? idx[static_cast<size_t>(b) * k_max + r] : -1;
    const bool ok = p >= 0 && p < seq;
    const char* s = src + (static_cast<size_t>(b) * seq + (ok ? p : 0)) * row_bytes;
    char* d = dst + (static_cast<size_t>(b) * k_max + r) * row_bytes;
    for (int c = 16 * threadIdx.x; c < row_bytes; c += 16 * kRowBlock)
        st16(d + c, ok ? ld16(s + c) : make_uint4(0u, 0u, 0u, 0u));
}

// dst[b][idx[b][r]] = src[b][r] for r < count[b] (entries outside [0, seq)
// skipped); grid (k_max, batch)
__global__ __launch_bounds__(kRowBlock) void scatter_rows_kernel(const char* __restrict__ src, char* __restrict__ dst,
                                                                 int seq, int row_bytes, const int32_t* __restrict__ idx,
                                                                 const int32_t* __restrict__ count, int k_max) {
    const int r = blockIdx.x, b = blockIdx.y;
    const int cnt = min(max(count[b], 0), k_max);
    if (r >= cnt) return;
    const int p = idx[static_cast<size_t>(b) * k_max + r];
    if (p < 0 || p >= seq) return;
    const char* s = src + (static_cast<size_t>(b) * k_max + r) * row_bytes;
    char* d = dst + (static_cast<size_t>(b) * seq + p) * row_bytes;
    for (int c = 16 * threadIdx.x; c < row_bytes; c += 16 * kRowBlock) st16(d + c, ld16(s + c));
}

int grid_for(long n4) {
    const long g = (n4 + kRowBlock - 1) / kRowBlock;
    return static_cast<int>(g < 8192 ? (g > 0 ? g : 1) : 8192);
}

}  // namespace
}  // namespace ps

extern "C" polestar_status polestar_embed(polestar_dtype dtype, int batch, int seq, int d, const int32_t* ids,
                                          int lo, int n_rows, const void* tok_emb, int vocab,
                                          const void* pos_emb, float* x, hipStream_t stream) {
    using namespace ps;
    if (!dtype_ok(dtype) || batch <= 0 || seq <= 0 || d <= 0 || vocab <= 0 || n_rows <= 0 || lo < 0 ||
        lo > seq - n_rows || !ids || !tok_emb || !pos_emb || !x)
        return POLESTAR_ERR_INVALID_ARGUMENT;
    if (d % 4 != 0 || !aligned16(x) || !aligned16(tok_emb) || !aligned16(pos_emb) || batch > 65535 ||
        n_rows > 0x7fffffff)
        return POLESTAR_ERR_UNSUPPORTED;
    const dim3 grid(n_rows, batch);
    if (dtype == POLESTAR_BF16)
        hipLaunchKernelGGL((embed_kernel<true>), grid, dim3(kRowBlock), 0, stream, ids, seq, lo, n_rows, d,
                           static_cast<const char*>(tok_emb), vocab, static_cast<const char*>(pos_emb), x);
    else
        hipLaunchKernelGGL((embed_kernel<false>), grid, dim3(kRowBlock), 0, stream, ids, seq, lo, n_rows, d,
                           static_cast<const char*>(tok_emb), vocab, static_cast<const char*>(pos_emb), x);
    return launch_status();
}

extern "C" polestar_status polestar_rmsnorm(polestar_dtype dtype, int batch, int n_rows, int d, const float* x,
                                            int x_seq, int x_start, float eps, void* out, int out_seq,
                                            int out_start, hipStream_t stream) {
    using namespace ps;
    if (!dtype_ok(dtype) || batch <= 0 || n_rows <= 0 || d <= 0 || !x || !out || !(eps >= 0.f) ||
        x_start < 0 || x_start > x_seq - n_rows || out_start < 0 || out_start > out_seq - n_rows)
        return POLESTAR_ERR_INVALID_ARGUMENT;
    if (d % 4 != 0 || d > 4 * kRowBlock * 16 || !aligned16(x) || !aligned16(out) || batch > 65535)
        return POLESTAR_ERR_UNSUPPORTED;
    const dim3 grid(n_rows, batch);
    const int per = ceil_div(d, 4 * kRowBlock);
    char* o = static_cast<char*>(out);
#define PS_NORM(BF, P)                                                                                    \
    hipLaunchKernelGGL((rmsnorm_kernel<BF, P>), grid, dim3(kRowBlock), 0, stream, x, x_seq, x_start, d, eps, \
                       o, out_seq, out_start)
    const bool bf16 = dtype == POLESTAR_BF16;
    if (per <= 4) { if (bf16) PS_NORM(true, 4); else PS_NORM(false, 4); }
    else if (per <= 8) { if (bf16) PS_NORM(true, 8); else PS_NORM(false, 8); }
    else { if (bf16) PS_NORM(true, 16); else PS_NORM(false, 16); }
#undef PS_NORM
    return launch_status();
}

extern "C" polestar_status polestar_residual_add(polestar_dtype dtype, long n, float* x, const void* y,
                                                 hipStream_t stream) {
    using namespace ps;
    if (!dtype_ok(dtype) || n < 0 || (n > 0 && (!x || !y))) return POLESTAR_ERR_INVALID_ARGUMENT;
    if (n % 4 != 0 || !aligned16(x) || !aligned16(y)) return POLESTAR_ERR_UNSUPPORTED;
    if (n == 0) return POLESTAR_OK;
    const long n4 = n / 4;
    if (dtype == POLESTAR_BF16)
        hipLaunchKernelGGL((residual_add_kernel<true>), dim3(grid_for(n4)), dim3(kRowBlock), 0, stream, x,
                           static_cast<const char*>(y), n4);
    else
        hipLaunchKernelGGL((residual_add_kernel<false>), dim3(grid_for(n4)), dim3(kRowBlock), 0, stream, x,
                           static_cast<const char*>(y), n4);
    return launch_status();
}

extern "C" polestar_status polestar_swiglu(polestar_dtype dtype, long rows, int ffn, const void* gate_up,
                                           void* out, hipStream_t stream) {
    using namespace ps;
    if (!dtype_ok(dtype) || rows < 0 || ffn <= 0 || (rows > 0 && (!gate_up || !out)))
        return POLESTAR_ERR_INVALID_ARGUMENT;
    if (ffn % 4 != 0 || !aligned16(gate_up) || !aligned16(out)) return POLESTAR_ERR_UNSUPPORTED;
    if (rows == 0) return POLESTAR_OK;
    const long n4 = rows * (ffn / 4);
    if (dtype == POLESTAR_BF16)
        hipLaunchKernelGGL((swiglu_kernel<true>), dim3(grid_for(n4)), dim3(kRowBlock), 0, stream,
                           static_cast<const char*>(gate_up), ffn, static_cast<char*>(out), rows);
    else
        hipLaunchKernelGGL((swiglu_kernel<false>), dim3(grid_for(n4)), dim3(kRowBlock), 0, stream,
                           static_cast<const char*>(gate_up), ffn, static_cast<char*>(out), rows);
    return launch_status();
}

extern "C" polestar_status polestar_copy_rows(polestar_dtype dtype, int batch, int seq, int d, const void* src,
                                              void* dst, const int32_t* stale_idx, const int32_t* stale_count,
                                              int k_max, int block_start, int block_len, hipStream_t stream) {
    using namespace ps;
    if (!dtype_ok(dtype) || batch <= 0 || seq <= 0 || d <= 0 || k_max < 0 || block_len < 0 ||
        block_start < 0 || block_start > seq - block_len || !src || !dst ||
        (k_max > 0 && (!stale_idx || !stale_count)))
        return POLESTAR_ERR_INVALID_ARGUMENT;
    const int es = dtype == POLESTAR_BF16 ? 2 : 4;
    if ((static_cast<long>(d) * es) % 16 != 0 || !aligned16(src) || !aligned16(dst) || batch > 65535)
        return POLESTAR_ERR_UNSUPPORTED;
    if (k_max + block_len == 0) return POLESTAR_OK;
    hipLaunchKernelGGL(copy_rows_kernel, dim3(k_max + block_len, batch), dim3(kRowBlock), 0, stream,
                       static_cast<const char*>(src), static_cast<char*>(dst), seq, d * es,
                       k_max > 0 ? stale_idx : nullptr, k_max > 0 ? stale_count : nullptr, k_max, block_start,
                       block_len);
    return launch_status();
}

extern "C" size_t polestar_linear_workspace_size(polestar_dtype dtype, int batch, int n_rows, int n_out,
                                                 int n_in) {
    using namespace ps;
    if (!dtype_ok(dtype) || batch <= 0 || n_rows <= 0 || n_out <= 0 || n_in <= 0) return 0;
    return gemm_plan(dtype == POLESTAR_BF16, static_cast<long>(batch) * n_rows, n_out, n_in).ws_bytes;
}

extern "C" polestar_status polestar_linear(polestar_dtype dtype, int batch, int seq, int n_in, int n_out,
                                           int row_start, int n_rows, const void* x, const void* w, void* y,
                                           void* workspace, size_t workspace_bytes, hipStream_t stream) {
    using namespace ps;
    if (!dtype_ok(dtype) || batch <= 0 || seq <= 0 || n_in <= 0 || n_out <= 0 || n_rows <= 0 ||
        row_start < 0 || row_start > seq - n_rows || !x || !w || !y)
        return POLESTAR_ERR_INVALID_ARGUMENT;
    const bool bf16 = dtype == POLESTAR_BF16;
    if (!gemm_k_ok(bf16, n_in) || n_out % 16 != 0 || !aligned16(x) || !aligned16(w) || !aligned16(y) ||
        !aligned16(workspace) || batch > 65535 || static_cast<long>(batch) * n_rows > 0x7fffffffL / 4)
        return POLESTAR_ERR_UNSUPPORTED;
    const GemmPlan plan = gemm_plan(bf16, static_cast<long>(batch) * n_rows, n_out, n_in);
    if (workspace_bytes < plan.ws_bytes || (plan.ws_bytes > 0 && !workspace)) return POLESTAR_ERR_WORKSPACE;
    GemmArgs g{};
    g.x = static_cast<const char*>(x);
    g.w0 = static_cast<const char*>(w);
    g.w1 = nullptr;
    g.n0 = n_out;
    g.N = n_out;
    g.K = n_in;
    g.mode = kGemmBlockRows;
    g.batch = batch;
    g.seq = seq;
    g.block_start = row_start;
    g.block_len = n_rows;
    g.out0 = static_cast<char*>(y);
    g.ws = static_cast<float*>(workspace);
    g.m_max = batch * n_rows;
    return gemm_run(bf16, plan, g, stream);
}

extern "C" polestar_status polestar_gather_rows(int batch, int seq, int row_bytes, const void* src,
                                                const int32_t* idx, const int32_t* count, int k_max, void* dst,
                                                hipStream_t stream) {
    using namespace ps;
    if (batch <= 0 || seq <= 0 || row_bytes <= 0 || k_max < 0 || (k_max > 0 && (!src || !idx || !count || !dst)))
        return POLESTAR_ERR_INVALID_ARGUMENT;
    if (row_bytes % 16 != 0 || !aligned16(src) || !aligned16(dst) || batch > 65535) return POLESTAR_ERR_UNSUPPORTED;
    if (k_max == 0) return POLESTAR_OK;
    hipLaunchKernelGGL(gather_rows_kernel, dim3(k_max, batch), dim3(kRowBlock), 0, stream,
                       static_cast<const char*>(src), static_cast<char*>(dst), seq, row_bytes, idx, count, k_max);
    return launch_status();
}

extern "C" polestar_status polestar_scatter_rows(int batch, int seq, int row_bytes, const void* src,
                                                 const int32_t* idx, const int32_t* count, int k_max, void* dst,
                                                 hipStream_t stream) {
    using namespace ps;
    if (batch <= 0 || seq <= 0 || row_bytes <= 0 || k_max < 0 || (k_max > 0 && (!src || !idx || !count || !dst)))
        return POLESTAR_ERR_INVALID_ARGUMENT;
    if (row_bytes % 16 != 0 || !aligned16(src) || !aligned16(dst) || batch > 65535) return POLESTAR_ERR_UNSUPPORTED;
    if (k_max == 0) return POLESTAR_OK;
    hipLaunchKernelGGL(scatter_rows_kernel, dim3(k_max, batch), dim3(kRowBlock), 0, stream,
                       static_cast<const char*>(src), static_cast<char*>(dst), seq, row_bytes, idx, count, k_max);
    return launch_status();
}
