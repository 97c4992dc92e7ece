// Gather -> MFMA GEMM -> scatter, the core of the sparse K/V refresh
// (Sec. 4.1: re-project the stale rows and the active block; Corollary 1 of
// App. B: K = W_K h, V = W_V h) and of the Q projection of the active block.
//
// The product is skinny: a few hundred gathered rows times a [N][K] weight
// read once from HBM.  A workgroup (4 waves) owns BM = 16*MT rows and 128
// output columns, wave w the columns 32w..32w+31 (two 16x16 MFMA tiles).
// Per super-step of 256 bytes of K:
//  - the gathered input rows are staged through LDS (16-byte coalesced loads,
//    row pitch padded to 272 bytes so the MFMA reads are bank-conflict free)
//    and shared by the four waves;
//  - each wave streams its weight rows straight from HBM into registers,
//    64 contiguous bytes per lane, two super-steps ahead;
//  - one MFMA step consumes a 16-byte slice of A and B per lane.  A and B
//    use the same lane -> k assignment, so k may be visited in any order.
// When the row x column tiles alone do not fill the chip, K is split over
// workgroups; fp32 partials go to the workspace and a second kernel sums
// them in split order (deterministic), rounds and scatters 16-byte rows.
#include "common.hpp"
#include "gemm.hpp"
#include "host_common.hpp"

namespace ps {
namespace {

constexpr int kGemmBlock = 256;
constexpr int kBN = 128;          // columns per workgroup
constexpr int kLda = 272;         // LDS row pitch (bytes) of the staged input rows
constexpr int kTargetWgs = 256;   // one workgroup per compute unit on MI355X

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

template <bool BF16, int MT>
__global__ __launch_bounds__(kGemmBlock) void gemm_kernel(GemmArgs g) {
    using T = Elem<BF16>;
    constexpr int BM = MT * 16;
    constexpr int ES = T::kBytes;
    constexpr int KS = 256 / ES;      // k elements per super-step
    __shared__ __align__(16) char sa[2][BM * kLda];
    __shared__ int rowb[BM], rowp[BM];
    __shared__ int scan_tmp[17];
    extern __shared__ int pre[];      // batch + 1 (refresh mode)

    const int t = threadIdx.x;
    const int lane = t & 63;
    const int w = t >> 6;
    const int m0 = blockIdx.y * BM;
    const int total = g.mode == kGemmRefresh ? build_prefix(g, pre, scan_tmp)
                                             : g.batch * g.block_len;
    if (m0 >= total) return;          // uniform over the workgroup
    if (t < BM) {
        int b, pos;
        map_row(g, pre, total, m0 + t, b, pos);
        rowb[t] = b;
        rowp[t] = pos;
    }
    __syncthreads();

    // Input rows this thread stages: r = t/16 + 16 i, 16 bytes at acol.
    const char* arow[MT];
#pragma unroll
    for (int i = 0; i < MT; ++i) {
        const int r = (t >> 4) + 16 * i;
        const int b = rowb[r];
        arow[i] = b >= 0 ? g.x + (static_cast<size_t>(b) * g.seq + rowp[r]) * g.K * ES : nullptr;
    }
    const int acol = (t & 15) * 16;

    // Weight rows this lane streams: two 16-column tiles of wave w.
    const int col0 = blockIdx.x * kBN + w * 32;
    const char* brow[2];
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
        const int n = col0 + nt * 16 + (lane & 15);
        brow[nt] = n >= g.N ? nullptr
                 : n < g.n0 ? g.w0 + static_cast<size_t>(n) * g.K * ES
                            : g.w1 + static_cast<size_t>(n - g.n0) * g.K * ES;
    }
    const int bcol = (lane >> 4) * 64;

    const int nsteps = (g.K + KS - 1) / KS;
    const int s0 = blockIdx.z * g.steps_per_split;
    const int s1 = min(nsteps, s0 + g.steps_per_split);

    floatx4 acc[MT][2];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

    auto load_a = [&](int step, uint4 (&ra)[MT]) {
        const int kb = step * 256 + acol;
        const bool kin = kb / ES < g.K;
#pragma unroll
        for (int i = 0; i < MT; ++i) ra[i] = (arow[i] && kin) ? ld16(arow[i] + kb) : zero16();
    };
    auto store_a = [&](int buf, const uint4 (&ra)[MT]) {
#pragma unroll
        for (int i = 0; i < MT; ++i) st16(&sa[buf][((t >> 4) + 16 * i) * kLda + acol], ra[i]);
    };
    auto load_b = [&](int step, uint4 (&rb)[2][4]) {
#pragma unroll
        for (int nt = 0; nt < 2; ++nt)
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const int kb = step * 256 + bcol + 16 * s;
                rb[nt][s] = (brow[nt] && kb / ES < g.K) ? ld16(brow[nt] + kb) : zero16();
            }
    };

    uint4 b0[2][4], b1[2][4];
    {
        uint4 ra[MT];
        load_a(s0, ra);
        load_b(s0, b0);
        if (s0 + 1 < s1) load_b(s0 + 1, b1);
        store_a(0, ra);
    }
    __syncthreads();

    for (int step = s0; step < s1; ++step) {
        const int buf = (step - s0) & 1;
        uint4 ra[MT];
        uint4 b2[2][4];
        if (step + 1 < s1) load_a(step + 1, ra);
        if (step + 2 < s1) load_b(step + 2, b2);
        const char* abase = &sa[buf][(lane & 15) * kLda + (lane >> 4) * 64];
#pragma unroll
        for (int s = 0; s < 4; ++s) {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const uint4 a = *reinterpret_cast<const uint4*>(abase + mt * 16 * kLda + 16 * s);
#pragma unroll
                for (int nt = 0; nt < 2; ++nt)
                    acc[mt][nt] = Mma<BF16>::step(a, b0[nt][s], acc[mt][nt]);
            }
        }
        if (step + 1 < s1) store_a(buf ^ 1, ra);
        __syncthreads();
#pragma unroll
        for (int nt = 0; nt < 2; ++nt)
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                b0[nt][s] = b1[nt][s];
                b1[nt][s] = b2[nt][s];
            }
    }

    // Epilogue: lane holds rows mt*16 + 4*(lane/16) + i of column n.
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
            const int n = col0 + nt * 16 + (lane & 15);
            if (n >= g.N) continue;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int r = mt * 16 + 4 * (lane >> 4) + i;
                const int b = rowb[r];
                if (b < 0) continue;
                const float v = acc[mt][nt][i];
                if (g.ksplit == 1)
                    store_elem<BF16>(out_ptr<BF16>(g, b, rowp[r], m0 + r, n), v);
                else
                    g.ws[(static_cast<size_t>(blockIdx.z) * g.m_max + (m0 + r)) * g.N + n] = v;
            }
        }
}

// Sum of the split-K partials of one output row per workgroup, rounded and
// written with 16-byte stores (8 consecutive columns per thread).
template <bool BF16>
__global__ __launch_bounds__(kGemmBlock) void gemm_reduce_kernel(GemmArgs g) {
    __shared__ int scan_tmp[17];
    __shared__ int rowinfo[2];
    extern __shared__ int pre[];
    const int m = blockIdx.x;
    const int total = g.mode == kGemmRefresh ? build_prefix(g, pre, scan_tmp)
                                             : g.batch * g.block_len;
    if (m >= total) return;
    if (threadIdx.x == 0) {
        int b, pos;
        map_row(g, pre, total, m, b, pos);
        rowinfo[0] = b;
        rowinfo[1] = pos;
    }
    __syncthreads();
    const int b = rowinfo[0], pos = rowinfo[1];
    if (b < 0) return;
    const size_t split_stride = static_cast<size_t>(g.m_max) * g.N;
    for (int c = threadIdx.x; c < g.N / 8; c += blockDim.x) {
        const int n = c * 8;
        const float* src = g.ws + static_cast<size_t>(m) * g.N + n;
        float v[8];
        {
            const float4 x0 = *reinterpret_cast<const float4*>(src);
            const float4 x1 = *reinterpret_cast<const float4*>(src + 4);
            v[0] = x0.x; v[1] = x0.y; v[2] = x0.z; v[3] = x0.w;
            v[4] = x1.x; v[5] = x1.y; v[6] = x1.z; v[7] = x1.w;
        }
        for (int s = 1; s < g.ksplit; ++s) {
            const float4 x0 = *reinterpret_cast<const float4*>(src + s * split_stride);
            const float4 x1 = *reinterpret_cast<const float4*>(src + s * split_stride + 4);
            v[0] += x0.x; v[1] += x0.y; v[2] += x0.z; v[3] += x0.w;
            v[4] += x1.x; v[5] += x1.y; v[6] += x1.z; v[7] += x1.w;
        }
        char* dst = out_ptr<BF16>(g, b, pos, m, n);
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
}

template <bool BF16, int MT>
void launch_gemm(const GemmPlan& p, const GemmArgs& g, size_t dyn, hipStream_t s) {
    dim3 grid(p.col_tiles, p.row_tiles, p.ksplit);
    hipLaunchKernelGGL((gemm_kernel<BF16, MT>), grid, dim3(kGemmBlock), dyn, s, g);
}

template <bool BF16>
bool dispatch_gemm(const GemmPlan& p, const GemmArgs& g, size_t dyn, hipStream_t s) {
    switch (p.mt) {
        case 1: launch_gemm<BF16, 1>(p, g, dyn, s); return true;
        case 2: launch_gemm<BF16, 2>(p, g, dyn, s); return true;
        case 3: launch_gemm<BF16, 3>(p, g, dyn, s); return true;
        case 4: launch_gemm<BF16, 4>(p, g, dyn, s); return true;
        case 5: launch_gemm<BF16, 5>(p, g, dyn, s); return true;
        case 6: launch_gemm<BF16, 6>(p, g, dyn, s); return true;
        case 7: launch_gemm<BF16, 7>(p, g, dyn, s); return true;
        case 8: launch_gemm<BF16, 8>(p, g, dyn, s); return true;
        case 9: launch_gemm<BF16, 9>(p, g, dyn, s); return true;
        case 10: launch_gemm<BF16, 10>(p, g, dyn, s); return true;
        case 11: launch_gemm<BF16, 11>(p, g, dyn, s); return true;
        case 12: launch_gemm<BF16, 12>(p, g, dyn, s); return true;
        case 13: launch_gemm<BF16, 13>(p, g, dyn, s); return true;
        case 14: launch_gemm<BF16, 14>(p, g, dyn, s); return true;
        case 15: launch_gemm<BF16, 15>(p, g, dyn, s); return true;
        case 16: launch_gemm<BF16, 16>(p, g, dyn, s); return true;
        default: return false;
    }
}

}  // namespace

GemmPlan gemm_plan(bool bf16, long m_max, int N, int K) {
    GemmPlan p{};
    const int ks = bf16 ? 128 : 64;
    const int nsteps = ceil_div(K, ks);
    if (m_max <= 0) m_max = 1;
    p.row_tiles = ceil_div(m_max, 256);
    p.mt = ceil_div(m_max, 16L * p.row_tiles);
    p.col_tiles = ceil_div(N, kBN);
    const long wgs = static_cast<long>(p.row_tiles) * p.col_tiles;
    int ksplit = 1;
    if (wgs < kTargetWgs) ksplit = ceil_div(kTargetWgs, wgs);
    if (ksplit > 8) ksplit = 8;
    if (ksplit > nsteps) ksplit = nsteps;
    p.steps_per_split = ceil_div(nsteps, ksplit);
    p.ksplit = ceil_div(nsteps, p.steps_per_split);
    p.ws_bytes = p.ksplit > 1 ? static_cast<size_t>(p.ksplit) * m_max * N * sizeof(float) : 0;
    return p;
}

polestar_status gemm_run(bool bf16, const GemmPlan& p, GemmArgs g, hipStream_t stream) {
    g.ksplit = p.ksplit;
    g.steps_per_split = p.steps_per_split;
    const size_t dyn = g.mode == kGemmRefresh ? (static_cast<size_t>(g.batch) + 1) * sizeof(int) : 0;
    const bool ok = bf16 ? dispatch_gemm<true>(p, g, dyn, stream)
                         : dispatch_gemm<false>(p, g, dyn, stream);
    if (!ok) return POLESTAR_ERR_UNSUPPORTED;
    polestar_status st = launch_status();
    if (st != POLESTAR_OK || p.ksplit == 1) return st;
    if (bf16)
        hipLaunchKernelGGL((gemm_reduce_kernel<true>), dim3(g.m_max), dim3(kGemmBlock), dyn, stream, g);
    else
        hipLaunchKernelGGL((gemm_reduce_kernel<false>), dim3(g.m_max), dim3(kGemmBlock), dyn, stream, g);
    return launch_status();
}

}  // namespace ps

extern "C" size_t polestar_refresh_kv_workspace_size(polestar_dtype dtype, int batch, int d,
                                                     int n_kv_heads, int head_dim, int k_max,
                                                     int block_len) {
    using namespace ps;
    if (!dtype_ok(dtype) || batch <= 0 || d <= 0 || n_kv_heads <= 0 || head_dim <= 0 ||
        k_max < 0 || block_len < 0)
        return 0;
    const long m_max = static_cast<long>(batch) * (k_max + block_len);
    const int N = 2 * n_kv_heads * head_dim;
    return gemm_plan(dtype == POLESTAR_BF16, m_max, N, d).ws_bytes;
}

extern "C" polestar_status polestar_refresh_kv(polestar_dtype dtype, int batch, int seq, int d,
                                               int n_kv_heads, int head_dim, const void* h_cur,
                                               const int32_t* stale_idx,
                                               const int32_t* stale_count, int k_max,
                                               int block_start, int block_len, const void* w_k,
                                               const void* w_v, void* k_cache, void* v_cache,
                                               void* workspace, size_t workspace_bytes,
                                               hipStream_t stream) {
    using namespace ps;
    if (!dtype_ok(dtype) || batch <= 0 || seq <= 0 || d <= 0 || n_kv_heads <= 0 ||
        head_dim <= 0 || k_max < 0 || k_max > seq || block_start < 0 || block_len < 0 ||
        block_start > seq - block_len || !h_cur || !w_k || !w_v || !k_cache || !v_cache ||
        (k_max > 0 && (!stale_idx || !stale_count)))
        return POLESTAR_ERR_INVALID_ARGUMENT;
    if ((head_dim != 64 && head_dim != 128) || !row_ok(dtype, d) || !aligned16(h_cur) ||
        !aligned16(w_k) || !aligned16(w_v) || !aligned16(k_cache) || !aligned16(v_cache) ||
        !aligned16(workspace))
        return POLESTAR_ERR_UNSUPPORTED;
    if (batch > 65536) return POLESTAR_ERR_UNSUPPORTED;
    const long m_max = static_cast<long>(batch) * (k_max + block_len);
    if (m_max == 0) return POLESTAR_OK;
    if (m_max > 0x7fffffffL / 4) return POLESTAR_ERR_UNSUPPORTED;
    const bool bf16 = dtype == POLESTAR_BF16;
    const int kvd = n_kv_heads * head_dim;
    const GemmPlan p = gemm_plan(bf16, m_max, 2 * kvd, d);
    if (workspace_bytes < p.ws_bytes || (p.ws_bytes > 0 && !workspace)) return POLESTAR_ERR_WORKSPACE;
    GemmArgs g{};
    g.x = static_cast<const char*>(h_cur);
    g.w0 = static_cast<const char*>(w_k);
    g.w1 = static_cast<const char*>(w_v);
    g.n0 = kvd;
    g.N = 2 * kvd;
    g.K = d;
    g.mode = kGemmRefresh;
    g.batch = batch;
    g.seq = seq;
    g.stale_idx = k_max > 0 ? stale_idx : nullptr;
    g.stale_count = k_max > 0 ? stale_count : nullptr;
    g.k_max = k_max;
    g.block_start = block_start;
    g.block_len = block_len;
    g.out0 = static_cast<char*>(k_cache);
    g.out1 = static_cast<char*>(v_cache);
    g.ws = static_cast<float*>(workspace);
    g.m_max = static_cast<int>(m_max);
    return gemm_run(bf16, p, g, stream);
}
