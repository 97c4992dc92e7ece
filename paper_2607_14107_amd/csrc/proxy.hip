// Clustered proxy drift, Polestar's own drift estimator (Sec. 4.1 "Cluster
// and Quantize Hidden States", "Measuring Drift and Layer-wise KV Updates";
// Alg. 1 block entry and per-layer loop):
//
//   polestar_cluster         spherical K-means of the local window's hidden
//                            states at block entry -> labels, cluster sums,
//                            counts, unit centroids
//   polestar_proxy_drift     per step: proxy token per cluster (members'
//                            mean) -> query (shared skinny GEMM) -> scores
//                            over the whole cache -> KL against the previous
//                            step's scores, averaged over heads
//   polestar_cluster_select  top-k clusters -> their window positions,
//                            ascending (the rows polestar_refresh_kv takes)
//   polestar_cluster_update  after the refresh: cluster sums move by the
//                            refreshed rows' change
//
// The per-step work is small (K proxy queries): a token kernel, the GEMM
// (W_q read once), a score kernel reading K once, and a KL kernel over the
// scores.  The K-means runs once per block, one workgroup per sequence with
// the centroids held in LDS.
#include "common.hpp"
#include "gemm.hpp"
#include "host_common.hpp"

namespace ps {
namespace {

constexpr int kKmBlock = 1024;               // K-means: 16 waves per sequence
constexpr int kKmWaves = kKmBlock / kWave;
constexpr int kMaxClusters = 16;
constexpr int kMaxWin = 2048;                // window positions per sequence
constexpr int kMaxCentroidFloats = 32768;    // K * d held in LDS (128 KB)
constexpr int kChunkGroup = 8;               // 16-byte chunks per lane loaded together in the K-means

template <bool BF16>
__device__ __forceinline__ float load_elem(const char* row, int c) {
    if constexpr (BF16) return bf16_to_f32(reinterpret_cast<const uint16_t*>(row)[c]);
    else return reinterpret_cast<const float*>(row)[c];
}

// ---------------------------------------------------------------------------
// polestar_cluster: one workgroup per sequence.
//   1. inverse norm of every window point (one wave per point);
//   2. centroid j starts at the point of window rank floor(j*n/K);
//   3. `iters` rounds: assignment (one wave per point, K dot products with
//      the LDS centroids, largest cosine, lowest cluster on ties), then each
//      centroid = normalised sum of its members' directions, accumulated in
//      point order (thread per channel: deterministic); empty clusters keep
//      their centroid;
//   4. a final assignment to the final centroids, then the raw sums and
//      counts of those clusters and the labels scattered by position (-1
//      outside the window).
// ---------------------------------------------------------------------------

// Four consecutive channels of a row as fp32 (8-byte bf16 / 16-byte fp32 load).
template <bool BF16>
__device__ __forceinline__ float4 load4(const char* row, int c) {
    if constexpr (BF16) {
        const uint2 v = *reinterpret_cast<const uint2*>(row + 2 * c);
        return make_float4(bf16_lo(v.x), bf16_hi(v.x), bf16_lo(v.y), bf16_hi(v.y));
    } else {
        return *reinterpret_cast<const float4*>(row + 4 * c);
    }
}

// Per-cluster sums over the window of one channel quad, points in order:
// acc[k] += direction (or raw state) of every member of cluster k.  Loads
// of sixteen points are issued before any of them is used.
template <bool BF16, bool UNIT>
__device__ __forceinline__ void quad_sums(const char* hb, const int32_t* wi, int seq, int n_win, int d, int c,
                                          const float* inv_norm, const int* lab, float4 (&acc)[kMaxClusters]) {
    constexpr int ES = Elem<BF16>::kBytes;
#pragma unroll
    for (int k = 0; k < kMaxClusters; ++k) acc[k] = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int i0 = 0; i0 < n_win; i0 += 16) {
        float4 v[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) {
            const int i = min(i0 + u, n_win - 1);
            const int p = min(max(wi[i], 0), seq - 1);
            v[u] = load4<BF16>(hb + static_cast<size_t>(p) * d * ES, c);
        }
#pragma unroll
        for (int u = 0; u < 16; ++u) {
            const int i = i0 + u;
            if (i >= n_win) break;
            const float f = UNIT ? inv_norm[i] : 1.f;
            const int li = lab[i];
#pragma unroll
            for (int k = 0; k < kMaxClusters; ++k) {
                const float sel = li == k ? f : 0.f;
                acc[k].x = fmaf(v[u].x, sel, acc[k].x);
                acc[k].y = fmaf(v[u].y, sel, acc[k].y);
                acc[k].z = fmaf(v[u].z, sel, acc[k].z);
                acc[k].w = fmaf(v[u].w, sel, acc[k].w);
            }
        }
    }
}

template <bool BF16>
__global__ __launch_bounds__(kKmBlock) void kmeans_kernel(const char* __restrict__ h, int seq, int d,
                                                          const int32_t* __restrict__ win_idx, int n_win,
                                                          int K, int iters, int32_t* __restrict__ labels_out,
                                                          float* __restrict__ sums, int32_t* __restrict__ counts,
                                                          float* __restrict__ centroids) {
    extern __shared__ float zs[];               // [K][d] unit centroids
    __shared__ float inv_norm[kMaxWin];
    __shared__ int lab[kMaxWin];
    __shared__ float red[kKmWaves][kMaxClusters];
    __shared__ int cnt_s[kMaxClusters];
    using T = Elem<BF16>;
    constexpr int ES = T::kBytes;
    constexpr int E = T::E;                     // channels per 16-byte chunk
    const int b = blockIdx.x;
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    const char* hb = h + static_cast<size_t>(b) * seq * d * ES;
    const int32_t* wi = win_idx + static_cast<size_t>(b) * n_win;
    // window entries are clamped into [0, seq): a bad index cannot leave the rows
    auto pos = [&](int i) { return min(max(wi[i], 0), seq - 1); };
    auto row = [&](int i) { return hb + static_cast<size_t>(pos(i)) * d * ES; };
    const int nch = d / (kWave * E);            // 16-byte chunks per lane of a row (d % (64 E) == 0)
    float* zg = centroids + static_cast<size_t>(b) * K * d;

    // kChunkGroup 16-byte chunks of a point's row per lane, starting at
    // chunk q0, loaded together (chunks past nch re-read the last one; the
    // callers skip them).
    auto load_group = [&](int i, int q0, uint4 (&raw)[kChunkGroup]) {
        const char* r = row(i);
#pragma unroll
        for (int u = 0; u < kChunkGroup; ++u)
            raw[u] = ld16(r + static_cast<size_t>(lane + kWave * min(q0 + u, nch - 1)) * 16);
    };

    // 1. inverse norms: wave per point
    for (int i = w; i < n_win; i += kKmWaves) {
        float s = 0.f;
        for (int q0 = 0; q0 < nch; q0 += kChunkGroup) {
            uint4 raw[kChunkGroup];
            load_group(i, q0, raw);
#pragma unroll
            for (int u = 0; u < kChunkGroup; ++u) {
                float f[E];
                T::unpack(raw[u], f);
                const float m = q0 + u < nch ? 1.f : 0.f;
#pragma unroll
                for (int e = 0; e < E; ++e) s = fmaf(f[e] * m, f[e], s);
            }
        }
        s = wave_sum(s);
        if (lane == 0) inv_norm[i] = s > 0.f ? 1.0f / sqrtf(s) : 0.f;
    }
    __syncthreads();
    // 2. start points: thread per channel quad, every cluster's start row
    // loaded together
    for (int c = 4 * t; c < d; c += 4 * kKmBlock) {
        float4 v[kMaxClusters];
#pragma unroll
        for (int k = 0; k < kMaxClusters; ++k) {
            const int i = static_cast<int>((static_cast<long>(min(k, K - 1)) * n_win) / K);
            v[k] = load4<BF16>(row(i), c);
        }
#pragma unroll
        for (int k = 0; k < kMaxClusters; ++k) {
            if (k < K) {
                const float f = inv_norm[static_cast<int>((static_cast<long>(k) * n_win) / K)];
                const float4 z = make_float4(v[k].x * f, v[k].y * f, v[k].z * f, v[k].w * f);
                *reinterpret_cast<float4*>(zs + k * d + c) = z;
                *reinterpret_cast<float4*>(zg + k * d + c) = z;   // previous-round copy
            }
        }
    }
    __syncthreads();

    for (int it = 0; it <= iters; ++it) {
        // assignment: wave per point, lane chunks of E channels, K dot products
        for (int i = w; i < n_win; i += kKmWaves) {
            float dot[kMaxClusters];
#pragma unroll
            for (int k = 0; k < kMaxClusters; ++k) dot[k] = 0.f;
            for (int q0 = 0; q0 < nch; q0 += kChunkGroup) {
                uint4 raw[kChunkGroup];
                load_group(i, q0, raw);
#pragma unroll
                for (int u = 0; u < kChunkGroup; ++u) {
                    if (q0 + u < nch) {
                        const int c0 = (lane + kWave * (q0 + u)) * E;
                        float f[E];
                        T::unpack(raw[u], f);
#pragma unroll
                        for (int k = 0; k < kMaxClusters; ++k) {
                            if (k < K) {
                                const float4* zk = reinterpret_cast<const float4*>(zs + k * d + c0);
#pragma unroll
                                for (int e4 = 0; e4 < E / 4; ++e4) {
                                    const float4 z4 = zk[e4];
                                    dot[k] = fmaf(f[4 * e4], z4.x, dot[k]);
                                    dot[k] = fmaf(f[4 * e4 + 1], z4.y, dot[k]);
                                    dot[k] = fmaf(f[4 * e4 + 2], z4.z, dot[k]);
                                    dot[k] = fmaf(f[4 * e4 + 3], z4.w, dot[k]);
                                }
                            }
                        }
                    }
                }
            }
            int best = 0;
            float bv = -INFINITY;
#pragma unroll
            for (int k = 0; k < kMaxClusters; ++k) {
                if (k < K) {
                    const float sdot = wave_sum(dot[k]) * inv_norm[i];
                    if (sdot > bv) { bv = sdot; best = k; }   // strict: lowest cluster on ties
                }
            }
            if (lane == 0) lab[i] = best;
        }
        __syncthreads();
        if (it == iters) break;                       // the last round only assigns
        // update: thread per channel quad, members' directions summed in point order
        for (int c = 4 * t; c < d; c += 4 * kKmBlock) {
            float4 acc[kMaxClusters];
            quad_sums<BF16, true>(hb, wi, seq, n_win, d, c, inv_norm, lab, acc);
#pragma unroll
            for (int k = 0; k < kMaxClusters; ++k)
                if (k < K) *reinterpret_cast<float4*>(zs + k * d + c) = acc[k];   // unnormalised for now
        }
        __syncthreads();
        // norms of the new sums; clusters with no member keep the old centroid
        float part[kMaxClusters];
#pragma unroll
        for (int k = 0; k < kMaxClusters; ++k) part[k] = 0.f;
        for (int c = t; c < d; c += kKmBlock) {
#pragma unroll
            for (int k = 0; k < kMaxClusters; ++k)
                if (k < K) part[k] = fmaf(zs[k * d + c], zs[k * d + c], part[k]);
        }
#pragma unroll
        for (int k = 0; k < kMaxClusters; ++k) {
            const float sk = wave_sum(part[k]);
            if (lane == 0) red[w][k] = sk;
        }
        if (t < kMaxClusters) cnt_s[t] = 0;
        __syncthreads();
        for (int i = t; i < n_win; i += kKmBlock) atomicAdd(&cnt_s[lab[i]], 1);
        __syncthreads();
        for (int k = 0; k < K; ++k) {
            float nrm = 0.f;
            for (int q = 0; q < kKmWaves; ++q) nrm += red[q][k];
            const bool keep = !(cnt_s[k] > 0 && nrm > 0.f);
            const float sc = keep ? 0.f : 1.0f / sqrtf(nrm);
            for (int c = t; c < d; c += kKmBlock) {
                const float v = keep ? zg[k * d + c] : zs[k * d + c] * sc;
                zs[k * d + c] = v;
                zg[k * d + c] = v;
            }
        }
        __syncthreads();
    }

    // 4. outputs: raw sums and counts of the final clusters, labels by position
    for (int c = 4 * t; c < d; c += 4 * kKmBlock) {
        float4 acc[kMaxClusters];
        quad_sums<BF16, false>(hb, wi, seq, n_win, d, c, inv_norm, lab, acc);
#pragma unroll
        for (int k = 0; k < kMaxClusters; ++k)
            if (k < K) *reinterpret_cast<float4*>(sums + (static_cast<size_t>(b) * K + k) * d + c) = acc[k];
    }
    if (t < kMaxClusters) cnt_s[t] = 0;
    __syncthreads();
    for (int i = t; i < n_win; i += kKmBlock) atomicAdd(&cnt_s[lab[i]], 1);
    for (int p = t; p < seq; p += kKmBlock) labels_out[static_cast<size_t>(b) * seq + p] = -1;
    __syncthreads();
    for (int i = t; i < n_win; i += kKmBlock) labels_out[static_cast<size_t>(b) * seq + pos(i)] = lab[i];
    if (t < K) counts[static_cast<size_t>(b) * K + t] = cnt_s[t];
}

// ---------------------------------------------------------------------------
// polestar_cluster for windows of at most kGramMaxWin positions: the same
// K-means, run on the window's Gram matrix.  Every centroid is a combination
// z_k = sum_j C[k][j] u_j of the window's directions u_j = h_j / |h_j| (a
// start point, or the normalised sum of a cluster's members), hence
//   cos(u_i, z_k) = sum_j C[k][j] (u_i . u_j),
//   |sum_{j in M} u_j|^2 = sum_{j, l in M} u_j . u_l.
// kmeans_gram_kernel, one workgroup per sequence:
//   1. G = (h_i . h_j) with MFMAs, the window rows staged in LDS 256 bytes of
//      each row at a time (upper-triangle tiles); G is symmetric and only its
//      upper triangle is kept (row i holds j = i .. n-1), so windows of up to
//      224 positions fit in LDS;
//   2. the rounds on G_ij / (|h_i| |h_j|) and C, all in LDS: the cosines are
//      G C^T and a new centroid's squared norm is the sum of G over its
//      member pairs, both as small fp32 MFMA products (fixed order:
//      deterministic);
//   3. labels and counts.
// Then, over many workgroups (channel ranges), kmeans_out_kernel writes
// the unit centroids sum_j C[k][j] u_j and then the raw sums.  Windows of
// more than 64 positions compute G itself over many workgroups first
// (kmeans_gram_tiles_kernel, 32 x 32 blocks) and phase 1 only loads it.  The
// rows are read a fixed number of times instead of twice per round.
// ---------------------------------------------------------------------------

constexpr int kGramBlock = 512;                 // 8 waves
constexpr int kGramWaves = kGramBlock / kWave;
constexpr int kGramMaxWin = 224;                // 14 row tiles: the upper triangle of G fits in LDS
constexpr int kGramTiles = kGramMaxWin / 16;
constexpr int kGramPairs = kGramTiles * (kGramTiles + 1) / 2;
constexpr int kGramPairsPerWave = (kGramPairs + kGramWaves - 1) / kGramWaves;
constexpr int kGramLda = 272;                   // staged row pitch (bytes): conflict-free fragments
constexpr int kGramRowsPerThread = (kGramMaxWin * 16 + kGramBlock - 1) / kGramBlock;
constexpr int kGramStageBytes = 2 * kGramMaxWin * kGramLda;
constexpr int kGramBytes = kGramMaxWin * (kGramMaxWin + 1) / 2 * 4;   // upper triangle of G, fp32
constexpr int kGramUnionBytes = kGramStageBytes > kGramBytes ? kGramStageBytes : kGramBytes;

// gin: G of every sequence already computed by kmeans_gram_tiles_kernel
// (packed upper triangle, gstride floats apart), else null and phase 1 below
// computes it.
template <bool BF16>
__global__ __launch_bounds__(kGramBlock) void kmeans_gram_kernel(const char* __restrict__ h, int seq, int d,
                                                                 const int32_t* __restrict__ win_idx, int n,
                                                                 int K, int iters, int32_t* __restrict__ labels_out,
                                                                 float* __restrict__ sums,
                                                                 int32_t* __restrict__ counts,
                                                                 const float* __restrict__ gin, size_t gstride) {
    __shared__ __align__(16) char un[kGramUnionBytes];   // staging (phase 1), then G
    // C; rows padded by four floats so that a 16-row column read hits 16 banks
    __shared__ __align__(16) float cf[kMaxClusters][kGramMaxWin + 4];
    __shared__ float cosv[kGramMaxWin][kMaxClusters + 1];
    __shared__ float invn[kGramMaxWin];
    __shared__ float tsum[kGramMaxWin];
    __shared__ __align__(16) int lab[kGramMaxWin];
    __shared__ int posw[kGramMaxWin];
    __shared__ float nrm[kMaxClusters];
    __shared__ int cnt_s[kMaxClusters];
    using T = Elem<BF16>;
    constexpr int ES = T::kBytes;
    const int b = blockIdx.x;
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    const char* hb = h + static_cast<size_t>(b) * seq * d * ES;
    const int32_t* wi = win_idx + static_cast<size_t>(b) * n;
    float* G = reinterpret_cast<float*>(un);
    // G[i][j] of the upper triangle (the pair ordered so that i <= j)
    auto gidx = [n](int i, int j) {
        const int lo = min(i, j), hi = max(i, j);
        return lo * n - (lo * (lo - 1)) / 2 + (hi - lo);
    };
    const int nt = (n + 15) / 16;
    const int npairs = nt * (nt + 1) / 2;

    // window entries are clamped into [0, seq): a bad index cannot leave the rows
    for (int i = t; i < n; i += kGramBlock) posw[i] = min(max(wi[i], 0), seq - 1);
    __syncthreads();

    // 1. Gram matrix.  Wave w owns the upper-triangle tile pairs w, w + 8, ...
    if (gin) {
        const float* gs = gin + static_cast<size_t>(b) * gstride;
        for (int e = t; e < n * (n + 1) / 2; e += kGramBlock) G[e] = gs[e];
    } else {
    int pti[kGramPairsPerWave], ptj[kGramPairsPerWave];
#pragma unroll
    for (int r = 0; r < kGramPairsPerWave; ++r) {
        int q = w + kGramWaves * r, ti = 0;
        if (q >= npairs) q = 0;                          // idle slot: computes pair 0, never stored
        while (q >= nt - ti) { q -= nt - ti; ++ti; }
        pti[r] = ti;
        ptj[r] = ti + q;
    }
    floatx4 acc[kGramPairsPerWave];
#pragma unroll
    for (int r = 0; r < kGramPairsPerWave; ++r) acc[r] = floatx4{0.f, 0.f, 0.f, 0.f};
    // staging thread t moves 16-byte chunk t%16 of rows t/16 + 32r; rows past
    // the window read the first window row and are stored as zeros
    const char* srow[kGramRowsPerThread];
#pragma unroll
    for (int r = 0; r < kGramRowsPerThread; ++r) {
        const int row = (t >> 4) + 32 * r;
        srow[r] = hb + static_cast<size_t>(posw[row < n ? row : 0]) * d * ES + (t & 15) * 16;
    }
    const int nstages = d * ES / 256;
    auto load_stage = [&](int st, uint4 (&ra)[kGramRowsPerThread]) {
#pragma unroll
        for (int r = 0; r < kGramRowsPerThread; ++r) ra[r] = ld16(srow[r] + min(st, nstages - 1) * 256);
    };
    auto store_stage = [&](int buf, const uint4 (&ra)[kGramRowsPerThread]) {
#pragma unroll
        for (int r = 0; r < kGramRowsPerThread; ++r) {
            const int row = (t >> 4) + 32 * r;
            if (row < nt * 16) st16(un + buf * (kGramMaxWin * kGramLda) + row * kGramLda + (t & 15) * 16,
                                    row < n ? ra[r] : zero16());
        }
    };
    const int frag = (lane & 15) * kGramLda + (lane >> 4) * 16;
    auto compute = [&](int buf) {
        const char* sb = un + buf * (kGramMaxWin * kGramLda) + frag;
#pragma unroll
        for (int r = 0; r < kGramPairsPerWave; ++r) {
            if (w + kGramWaves * r < npairs) {
#pragma unroll
                for (int p = 0; p < 4; ++p) {
                    const uint4 a = *reinterpret_cast<const uint4*>(sb + pti[r] * 16 * kGramLda + 64 * p);
                    const uint4 bb = *reinterpret_cast<const uint4*>(sb + ptj[r] * 16 * kGramLda + 64 * p);
                    acc[r] = Mma<BF16>::step(a, bb, acc[r]);
                }
            }
        }
    };
    // two stages in flight (register ring of three): stage st+1 is stored
    // into LDS at the end of stage st while stage st+2 is still loading
    uint4 q0[kGramRowsPerThread], q1[kGramRowsPerThread], q2[kGramRowsPerThread];
    load_stage(0, q0);
    load_stage(1, q1);
    load_stage(2, q2);
    store_stage(0, q0);
    __syncthreads();
#define PS_GRAM_STEP(ST, Q_STORE, Q_LOAD)                                   \
    {                                                                       \
        const int st_ = (ST);                                               \
        compute(st_ & 1);                                                   \
        if (st_ + 1 < nstages) store_stage((st_ + 1) & 1, Q_STORE);         \
        __syncthreads();                                                    \
        load_stage(st_ + 3, Q_LOAD);                                        \
    }
    int sc = 0;
    for (; sc + 3 <= nstages; sc += 3) {   // stage st sits in q(st % 3)
        PS_GRAM_STEP(sc, q1, q0)
        PS_GRAM_STEP(sc + 1, q2, q1)
        PS_GRAM_STEP(sc + 2, q0, q2)
    }
    if (sc < nstages) PS_GRAM_STEP(sc, q1, q0)
    if (sc + 1 < nstages) PS_GRAM_STEP(sc + 1, q2, q1)
#undef PS_GRAM_STEP
    // lane l holds G[16 ti + 4 (l/16) + i][16 tj + l%16], i = 0..3 (and its mirror)
#pragma unroll
    for (int r = 0; r < kGramPairsPerWave; ++r) {
        if (w + kGramWaves * r < npairs) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int gi = pti[r] * 16 + 4 * (lane >> 4) + i, gj = ptj[r] * 16 + (lane & 15);
                if (gi <= gj && gj < n) G[gidx(gi, gj)] = acc[r][i];   // a diagonal tile holds both halves
            }
        }
    }
    }   // phase 1
    __syncthreads();

    // 2. rounds on the cosine Gram matrix
    for (int i = t; i < n; i += kGramBlock) {
        const float g = G[gidx(i, i)];
        invn[i] = g > 0.f ? 1.0f / sqrtf(g) : 0.f;
    }
    // (the cosines G_ij / (|h_i| |h_j|) are formed as the rounds' registers are
    // loaded below)
    // centroid k starts at the point of window rank floor(k n / K); C (all 16
    // rows) and the labels are padded with zeros / -1 to n4 = n rounded up to 4
    const int n4 = (n + 3) & ~3;
    for (int e = t; e < kMaxClusters * n4; e += kGramBlock) {
        const int k = e / n4, j = e - k * n4;
        cf[k][j] = k < K && j == static_cast<int>((static_cast<long>(k) * n) / K) ? 1.f : 0.f;
    }
    for (int j = n + t; j < n4; j += kGramBlock) lab[j] = -1;
    __syncthreads();
    // Products of G with 16 columns (one per cluster), v_mfma_f32_16x16x4f32
    // over j in order: wave w takes the 16-point tiles w, w + 8.  Lane l
    // feeds G[i0 + l%16][j0 + l/16] and column l%16 at j0 + l/16, and holds
    // the result of points i0 + 4 (l/16) + r, column l%16.
    //   mode 0: column k = C[k][.]            -> cosines of the points
    //   mode 1: column k = (label == k)        -> sum of G over the point's cluster
    // The rounds never change G, so each wave keeps its tiles' A operands in
    // registers (ga[tt][s] = cosine of points i0 + l%16 and 4 s + l/16, zero
    // past the window) and every round reads only the columns from LDS.
    constexpr int kWaveTiles = (kGramTiles + kGramWaves - 1) / kGramWaves;
    constexpr int kSteps = kGramMaxWin / 4;        // four-column steps of a row
    float ga[kWaveTiles][kSteps];
#pragma unroll
    for (int tt = 0; tt < kWaveTiles; ++tt) {
        const int ia = (w + kGramWaves * tt) * 16 + (lane & 15);
#pragma unroll
        for (int st = 0; st < kSteps; ++st) {
            const int j = 4 * st + (lane >> 4);
            const int lo = min(ia, j), hi = max(ia, j);
            ga[tt][st] = ia < n && j < n ? G[gidx(lo, hi)] * invn[lo] * invn[hi] : 0.f;
        }
    }
    // Columns go in chunks of eight four-column steps: a chunk's eight LDS
    // reads are issued together (addresses stay inside the arrays; steps past
    // n4 read zero), then its MFMAs run on every tile of the wave.  Steps past
    // the window multiply zeros, so the sums are those of the steps up to n4.
    constexpr int kChunk = 8;
    static_assert(kSteps % kChunk == 0, "whole chunks");
    auto gram_product = [&](int mode) {
        const int col = lane & 15;
        // two interleaved chains per tile (even steps: j0 = 0, 8, 16, ...; odd
        // steps: 4, 12, ...), then summed
        floatx4 c0[kWaveTiles], c1[kWaveTiles];
#pragma unroll
        for (int tt = 0; tt < kWaveTiles; ++tt) c0[tt] = c1[tt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ch = 0; ch < kSteps / kChunk; ++ch) {
            if (4 * kChunk * ch >= n4) break;
            float bv[kChunk];
#pragma unroll
            for (int q = 0; q < kChunk; ++q) {
                const int j = 4 * (kChunk * ch + q) + (lane >> 4);
                const float v = mode == 0 ? cf[col][j] : (lab[j] == col ? 1.f : 0.f);
                bv[q] = j < n4 ? v : 0.f;
            }
#pragma unroll
            for (int tt = 0; tt < kWaveTiles; ++tt) {
                if (w + kGramWaves * tt >= nt) break;
#pragma unroll
                for (int q = 0; q < kChunk; q += 2) {
                    c0[tt] = __builtin_amdgcn_mfma_f32_16x16x4f32(ga[tt][kChunk * ch + q], bv[q], c0[tt], 0, 0, 0);
                    c1[tt] = __builtin_amdgcn_mfma_f32_16x16x4f32(ga[tt][kChunk * ch + q + 1], bv[q + 1], c1[tt],
                                                                  0, 0, 0);
                }
            }
        }
#pragma unroll
        for (int tt = 0; tt < kWaveTiles; ++tt) {
            const int tile = w + kGramWaves * tt;
            if (tile >= nt) break;
            const floatx4 c = c0[tt] + c1[tt];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int i = tile * 16 + 4 * (lane >> 4) + r;
                if (i >= n || col >= K) continue;
                if (mode == 0) cosv[i][col] = c[r];
                else if (lab[i] == col) tsum[i] = c[r];
            }
        }
    };
    for (int it = 0; it <= iters; ++it) {
        // assignment: cos(point i, centroid k) = sum_j C[k][j] G[i][j]
        gram_product(0);
        __syncthreads();
        for (int i = t; i < n; i += kGramBlock) {
            int best = 0;
            float bv = -INFINITY;
            for (int k = 0; k < K; ++k)
                if (cosv[i][k] > bv) { bv = cosv[i][k]; best = k; }   // strict: lowest cluster on ties
            lab[i] = best;
        }
        if (t < kMaxClusters) cnt_s[t] = 0;
        __syncthreads();
        if (it == iters) break;                          // the last round only assigns
        // update: |sum of the members' directions|^2 = sum over member pairs of
        // G; a cluster's wave also counts its members
        gram_product(1);
        __syncthreads();
        for (int k = w; k < K; k += kGramWaves) {
            float s2 = 0.f;
            int c = 0;
            for (int j = lane; j < n; j += kWave) {
                const bool m = lab[j] == k;
                s2 += m ? tsum[j] : 0.f;
                c += __popcll(__ballot(m));
            }
            s2 = wave_sum(s2);
            if (lane == 0) {
                nrm[k] = s2;
                cnt_s[k] = c;
            }
        }
        __syncthreads();
        // clusters with no member keep their centroid
        for (int e = t; e < K * n4; e += kGramBlock) {
            const int k = e / n4, j = e - k * n4;
            if (cnt_s[k] > 0 && nrm[k] > 0.f) cf[k][j] = lab[j] == k ? 1.0f / sqrtf(nrm[k]) : 0.f;
        }
        __syncthreads();
    }

    // 3. outputs: labels by position, counts, raw sums, unit centroids
    for (int i = t; i < n; i += kGramBlock) atomicAdd(&cnt_s[lab[i]], 1);
    for (int p = t; p < seq; p += kGramBlock) labels_out[static_cast<size_t>(b) * seq + p] = -1;
    __syncthreads();
    for (int i = t; i < n; i += kGramBlock) labels_out[static_cast<size_t>(b) * seq + posw[i]] = lab[i];
    if (t < K) counts[static_cast<size_t>(b) * K + t] = cnt_s[t];
    // the final C and 1/|h_i| go to the caller's sums array (K*n + n <= K*d
    // floats) for the centroid launch of kmeans_out_kernel, which its sum launch then
    // overwrites with the raw sums
    float* stash = sums + static_cast<size_t>(b) * K * d;
    for (int e = t; e < K * n; e += kGramBlock) {
        const int k = e / n, j = e - k * n;
        stash[e] = cf[k][j];
    }
    for (int i = t; i < n; i += kGramBlock) stash[K * n + i] = invn[i];
}

// The Gram matrix of a window over many workgroups: one 32 x 32 block (bi,
// bj), bi <= bj, of G per workgroup, its four waves one 16 x 16 tile each.
// Every tile runs the MFMA chain of kmeans_gram_kernel's phase 1 (the same
// staged fragments, stages and k order), so G is bit-identical; it is written
// in the kernel's packed upper-triangle layout for kmeans_gram_kernel to load.
constexpr int kGtBlock = 256;

template <bool BF16>
__global__ __launch_bounds__(kGtBlock) void kmeans_gram_tiles_kernel(const char* __restrict__ h, int seq, int d,
                                                                     const int32_t* __restrict__ win_idx, int n,
                                                                     float* __restrict__ gout, size_t gstride) {
    using T = Elem<BF16>;
    constexpr int ES = T::kBytes;
    __shared__ __align__(16) char sa[2][64 * kGramLda];   // staged rows: 0..31 block bi, 32..63 block bj
    const int b = blockIdx.y;
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    const int nb = (n + 31) / 32;
    int q = blockIdx.x, bi = 0;
    while (q >= nb - bi) {
        q -= nb - bi;
        ++bi;
    }
    const int bj = bi + q;
    const char* hb = h + static_cast<size_t>(b) * seq * d * ES;
    const int32_t* wi = win_idx + static_cast<size_t>(b) * n;
    // thread t moves 16-byte chunk t%16 of staged rows t/16 + 16 r; points
    // past the window read the first window row and are stored as zeros
    const char* srow[4];
    bool live[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int sr = (t >> 4) + 16 * r;
        const int pt = sr < 32 ? 32 * bi + sr : 32 * bj + sr - 32;
        live[r] = pt < n;
        const int pos = min(max(wi[live[r] ? pt : 0], 0), seq - 1);
        srow[r] = hb + static_cast<size_t>(pos) * d * ES + (t & 15) * 16;
    }
    const int nstages = d * ES / 256;
    auto load_stage = [&](int st, uint4 (&ra)[4]) {
#pragma unroll
        for (int r = 0; r < 4; ++r) ra[r] = ld16(srow[r] + min(st, nstages - 1) * 256);
    };
    auto store_stage = [&](int buf, const uint4 (&ra)[4]) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
            st16(sa[buf] + ((t >> 4) + 16 * r) * kGramLda + (t & 15) * 16, live[r] ? ra[r] : zero16());
    };
    // wave w: rows 16 (w / 2) .. of block bi against rows 16 (w % 2) .. of block bj
    const int frag = (lane & 15) * kGramLda + (lane >> 4) * 16;
    const int aoff = 16 * (w >> 1) * kGramLda + frag, boff = (32 + 16 * (w & 1)) * kGramLda + frag;
    floatx4 acc = {0.f, 0.f, 0.f, 0.f};
    auto compute = [&](int buf) {
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            const uint4 a = *reinterpret_cast<const uint4*>(sa[buf] + aoff + 64 * p);
            const uint4 bb = *reinterpret_cast<const uint4*>(sa[buf] + boff + 64 * p);
            acc = Mma<BF16>::step(a, bb, acc);
        }
    };
    uint4 q0[4], q1[4], q2[4];
    load_stage(0, q0);
    load_stage(1, q1);
    load_stage(2, q2);
    store_stage(0, q0);
    __syncthreads();
#define PS_GT_STEP(ST, Q_STORE, Q_LOAD)                                     \
    {                                                                       \
        const int st_ = (ST);                                               \
        compute(st_ & 1);                                                   \
        if (st_ + 1 < nstages) store_stage((st_ + 1) & 1, Q_STORE);         \
        __syncthreads();                                                    \
        load_stage(st_ + 3, Q_LOAD);                                        \
    }
    int sc = 0;
    for (; sc + 3 <= nstages; sc += 3) {   // stage st sits in q(st % 3)
        PS_GT_STEP(sc, q1, q0)
        PS_GT_STEP(sc + 1, q2, q1)
        PS_GT_STEP(sc + 2, q0, q2)
    }
    if (sc < nstages) PS_GT_STEP(sc, q1, q0)
    if (sc + 1 < nstages) PS_GT_STEP(sc + 1, q2, q1)
#undef PS_GT_STEP
    // lane l holds G[gi0 + 4 (l/16) + i][gj0 + l%16]
    float* gs = gout + static_cast<size_t>(b) * gstride;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int gi = 32 * bi + 16 * (w >> 1) + 4 * (lane >> 4) + i, gj = 32 * bj + 16 * (w & 1) + (lane & 15);
        if (gi <= gj && gj < n) gs[gi * n - (gi * (gi - 1)) / 2 + (gj - gi)] = acc[i];
    }
}


// Per-cluster weighted sums of the window rows, 256 channels per workgroup
// (a lane's four channels), for the Gram path's outputs:
//   UNITC: the unit centroids z_k = sum_i C[k][i] h_i / |h_i|, from the stash
//          kmeans_gram_kernel leaves in the sums array;
//   else:  the raw sums of the final clusters (one-hot labels), written over
//          the sums array (after the centroid launch has read the stash).
// Wave w takes points w, w + 8, ... in order (loads of eight points issued
// before any is used); the eight waves' sums are then added in wave order.
constexpr int kKmOutWaves = 8;
constexpr int kKmOutThreads = kKmOutWaves * 64;

template <bool BF16, bool UNITC>
__global__ __launch_bounds__(kKmOutThreads) void kmeans_out_kernel(const char* __restrict__ h, int seq, int d,
                                                                  const int32_t* __restrict__ win_idx, int n, int K,
                                                                  const float* __restrict__ stash_all,
                                                                  const int32_t* __restrict__ labels,
                                                                  float* __restrict__ out) {
    __shared__ float w_s[UNITC ? kMaxClusters : 1][kGramMaxWin];   // C[k][i] / |h_i|
    __shared__ int lab_s[kGramMaxWin];
    __shared__ int pos_s[kGramMaxWin];
    __shared__ float4 red[kKmOutWaves - 1][kMaxClusters][64];
    constexpr int ES = Elem<BF16>::kBytes;
    const int b = blockIdx.y;
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    for (int i = t; i < n; i += kKmOutThreads) {
        pos_s[i] = min(max(win_idx[static_cast<size_t>(b) * n + i], 0), seq - 1);
        if (!UNITC) lab_s[i] = labels[static_cast<size_t>(b) * seq + pos_s[i]];
    }
    if constexpr (UNITC) {
        const float* stash = stash_all + static_cast<size_t>(b) * K * d;
        for (int e = t; e < K * n; e += kKmOutThreads) {
            const int k = e / n, i = e - k * n;
            w_s[k][i] = stash[e] * stash[K * n + i];
        }
    }
    __syncthreads();
    const int c = min((blockIdx.x * 64 + lane) * 4, d - 4);   // lanes past d repeat the last quad, never stored
    const char* hb = h + static_cast<size_t>(b) * seq * d * ES;
    float4 acc[kMaxClusters];
#pragma unroll
    for (int k = 0; k < kMaxClusters; ++k) acc[k] = make_float4(0.f, 0.f, 0.f, 0.f);
    constexpr int kBatch = 8;
    for (int i0 = w; i0 < n; i0 += kBatch * kKmOutWaves) {
        float4 v[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u)
            v[u] = load4<BF16>(hb + static_cast<size_t>(pos_s[min(i0 + kKmOutWaves * u, n - 1)]) * d * ES, c);
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int i = i0 + kKmOutWaves * u;
            if (i >= n) break;
            const int li = UNITC ? 0 : lab_s[i];
#pragma unroll
            for (int k = 0; k < kMaxClusters; ++k) {
                if (k < K) {
                    const float wk = UNITC ? w_s[k][i] : (li == k ? 1.f : 0.f);
                    acc[k].x = fmaf(v[u].x, wk, acc[k].x);
                    acc[k].y = fmaf(v[u].y, wk, acc[k].y);
                    acc[k].z = fmaf(v[u].z, wk, acc[k].z);
                    acc[k].w = fmaf(v[u].w, wk, acc[k].w);
                }
            }
        }
    }
    if (w > 0) {
#pragma unroll
        for (int k = 0; k < kMaxClusters; ++k)
            if (k < K) red[w - 1][k][lane] = acc[k];
    }
    __syncthreads();
    if (w > 0 || (blockIdx.x * 64 + lane) * 4 >= d) return;
#pragma unroll
    for (int k = 0; k < kMaxClusters; ++k) {
        if (k >= K) continue;
        float4 s = acc[k];
#pragma unroll
        for (int ww = 0; ww < kKmOutWaves - 1; ++ww) {
            const float4 r = red[ww][k][lane];
            s.x += r.x;
            s.y += r.y;
            s.z += r.z;
            s.w += r.w;
        }
        *reinterpret_cast<float4*>(out + (static_cast<size_t>(b) * K + k) * d + c) = s;
    }
}

// ---------------------------------------------------------------------------
// polestar_proxy_drift kernels
// ---------------------------------------------------------------------------

// token[b][k][:] = dtype(sums / count), zero for an empty cluster; thread
// per 4 channels (d % 4 == 0), workgroups over (cluster, channel range).
template <bool BF16>
__global__ __launch_bounds__(256) void token_kernel(const float* __restrict__ sums,
                                                    const int32_t* __restrict__ counts, int d,
                                                    char* __restrict__ tok) {
    const int bk = blockIdx.y;
    const int c = (blockIdx.x * 256 + threadIdx.x) * 4;
    if (c >= d) return;
    const int n = counts[bk];
    const float4 v = *reinterpret_cast<const float4*>(sums + static_cast<size_t>(bk) * d + c);
    const float f = n > 0 ? static_cast<float>(n) : 1.f;
    const float x0 = n > 0 ? v.x / f : 0.f, x1 = n > 0 ? v.y / f : 0.f;
    const float x2 = n > 0 ? v.z / f : 0.f, x3 = n > 0 ? v.w / f : 0.f;
    if constexpr (BF16)
        *reinterpret_cast<uint2*>(tok + (static_cast<size_t>(bk) * d + c) * 2) =
            make_uint2(pack_bf16x2(x0, x1), pack_bf16x2(x2, x3));
    else
        *reinterpret_cast<float4*>(tok + (static_cast<size_t>(bk) * d + c) * 4) = make_float4(x0, x1, x2, x3);
}

// ---------------------------------------------------------------------------
// Scores of R query rows over every cache position and their KL against the
// previous step's scores: the proxy drift of the clusters (R = K proxy
// queries) and the commit drift of the block's queries.  S^T = K Q^T on
// MFMA: a wave takes 16-key tiles, the query rows sit in registers as B
// fragments.  Nothing is staged: each lane folds its scores into an online
// (m, Z, W) per query row,
//     Z = sum_j e^(s_j - m),   W = sum_j e^(s_j - m) (s_j - s'_j),
// so that KL(p || p') = W / Z - (m + log Z) + lse' with p = softmax(s), and
// each score replaces the previous one in place (read and written by the
// same lane).  grid (key splits, heads, batch); the partials of a split go to
// part[b][r][h][split][3] and qkl_merge_kernel combines them.
// ---------------------------------------------------------------------------
constexpr int kQkBlock = 256;
constexpr int kQkWaves = kQkBlock / kWave;
constexpr int kQkMaxRows = 64;              // four 16-row query tiles
constexpr int kQkMaxSplits = 16;

struct QklArgs {
    const char* q;        // [b][R][H][hd]
    const char* kc;       // [b][S][Hkv][hd]
    float* scores;        // [b][R][H][S], the previous step's in, this step's out
    float* part;          // [b][R][H][splits][3]
    int R, S, H, Hkv, splits, tiles_per_split, first;
    float scale;
};

// (m, z, w) <- merge with (m2, z2, w2)
__device__ __forceinline__ void mzw_merge(float& m, float& z, float& w, float m2, float z2, float w2) {
    const float mn = fmaxf(m, m2);
    const float f1 = m == mn ? 1.f : __expf(m - mn);
    const float f2 = m2 == mn ? 1.f : __expf(m2 - mn);
    z = z * f1 + z2 * f2;
    w = w * f1 + w2 * f2;
    m = mn;
}

template <bool BF16, int HD, int RT>
__global__ __launch_bounds__(kQkBlock) void qkl_kernel(QklArgs a) {
    using T = Elem<BF16>;
    constexpr int ES = T::kBytes;
    constexpr int E = T::E;                  // elements per 16-byte chunk
    constexpr int NC = HD / (4 * E);         // chunks per row and lane (k-group g of each MFMA step)
    constexpr int TB = RT * NC <= 8 ? 4 : (RT * NC <= 16 ? 2 : 1);   // key tiles loaded together
    __shared__ float red[kQkWaves][RT * 16][3];
    const int split = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    const int g = lane >> 4, li = lane & 15;
    const int kvh = h / (a.H / a.Hkv);

    // query fragments: row 16 rt + li (rows past R repeat the last one and are
    // never stored), chunk c holds elements [4E c + E g, +E)
    uint4 qf[RT][NC];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
        const int r = min(16 * rt + li, a.R - 1);
        const char* qrow = a.q + ((static_cast<size_t>(b) * a.R + r) * a.H + h) * HD * ES;
#pragma unroll
        for (int c = 0; c < NC; ++c) qf[rt][c] = ld16(qrow + (c * 4 * E + g * E) * ES);
    }
    float pm[RT], pz[RT], pw[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) { pm[rt] = -INFINITY; pz[rt] = 0.f; pw[rt] = 0.f; }

    const int ntiles = (a.S + 15) / 16;
    const int t0 = split * a.tiles_per_split;
    const int t1 = min(ntiles, t0 + a.tiles_per_split);
    const size_t krow = static_cast<size_t>(a.Hkv) * HD * ES;
    const char* kbase = a.kc + (static_cast<size_t>(b) * a.S * a.Hkv + kvh) * HD * ES;
    // with S a multiple of 16 (and 16-byte aligned scores) every tile is whole
    // and the lane's four scores load and store as one float4
    const bool full = (a.S & 15) == 0 && (reinterpret_cast<uintptr_t>(a.scores) & 15) == 0;
    for (int tb = t0 + w; tb < t1; tb += kQkWaves * TB) {
        // every load of this round first: key fragments of TB tiles and the
        // previous scores the lane will fold in (clamped, unused when invalid)
        uint4 kf[TB][NC];
        float sp[TB][RT][4];
#pragma unroll
        for (int u = 0; u < TB; ++u) {
            const int tile = min(tb + u * kQkWaves, t1 - 1);
            const int key = min(tile * 16 + li, a.S - 1);
#pragma unroll
            for (int c = 0; c < NC; ++c) kf[u][c] = ld16(kbase + key * krow + (c * 4 * E + g * E) * ES);
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
                const int r = min(16 * rt + li, a.R - 1);
                const float* srow = a.scores + ((static_cast<size_t>(b) * a.R + r) * a.H + h) * a.S;
                if (full) {   // the lane's four scores in one 16-byte load
                    const float4 v = *reinterpret_cast<const float4*>(srow + tile * 16 + 4 * g);
                    sp[u][rt][0] = v.x;
                    sp[u][rt][1] = v.y;
                    sp[u][rt][2] = v.z;
                    sp[u][rt][3] = v.w;
                } else {
#pragma unroll
                    for (int i = 0; i < 4; ++i) sp[u][rt][i] = srow[min(tile * 16 + 4 * g + i, a.S - 1)];
                }
            }
        }
#pragma unroll
        for (int u = 0; u < TB; ++u) {
            const int tile = tb + u * kQkWaves;
            if (tile < t1) {
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) {
                    floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int c = 0; c < NC; ++c) acc = Mma<BF16>::step(kf[u][c], qf[rt][c], acc);
                    // lane holds S^T[key 16 tile + 4 g + i][query 16 rt + li]
                    const int r = 16 * rt + li;
                    float* srow = a.scores + ((static_cast<size_t>(b) * a.R + min(r, a.R - 1)) * a.H + h) * a.S;
                    float sv[4];
                    bool ok[4];
                    float mx = pm[rt];
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int key = tile * 16 + 4 * g + i;
                        ok[i] = (r < a.R) & (key < a.S);
                        sv[i] = acc[i] * a.scale;
                        mx = ok[i] ? fmaxf(mx, sv[i]) : mx;
                    }
                    const float f = pm[rt] == mx ? 1.f : __expf(pm[rt] - mx);
                    float z = pz[rt] * f, ww = pw[rt] * f;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        if (ok[i]) {
                            const float e = __expf(sv[i] - mx);
                            z += e;
                            ww = fmaf(e, sv[i] - sp[u][rt][i], ww);
                            if (!full) srow[tile * 16 + 4 * g + i] = sv[i];
                        }
                    }
                    if (full && r < a.R)
                        *reinterpret_cast<float4*>(srow + tile * 16 + 4 * g) = make_float4(sv[0], sv[1], sv[2], sv[3]);
                    pm[rt] = mx;
                    pz[rt] = z;
                    pw[rt] = ww;
                }
            }
        }
    }
    // lanes li, li+16, li+32, li+48 hold the same query rows: merge, then the waves
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
        for (int off = 16; off <= 32; off <<= 1) {
            const float m2 = __shfl_xor(pm[rt], off), z2 = __shfl_xor(pz[rt], off), w2 = __shfl_xor(pw[rt], off);
            mzw_merge(pm[rt], pz[rt], pw[rt], m2, z2, w2);
        }
        if (g == 0) {
            red[w][16 * rt + li][0] = pm[rt];
            red[w][16 * rt + li][1] = pz[rt];
            red[w][16 * rt + li][2] = pw[rt];
        }
    }
    __syncthreads();
    if (t < RT * 16 && t < a.R) {
        float m = red[0][t][0], z = red[0][t][1], ww = red[0][t][2];
#pragma unroll
        for (int q = 1; q < kQkWaves; ++q) mzw_merge(m, z, ww, red[q][t][0], red[q][t][1], red[q][t][2]);
        float* pp = a.part + (((static_cast<size_t>(b) * a.R + t) * a.H + h) * a.splits + split) * 3;
        pp[0] = m;
        pp[1] = z;
        pp[2] = ww;
    }
}

// One wave per (sequence, query row): lane h merges head h's splits, then
//   lse = m + log Z,   KL = first ? 0 : W / Z - lse + lse_prev,
// lse replaces lse_prev, and drift = the mean of KL over the heads.
__global__ __launch_bounds__(256) void qkl_merge_kernel(const float* __restrict__ part, int BR, int H, int splits,
                                                        int first, float* __restrict__ lse,
                                                        float* __restrict__ drift) {
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= BR) return;                              // uniform per wave
    float acc = 0.f;
    for (int h = lane; h < H; h += kWave) {
        const float* pp = part + (static_cast<size_t>(row) * H + h) * splits * 3;
        float v[kQkMaxSplits][3];
#pragma unroll
        for (int s = 0; s < kQkMaxSplits; ++s) {
            const int sc = min(s, splits - 1);
            v[s][0] = pp[3 * sc];
            v[s][1] = pp[3 * sc + 1];
            v[s][2] = pp[3 * sc + 2];
        }
        float m = v[0][0], z = v[0][1], w = v[0][2];
#pragma unroll
        for (int s = 1; s < kQkMaxSplits; ++s)
            if (s < splits) mzw_merge(m, z, w, v[s][0], v[s][1], v[s][2]);
        const size_t id = static_cast<size_t>(row) * H + h;
        const float l = m + logf(z);
        const float kl = first ? 0.f : w / z - l + lse[id];
        lse[id] = l;
        acc += kl;
    }
    acc = wave_sum(acc);
    if (lane == 0) drift[row] = acc / static_cast<float>(H);
}

struct QklPlan {
    int splits, tiles_per_split;
    size_t part_bytes;
};

// Key splits: at least about 256 workgroups, and at most 16 key tiles per
// workgroup, so that a wave's tiles (four at a time for bf16 rows of up to
// 32 query rows at head_dim 128) are loaded in one round instead of several
// dependent ones: the batch-8 LLaDA-8B shape (8 x 32 heads, 96 tiles) went
// from one split to six, the Dream-7B one (4 x 28 heads, 128 tiles) from
// three to eight.  Several workgroups fit per CU.
QklPlan qkl_plan(int batch, int seq, int R, int H) {
    QklPlan p{};
    const int ntiles = ceil_div(seq, 16);
    const long base = static_cast<long>(batch) * H;
    int splits = max(static_cast<int>((256 + base - 1) / base), ceil_div(ntiles, 16));
    splits = min(splits, max(1, ntiles / kQkWaves));
    splits = max(1, min(splits, kQkMaxSplits));
    p.tiles_per_split = ceil_div(ntiles, splits);
    p.splits = ceil_div(ntiles, p.tiles_per_split);
    p.part_bytes = align_up(static_cast<size_t>(batch) * R * H * p.splits * 3 * sizeof(float), 256);
    return p;
}

template <bool BF16, int HD>
void launch_qkl_rt(const QklArgs& a, int batch, hipStream_t s) {
    const dim3 grid(a.splits, a.H, batch);
    const int rt = ceil_div(a.R, 16);
    if (rt == 1) hipLaunchKernelGGL((qkl_kernel<BF16, HD, 1>), grid, dim3(kQkBlock), 0, s, a);
    else if (rt == 2) hipLaunchKernelGGL((qkl_kernel<BF16, HD, 2>), grid, dim3(kQkBlock), 0, s, a);
    else if (rt == 3) hipLaunchKernelGGL((qkl_kernel<BF16, HD, 3>), grid, dim3(kQkBlock), 0, s, a);
    else hipLaunchKernelGGL((qkl_kernel<BF16, HD, 4>), grid, dim3(kQkBlock), 0, s, a);
}

// scores + KL of R query rows, then the merge.  The caller has validated
// shapes (R <= kQkMaxRows, hd 64 or 128, H % Hkv == 0) and sized `part`.
polestar_status run_qkl(bool bf16, int batch, int seq, int R, int H, int Hkv, int hd, const char* q,
                        const char* kc, float scale, float* scores, float* lse, int first, float* part,
                        float* drift, hipStream_t stream) {
    const QklPlan p = qkl_plan(batch, seq, R, H);
    QklArgs a{};
    a.q = q;
    a.kc = kc;
    a.scores = scores;
    a.part = part;
    a.R = R;
    a.S = seq;
    a.H = H;
    a.Hkv = Hkv;
    a.splits = p.splits;
    a.tiles_per_split = p.tiles_per_split;
    a.first = first;
    a.scale = scale > 0.f ? scale : 1.0f / sqrtf(static_cast<float>(hd));
    if (bf16) { if (hd == 128) launch_qkl_rt<true, 128>(a, batch, stream); else launch_qkl_rt<true, 64>(a, batch, stream); }
    else { if (hd == 128) launch_qkl_rt<false, 128>(a, batch, stream); else launch_qkl_rt<false, 64>(a, batch, stream); }
    polestar_status st = launch_status();
    if (st != POLESTAR_OK) return st;
    const int BR = batch * R;
    hipLaunchKernelGGL(qkl_merge_kernel, dim3(ceil_div(BR, 4)), dim3(256), 0, stream, part, BR, H, p.splits, first,
                       lse, drift);
    return launch_status();
}

// ---------------------------------------------------------------------------
// polestar_cluster_select: one 256-thread workgroup per sequence.  Rank of
// cluster k = clusters with larger drift, or equal drift and a lower index;
// selected if rank < k_top.  Positions are then streamed in order and the
// members of selected clusters written ascending (block prefix sums).
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(256) void cluster_select_kernel(const int32_t* __restrict__ labels, int seq,
                                                             const float* __restrict__ drift, int K, int k_top,
                                                             int32_t* __restrict__ idx, int k_max,
                                                             int32_t* __restrict__ cnt) {
    __shared__ int sel[kMaxClusters];
    __shared__ int scan_tmp[17];
    const int b = blockIdx.x, t = threadIdx.x;
    if (t < K) {
        const float dt = drift[static_cast<size_t>(b) * K + t];
        int rank = 0;
        for (int j = 0; j < K; ++j) {
            const float dj = drift[static_cast<size_t>(b) * K + j];
            rank += (dj > dt || (dj == dt && j < t)) ? 1 : 0;
        }
        sel[t] = rank < k_top ? 1 : 0;
    }
    __syncthreads();
    const int32_t* lb = labels + static_cast<size_t>(b) * seq;
    int32_t* out = idx + static_cast<size_t>(b) * k_max;
    int written = 0;
    for (int p0 = 0; p0 < seq; p0 += 256) {
        const int p = p0 + t;
        const int l = p < seq ? lb[p] : -1;
        const int take = (l >= 0 && l < K && sel[l]) ? 1 : 0;
        int total;
        const int ex = block_excl_scan(take, scan_tmp, &total);
        if (take && written + ex < k_max) out[written + ex] = p;
        written += total;
    }
    const int n = min(written, k_max);
    for (int i = n + t; i < k_max; i += 256) out[i] = -1;
    if (t == 0) cnt[b] = n;
}

// ---------------------------------------------------------------------------
// polestar_cluster_update: thread per 4 channels of one sequence; the
// refreshed rows are taken in list order and each channel's per-cluster
// change accumulated in registers (deterministic), then added to the sums.
// ---------------------------------------------------------------------------

template <bool BF16>
__global__ __launch_bounds__(256) void cluster_update_kernel(const char* __restrict__ h_new,
                                                             const char* __restrict__ h_old, int seq, int d,
                                                             const int32_t* __restrict__ labels, int K,
                                                             const int32_t* __restrict__ idx,
                                                             const int32_t* __restrict__ cnt, int k_max,
                                                             float* __restrict__ sums) {
    constexpr int ES = Elem<BF16>::kBytes;
    const int b = blockIdx.y;
    const int c0 = (blockIdx.x * 256 + threadIdx.x) * 4;
    if (c0 >= d) return;
    float acc[kMaxClusters][4];
#pragma unroll
    for (int k = 0; k < kMaxClusters; ++k)
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[k][e] = 0.f;
    const int n = min(max(cnt[b], 0), k_max);
    const int32_t* ib = idx + static_cast<size_t>(b) * k_max;
    const int32_t* lb = labels + static_cast<size_t>(b) * seq;
    for (int r = 0; r < n; ++r) {
        const int p = ib[r];
        if (p < 0 || p >= seq) continue;
        const int l = lb[p];
        if (l < 0 || l >= K) continue;
        const size_t off = (static_cast<size_t>(b) * seq + p) * d + c0;
        float dv[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) dv[e] = load_elem<BF16>(h_new + off * ES, e) - load_elem<BF16>(h_old + off * ES, e);
#pragma unroll
        for (int k = 0; k < kMaxClusters; ++k)
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[k][e] += (l == k) ? dv[e] : 0.f;
    }
#pragma unroll
    for (int k = 0; k < kMaxClusters; ++k) {
        if (k < K) {
            float* s = sums + (static_cast<size_t>(b) * K + k) * d + c0;
#pragma unroll
            for (int e = 0; e < 4; ++e) s[e] += acc[k][e];
        }
    }
}

// Workspace of polestar_proxy_drift: tokens, queries, the GEMM's partials,
// the score/KL partials.
struct ProxyLayout {
    GemmPlan qp;
    size_t tok, q, gemm, part, total;
};

ProxyLayout proxy_layout(bool bf16, int batch, int seq, int d, int H, int hd, int K) {
    ProxyLayout L{};
    const size_t es = bf16 ? 2 : 4;
    L.qp = gemm_plan(bf16, static_cast<long>(batch) * K, H * hd, d);
    L.tok = 0;
    L.q = align_up(static_cast<size_t>(batch) * K * d * es, 256);
    L.gemm = L.q + align_up(static_cast<size_t>(batch) * K * H * hd * es, 256);
    L.part = L.gemm + align_up(L.qp.ws_bytes, 256);
    L.total = L.part + qkl_plan(batch, seq, K, H).part_bytes;
    return L;
}

}  // namespace
}  // namespace ps

extern "C" polestar_status polestar_cluster(polestar_dtype dtype, int batch, int seq, int d, const void* h,
                                            const int32_t* win_idx, int n_win, int n_clusters, int iters,
                                            int32_t* labels, float* sums, int32_t* counts, float* centroids,
                                            hipStream_t stream) {
    using namespace ps;
    if (!dtype_ok(dtype) || batch <= 0 || seq <= 0 || d <= 0 || n_win <= 0 || n_win > seq ||
        n_clusters <= 0 || n_clusters > n_win || iters < 0 || !h || !win_idx || !labels || !sums ||
        !counts || !centroids)
        return POLESTAR_ERR_INVALID_ARGUMENT;
    if (n_clusters > kMaxClusters || n_win > kMaxWin ||
        static_cast<long>(n_clusters) * d > kMaxCentroidFloats || batch > 65535 ||
        d % (dtype == POLESTAR_BF16 ? 512 : 256) != 0 || !aligned16(h) || !aligned16(sums) ||
        !aligned16(centroids))
        return POLESTAR_ERR_UNSUPPORTED;
    // the Gram path stashes (K + 1) * n_win floats in each sequence's K * d sums
    if (n_win <= kGramMaxWin && static_cast<long>(n_clusters) * d >= static_cast<long>(n_clusters + 1) * n_win) {
        const char* hc = static_cast<const char*>(h);
        const dim3 out_grid(ceil_div(d, 256), batch);
        // windows longer than 64: G over many workgroups, held in the centroid
        // output (free until the centroid launch) when it fits there
        const size_t gstride = static_cast<size_t>(n_clusters) * d;
        const bool tiles = n_win > 64 && gstride >= static_cast<size_t>(n_win) * (n_win + 1) / 2;
        const float* gin = tiles ? centroids : nullptr;
        const int nb = ceil_div(n_win, 32);
        const dim3 tgrid(nb * (nb + 1) / 2, batch);
        if (dtype == POLESTAR_BF16) {
            if (tiles)
                hipLaunchKernelGGL((kmeans_gram_tiles_kernel<true>), tgrid, dim3(kGtBlock), 0, stream, hc, seq, d,
                                   win_idx, n_win, centroids, gstride);
            hipLaunchKernelGGL((kmeans_gram_kernel<true>), dim3(batch), dim3(kGramBlock), 0, stream, hc, seq, d,
                               win_idx, n_win, n_clusters, iters, labels, sums, counts, gin, gstride);
            hipLaunchKernelGGL((kmeans_out_kernel<true, true>), out_grid, dim3(kKmOutThreads), 0, stream, hc,
                               seq, d, win_idx, n_win, n_clusters, sums, labels, centroids);
            hipLaunchKernelGGL((kmeans_out_kernel<true, false>), out_grid, dim3(kKmOutThreads), 0, stream, hc,
                               seq, d, win_idx, n_win, n_clusters, sums, labels, sums);
        } else {
            if (tiles)
                hipLaunchKernelGGL((kmeans_gram_tiles_kernel<false>), tgrid, dim3(kGtBlock), 0, stream, hc, seq, d,
                                   win_idx, n_win, centroids, gstride);
            hipLaunchKernelGGL((kmeans_gram_kernel<false>), dim3(batch), dim3(kGramBlock), 0, stream, hc, seq, d,
                               win_idx, n_win, n_clusters, iters, labels, sums, counts, gin, gstride);
            hipLaunchKernelGGL((kmeans_out_kernel<false, true>), out_grid, dim3(kKmOutThreads), 0, stream, hc,
                               seq, d, win_idx, n_win, n_clusters, sums, labels, centroids);
            hipLaunchKernelGGL((kmeans_out_kernel<false, false>), out_grid, dim3(kKmOutThreads), 0, stream, hc,
                               seq, d, win_idx, n_win, n_clusters, sums, labels, sums);
        }
        return launch_status();
    }
    const size_t lds = static_cast<size_t>(n_clusters) * d * sizeof(float);
    if (dtype == POLESTAR_BF16)
        hipLaunchKernelGGL((kmeans_kernel<true>), dim3(batch), dim3(kKmBlock), lds, stream,
                           static_cast<const char*>(h), seq, d, win_idx, n_win, n_clusters, iters, labels, sums,
                           counts, centroids);
    else
        hipLaunchKernelGGL((kmeans_kernel<false>), dim3(batch), dim3(kKmBlock), lds, stream,
                           static_cast<const char*>(h), seq, d, win_idx, n_win, n_clusters, iters, labels, sums,
                           counts, centroids);
    return launch_status();
}

extern "C" size_t polestar_proxy_drift_workspace_size(polestar_dtype dtype, int batch, int seq, int d,
                                                      int n_heads, int head_dim, int n_clusters) {
    using namespace ps;
    if (!dtype_ok(dtype) || batch <= 0 || seq <= 0 || d <= 0 || n_heads <= 0 || head_dim <= 0 ||
        n_clusters <= 0)
        return 0;
    return proxy_layout(dtype == POLESTAR_BF16, batch, seq, d, n_heads, head_dim, n_clusters).total;
}

extern "C" polestar_status polestar_proxy_drift(polestar_dtype dtype, int batch, int seq, int d, int n_heads,
                                                int n_kv_heads, int head_dim, int n_clusters,
                                                const float* sums, const int32_t* counts, const void* w_q,
                                                const void* k_cache, float scale, float* scores, float* lse,
                                                int first, float* drift, void* workspace,
                                                size_t workspace_bytes, hipStream_t stream) {
    using namespace ps;
    if (!dtype_ok(dtype) || batch <= 0 || seq <= 0 || d <= 0 || n_heads <= 0 || n_kv_heads <= 0 ||
        head_dim <= 0 || n_clusters <= 0 || n_heads % n_kv_heads != 0 || !sums || !counts || !w_q ||
        !k_cache || !scores || !lse || !drift)
        return POLESTAR_ERR_INVALID_ARGUMENT;
    const bool bf16 = dtype == POLESTAR_BF16;
    if ((head_dim != 64 && head_dim != 128) || !gemm_k_ok(bf16, d) || n_clusters > kMaxClusters ||
        !aligned16(w_q) || !aligned16(k_cache) || !aligned16(workspace) || !aligned16(sums) ||
        batch > 65535 || n_heads > 65535)
        return POLESTAR_ERR_UNSUPPORTED;
    const ProxyLayout L = proxy_layout(bf16, batch, seq, d, n_heads, head_dim, n_clusters);
    if (workspace_bytes < L.total || !workspace) return POLESTAR_ERR_WORKSPACE;
    char* ws = static_cast<char*>(workspace);
    const int BK = batch * n_clusters;
    const dim3 tgrid(ceil_div(d, 1024), BK);
    if (bf16) hipLaunchKernelGGL((token_kernel<true>), tgrid, dim3(256), 0, stream, sums, counts, d, ws + L.tok);
    else hipLaunchKernelGGL((token_kernel<false>), tgrid, dim3(256), 0, stream, sums, counts, d, ws + L.tok);
    polestar_status st = launch_status();
    if (st != POLESTAR_OK) return st;
    // queries: the tokens as the "block rows" of a [batch][K][d] input
    GemmArgs g{};
    g.x = ws + L.tok;
    g.w0 = static_cast<const char*>(w_q);
    g.n0 = n_heads * head_dim;
    g.N = n_heads * head_dim;
    g.K = d;
    g.mode = kGemmBlockRows;
    g.batch = batch;
    g.seq = n_clusters;
    g.block_start = 0;
    g.block_len = n_clusters;
    g.out0 = ws + L.q;
    g.ws = reinterpret_cast<float*>(ws + L.gemm);
    g.m_max = BK;
    st = gemm_run(bf16, L.qp, g, stream);
    if (st != POLESTAR_OK) return st;
    return run_qkl(bf16, batch, seq, n_clusters, n_heads, n_kv_heads, head_dim, ws + L.q,
                   static_cast<const char*>(k_cache), scale, scores, lse, first,
                   reinterpret_cast<float*>(ws + L.part), drift, stream);
}

extern "C" size_t polestar_attention_drift_workspace_size(int batch, int seq, int n_rows, int n_heads) {
    using namespace ps;
    if (batch <= 0 || seq <= 0 || n_rows <= 0 || n_heads <= 0) return 0;
    return qkl_plan(batch, seq, n_rows, n_heads).part_bytes;
}

// Drift of the attention distributions of given query rows (the commit drift
// of Alg. 1 for the block's queries of the last layer).
extern "C" polestar_status polestar_attention_drift(polestar_dtype dtype, int batch, int seq, int n_rows,
                                                    int n_heads, int n_kv_heads, int head_dim, const void* q,
                                                    const void* k_cache, float scale, float* scores, float* lse,
                                                    int first, float* drift, void* workspace,
                                                    size_t workspace_bytes, hipStream_t stream) {
    using namespace ps;
    if (!dtype_ok(dtype) || batch <= 0 || seq <= 0 || n_rows <= 0 || n_heads <= 0 || n_kv_heads <= 0 ||
        head_dim <= 0 || n_heads % n_kv_heads != 0 || !q || !k_cache || !scores || !lse || !drift)
        return POLESTAR_ERR_INVALID_ARGUMENT;
    if ((head_dim != 64 && head_dim != 128) || n_rows > kQkMaxRows || !aligned16(q) || !aligned16(k_cache) ||
        batch > 65535 || n_heads > 65535)
        return POLESTAR_ERR_UNSUPPORTED;
    const QklPlan p = qkl_plan(batch, seq, n_rows, n_heads);
    if (workspace_bytes < p.part_bytes || !workspace) return POLESTAR_ERR_WORKSPACE;
    return run_qkl(dtype == POLESTAR_BF16, batch, seq, n_rows, n_heads, n_kv_heads, head_dim,
                   static_cast<const char*>(q), static_cast<const char*>(k_cache), scale, scores, lse, first,
                   static_cast<float*>(workspace), drift, stream);
}

extern "C" polestar_status polestar_cluster_select(int batch, int seq, const int32_t* labels, int n_clusters,
                                                   const float* drift, int k_top, int32_t* stale_idx, int k_max,
                                                   int32_t* stale_count, hipStream_t stream) {
    using namespace ps;
    if (batch <= 0 || seq <= 0 || n_clusters <= 0 || k_top < 0 || k_max < 0 || !labels || !drift ||
        !stale_count || (k_max > 0 && !stale_idx))
        return POLESTAR_ERR_INVALID_ARGUMENT;
    if (n_clusters > kMaxClusters || batch > 65535) return POLESTAR_ERR_UNSUPPORTED;
    hipLaunchKernelGGL(cluster_select_kernel, dim3(batch), dim3(256), 0, stream, labels, seq, drift, n_clusters,
                       k_top, stale_idx, k_max, stale_count);
    return launch_status();
}

extern "C" polestar_status polestar_cluster_update(polestar_dtype dtype, int batch, int seq, int d,
                                                   const void* h_new, const void* h_old, const int32_t* labels,
                                                   int n_clusters, const int32_t* stale_idx,
                                                   const int32_t* stale_count, int k_max, float* sums,
                                                   hipStream_t stream) {
    using namespace ps;
    if (!dtype_ok(dtype) || batch <= 0 || seq <= 0 || d <= 0 || n_clusters <= 0 || k_max < 0 || !h_new ||
        !h_old || !labels || !stale_count || !sums || (k_max > 0 && !stale_idx))
        return POLESTAR_ERR_INVALID_ARGUMENT;
    if (n_clusters > kMaxClusters || batch > 65535 || d % 4 != 0) return POLESTAR_ERR_UNSUPPORTED;
    if (k_max == 0) return POLESTAR_OK;
    const dim3 grid(ceil_div(d, 1024), batch);
    if (dtype == POLESTAR_BF16)
        hipLaunchKernelGGL((cluster_update_kernel<true>), grid, dim3(256), 0, stream,
                           static_cast<const char*>(h_new), static_cast<const char*>(h_old), seq, d, labels,
                           n_clusters, stale_idx, stale_count, k_max, sums);
    else
        hipLaunchKernelGGL((cluster_update_kernel<false>), grid, dim3(256), 0, stream,
                           static_cast<const char*>(h_new), static_cast<const char*>(h_old), seq, d, labels,
                           n_clusters, stale_idx, stale_count, k_max, sums);
    return launch_status();
}
