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
constexpr long kMaxProxyScores = 36864;      // K * (seq + head_dim) floats in LDS (144 KB)
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

// Scores and drift of one (sequence b, head h), all K clusters at once:
//   1. the K queries of head h go to LDS (fp32);
//   2. thread j loads key row j (16-byte loads) and writes the K scores
//      s_(k,j) to LDS (sc[k][j], fp32);
//   3. wave w takes clusters w, w+4, ...: max and sum of exp over j (shuffles)
//      give lse; then KL_(k,h) = sum_j p_j ((s_j - lse) - (s'_j - lse')) with
//      the previous scores s' read from `prev`, which then receives s_j, and
//      lse replaces lse'.
// The per-head KL goes to kl[b][k][h]; head_mean_kernel averages it.
constexpr int kPdBlock = 1024;
constexpr int kPdPer = 16;                  // positions per lane per pass of the KL stage

template <bool BF16, int HD>
__global__ __launch_bounds__(kPdBlock) void proxy_kl_kernel(const char* __restrict__ q, const char* __restrict__ kc,
                                                            int seq, int K, int H, int Hkv, float scale,
                                                            float* __restrict__ prev, float* __restrict__ prev_lse,
                                                            int first, float* __restrict__ kl) {
    extern __shared__ float sm[];               // [K][HD] queries, then [K][seq] scores
    float* qs = sm;
    float* sc = sm + K * HD;
    using T = Elem<BF16>;
    constexpr int ES = T::kBytes;
    constexpr int E = T::E;
    constexpr int NC = HD * ES / 16;            // 16-byte chunks of a key row
    const int h = blockIdx.x, b = blockIdx.y;
    const int g = h / (H / Hkv);
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    for (int e = t; e < K * HD; e += kPdBlock) {
        const int k = e / HD, c = e - k * HD;
        qs[e] = load_elem<BF16>(q + ((static_cast<size_t>(b) * K + k) * H + h) * HD * ES, c);
    }
    __syncthreads();
    // scores: thread per key; the key row's chunks are loaded together, then
    // every cluster's dot product is accumulated chunk by chunk
    for (int j = t; j < seq; j += kPdBlock) {
        const char* kr = kc + ((static_cast<size_t>(b) * seq + j) * Hkv + g) * HD * ES;
        float acc[kMaxClusters];
#pragma unroll
        for (int k = 0; k < kMaxClusters; ++k) acc[k] = 0.f;
        constexpr int G = NC < 16 ? NC : 16;    // chunks held at once
        uint4 raw[G];
#pragma unroll
        for (int cc = 0; cc < NC; ++cc) {
            if (cc % G == 0) {
#pragma unroll
                for (int u = 0; u < G; ++u) raw[u] = ld16(kr + 16 * (cc + u));
            }
            float kv[E];
            T::unpack(raw[cc % G], kv);
#pragma unroll
            for (int k = 0; k < kMaxClusters; ++k) {
                if (k < K) {
                    const float4* qk = reinterpret_cast<const float4*>(qs + k * HD + cc * E);   // broadcast
#pragma unroll
                    for (int e4 = 0; e4 < E / 4; ++e4) {
                        const float4 qv = qk[e4];
                        acc[k] = fmaf(qv.x, kv[4 * e4], acc[k]);
                        acc[k] = fmaf(qv.y, kv[4 * e4 + 1], acc[k]);
                        acc[k] = fmaf(qv.z, kv[4 * e4 + 2], acc[k]);
                        acc[k] = fmaf(qv.w, kv[4 * e4 + 3], acc[k]);
                    }
                }
            }
        }
#pragma unroll
        for (int k = 0; k < kMaxClusters; ++k)
            if (k < K) sc[k * seq + j] = acc[k] * scale;
    }
    __syncthreads();
    // KL per cluster: wave per cluster; the previous scores of a pass of
    // kPdPer positions per lane are loaded before they are used
    for (int k = w; k < K; k += kPdBlock / kWave) {
        const float* srow = sc + k * seq;
        float m = -INFINITY;
        for (int j = lane; j < seq; j += kWave) m = fmaxf(m, srow[j]);
        m = wave_max(m);
        float z = 0.f;
        for (int j = lane; j < seq; j += kWave) z += fast_exp2((srow[j] - m) * kLog2e);
        z = wave_sum(z);
        const float lse = m + logf(z);
        const size_t rowid = (static_cast<size_t>(b) * K + k) * H + h;
        const float lse_prev = prev_lse[rowid];
        float* pr = prev + rowid * seq;
        float acc = 0.f;
        for (int j0 = 0; j0 < seq; j0 += kWave * kPdPer) {
            float pv[kPdPer];
#pragma unroll
            for (int u = 0; u < kPdPer; ++u) pv[u] = pr[min(j0 + u * kWave + lane, seq - 1)];
#pragma unroll
            for (int u = 0; u < kPdPer; ++u) {
                const int j = j0 + u * kWave + lane;
                if (j < seq) {
                    const float sj = srow[j];
                    const float lp = sj - lse;
                    acc = first ? acc : fmaf(fast_exp2(lp * kLog2e), lp - (pv[u] - lse_prev), acc);
                    pr[j] = sj;
                }
            }
        }
        acc = wave_sum(acc);
        if (lane == 0) {
            kl[rowid] = first ? 0.f : acc;
            prev_lse[rowid] = lse;
        }
    }
}

// drift[b][k] = mean over heads of kl[b][k][h], summed in head order.
__global__ __launch_bounds__(256) void head_mean_kernel(const float* __restrict__ kl, int BK, int H,
                                                        float* __restrict__ drift) {
    const int bk = blockIdx.x * 256 + threadIdx.x;
    if (bk >= BK) return;
    float s = 0.f;
    for (int h = 0; h < H; ++h) s += kl[static_cast<size_t>(bk) * H + h];
    drift[bk] = s / static_cast<float>(H);
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
// the per-head KL.
struct ProxyLayout {
    GemmPlan qp;
    size_t tok, q, gemm, kl, total;
};

ProxyLayout proxy_layout(bool bf16, int batch, int seq, int d, int H, int hd, int K) {
    ProxyLayout L{};
    const size_t es = bf16 ? 2 : 4;
    L.qp = gemm_plan(bf16, static_cast<long>(batch) * K, H * hd, d);
    L.tok = 0;
    L.q = align_up(static_cast<size_t>(batch) * K * d * es, 256);
    L.gemm = L.q + align_up(static_cast<size_t>(batch) * K * H * hd * es, 256);
    L.kl = L.gemm + align_up(L.qp.ws_bytes, 256);
    L.total = L.kl + align_up(static_cast<size_t>(batch) * K * H * sizeof(float), 256);
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
        batch > 65535 || n_heads > 65535 ||
        static_cast<long>(n_clusters) * (seq + head_dim) > kMaxProxyScores)
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
    const float sc = scale > 0.f ? scale : 1.0f / sqrtf(static_cast<float>(head_dim));
    const dim3 pgrid(n_heads, batch);
    const size_t plds = (static_cast<size_t>(n_clusters) * head_dim + static_cast<size_t>(n_clusters) * seq) *
                        sizeof(float);
    float* kl = reinterpret_cast<float*>(ws + L.kl);
    const char* qb = ws + L.q;
    const char* kcb = static_cast<const char*>(k_cache);
    if (bf16) {
        if (head_dim == 128) hipLaunchKernelGGL((proxy_kl_kernel<true, 128>), pgrid, dim3(kPdBlock), plds, stream, qb, kcb, seq, n_clusters, n_heads, n_kv_heads, sc, scores, lse, first, kl);
        else hipLaunchKernelGGL((proxy_kl_kernel<true, 64>), pgrid, dim3(kPdBlock), plds, stream, qb, kcb, seq, n_clusters, n_heads, n_kv_heads, sc, scores, lse, first, kl);
    } else {
        if (head_dim == 128) hipLaunchKernelGGL((proxy_kl_kernel<false, 128>), pgrid, dim3(kPdBlock), plds, stream, qb, kcb, seq, n_clusters, n_heads, n_kv_heads, sc, scores, lse, first, kl);
        else hipLaunchKernelGGL((proxy_kl_kernel<false, 64>), pgrid, dim3(kPdBlock), plds, stream, qb, kcb, seq, n_clusters, n_heads, n_kv_heads, sc, scores, lse, first, kl);
    }
    st = launch_status();
    if (st != POLESTAR_OK) return st;
    hipLaunchKernelGGL(head_mean_kernel, dim3(ceil_div(BK, 256)), dim3(256), 0, stream, kl, BK, n_heads, drift);
    return launch_status();
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
