// Device side of polestar_attend, shared by attend.hip and the fused step.
// (Grouped KV heads take attend_group_kernel, described at its definition.)
//
// Bidirectional attention of the active block over the whole
// cache (Sec. 2, eq. 3: queries of J_b attend to the cached K/V of I and the
// recomputed K/V of J_b, here all held in the refreshed cache; App. B setup:
// l = q.k / sqrt(d_h), a = softmax(l), o = sum a v).  No causal mask.
//
// The queries come from the Q projection (the shared skinny GEMM of
// gemm.hip).  Split-key flash attention:
//  - workgroup = (sequence b, query head h, group of 32 queries, key split);
//    its 4 waves take 32-key tiles in turn and keep an online softmax;
//  - S^T = K Q^T on MFMA with K as the A operand, so each lane ends up with
//    the scores of one query for 8 keys -- exactly the B-operand slice of
//    O^T = V^T P^T.  V^T is staged in LDS with its keys in the same order;
//  - the 4 waves are merged in LDS; with one split the workgroup writes the
//    output directly, otherwise (m, l, O) partials go to the workspace and a
//    merge kernel combines the splits in order with their log-sum-exp.
// Scores are kept in base-2 units (scale * log2 e folded in) for exp2.
#pragma once

#include "common.hpp"
#include "host_common.hpp"

namespace ps {
namespace {

constexpr int kAttBlock = 256;   // 4 waves
constexpr int kQG = 32;          // queries per workgroup
constexpr int kKT = 32;          // keys per tile
constexpr float kLazy = 8.f;     // log2 headroom of the lazy softmax reference

}  // namespace

// Outside the anonymous namespace: the ring kernel (attend_ring.hip) is
// launched from the other files through launch_att_ring.
struct AttArgs {
    const char* q;       // [batch][nq][H][hd]
    const char* k;       // [batch][seq][Hkv][hd]
    const char* v;
    char* out;           // [batch][nq][H][hd]
    float* lse;          // [batch][H][nq] or null
    float* part_o;       // [batch][H][nq][splits][hd]
    float* part_ml;      // [batch][H][nq][splits][2]
    int batch, seq, nq, H, Hkv;
    int splits, tiles_per_split;
    float scale_log2;    // scale * log2(e)
};

// attend_ring_kernel<hd> over `grid` (attend_ring.hip; hd 64 or 128, bf16).
void launch_att_ring(int hd, dim3 grid, const AttArgs& a, hipStream_t s);

namespace {

// Position of key kk (0..31) of a tile in the LDS row of V^T: lane group g
// reads slots 8g..8g+7 = keys 4g..4g+3 and 16+4g..16+4g+3 (bf16 path).
__device__ __forceinline__ int vslot(int kk) {
    return kk < 16 ? 8 * (kk >> 2) + (kk & 3) : 8 * ((kk - 16) >> 2) + 4 + (kk & 3);
}

// Physical LDS row of V^T row r (d index) in attend_kernel's bf16 path.  A
// transposing store instruction writes rows 8 dc + e (dc = 16-byte chunk of
// d, one per lane, e fixed), which with the 80-byte pitch fall on only two
// bank offsets; XOR-ing the low three bits of the row with bits 4..6 spreads
// them over 16, while the fragment reads (16 consecutive rows) stay a
// permutation of 16 rows.
__device__ __forceinline__ int vrow(int r) { return r ^ ((r >> 4) & 7); }

template <bool BF16, int HD>
__global__ __launch_bounds__(kAttBlock, 2) void attend_kernel(AttArgs a) {
    using T = Elem<BF16>;
    constexpr int ES = T::kBytes;
    constexpr int NC = HD * ES / 64;        // 16-byte chunks of one lane's d-range
    constexpr int DPL = HD / 4;             // d values per lane group
    constexpr int DT = HD / 16;             // 16-row d tiles of O^T
    // V^T rows: bf16 32 keys (64 B) + 16 B pad; fp32 32 keys (128 B) + 16 B pad
    constexpr int VP = BF16 ? 80 : 144;
    // The V^T staging of the loop and the wave merge after it share one LDS
    // array (two workgroups fit per CU instead of one).
    constexpr int kVtBytes = 4 * HD * VP;
    constexpr int kWoBytes = 4 * kQG * (HD + 4) * 4;
    __shared__ __align__(16) char smem[kVtBytes > kWoBytes ? kVtBytes : kWoBytes];
    __shared__ float wm[4][kQG], wl[4][kQG];
    auto wo = reinterpret_cast<float (*)[kQG][HD + 4]>(smem);

    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const int g = lane >> 4;
    const int split = blockIdx.x;
    const int qgroups = (a.nq + kQG - 1) / kQG;
    const int h = blockIdx.y / qgroups;
    const int qg = blockIdx.y - h * qgroups;
    const int b = blockIdx.z;
    const int kvh = h / (a.H / a.Hkv);

    const size_t krow = static_cast<size_t>(a.Hkv) * HD * ES;   // bytes per cache row
    const char* kbase = a.k + (static_cast<size_t>(b) * a.seq * a.Hkv + kvh) * HD * ES;
    const char* vbase = a.v + (static_cast<size_t>(b) * a.seq * a.Hkv + kvh) * HD * ES;

    // Q fragments (B operand of S^T): query 16u + (lane & 15), d in [DPL g, DPL g + DPL).
    // All loads are unconditional: queries past nq and keys past seq read the
    // last row (finite values whose results are masked or never stored), so
    // no load sits behind an exec mask and the wait counts stay static.
    uint4 qf[2][NC];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int q = min(qg * kQG + 16 * u + (lane & 15), a.nq - 1);
        const char* qp = a.q + ((static_cast<size_t>(b) * a.nq + q) * a.H + h) * HD * ES + g * DPL * ES;
#pragma unroll
        for (int c = 0; c < NC; ++c) qf[u][c] = ld16(qp + 16 * c);
    }

    floatx4 o[DT][2];
#pragma unroll
    for (int i = 0; i < DT; ++i) o[i][0] = o[i][1] = floatx4{0.f, 0.f, 0.f, 0.f};
    float mrun[2] = {-INFINITY, -INFINITY};
    float lrun[2] = {0.f, 0.f};

    const int ntiles = (a.seq + kKT - 1) / kKT;
    const int t_begin = split * a.tiles_per_split;
    const int t_end = min(ntiles, t_begin + a.tiles_per_split);
    // Each wave stages and reads only its own V^T region, so no workgroup
    // barrier is needed until the waves are merged.
    char* myvt = smem + w * HD * VP;
    const int wu = __builtin_amdgcn_readfirstlane(w);   // wave-uniform tile choice

    // K fragments (A operand of S^T: key key0 + 16 t + (lane & 15)) and the V
    // tile (item pr = lane + 64 it: 4 keys x one 16-byte chunk of d) of one
    // tile, loaded into registers.  In bf16 the next tile's loads are issued
    // as soon as this tile's registers are consumed -- V transposed into LDS,
    // the score MFMAs issued -- so they are in flight during the softmax and
    // PV work instead of after it.
    constexpr int DCV = BF16 ? HD / 8 : HD / 4;   // 16-byte chunks of a V row
    constexpr int ITV = DCV * 8 / 64;
    uint4 kf[2][NC];
    uint4 vv[ITV][4];
    // V item `it` of this lane: 16-byte chunk dc of d for the 4 keys of group
    // kg.  bf16: the 4 key groups a store instruction covers are it, it + IT,
    // it + 2 IT, ... so that they use both 8-byte halves of a 16-byte slot
    // group (with vrow, a 2-way bank conflict, the minimum for a 512-byte
    // store); the loads stay 256 contiguous bytes per 16 lanes.
    auto vitem = [&](int it, int& dc, int& kg) {
        if constexpr (BF16) {
            dc = lane % DCV;
            kg = it + ITV * (lane / DCV);
        } else {
            const int pr = lane + 64 * it;
            dc = pr % DCV;
            kg = pr / DCV;
        }
    };
    auto load_tile = [&](int tile) {
        const int key0 = tile * kKT;
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            const int key = min(key0 + 16 * t + (lane & 15), a.seq - 1);
            const char* kp = kbase + static_cast<size_t>(key) * krow + g * DPL * ES;
#pragma unroll
            for (int c = 0; c < NC; ++c) kf[t][c] = ld16(kp + 16 * c);
        }
#pragma unroll
        for (int it = 0; it < ITV; ++it) {
            int dc, kg;
            vitem(it, dc, kg);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int key = min(key0 + 4 * kg + j, a.seq - 1);
                vv[it][j] = ld16(vbase + static_cast<size_t>(key) * krow + dc * 16);
            }
        }
    };

    // Wave w takes tiles t_begin + w, t_begin + w + 4, ... (no barrier inside
    // the loop, so the waves' trip counts may differ).
    int tile = t_begin + wu;
    if constexpr (BF16) {
        if (tile < t_end) load_tile(tile);
    }
    for (; tile < t_end; tile += 4) {
        {
            // fp32 tiles are twice as wide: there the registers do not hold
            // the next tile across the softmax and PV work, so it loads here
            if constexpr (!BF16) load_tile(tile);
            const int key0 = tile * kKT;
            floatx4 st[2][2];
            // V tile (loaded into vv) -> LDS, transposed to [d][key slot].
            if constexpr (BF16) {
                // 8 groups of 4 keys x HD/8 chunks of 8 d; item pr = lane + 64 it
                constexpr int DC = HD / 8;
                constexpr int IT = DC * 8 / 64;
#pragma unroll
                for (int it = 0; it < IT; ++it) {
                    int dc, kg;
                    vitem(it, dc, kg);
                    const uint32_t* x0 = reinterpret_cast<const uint32_t*>(&vv[it][0]);
                    const uint32_t* x1 = reinterpret_cast<const uint32_t*>(&vv[it][1]);
                    const uint32_t* x2 = reinterpret_cast<const uint32_t*>(&vv[it][2]);
                    const uint32_t* x3 = reinterpret_cast<const uint32_t*>(&vv[it][3]);
                    const int slot = vslot(4 * kg);
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        // d = 8 dc + e of the 4 keys: the low (e even) or high
                        // (e odd) halves of word e / 2, two keys per byte permute
                        const uint32_t sel = (e & 1) ? 0x07060302u : 0x05040100u;
                        const uint2 pk = make_uint2(__builtin_amdgcn_perm(x1[e >> 1], x0[e >> 1], sel),
                                                    __builtin_amdgcn_perm(x3[e >> 1], x2[e >> 1], sel));
                        *reinterpret_cast<uint2*>(myvt + vrow(dc * 8 + e) * VP + slot * 2) = pk;
                    }
                }
            } else {
                constexpr int DC = HD / 4;
                constexpr int IT = DC * 8 / 64;
#pragma unroll
                for (int it = 0; it < IT; ++it) {
                    int dc, kg;
                    vitem(it, dc, kg);
                    const uint32_t* x0 = reinterpret_cast<const uint32_t*>(&vv[it][0]);
                    const uint32_t* x1 = reinterpret_cast<const uint32_t*>(&vv[it][1]);
                    const uint32_t* x2 = reinterpret_cast<const uint32_t*>(&vv[it][2]);
                    const uint32_t* x3 = reinterpret_cast<const uint32_t*>(&vv[it][3]);
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        *reinterpret_cast<uint4*>(myvt + (dc * 4 + e) * VP + 16 * kg) =
                            make_uint4(x0[e], x1[e], x2[e], x3[e]);
                }
            }
            // S^T tiles: st[t][u] = K_t Q_u^T.
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    floatx4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int c = 0; c < NC; ++c) s = Mma<BF16>::step(kf[t][c], qf[u][c], s);
                    st[t][u] = s;
                }
            if constexpr (BF16) {
                if (tile + 4 < t_end) load_tile(tile + 4);
            }
            // Keys past seq exist only in a partial last tile.
            if (__builtin_expect(key0 + kKT > a.seq, 0)) {
#pragma unroll
                for (int t = 0; t < 2; ++t)
#pragma unroll
                    for (int u = 0; u < 2; ++u)
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            if (key0 + 16 * t + 4 * g + i >= a.seq) st[t][u][i] = -INFINITY;
            }
            // Online softmax in base-2 units with a lazy exponent reference:
            // the reference moves (and O, l are rescaled) only when some
            // query's maximum exceeds it by more than kLazy, so exponents stay
            // below 2^kLazy; (m, l, O) are exact for any reference.
            float p[2][2][4];   // [t][u][i]
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                float mx = -INFINITY;
#pragma unroll
                for (int t = 0; t < 2; ++t)
#pragma unroll
                    for (int i = 0; i < 4; ++i) mx = fmaxf(mx, st[t][u][i]);
                mx = fmaxf(mx, __shfl_xor(mx, 16));
                mx = fmaxf(mx, __shfl_xor(mx, 32));
                const float mcand = fmaxf(mrun[u], mx * a.scale_log2);
                const bool any = __builtin_amdgcn_ballot_w64(mcand > mrun[u] + kLazy) != 0;
                const float alpha = any ? fast_exp2(mrun[u] - (mcand == -INFINITY ? 0.f : mcand)) : 1.f;
                if (any) mrun[u] = mcand;
                const float mref = mrun[u] == -INFINITY ? 0.f : mrun[u];
                float sum = 0.f;
#pragma unroll
                for (int t = 0; t < 2; ++t)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const float e = fast_exp2(fmaf(st[t][u][i], a.scale_log2, -mref));
                        p[t][u][i] = e;
                        sum += e;
                    }
                sum += __shfl_xor(sum, 16);
                sum += __shfl_xor(sum, 32);
                lrun[u] = fmaf(lrun[u], alpha, sum);
                if (any) {
#pragma unroll
                    for (int dt = 0; dt < DT; ++dt) o[dt][u] *= alpha;
                }
            }
            // O^T += V^T P^T
            if constexpr (BF16) {
                uint4 pf[2];
#pragma unroll
                for (int u = 0; u < 2; ++u)
                    pf[u] = make_uint4(cvt_pk_bf16(p[0][u][0], p[0][u][1]), cvt_pk_bf16(p[0][u][2], p[0][u][3]),
                                       cvt_pk_bf16(p[1][u][0], p[1][u][1]), cvt_pk_bf16(p[1][u][2], p[1][u][3]));
#pragma unroll
                for (int dt = 0; dt < DT; ++dt) {
                    const uint4 va = *reinterpret_cast<const uint4*>(myvt + vrow(dt * 16 + (lane & 15)) * VP + g * 16);
#pragma unroll
                    for (int u = 0; u < 2; ++u) o[dt][u] = mfma_bf16(va, pf[u], o[dt][u]);
                }
            } else {
#pragma unroll
                for (int dt = 0; dt < DT; ++dt) {
                    const float* vrow = reinterpret_cast<const float*>(myvt + (dt * 16 + (lane & 15)) * VP);
#pragma unroll
                    for (int t = 0; t < 2; ++t)
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const float va = vrow[16 * t + 4 * g + i];
#pragma unroll
                            for (int u = 0; u < 2; ++u) o[dt][u] = mfma_f32(va, p[t][u][i], o[dt][u]);
                        }
                }
            }
        }
    }

    // Merge the four waves.  Lane holds O^T[d = 16 dt + 4 g + i][q = 16 u + (lane & 15)].
    // The merge buffer overlays the V^T staging: every wave must be done with
    // its tiles first (all waves run the same number of loop trips).
    __syncthreads();
    if (lane < 16) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            wm[w][16 * u + lane] = mrun[u];
            wl[w][16 * u + lane] = lrun[u];
        }
    }
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int i = 0; i < 4; ++i) wo[w][16 * u + (lane & 15)][dt * 16 + 4 * g + i] = o[dt][u][i];
    __syncthreads();

    // Each thread finishes 32*HD/256 outputs: query qi, d range.
    constexpr int PER = kQG * HD / kAttBlock;   // 8 (HD 64) or 16 (HD 128)
    const int qi = threadIdx.x / (HD / PER);
    const int d0 = (threadIdx.x % (HD / PER)) * PER;
    const int q = qg * kQG + qi;
    float M = -INFINITY;
#pragma unroll
    for (int ww = 0; ww < 4; ++ww) M = fmaxf(M, wm[ww][qi]);
    const float Mref = M == -INFINITY ? 0.f : M;
    float wgt[4], L = 0.f;
#pragma unroll
    for (int ww = 0; ww < 4; ++ww) {
        wgt[ww] = fast_exp2(wm[ww][qi] - Mref);
        L += wl[ww][qi] * wgt[ww];
    }
    float acc[PER];
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        float s = 0.f;
#pragma unroll
        for (int ww = 0; ww < 4; ++ww) s += wo[ww][qi][d0 + j] * wgt[ww];
        acc[j] = s;
    }
    if (q >= a.nq) return;
    const size_t row = (static_cast<size_t>(b) * a.nq + q) * a.H + h;   // [b][q][h]
    if (a.splits == 1) {
        const float inv = 1.f / L;
        char* op = a.out + (row * HD + d0) * ES;
#pragma unroll
        for (int j = 0; j < PER; j += 8) {
            if constexpr (BF16) {
                st16(op + 2 * j, make_uint4(pack_bf16x2(acc[j] * inv, acc[j + 1] * inv),
                                            pack_bf16x2(acc[j + 2] * inv, acc[j + 3] * inv),
                                            pack_bf16x2(acc[j + 4] * inv, acc[j + 5] * inv),
                                            pack_bf16x2(acc[j + 6] * inv, acc[j + 7] * inv)));
            } else {
                float* fp = reinterpret_cast<float*>(op) + j;
                *reinterpret_cast<float4*>(fp) = make_float4(acc[j] * inv, acc[j + 1] * inv,
                                                             acc[j + 2] * inv, acc[j + 3] * inv);
                *reinterpret_cast<float4*>(fp + 4) = make_float4(acc[j + 4] * inv, acc[j + 5] * inv,
                                                                 acc[j + 6] * inv, acc[j + 7] * inv);
            }
        }
        if (a.lse && d0 == 0)
            a.lse[(static_cast<size_t>(b) * a.H + h) * a.nq + q] = (M + __log2f(L)) * kLn2;
    } else {
        const size_t prow = ((static_cast<size_t>(b) * a.H + h) * a.nq + q) * a.splits + split;
        float* po = a.part_o + prow * HD + d0;
#pragma unroll
        for (int j = 0; j < PER; j += 4)
            *reinterpret_cast<float4*>(po + j) = make_float4(acc[j], acc[j + 1], acc[j + 2], acc[j + 3]);
        if (d0 == 0) {
            a.part_ml[prow * 2] = M;
            a.part_ml[prow * 2 + 1] = L;
        }
    }
}

// Combine the key splits of one (b, h, q) row: one wave per row, lanes over d.
// Splits are taken eight at a time with every load of the chunk issued
// before any arithmetic (indices clamped, extra splits weighted zero), and
// merged in split order with a running maximum.
template <bool BF16, int HD>
__device__ __forceinline__ void merge_body(const AttArgs& a, int blk) {
    constexpr int ES = Elem<BF16>::kBytes;
    constexpr int PL = HD / 64;   // d values per lane (1 or 2)
    constexpr int CH = 8;         // splits per chunk
    const int lane = threadIdx.x & 63;
    const long rowid = static_cast<long>(blk) * 4 + (threadIdx.x >> 6);   // over [b][h][q]
    const long nrows = static_cast<long>(a.batch) * a.H * a.nq;
    if (rowid >= nrows) return;
    const int q = static_cast<int>(rowid % a.nq);
    const long bh = rowid / a.nq;
    const int h = static_cast<int>(bh % a.H);
    const int b = static_cast<int>(bh / a.H);
    const size_t prow0 = static_cast<size_t>(rowid) * a.splits;
    float M = -INFINITY, L = 0.f, acc[PL];
#pragma unroll
    for (int j = 0; j < PL; ++j) acc[j] = 0.f;
    for (int s0 = 0; s0 < a.splits; s0 += CH) {
        float2 ml[CH];
        float po[CH][PL];
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const size_t pr = prow0 + min(s0 + c, a.splits - 1);
            ml[c] = *reinterpret_cast<const float2*>(a.part_ml + pr * 2);
#pragma unroll
            for (int j = 0; j < PL; ++j) po[c][j] = a.part_o[pr * HD + lane * PL + j];
        }
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const float m = s0 + c < a.splits ? ml[c].x : -INFINITY;
            const float mn = fmaxf(M, m);
            const float mref = mn == -INFINITY ? 0.f : mn;
            const float wold = fast_exp2(M - mref), wnew = fast_exp2(m - mref);
            L = L * wold + ml[c].y * wnew;
#pragma unroll
            for (int j = 0; j < PL; ++j) acc[j] = acc[j] * wold + po[c][j] * wnew;
            M = mn;
        }
    }
    const float inv = 1.f / L;
    const size_t row = (static_cast<size_t>(b) * a.nq + q) * a.H + h;
    char* op = a.out + (row * HD + lane * PL) * ES;
    if constexpr (BF16) {
        if constexpr (PL == 2) *reinterpret_cast<uint32_t*>(op) = pack_bf16x2(acc[0] * inv, acc[1] * inv);
        else *reinterpret_cast<uint16_t*>(op) = static_cast<uint16_t>(f32_to_bf16_bits(acc[0] * inv));
    } else {
#pragma unroll
        for (int j = 0; j < PL; ++j) reinterpret_cast<float*>(op)[j] = acc[j] * inv;
    }
    if (a.lse && lane == 0) a.lse[(static_cast<size_t>(b) * a.H + h) * a.nq + q] = (M + __log2f(L)) * kLn2;
}

// Grouped-query attention (bf16).  The H / Hkv query heads of a KV group all
// read that group's K/V, so the workgroup is (sequence b, KV head, row block,
// key split): its NW waves each own one (query head, 32-query group) pair of
// the group and walk the same keys, which the whole workgroup stages once in
// LDS -- K as [key][d] rows, V^T as [d][key slot] rows -- 64 keys per step,
// double-buffered with one barrier per step (the next step's loads are in
// flight while the current one is computed).  Both products run on
// v_mfma_f32_32x32x16_bf16 (on gfx950 twice the rate of the 16x16x32 form):
// S^T = K Q^T for 32 keys x the wave's 32 queries, then O^T += V^T P^T, 16
// keys at a time.  A lane ends S^T with 16 scores of one query (query
// lane % 32), which are exactly the eight-key slices of P^T that the second
// product takes as its B operand -- keys 4h..4h+3 and 8+4h..8+4h+3 of each
// 16-key block for lane half h -- so V^T is staged with the 4-key groups of a
// block in slot order 0, 2, 1, 3 and the probabilities never leave the
// registers.  There is no wave merge: each wave writes its own output (one
// split) or its (m, l, O) partial in the layout the merge kernel reads.
// Waves past the group's last pair help stage and skip the arithmetic.
constexpr int kGKT = 64;   // keys per step of the grouped kernel

// LDS slot of the first key of 4-key group kg (0..15) of a step in a V^T row.
__device__ __forceinline__ int gslot(int kg) {
    constexpr int kOrder[4] = {0, 8, 4, 12};
    return 16 * (kg >> 2) + kOrder[kg & 3];
}

template <int HD, int NW>
__global__ __launch_bounds__(64 * NW) void attend_group_kernel(AttArgs a) {
    constexpr int NT = 64 * NW;
    constexpr int KS = HD / 16;              // 16-wide d steps of S^T = K Q^T
    constexpr int DT = HD / 32;              // 32-row d tiles of O^T
    constexpr int KP = HD * 2 + 16;          // K row + 16 B pad
    constexpr int VP = kGKT * 2 + 16;        // V^T row: 64 key slots + 16 B pad (16-row reads on distinct banks)
    constexpr int KCH = kGKT * HD * 2 / 16;  // 16-byte chunks of a step's K
    constexpr int KI = (KCH + NT - 1) / NT;
    constexpr int VU = (kGKT / 4) * (HD / 2);   // V staging units: 4 keys x 2 d
    constexpr int VI = (VU + NT - 1) / NT;
    __shared__ __align__(16) char ks[2][kGKT * KP];
    __shared__ __align__(16) char vs[2][HD * VP];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int l32 = lane & 31, h32 = lane >> 5;
    const int w = tid >> 6;
    const int split = blockIdx.x;
    const int G = a.H / a.Hkv;
    const int qgroups = (a.nq + kQG - 1) / kQG;
    const int npairs = G * qgroups;
    const int pair_raw = blockIdx.y * NW + w;
    const bool active = pair_raw < npairs;   // wave-uniform
    const int pair = min(pair_raw, npairs - 1);
    const int hh = pair / qgroups;
    const int qg = pair - hh * qgroups;
    const int b = blockIdx.z / a.Hkv;
    const int kvh = blockIdx.z - b * a.Hkv;
    const int h = kvh * G + hh;

    const size_t krow = static_cast<size_t>(a.Hkv) * HD * 2;   // bytes per cache row
    const char* kbase = a.k + (static_cast<size_t>(b) * a.seq * a.Hkv + kvh) * HD * 2;
    const char* vbase = a.v + (static_cast<size_t>(b) * a.seq * a.Hkv + kvh) * HD * 2;

    // Q fragments (B operand of S^T: 16 d x 32 queries): query qg*32 + lane % 32,
    // d = 16 kk + 8 h32 .. +8.  Queries past nq read the last row (never stored).
    uint4 qf[KS];
    {
        const int q = min(qg * kQG + l32, a.nq - 1);
        const char* qp = a.q + ((static_cast<size_t>(b) * a.nq + q) * a.H + h) * HD * 2 + h32 * 16;
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) qf[kk] = ld16(qp + 32 * kk);
    }

    floatx16 o[DT];
#pragma unroll
    for (int i = 0; i < DT; ++i)
#pragma unroll
        for (int j = 0; j < 16; ++j) o[i][j] = 0.f;
    float mrun = -INFINITY, lrun = 0.f;

    const int nsteps = (a.seq + kGKT - 1) / kGKT;
    const int s_begin = split * a.tiles_per_split;
    const int s_end = min(nsteps, s_begin + a.tiles_per_split);

    // Staging registers of one step: K chunks (16 B) and V units (4 keys x 2 d).
    // Each thread's offsets inside a step are fixed: a step wholly inside the
    // sequence loads from the step's first row plus them; the last step of a
    // sequence whose length is not a multiple of 64 clamps its keys to the
    // last row (their scores are masked).  Indices past the step are clamped
    // on load and skipped on store.
    uint32_t koff[KI], voff[VI];
#pragma unroll
    for (int i = 0; i < KI; ++i) {
        const int c = min(tid + i * NT, KCH - 1);
        koff[i] = static_cast<uint32_t>((c / (HD / 8)) * krow + (c % (HD / 8)) * 16);
    }
#pragma unroll
    for (int i = 0; i < VI; ++i) {
        const int u = min(tid + i * NT, VU - 1);
        voff[i] = static_cast<uint32_t>(4 * (u / (HD / 2)) * krow + (u % (HD / 2)) * 4);
    }
    auto load_step = [&](int step, uint4 (&kr)[KI], uint32_t (&vr)[VI][4]) {
        const int key0 = step * kGKT;
        if (key0 + kGKT <= a.seq) {
            const char* kp = kbase + static_cast<size_t>(key0) * krow;
            const char* vp = vbase + static_cast<size_t>(key0) * krow;
#pragma unroll
            for (int i = 0; i < KI; ++i) kr[i] = ld16(kp + koff[i]);
#pragma unroll
            for (int i = 0; i < VI; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    vr[i][j] = *reinterpret_cast<const uint32_t*>((vp + j * krow) + voff[i]);
            return;
        }
#pragma unroll
        for (int i = 0; i < KI; ++i) {
            const int c = min(tid + i * NT, KCH - 1);
            const int key = min(key0 + c / (HD / 8), a.seq - 1);
            kr[i] = ld16(kbase + static_cast<size_t>(key) * krow + (c % (HD / 8)) * 16);
        }
#pragma unroll
        for (int i = 0; i < VI; ++i) {
            const int u = min(tid + i * NT, VU - 1);
            const int dp = u % (HD / 2), kg = u / (HD / 2);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int key = min(key0 + 4 * kg + j, a.seq - 1);
                vr[i][j] = *reinterpret_cast<const uint32_t*>(vbase + static_cast<size_t>(key) * krow + dp * 4);
            }
        }
    };
    auto store_step = [&](int buf, const uint4 (&kr)[KI], const uint32_t (&vr)[VI][4]) {
#pragma unroll
        for (int i = 0; i < KI; ++i) {
            const int c = tid + i * NT;
            if (KCH % NT == 0 || c < KCH)
                st16(ks[buf] + (c / (HD / 8)) * KP + (c % (HD / 8)) * 16, kr[i]);
        }
#pragma unroll
        for (int i = 0; i < VI; ++i) {
            const int u = tid + i * NT;
            if (VU % NT == 0 || u < VU) {
                const int dp = u % (HD / 2), kg = u / (HD / 2);
                const int slot = gslot(kg);
                // low halves (d = 2 dp) and high halves (d = 2 dp + 1) of the 4 keys
                const uint2 lo = make_uint2(__builtin_amdgcn_perm(vr[i][1], vr[i][0], 0x05040100u),
                                            __builtin_amdgcn_perm(vr[i][3], vr[i][2], 0x05040100u));
                const uint2 hi = make_uint2(__builtin_amdgcn_perm(vr[i][1], vr[i][0], 0x07060302u),
                                            __builtin_amdgcn_perm(vr[i][3], vr[i][2], 0x07060302u));
                *reinterpret_cast<uint2*>(vs[buf] + (2 * dp) * VP + slot * 2) = lo;
                *reinterpret_cast<uint2*>(vs[buf] + (2 * dp + 1) * VP + slot * 2) = hi;
            }
        }
    };
    auto compute_step = [&](int buf, int step) {
        const int key0 = step * kGKT;
        const char* kb = ks[buf];
        const char* vb = vs[buf];
        // S^T for the two 32-key tiles of the step; register j of st[kt] is key
        // key0 + 32 kt + mfma32_row(lane, j) of query lane % 32.
        floatx16 st[2];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
            floatx16 sacc;
#pragma unroll
            for (int j = 0; j < 16; ++j) sacc[j] = 0.f;
#pragma unroll
            for (int kk = 0; kk < KS; ++kk) {
                const uint4 kf = *reinterpret_cast<const uint4*>(kb + (32 * kt + l32) * KP + 32 * kk + 16 * h32);
                sacc = Mma32<true>::step(kf, qf[kk], sacc);
            }
            st[kt] = sacc;
        }
        // Keys past seq exist only in a partial last step.
        if (__builtin_expect(key0 + kGKT > a.seq, 0)) {
#pragma unroll
            for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                for (int j = 0; j < 16; ++j)
                    if (key0 + 32 * kt + mfma32_row(lane, j) >= a.seq) st[kt][j] = -INFINITY;
        }
        // Online softmax in base-2 units: the maximum of the raw scores times
        // the positive scale is the maximum of the scaled scores, and each
        // exponent is one fma of the raw score.
        float mx = -INFINITY;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int j = 0; j < 16; ++j) mx = fmaxf(mx, st[kt][j]);
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float mcand = fmaxf(mrun, mx * a.scale_log2);
        const bool any = __builtin_amdgcn_ballot_w64(mcand > mrun + kLazy) != 0;
        const float alpha = any ? fast_exp2(mrun - (mcand == -INFINITY ? 0.f : mcand)) : 1.f;
        if (any) mrun = mcand;
        const float mref = mrun == -INFINITY ? 0.f : mrun;
        float sum = 0.f;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const float e = fast_exp2(fmaf(st[kt][j], a.scale_log2, -mref));
                st[kt][j] = e;
                sum += e;
            }
        sum += __shfl_xor(sum, 32);
        lrun = fmaf(lrun, alpha, sum);
        if (any) {
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) o[dt] *= alpha;
        }
        // O^T += V^T P^T over the four 16-key blocks: the B operand is
        // registers 8 kb' .. 8 kb' + 7 of st[kt] (kb' = block within the tile).
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int kb2 = 0; kb2 < 2; ++kb2) {
                const int r = 8 * kb2;
                const uint4 pf = make_uint4(cvt_pk_bf16(st[kt][r + 0], st[kt][r + 1]),
                                            cvt_pk_bf16(st[kt][r + 2], st[kt][r + 3]),
                                            cvt_pk_bf16(st[kt][r + 4], st[kt][r + 5]),
                                            cvt_pk_bf16(st[kt][r + 6], st[kt][r + 7]));
                const int soff = (32 * kt + 16 * kb2 + 8 * h32) * 2;
#pragma unroll
                for (int dt = 0; dt < DT; ++dt) {
                    const uint4 va = *reinterpret_cast<const uint4*>(vb + (32 * dt + l32) * VP + soff);
                    o[dt] = Mma32<true>::step(va, pf, o[dt]);
                }
            }
    };

    // Three register sets: while step i is stored to LDS buffer i % 2, steps
    // i + 1 and i + 2 are being loaded (one step of compute does not cover a
    // global load's latency).  Buffer i % 2 is rewritten two steps after it
    // was read; the barrier of the step in between orders every wave's reads
    // before the rewrite.  The loop is unrolled by three so that the register
    // sets are fixed per position.
    constexpr int PD = 3;
    uint4 kr[PD][KI];
    uint32_t vr[PD][VI][4];
    const int n = s_end - s_begin;
#pragma unroll
    for (int j = 0; j < PD - 1; ++j)
        if (j < n) load_step(s_begin + j, kr[j], vr[j]);
    for (int base = 0; base < n; base += PD) {
#pragma unroll
        for (int j = 0; j < PD; ++j) {
            const int i = base + j;
            if (i < n) {
                store_step(i & 1, kr[j], vr[j]);
                if (i + PD - 1 < n) load_step(s_begin + i + PD - 1, kr[(j + PD - 1) % PD], vr[(j + PD - 1) % PD]);
                __syncthreads();
                if (active) compute_step(i & 1, s_begin + i);
            }
        }
    }
    if (!active) return;

    // Register j of o[dt] is O^T[d = 32 dt + mfma32_row(lane, j)][query lane % 32]:
    // groups of four consecutive d per lane.
    const int q = qg * kQG + l32;
    if (q >= a.nq) return;
    const size_t row = (static_cast<size_t>(b) * a.nq + q) * a.H + h;   // [b][q][h]
    if (a.splits == 1) {
        const float inv = 1.f / lrun;
        char* op = a.out + row * HD * 2;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int g4 = 0; g4 < 4; ++g4)
                *reinterpret_cast<uint2*>(op + (32 * dt + 8 * g4 + 4 * h32) * 2) =
                    make_uint2(pack_bf16x2(o[dt][4 * g4] * inv, o[dt][4 * g4 + 1] * inv),
                               pack_bf16x2(o[dt][4 * g4 + 2] * inv, o[dt][4 * g4 + 3] * inv));
        if (a.lse && h32 == 0)
            a.lse[(static_cast<size_t>(b) * a.H + h) * a.nq + q] = (mrun + __log2f(lrun)) * kLn2;
    } else {
        const size_t prow = ((static_cast<size_t>(b) * a.H + h) * a.nq + q) * a.splits + split;
        float* po = a.part_o + prow * HD;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int g4 = 0; g4 < 4; ++g4)
                *reinterpret_cast<float4*>(po + 32 * dt + 8 * g4 + 4 * h32) =
                    make_float4(o[dt][4 * g4], o[dt][4 * g4 + 1], o[dt][4 * g4 + 2], o[dt][4 * g4 + 3]);
        if (h32 == 0) {
            a.part_ml[prow * 2] = mrun;
            a.part_ml[prow * 2 + 1] = lrun;
        }
    }
}

struct AttPlan {
    int splits;
    int tiles_per_split;
    size_t part_bytes;   // partial O + (m, l)
    int group_waves;     // 0: attend_kernel; 8: attend_group_kernel (its tiles_per_split then counts
                         // 64-key steps)
    int row_blocks;      // grouped: workgroups per (sequence, KV head, split)
    bool ring;           // attend_ring_kernel (attend_ring.hip): one workgroup per CU, three tiles in flight per wave
};

// Plan of the attention launch.  Grouped heads (bf16, at least four (query
// head, 32-query group) pairs per KV head) take attend_group_kernel: 8-wave
// workgroups (two waves per SIMD), keys split so that about 256 workgroups
// run (one round, one per CU); each split adds an fp32 (m, l, O) partial per
// query row, so no more splits than that.  bf16 with at least four tiles per
// wave at about 256 workgroups: attend_ring_kernel.  Everything else
// attend_kernel.
inline AttPlan att_plan(bool bf16, int batch, int seq, int H, int Hkv, int nq, int hd) {
    AttPlan p{};
    const int ntiles = ceil_div(seq, kKT);
    const int npairs = (H / Hkv) * ceil_div(nq, kQG);
    if (bf16 && npairs >= 4 && static_cast<long>(batch) * Hkv <= 65535) {
        p.group_waves = 8;
        p.row_blocks = ceil_div(npairs, p.group_waves);
        const int nsteps = ceil_div(seq, kGKT);          // tiles_per_split counts 64-key steps
        const long base = static_cast<long>(batch) * Hkv * p.row_blocks;
        int splits = static_cast<int>(256 / base);
        if (splits > nsteps) splits = nsteps;
        if (splits < 1) splits = 1;
        p.tiles_per_split = ceil_div(nsteps, splits);
        p.splits = ceil_div(nsteps, p.tiles_per_split);
        if (p.splits > 1) {
            const size_t rows = static_cast<size_t>(batch) * H * nq * p.splits;
            p.part_bytes = align_up(rows * hd * sizeof(float), 256) + align_up(rows * 2 * sizeof(float), 256);
        }
        return p;
    }
    const long base = static_cast<long>(batch) * H * ceil_div(nq, kQG);
    const int max_splits = ceil_div(ntiles, 4);      // at least one tile per wave
    // bf16 with long key ranges: the ring kernel, about 256 workgroups (one
    // per CU, one round), while every wave still walks at least 4 tiles (the
    // batch-8 LLaDA-8B layer: one split, 12 tiles per wave, attention + merge
    // 50.2 -> 45.2 us; at batch 1 the six splits leave one tile per wave and
    // the plain kernel stays; more than 256 (sequence, head, query group)
    // rows, as in a batch-16 stack, keep the plain kernel's one round)
    if (bf16 && base <= 256) {
        int rs = static_cast<int>(256 / base);
        if (rs > max_splits) rs = max_splits;
        if (rs < 1) rs = 1;
        const int tps = ceil_div(ntiles, rs);
        if (tps >= 16) {
            p.ring = true;
            p.tiles_per_split = tps;
            p.splits = ceil_div(ntiles, tps);
            if (p.splits > 1) {
                const size_t rows = static_cast<size_t>(batch) * H * nq * p.splits;
                p.part_bytes = align_up(rows * hd * sizeof(float), 256) + align_up(rows * 2 * sizeof(float), 256);
            }
            return p;
        }
    }
    // about 512 workgroups, rounded down: two fit per CU, so a grid of at most
    // 512 runs in one round without a partial second one
    int splits = static_cast<int>(512 / base);
    if (splits > max_splits) splits = max_splits;
    if (splits < 1) splits = 1;
    p.tiles_per_split = ceil_div(ntiles, splits);
    p.splits = ceil_div(ntiles, p.tiles_per_split);
    if (p.splits > 1) {
        const size_t rows = static_cast<size_t>(batch) * H * nq * p.splits;
        p.part_bytes = align_up(rows * hd * sizeof(float), 256) + align_up(rows * 2 * sizeof(float), 256);
    }
    return p;
}

template <bool BF16, int HD>
void launch_att(const AttPlan& p, const AttArgs& a, hipStream_t s) {
    if constexpr (BF16) {
        if (p.group_waves > 0) {
            const dim3 grid(p.splits, p.row_blocks, a.batch * a.Hkv);
            hipLaunchKernelGGL((attend_group_kernel<HD, 8>), grid, dim3(512), 0, s, a);
            return;
        }
    }
    dim3 grid(p.splits, a.H * ceil_div(a.nq, kQG), a.batch);
    if constexpr (BF16) {
        if (p.ring) {
            launch_att_ring(HD, grid, a, s);
            return;
        }
    }
    hipLaunchKernelGGL((attend_kernel<BF16, HD>), grid, dim3(kAttBlock), 0, s, a);
}

template <bool BF16, int HD>
__global__ __launch_bounds__(256) void attend_merge_kernel(AttArgs a) {
    merge_body<BF16, HD>(a, blockIdx.x);
}

template <bool BF16, int HD>
void launch_merge(const AttArgs& a, hipStream_t s) {
    const long rows = static_cast<long>(a.batch) * a.H * a.nq;
    hipLaunchKernelGGL((attend_merge_kernel<BF16, HD>), dim3(ceil_div(rows, 4)), dim3(256), 0, s, a);
}

// Attention arguments for a plan; `part` is the plan's partial buffer (null
// when the plan has one split).
inline AttArgs att_args(const AttPlan& p, int batch, int seq, int nq, int H, int Hkv, int hd,
                        const void* q, const void* k, const void* v, void* out, float* lse,
                        float scale, char* part) {
    AttArgs a{};
    a.q = static_cast<const char*>(q);
    a.k = static_cast<const char*>(k);
    a.v = static_cast<const char*>(v);
    a.out = static_cast<char*>(out);
    a.lse = lse;
    a.batch = batch;
    a.seq = seq;
    a.nq = nq;
    a.H = H;
    a.Hkv = Hkv;
    a.splits = p.splits;
    a.tiles_per_split = p.tiles_per_split;
    const float sc = scale > 0.f ? scale : 1.0f / sqrtf(static_cast<float>(hd));
    a.scale_log2 = sc * kLog2e;
    if (p.splits > 1) {
        const size_t rows = static_cast<size_t>(batch) * H * nq * p.splits;
        a.part_o = reinterpret_cast<float*>(part);
        a.part_ml = reinterpret_cast<float*>(part + align_up(rows * hd * sizeof(float), 256));
    }
    return a;
}

}  // namespace
}  // namespace ps
