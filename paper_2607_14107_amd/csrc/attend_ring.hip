// attend_ring_kernel: the split-key attention of attend_dev.hpp's
// attend_kernel (same tiles, fragments, online softmax and wave merge, same
// results up to the key split) with three tiles of K/V loads in flight per
// wave instead of one, in a ring of register sets.  The sets take up to 432
// registers, so one four-wave workgroup runs per CU, which keeps up to 192 KB
// of K/V loads in flight where two attend_kernel workgroups keep at most
// 128 KB; the plan takes it for long key ranges of bf16 caches (the batch-8
// LLaDA-8B layer: attention + merge 50.2 -> 45.2 us).
//
// A kernel of its own, in a file of its own: with the ring folded into
// attend_kernel's body as a template parameter, the batch-1 layer step (which
// keeps attend_kernel, one tile per wave) ran 0.5 us slower -- different
// instruction schedules in attend_kernel and in the unchanged kernels
// compiled beside it -- so attend_kernel and its translation units keep their
// code, and the ring body repeats the per-tile arithmetic.

#include "attend_dev.hpp"

namespace ps {
namespace {

template <int HD>
__global__ __launch_bounds__(kAttBlock, 1) void attend_ring_kernel(AttArgs a) {
    constexpr int PF = 3;                   // tiles in flight per wave
    using T = Elem<true>;
    constexpr int ES = T::kBytes;
    constexpr int NC = HD * ES / 64;        // 16-byte chunks of one lane's d-range
    constexpr int DPL = HD / 4;             // d values per lane group
    constexpr int DT = HD / 16;             // 16-row d tiles of O^T
    constexpr int VP = 80;                  // V^T rows: 32 keys (64 B) + 16 B pad
    // The V^T staging of the loop and the wave merge after it share one LDS
    // array.
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
    // tile (item pr = lane + 64 it: 4 keys x one 16-byte chunk of d) of a
    // tile, loaded into one of PF register sets.  A set is refilled with the
    // tile PF trips ahead as soon as its tile is consumed -- V transposed into
    // LDS, the score MFMAs issued -- so PF - 1 further tiles stay in flight
    // through the softmax and PV work.
    constexpr int DCV = HD / 8;             // 16-byte chunks of a V row
    constexpr int ITV = DCV * 8 / 64;
    uint4 kf[PF][2][NC];
    uint4 vv[PF][ITV][4];
    // V item `it` of this lane: 16-byte chunk dc of d for the 4 keys of group
    // kg: the 4 key groups a store instruction covers are it, it + IT,
    // it + 2 IT, ... so that they use both 8-byte halves of a 16-byte slot
    // group (with vrow, a 2-way bank conflict, the minimum for a 512-byte
    // store); the loads stay 256 contiguous bytes per 16 lanes.
    auto vitem = [&](int it, int& dc, int& kg) {
        dc = lane % DCV;
        kg = it + ITV * (lane / DCV);
    };
    auto load_tile = [&](int tile, uint4 (&kf_)[2][NC], uint4 (&vv_)[ITV][4]) {
        const int key0 = tile * kKT;
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            const int key = min(key0 + 16 * t + (lane & 15), a.seq - 1);
            const char* kp = kbase + static_cast<size_t>(key) * krow + g * DPL * ES;
#pragma unroll
            for (int c = 0; c < NC; ++c) kf_[t][c] = ld16(kp + 16 * c);
        }
#pragma unroll
        for (int it = 0; it < ITV; ++it) {
            int dc, kg;
            vitem(it, dc, kg);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int key = min(key0 + 4 * kg + j, a.seq - 1);
                vv_[it][j] = ld16(vbase + static_cast<size_t>(key) * krow + dc * 16);
            }
        }
    };

    // Wave w takes tiles t_begin + w, t_begin + w + 4, ... (no barrier inside
    // the loop, so the waves' trip counts may differ); tile t_begin + w + 4i
    // goes through register set i % PF.
    auto step = [&](int tile, uint4 (&kf_)[2][NC], uint4 (&vv_)[ITV][4]) {
        const int key0 = tile * kKT;
        floatx4 st[2][2];
        // V tile (loaded into vv) -> LDS, transposed to [d][key slot].
        {
            // 8 groups of 4 keys x HD/8 chunks of 8 d; item pr = lane + 64 it
            constexpr int DC = HD / 8;
            constexpr int IT = DC * 8 / 64;
#pragma unroll
            for (int it = 0; it < IT; ++it) {
                int dc, kg;
                vitem(it, dc, kg);
                const uint32_t* x0 = reinterpret_cast<const uint32_t*>(&vv_[it][0]);
                const uint32_t* x1 = reinterpret_cast<const uint32_t*>(&vv_[it][1]);
                const uint32_t* x2 = reinterpret_cast<const uint32_t*>(&vv_[it][2]);
                const uint32_t* x3 = reinterpret_cast<const uint32_t*>(&vv_[it][3]);
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
        }
        // S^T tiles: st[t][u] = K_t Q_u^T.
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                floatx4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int c = 0; c < NC; ++c) s = Mma<true>::step(kf_[t][c], qf[u][c], s);
                st[t][u] = s;
            }
        if (tile + 4 * PF < t_end) load_tile(tile + 4 * PF, kf_, vv_);
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
        {
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
        }
    };
    const int t0 = t_begin + wu;
#pragma unroll
    for (int j = 0; j < PF; ++j)
        if (t0 + 4 * j < t_end) load_tile(t0 + 4 * j, kf[j], vv[j]);
    for (int base = t0; base < t_end; base += 4 * PF) {
#pragma unroll
        for (int j = 0; j < PF; ++j) {
            const int tile = base + 4 * j;
            if (tile < t_end) step(tile, kf[j], vv[j]);
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
        for (int j = 0; j < PER; j += 8)
            st16(op + 2 * j, make_uint4(pack_bf16x2(acc[j] * inv, acc[j + 1] * inv),
                                        pack_bf16x2(acc[j + 2] * inv, acc[j + 3] * inv),
                                        pack_bf16x2(acc[j + 4] * inv, acc[j + 5] * inv),
                                        pack_bf16x2(acc[j + 6] * inv, acc[j + 7] * inv)));
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

}  // namespace

void launch_att_ring(int hd, dim3 grid, const AttArgs& a, hipStream_t s) {
    if (hd == 128)
        hipLaunchKernelGGL((attend_ring_kernel<128>), grid, dim3(kAttBlock), 0, s, a);
    else
        hipLaunchKernelGGL((attend_ring_kernel<64>), grid, dim3(kAttBlock), 0, s, a);
}

}  // namespace ps
