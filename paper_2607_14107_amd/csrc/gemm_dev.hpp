// Device side of the skinny "gather rows -> MFMA GEMM -> scatter rows": row
// bookkeeping, output addressing and the small-M kernel body, shared by the
// GEMM kernels and the fused step kernel.  Internal to the library.
#pragma once

#include "common.hpp"
#include "gemm.hpp"

namespace ps {
namespace {

constexpr int kGemmBlock = 256;
constexpr int kSmallWaves = 4;    // gemm_small_kernel: waves per workgroup
constexpr int kSmallBlock = kSmallWaves * 64;

// Row bookkeeping --------------------------------------------------------------
// Refresh mode: sequence b owns rows [b*R, (b+1)*R), R = k_max + block_len:
// its first count_b rows are its stale positions, the last block_len rows
// its active block; rows in between (count_b < k_max) map to nothing.  A
// fixed stride costs no prefix over the counts, so a row's position is one
// load away.  Block-rows mode: row m is position block_start + m % block_len
// of sequence m / block_len.
__device__ __forceinline__ int gemm_rows_total(const GemmArgs& g) {
    return g.batch * (g.mode == kGemmRefresh ? g.k_max + g.block_len : g.block_len);
}

// Row m -> (sequence, position); b = -1 when the row maps to nothing.
__device__ __forceinline__ void map_row(const GemmArgs& g, int m, int& b, int& pos) {
    b = -1;
    pos = 0;
    if (m < 0 || m >= gemm_rows_total(g)) return;
    if (g.mode == kGemmBlockRows) {
        b = m / g.block_len;
        pos = g.block_start + (m - b * g.block_len);
        return;
    }
    const int R = g.k_max + g.block_len;
    const int sb = m / R;
    const int local = m - sb * R;
    if (local >= g.k_max) {
        b = sb;
        pos = g.block_start + (local - g.k_max);
        return;
    }
    int c = g.stale_count[sb];
    const int p = g.stale_idx[static_cast<size_t>(sb) * g.k_max + local];
    c = c < 0 ? 0 : (c > g.k_max ? g.k_max : c);
    if (local >= c || p < 0 || p >= g.seq) return;   // unused slot or out-of-range entry: refresh nothing
    b = sb;
    pos = p;
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

// 8 consecutive fp32 values -> destination (16-byte bf16 or 2x16-byte fp32 store).
template <bool BF16>
__device__ __forceinline__ void store8(char* dst, const float* v) {
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

// Weight row of output column n (nullptr past N).
__device__ __forceinline__ const char* weight_row(const GemmArgs& g, int n, int es) {
    if (n >= g.N) return nullptr;
    return n < g.n0 ? g.w0 + static_cast<size_t>(n) * g.K * es
                    : g.w1 + static_cast<size_t>(n - g.n0) * g.K * es;
}

// ---------------------------------------------------------------------------
// gemm_small_kernel: at most 16*MT rows, 16 columns per workgroup, the 4
// waves take super-steps w, w+4, w+8, ... of K and are summed in LDS.
// ---------------------------------------------------------------------------

template <bool BF16, int MT>
__device__ __forceinline__ void small_body(const GemmArgs& g, int bx, int by) {
    using T = Elem<BF16>;
    constexpr int ES = T::kBytes;
    constexpr int BM = MT * 16;
    __shared__ int rowb[BM], rowp[BM];
    __shared__ float red[kSmallWaves][BM][17];

    const int t = threadIdx.x;
    const int lane = t & 63;
    const int w = t >> 6;
    const int col0 = bx * 16;
    const int m0 = by * BM;
    const int kcol = (lane >> 4) * 16;   // lane group g reads bytes 16g + 64s: 64 contiguous bytes of a row per load
    const int nsteps = g.K / (256 / ES);
    // wave w: super-steps w, w+W, ...; the last one it owns is slast
    // (prefetches past it re-read slast and are ignored).
    constexpr int W = kSmallWaves;
    const int nmine = w < nsteps ? (nsteps - 1 - w) / W + 1 : 0;
    const int slast = w < nsteps ? w + W * (nmine - 1) : 0;

    // Weight row of column col0 + lane%16 (past N: row 0, never stored); its
    // first two super-steps are requested before the row bookkeeping.
    const char* brow = weight_row(g, col0 + (lane & 15), ES);
    if (!brow) brow = g.w0;
    auto load_b = [&](int step, uint4 (&rb)[4]) {
#pragma unroll
        for (int s = 0; s < 4; ++s) rb[s] = ld16(brow + step * 256 + 64 * s + kcol);
    };
    uint4 q0[4], q1[4], q2[4];
    load_b(min(w, slast), q0);
    load_b(min(w + W, slast), q1);

    if (m0 >= gemm_rows_total(g)) return;
    if (t < BM) {
        int b, pos;
        map_row(g, m0 + t, b, pos);
        rowb[t] = b;
        rowp[t] = pos;
    }
    __syncthreads();

    // Rows past the end read row 0 and are never stored.
    const char* arow[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const int r = mt * 16 + (lane & 15);
        const int b = rowb[r];
        arow[mt] = b >= 0 ? g.x + (static_cast<size_t>(b) * g.seq + rowp[r]) * g.K * ES : g.x;
    }
    auto load_a = [&](int step, uint4 (&ra)[MT][4]) {
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) ra[mt][s] = ld16(arow[mt] + step * 256 + 64 * s + kcol);
    };
    floatx4 acc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[mt] = floatx4{0.f, 0.f, 0.f, 0.f};
    auto compute = [&](const uint4 (&ra)[MT][4], const uint4 (&rb)[4]) {
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) acc[mt] = Mma<BF16>::step(ra[mt][s], rb[s], acc[mt]);
    };

    uint4 a0[MT][4], a1[MT][4], a2[MT][4];
    load_a(min(w, slast), a0);
    load_a(min(w + W, slast), a1);
#define PS_SMALL_STEP(I, A_USE, B_USE, A_LOAD, B_LOAD)                      \
    {                                                                       \
        __builtin_amdgcn_sched_barrier(0);                                  \
        load_a(min(w + W * ((I) + 2), slast), A_LOAD);                      \
        load_b(min(w + W * ((I) + 2), slast), B_LOAD);                      \
        __builtin_amdgcn_sched_barrier(0);                                  \
        compute(A_USE, B_USE);                                              \
    }
    int ic = 0;
    for (; ic + 3 <= nmine; ic += 3) {
        PS_SMALL_STEP(ic, a0, q0, a2, q2)
        PS_SMALL_STEP(ic + 1, a1, q1, a0, q0)
        PS_SMALL_STEP(ic + 2, a2, q2, a1, q1)
    }
    if (ic < nmine) PS_SMALL_STEP(ic, a0, q0, a2, q2)
    if (ic + 1 < nmine) PS_SMALL_STEP(ic + 1, a1, q1, a0, q0)
#undef PS_SMALL_STEP

    // sum the waves in order: lane holds rows mt*16 + 4*(lane/16) + i, column lane%16
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) red[w][mt * 16 + 4 * (lane >> 4) + i][lane & 15] = acc[mt][i];
    __syncthreads();
    // thread -> (row r, 8 columns c)
    for (int idx = t; idx < BM * 2; idx += kSmallBlock) {
        const int r = idx >> 1, c = (idx & 1) * 8;
        const int b = rowb[r];
        const int n = col0 + c;
        if (b < 0 || n >= g.N) continue;
        float v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            float acc_j = red[0][r][c + j];
#pragma unroll
            for (int q = 1; q < kSmallWaves; ++q) acc_j += red[q][r][c + j];
            v[j] = acc_j;
        }
        store8<BF16>(out_ptr<BF16>(g, b, rowp[r], m0 + r, n), v);
    }
}

constexpr int kMaxSplit = 8;      // largest split-K factor of a plan

// ---------------------------------------------------------------------------
// dma_body (gemm_dma_kernel, and the fused step's Q projection): BM = 16*MT rows (one row tile) x 128 columns; wave w owns
// columns 32w..32w+31 as two 16-column tiles of v_mfma_f32_16x16x32_bf16.
// ---------------------------------------------------------------------------

constexpr int kDmaStage = 128;               // bytes of each row per stage
constexpr int kDmaMaxRowTiles = 10;          // 160 rows
// One 16-byte global -> LDS transfer per lane (the wave's lanes land
// contiguously from lds_base).  A plain device function, so the builtin never
// appears in a kernel template's host-side instantiation.
__device__ __forceinline__ void dma16(const void* src, void* lds_base) {
    __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void*)lds_base, 16, 0, 0);
}
// The same transfer marked non-temporal (cache policy nt): for weights that a
// single row tile reads once.
__device__ __forceinline__ void dma16_nt(const void* src, void* lds_base) {
    __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void*)lds_base, 16, 0, 2);
}

// s_waitcnt immediates (gfx9 encoding: vmcnt in bits 3:0 and 15:14, expcnt
// 6:4, lgkmcnt 11:8): wait until at most n vector-memory operations of this
// wave are outstanding / until its LDS reads are done.
constexpr int wait_vm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
constexpr int kWaitLgkm0 = 15 | (3 << 14) | (7 << 4);

// LDS offset of 16-byte chunk c of row r in a stage (rows of kDmaStage bytes).
__device__ __forceinline__ int dma_swz(int r, int c) { return r * kDmaStage + ((c ^ ((r >> 1) & 7)) << 4); }

// NS: LDS slots per operand (4: three stages in flight; 3: two, for a
// workgroup that must share its compute unit).  NTW: the plan has one row
// tile, so every weight byte is read once and its DMA is marked non-temporal
// (a compile-time choice: a branch inside the unrolled stage loop costs more
// than the hint saves).  REG: the operands go through registers instead of
// global -> LDS transfers (below); taken for row tiles of at most 64 rows,
// where it made the batch-1 Q projection 13.8 -> 13.3 us, while the 144- and
// 160-row refreshes ran 27.5 -> 31.1 and 25.4 -> 28.0 us with it.
template <bool BF16, int MT, int NST, int NS = 4, bool NTW = false, bool REG = (MT <= 4)>
__device__ __forceinline__ void dma_body(const GemmArgs& g, int blk) {
    static_assert(NS == 3 || NS == 4, "three or four LDS slots");
    using T = Elem<BF16>;
    constexpr int ES = T::kBytes;
    constexpr int BM = MT * 16;
    constexpr int BN = 128;
    constexpr int ASZ = BM * kDmaStage, BSZ = BN * kDmaStage;
    constexpr int AG = BM / 8;                          // 8-row groups of A per stage (one DMA instruction each)
    constexpr int AIW = (AG + 3) / 4;                   // per wave (surplus ones repeat the last group)
    constexpr int NDMA = 4 + AIW;                       // DMA instructions per wave per stage
    static_assert(2 * NDMA <= 63, "outstanding DMA must fit the vmcnt counter");
    // one LDS object per slot and operand: the compiler can tell them apart
    __shared__ __align__(16) char sa0[ASZ], sa1[ASZ], sa2[REG ? 16 : ASZ], sa3[NS == 4 && !REG ? ASZ : 16];
    __shared__ __align__(16) char sb0[BSZ], sb1[BSZ], sb2[REG ? 16 : BSZ], sb3[NS == 4 && !REG ? BSZ : 16];
    __shared__ __align__(16) int rowb[BM];
    __shared__ int rowp[BM];

    const int tile = blk / g.ksplit;
    const int split = blk - tile * g.ksplit;
    const int col_tile = tile % g.col_tiles;
    const int m0 = (tile / g.col_tiles) * BM;           // up to eight row tiles
    const int t = threadIdx.x;
    const int lane = t & 63;
    const int w = t >> 6;
    const int s0b = split * g.steps_per_split * 256;    // byte offset of the split in a row
    constexpr int nst_here = NST;                       // 128-byte stages of every split (the plan divides K evenly)

    // weights: wave w moves rows 32w + 8i + l/8 (i < 4) of the tile's 128
    // columns; lane l fills slot l%8 of its row
    const char* bsrc[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = 32 * w + 8 * i + (lane >> 3);
        const char* row = weight_row(g, col_tile * BN + r, ES);
        bsrc[i] = (row ? row : g.w0) + s0b + (((lane & 7) ^ ((r >> 1) & 7)) << 4);
    }
    auto issue_b = [&](int st, char* buf) {
        const int off = min(st, nst_here - 1) * kDmaStage;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            if constexpr (NTW) dma16_nt(bsrc[i] + off, buf + (32 * w + 8 * i) * kDmaStage);
            else dma16(bsrc[i] + off, buf + (32 * w + 8 * i) * kDmaStage);
        }
    };
    // Row bookkeeping (one load per row); the first workgroup publishes the
    // map for the split-K reduction.
    int rb_ = -1, rp_ = 0;
    if (t < BM) map_row(g, m0 + t, rb_, rp_);
    if (t < BM) {
        rowb[t] = rb_;
        rowp[t] = rp_;
        if (g.ksplit > 1 && split == 0 && col_tile == 0 && m0 + t < g.m_max)
            *reinterpret_cast<int2*>(g.rowmap + 2 * (m0 + t)) = make_int2(rb_, rp_);
    }
    if (!__syncthreads_or(rb_ >= 0)) return;            // no row of this tile maps anywhere (uniform)
    // input rows: wave w moves groups w, w + 4, ... (8 rows each); rows that
    // map to nothing read row 0 and are never stored
    const char* asrc[AIW];
#pragma unroll
    for (int i = 0; i < AIW; ++i) {
        const int r = 8 * min(w + 4 * i, AG - 1) + (lane >> 3);
        const int b = rowb[r];
        const char* row = b >= 0 ? g.x + (static_cast<size_t>(b) * g.seq + rowp[r]) * g.K * ES : g.x;
        asrc[i] = row + s0b + (((lane & 7) ^ ((r >> 1) & 7)) << 4);
    }
    auto issue_a = [&](int st, char* buf) {
        const int off = min(st, nst_here - 1) * kDmaStage;
#pragma unroll
        for (int i = 0; i < AIW; ++i)
            dma16(asrc[i] + off, buf + 8 * min(w + 4 * i, AG - 1) * kDmaStage);
    };
    floatx4 acc[2][MT];
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int i = 0; i < MT; ++i) acc[c][i] = floatx4{0.f, 0.f, 0.f, 0.f};
    // a stage is two 64-byte pieces; lane l reads chunk 4p + l/16 of rows
    // 16mt + l%16 (A) and 32w + 16c + l%16 (B)
    auto compute = [&](const char* abuf, const char* bbuf) {
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            const int c = 4 * p + (lane >> 4);
            const uint4 bf0 = *reinterpret_cast<const uint4*>(bbuf + dma_swz(32 * w + (lane & 15), c));
            const uint4 bf1 = *reinterpret_cast<const uint4*>(bbuf + dma_swz(32 * w + 16 + (lane & 15), c));
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const uint4 af = *reinterpret_cast<const uint4*>(abuf + dma_swz(16 * mt + (lane & 15), c));
                acc[0][mt] = Mma<BF16>::step(af, bf0, acc[0][mt]);
                acc[1][mt] = Mma<BF16>::step(af, bf1, acc[1][mt]);
            }
        }
    };
    if constexpr (!REG) {
        issue_b(0, sb0);
        issue_a(0, sa0);
        issue_b(1, sb1);
        issue_a(1, sa1);
        if constexpr (NS == 4) {
            issue_b(2, sb2);
            issue_a(2, sa2);
        }

        // Stage s: wait for this wave's DMA of stage s and its own earlier LDS
        // reads; barrier (stage s is in LDS for every wave, and the slot of stage
        // s-1 is free); issue stage s+NS-1 into that slot; compute stage s.
        // Issue order (NS = 4) B0 A0 B1 A1 B2 A2 | B3 A3 | ...: the wait leaves
        // exactly the NS-2 newer stages outstanding.  Stages past the split
        // re-read its last stage, so every stage issues the same DMA count.
    #define PS_DMA_STEP(S, WAIT, AUSE, BUSE, ANEXT, BNEXT)                      \
        {                                                                       \
            __builtin_amdgcn_s_waitcnt(WAIT);                                   \
            __builtin_amdgcn_s_waitcnt(kWaitLgkm0);                             \
            __builtin_amdgcn_s_barrier();                                       \
            issue_b((S) + NS - 1, BNEXT);                                       \
            issue_a((S) + NS - 1, ANEXT);                                       \
            compute(AUSE, BUSE);                                                \
        }
        constexpr int WS = wait_vm((NS - 2) * NDMA);        // after stage s: stages s+1 .. s+NS-2
        char* const sa[4] = {sa0, sa1, sa2, sa3};
        char* const sb[4] = {sb0, sb1, sb2, sb3};
        // fully unrolled: every slot index is a constant and the compiler sees the
        // whole issue order (a loop would make it drain the DMA at the loop head)
    #pragma unroll
        for (int st = 0; st < NST; ++st)
            PS_DMA_STEP(st, WS, sa[st % NS], sb[st % NS], sa[(st + NS - 1) % NS], sb[(st + NS - 1) % NS])
    #undef PS_DMA_STEP
        __builtin_amdgcn_s_waitcnt(0);                      // the re-read tail DMA lands before the workgroup ends
    } else {
        // Register staging: each stage's chunks are loaded into registers P
        // stages ahead and written to the same LDS positions the DMA fills
        // (lane l of an instruction at base + 16 l), into two LDS slots.
        // Plain loads stream faster than global -> LDS transfers (a probe
        // with the batch-8 Q projection's addresses and no arithmetic: 14.4
        // against 18.4 us, 9.1 against 13.4 us when the data is in L2), but
        // the stores to LDS cost the large tiles more than that.  Iteration
        // s: compute slot s%2; wait for stage s+1's registers, write them to
        // slot (s+1)%2 (computed an iteration back), load stage s+1+P into
        // the freed set; barrier.  Stages past the split re-read its last
        // stage, so every iteration issues the same load count.
        constexpr int P = 3;
        static_assert(P * NDMA <= 63, "outstanding loads must fit the vmcnt counter");
        uint4 rs[P][NDMA];
        auto load_stage = [&](int st, uint4 (&r)[NDMA]) {
            const int off = min(st, nst_here - 1) * kDmaStage;
#pragma unroll
            for (int i = 0; i < 4; ++i) r[i] = NTW ? ld16_nt(bsrc[i] + off) : ld16(bsrc[i] + off);
#pragma unroll
            for (int i = 0; i < AIW; ++i) r[4 + i] = ld16(asrc[i] + off);
        };
        auto store_stage = [&](const uint4 (&r)[NDMA], char* abuf, char* bbuf) {
#pragma unroll
            for (int i = 0; i < 4; ++i) st16(bbuf + (32 * w + 8 * i) * kDmaStage + 16 * lane, r[i]);
#pragma unroll
            for (int i = 0; i < AIW; ++i)
                if (AG % 4 == 0 || w + 4 * i < AG)   // surplus instructions repeat the last group: no store
                    st16(abuf + 8 * (w + 4 * i) * kDmaStage + 16 * lane, r[4 + i]);
        };
#pragma unroll
        for (int j = 0; j < P; ++j) load_stage(j, rs[j]);
        __builtin_amdgcn_s_waitcnt(wait_vm((P - 1) * NDMA));
        store_stage(rs[0], sa0, sb0);
        load_stage(P, rs[0]);
        __syncthreads();
        constexpr int WR = wait_vm((P - 1) * NDMA);     // stages s+2 .. s+P stay in flight
#pragma unroll
        for (int st = 0; st < NST; ++st) {
            compute(st % 2 ? sa1 : sa0, st % 2 ? sb1 : sb0);
            if (st + 1 < NST) {
                __builtin_amdgcn_s_waitcnt(WR);
                store_stage(rs[(st + 1) % P], (st + 1) % 2 ? sa1 : sa0, (st + 1) % 2 ? sb1 : sb0);
                load_stage(st + 1 + P, rs[(st + 1) % P]);
            }
            __syncthreads();
        }
        __builtin_amdgcn_s_waitcnt(0);                  // the re-read tail loads land before the workgroup ends
    }

    // results straight from registers: register i of acc[c][mt] is row
    // 16mt + 4(l/16) + i, column 32w + 16c + l%16.  Split K (the usual case):
    // fp32 partials, the lane's four row flags read once per row tile.
    if (g.ksplit > 1) {
        float* part = g.ws + (static_cast<size_t>(split) * g.col_tiles + col_tile) * g.m_max * BN +
                      32 * w + (lane & 15);
        const bool c0 = col_tile * BN + 32 * w + (lane & 15) < g.N;
        const bool c1 = col_tile * BN + 32 * w + 16 + (lane & 15) < g.N;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const int r0 = 16 * mt + 4 * (lane >> 4);
            const int4 rb4 = *reinterpret_cast<const int4*>(&rowb[r0]);
            const int rv[4] = {rb4.x, rb4.y, rb4.z, rb4.w};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                float* dst = part + static_cast<size_t>(m0 + r0 + i) * BN;
                if (rv[i] >= 0 && c0) dst[0] = acc[0][mt][i];
                if (rv[i] >= 0 && c1) dst[16] = acc[1][mt][i];
            }
        }
        return;
    }
#pragma unroll
    for (int c = 0; c < 2; ++c) {
        const int n = col_tile * BN + 32 * w + 16 * c + (lane & 15);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int r = 16 * mt + 4 * (lane >> 4) + i;
                const int b = rowb[r];
                if (b >= 0 && n < g.N) store_elem<BF16>(out_ptr<BF16>(g, b, rowp[r], m0 + r, n), acc[c][mt][i]);
            }
    }
}


// ---------------------------------------------------------------------------
// tile_body (gemm_tile_kernel, and the fused step's refresh): 256 or 192
// rows x 256 or 192 columns of outputs per workgroup for row sets of more
// than one DMA tile (the refresh of a whole batch, the dense rows of a
// stack).  The four waves form a 2 x 2 grid of blocks of MI x NJ tiles of
// v_mfma_f32_32x32x16_bf16 (MI, NJ = 4 or 3), so every fragment read from LDS
// feeds three or four MFMAs (the row kernels of gemm.hip read one A fragment
// per MFMA).  The plan takes 192-row or 192-column tiles where 256 x 256 ones
// would leave compute units idle (1488 rows x 8192 columns: 256 tiles of 192
// rows instead of 192 tiles; 512 rows x 12288: 128 tiles of 192 columns in
// two splits instead of 96).
// Both operands arrive by DMA in stages of 64 bytes (32 bf16) of each row,
// four LDS slots, three stages in flight; the DMA wait and barrier for stage
// s+1 sit between the two halves of stage s, so the first fragments of s+1
// are read while the second half's MFMAs run.
// ---------------------------------------------------------------------------

constexpr int kTileStage = 64;                 // bytes of each row per stage
constexpr int kTileDim = 256;                  // columns (and at most rows) per workgroup
constexpr int kTileGroupRows = 4;              // row tiles per band of the launch order
constexpr int kTileSlot = kTileDim * kTileStage;

// LDS offset of 16-byte chunk c (0..3) of row r in a stage: the chunk is
// XOR-ed with (r/4) % 4.  Measured on gfx950, fragment reads (lane l: row
// l%32, chunk l/32) with this layout run at the full ds_read_b128 rate;
// ((r/2) ^ (r/8)) % 4 or (r/2) % 4 reach half of it.
__device__ __forceinline__ int tile_sw(int r) { return (r >> 2) & 3; }

// Workgroup blk -> (split, row tile, column tile).  Consecutive workgroups go
// to different XCDs, so the ids are first regrouped per XCD; each XCD then
// walks bands of kTileGroupRows row tiles column by column, which keeps the
// input rows and weight rows its compute units share in its own L2.  (The
// tile workgroups must be the first ones of their launch.)
__device__ __forceinline__ void tile_coords(const GemmArgs& g, int bn, int blk, int& split, int& rt, int& ct) {
    const int ntc = (g.N + bn - 1) / bn;
    const int ntiles = g.row_tiles * ntc;
    const int nb = ntiles * g.ksplit;
    int bid = blk;
    if (nb % 8 == 0) bid = (bid % 8) * (nb / 8) + bid / 8;
    split = bid / ntiles;
    const int tl = bid - split * ntiles;
    const int band = tl / (kTileGroupRows * ntc);
    const int rows_here = min(kTileGroupRows, g.row_tiles - band * kTileGroupRows);
    const int in = tl - band * kTileGroupRows * ntc;
    ct = in / rows_here;
    rt = band * kTileGroupRows + (in - ct * rows_here);
}

constexpr int kTileThreads = 256;             // four waves, one per SIMD

// MI / NJ: 32-row / 32-column MFMA tiles per wave: 4 (256-row or -column
// tiles) or 3 (192), for shapes where 256 x 256 tiles would leave compute
// units idle.
template <int MI, int NJ>
__device__ __forceinline__ void tile_body(const GemmArgs& g, int blk) {
    static_assert((MI == 3 || MI == 4) && (NJ == 3 || NJ == 4), "192- or 256-row and -column tiles");
    constexpr int ES = 2;                                // bf16 operands
    constexpr int BMT = 64 * MI;                         // rows per tile (two waves down, MI tiles each)
    constexpr int BNT = 64 * NJ;                         // columns per tile (two waves across, NJ tiles each)
    constexpr int ASLOT = BMT * kTileStage;
    constexpr int BSLOT = BNT * kTileStage;
    constexpr int NDMA = MI + NJ;                        // DMA instructions per wave per stage (MI A, NJ B)
    __shared__ __align__(16) char sa0[ASLOT], sa1[ASLOT], sa2[ASLOT], sa3[ASLOT];
    __shared__ __align__(16) char sb0[BSLOT], sb1[BSLOT], sb2[BSLOT], sb3[BSLOT];
    __shared__ int rowb[kTileDim], rowp[kTileDim];

    int split, rt, ct;
    tile_coords(g, BNT, blk, split, rt, ct);
    const int t = threadIdx.x;
    const int lane = t & 63;
    const int w = t >> 6;
    const int wm = w & 1, wn = w >> 1;
    const int m0 = rt * BMT;
    const int n0 = ct * BNT;
    const int nss = g.steps_per_split;                   // stages of this split (a multiple of 4)
    const size_t k0b = static_cast<size_t>(split) * nss * kTileStage;

    // Row bookkeeping: thread t < BMT maps row m0 + t; the first workgroup of
    // each row tile publishes the map for the split-K reduction.
    int rb_ = -1, rp_ = 0;
    if (t < BMT) map_row(g, m0 + t, rb_, rp_);
    rowb[t] = rb_;
    rowp[t] = rp_;
    if (g.ksplit > 1 && split == 0 && ct == 0 && t < BMT && m0 + t < g.m_max)
        *reinterpret_cast<int2*>(g.rowmap + 2 * (m0 + t)) = make_int2(rb_, rp_);
    if (!__syncthreads_or(rb_ >= 0)) return;             // no row of this tile maps anywhere (uniform)

    // DMA sources: instruction i of wave w moves rows 16(w + 4i) .. +15 of a
    // slot (i < MI for the input rows, i < NJ for the weight rows); lane l
    // fills chunk l%4 of row 16(w + 4i) + l/4, i.e. logical chunk
    // (l%4) ^ swizzle(row).  Rows that map to nothing read row 0 of the
    // input, columns past N weight row 0; neither is stored.
    const char* asrc[MI];
    const char* bsrc[NJ];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = 16 * (w + 4 * i) + (lane >> 2);
        const int chunk = ((lane & 3) ^ tile_sw(r)) << 4;
        if (i < MI) {
            const int b = rowb[r];
            const char* arow = b >= 0 ? g.x + (static_cast<size_t>(b) * g.seq + rowp[r]) * g.K * ES : g.x;
            asrc[i] = arow + k0b + chunk;
        }
        if (i < NJ) {
            const char* brow = weight_row(g, n0 + r, ES);
            bsrc[i] = (brow ? brow : g.w0) + k0b + chunk;
        }
    }
    auto issue = [&](int st, char* abuf, char* bbuf) {
        const int off = min(st, nss - 1) * kTileStage;   // past the split: re-read its last stage
#pragma unroll
        for (int i = 0; i < NJ; ++i) dma16(bsrc[i] + off, bbuf + 16 * (w + 4 * i) * kTileStage);
#pragma unroll
        for (int i = 0; i < MI; ++i) dma16(asrc[i] + off, abuf + 16 * (w + 4 * i) * kTileStage);
    };

    // Fragment offsets: lane l reads row 32i + l%32 of its wave's block at
    // k-group l/32 of half kk; the swizzle depends on l%32 only.
    const int fr = lane & 31;
    const int fsw = tile_sw(fr);                         // = tile_sw(32i + fr)
    const int h = lane >> 5;
    const int aoff0 = (32 * MI * wm + fr) * kTileStage + (((0 + h) ^ fsw) << 4);
    const int aoff1 = (32 * MI * wm + fr) * kTileStage + (((2 + h) ^ fsw) << 4);
    const int boff0 = (32 * NJ * wn + fr) * kTileStage + (((0 + h) ^ fsw) << 4);
    const int boff1 = (32 * NJ * wn + fr) * kTileStage + (((2 + h) ^ fsw) << 4);

    floatx16 acc[MI][NJ];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

    uint4 fa0[MI], fb0[NJ], fa1[MI], fb1[NJ];            // fragments of half 0 / half 1
    auto read_half = [&](const char* abuf, const char* bbuf, int aoff, int boff, uint4 (&fa)[MI], uint4 (&fb)[NJ]) {
#pragma unroll
        for (int i = 0; i < MI; ++i) fa[i] = *reinterpret_cast<const uint4*>(abuf + aoff + i * 32 * kTileStage);
#pragma unroll
        for (int j = 0; j < NJ; ++j) fb[j] = *reinterpret_cast<const uint4*>(bbuf + boff + j * 32 * kTileStage);
    };
    auto mfma_half = [&](const uint4 (&fa)[MI], const uint4 (&fb)[NJ]) {
#pragma unroll
        for (int i = 0; i < MI; ++i)
#pragma unroll
            for (int j = 0; j < NJ; ++j) acc[i][j] = Mma32<true>::step(fa[i], fb[j], acc[i][j]);
    };
    // Instruction order of a half: the MI + NJ fragment reads for the next
    // half go out behind the first two MFMAs (so they land well before the
    // next half starts), the NDMA DMA instructions (second half only) two
    // behind each of the next MFMAs, then the remaining MFMAs.
    auto interleave = [&](bool with_dma) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, NJ, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, MI, 0);
        if (with_dma) {
#pragma unroll
            for (int q = 0; q < NDMA / 2; ++q) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x020, 2, 0);
            }
            if constexpr (NDMA % 2) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
            }
            __builtin_amdgcn_sched_group_barrier(0x008, NJ * MI - 2 - (NDMA + 1) / 2, 0);
        } else {
            __builtin_amdgcn_sched_group_barrier(0x008, NJ * MI - 2, 0);
        }
    };

    constexpr int WS = wait_vm(2 * NDMA);                // two newer stages stay in flight
    issue(0, sa0, sb0);
    issue(1, sa1, sb1);
    issue(2, sa2, sb2);
    issue(3, sa3, sb3);
    __builtin_amdgcn_s_waitcnt(wait_vm(3 * NDMA));
    __builtin_amdgcn_s_barrier();
    read_half(sa0, sb0, aoff0, boff0, fa0, fb0);

    // Stage S in slot S%4: half 1 of S is read while half 0's MFMAs run;
    // then (own reads done, stage S+1 landed for this wave) a barrier makes
    // S+1 visible to all waves and frees slot S%4, which takes stage S+4;
    // half 0 of S+1 is read while half 1's MFMAs run.
#define PS_TILE_STEP(S, AU, BU, AX, BX)                                     \
    {                                                                       \
        __builtin_amdgcn_sched_barrier(0);                                  \
        read_half(AU, BU, aoff1, boff1, fa1, fb1);                          \
        mfma_half(fa0, fb0);                                                \
        interleave(false);                                                  \
        __builtin_amdgcn_sched_barrier(0);                                  \
        __builtin_amdgcn_s_waitcnt(WS);                                     \
        __builtin_amdgcn_s_waitcnt(kWaitLgkm0);                             \
        __builtin_amdgcn_s_barrier();                                       \
        __builtin_amdgcn_sched_barrier(0);                                  \
        issue((S) + 4, AU, BU);                                             \
        read_half(AX, BX, aoff0, boff0, fa0, fb0);                          \
        mfma_half(fa1, fb1);                                                \
        interleave(true);                                                   \
        __builtin_amdgcn_sched_barrier(0);                                  \
    }
    for (int st = 0; st < nss; st += 4) {
        PS_TILE_STEP(st + 0, sa0, sb0, sa1, sb1)
        PS_TILE_STEP(st + 1, sa1, sb1, sa2, sb2)
        PS_TILE_STEP(st + 2, sa2, sb2, sa3, sb3)
        PS_TILE_STEP(st + 3, sa3, sb3, sa0, sb0)
    }
#undef PS_TILE_STEP
    __builtin_amdgcn_s_waitcnt(0);                       // every DMA (the re-read tail too) has landed
    __syncthreads();                                     // and every wave is done with the slots

    // Epilogue through LDS, per wave, 16 rows at a time: register e of
    // acc[i][j] is row 32i + 8(e/4) + 4(l/32) + e%4, column 32j + l%32 of the
    // wave's block; each lane then moves 8 consecutive columns of a row.
    constexpr int EP = 132;                              // fp32 pitch of a staged row
    static_assert(16 * EP * 4 <= ASLOT, "a wave's 16 staged rows fit its input slot");
    float* ep = reinterpret_cast<float*>(w == 0 ? sa0 : w == 1 ? sa1 : w == 2 ? sa2 : sa3);
    const int cbase = n0 + 32 * NJ * wn;
#pragma unroll
    for (int i = 0; i < MI; ++i) {
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
#pragma unroll
            for (int j = 0; j < NJ; ++j)
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int ee = 8 * hh + e;
                    const int r = 8 * (e >> 2) + 4 * h + (e & 3);
                    ep[r * EP + 32 * j + fr] = acc[i][j][ee];
                }
            __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
            __builtin_amdgcn_wave_barrier();
#pragma unroll
            for (int q = 0; q < NJ; ++q) {
                const int idx = 64 * q + lane;           // 16 rows x 4 NJ chunks of 8 columns
                const int r = idx / (4 * NJ), c = (idx % (4 * NJ)) * 8;
                const int lr = 32 * MI * wm + 32 * i + 16 * hh + r;   // row within the tile
                const int b = rowb[lr];
                const int n = cbase + c;
                const float* v = ep + r * EP + c;
                if (b >= 0 && n < g.N) {
                    if (g.ksplit == 1) {
                        store8<true>(out_ptr<true>(g, b, rowp[lr], m0 + lr, n), v);
                    } else {
                        float* dst = g.ws + ((static_cast<size_t>(split) * g.col_tiles + (n >> 7)) * g.m_max +
                                             (m0 + lr)) * 128 + (n & 127);
                        *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
                        *reinterpret_cast<float4*>(dst + 4) = make_float4(v[4], v[5], v[6], v[7]);
                    }
                }
            }
            __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
            __builtin_amdgcn_wave_barrier();
        }
    }
}

// Split-K reduction: thread = (column tile, row, 8 columns); sums the splits
// in order and stores the row through the published row map.  One
// kGemmBlock workgroup per 16 rows of a column tile.
template <bool BF16>
__device__ __forceinline__ void reduce_body(const GemmArgs& g, int blk) {
    const long id = static_cast<long>(blk) * kGemmBlock + threadIdx.x;
    const long per_tile = static_cast<long>(g.m_max) * 16;
    const int ct = static_cast<int>(id / per_tile);
    if (ct >= g.col_tiles) return;
    const int rem = static_cast<int>(id - ct * per_tile);
    const int m = rem >> 4;
    const int c = (rem & 15) * 8;
    const size_t stride = static_cast<size_t>(g.col_tiles) * g.m_max * 128;   // one split
    const float* src = g.ws + (static_cast<size_t>(ct) * g.m_max + m) * 128 + c;
    float4 x[2 * kMaxSplit];
#pragma unroll
    for (int s = 0; s < kMaxSplit; ++s) {
        if (s < g.ksplit) {
            x[2 * s] = *reinterpret_cast<const float4*>(src + s * stride);
            x[2 * s + 1] = *reinterpret_cast<const float4*>(src + s * stride + 4);
        }
    }
    const int2 mp = *reinterpret_cast<const int2*>(g.rowmap + 2 * m);
    const int n = ct * 128 + c;
    if (mp.x < 0 || n >= g.N) return;
    float v[8] = {x[0].x, x[0].y, x[0].z, x[0].w, x[1].x, x[1].y, x[1].z, x[1].w};
#pragma unroll
    for (int s = 1; s < kMaxSplit; ++s) {
        if (s < g.ksplit) {
            v[0] += x[2 * s].x; v[1] += x[2 * s].y; v[2] += x[2 * s].z; v[3] += x[2 * s].w;
            v[4] += x[2 * s + 1].x; v[5] += x[2 * s + 1].y; v[6] += x[2 * s + 1].z; v[7] += x[2 * s + 1].w;
        }
    }
    store8<BF16>(out_ptr<BF16>(g, mp.x, mp.y, m, n), v);
}

}  // namespace
}  // namespace ps
