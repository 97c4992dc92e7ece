// Gather -> MFMA GEMM -> scatter, the core of the sparse K/V refresh
// (Sec. 4.1: re-project the stale rows and the active block; Corollary 1 of
// App. B: K = W_K h, V = W_V h) and of the Q projection of the active block.
//
// The product is skinny: a few hundred gathered rows times a [N][K] weight
// that is read once from HBM.  Two kernels:
//
// gemm_rows_kernel (more than 64 rows): a workgroup of 4 waves owns
//   BM = 32*MT rows and 128 columns; wave w computes all BM rows of columns
//   32w..32w+31 with v_mfma_f32_32x32x16_bf16 (on gfx950 it does twice the
//   work per issue slot of the 16x16x32 form).  Per super-step of 256 bytes
//   of K:
//   - the gathered input rows are staged in LDS (16-byte coalesced loads,
//     272-byte row pitch: conflict-free MFMA reads) and shared by the waves;
//     a wave reads the fragments of the next 16-k chunk while the MFMAs of
//     the current one run;
//   - each wave streams its weight rows from HBM straight into registers,
//     128 contiguous bytes per lane, two super-steps ahead (triple buffer,
//     loop unrolled three times so the buffers rotate without copies).
//   A row's (sequence, position) is one load away (fixed stride of
//   k_max + block_len rows per sequence), so the first input rows follow
//   the weight prefetch closely.
//   When rows x columns do not fill the chip, K is split over workgroups;
//   each writes its fp32 partial tile as one contiguous block of the
//   workspace ([split][column tile][row][128]: long DRAM bursts, not 512-byte
//   pieces 32 KB apart), the row map goes next to it, and gemm_reduce_kernel
//   sums the partials in split order (deterministic) and scatters 16-byte
//   rows.
//
// gemm_dma_kernel (65 to 320 rows, e.g. the refresh of one sequence's stale
//   rows and block, or the Q projection of a batch's blocks; up to 1280 rows
//   for outputs of at most 1024 columns): one of up to two row tiles (eight
//   for narrow outputs) of up to 160 rows and 128 columns per workgroup, both operands
//   (bf16) brought into LDS by global_load_lds_dwordx4 (no VGPR staging, so the
//   weight loads never wait behind registers that MFMAs still read), in
//   stages of 128 bytes of each row; four LDS slots, three stages in flight,
//   one barrier per stage.  A stage's rows are XOR-swizzled in 16-byte chunks
//   (chunk c of row r at slot c ^ (r/2 % 8)) so that 16-row fragment reads
//   are conflict-free; the swizzle is applied to each lane's global address,
//   since a DMA instruction writes its lanes' data contiguously.  The waits
//   for the DMA are explicit s_waitcnt immediates (each wave issues the same
//   number of DMA instructions per stage), and each slot's LDS arrays are
//   separate objects so the compiler does not add waits of its own.
//   Measured on the batch-1 LLaDA-8B refresh (138 rows x 8192 x 4096): 18.6 us for
//   the split-K GEMM against 25.9 us for gemm_rows_kernel.
//
// gemm_small_kernel (at most 64 rows, e.g. the Q projection): a workgroup
//   owns all rows and 16 columns; its 4 waves take interleaved super-steps
//   of the full K with both operands loaded straight into registers and are
//   summed in LDS, so no partials leave the chip.  A load instruction covers
//   64 contiguous bytes of each of 16 rows.
//
// In both, A and B use the same lane -> k assignment, so k may be visited in
// any order.  All loads are unconditional (rows or columns past the end read
// row 0 and are never stored) so the compiler's wait counts stay static.
#include <mutex>

#include "gemm_dev.hpp"
#include "host_common.hpp"

namespace ps {
namespace {

constexpr int kLda = 272;         // LDS row pitch (bytes) of the staged input rows
constexpr int kTargetWgs = 256;   // one workgroup per compute unit on MI355X
// Per-CU rate of a 192-row tile relative to a 256-row one in the plan's
// estimate.  Unsplit, the batch-8 LLaDA-8B refresh (1488 x 8192 x 4096 in
// one round) measures 0.86 (256 tiles of 192 rows 112.9 us against 192 of
// 256 rows 130 us); 0.95 is the value whose choices matched the faster
// plan on every shape measured through polestar_linear (with 0.86 the
// 1250 x 2512 x 2048 product takes 256-row tiles in four splits, 45.4 us,
// against 43.8 us for 192-row tiles in two).
constexpr double kTile192Rate = 0.95;

// ---------------------------------------------------------------------------
// gemm_rows_kernel: BM = 32*MT rows x 128 columns per workgroup; wave w owns
// columns 32w..32w+31 of all rows (v_mfma_f32_32x32x16_bf16: lane l carries
// row/column l%32 and k-group l/32, 128 contiguous bytes per super-step).
// ---------------------------------------------------------------------------

template <bool BF16, int MT>
__global__ __launch_bounds__(kGemmBlock) void gemm_rows_kernel(GemmArgs g) {
    using T = Elem<BF16>;
    constexpr int BM = MT * 32;
    constexpr int BN = 128;
    constexpr int RA = BM / 16;            // 16-byte chunks each thread stages per super-step
    constexpr int ES = T::kBytes;
    __shared__ __align__(16) char sa[2][BM * kLda];
    __shared__ int rowb[BM], rowp[BM];

    const int tile = blockIdx.x / g.ksplit;
    const int split = blockIdx.x - tile * g.ksplit;
    const int col_tile = tile % g.col_tiles;
    const int row_tile = tile / g.col_tiles;

    const int t = threadIdx.x;
    const int lane = t & 63;
    const int w = t >> 6;
    const int m0 = row_tile * BM;

    // The weight row this lane streams (column n of wave w; past N: row 0,
    // never stored), 128 contiguous bytes per super-step at k-group lane/32.
    // Its first two super-steps are requested before the row bookkeeping,
    // whose dependent loads (counts, prefix, stale indices) would otherwise
    // delay the weight stream.
    const int n = col_tile * BN + w * 32 + (lane & 31);
    const char* brow = weight_row(g, n, ES);
    if (!brow) brow = g.w0;
    brow += (lane >> 5) * 128;
    const int nsteps = g.K / (256 / ES);
    const int s0 = split * g.steps_per_split;
    const int s1 = min(nsteps, s0 + g.steps_per_split);
    const int slast = s1 - 1;
    auto load_b = [&](int step, uint4 (&rb)[8]) {
#pragma unroll
        for (int s = 0; s < 8; ++s) rb[s] = ld16(brow + step * 256 + 16 * s);
    };
    uint4 b0[8], b1[8], b2[8];
    load_b(s0, b0);
    load_b(min(s0 + 1, slast), b1);

    // Row bookkeeping: one load per row.  The first workgroup of each row
    // tile also publishes the map for the split-K reduction.
    int rb_ = -1, rp_ = 0;
    if (t < BM) map_row(g, m0 + t, rb_, rp_);
    if (t < BM) {
        rowb[t] = rb_;
        rowp[t] = rp_;
        if (g.ksplit > 1 && split == 0 && col_tile == 0 && m0 + t < g.m_max)
            *reinterpret_cast<int2*>(g.rowmap + 2 * (m0 + t)) = make_int2(rb_, rp_);
    }
    if (!__syncthreads_or(rb_ >= 0)) return;   // no row of this tile maps anywhere (uniform)

    // Rows that map to nothing read row 0 instead: their accumulators are
    // never stored, and every load stays unconditional (static wait counts).
    const char* arow[RA];
#pragma unroll
    for (int i = 0; i < RA; ++i) {
        const int r = (t >> 4) + 16 * i;
        const int b = rowb[r];
        arow[i] = b >= 0 ? g.x + (static_cast<size_t>(b) * g.seq + rowp[r]) * g.K * ES : g.x;
    }
    const int acol = (t & 15) * 16;

    floatx16 acc[MT];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < 16; ++j) acc[i][j] = 0.f;

    auto load_a = [&](int step, uint4 (&ra)[RA]) {
#pragma unroll
        for (int i = 0; i < RA; ++i) ra[i] = ld16(arow[i] + step * 256 + acol);
    };
    auto store_a = [&](int buf, const uint4 (&ra)[RA]) {
#pragma unroll
        for (int i = 0; i < RA; ++i) st16(&sa[buf][((t >> 4) + 16 * i) * kLda + acol], ra[i]);
    };
    // The MT fragments of chunk s+1 are read from LDS while the MFMAs of
    // chunk s run (two register sets; the scheduling barriers keep that
    // order), so LDS latency is not exposed per MFMA.
    auto compute = [&](int buf, const uint4 (&rb)[8]) {
        const char* abase = &sa[buf][(lane & 31) * kLda + (lane >> 5) * 128];
        uint4 af[2][MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) af[0][mt] = *reinterpret_cast<const uint4*>(abase + mt * 32 * kLda);
#pragma unroll
        for (int s = 0; s < 8; ++s) {
            __builtin_amdgcn_sched_barrier(0);
            if (s + 1 < 8) {
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    af[(s + 1) & 1][mt] = *reinterpret_cast<const uint4*>(abase + mt * 32 * kLda + 16 * (s + 1));
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) acc[mt] = Mma32<BF16>::step(af[s & 1][mt], rb[s], acc[mt]);
        }
        __builtin_amdgcn_sched_barrier(0);
    };

    // Software pipeline.  Issue order of the loads: ... B(s+1), A(s+1),
    // B(s+2), A(s+2) ...  Waiting for A(s+1) at the end of step s (to stage
    // it in LDS) therefore also covers B(s+1), which step s+1 needs, while
    // B(s+2) stays in flight: weights get two compute phases of latency
    // cover, the (L2-resident) input rows one.  (Two phases for the input
    // rows too, with a second register buffer, measured no faster.)
    // Prefetches past s1 - 1 re-read step s1 - 1 (cache hits, ignored) so
    // every iteration issues the same loads and the wait counts stay static.
    uint4 ra[RA];
    load_a(s0, ra);
    store_a(0, ra);                       // waits for A(s0) (and B(s0), B(s0+1))
    load_a(min(s0 + 1, slast), ra);
    __syncthreads();

    // step S: issue B(S+2) -> B_LOAD; compute with LDS[(S-s0)%2] and B_USE;
    // stage A(S+1) -> LDS[(S-s0+1)%2]; then issue A(S+2).
#define PS_GEMM_STEP(S, B_USE, B_LOAD)                                      \
    {                                                                       \
        const int s_ = (S);                                                 \
        __builtin_amdgcn_sched_barrier(0);                                  \
        load_b(min(s_ + 2, slast), B_LOAD);                                 \
        __builtin_amdgcn_sched_barrier(0);                                  \
        compute((s_ - s0) & 1, B_USE);                                      \
        if (s_ + 1 < s1) store_a((s_ - s0 + 1) & 1, ra);                    \
        __syncthreads();                                                    \
        load_a(min(s_ + 2, slast), ra);                                     \
    }
    int sc = s0;
    for (; sc + 3 <= s1; sc += 3) {      // single exit: buffers rotate b0 -> b1 -> b2
        PS_GEMM_STEP(sc, b0, b2)
        PS_GEMM_STEP(sc + 1, b1, b0)
        PS_GEMM_STEP(sc + 2, b2, b1)
    }
    if (sc < s1) PS_GEMM_STEP(sc, b0, b2)
    if (sc + 1 < s1) PS_GEMM_STEP(sc + 1, b1, b0)
#undef PS_GEMM_STEP

    // Epilogue, staged through LDS (the input staging buffers are free now):
    // register j of acc[mt] is row mt*32 + mfma32_row(lane, j) of column
    // 32w + lane%32; then each thread writes 8 consecutive columns of a row
    // (16-byte stores, 512 contiguous bytes per row of the tile).
    constexpr int EP = BN + 4;            // fp32 pitch of the staged tile
    static_assert(static_cast<size_t>(BM) * EP * 4 <= sizeof(sa), "epilogue tile must fit");
    float* ep = reinterpret_cast<float*>(&sa[0][0]);
    __syncthreads();                      // every wave is done reading sa
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int j = 0; j < 16; ++j)
            ep[(mt * 32 + mfma32_row(lane, j)) * EP + w * 32 + (lane & 31)] = acc[mt][j];
    __syncthreads();
    for (int idx = t; idx < BM * (BN / 8); idx += kGemmBlock) {
        const int r = idx / (BN / 8);
        const int c = (idx % (BN / 8)) * 8;
        const int b = rowb[r];
        const int nc = col_tile * BN + c;
        if (b < 0 || nc >= g.N) continue;
        const float* v = ep + r * EP + c;
        if (g.ksplit == 1) {
            store8<BF16>(out_ptr<BF16>(g, b, rowp[r], m0 + r, nc), v);
        } else {
            float* dst = g.ws + ((static_cast<size_t>(split) * g.col_tiles + col_tile) * g.m_max + (m0 + r)) * BN + c;
            *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
            *reinterpret_cast<float4*>(dst + 4) = make_float4(v[4], v[5], v[6], v[7]);
        }
    }
}

// ---------------------------------------------------------------------------
// gemm_dma_kernel: the DMA-staged body of gemm_dev.hpp (dma_body).
// ---------------------------------------------------------------------------

template <bool BF16, int MT, int NST, bool NTW>
__global__ __launch_bounds__(kGemmBlock) void gemm_dma_kernel(GemmArgs g) {
    dma_body<BF16, MT, NST, 4, NTW>(g, blockIdx.x);
}

template <int MI, int NJ>
__global__ __launch_bounds__(kTileThreads) void gemm_tile_kernel(GemmArgs g) { tile_body<MI, NJ>(g, blockIdx.x); }

// Sum of the split-K partials, in split order (deterministic): thread ->
// (column tile, row, 8 columns) so that consecutive threads read consecutive
// 32-byte pieces of the contiguous partial tiles; the partial and row-map
// loads are independent, then one rounded 16-byte store.
template <bool BF16>
__global__ __launch_bounds__(kGemmBlock) void gemm_reduce_kernel(GemmArgs g) {
    reduce_body<BF16>(g, blockIdx.x);
}

template <bool BF16, int MT>
__global__ __launch_bounds__(kSmallBlock) void gemm_small_kernel(GemmArgs g) {
    small_body<BF16, MT>(g, blockIdx.x, blockIdx.y);
}

template <bool BF16, int MT>
void launch_rows(const GemmPlan& p, const GemmArgs& g, hipStream_t s) {
    hipLaunchKernelGGL((gemm_rows_kernel<BF16, MT>), dim3(p.grid), dim3(kGemmBlock), 0, s, g);
}

template <bool BF16>
bool dispatch_rows(const GemmPlan& p, const GemmArgs& g, hipStream_t s) {
    switch (p.mt) {   // 32-row tiles per workgroup
        case 1: launch_rows<BF16, 1>(p, g, s); return true;
        case 2: launch_rows<BF16, 2>(p, g, s); return true;
        case 3: launch_rows<BF16, 3>(p, g, s); return true;
        case 4: launch_rows<BF16, 4>(p, g, s); return true;
        case 5: launch_rows<BF16, 5>(p, g, s); return true;
        case 6: launch_rows<BF16, 6>(p, g, s); return true;
        case 7: launch_rows<BF16, 7>(p, g, s); return true;
        case 8: launch_rows<BF16, 8>(p, g, s); return true;
        default: return false;
    }
}

template <bool BF16, int NST, bool NTW>
bool dispatch_dma_mt(const GemmPlan& p, const GemmArgs& g, hipStream_t s) {
    const dim3 grid(p.grid), block(kGemmBlock);
    switch (p.mt) {   // 16-row tiles
        case 2: hipLaunchKernelGGL((gemm_dma_kernel<BF16, 2, NST, NTW>), grid, block, 0, s, g); return true;
        case 3: hipLaunchKernelGGL((gemm_dma_kernel<BF16, 3, NST, NTW>), grid, block, 0, s, g); return true;
        case 4: hipLaunchKernelGGL((gemm_dma_kernel<BF16, 4, NST, NTW>), grid, block, 0, s, g); return true;
        case 5: hipLaunchKernelGGL((gemm_dma_kernel<BF16, 5, NST, NTW>), grid, block, 0, s, g); return true;
        case 6: hipLaunchKernelGGL((gemm_dma_kernel<BF16, 6, NST, NTW>), grid, block, 0, s, g); return true;
        case 7: hipLaunchKernelGGL((gemm_dma_kernel<BF16, 7, NST, NTW>), grid, block, 0, s, g); return true;
        case 8: hipLaunchKernelGGL((gemm_dma_kernel<BF16, 8, NST, NTW>), grid, block, 0, s, g); return true;
        case 9: hipLaunchKernelGGL((gemm_dma_kernel<BF16, 9, NST, NTW>), grid, block, 0, s, g); return true;
        case 10: hipLaunchKernelGGL((gemm_dma_kernel<BF16, 10, NST, NTW>), grid, block, 0, s, g); return true;
        default: return false;
    }
}

template <bool BF16>
bool dispatch_dma(const GemmPlan& p, const GemmArgs& g, hipStream_t s) {
    static_assert(kDmaMaxRowTiles == 10, "dispatch covers 2..kDmaMaxRowTiles");
    // one row tile reads every weight byte once: non-temporal weight stream
    if (p.row_tiles == 1) {
        switch (2 * p.steps_per_split) {   // 128-byte stages per split
            case 8: return dispatch_dma_mt<BF16, 8, true>(p, g, s);
            case 10: return dispatch_dma_mt<BF16, 10, true>(p, g, s);
            case 12: return dispatch_dma_mt<BF16, 12, true>(p, g, s);
            case 14: return dispatch_dma_mt<BF16, 14, true>(p, g, s);
            case 16: return dispatch_dma_mt<BF16, 16, true>(p, g, s);
            default: return false;
        }
    }
    switch (2 * p.steps_per_split) {
        case 8: return dispatch_dma_mt<BF16, 8, false>(p, g, s);
        case 10: return dispatch_dma_mt<BF16, 10, false>(p, g, s);
        case 12: return dispatch_dma_mt<BF16, 12, false>(p, g, s);
        case 14: return dispatch_dma_mt<BF16, 14, false>(p, g, s);
        case 16: return dispatch_dma_mt<BF16, 16, false>(p, g, s);
        default: return false;
    }
}

template <bool BF16>
bool dispatch_small(const GemmPlan& p, const GemmArgs& g, hipStream_t s) {
    dim3 grid(p.col_tiles, p.row_tiles);
    switch (p.mt) {
        case 1: hipLaunchKernelGGL((gemm_small_kernel<BF16, 1>), grid, dim3(kSmallBlock), 0, s, g); return true;
        case 2: hipLaunchKernelGGL((gemm_small_kernel<BF16, 2>), grid, dim3(kSmallBlock), 0, s, g); return true;
        case 3: hipLaunchKernelGGL((gemm_small_kernel<BF16, 3>), grid, dim3(kSmallBlock), 0, s, g); return true;
        case 4: hipLaunchKernelGGL((gemm_small_kernel<BF16, 4>), grid, dim3(kSmallBlock), 0, s, g); return true;
        default: return false;
    }
}

}  // namespace

// Partial tiles of a split-K plan, [ksplit][col_tiles][m_max][128] fp32.
static size_t partial_bytes(const GemmPlan& p, long m_max) {
    return align_up(static_cast<size_t>(p.ksplit) * p.col_tiles * m_max * 128 * sizeof(float), 256);
}

GemmPlan gemm_plan(bool bf16, long m_max, int N, int K) {
    GemmPlan p{};
    const int ks = bf16 ? 128 : 64;
    const int nsteps = ceil_div(K, ks);
    if (m_max <= 0) m_max = 1;
    // 17..64 rows (bf16): the DMA kernel with split-K partials streams each
    // weight once with its A rows shared through LDS, where the small kernel
    // re-reads the rows once per 16 columns (the 32-row LLaDA-8B block
    // projection: 12.4 against 13.7 us with the reduce, 64 rows 13.6 against
    // 21.0); other shapes, or when K does not split into 8 or 16 stages, the
    // small kernel
    if (m_max <= 64 && bf16 && m_max > 16) {
        const int col_tiles = ceil_div(N, 128);
        for (int ks = ceil_div(kTargetWgs, col_tiles); ks <= kMaxSplit; ++ks) {
            if (nsteps % ks == 0 && (nsteps / ks == 4 || nsteps / ks == 8)) {
                p.dma = true;
                p.row_tiles = 1;
                p.col_tiles = col_tiles;
                p.ksplit = ks;
                p.steps_per_split = nsteps / ks;
                p.mt = ceil_div(m_max, 16);
                p.grid = col_tiles * ks;
                if (ks > 1)
                    p.ws_bytes = partial_bytes(p, m_max) + align_up(static_cast<size_t>(m_max) * 2 * sizeof(int), 256);
                return p;
            }
        }
    }
    if (m_max <= 64) {
        p.small = true;
        p.mt = ceil_div(m_max, 16);
        p.row_tiles = 1;
        p.col_tiles = ceil_div(N, 16);
        p.ksplit = 1;
        p.steps_per_split = nsteps;
        p.grid = p.col_tiles;
        return p;
    }
    p.small = false;
    p.col_tiles = ceil_div(N, 128);                     // split-K partials: 128-column tiles
    // Tile kernel: more rows than one DMA tile; 256- or 192-row x 256- or 192-column tiles, K split
    // while the tiles alone leave compute units idle.  Measured against the
    // other kernels it wins when it launches at least 128 workgroups and at
    // most four splits fill the chip, each split still runs 48 stages or
    // more, or there are four row tiles or more; short splits of one or two
    // row tiles (256 or 512 rows of a 4096 x 4096 projection) stay on the DMA
    // or row kernel.
    // Narrow outputs (at most 1024 columns: four 256-wide tiles across) take
    // the DMA kernel's 128-column tiles instead, up to eight row tiles: the
    // Dream-7B refresh (1052 rows x 1024 x 3584) runs 56 tiles in four splits
    // (224 workgroups, 17 MB of partials) in 27.7 us, where the tile kernel's
    // 20 tiles needed seven splits (30 MB of partials) and 37.5 us.
    // Only where the DMA kernel can take K: some split into 4 to 8 steps of
    // 256 bytes (K = 2816, 22 steps, has none and stays on the tile kernel).
    bool dma_k = false;
    for (int ks = 1; ks <= kMaxSplit && !dma_k; ++ks) dma_k = nsteps % ks == 0 && nsteps / ks >= 4 && nsteps / ks <= 8;
    const bool narrow_dma = bf16 && dma_k && N <= 4 * kTileDim && m_max <= 8L * 16 * kDmaMaxRowTiles;
    if (bf16 && m_max > 16L * kDmaMaxRowTiles && K % kTileStage == 0 && !narrow_dma) {
        const int nstage = K / (kTileStage / 2);
        // The tile shape and split with the least estimated time: ceil(tiles
        // * k / 256) rounds of one workgroup per CU, each 1/k of a tile's
        // work (a whole 256 x 256 x K tile at the ~1 PFLOP/s this kernel
        // sustains: 3.9 GFLOP/ms per CU; a 192-row or 192-column tile at
        // kTile192Rate of that rate, 192 x 192 at its square), plus the fp32
        // partials of a split run written and read back (8 k M N bytes at
        // ~5 TB/s); ties keep the larger tile, rows before columns.
        // Measured on the batch-8 LLaDA-8B refresh: 192 tiles of 256 rows
        // (10% stale) unsplit in one round 130 us, in two splits (384
        // workgroups, a round and a half, 98 MB of partials) 159 us, as 256
        // tiles of 192 rows 112.9 us; 64 tiles (2%) best in four splits; 20
        // tiles (the Dream-7B refresh) in seven.  Through polestar_linear the
        // 192-row plans it picks ran 3-15% faster than the best 256-row ones
        // (512 x 4096 x 4096: 47.6 against 50.9 us; 1264 x 8192 x 4096: 95.1
        // against 110.3 us).  Every split runs a whole number of 4-stage loop
        // trips and at least 16 stages.  192-column tiles moved the 512-row
        // projections of a 32-layer stack's block-only forwards (12288 and
        // 24576 columns) from 192 to 256 workgroups: those forwards 13.9 ->
        // 13.4 ms.
        int ksplit = 1, mi = 4, nj = 4;
        double best = 1e30;
        for (int cm = 4; cm >= 3; --cm) {
            for (int cn = 4; cn >= 3; --cn) {
                const int rows = 64 * cm, cols = 64 * cn;
                const long tiles = static_cast<long>(ceil_div(m_max, rows)) * ceil_div(N, cols);
                const double rate = (cm == 4 ? 1.0 : kTile192Rate) * (cn == 4 ? 1.0 : kTile192Rate);
                const double tile_us = static_cast<double>(rows) * cols * 2.0 * K / (3.9e6 * rate);
                for (int k = 1; k <= kMaxSplit; ++k) {
                    if (nstage % (4 * k) != 0 || nstage / k < 16) continue;
                    const double rounds = static_cast<double>((tiles * k + kTargetWgs - 1) / kTargetWgs);
                    const double cost = rounds * tile_us / k + (k > 1 ? 8.0 * k * m_max * N / 5e6 : 0.0);
                    if (cost < best) {
                        best = cost;
                        ksplit = k;
                        mi = cm;
                        nj = cn;
                    }
                }
            }
        }
        p.tile_mi = mi;
        p.tile_nj = nj;
        p.row_tiles = ceil_div(m_max, 64 * mi);
        const long tiles = static_cast<long>(p.row_tiles) * ceil_div(N, 64 * nj);
        p.tile = tiles * ksplit >= kTargetWgs / 2 &&
                 (ksplit <= 4 || nstage / ksplit >= 48 || p.row_tiles >= 4);
        p.ksplit = ksplit;
    }
    if (p.tile) {
        const int nstage = K / (kTileStage / 2);
        const long tiles = static_cast<long>(p.row_tiles) * ceil_div(N, 64 * p.tile_nj);
        const int ksplit = p.ksplit;
        p.steps_per_split = nstage / ksplit;
        p.mt = 2 * p.tile_mi;
        p.grid = static_cast<int>(tiles * ksplit);
        if (p.ksplit > 1)
            p.ws_bytes = partial_bytes(p, m_max) + align_up(static_cast<size_t>(m_max) * 2 * sizeof(int), 256);
        return p;
    }
    // DMA kernel: up to two row tiles of at most 160 rows (eight for narrow
    // outputs), K split evenly
    // into 8 to 16 stages of 128 bytes per row; the split with the fewest
    // rounds of one workgroup per CU times stages per split, the smaller
    // split on ties (the Dream-7B Q projection, 56 tiles of K = 3584: four
    // splits of 14 stages in one round rather than seven of 8 in two)
    const bool dma_rows = bf16 && (m_max <= 2L * 16 * kDmaMaxRowTiles || narrow_dma);
    p.row_tiles = dma_rows ? ceil_div(m_max, 16L * kDmaMaxRowTiles) : ceil_div(m_max, 256);
    const long tiles = static_cast<long>(p.row_tiles) * p.col_tiles;
    int ksplit = 1;
    if (tiles < kTargetWgs) ksplit = ceil_div(kTargetWgs, tiles);
    if (ksplit > kMaxSplit) ksplit = kMaxSplit;
    if (ksplit > nsteps) ksplit = nsteps;
    p.steps_per_split = ceil_div(nsteps, ksplit);
    p.ksplit = ceil_div(nsteps, p.steps_per_split);
    p.dma = false;
    long best = -1;
    for (int ks = 1; dma_rows && ks <= kMaxSplit; ++ks) {
        if (nsteps % ks != 0 || nsteps / ks < 4 || nsteps / ks > 8) continue;
        const long cost = (tiles * ks + kTargetWgs - 1) / kTargetWgs * (nsteps / ks);
        if (best < 0 || cost < best) {
            best = cost;
            p.dma = true;
            p.ksplit = ks;
            p.steps_per_split = nsteps / ks;
        }
    }
    if (!p.dma) p.row_tiles = ceil_div(m_max, 256);
    p.mt = p.dma ? ceil_div(ceil_div(m_max, p.row_tiles), 16) : ceil_div(m_max, 32L * p.row_tiles);
    p.grid = static_cast<int>(static_cast<long>(p.row_tiles) * p.col_tiles * p.ksplit);
    if (p.ksplit > 1)
        p.ws_bytes = partial_bytes(p, m_max) + align_up(static_cast<size_t>(m_max) * 2 * sizeof(int), 256);
    return p;
}

GemmArgs refresh_gemm_args(int batch, int seq, int d, int kvd, const void* h_cur, const int32_t* stale_idx,
                           const int32_t* stale_count, int k_max, int block_start, int block_len,
                           const void* w_k, const void* w_v, void* k_cache, void* v_cache, void* workspace) {
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
    g.m_max = batch * (k_max + block_len);
    return g;
}

void gemm_finalize_args(const GemmPlan& p, GemmArgs& g) {
    g.rowmap = p.ksplit > 1 ? reinterpret_cast<int*>(reinterpret_cast<char*>(g.ws) + partial_bytes(p, g.m_max))
                            : nullptr;
    g.ksplit = p.ksplit;
    g.steps_per_split = p.steps_per_split;
    g.row_tiles = p.row_tiles;
    g.col_tiles = p.col_tiles;
}

int gemm_reduce_blocks(const GemmPlan& p, const GemmArgs& g) {
    if (p.small || p.ksplit == 1) return 0;
    return ceil_div(static_cast<long>(p.col_tiles) * g.m_max * 16, kGemmBlock);
}

// The tile kernel of the plan's tile shape (false for a shape not instantiated).
static bool launch_tile(const GemmPlan& p, const GemmArgs& g, hipStream_t stream) {
    const dim3 grid(p.grid), block(kTileThreads);
    switch (10 * p.tile_mi + p.tile_nj) {
        case 44: hipLaunchKernelGGL((gemm_tile_kernel<4, 4>), grid, block, 0, stream, g); return true;
        case 43: hipLaunchKernelGGL((gemm_tile_kernel<4, 3>), grid, block, 0, stream, g); return true;
        case 34: hipLaunchKernelGGL((gemm_tile_kernel<3, 4>), grid, block, 0, stream, g); return true;
        case 33: hipLaunchKernelGGL((gemm_tile_kernel<3, 3>), grid, block, 0, stream, g); return true;
        default: return false;
    }
}

polestar_status gemm_run(bool bf16, const GemmPlan& p, GemmArgs g, hipStream_t stream, GemmArgs* deferred) {
    gemm_finalize_args(p, g);
    bool ok;
    if (p.small) ok = bf16 ? dispatch_small<true>(p, g, stream) : dispatch_small<false>(p, g, stream);
    else if (p.tile) {
        ok = bf16 && p.steps_per_split % 4 == 0;
        if (ok) ok = launch_tile(p, g, stream);
    } else if (p.dma) ok = bf16 && dispatch_dma<true>(p, g, stream);
    else ok = bf16 ? dispatch_rows<true>(p, g, stream) : dispatch_rows<false>(p, g, stream);
    if (!ok) return POLESTAR_ERR_UNSUPPORTED;
    polestar_status st = launch_status();
    if (st != POLESTAR_OK || p.small || p.ksplit == 1) return st;
    if (deferred) {   // the caller launches the reduction (fused with other work)
        *deferred = g;
        return POLESTAR_OK;
    }
    const int blocks = gemm_reduce_blocks(p, g);
    if (bf16)
        hipLaunchKernelGGL((gemm_reduce_kernel<true>), dim3(blocks), dim3(kGemmBlock), 0, stream, g);
    else
        hipLaunchKernelGGL((gemm_reduce_kernel<false>), dim3(blocks), dim3(kGemmBlock), 0, stream, g);
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
    if ((head_dim != 64 && head_dim != 128) || !gemm_k_ok(dtype == POLESTAR_BF16, d) ||
        !aligned16(h_cur) || !aligned16(w_k) || !aligned16(w_v) || !aligned16(k_cache) ||
        !aligned16(v_cache) || !aligned16(workspace))
        return POLESTAR_ERR_UNSUPPORTED;
    if (batch > 65536) return POLESTAR_ERR_UNSUPPORTED;
    const long m_max = static_cast<long>(batch) * (k_max + block_len);
    if (m_max == 0) return POLESTAR_OK;
    if (m_max > 0x7fffffffL / 4) return POLESTAR_ERR_UNSUPPORTED;
    const bool bf16 = dtype == POLESTAR_BF16;
    const int kvd = n_kv_heads * head_dim;
    const GemmPlan p = gemm_plan(bf16, m_max, 2 * kvd, d);
    if (workspace_bytes < p.ws_bytes || (p.ws_bytes > 0 && !workspace)) return POLESTAR_ERR_WORKSPACE;
    const GemmArgs g = refresh_gemm_args(batch, seq, d, kvd, h_cur, stale_idx, stale_count, k_max, block_start,
                                         block_len, w_k, w_v, k_cache, v_cache, workspace);
    return gemm_run(bf16, p, g, stream);
}

// ---------------------------------------------------------------------------
// polestar_refresh_kv_noalloc: polestar_refresh_kv with its split-K partials
// and row map in a file-scope device array instead of a caller workspace.
// Each device holds its own copy of the array; its address on a device is
// looked up once (hipGetSymbolAddress, with that device current) and kept,
// since the array's name in host code is only a host-side stand-in.  The
// kernels need no initialised scratch (every partial that the reduction
// reads is written first in the same call), so nothing is cleared.
// ---------------------------------------------------------------------------

namespace ps {
namespace {
constexpr size_t kScratchBytes = size_t{64} << 20;
constexpr int kMaxDevices = 64;
}  // namespace
}  // namespace ps

static __device__ __align__(256) char scratch[ps::kScratchBytes];

namespace ps {
namespace {

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's copy of the array, or nullptr if its address cannot
// be obtained (status in *st).
void* device_scratch(polestar_status* st) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
        *st = dev >= kMaxDevices ? POLESTAR_ERR_UNSUPPORTED : POLESTAR_ERR_LAUNCH;
        return nullptr;
    }
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
            *st = POLESTAR_ERR_LAUNCH;
            return nullptr;
        }
        g_scratch_ptr[dev] = p;
    }
    return g_scratch_ptr[dev];
}

}  // namespace
}  // namespace ps

extern "C" size_t polestar_refresh_kv_noalloc_max_bytes(void) { return ps::kScratchBytes; }

extern "C" polestar_status polestar_refresh_kv_noalloc(polestar_dtype dtype, int batch, int seq, int d,
                                                       int n_kv_heads, int head_dim, const void* h_cur,
                                                       const int32_t* stale_idx,
                                                       const int32_t* stale_count, int k_max,
                                                       int block_start, int block_len, const void* w_k,
                                                       const void* w_v, void* k_cache, void* v_cache,
                                                       hipStream_t stream) {
    using namespace ps;
    // The same validation as polestar_refresh_kv, before the scratch lookup.
    if (!dtype_ok(dtype) || batch <= 0 || seq <= 0 || d <= 0 || n_kv_heads <= 0 ||
        head_dim <= 0 || k_max < 0 || k_max > seq || block_start < 0 || block_len < 0 ||
        block_start > seq - block_len || !h_cur || !w_k || !w_v || !k_cache || !v_cache ||
        (k_max > 0 && (!stale_idx || !stale_count)))
        return POLESTAR_ERR_INVALID_ARGUMENT;
    if ((head_dim != 64 && head_dim != 128) || !gemm_k_ok(dtype == POLESTAR_BF16, d) ||
        !aligned16(h_cur) || !aligned16(w_k) || !aligned16(w_v) || !aligned16(k_cache) ||
        !aligned16(v_cache))
        return POLESTAR_ERR_UNSUPPORTED;
    if (batch > 65536) return POLESTAR_ERR_UNSUPPORTED;
    const long m_max = static_cast<long>(batch) * (k_max + block_len);
    if (m_max == 0) return POLESTAR_OK;
    if (m_max > 0x7fffffffL / 4) return POLESTAR_ERR_UNSUPPORTED;
    const bool bf16 = dtype == POLESTAR_BF16;
    const int kvd = n_kv_heads * head_dim;
    const GemmPlan p = gemm_plan(bf16, m_max, 2 * kvd, d);
    if (p.ws_bytes > kScratchBytes) return POLESTAR_ERR_WORKSPACE;
    void* ws = nullptr;
    if (p.ws_bytes > 0) {
        polestar_status st = POLESTAR_OK;
        ws = device_scratch(&st);
        if (!ws) return st;
    }
    const GemmArgs g = refresh_gemm_args(batch, seq, d, kvd, h_cur, stale_idx, stale_count, k_max, block_start,
                                         block_len, w_k, w_v, k_cache, v_cache, ws);
    return gemm_run(bf16, p, g, stream);
}
