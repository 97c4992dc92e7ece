// Skinny "gather rows -> MFMA GEMM -> scatter rows" used by the K/V refresh
// (stale rows plus the active block, scattered into the caches) and by the
// Q projection of the active block (dense output).  Internal to the library.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "polestar.h"

namespace ps {

enum GemmMode : int { kGemmRefresh = 0, kGemmBlockRows = 1 };

// Y[m][n] = sum_k X[row(m)][k] * W[n][k], W = w0 for n < n0, else w1 (row n - n0).
struct GemmArgs {
    const char* x;        // [batch][seq][K] input rows
    const char* w0;
    const char* w1;
    int n0;
    int N, K;
    int mode;
    int batch, seq;
    const int32_t* stale_idx;    // refresh mode: [batch][k_max]
    const int32_t* stale_count;  // refresh mode: [batch]
    int k_max;
    int block_start, block_len;
    char* out0;   // refresh: k_cache (row pitch n0); block rows: [rows][N]
    char* out1;   // refresh: v_cache (row pitch N - n0)
    float* ws;          // split-K partials [split][col_tile][m_max][128] fp32
    int* rowmap;        // split-K: [m_max][2] (sequence, position) of row m, -1: none
    int m_max;
    int ksplit;
    int steps_per_split;   // 256-byte super-steps per split (tile kernel: 64-byte stages)
    int row_tiles, col_tiles;
};

struct GemmPlan {
    bool small;         // gemm_small_kernel (<= 64 rows) instead of gemm_rows_kernel
    bool dma;           // gemm_dma_kernel (17..320 rows in up to two row tiles, up to 1280 in eight for
                        // outputs of <= 1024 columns; operands DMA'd into LDS)
    bool tile;          // gemm_tile_kernel (bf16, more than 160 rows: 256- or 192-row x 256- or 192-column tiles)
    int tile_mi;        // tile kernel: 32-row MFMA tiles per wave down the rows (4: 256-row tiles, 3: 192)
    int tile_nj;        // tile kernel: 32-column MFMA tiles per wave across (4: 256-column tiles, 3: 192)
    int mt;             // MFMA row tiles per workgroup (16 rows: small and dma kernels; 32: rows and tile kernels)
    int row_tiles;
    int col_tiles;
    int ksplit;
    int steps_per_split;   // 256-byte super-steps per split (tile kernel: 64-byte stages)
    int grid;           // workgroups of gemm_rows_kernel
    size_t ws_bytes;    // fp32 partials + row map, 0 when ksplit == 1
};

GemmPlan gemm_plan(bool bf16, long m_max, int N, int K);

// The GEMMs stream K in super-steps of 256 bytes per row: 128 bf16 or 64 fp32.
inline bool gemm_k_ok(bool bf16, int K) { return K > 0 && K % (bf16 ? 128 : 64) == 0; }

// Enqueue the GEMM (and the split-K reduction when the plan splits K).
// `g.ws` must hold plan.ws_bytes.  With `deferred`, a plan that needs the
// reduction leaves it to the caller: *deferred receives the arguments of
// the reduction (reduce_body, gemm_reduce_blocks workgroups).  Returns
// POLESTAR_OK or a launch error.
polestar_status gemm_run(bool bf16, const GemmPlan& plan, GemmArgs g, hipStream_t stream,
                         GemmArgs* deferred = nullptr);

// Arguments of the K/V refresh GEMM (polestar_refresh_kv's, after its checks):
// rows = the stale positions and the active block of every sequence, output
// columns [0, kvd) to k_cache and [kvd, 2 kvd) to v_cache.
GemmArgs refresh_gemm_args(int batch, int seq, int d, int kvd, const void* h_cur, const int32_t* stale_idx,
                           const int32_t* stale_count, int k_max, int block_start, int block_len,
                           const void* w_k, const void* w_v, void* k_cache, void* v_cache, void* workspace);

// The plan's fields of the arguments (split, tiles, row map in the workspace).
void gemm_finalize_args(const GemmPlan& plan, GemmArgs& g);

// Workgroups of the split-K reduction of a plan (0: none).
int gemm_reduce_blocks(const GemmPlan& plan, const GemmArgs& g);

}  // namespace ps
