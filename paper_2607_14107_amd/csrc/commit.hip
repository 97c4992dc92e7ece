// polestar_commit: Polestar-Commit for the current block (Sec. 4.2, Alg. 1)
// on top of the confidence of Sec. 2 / eq. 1.  The device code lives in
// commit_dev.hpp; this file launches the vocabulary scan (workgroup per
// token and vocabulary slice) and the finalize step (workgroup per sequence).
#include "commit_dev.hpp"
#include "host_common.hpp"

namespace ps {
namespace {

template <bool BF16>
__global__ __launch_bounds__(kScanBlock) void scan_kernel(const char* __restrict__ logits, int vocab,
                                                          int nq, int chunk, int splits, int mask_id,
                                                          ScanPart* __restrict__ parts) {
    scan_body<BF16>(logits, vocab, nq, chunk, splits, mask_id, parts, blockIdx.x, blockIdx.y, blockIdx.z);
}

__global__ __launch_bounds__(1024) void finalize_kernel(const ScanPart* __restrict__ parts, int splits,
                                                        int nq, const uint8_t* __restrict__ masked,
                                                        const uint8_t* __restrict__ eligible,
                                                        const float* __restrict__ drift, int seq,
                                                        int block_start, float* hist, int32_t* hist_len,
                                                        int h, float tau_s, float alpha, int force_one,
                                                        int32_t* __restrict__ token,
                                                        float* __restrict__ conf,
                                                        uint8_t* __restrict__ commit) {
    finalize_body(parts, splits, nq, masked, eligible, drift, seq, block_start, hist, hist_len, h, tau_s, alpha,
                  force_one, token, conf, commit, blockIdx.x);
}

polestar_status launch_scan(bool bf16, const CommitPlan& p, int batch, int nq, int vocab, const void* logits,
                            int mask_token_id, ScanPart* parts, hipStream_t stream) {
    dim3 grid(p.splits, nq, batch);
    if (bf16)
        hipLaunchKernelGGL((scan_kernel<true>), grid, dim3(kScanBlock), 0, stream,
                           static_cast<const char*>(logits), vocab, nq, p.chunk, p.splits, mask_token_id, parts);
    else
        hipLaunchKernelGGL((scan_kernel<false>), grid, dim3(kScanBlock), 0, stream,
                           static_cast<const char*>(logits), vocab, nq, p.chunk, p.splits, mask_token_id, parts);
    return launch_status();
}

}  // namespace
}  // namespace ps

extern "C" size_t polestar_commit_workspace_size(polestar_dtype dtype, int batch, int block_len,
                                                 int vocab) {
    using namespace ps;
    if (!dtype_ok(dtype) || batch <= 0 || block_len <= 0 || vocab <= 0) return 0;
    return commit_plan(dtype == POLESTAR_BF16, batch, block_len, vocab).ws_bytes;
}

extern "C" polestar_status polestar_commit(polestar_dtype dtype, int batch, int block_len, int vocab,
                                           const void* logits, const uint8_t* masked,
                                           const float* drift, int seq, int block_start,
                                           float* hist, int32_t* hist_len, int h,
                                           int mask_token_id, float tau_s, float alpha,
                                           int force_one, int32_t* token, float* conf,
                                           uint8_t* commit, void* workspace,
                                           size_t workspace_bytes, hipStream_t stream) {
    using namespace ps;
    if (!dtype_ok(dtype) || batch <= 0 || block_len <= 0 || vocab <= 0 || h < 0 || !logits ||
        !masked || !token || !conf || !commit || mask_token_id >= vocab ||
        (h > 0 && drift && (!hist || !hist_len)) ||
        (drift && (seq <= 0 || block_start < 0 || block_start > seq - block_len)))
        return POLESTAR_ERR_INVALID_ARGUMENT;
    if (!row_ok(dtype, vocab) || !aligned16(logits) || block_len > 1024 || batch > 65535 ||
        h > kMaxHist)
        return POLESTAR_ERR_UNSUPPORTED;
    const bool bf16 = dtype == POLESTAR_BF16;
    const CommitPlan p = commit_plan(bf16, batch, block_len, vocab);
    if (workspace_bytes < p.ws_bytes || !workspace) return POLESTAR_ERR_WORKSPACE;
    ScanPart* parts = static_cast<ScanPart*>(workspace);
    polestar_status st = launch_scan(bf16, p, batch, block_len, vocab, logits, mask_token_id, parts, stream);
    if (st != POLESTAR_OK) return st;
    const int threads = ceil_div(block_len, 64) * 64;
    const bool use_hist = h > 0 && drift;
    hipLaunchKernelGGL(finalize_kernel, dim3(batch), dim3(threads), 0, stream, parts, p.splits,
                       block_len, masked, nullptr, drift, seq, block_start, use_hist ? hist : nullptr,
                       use_hist ? hist_len : nullptr, use_hist ? h : 0, tau_s, alpha, force_one,
                       token, conf, commit);
    return launch_status();
}

// Suffix-block commit (Sec. 4.2 "Suffix Block Commit"; Alg. 1, last commit of
// a step): the vocabulary scan of the packet rows, then the confidence rule
// alone on the positions that are masked and eligible.
extern "C" polestar_status polestar_suffix_commit(polestar_dtype dtype, int batch, int n_rows, int vocab,
                                                  const void* logits, const uint8_t* masked,
                                                  const uint8_t* eligible, int mask_token_id, float tau_s,
                                                  int32_t* token, float* conf, uint8_t* commit,
                                                  void* workspace, size_t workspace_bytes,
                                                  hipStream_t stream) {
    using namespace ps;
    if (!dtype_ok(dtype) || batch <= 0 || n_rows <= 0 || vocab <= 0 || !logits || !masked || !eligible ||
        !token || !conf || !commit || mask_token_id >= vocab)
        return POLESTAR_ERR_INVALID_ARGUMENT;
    if (!row_ok(dtype, vocab) || !aligned16(logits) || n_rows > 1024 || batch > 65535)
        return POLESTAR_ERR_UNSUPPORTED;
    const bool bf16 = dtype == POLESTAR_BF16;
    const CommitPlan p = commit_plan(bf16, batch, n_rows, vocab);
    if (workspace_bytes < p.ws_bytes || !workspace) return POLESTAR_ERR_WORKSPACE;
    ScanPart* parts = static_cast<ScanPart*>(workspace);
    polestar_status st = launch_scan(bf16, p, batch, n_rows, vocab, logits, mask_token_id, parts, stream);
    if (st != POLESTAR_OK) return st;
    const int threads = ceil_div(n_rows, 64) * 64;
    hipLaunchKernelGGL(finalize_kernel, dim3(batch), dim3(threads), 0, stream, parts, p.splits, n_rows, masked,
                       eligible, nullptr, 0, 0, nullptr, nullptr, 0, tau_s, 0.f, 0, token, conf, commit);
    return launch_status();
}
