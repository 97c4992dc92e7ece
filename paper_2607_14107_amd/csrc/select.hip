// polestar_select: TopK of the drift over the cached positions of each
// sequence (Alg. 1, TopK; cached set I = J \ J_b of Sec. 2).  The algorithm
// lives in select_dev.hpp; this file launches it, one workgroup per sequence.
#include "host_common.hpp"
#include "select_dev.hpp"

namespace ps {
namespace {

template <int IPT>
__global__ __launch_bounds__(kSelBlock) void select_kernel(const float* __restrict__ drift,
                                                           const uint8_t* __restrict__ elig,
                                                           int seq, int bs, int bl, int k,
                                                           int32_t* __restrict__ idx,
                                                           int32_t* __restrict__ cnt) {
    select_body<IPT>(drift, elig, seq, bs, bl, k, idx, cnt, blockIdx.x);
}

template <int IPT>
void launch(int batch, int seq, const float* drift, const uint8_t* elig, int bs, int bl, int k,
            int32_t* idx, int32_t* cnt, hipStream_t s) {
    hipLaunchKernelGGL((select_kernel<IPT>), dim3(batch), dim3(kSelBlock), 0, s, drift, elig, seq,
                       bs, bl, k, idx, cnt);
}

}  // namespace
}  // namespace ps

extern "C" polestar_status polestar_select(int batch, int seq, const float* drift,
                                           const uint8_t* eligible, int block_start,
                                           int block_len, int k, int32_t* stale_idx,
                                           int32_t* stale_count, hipStream_t stream) {
    using namespace ps;
    if (batch <= 0 || seq <= 0 || !drift || !stale_count || block_start < 0 || block_len < 0 ||
        block_start > seq - block_len || k < 0 || k > seq || (k > 0 && !stale_idx))
        return POLESTAR_ERR_INVALID_ARGUMENT;
    const int ipt = ceil_div(seq, kSelBlock);
    int32_t* idx = stale_idx;
    if (ipt <= 1) launch<1>(batch, seq, drift, eligible, block_start, block_len, k, idx, stale_count, stream);
    else if (ipt <= 2) launch<2>(batch, seq, drift, eligible, block_start, block_len, k, idx, stale_count, stream);
    else if (ipt <= 3) launch<3>(batch, seq, drift, eligible, block_start, block_len, k, idx, stale_count, stream);
    else if (ipt <= 4) launch<4>(batch, seq, drift, eligible, block_start, block_len, k, idx, stale_count, stream);
    else if (ipt <= 6) launch<6>(batch, seq, drift, eligible, block_start, block_len, k, idx, stale_count, stream);
    else if (ipt <= 8) launch<8>(batch, seq, drift, eligible, block_start, block_len, k, idx, stale_count, stream);
    else if (ipt <= 16) launch<16>(batch, seq, drift, eligible, block_start, block_len, k, idx, stale_count, stream);
    else if (ipt <= 32) launch<32>(batch, seq, drift, eligible, block_start, block_len, k, idx, stale_count, stream);
    else if (ipt <= 64) launch<64>(batch, seq, drift, eligible, block_start, block_len, k, idx, stale_count, stream);
    else return POLESTAR_ERR_UNSUPPORTED;   // seq above 16384
    return launch_status();
}
