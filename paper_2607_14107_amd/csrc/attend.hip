// polestar_attend and polestar_project_q: the Q projection of the active
// block (the shared skinny GEMM of gemm.hip) and the split-key flash
// attention of attend_dev.hpp, launched with their plans and workspaces.
#include "attend_dev.hpp"
#include "gemm.hpp"
#include "host_common.hpp"

namespace ps {
namespace {

struct AttendLayout {
    GemmPlan qp;
    AttPlan ap;
    size_t q_ws;       // offset of attention partials
    size_t total;
};

// Q = W_q h_cur[b][block rows] through the shared GEMM (block-rows mode).
polestar_status run_q_projection(bool bf16, const GemmPlan& plan, int batch, int seq, int d, int H,
                                 int hd, int block_start, int block_len, const void* h_cur,
                                 const void* w_q, void* q, char* ws, hipStream_t stream) {
    GemmArgs g{};
    g.x = static_cast<const char*>(h_cur);
    g.w0 = static_cast<const char*>(w_q);
    g.w1 = nullptr;
    g.n0 = H * hd;
    g.N = H * hd;
    g.K = d;
    g.mode = kGemmBlockRows;
    g.batch = batch;
    g.seq = seq;
    g.block_start = block_start;
    g.block_len = block_len;
    g.out0 = static_cast<char*>(q);
    g.ws = reinterpret_cast<float*>(ws);
    g.m_max = batch * block_len;
    return gemm_run(bf16, plan, g, stream);
}

}  // namespace
}  // namespace ps

extern "C" size_t polestar_project_q_workspace_size(polestar_dtype dtype, int batch, int d,
                                                    int n_heads, int head_dim, int block_len) {
    using namespace ps;
    if (!dtype_ok(dtype) || batch <= 0 || d <= 0 || n_heads <= 0 || head_dim <= 0 || block_len <= 0)
        return 0;
    return gemm_plan(dtype == POLESTAR_BF16, static_cast<long>(batch) * block_len, n_heads * head_dim, d)
        .ws_bytes;
}

extern "C" polestar_status polestar_project_q(polestar_dtype dtype, int batch, int seq, int d,
                                              int n_heads, int head_dim, int block_start,
                                              int block_len, const void* h_cur, const void* w_q,
                                              void* q, void* workspace, size_t workspace_bytes,
                                              hipStream_t stream) {
    using namespace ps;
    if (!dtype_ok(dtype) || batch <= 0 || seq <= 0 || d <= 0 || n_heads <= 0 || head_dim <= 0 ||
        block_len <= 0 || block_start < 0 || block_start > seq - block_len || !h_cur || !w_q || !q)
        return POLESTAR_ERR_INVALID_ARGUMENT;
    const bool bf16 = dtype == POLESTAR_BF16;
    if ((head_dim != 64 && head_dim != 128) || !gemm_k_ok(bf16, d) || !aligned16(h_cur) ||
        !aligned16(w_q) || !aligned16(q) || !aligned16(workspace) || batch > 65535 ||
        static_cast<long>(batch) * block_len > 0x7fffffffL / 4)
        return POLESTAR_ERR_UNSUPPORTED;
    const GemmPlan plan = gemm_plan(bf16, static_cast<long>(batch) * block_len, n_heads * head_dim, d);
    if (workspace_bytes < plan.ws_bytes || (plan.ws_bytes > 0 && !workspace)) return POLESTAR_ERR_WORKSPACE;
    return run_q_projection(bf16, plan, batch, seq, d, n_heads, head_dim, block_start, block_len, h_cur,
                            w_q, q, static_cast<char*>(workspace), stream);
}

namespace ps {
namespace {
AttendLayout attend_layout(bool bf16, int batch, int seq, int d, int H, int Hkv, int hd, int nq,
                           bool project) {
    AttendLayout L{};
    if (project) L.qp = gemm_plan(bf16, static_cast<long>(batch) * nq, H * hd, d);
    L.ap = att_plan(bf16, batch, seq, H, Hkv, nq, hd);
    L.q_ws = align_up(L.qp.ws_bytes, 256);
    L.total = L.q_ws + L.ap.part_bytes;
    return L;
}

}  // namespace
}  // namespace ps

extern "C" size_t polestar_attend_workspace_size(polestar_dtype dtype, int batch, int seq, int d,
                                                 int n_heads, int n_kv_heads, int head_dim,
                                                 int block_len) {
    using namespace ps;
    if (!dtype_ok(dtype) || batch <= 0 || seq <= 0 || d <= 0 || n_heads <= 0 || n_kv_heads <= 0 ||
        head_dim <= 0 || block_len <= 0)
        return 0;
    return attend_layout(dtype == POLESTAR_BF16, batch, seq, d, n_heads, n_kv_heads, head_dim, block_len, true)
        .total;
}

extern "C" polestar_status polestar_attend(polestar_dtype dtype, int batch, int seq, int d,
                                           int n_heads, int n_kv_heads, int head_dim,
                                           int block_start, int block_len, const void* h_cur,
                                           const void* w_q, void* q_buf, const void* k_cache,
                                           const void* v_cache, float scale, void* out, float* lse,
                                           void* workspace, size_t workspace_bytes,
                                           hipStream_t stream) {
    using namespace ps;
    if (!dtype_ok(dtype) || batch <= 0 || seq <= 0 || d <= 0 || n_heads <= 0 || n_kv_heads <= 0 ||
        head_dim <= 0 || block_len <= 0 || block_start < 0 || block_start > seq - block_len ||
        n_heads % n_kv_heads != 0 || !q_buf || !k_cache || !v_cache || !out ||
        (w_q && !h_cur))
        return POLESTAR_ERR_INVALID_ARGUMENT;
    if ((head_dim != 64 && head_dim != 128) || (w_q && !gemm_k_ok(dtype == POLESTAR_BF16, d)) ||
        !aligned16(q_buf) ||
        !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(out) || !aligned16(workspace) ||
        (w_q && (!aligned16(w_q) || !aligned16(h_cur))))
        return POLESTAR_ERR_UNSUPPORTED;
    if (batch > 65535 || static_cast<long>(n_heads) * ceil_div(block_len, kQG) > 65535)
        return POLESTAR_ERR_UNSUPPORTED;
    const bool bf16 = dtype == POLESTAR_BF16;
    const AttendLayout L =
        attend_layout(bf16, batch, seq, d, n_heads, n_kv_heads, head_dim, block_len, w_q != nullptr);
    if (workspace_bytes < L.total || (L.total > 0 && !workspace)) return POLESTAR_ERR_WORKSPACE;
    char* ws = static_cast<char*>(workspace);

    if (w_q) {
        polestar_status st = run_q_projection(bf16, L.qp, batch, seq, d, n_heads, head_dim, block_start,
                                              block_len, h_cur, w_q, q_buf, ws, stream);
        if (st != POLESTAR_OK) return st;
    }

    const AttArgs a = att_args(L.ap, batch, seq, block_len, n_heads, n_kv_heads, head_dim, q_buf, k_cache,
                               v_cache, out, lse, scale, L.ap.splits > 1 ? ws + L.q_ws : nullptr);
    if (bf16) {
        if (head_dim == 128) launch_att<true, 128>(L.ap, a, stream);
        else launch_att<true, 64>(L.ap, a, stream);
    } else {
        if (head_dim == 128) launch_att<false, 128>(L.ap, a, stream);
        else launch_att<false, 64>(L.ap, a, stream);
    }
    polestar_status st = launch_status();
    if (st != POLESTAR_OK || L.ap.splits == 1) return st;
    if (bf16) {
        if (head_dim == 128) launch_merge<true, 128>(a, stream);
        else launch_merge<true, 64>(a, stream);
    } else {
        if (head_dim == 128) launch_merge<false, 128>(a, stream);
        else launch_merge<false, 64>(a, stream);
    }
    return launch_status();
}
