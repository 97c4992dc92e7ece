// polestar_step: one whole layer step (drift -> select -> K/V refresh -> Q
// projection -> attention -> commit) on one stream, with the work that does
// not depend on the previous launch fused into shared launches:
//
//   1. drift                          (every position)
//   2. front: select | Q projection | vocabulary scan
//      The select of a sequence is one latency-bound workgroup; the Q
//      projection and the logit scan read only the step's inputs, so they
//      fill the GPU while it runs.
//   3. refresh: gather -> GEMM -> split-K reduce -> scatter (needs 2)
//   4. attention over the refreshed cache (needs 2, 3)
//   5. back: attention merge | commit finalize (needs 4, and 1-2)
//
// Five launch groups instead of nine kernels on their own.  Workgroups of a
// fused launch take their role from their block index; each role is the
// device body the stand-alone kernel runs, so results are bit-identical to
// calling the six entry points in order.  Shapes outside the fused kernels'
// instantiations (more than 2048 positions, more than 64 query rows, blocks
// longer than 256) run exactly that sequence of entry points instead.
#include "attend_dev.hpp"
#include "commit_dev.hpp"
#include "gemm_dev.hpp"
#include "host_common.hpp"
#include "select_dev.hpp"

namespace ps {
namespace {

constexpr int kStepBlock = 256;
static_assert(kSelBlock == kStepBlock && kSmallBlock == kStepBlock && kScanBlock == kStepBlock &&
                  kAttBlock == kStepBlock,
              "fused roles share one workgroup size");

struct FrontArgs {
    // select
    const float* drift;
    const uint8_t* elig;
    int seq, bs, bl, k;
    int32_t* idx;
    int32_t* cnt;
    // Q projection (block rows, at most 64 of them)
    GemmArgs q;
    // vocabulary scan
    const char* logits;
    int vocab, nq, chunk, splits, mask_id;
    ScanPart* parts;
    // workgroups per role, in launch order
    int n_sel, n_q;
};

template <bool BF16, int IPT, int MT>
__global__ __launch_bounds__(kStepBlock) void front_kernel(FrontArgs f) {
    int vb = blockIdx.x;
    if (vb < f.n_sel) {
        select_body<IPT>(f.drift, f.elig, f.seq, f.bs, f.bl, f.k, f.idx, f.cnt, vb);
        return;
    }
    vb -= f.n_sel;
    if (vb < f.n_q) {
        small_body<BF16, MT>(f.q, vb, 0);
        return;
    }
    vb -= f.n_q;
    const int split = vb % f.splits;
    const int tok = vb / f.splits;
    scan_body<BF16>(f.logits, f.vocab, f.nq, f.chunk, f.splits, f.mask_id, f.parts, split, tok % f.nq,
                    tok / f.nq);
}

struct BackArgs {
    AttArgs att;
    int n_merge;
    const ScanPart* parts;
    int splits, nq;
    const uint8_t* masked;
    const float* drift;
    int seq, block_start;
    float* hist;
    int32_t* hist_len;
    int h;
    float tau_s, alpha;
    int force_one;
    int32_t* token;
    float* conf;
    uint8_t* commit;
};

template <bool BF16, int HD>
__global__ __launch_bounds__(kStepBlock) void back_kernel(BackArgs k) {
    if (static_cast<int>(blockIdx.x) < k.n_merge) {
        merge_body<BF16, HD>(k.att, blockIdx.x);
        return;
    }
    finalize_body(k.parts, k.splits, k.nq, k.masked, nullptr, k.drift, k.seq, k.block_start, k.hist, k.hist_len,
                  k.h, k.tau_s, k.alpha, k.force_one, k.token, k.conf, k.commit,
                  blockIdx.x - k.n_merge);
}

template <bool BF16, int IPT>
bool launch_front_mt(int mt, dim3 grid, const FrontArgs& f, hipStream_t s) {
    switch (mt) {
        case 1: hipLaunchKernelGGL((front_kernel<BF16, IPT, 1>), grid, dim3(kStepBlock), 0, s, f); return true;
        case 2: hipLaunchKernelGGL((front_kernel<BF16, IPT, 2>), grid, dim3(kStepBlock), 0, s, f); return true;
        case 3: hipLaunchKernelGGL((front_kernel<BF16, IPT, 3>), grid, dim3(kStepBlock), 0, s, f); return true;
        case 4: hipLaunchKernelGGL((front_kernel<BF16, IPT, 4>), grid, dim3(kStepBlock), 0, s, f); return true;
        default: return false;
    }
}

template <bool BF16>
bool launch_front(int ipt, int mt, dim3 grid, const FrontArgs& f, hipStream_t s) {
    switch (ipt) {
        case 1: return launch_front_mt<BF16, 1>(mt, grid, f, s);
        case 2: return launch_front_mt<BF16, 2>(mt, grid, f, s);
        case 3: return launch_front_mt<BF16, 3>(mt, grid, f, s);
        case 4: return launch_front_mt<BF16, 4>(mt, grid, f, s);
        case 6: return launch_front_mt<BF16, 6>(mt, grid, f, s);
        case 8: return launch_front_mt<BF16, 8>(mt, grid, f, s);
        default: return false;
    }
}

template <bool BF16>
void launch_back(int hd, dim3 grid, const BackArgs& k, hipStream_t s) {
    if (hd == 128) hipLaunchKernelGGL((back_kernel<BF16, 128>), grid, dim3(kStepBlock), 0, s, k);
    else hipLaunchKernelGGL((back_kernel<BF16, 64>), grid, dim3(kStepBlock), 0, s, k);
}

template <bool BF16>
void launch_attention(int hd, const AttPlan& p, const AttArgs& a, hipStream_t s) {
    if (hd == 128) launch_att<BF16, 128>(p, a, s);
    else launch_att<BF16, 64>(p, a, s);
}

// Workspace of the fused path: refresh partials, attention partials, scan
// partials, each 256-byte aligned.
struct StepLayout {
    GemmPlan qp;        // Q projection plan (small path when fused)
    AttPlan ap;
    CommitPlan cp;
    size_t refresh_bytes, att_off, scan_off, total;
    bool fused;
    int ipt;
};

StepLayout step_layout(const polestar_step_args& a) {
    StepLayout L{};
    const bool bf16 = a.dtype == POLESTAR_BF16;
    L.refresh_bytes = polestar_refresh_kv_workspace_size(a.dtype, a.batch, a.d, a.n_kv_heads, a.head_dim, a.k,
                                                         a.block_len);
    L.qp = gemm_plan(bf16, static_cast<long>(a.batch) * a.block_len, a.n_heads * a.head_dim, a.d);
    L.ap = att_plan(bf16, a.batch, a.seq, a.n_heads, a.n_kv_heads, a.block_len, a.head_dim);
    L.cp = commit_plan(bf16, a.batch, a.block_len, a.vocab);
    L.ipt = select_ipt(a.seq);
    L.fused = L.ipt >= 1 && L.ipt <= 8 && L.qp.small && a.block_len <= kStepBlock &&
              (a.head_dim == 64 || a.head_dim == 128);
    L.att_off = align_up(L.refresh_bytes, 256);
    L.scan_off = L.att_off + align_up(L.ap.part_bytes, 256);
    const size_t q_ws = align_up(L.qp.ws_bytes, 256);   // unfused path: stand-alone Q projection
    L.total = L.scan_off + align_up(L.cp.ws_bytes, 256) + (L.fused ? 0 : q_ws);
    return L;
}

// The six entry points in order (shapes the fused kernels do not cover).
polestar_status run_unfused(const polestar_step_args& a, const StepLayout& L, char* ws,
                            hipEvent_t ev0, hipEvent_t ev1, hipStream_t s) {
    polestar_status st = polestar_drift(a.dtype, a.batch, a.seq, a.d, a.h_cur, a.h_prev, a.drift, s);
    if (st != POLESTAR_OK) return st;
    st = polestar_select(a.batch, a.seq, a.drift, a.eligible, a.block_start, a.block_len, a.k, a.stale_idx,
                         a.stale_count, s);
    if (st != POLESTAR_OK) return st;
    if (ev0 && hipEventRecord(ev0, s) != hipSuccess) return POLESTAR_ERR_LAUNCH;
    st = polestar_refresh_kv(a.dtype, a.batch, a.seq, a.d, a.n_kv_heads, a.head_dim, a.h_cur, a.stale_idx,
                             a.stale_count, a.k, a.block_start, a.block_len, a.w_k, a.w_v, a.k_cache,
                             a.v_cache, ws, L.refresh_bytes, s);
    if (st != POLESTAR_OK) return st;
    if (ev1 && hipEventRecord(ev1, s) != hipSuccess) return POLESTAR_ERR_LAUNCH;
    const size_t q_off = L.scan_off + align_up(L.cp.ws_bytes, 256);
    st = polestar_project_q(a.dtype, a.batch, a.seq, a.d, a.n_heads, a.head_dim, a.block_start, a.block_len,
                            a.h_cur, a.w_q, a.q, L.qp.ws_bytes ? ws + q_off : nullptr, L.qp.ws_bytes, s);
    if (st != POLESTAR_OK) return st;
    st = polestar_attend(a.dtype, a.batch, a.seq, a.d, a.n_heads, a.n_kv_heads, a.head_dim, a.block_start,
                         a.block_len, nullptr, nullptr, a.q, a.k_cache, a.v_cache, a.scale, a.out, a.lse,
                         L.ap.part_bytes ? ws + L.att_off : nullptr, L.ap.part_bytes, s);
    if (st != POLESTAR_OK) return st;
    return polestar_commit(a.dtype, a.batch, a.block_len, a.vocab, a.logits, a.masked, a.drift, a.seq,
                           a.block_start, a.hist, a.hist_len, a.h, a.mask_token_id, a.tau_s, a.alpha,
                           a.force_one, a.token, a.conf, a.commit, ws + L.scan_off, L.cp.ws_bytes, s);
}

}  // namespace
}  // namespace ps

extern "C" size_t polestar_step_workspace_size(const polestar_step_args* a) {
    using namespace ps;
    if (!a || !dtype_ok(a->dtype) || a->batch <= 0 || a->seq <= 0 || a->d <= 0 || a->n_heads <= 0 ||
        a->n_kv_heads <= 0 || a->head_dim <= 0 || a->block_len <= 0 || a->vocab <= 0 || a->k < 0)
        return 0;
    return step_layout(*a).total;
}

extern "C" polestar_status polestar_step(const polestar_step_args* a, void* workspace,
                                         size_t workspace_bytes, hipEvent_t refresh_begin,
                                         hipEvent_t refresh_end, hipStream_t stream) {
    using namespace ps;
    if (!a || !dtype_ok(a->dtype) || a->batch <= 0 || a->seq <= 0 || a->d <= 0 || a->n_heads <= 0 ||
        a->n_kv_heads <= 0 || a->head_dim <= 0 || a->block_len <= 0 || a->vocab <= 0 || a->k < 0 ||
        a->k > a->seq || a->h < 0 || a->block_start < 0 || a->block_start > a->seq - a->block_len ||
        a->n_heads % a->n_kv_heads != 0 || !a->h_cur || !a->h_prev || !a->w_q || !a->w_k || !a->w_v ||
        !a->k_cache || !a->v_cache || !a->logits || !a->masked || !a->drift || !a->stale_count ||
        (a->k > 0 && !a->stale_idx) || !a->q || !a->out || !a->token || !a->conf || !a->commit ||
        a->mask_token_id >= a->vocab || (a->h > 0 && (!a->hist || !a->hist_len)))
        return POLESTAR_ERR_INVALID_ARGUMENT;
    const StepLayout L = step_layout(*a);
    if (workspace_bytes < L.total || !workspace) return POLESTAR_ERR_WORKSPACE;
    char* ws = static_cast<char*>(workspace);
    if (!L.fused) return run_unfused(*a, L, ws, refresh_begin, refresh_end, stream);

    const bool bf16 = a->dtype == POLESTAR_BF16;
    // Every check of the fused launches' stand-alone entry points, before
    // anything is enqueued.
    if (!row_ok(a->dtype, a->d) || !aligned16(a->h_cur) || !aligned16(a->h_prev) || !aligned16(a->drift) ||
        !gemm_k_ok(bf16, a->d) || !aligned16(a->w_q) || !aligned16(a->w_k) || !aligned16(a->w_v) ||
        !aligned16(a->q) || !aligned16(a->k_cache) || !aligned16(a->v_cache) || !aligned16(a->out) ||
        !aligned16(workspace) || !row_ok(a->dtype, a->vocab) || !aligned16(a->logits) || a->h > kMaxHist ||
        a->batch > 65535 || static_cast<long>(a->n_heads) * ceil_div(a->block_len, kQG) > 65535)
        return POLESTAR_ERR_UNSUPPORTED;

    // 1. drift
    polestar_status st = polestar_drift(a->dtype, a->batch, a->seq, a->d, a->h_cur, a->h_prev, a->drift, stream);
    if (st != POLESTAR_OK) return st;

    // 2. select | Q projection | vocabulary scan
    FrontArgs f{};
    f.drift = a->drift;
    f.elig = a->eligible;
    f.seq = a->seq;
    f.bs = a->block_start;
    f.bl = a->block_len;
    f.k = a->k;
    f.idx = a->stale_idx;
    f.cnt = a->stale_count;
    f.q.x = static_cast<const char*>(a->h_cur);
    f.q.w0 = static_cast<const char*>(a->w_q);
    f.q.n0 = a->n_heads * a->head_dim;
    f.q.N = a->n_heads * a->head_dim;
    f.q.K = a->d;
    f.q.mode = kGemmBlockRows;
    f.q.batch = a->batch;
    f.q.seq = a->seq;
    f.q.block_start = a->block_start;
    f.q.block_len = a->block_len;
    f.q.out0 = static_cast<char*>(a->q);
    f.q.m_max = a->batch * a->block_len;
    f.q.ksplit = 1;
    f.q.steps_per_split = L.qp.steps_per_split;
    f.q.row_tiles = 1;
    f.q.col_tiles = L.qp.col_tiles;
    f.logits = static_cast<const char*>(a->logits);
    f.vocab = a->vocab;
    f.nq = a->block_len;
    f.chunk = L.cp.chunk;
    f.splits = L.cp.splits;
    f.mask_id = a->mask_token_id;
    f.parts = reinterpret_cast<ScanPart*>(ws + L.scan_off);
    f.n_sel = a->batch;
    f.n_q = L.qp.col_tiles;
    const long n_front = static_cast<long>(f.n_sel) + f.n_q + static_cast<long>(L.cp.splits) * a->block_len * a->batch;
    if (n_front > 0x7fffffffL) return POLESTAR_ERR_UNSUPPORTED;
    const bool ok = bf16 ? launch_front<true>(L.ipt, L.qp.mt, dim3(n_front), f, stream)
                         : launch_front<false>(L.ipt, L.qp.mt, dim3(n_front), f, stream);
    if (!ok) return POLESTAR_ERR_UNSUPPORTED;
    st = launch_status();
    if (st != POLESTAR_OK) return st;

    // 3. refresh (the caller's events bracket exactly this launch group)
    if (refresh_begin && hipEventRecord(refresh_begin, stream) != hipSuccess) return POLESTAR_ERR_LAUNCH;
    st = polestar_refresh_kv(a->dtype, a->batch, a->seq, a->d, a->n_kv_heads, a->head_dim, a->h_cur,
                             a->stale_idx, a->stale_count, a->k, a->block_start, a->block_len, a->w_k, a->w_v,
                             a->k_cache, a->v_cache, ws, L.refresh_bytes, stream);
    if (st != POLESTAR_OK) return st;
    if (refresh_end && hipEventRecord(refresh_end, stream) != hipSuccess) return POLESTAR_ERR_LAUNCH;

    // 4. attention
    const AttArgs att = att_args(L.ap, a->batch, a->seq, a->block_len, a->n_heads, a->n_kv_heads, a->head_dim,
                                 a->q, a->k_cache, a->v_cache, a->out, a->lse, a->scale,
                                 L.ap.splits > 1 ? ws + L.att_off : nullptr);
    if (bf16) launch_attention<true>(a->head_dim, L.ap, att, stream);
    else launch_attention<false>(a->head_dim, L.ap, att, stream);
    st = launch_status();
    if (st != POLESTAR_OK) return st;

    // 5. attention merge | commit finalize
    BackArgs k{};
    k.att = att;
    k.n_merge = L.ap.splits > 1 ? static_cast<int>(ceil_div(static_cast<long>(a->batch) * a->n_heads * a->block_len, 4)) : 0;
    k.parts = f.parts;
    k.splits = L.cp.splits;
    k.nq = a->block_len;
    k.masked = a->masked;
    k.drift = a->drift;
    k.seq = a->seq;
    k.block_start = a->block_start;
    const bool use_hist = a->h > 0;
    k.hist = use_hist ? a->hist : nullptr;
    k.hist_len = use_hist ? a->hist_len : nullptr;
    k.h = use_hist ? a->h : 0;
    k.tau_s = a->tau_s;
    k.alpha = a->alpha;
    k.force_one = a->force_one;
    k.token = a->token;
    k.conf = a->conf;
    k.commit = a->commit;
    const dim3 gb(k.n_merge + a->batch);
    if (bf16) launch_back<true>(a->head_dim, gb, k, stream);
    else launch_back<false>(a->head_dim, gb, k, stream);
    return launch_status();
}
