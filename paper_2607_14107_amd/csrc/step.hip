// polestar_step: one whole layer step (drift -> select -> K/V refresh -> Q
// projection -> attention -> commit) on one stream, with the work that does
// not depend on the previous launch fused into shared launches:
//
//   1. lead: drift | vocabulary scan   (both read only the step's inputs)
//   2. front: select | Q projection
//      The select of a sequence is one latency-bound workgroup; the Q
//      projection (split-K partials when the plan splits K) reads only the
//      inputs, so it fills the GPU while select runs.
//   3. refresh GEMM: gather -> MFMA -> split-K partials (needs 2)
//   4. reduce: refresh split-K reduce + scatter | Q split-K reduce
//      (an unsplit refresh on the tile kernel takes the Q reduce into its
//      own launch instead: five launches)
//   5. attention over the refreshed cache (needs 2, 3, 4)
//   6. back: attention merge | commit finalize (needs 5, and 1-2)
//
// Six launches instead of eleven kernels on their own.  Workgroups of a
// fused launch take their role from their block index; each role is the
// device body the stand-alone kernel runs, so results are bit-identical to
// calling the six entry points in order.  With more than 2048 positions, or
// a Q projection other than one DMA row tile of up to 64 rows or two of 128
// whose grid and select's workgroups overflow one round by at most 16,
// select and the Q projection run as two launches of their own (seven in
// all); shapes
// outside the other fused kernels
// (blocks longer than 256, head_dim other than 64/128, rows above the
// drift kernel's) run exactly the sequence of entry points instead.
#include "attend_dev.hpp"
#include "commit_dev.hpp"
#include "drift_dev.hpp"
#include "gemm_dev.hpp"
#include "host_common.hpp"
#include "select_dev.hpp"

namespace ps {
namespace {

constexpr int kStepBlock = 256;
constexpr long kCus = 256;   // compute units of MI355X: one round of one workgroup each
static_assert(kSelBlock == kStepBlock && kSmallBlock == kStepBlock && kScanBlock == kStepBlock &&
                  kAttBlock == kStepBlock && kDriftBlock == kStepBlock && kGemmBlock == kStepBlock,
              "fused roles share one workgroup size");

struct LeadArgs {
    // drift
    const char* hc;
    const char* hp;
    float* drift;
    int rows, d;
    // vocabulary scan
    const char* logits;
    int vocab, nq, chunk, splits, mask_id;
    ScanPart* parts;
    int n_drift;   // workgroups of the drift role, first in launch order
};

template <bool BF16, int TPR, int NCH>
__global__ __launch_bounds__(kStepBlock) void lead_kernel(LeadArgs l) {
    const int vb = blockIdx.x;
    if (vb < l.n_drift) {
        drift_body<BF16, TPR, NCH>(l.hc, l.hp, l.drift, l.rows, l.d, vb);
        return;
    }
    const int r = vb - l.n_drift;
    const int split = r % l.splits;
    const int tok = r / l.splits;
    scan_body<BF16>(l.logits, l.vocab, l.nq, l.chunk, l.splits, l.mask_id, l.parts, split, tok % l.nq,
                    tok / l.nq);
}

struct FrontArgs {
    // select
    const float* drift;
    const uint8_t* elig;
    int seq, bs, bl, k;
    int32_t* idx;
    int32_t* cnt;
    // Q projection (block rows, at most 64 of them)
    GemmArgs q;
    int n_sel;     // workgroups of the select role, first in launch order
};

// select | Q projection on the small-M kernel (no partials)
template <bool BF16, int IPT, int MT>
__global__ __launch_bounds__(kStepBlock) void front_kernel(FrontArgs f) {
    const int vb = blockIdx.x;
    if (vb < f.n_sel) {
        select_body<IPT>(f.drift, f.elig, f.seq, f.bs, f.bl, f.k, f.idx, f.cnt, vb);
        return;
    }
    small_body<BF16, MT>(f.q, vb - f.n_sel, 0);
}

// select | Q projection on the DMA-staged kernel (bf16; split-K partials
// reduced in launch 4).  With three LDS slots two workgroups of up to four
// 16-row tiles fit per compute unit, so the select workgroups do not push the
// Q projection's one-per-CU grid into a second round; the 256-row block
// projections (two row tiles of eight) run one workgroup per CU and are fused
// only when the whole grid fits one round.  NTW: one row tile, so the weight
// stream is non-temporal.
template <int IPT, int MT, int NST, bool NTW>
__global__ __launch_bounds__(kStepBlock) void front_dma_kernel(FrontArgs f) {
    const int vb = blockIdx.x;
    if (vb < f.n_sel) {
        select_body<IPT>(f.drift, f.elig, f.seq, f.bs, f.bl, f.k, f.idx, f.cnt, vb);
        return;
    }
    dma_body<true, MT, NST, 3, NTW>(f.q, vb - f.n_sel);
}

struct ReduceArgs {
    GemmArgs r;    // refresh (n_r workgroups, first)
    GemmArgs q;    // Q projection
    int n_r;
};

// refresh on the tile kernel, unsplit | Q split-K reduce: the tile
// workgroups come first (tile_body's XCD-aware order counts from id 0), the
// reduction's after them, on compute units the tiles leave free or as a short
// tail, so the Q reduce needs no launch of its own (bf16 only, as the tile
// kernel).
struct TileQArgs {
    GemmArgs r;    // refresh (n_tile workgroups, first)
    GemmArgs q;    // Q projection
    int n_tile;
};

static_assert(kTileThreads == kGemmBlock, "the tile and reduce roles share one workgroup size");

template <int MI, int NJ>
__global__ __launch_bounds__(kTileThreads) void tile_qred_kernel(TileQArgs k) {
    if (static_cast<int>(blockIdx.x) < k.n_tile) {
        tile_body<MI, NJ>(k.r, blockIdx.x);
        return;
    }
    reduce_body<true>(k.q, blockIdx.x - k.n_tile);
}

template <bool BF16>
__global__ __launch_bounds__(kStepBlock) void reduce2_kernel(ReduceArgs k) {
    if (static_cast<int>(blockIdx.x) < k.n_r) {
        reduce_body<BF16>(k.r, blockIdx.x);
        return;
    }
    reduce_body<BF16>(k.q, blockIdx.x - k.n_r);
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

template <bool BF16, int TPR, int NCH>
void launch_lead1(dim3 grid, const LeadArgs& l, hipStream_t s) {
    hipLaunchKernelGGL((lead_kernel<BF16, TPR, NCH>), grid, dim3(kStepBlock), 0, s, l);
}

template <bool BF16>
bool launch_lead(int tpr, int nch, dim3 grid, const LeadArgs& l, hipStream_t s) {
    switch (tpr * 16 + nch) {
#define PS_CASE(TPR, NCH) \
        case TPR * 16 + NCH: launch_lead1<BF16, TPR, NCH>(grid, l, s); return true;
        PS_DRIFT_SHAPES(PS_CASE)
#undef PS_CASE
        default: return false;
    }
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

// one row tile of 2..4 16-row tiles (NST 8 or 16, non-temporal weights), or
// two row tiles of 8 (NST 8, 14 or 16)
template <int IPT, int NST>
bool launch_front_dma_mt(int mt, dim3 grid, const FrontArgs& f, hipStream_t s) {
    switch (mt) {
        case 2: hipLaunchKernelGGL((front_dma_kernel<IPT, 2, NST, true>), grid, dim3(kStepBlock), 0, s, f); return true;
        case 3: hipLaunchKernelGGL((front_dma_kernel<IPT, 3, NST, true>), grid, dim3(kStepBlock), 0, s, f); return true;
        case 4: hipLaunchKernelGGL((front_dma_kernel<IPT, 4, NST, true>), grid, dim3(kStepBlock), 0, s, f); return true;
        case 8: hipLaunchKernelGGL((front_dma_kernel<IPT, 8, NST, false>), grid, dim3(kStepBlock), 0, s, f); return true;
        default: return false;
    }
}

template <int IPT>
bool launch_front_dma_nst(int nst, int mt, dim3 grid, const FrontArgs& f, hipStream_t s) {
    if (nst == 8) return launch_front_dma_mt<IPT, 8>(mt, grid, f, s);
    if (nst == 16) return launch_front_dma_mt<IPT, 16>(mt, grid, f, s);
    if (nst == 14 && mt == 8) {
        hipLaunchKernelGGL((front_dma_kernel<IPT, 8, 14, false>), grid, dim3(kStepBlock), 0, s, f);
        return true;
    }
    return false;
}

// dma: the Q plan takes the DMA kernel (bf16), nst its 128-byte stages per split
template <bool BF16>
bool launch_front(int ipt, bool dma, int nst, int mt, dim3 grid, const FrontArgs& f, hipStream_t s) {
    if (dma) {
        if constexpr (!BF16) return false;
        switch (ipt) {
            case 1: return launch_front_dma_nst<1>(nst, mt, grid, f, s);
            case 2: return launch_front_dma_nst<2>(nst, mt, grid, f, s);
            case 3: return launch_front_dma_nst<3>(nst, mt, grid, f, s);
            case 4: return launch_front_dma_nst<4>(nst, mt, grid, f, s);
            case 6: return launch_front_dma_nst<6>(nst, mt, grid, f, s);
            case 8: return launch_front_dma_nst<8>(nst, mt, grid, f, s);
            default: return false;
        }
    }
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

// Workspace of the step: refresh partials, attention partials, scan
// partials, Q-projection partials, each 256-byte aligned.
struct StepLayout {
    GemmPlan qp;        // Q projection plan
    GemmPlan rp;        // refresh plan
    AttPlan ap;
    CommitPlan cp;
    size_t refresh_bytes, att_off, scan_off, q_off, total;
    bool fused;         // all six launches fused (select | Q projection in one)
    bool semi;          // the same launches with select and the Q projection as their own
    int ipt;
    int drift_tpr, drift_nch;
};

StepLayout step_layout(const polestar_step_args& a) {
    StepLayout L{};
    const bool bf16 = a.dtype == POLESTAR_BF16;
    L.refresh_bytes = polestar_refresh_kv_workspace_size(a.dtype, a.batch, a.d, a.n_kv_heads, a.head_dim, a.k,
                                                         a.block_len);
    L.qp = gemm_plan(bf16, static_cast<long>(a.batch) * a.block_len, a.n_heads * a.head_dim, a.d);
    L.rp = gemm_plan(bf16, static_cast<long>(a.batch) * (a.k + a.block_len), 2 * a.n_kv_heads * a.head_dim, a.d);
    L.ap = att_plan(bf16, a.batch, a.seq, a.n_heads, a.n_kv_heads, a.block_len, a.head_dim);
    L.cp = commit_plan(bf16, a.batch, a.block_len, a.vocab);
    L.ipt = select_ipt(a.seq);
    const int qnst = 2 * L.qp.steps_per_split;
    const bool q_dma1 = bf16 && L.qp.dma && L.qp.row_tiles == 1 && L.qp.mt >= 2 && L.qp.mt <= 4 &&
                        (qnst == 8 || qnst == 16);
    // the 256-row block projections (two row tiles of eight 16-row tiles):
    // one workgroup per CU, so fused when select's workgroups and the
    // projection's fit one round, or overflow it by at most 16: the select
    // workgroups go first and are short, so the projection's last few start
    // when they end (batch-8 LLaDA-8B layer, 256 + 8 workgroups: 202-380 us
    // per step against 207-385 us with select launched on its own)
    const bool q_dma2 = bf16 && L.qp.dma && L.qp.row_tiles == 2 && L.qp.mt == 8 &&
                        (qnst == 8 || qnst == 14 || qnst == 16) &&
                        static_cast<long>(L.qp.grid) + a.batch <= kCus + 16;
    const bool q_dma = q_dma1 || q_dma2;
    const bool drift_ok = drift_config(a.d / (bf16 ? 8 : 4), static_cast<long>(a.batch) * a.seq, L.drift_tpr,
                                       L.drift_nch);
    const bool common = drift_ok && a.block_len <= kStepBlock && (a.head_dim == 64 || a.head_dim == 128);
    L.fused = common && L.ipt >= 1 && L.ipt <= 8 && (L.qp.small || q_dma);
    // more query rows than the front kernel takes (or a longer sequence):
    // select and the Q projection run as their own launches, the rest fused
    L.semi = !L.fused && common && L.ipt >= 1;
    L.att_off = align_up(L.refresh_bytes, 256);
    L.scan_off = L.att_off + align_up(L.ap.part_bytes, 256);
    L.q_off = L.scan_off + align_up(L.cp.ws_bytes, 256);   // Q projection partials (when its plan splits K)
    L.total = L.q_off + align_up(L.qp.ws_bytes, 256);
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
    st = polestar_project_q(a.dtype, a.batch, a.seq, a.d, a.n_heads, a.head_dim, a.block_start, a.block_len,
                            a.h_cur, a.w_q, a.q, L.qp.ws_bytes ? ws + L.q_off : nullptr, L.qp.ws_bytes, s);
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
    if (!L.fused && !L.semi) return run_unfused(*a, L, ws, refresh_begin, refresh_end, stream);

    const bool bf16 = a->dtype == POLESTAR_BF16;
    // Every check of the fused launches' stand-alone entry points, before
    // anything is enqueued.
    if (!row_ok(a->dtype, a->d) || !aligned16(a->h_cur) || !aligned16(a->h_prev) || !aligned16(a->drift) ||
        !gemm_k_ok(bf16, a->d) || !aligned16(a->w_q) || !aligned16(a->w_k) || !aligned16(a->w_v) ||
        !aligned16(a->q) || !aligned16(a->k_cache) || !aligned16(a->v_cache) || !aligned16(a->out) ||
        !aligned16(workspace) || !row_ok(a->dtype, a->vocab) || !aligned16(a->logits) || a->h > kMaxHist ||
        a->batch > 65535 || static_cast<long>(a->n_heads) * ceil_div(a->block_len, kQG) > 65535)
        return POLESTAR_ERR_UNSUPPORTED;

    // 1. drift | vocabulary scan
    LeadArgs l{};
    l.hc = static_cast<const char*>(a->h_cur);
    l.hp = static_cast<const char*>(a->h_prev);
    l.drift = a->drift;
    l.rows = a->batch * a->seq;
    l.d = a->d;
    l.logits = static_cast<const char*>(a->logits);
    l.vocab = a->vocab;
    l.nq = a->block_len;
    l.chunk = L.cp.chunk;
    l.splits = L.cp.splits;
    l.mask_id = a->mask_token_id;
    l.parts = reinterpret_cast<ScanPart*>(ws + L.scan_off);
    l.n_drift = ceil_div(l.rows, kDriftBlock / L.drift_tpr);
    const long n_lead = static_cast<long>(l.n_drift) + static_cast<long>(L.cp.splits) * a->block_len * a->batch;
    if (n_lead > 0x7fffffffL) return POLESTAR_ERR_UNSUPPORTED;
    const bool lok = bf16 ? launch_lead<true>(L.drift_tpr, L.drift_nch, dim3(n_lead), l, stream)
                          : launch_lead<false>(L.drift_tpr, L.drift_nch, dim3(n_lead), l, stream);
    if (!lok) return POLESTAR_ERR_UNSUPPORTED;
    polestar_status st = launch_status();
    if (st != POLESTAR_OK) return st;

    // 2. select | Q projection
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
    f.q.ws = reinterpret_cast<float*>(ws + L.q_off);
    gemm_finalize_args(L.qp, f.q);
    f.n_sel = a->batch;
    if (L.fused) {
        const int n_q = L.qp.small ? L.qp.col_tiles : L.qp.grid;
        const bool ok = bf16 ? launch_front<true>(L.ipt, !L.qp.small, 2 * L.qp.steps_per_split, L.qp.mt,
                                                  dim3(f.n_sel + n_q), f, stream)
                             : launch_front<false>(L.ipt, !L.qp.small, 2 * L.qp.steps_per_split, L.qp.mt,
                                                   dim3(f.n_sel + n_q), f, stream);
        if (!ok) return POLESTAR_ERR_UNSUPPORTED;
        st = launch_status();
    } else {
        // the same two pieces as separate launches; the Q projection's split-K
        // reduction still joins the refresh's in launch 4
        st = polestar_select(a->batch, a->seq, a->drift, a->eligible, a->block_start, a->block_len, a->k,
                             a->stale_idx, a->stale_count, stream);
        if (st != POLESTAR_OK) return st;
        GemmArgs qdef{};
        st = gemm_run(bf16, L.qp, f.q, stream, &qdef);
    }
    if (st != POLESTAR_OK) return st;

    // 3. refresh GEMM, 4. refresh reduce | Q reduce (the caller's events
    // bracket exactly these two launches)
    if (refresh_begin && hipEventRecord(refresh_begin, stream) != hipSuccess) return POLESTAR_ERR_LAUNCH;
    ReduceArgs rk{};
    GemmArgs rg = refresh_gemm_args(a->batch, a->seq, a->d, a->n_kv_heads * a->head_dim, a->h_cur, a->stale_idx,
                                    a->stale_count, a->k, a->block_start, a->block_len, a->w_k, a->w_v,
                                    a->k_cache, a->v_cache, ws);
    const int n_qred = gemm_reduce_blocks(L.qp, f.q);
    if (bf16 && L.rp.tile && L.rp.ksplit == 1 && L.rp.steps_per_split % 4 == 0 && n_qred > 0) {
        TileQArgs tq{};
        gemm_finalize_args(L.rp, rg);
        tq.r = rg;
        tq.q = f.q;
        tq.n_tile = L.rp.grid;
        const dim3 grid(L.rp.grid + n_qred), block(kTileThreads);
        switch (10 * L.rp.tile_mi + L.rp.tile_nj) {
            case 44: hipLaunchKernelGGL((tile_qred_kernel<4, 4>), grid, block, 0, stream, tq); break;
            case 43: hipLaunchKernelGGL((tile_qred_kernel<4, 3>), grid, block, 0, stream, tq); break;
            case 34: hipLaunchKernelGGL((tile_qred_kernel<3, 4>), grid, block, 0, stream, tq); break;
            case 33: hipLaunchKernelGGL((tile_qred_kernel<3, 3>), grid, block, 0, stream, tq); break;
            default: return POLESTAR_ERR_UNSUPPORTED;
        }
        st = launch_status();
        if (st != POLESTAR_OK) return st;
    } else {
        st = gemm_run(bf16, L.rp, rg, stream, &rk.r);
        if (st != POLESTAR_OK) return st;
        gemm_finalize_args(L.rp, rg);
        rk.n_r = gemm_reduce_blocks(L.rp, rg);
        rk.q = f.q;
        const int n_red = rk.n_r + n_qred;
        if (n_red > 0) {
            if (bf16) hipLaunchKernelGGL(reduce2_kernel<true>, dim3(n_red), dim3(kStepBlock), 0, stream, rk);
            else hipLaunchKernelGGL(reduce2_kernel<false>, dim3(n_red), dim3(kStepBlock), 0, stream, rk);
            st = launch_status();
            if (st != POLESTAR_OK) return st;
        }
    }
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
    k.parts = l.parts;
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
