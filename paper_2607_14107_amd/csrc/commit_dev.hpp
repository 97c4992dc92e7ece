// Device side of polestar_commit (Sec. 4.2, Alg. 1; confidence of Sec. 2 and
// eq. 1), shared by the stand-alone kernels and the fused step kernels.
//
// The vocabulary scan is an HBM-bound stream: workgroup (split, j, b)
// reduces one slice of the vocabulary of token (b, j) to
//   (m, s, best value, best id):  m = max_v l_v,  s = sum_v exp(l_v - m),
//   best = argmax over v != mask id (lowest id on ties)
// with 16-byte loads, per-lane running values and wavefront shuffles.
// The finalize step (one workgroup per sequence, one thread per block
// position) merges the slices in order, forms conf = exp(best - m) / s,
// applies the fp32 commit rule with the operation order of the header (no
// contraction), the force-one fallback and the history push.
#pragma once

#include "common.hpp"
#include "host_common.hpp"

namespace ps {
namespace {

constexpr int kScanBlock = 256;
constexpr int kScanInFlight = 8;   // 16-byte chunks per lane kept in flight by scan_body
constexpr int kMaxSplits = 16;    // vocabulary slices per token
constexpr int kMaxHist = 16;      // drift history depth h

struct ScanPart {
    float m;
    float s;
    float best;
    int idx;
};

// Argmax step: (v, i) replaces (bv, bi) if larger, or equal with a lower id.
// Written as selects so that it compiles to straight-line code.
__device__ __forceinline__ void better(float& bv, int& bi, float v, int i, bool valid = true) {
    const bool take = valid & ((v > bv) | ((v == bv) & (i < bi)));   // no short-circuit: no branches
    bv = take ? v : bv;
    bi = take ? i : bi;
}

// (m, s) <- merge with (m2, s2), s = sum exp(l - m); all -inf stays (-inf, 0).
__device__ __forceinline__ void merge_ms(float& m, float& s, float m2, float s2) {
    const float mn = fmaxf(m, m2);
    const float mref = mn == -INFINITY ? 0.f : mn;
    s = s * fast_exp2((m - mref) * kLog2e) + s2 * fast_exp2((m2 - mref) * kLog2e);
    m = mn;
}

// Slice `split` of the vocabulary of token (b, j), one 256-thread workgroup.
template <bool BF16>
__device__ __forceinline__ void scan_body(const char* __restrict__ logits, int vocab, int nq,
                                          int chunk, int splits, int mask_id,
                                          ScanPart* __restrict__ parts, int split, int j, int b) {
    using T = Elem<BF16>;
    constexpr int ES = T::kBytes;
    constexpr int G = kScanInFlight;
    __shared__ float sm[4], ss[4], sb[4];
    __shared__ int si[4];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const size_t tok = static_cast<size_t>(b) * nq + j;
    const int v0 = split * chunk;
    const int v1 = min(vocab, v0 + chunk);
    const char* row = logits + tok * vocab * ES;

    float m = -INFINITY, s = 0.f, bv = -INFINITY;
    int bi = 0x7fffffff;
    // Elements [v0, v1) in 16-byte chunks; chunk c starts at element v0 + c*E.
    // Straight-line loads: chunks past the slice re-read chunk 0 and count as
    // -inf (no exp contribution, never the argmax); the mask id takes part in
    // the softmax but not in the argmax.  A thread visits its elements in
    // increasing id order, so the lowest id of the largest value is the first
    // element equal to the largest chunk maximum in the first chunk that
    // reaches it.  Each round therefore keeps only that chunk (its maximum
    // over ids other than the mask id, and its data, by selects) and searches
    // it once at the end of the round; an element-wise search of every chunk
    // that might hold a new best ran for almost every chunk, since some lane
    // of the wave nearly always needed it.
    const int nchunks = (v1 - v0) / T::E;
    for (int c0 = 0; c0 < nchunks; c0 += kScanBlock * G) {
        uint4 r[G];
        bool ok[G];
#pragma unroll
        for (int gq = 0; gq < G; ++gq) {
            const int c = c0 + gq * kScanBlock + threadIdx.x;
            ok[gq] = c < nchunks;
            r[gq] = ld16_nt(row + static_cast<size_t>(v0 + (ok[gq] ? c : 0) * T::E) * ES);   // read once
        }
        __builtin_amdgcn_sched_barrier(0);   // all G loads in flight before any use
        float lm = -INFINITY;
        // the round's candidate chunk: maximum rbv (mask id excluded), data rdat, first id rvb
        float rbv = -INFINITY;
        bool rhave = false;
        uint4 rdat = r[0];
        int rvb = 0;
#pragma unroll
        for (int gq = 0; gq < G; ++gq) {
            float f[T::E];
            T::unpack(r[gq], f);
            float cm = f[0];
#pragma unroll
            for (int e = 1; e < T::E; ++e) cm = fmaxf(cm, f[e]);
            lm = fmaxf(lm, ok[gq] ? cm : -INFINITY);
            const int vb = v0 + (c0 + gq * kScanBlock + threadIdx.x) * T::E;
            float ca = cm;
            if (__builtin_expect(static_cast<unsigned>(mask_id - vb) < static_cast<unsigned>(T::E), 0)) {
                ca = -INFINITY;
#pragma unroll
                for (int e = 0; e < T::E; ++e) ca = vb + e != mask_id ? fmaxf(ca, f[e]) : ca;
            }
            // a later chunk replaces the candidate only with a strictly larger
            // maximum; the first valid chunk is taken even at -inf (a NaN
            // maximum, from a chunk of NaNs, never is)
            const bool take = ok[gq] & ((ca > rbv) | (!rhave & (ca == ca)));
            rbv = take ? ca : rbv;
            rdat.x = take ? r[gq].x : rdat.x;
            rdat.y = take ? r[gq].y : rdat.y;
            rdat.z = take ? r[gq].z : rdat.z;
            rdat.w = take ? r[gq].w : rdat.w;
            rvb = take ? vb : rvb;
            rhave |= take;
        }
        if (rhave) {
            // the candidate's first element equal to its maximum (mask id
            // excluded), merged into the running best: earlier rounds hold
            // lower ids, so on a tie the running best stays
            float f[T::E];
            T::unpack(rdat, f);
            int ie = -1;
            float fv = rbv;
#pragma unroll
            for (int e = T::E - 1; e >= 0; --e) {
                const bool hit = (f[e] == rbv) & (rvb + e != mask_id);
                ie = hit ? e : ie;
                fv = hit ? f[e] : fv;
            }
            if (ie >= 0) better(bv, bi, fv, rvb + ie);
        }
        // The exponentials unpack the chunks again: keeping every chunk's
        // floats live from the first pass took 123 registers against 65 (the
        // fused launch that runs this beside the drift takes the larger count).
#pragma unroll
        for (int gq = 0; gq < G; ++gq) asm volatile("" : "+v"(r[gq].x), "+v"(r[gq].y), "+v"(r[gq].z), "+v"(r[gq].w));
        const float mn = fmaxf(m, lm);
        const float mref = mn == -INFINITY ? 0.f : mn;
        const float mnl = mref * kLog2e;
        float ls = 0.f;
#pragma unroll
        for (int gq = 0; gq < G; ++gq) {
            float f[T::E];
            T::unpack(r[gq], f);
            float cs = 0.f;
#pragma unroll
            for (int e = 0; e < T::E; ++e) cs += fast_exp2(fmaf(f[e], kLog2e, -mnl));
            ls += ok[gq] ? cs : 0.f;
        }
        s = s * fast_exp2((m - mref) * kLog2e) + ls;
        m = mn;
    }
    // wavefront reduction
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const float m2 = __shfl_xor(m, o), s2 = __shfl_xor(s, o);
        const float b2 = __shfl_xor(bv, o);
        const int i2 = __shfl_xor(bi, o);
        merge_ms(m, s, m2, s2);
        better(bv, bi, b2, i2);
    }
    if (lane == 0) {
        sm[w] = m; ss[w] = s; sb[w] = bv; si[w] = bi;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int q = 1; q < 4; ++q) {
            merge_ms(m, s, sm[q], ss[q]);
            better(bv, bi, sb[q], si[q]);
        }
        parts[tok * splits + split] = ScanPart{m, s, bv, bi};
    }
}

// The fp32 rule, written without contraction so that the operation order is
// the documented one.
#pragma clang fp contract(off)
__device__ bool commit_rule(float c, float dlt, bool use_drift, const float* hv, int n, float tau_s,
                            float alpha) {
    if (c > tau_s) return true;
    if (!use_drift) return false;
    float mu = 0.f;
    if (n > 0) {
        float s = 0.f;
#pragma unroll
        for (int r = 0; r < kMaxHist; ++r)
            if (r < n) s = s + hv[r];
        mu = s / static_cast<float>(n);
    }
    const float D = dlt - mu;
    const float t = tau_s - c;
    const float tau_d = (alpha * t) * t;
    return D > tau_d;
}
#pragma clang fp contract(on)

// Sequence b: one thread per block position j (blockDim.x >= nq).  `eligible`
// (nullable) further restricts the positions that may commit.
__device__ __forceinline__ void finalize_body(const ScanPart* __restrict__ parts, int splits, int nq,
                                              const uint8_t* __restrict__ masked,
                                              const uint8_t* __restrict__ eligible,
                                              const float* __restrict__ drift, int seq,
                                              int block_start, float* hist, int32_t* hist_len, int h,
                                              float tau_s, float alpha, int force_one,
                                              int32_t* __restrict__ token, float* __restrict__ conf,
                                              uint8_t* __restrict__ commit, int b) {
    __shared__ int any_commit;
    __shared__ unsigned long long best_key;
    const int j = threadIdx.x;
    const bool inb = j < nq;
    const int jc = inb ? j : 0;
    const size_t tok = static_cast<size_t>(b) * nq + jc;

    // Every load of this thread is issued up front (one memory round trip):
    // the slice partials, the mask, the drift and the history column.
    ScanPart pv[kMaxSplits];
#pragma unroll
    for (int q = 0; q < kMaxSplits; ++q) pv[q] = parts[tok * splits + (q < splits ? q : 0)];
    const int n = (h > 0 && hist_len) ? min(max(hist_len[b], 0), h) : 0;
    // a position may commit only if it is masked (and eligible, when a mask is given)
    const bool is_masked = (masked[tok] != 0) & (eligible == nullptr || eligible[tok] != 0);
    const float dlt = drift ? drift[static_cast<size_t>(b) * seq + block_start + jc] : 0.f;
    float hv[kMaxHist];
    float* hcol = hist ? hist + static_cast<size_t>(b) * h * nq + jc : nullptr;
#pragma unroll
    for (int r = 0; r < kMaxHist; ++r) hv[r] = (hcol && r < h) ? hcol[r * nq] : 0.f;

    if (j == 0) {
        any_commit = 0;
        best_key = 0ull;
    }
    float m = pv[0].m, ssum = pv[0].s, bv = pv[0].best;
    int bi = pv[0].idx;
#pragma unroll
    for (int q = 1; q < kMaxSplits; ++q) {
        if (q < splits) {
            merge_ms(m, ssum, pv[q].m, pv[q].s);
            better(bv, bi, pv[q].best, pv[q].idx);
        }
    }
    const float c = fast_exp2((bv - m) * kLog2e) / ssum;
    bool cm = inb && is_masked && commit_rule(c, dlt, drift != nullptr, hv, n, tau_s, alpha);
    __syncthreads();                        // any_commit / best_key initialised
    if (cm) atomicOr(&any_commit, 1);
    __syncthreads();
    if (force_one && !any_commit && inb && is_masked) {
        // largest confidence, then lowest position: key = (conf bits, ~j)
        const unsigned long long key =
            (static_cast<unsigned long long>(__float_as_uint(c)) << 32) | (0xffffffffu - j);
        atomicMax(&best_key, key);
    }
    __syncthreads();
    if (force_one && !any_commit && inb && is_masked && best_key != 0ull &&
        static_cast<int>(0xffffffffu - static_cast<uint32_t>(best_key & 0xffffffffull)) == j)
        cm = true;
    if (inb) {
        token[tok] = bi;
        conf[tok] = c;
        commit[tok] = cm ? 1 : 0;
        // history push (all block positions), entries oldest first
        if (h > 0 && drift && hist) {
            if (n < h) {
                hcol[n * nq] = dlt;
            } else {
#pragma unroll
                for (int r = 0; r + 1 < kMaxHist; ++r)
                    if (r + 1 < h) hcol[r * nq] = hv[r + 1];
                hcol[(h - 1) * nq] = dlt;
            }
        }
    }
    if (j == 0 && h > 0 && drift && hist_len) hist_len[b] = min(n + 1, h);
}

struct CommitPlan {
    int splits;
    int chunk;
    size_t ws_bytes;
};

inline CommitPlan commit_plan(bool bf16, int batch, int nq, int vocab) {
    CommitPlan p{};
    const int e = bf16 ? 8 : 4;
    const long toks = static_cast<long>(batch) * nq;
    int splits = static_cast<int>((2048 + toks - 1) / toks);   // ~2048 workgroups: several resident per CU
    // and no slice longer than one round of loads (kScanInFlight chunks per
    // thread): a vocabulary of 152064 in 8 slices took a second, mostly
    // empty, round per workgroup (25.4 us for 78 MB)
    const int one_round = kScanBlock * kScanInFlight * e;
    if (splits < ceil_div(vocab, one_round)) splits = ceil_div(vocab, one_round);
    const int max_splits = ceil_div(vocab, 2048);
    if (splits > max_splits) splits = max_splits;
    if (splits > kMaxSplits) splits = kMaxSplits;
    if (splits < 1) splits = 1;
    p.chunk = ceil_div(ceil_div(vocab, splits), e) * e;
    p.splits = ceil_div(vocab, p.chunk);
    p.ws_bytes = static_cast<size_t>(toks) * p.splits * sizeof(ScanPart);
    return p;
}

}  // namespace
}  // namespace ps
