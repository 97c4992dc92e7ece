"""CPU oracle for one cached denoising step of Polestar (arxiv 2607.14107).

TEST INFRASTRUCTURE ONLY.  This module is the slow, plain reference that the
HIP path is checked against.  Only the test suite, the smoke check of the
package entry file and the `cpu_baseline` leg of the benchmark may import it;
the product path never does.  It shares no code with the HIP kernels or their
host code, and it never consumes a value produced by them.

Everything is float64 NumPy written for readability, not speed: dense
contractions use NumPy's matmul, everything else is plain NumPy following the
paper's definitions step by step.  Inputs arrive as float64 arrays already
decoded from the bytes the GPU receives (see `decode`).

Step order of one layer step (the data-parallel hot path):
  1. drift       -- token representation drift, eq. (drift), Sec. 3
  2. select      -- TopK of drift over cached positions, Alg. 1 (TopK step)
  3. refresh_kv  -- sparse K/V re-projection of the stale rows plus the
                    active block, Sec. 4.1 "Measuring Drift and Layer-wise KV
                    Updates" and Corollary 1 (App. B)
  4. attend      -- bidirectional attention of the active block over the
                    whole cache, eq. (3) and the setup of App. B
  5. commit      -- Polestar-Commit current-block rule, Sec. 4.2 and Alg. 1
                    (confidence, drift delta, dynamic threshold, commit)

Readings of passages that are ambiguous are written next to the code that
takes them.
"""

from __future__ import annotations

import numpy as np

# ---------------------------------------------------------------------------
# Dtype handling.  The GPU receives fp32 arrays or bf16 bit patterns; the
# oracle decodes them exactly into float64.  Rounding of float64 results to
# bf16 (round to nearest, ties to even) is done here from the definition of
# the format: 8 significant bits.
# ---------------------------------------------------------------------------


def decode(x: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 values of an fp32 array or of bf16 bit patterns (uint16)."""
    if dtype == "fp32":
        return np.asarray(x, dtype=np.float32).astype(np.float64)
    if dtype == "bf16":
        bits = np.asarray(x, dtype=np.uint16).astype(np.uint32) << 16
        return bits.view(np.float32).astype(np.float64)
    raise ValueError(dtype)


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """float64 -> nearest bf16 value (ties to even), returned as float64.

    A bf16 number has an 8-bit significand.  frexp gives x = m * 2**e with
    0.5 <= |m| < 1, so m * 2**8 is the significand scaled to an integer range
    and np.rint rounds it half-to-even.  Values here are O(1): the subnormal
    and overflow ranges are not reached.
    """
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)
    return np.ldexp(np.rint(m * 256.0), e - 8)


def round_to(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round float64 results to the stored dtype (as float64 values)."""
    if dtype == "fp32":
        return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)
    if dtype == "bf16":
        return round_to_bf16(x)
    raise ValueError(dtype)


# ---------------------------------------------------------------------------
# Step 1 -- drift.
#
# The paper measures a token's drift as KL(current || previous) of its
# distribution between two consecutive denoising steps (eq. drift, Sec. 3).
# Reading used on the hot path: the distribution of a token is the softmax of
# its layer-input hidden state over the d channels, so the drift is a
# per-token reduction between the current and previous hidden states.  KL is
# in nats, argument order current || previous.
# ---------------------------------------------------------------------------


def log_softmax(x: np.ndarray, axis: int = -1) -> np.ndarray:
    m = np.max(x, axis=axis, keepdims=True)
    z = x - m
    return z - np.log(np.sum(np.exp(z), axis=axis, keepdims=True))


def kl(logp: np.ndarray, logq: np.ndarray, axis: int = -1) -> np.ndarray:
    """KL(p || q) = sum_c p_c (log p_c - log q_c), from log-probabilities."""
    return np.sum(np.exp(logp) * (logp - logq), axis=axis)


def drift(h_cur: np.ndarray, h_prev: np.ndarray) -> np.ndarray:
    """D[b, i] = KL(softmax(h_cur[b, i]) || softmax(h_prev[b, i])).

    h_cur, h_prev: [batch][seq][d] float64.  Returns [batch][seq] float64.
    """
    return kl(log_softmax(h_cur), log_softmax(h_prev))


def attention_logits(h: np.ndarray, w_q: np.ndarray, w_k: np.ndarray,
                     n_heads: int, n_kv_heads: int, head_dim: int,
                     scale: float | None = None) -> np.ndarray:
    """Full-sequence attention logits l_ij = q_i . k_j / sqrt(d_h), per head.

    App. B setup: q = W_Q x, k = W_K x.  Returns [batch][heads][seq][seq].
    """
    b, s, _ = h.shape
    if scale is None:
        scale = 1.0 / np.sqrt(head_dim)
    q = (h @ w_q.T).reshape(b, s, n_heads, head_dim).transpose(0, 2, 1, 3)
    k = (h @ w_k.T).reshape(b, s, n_kv_heads, head_dim).transpose(0, 2, 1, 3)
    group = n_heads // n_kv_heads
    k = np.repeat(k, group, axis=1)
    return (q @ k.transpose(0, 1, 3, 2)) * scale


def drift_attention_exact(h_cur: np.ndarray, h_prev: np.ndarray,
                          w_q: np.ndarray, w_k: np.ndarray,
                          n_heads: int, n_kv_heads: int, head_dim: int) -> np.ndarray:
    """The paper's drift taken literally: KL of each token's attention
    distribution A_i^(t) || A_i^(t-1) (eq. drift), with both steps fully
    recomputed from their hidden states, per head and then averaged over heads
    (heads averaged as in the staleness metric of App. C.2).

    Used only for the fidelity report of the hot-path reading; O(S^2).
    """
    lc = log_softmax(attention_logits(h_cur, w_q, w_k, n_heads, n_kv_heads, head_dim))
    lp = log_softmax(attention_logits(h_prev, w_q, w_k, n_heads, n_kv_heads, head_dim))
    return kl(lc, lp).mean(axis=1)


def staleness(k_cached: np.ndarray, v_cached: np.ndarray,
              k_ref: np.ndarray, v_ref: np.ndarray) -> np.ndarray:
    """KV-cache staleness E_i (App. C.2): 1 - (cos(K, K_ref) + cos(V, V_ref)) / 2,
    cosine taken per head and averaged over heads.

    Arrays: [batch][seq][kv_heads][head_dim].  Returns [batch][seq].
    """
    def cos(a, b):
        num = np.sum(a * b, axis=-1)
        den = np.linalg.norm(a, axis=-1) * np.linalg.norm(b, axis=-1)
        return num / den
    return 1.0 - 0.5 * (cos(k_cached, k_ref).mean(axis=-1) + cos(v_cached, v_ref).mean(axis=-1))


# ---------------------------------------------------------------------------
# Step 2 -- select.
#
# Alg. 1 takes the TopK of the drift to find the positions whose cached K/V
# are refreshed.  Candidates are the cached positions I = J \ J_b (Sec. 2,
# block-wise KV caching): the active block is recomputed every step anyway.
# An optional eligibility mask narrows the candidates (the local window of
# Sec. 4.1).  Order: larger drift first, equal drift -> lower position first;
# the chosen set is returned sorted by ascending position, padded with -1.
# ---------------------------------------------------------------------------


def select(drift_vals: np.ndarray, k: int, block_start: int, block_len: int,
           eligible: np.ndarray | None = None):
    """Returns (stale_idx [batch][k] int32, stale_count [batch] int32)."""
    drift_vals = np.asarray(drift_vals, dtype=np.float64)
    batch, seq = drift_vals.shape
    idx = np.full((batch, k), -1, dtype=np.int32)
    cnt = np.zeros(batch, dtype=np.int32)
    for b in range(batch):
        cands = [i for i in range(seq)
                 if not (block_start <= i < block_start + block_len)
                 and (eligible is None or eligible[b, i])]
        # -0.0 and +0.0 compare equal, so they tie and fall back to the index.
        ranked = sorted(cands, key=lambda i: (-drift_vals[b, i], i))
        chosen = sorted(ranked[:k])
        cnt[b] = len(chosen)
        idx[b, :len(chosen)] = chosen
    return idx, cnt


# ---------------------------------------------------------------------------
# Step 3 -- sparse K/V refresh.
#
# Rows R = stale positions U J_b: the active block's K/V are computed every
# step (Sec. 2, block-wise KV caching) and the selected stale positions are
# re-projected from their current hidden states (Sec. 4.1).  For each r in R:
# K_r = W_K h_r and V_r = W_V h_r (App. B setup; Corollary 1 gives the change
# as W_K dH, W_V dH).  Rows outside R keep their cached values.
# Weights are [kv_heads*head_dim][d] (output x input), caches are
# [batch][seq][kv_heads][head_dim].
# ---------------------------------------------------------------------------


def refresh_rows(stale_idx: np.ndarray, stale_count: np.ndarray,
                 block_start: int, block_len: int) -> list[list[int]]:
    """The row set R of every sequence, ascending and without duplicates."""
    rows = []
    for b in range(stale_idx.shape[0]):
        r = set(int(i) for i in stale_idx[b, :int(stale_count[b])])
        r.update(range(block_start, block_start + block_len))
        rows.append(sorted(r))
    return rows


def refresh_kv(h_cur: np.ndarray, w_k: np.ndarray, w_v: np.ndarray,
               k_cache: np.ndarray, v_cache: np.ndarray,
               stale_idx: np.ndarray, stale_count: np.ndarray,
               block_start: int, block_len: int):
    """Returns (k_new, v_new, rows) in float64.  k_new/v_new equal the input
    caches outside the refreshed rows and hold the exact float64 projections
    on them (rounding to the stored dtype is the caller's choice)."""
    batch, seq, kvh, hd = k_cache.shape
    k_new = np.array(k_cache, dtype=np.float64, copy=True)
    v_new = np.array(v_cache, dtype=np.float64, copy=True)
    rows = refresh_rows(stale_idx, stale_count, block_start, block_len)
    for b in range(batch):
        r = np.asarray(rows[b], dtype=np.int64)
        if r.size == 0:
            continue
        x = h_cur[b, r, :]
        k_new[b, r] = (x @ w_k.T).reshape(r.size, kvh, hd)
        v_new[b, r] = (x @ w_v.T).reshape(r.size, kvh, hd)
    return k_new, v_new, rows


def project_rows(h: np.ndarray, w: np.ndarray, rows: np.ndarray) -> np.ndarray:
    """W h_r for a list of rows of one sequence (used for sampled checks)."""
    return h[np.asarray(rows, dtype=np.int64), :] @ w.T


# ---------------------------------------------------------------------------
# Step 4 -- attention of the active block over the whole cache.
#
# eq. (3): queries of J_b attend jointly to the cached K/V of I and the
# recomputed K/V of J_b; with the refreshed cache holding both, this is
# softmax attention over all seq slots, without a causal or padding mask
# (bidirectional dLLM attention).  Per head (App. B setup):
# l_ij = q_i . k_j / sqrt(d_h), a = softmax_j(l), o_i = sum_j a_ij v_j.
# Grouped-query attention: query head h reads KV head h // (heads / kv_heads),
# i.e. consecutive query heads share one KV head.
# ---------------------------------------------------------------------------


def q_project(h_cur: np.ndarray, w_q: np.ndarray, block_start: int, block_len: int,
              n_heads: int, head_dim: int) -> np.ndarray:
    """Q = W_Q h for the active-block rows -> [batch][block_len][heads][head_dim]."""
    x = h_cur[:, block_start:block_start + block_len, :]
    b = x.shape[0]
    return (x @ w_q.T).reshape(b, block_len, n_heads, head_dim)


def attend(q: np.ndarray, k_cache: np.ndarray, v_cache: np.ndarray,
           scale: float | None = None):
    """q: [batch][nq][heads][head_dim]; caches [batch][seq][kv_heads][head_dim].

    Returns (out [batch][nq][heads][head_dim], lse [batch][heads][nq]) where
    lse is the natural log of sum_j exp(l_ij).
    """
    batch, nq, heads, hd = q.shape
    kvh = k_cache.shape[2]
    group = heads // kvh
    if scale is None:
        scale = 1.0 / np.sqrt(hd)
    out = np.zeros((batch, nq, heads, hd))
    lse = np.zeros((batch, heads, nq))
    for b in range(batch):
        for h in range(heads):
            g = h // group
            logits = (q[b, :, h, :] @ k_cache[b, :, g, :].T) * scale   # [nq][seq]
            m = logits.max(axis=1, keepdims=True)
            e = np.exp(logits - m)
            z = e.sum(axis=1, keepdims=True)
            out[b, :, h, :] = (e / z) @ v_cache[b, :, g, :]
            lse[b, h, :] = (m + np.log(z))[:, 0]
    return out, lse


# ---------------------------------------------------------------------------
# Step 5 -- Polestar-Commit, current block.
#
# Confidence (Sec. 2): the provisional token is the argmax over the vocabulary
# without [MASK] (eq. 1); its confidence c is its softmax probability
# (max-probability confidence of the cited Fast-dLLM rule).  Readings: the
# softmax denominator runs over the whole vocabulary, [MASK] included; equal
# logits resolve to the lowest vocabulary id.
#
# Rule (Sec. 4.2 and Alg. 1): drift delta = delta_j - mean of the last h drift
# values (mean over the entries present; 0 when there are none), dynamic
# threshold tau_d = alpha (tau_s - c)^2, commit a masked token when c > tau_s
# or delta > tau_d (Alg. 1 uses strict comparisons), then push delta_j into
# the history and keep its last h entries.  When no masked token of a
# sequence qualifies and force_one is set, the masked token with the largest
# confidence (lowest position on ties) is committed so that the denoising
# loop always progresses.
#
# The decision is taken in fp32 with a fixed operation order, the same order
# the kernel uses, so that decisions are comparable bit for bit:
#   mu   = (((hist[0] + hist[1]) + ...) + hist[n-1]) / n
#   D    = delta - mu
#   t    = tau_s - c
#   tau  = (alpha * t) * t
#   commit = masked and (c > tau_s or D > tau)
# ---------------------------------------------------------------------------


def confidence(logits: np.ndarray, mask_token_id: int = -1):
    """logits [batch][nq][vocab] float64 -> (token int32, conf float64)."""
    batch, nq, vocab = logits.shape
    token = np.zeros((batch, nq), dtype=np.int32)
    conf = np.zeros((batch, nq))
    for b in range(batch):
        for j in range(nq):
            row = logits[b, j]
            cand = row.copy()
            if 0 <= mask_token_id < vocab:
                cand[mask_token_id] = -np.inf
            y = int(np.argmax(cand))          # first maximal index
            m = row.max()
            token[b, j] = y
            conf[b, j] = np.exp(row[y] - m) / np.sum(np.exp(row - m))
    return token, conf


def commit_rule(conf32: np.ndarray, delta32: np.ndarray, masked: np.ndarray,
                hist32: np.ndarray, hist_len: np.ndarray, h: int,
                tau_s: float, alpha: float, force_one: bool):
    """The commit decision of one step, in fp32.

    conf32, delta32: [batch][nq] float32; masked: [batch][nq] bool;
    hist32: [batch][h][nq] float32 with entries 0..hist_len-1 valid, oldest
    first.  Returns (commit bool [batch][nq], new_hist, new_len).
    """
    f = np.float32
    batch, nq = conf32.shape
    tau_s = f(tau_s)
    alpha = f(alpha)
    commit = np.zeros((batch, nq), dtype=bool)
    new_hist = np.array(hist32, dtype=np.float32, copy=True)
    new_len = np.array(hist_len, dtype=np.int32, copy=True)
    for b in range(batch):
        n = int(hist_len[b]) if h > 0 else 0
        for j in range(nq):
            if not masked[b, j]:
                continue
            c = f(conf32[b, j])
            mu = f(0.0)
            if n > 0:
                s = f(0.0)
                for r in range(n):
                    s = f(s + f(hist32[b, r, j]))
                mu = f(s / f(n))
            d = f(f(delta32[b, j]) - mu)
            t = f(tau_s - c)
            tau_d = f(f(alpha * t) * t)
            commit[b, j] = bool(c > tau_s) or bool(d > tau_d)
        if force_one and not commit[b].any() and masked[b].any():
            best = None
            for j in range(nq):
                if masked[b, j] and (best is None or f(conf32[b, j]) > f(conf32[b, best])):
                    best = j
            commit[b, best] = True
        if h > 0:
            if n < h:
                new_hist[b, n, :] = delta32[b]
                new_len[b] = n + 1
            else:
                new_hist[b, :h - 1, :] = hist32[b, 1:h, :]
                new_hist[b, h - 1, :] = delta32[b]
                new_len[b] = h
    return commit, new_hist, new_len


def suffix_eligible(stale_idx: np.ndarray, stale_count: np.ndarray, suffix_start: int,
                    suffix_len: int) -> np.ndarray:
    """Suffix positions carried by the final layer's update packet (Sec. 4.2,
    "Suffix Block Commit"; Alg. 1, the positions of the packet that fall in
    the next block J_(b+1)): [batch][suffix_len] bool, True where position
    suffix_start + r is among the first stale_count[b] entries of stale_idx[b]."""
    batch = stale_idx.shape[0]
    out = np.zeros((batch, suffix_len), dtype=bool)
    for b in range(batch):
        for r in range(int(stale_count[b])):
            p = int(stale_idx[b, r])
            if suffix_start <= p < suffix_start + suffix_len:
                out[b, p - suffix_start] = True
    return out


def suffix_commit_rule(conf32: np.ndarray, masked: np.ndarray, eligible: np.ndarray,
                       tau_s: float) -> np.ndarray:
    """Suffix-block commit (Sec. 4.2, "Suffix Block Commit"): a suffix position
    commits when it is still masked, the packet carries it (eligible) and its
    confidence exceeds tau_s; compared in fp32, strictly, as in Alg. 1."""
    f = np.float32
    c = np.asarray(conf32, dtype=np.float32)
    return np.asarray(masked, bool) & np.asarray(eligible, bool) & (c > f(tau_s))


# ---------------------------------------------------------------------------
# One whole layer step, for end-to-end checks.
# ---------------------------------------------------------------------------


def layer_step(h_cur, h_prev, w_q, w_k, w_v, k_cache, v_cache, *, k: int,
               block_start: int, block_len: int, n_heads: int, n_kv_heads: int,
               head_dim: int, cache_dtype: str, eligible=None):
    """drift -> select -> refresh (stored rounded to cache_dtype) -> attend."""
    d = drift(h_cur, h_prev)
    idx, cnt = select(d, k, block_start, block_len, eligible)
    k_new, v_new, rows = refresh_kv(h_cur, w_k, w_v, k_cache, v_cache, idx, cnt,
                                    block_start, block_len)
    k_st = round_to(k_new, cache_dtype)
    v_st = round_to(v_new, cache_dtype)
    q = q_project(h_cur, w_q, block_start, block_len, n_heads, head_dim)
    out, lse = attend(q, k_st, v_st)
    return dict(drift=d, stale_idx=idx, stale_count=cnt, rows=rows,
                k_exact=k_new, v_exact=v_new, k_cache=k_st, v_cache=v_st,
                q=q, out=out, lse=lse)
