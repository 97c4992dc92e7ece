"""CPU oracle for Polestar's own drift estimator: clustered proxy drift.

TEST INFRASTRUCTURE ONLY, like `polestar_ref`: the slow plain reference the
HIP path is checked against; only the tests, the package's smoke check and
the benchmark's `cpu_baseline` leg may use it, and it never consumes a value
produced by the HIP path.  float64 NumPy throughout.

What it computes (Sec. 4.1, "Cluster and Quantize Hidden States" and
"Measuring Drift and Layer-wise KV Updates"; Alg. 1, block entry and the
per-layer loop):
  at block entry
    1. spherical K-means of the hidden states of the local window
       -> a cluster label per window position, and per cluster the sum and
          count of its members' hidden states;
  at every step
    2. proxy tokens: one per cluster (the members' mean hidden state);
    3. proxy attention: the tokens projected to queries attend over all
       cached positions, one softmax distribution per (cluster, head);
    4. drift per cluster: KL(current distribution || previous one);
    5. the top-k clusters by drift; their member positions are the rows to
       refresh, in ascending order;
    6. after the refresh, the cluster sums move by the refreshed rows'
       change (labels stay fixed until the next block entry).

Readings where the paper leaves the detail open:
  P-1  Spherical K-means clusters the directions h/|h| (cosine similarity).
  P-2  Initialisation is deterministic: centroid j starts at the window point
       of rank floor(j*n/K).  A fixed number of iterations (default 10):
       assign each point to the centroid of largest cosine (ties: lowest
       cluster), then each centroid becomes the normalised sum of its
       members' directions; a cluster left empty keeps its centroid.  The
       returned labels are the assignment to the final centroids.
  P-3  The proxy token of a cluster is the mean of its members' hidden
       states (not the unit centroid, whose scale would flatten attention),
       rounded to the activation dtype like any hidden state; its query is
       W_q times the token, rounded to the dtype like the block's queries.
  P-4  Proxy attention runs over all seq cache positions (cached rows and
       the recomputed active block), scale 1/sqrt(head_dim); the drift of a
       cluster is KL(P_t || P_{t-1}) in nats averaged over the query heads.
  P-5  Top-k clusters by drift, largest first, ties to the lower cluster
       index; the stale set is every window position whose cluster is
       selected, emitted in ascending position order.
  P-6  After the refresh, sum_k += h_new[i] - h_old[i] for every refreshed
       position i of cluster k; counts and labels are unchanged.
"""

from __future__ import annotations

import numpy as np

from oracle.polestar_ref import round_to


# ---------------------------------------------------------------------------
# 1. block entry: spherical K-means of the window's hidden states
# ---------------------------------------------------------------------------

def spherical_kmeans(h_win: np.ndarray, n_clusters: int, iters: int = 10):
    """h_win: [n][d] hidden states of the window positions (in position order).

    Returns (labels [n] int, centroids [K][d] unit vectors) after `iters`
    rounds of assignment and update; the labels assign every point to its
    nearest final centroid (readings P-1, P-2)."""
    n = h_win.shape[0]
    x = h_win / np.linalg.norm(h_win, axis=1, keepdims=True)          # directions (P-1)
    z = np.stack([x[(j * n) // n_clusters] for j in range(n_clusters)])   # deterministic start (P-2)
    labels = np.zeros(n, dtype=np.int64)
    for _ in range(iters):
        cos = x @ z.T                                   # [n][K]
        labels = np.argmax(cos, axis=1)                 # first maximum: lowest cluster on ties
        for k in range(n_clusters):
            members = x[labels == k]
            if len(members) == 0:
                continue                                # empty: keep the centroid (P-2)
            s = members.sum(axis=0)
            z[k] = s / np.linalg.norm(s)
    labels = np.argmax(x @ z.T, axis=1)                 # the final centroids' assignment (P-2)
    return labels, z


def cluster_sums(h_win: np.ndarray, labels: np.ndarray, n_clusters: int):
    """Per cluster: the sum of its members' hidden states [K][d] and the count [K]."""
    d = h_win.shape[1]
    sums = np.zeros((n_clusters, d))
    counts = np.zeros(n_clusters, dtype=np.int64)
    for i, k in enumerate(labels):
        sums[k] += h_win[i]
        counts[k] += 1
    return sums, counts


# ---------------------------------------------------------------------------
# 2-4. per step: proxy tokens, proxy attention, drift per cluster
# ---------------------------------------------------------------------------

def proxy_tokens(sums: np.ndarray, counts: np.ndarray, dtype: str) -> np.ndarray:
    """[..., K, d]: the members' mean, rounded to the activation dtype (P-3);
    an empty cluster gives the zero token."""
    c = np.asarray(counts, dtype=np.float64)[..., None]
    mean = np.divide(sums, c, out=np.zeros_like(sums, dtype=np.float64), where=c > 0)
    return round_to(mean, dtype)


def proxy_scores(tokens: np.ndarray, w_q: np.ndarray, k_cache: np.ndarray, n_heads: int,
                 dtype: str, scale: float | None = None) -> np.ndarray:
    """Attention logits of the proxy queries over every cache position.

    tokens [b][K][d], w_q [H*hd][d], k_cache [b][S][Hkv][hd]
    -> scores [b][K][H][S] = scale * q_(k,h) . k_(j, kv head of h)   (P-3, P-4)."""
    b, K, d = tokens.shape
    _, S, Hkv, hd = k_cache.shape
    q = round_to(tokens @ w_q.T, dtype).reshape(b, K, n_heads, hd)
    sc = 1.0 / np.sqrt(hd) if scale is None else scale
    group = n_heads // Hkv
    scores = np.empty((b, K, n_heads, S))
    for h in range(n_heads):
        keys = k_cache[:, :, h // group, :]                     # [b][S][hd]
        scores[:, :, h, :] = sc * np.einsum("bkd,bsd->bks", q[:, :, h, :], keys)
    return scores


def proxy_kl(scores: np.ndarray, prev_scores: np.ndarray) -> np.ndarray:
    """Drift per cluster [b][K]: KL(softmax(scores) || softmax(prev_scores))
    over the positions, in nats, averaged over the heads (P-4)."""
    def log_softmax(s):
        m = s.max(axis=-1, keepdims=True)
        return s - m - np.log(np.exp(s - m).sum(axis=-1, keepdims=True))
    lp, lq = log_softmax(scores), log_softmax(prev_scores)
    kl = (np.exp(lp) * (lp - lq)).sum(axis=-1)                  # [b][K][H]
    return kl.mean(axis=-1)


def query_scores(q: np.ndarray, k_cache: np.ndarray, scale: float | None = None) -> np.ndarray:
    """Attention logits of given queries over every cache position:
    q [b][R][H][hd], k_cache [b][S][Hkv][hd] -> [b][R][H][S] =
    scale * q_(r,h) . k_(j, kv head of h), scale 1/sqrt(hd) by default (eq. 3)."""
    b, R, H, hd = q.shape
    _, S, Hkv, _ = k_cache.shape
    sc = 1.0 / np.sqrt(hd) if scale is None else scale
    group = H // Hkv
    out = np.empty((b, R, H, S))
    for h in range(H):
        keys = k_cache[:, :, h // group, :]                     # [b][S][hd]
        out[:, :, h, :] = sc * np.einsum("brd,bsd->brs", q[:, :, h, :], keys)
    return out


def attention_drift(scores: np.ndarray, prev_scores: np.ndarray) -> np.ndarray:
    """The commit drift of Alg. 1: for each query row, KL(A_t || A_(t-1)) of its
    attention distributions over the positions, in nats, averaged over the
    heads (the drift functional of Sec. 3 on the main attention of the last
    layer).  scores, prev_scores [b][R][H][S] -> [b][R]."""
    return proxy_kl(scores, prev_scores)


def log_sum_exp(scores: np.ndarray) -> np.ndarray:
    """Natural-log normaliser of each distribution: [b][K][H]."""
    m = scores.max(axis=-1)
    return m + np.log(np.exp(scores - m[..., None]).sum(axis=-1))


# ---------------------------------------------------------------------------
# 5. top-k clusters -> stale positions
# ---------------------------------------------------------------------------

def select_clusters(drift: np.ndarray, k_top: int) -> np.ndarray:
    """[b][K] bool: the k_top clusters of largest drift, ties to the lower index (P-5)."""
    b, K = drift.shape
    sel = np.zeros((b, K), dtype=bool)
    for s in range(b):
        order = sorted(range(K), key=lambda k: (-drift[s, k], k))
        sel[s, order[:min(k_top, K)]] = True
    return sel


def cluster_members(labels_by_pos: np.ndarray, selected: np.ndarray):
    """labels_by_pos [b][S] (-1 outside the window), selected [b][K]
    -> (stale_idx [b][S] ascending, padded with -1; stale_count [b])."""
    b, S = labels_by_pos.shape
    idx = np.full((b, S), -1, dtype=np.int64)
    cnt = np.zeros(b, dtype=np.int64)
    for s in range(b):
        rows = [p for p in range(S) if labels_by_pos[s, p] >= 0 and selected[s, labels_by_pos[s, p]]]
        idx[s, :len(rows)] = rows
        cnt[s] = len(rows)
    return idx, cnt


# ---------------------------------------------------------------------------
# 6. cluster update after the refresh
# ---------------------------------------------------------------------------

def update_sums(sums: np.ndarray, labels_by_pos: np.ndarray, stale_idx: np.ndarray,
                stale_count: np.ndarray, h_new: np.ndarray, h_old: np.ndarray) -> np.ndarray:
    """sums [b][K][d] after adding h_new[p] - h_old[p] for every refreshed
    window position p to its cluster's sum (P-6)."""
    out = np.array(sums, dtype=np.float64, copy=True)
    for s in range(sums.shape[0]):
        for r in range(int(stale_count[s])):
            p = int(stale_idx[s, r])
            k = int(labels_by_pos[s, p]) if p >= 0 else -1
            if k >= 0:
                out[s, k] += h_new[s, p] - h_old[s, p]
    return out


def labels_by_position(win_idx: np.ndarray, labels: np.ndarray, seq: int) -> np.ndarray:
    """Scatter window labels to a [seq] array, -1 outside the window."""
    out = np.full(seq, -1, dtype=np.int64)
    out[np.asarray(win_idx)] = labels
    return out
