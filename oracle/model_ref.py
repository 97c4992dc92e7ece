"""CPU oracle of Polestar's denoising loop on a whole layer stack.

TEST INFRASTRUCTURE ONLY, like `polestar_ref`: the slow plain reference that
the GPU loop is checked against; only the tests, the package's smoke check and
the benchmark's `cpu_baseline` leg may use it, and it never consumes a value
produced by the HIP path except where a test feeds it the GPU's layer inputs
on purpose (replay).  float64 NumPy; the per-layer hot path is composed from
`polestar_ref` (drift, select, refresh_kv, attend, confidence, commit_rule).

The model (a masked-diffusion LM of the shape the paper evaluates, Sec. 5.1;
readings where the paper gives no detail):
  M-1  Pre-norm layers: x += W_o Attn(h), h = RMSNorm(x); then
       x += W_down (silu(W_gate g) * W_up g), g = RMSNorm(x).  Attention is
       bidirectional over every cache slot (eq. 3).
  M-2  RMSNorm(x) = x / sqrt(mean(x^2) + eps) with unit gain, eps = 1e-5.
  M-3  Positions enter as an absolute position table added to the token
       embedding (no rotary embedding): with random weights it only has to
       make positions distinguishable, and it keeps K/V a plain projection of
       the cached hidden state.
  M-4  Rounding: the residual stream x is kept in fp32 (here: exact); every
       other stored tensor is rounded to the activation dtype: h, g, q, K, V,
       the attention output, W_o's output, the gate/up outputs, the SwiGLU
       product, W_down's output and the logits.
  M-5  The layer's hidden state H (whose drift is measured, from which K/V
       are projected and which is cached) is h = RMSNorm(x) of the layer input.
  M-6  Logits = W_lm RMSNorm(x_final); mask id = vocab - 1.

The loop (Alg. 1 with the window-forward reading of the per-token drift):
  M-7  Block b: J_b = the block's 32 positions; local window
       Omega_b = [start - 2B, end + B) minus J_b, clipped to the sequence;
       R = Omega_b u J_b (a contiguous range).
  M-8  Block entry: even b -> forward every position (all K/V and H
       rewritten); odd b -> forward R against the cache (K/V and H of all of
       R rewritten).  Then the confidence-only commit of J_b (no fallback),
       and the drift history is emptied.
  M-9  Within the block, a step refreshes when the tokens committed since
       the last refreshing forward exceed tau_upd (Sec. 4.1 "Update
       Schedule"); the block entry counts as refreshing.  The count is kept
       per sequence and a batch refreshes when any of its sequences would.  A refreshing step
       forwards R: per layer drift on R's rows, the top ceil(|Omega|/2) of
       Omega refreshed (K/V and H) along with J_b, queries from all of R.  A
       plain step forwards J_b only (its K/V and H rewritten).  After the last
       layer: logits of J_b, delta_j = drift of J_b at the last layer, the
       Polestar-Commit rule (force_one), then the suffix commit of the
       suffix rows that the last layer refreshed (Sec. 4.2).
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

from oracle import polestar_ref as ref

EPS = 1e-5


# ---------------------------------------------------------------------------
# model pieces
# ---------------------------------------------------------------------------

def rmsnorm(x: np.ndarray, eps: float = EPS) -> np.ndarray:
    """M-2: x / sqrt(mean over the last axis of x^2 + eps)."""
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)


def silu(x: np.ndarray) -> np.ndarray:
    """x * sigmoid(x)."""
    return x / (1.0 + np.exp(-x))


@dataclass
class Shape:
    n_layers: int
    d: int
    n_heads: int
    head_dim: int
    ffn: int
    vocab: int
    seq: int
    dtype: str = "bf16"

    @property
    def mask_id(self) -> int:
        return self.vocab - 1                                   # M-6


def embed(tok_emb: np.ndarray, pos_emb: np.ndarray, ids: np.ndarray, lo: int, hi: int) -> np.ndarray:
    """M-3: x[b][r] = tok_emb[ids[b][lo + r]] + pos_emb[lo + r] for r < hi - lo."""
    return tok_emb[ids[:, lo:hi]] + pos_emb[None, lo:hi]


@dataclass
class LayerState:
    """The cached state of one layer: K/V caches [b][S][H][hd] and the cached
    hidden states H [b][S][d], all float64 holding dtype values."""
    k: np.ndarray
    v: np.ndarray
    h: np.ndarray


def layer_forward(x_rows: np.ndarray, lo: int, w: dict, st: LayerState, *, mode: str, block: tuple[int, int],
                  shape: Shape, k_top: int = 0, stale=None) -> dict:
    """One layer over the rows R = [lo, lo + m) of every sequence (M-1, M-5, M-9).

    mode: "all"     -- every K/V and H row of R rewritten (block entry);
          "refresh" -- drift on R, the top k_top of R minus the block
                       (eligible = Omega) and the block rewritten;
          "plain"   -- only the block rewritten (R must be the block).
    stale = (idx, cnt) replaces the refresh mode's own selection (replay of a
    selection taken elsewhere on the same drift).
    Returns a dict with the new state (st is not modified), the drift on R,
    the stale set, and x_out for the rows of R."""
    dt = shape.dtype
    b, m, d = x_rows.shape
    seq = st.h.shape[1]
    bs, bl = block
    h_rows = ref.round_to(rmsnorm(x_rows), dt)                               # M-5
    # drift against the cached hidden states, on the rows of R
    drift = np.zeros((b, seq))
    drift[:, lo:lo + m] = ref.drift(h_rows, st.h[:, lo:lo + m])
    if mode == "all":
        rows = list(range(lo, lo + m))
        idx = np.zeros((b, 0), np.int32)
        cnt = np.zeros(b, np.int32)
        kk, vv, _ = ref.refresh_kv(_place(h_rows, lo, st.h), w["w_k"], w["w_v"], st.k, st.v, idx, cnt, lo, m)
    else:
        eligible = np.zeros((b, seq), bool)
        if mode == "refresh":
            eligible[:, lo:lo + m] = True
            eligible[:, bs:bs + bl] = False
            idx, cnt = ref.select(drift, k_top, bs, bl, eligible) if stale is None else stale
        else:
            assert (lo, m) == (bs, bl)
            idx, cnt = np.zeros((b, 0), np.int32), np.zeros(b, np.int32)
        kk, vv, rows = ref.refresh_kv(_place(h_rows, lo, st.h), w["w_k"], w["w_v"], st.k, st.v, idx, cnt, bs, bl)
    new_h = np.array(st.h, copy=True)
    full_h = _place(h_rows, lo, st.h)
    if mode == "all":
        new_h[:, lo:lo + m] = h_rows
    else:
        for s in range(b):
            r = np.asarray(rows[s], np.int64)
            new_h[s, r] = full_h[s, r]
    new = LayerState(ref.round_to(kk, dt), ref.round_to(vv, dt), new_h)
    # attention of every row of R over the whole (updated) cache
    q = ref.round_to(h_rows @ w["w_q"].T, dt).reshape(b, m, shape.n_heads, shape.head_dim)
    o, _ = ref.attend(q, new.k, new.v)
    o = ref.round_to(o, dt).reshape(b, m, shape.n_heads * shape.head_dim)
    x = x_rows + ref.round_to(o @ w["w_o"].T, dt)
    g = ref.round_to(rmsnorm(x), dt)
    gu = ref.round_to(g @ w["w_gu"].T, dt)
    f = shape.ffn
    a = ref.round_to(silu(gu[..., :f]) * gu[..., f:], dt)
    x = x + ref.round_to(a @ w["w_down"].T, dt)
    return dict(state=new, drift=drift, stale_idx=idx, stale_count=cnt, h=h_rows, x_out=x)


def _place(h_rows: np.ndarray, lo: int, h_all: np.ndarray) -> np.ndarray:
    out = np.array(h_all, copy=True)
    out[:, lo:lo + h_rows.shape[1]] = h_rows
    return out


def logits(x_rows: np.ndarray, w_lm: np.ndarray, dtype: str) -> np.ndarray:
    """M-6: rounded W_lm RMSNorm(x) for the given rows."""
    return ref.round_to(ref.round_to(rmsnorm(x_rows), dtype) @ w_lm.T, dtype)


# ---------------------------------------------------------------------------
# loop control (pure functions of the block index and the commit history)
# ---------------------------------------------------------------------------

def block_bounds(prompt_len: int, block_len: int, b: int) -> tuple[int, int]:
    """J_b = [start, start + block_len)."""
    s = prompt_len + b * block_len
    return s, s + block_len


def window(prompt_len: int, block_len: int, seq: int, b: int, prefix: int, suffix: int) -> tuple[int, int]:
    """M-7: R = [max(0, start - prefix), min(seq, end + suffix))."""
    s, e = block_bounds(prompt_len, block_len, b)
    return max(0, s - prefix), min(seq, e + suffix)


def window_top_k(lo: int, hi: int, block_len: int, frac: float = 0.5) -> int:
    """M-9: ceil(frac * |Omega|), Omega = R minus the block (frac 1/2 by default)."""
    return int(math.ceil(frac * (hi - lo - block_len)))


def refreshes(committed_since: int, tau_upd: int) -> bool:
    """M-9 / Sec. 4.1 "Update Schedule": refresh once more than tau_upd tokens
    were decoded since the last refreshing forward."""
    return committed_since > tau_upd


# ---------------------------------------------------------------------------
# the whole loop, free running (small sizes)
# ---------------------------------------------------------------------------

@dataclass
class LoopParams:
    prompt_len: int
    gen_len: int
    block_len: int = 32
    prefix: int = 64
    suffix: int = 32
    tau_upd: int = 3
    h: int = 5
    alpha: float = 10.0
    tau_s: float = 0.9
    force_one: bool = True
    suffix_commit: bool = True
    window_frac: float = 0.5        # share of the window a refreshing step re-projects (window flow)


@dataclass
class Trace:
    forwards: list = field(default_factory=list)     # one dict per forward pass
    committed: int = 0


def generate(weights: dict, prompt: np.ndarray, shape: Shape, p: LoopParams) -> tuple[np.ndarray, Trace]:
    """Runs the loop of M-7..M-9 on prompt [b][prompt_len]; returns the final
    token ids [b][seq] and the trace of forwards."""
    b = prompt.shape[0]
    seq = p.prompt_len + p.gen_len
    assert seq == shape.seq
    dt = shape.dtype
    mask = shape.mask_id
    y = np.full((b, seq), mask, np.int64)
    y[:, :p.prompt_len] = prompt
    hd = shape.head_dim
    states = [LayerState(np.zeros((b, seq, shape.n_heads, hd)), np.zeros((b, seq, shape.n_heads, hd)),
                         np.zeros((b, seq, shape.d))) for _ in range(shape.n_layers)]
    tr = Trace()
    n_blocks = p.gen_len // p.block_len
    hist = np.zeros((b, max(p.h, 1), p.block_len), np.float32)
    for blk in range(n_blocks):
        bs, be = block_bounds(p.prompt_len, p.block_len, blk)
        lo, hi = window(p.prompt_len, p.block_len, seq, blk, p.prefix, p.suffix)
        # block entry (M-8)
        elo, ehi = (0, seq) if blk % 2 == 0 else (lo, hi)
        x = embed(weights["tok_emb"], weights["pos_emb"], y, elo, ehi)
        for li in range(shape.n_layers):
            r = layer_forward(x, elo, weights["layers"][li], states[li], mode="all", block=(bs, p.block_len),
                              shape=shape)
            states[li], x = r["state"], r["x_out"]
        lg = logits(x[:, bs - elo:be - elo], weights["w_lm"], dt)
        tok, conf = ref.confidence(lg, mask)
        masked = y[:, bs:be] == mask
        cm = masked & (conf.astype(np.float32) > np.float32(p.tau_s))
        y[:, bs:be] = np.where(cm, tok, y[:, bs:be])
        tr.forwards.append(dict(kind="entry_full" if blk % 2 == 0 else "entry_window", block=blk,
                                rows=(elo, ehi), commit=cm, token=tok))
        tr.committed += int(cm.sum())
        since = cm.sum(axis=1)                 # per sequence, decoded after the entry's (refreshing) forward
        hist_len = np.zeros(b, np.int32)
        while (y[:, bs:be] == mask).any():
            refresh = refreshes(int(since.max()), p.tau_upd)
            rlo, rhi = (lo, hi) if refresh else (bs, be)
            kt = window_top_k(lo, hi, p.block_len, p.window_frac) if refresh else 0
            x = embed(weights["tok_emb"], weights["pos_emb"], y, rlo, rhi)
            last = None
            for li in range(shape.n_layers):
                last = layer_forward(x, rlo, weights["layers"][li], states[li],
                                     mode="refresh" if refresh else "plain", block=(bs, p.block_len),
                                     shape=shape, k_top=kt)
                states[li], x = last["state"], last["x_out"]
            lg = logits(x[:, bs - rlo:be - rlo], weights["w_lm"], dt)
            tok, conf = ref.confidence(lg, mask)
            masked = y[:, bs:be] == mask
            delta = last["drift"][:, bs:be].astype(np.float32)
            cm, hist, hist_len = ref.commit_rule(conf.astype(np.float32), delta, masked, hist, hist_len, p.h,
                                                 p.tau_s, p.alpha, p.force_one)
            y[:, bs:be] = np.where(cm, tok, y[:, bs:be])
            n_commit = cm.sum(axis=1)
            scm = None
            if p.suffix_commit and refresh and be < hi:
                el = ref.suffix_eligible(last["stale_idx"], last["stale_count"], be, hi - be)
                slg = logits(x[:, be - rlo:hi - rlo], weights["w_lm"], dt)
                stok, sconf = ref.confidence(slg, mask)
                smask = y[:, be:hi] == mask
                scm = ref.suffix_commit_rule(sconf.astype(np.float32), smask, el, p.tau_s)
                y[:, be:hi] = np.where(scm, stok, y[:, be:hi])
                n_commit = n_commit + scm.sum(axis=1)
            tr.forwards.append(dict(kind="refresh" if refresh else "plain", block=blk, rows=(rlo, rhi),
                                    commit=cm, token=tok, suffix_commit=scm))
            tr.committed += int(n_commit.sum())
            since = n_commit if refresh else since + n_commit
    return y, tr


# ---------------------------------------------------------------------------
# The paper's own flow (Alg. 1, per-layer loop; Sec. 4.1 "Measuring Drift and
# Layer-wise KV Updates"): clustered proxy drift per layer and update packets
# passed from layer to layer.  Readings:
#   F3-1  each layer caches its inputs X (the residual stream, kept exact
#         here, fp32 on the GPU) besides K/V and H = RMSNorm(X); the local
#         window's H is clustered per layer at block entry (proxy_ref), and
#         the proxy scores of that entry are the first P;
#   F3-2  on a refreshing step (the tau_upd schedule), layer l: (1) patches
#         the rows of the packet U(l) it receives -- X and H of those rows,
#         their K/V and the cluster sums; (2) forwards the block; (3) takes
#         the proxy drift of its clusters against its last P and the members
#         of the top-k clusters as S(l); (4) forwards the rows S(l) from their
#         cached inputs, and their outputs are the packet U(l + 1);
#   F3-3  the packet of layer 0 holds the window rows whose token a suffix
#         commit changed since the last refreshing forward (new embeddings);
#   F3-5  with a codec (codec_ref, MXFP4 / MXFP8), the window rows' cached
#         inputs are kept as residuals to their cluster's mean input (taken
#         at block entry and fixed for the block); patched rows are
#         re-encoded, and a packet's forward starts from the decoded inputs;
#   F3-4  a plain step forwards the block only; the commit drift of the
#         block is the attention drift of its queries at the last layer
#         (proxy_ref.attention_drift), measured every forward after the entry
#         set its baseline; the suffix commit reads the last layer's packet
#         rows that lie in the suffix window.
# ---------------------------------------------------------------------------

from oracle import codec_ref as cr
from oracle import proxy_ref as pr


@dataclass
class PacketLayer:
    st: LayerState                 # K, V, H (= rounded RMSNorm of X)
    x: np.ndarray                  # [b][S][d] cached layer inputs
    labels: np.ndarray             # [b][S] cluster of each window position, -1 elsewhere
    sums: np.ndarray               # [b][K][d] sums of the members' H
    counts: np.ndarray             # [b][K]
    scores: np.ndarray             # [b][K][H][S] last proxy scores
    codec: dict | None = None      # F3-5: fmt, codes [b][S][d], exps [b][S][d/32], means [b][K][d]


def _mean_rows(codec: dict, labels: np.ndarray, s: int, rows) -> np.ndarray:
    """Each row's cluster mean (zeros outside every cluster)."""
    d = codec["means"].shape[2]
    return np.stack([codec["means"][s, labels[s, p]] if labels[s, p] >= 0 else np.zeros(d) for p in rows])


def encode_rows(codec: dict, x: np.ndarray, labels: np.ndarray, rows) -> dict:
    """F3-5: codes of the listed rows [b][...] of x against their cluster means."""
    out = dict(codec, codes=np.array(codec["codes"], copy=True), exps=np.array(codec["exps"], copy=True))
    for s in range(x.shape[0]):
        r = list(rows[s])
        if r:
            c, e = cr.encode(x[s, r], _mean_rows(codec, labels, s, r), codec["fmt"])
            out["codes"][s, r], out["exps"][s, r] = c, e
    return out


def decoded_rows(pl: "PacketLayer", s: int, rows) -> np.ndarray:
    """The cached inputs of rows of sequence s, decoded when a codec is on."""
    r = np.asarray(rows, np.int64)
    if pl.codec is None:
        return pl.x[s, r]
    c = pl.codec
    return cr.decode(c["codes"][s, r], c["exps"][s, r], _mean_rows(c, pl.labels, s, r), c["fmt"])


def patch(pl: PacketLayer, rows, x_new: np.ndarray, w: dict, shape: Shape) -> PacketLayer:
    """F3-2 (1): rows[b] = list of positions, x_new[b][i] their new inputs."""
    dt = shape.dtype
    k, v, h = (np.array(a, copy=True) for a in (pl.st.k, pl.st.v, pl.st.h))
    x = np.array(pl.x, copy=True)
    sums = np.array(pl.sums, copy=True)
    H, hd = shape.n_heads, shape.head_dim
    for s in range(x.shape[0]):
        for i, p in enumerate(rows[s]):
            hn = ref.round_to(rmsnorm(x_new[s][i]), dt)
            lab = int(pl.labels[s, p])
            if lab >= 0:
                sums[s, lab] += hn - h[s, p]                       # P-6
            h[s, p] = hn
            x[s, p] = x_new[s][i]
            k[s, p] = ref.round_to(hn @ w["w_k"].T, dt).reshape(H, hd)
            v[s, p] = ref.round_to(hn @ w["w_v"].T, dt).reshape(H, hd)
    codec = None if pl.codec is None else encode_rows(pl.codec, x, pl.labels, rows)
    return PacketLayer(LayerState(k, v, h), x, pl.labels, sums, pl.counts, pl.scores, codec)


def sparse_forward(pl: PacketLayer, rows, w: dict, shape: Shape) -> list:
    """F3-2 (4): the rows' outputs of this layer from their cached inputs,
    attending over the current cache; returns x_out[b] = [n_b][d]."""
    dt = shape.dtype
    out = []
    for s in range(pl.x.shape[0]):
        r = np.asarray(rows[s], np.int64)
        if r.size == 0:
            out.append(np.zeros((0, shape.d)))
            continue
        xr = decoded_rows(pl, s, r)[None]
        h = ref.round_to(rmsnorm(xr), dt)
        q = ref.round_to(h @ w["w_q"].T, dt).reshape(1, r.size, shape.n_heads, shape.head_dim)
        o, _ = ref.attend(q, pl.st.k[s:s + 1], pl.st.v[s:s + 1])
        o = ref.round_to(o, dt).reshape(1, r.size, -1)
        xx = xr + ref.round_to(o @ w["w_o"].T, dt)
        g = ref.round_to(rmsnorm(xx), dt)
        gu = ref.round_to(g @ w["w_gu"].T, dt)
        a = ref.round_to(silu(gu[..., :shape.ffn]) * gu[..., shape.ffn:], dt)
        out.append((xx + ref.round_to(a @ w["w_down"].T, dt))[0])
    return out


def proxy_select(pl: PacketLayer, w: dict, shape: Shape, k_top: int):
    """F3-2 (3): drift per cluster against the last proxy scores, the top
    k_top clusters and their member rows; returns (drift, rows, new scores)."""
    tok = pr.proxy_tokens(pl.sums, pl.counts, shape.dtype)
    sc = pr.proxy_scores(tok, w["w_q"], pl.st.k, shape.n_heads, shape.dtype)
    drift = pr.proxy_kl(sc, pl.scores)
    sel = pr.select_clusters(drift, k_top)
    idx, cnt = pr.cluster_members(pl.labels, sel)
    rows = [list(idx[s, :cnt[s]]) for s in range(idx.shape[0])]
    return drift, rows, sc


def _window_positions(lo: int, bs: int, be: int, hi: int) -> np.ndarray:
    return np.concatenate([np.arange(lo, bs), np.arange(be, hi)]).astype(np.int64)


def cluster_layer(h: np.ndarray, win: np.ndarray, n_clusters: int, iters: int):
    """Spherical K-means of every sequence's window rows of H (F3-1):
    (labels by position [b][S], sums [b][K][d], counts [b][K])."""
    b, seq, d = h.shape
    labels = np.full((b, seq), -1, np.int64)
    sums = np.zeros((b, n_clusters, d))
    counts = np.zeros((b, n_clusters), np.int64)
    for s in range(b):
        lab, _ = pr.spherical_kmeans(h[s, win], n_clusters, iters)
        sums[s], counts[s] = pr.cluster_sums(h[s, win], lab, n_clusters)
        labels[s] = pr.labels_by_position(win, lab, seq)
    return labels, sums, counts


def block_queries(h_block: np.ndarray, w_q: np.ndarray, shape: Shape) -> np.ndarray:
    """The block's rounded queries [b][B][H][hd] from its rows of H."""
    b, n, _ = h_block.shape
    return ref.round_to(h_block @ w_q.T, shape.dtype).reshape(b, n, shape.n_heads, shape.head_dim)


def generate_packets(weights: dict, prompt: np.ndarray, shape: Shape, p: LoopParams, n_clusters: int = 8,
                     k_top: int = 4, iters: int = 10, codec: str | None = None) -> tuple[np.ndarray, Trace]:
    """The loop of Alg. 1 with update packets and proxy drift (F3-1..F3-5)."""
    b = prompt.shape[0]
    seq = p.prompt_len + p.gen_len
    assert seq == shape.seq
    dt, mask, L = shape.dtype, shape.mask_id, shape.n_layers
    y = np.full((b, seq), mask, np.int64)
    y[:, :p.prompt_len] = prompt
    hd, H = shape.head_dim, shape.n_heads
    zeros = lambda *s: np.zeros(s)
    layers = [PacketLayer(LayerState(zeros(b, seq, H, hd), zeros(b, seq, H, hd), zeros(b, seq, shape.d)),
                          zeros(b, seq, shape.d), np.full((b, seq), -1, np.int64), zeros(b, n_clusters, shape.d),
                          np.zeros((b, n_clusters), np.int64), zeros(b, n_clusters, H, seq))
              for _ in range(L)]
    tr = Trace()
    hist = np.zeros((b, max(p.h, 1), p.block_len), np.float32)
    for blk in range(p.gen_len // p.block_len):
        bs, be = block_bounds(p.prompt_len, p.block_len, blk)
        lo, hi = window(p.prompt_len, p.block_len, seq, blk, p.prefix, p.suffix)
        win = _window_positions(lo, bs, be, hi)
        elo, ehi = (0, seq) if blk % 2 == 0 else (lo, hi)
        x = embed(weights["tok_emb"], weights["pos_emb"], y, elo, ehi)
        for li in range(L):
            w = weights["layers"][li]
            r = layer_forward(x, elo, w, layers[li].st, mode="all", block=(bs, p.block_len), shape=shape)
            xc = np.array(layers[li].x, copy=True)
            xc[:, elo:ehi] = x
            st = r["state"]
            labels, sums, counts = cluster_layer(st.h, win, n_clusters, iters)
            sc0 = pr.proxy_scores(pr.proxy_tokens(sums, counts, dt), w["w_q"], st.k, H, dt)
            cd = None
            if codec is not None:
                means = np.stack([cr.cluster_means(xc[s], labels[s], n_clusters) for s in range(b)])
                cd = dict(fmt=codec, codes=np.zeros((b, seq, shape.d), np.int64),
                          exps=np.zeros((b, seq, shape.d // cr.BLOCK), np.int64), means=means)
                cd = encode_rows(cd, xc, labels, [win] * b)
            layers[li] = PacketLayer(st, xc, labels, sums, counts, sc0, cd)
            if li == L - 1:
                att = pr.query_scores(block_queries(r["h"][:, bs - elo:be - elo], w["w_q"], shape), st.k)
            x = r["x_out"]
        lg = logits(x[:, bs - elo:be - elo], weights["w_lm"], dt)
        tok, conf = ref.confidence(lg, mask)
        masked = y[:, bs:be] == mask
        cm = masked & (conf.astype(np.float32) > np.float32(p.tau_s))
        y[:, bs:be] = np.where(cm, tok, y[:, bs:be])
        tr.forwards.append(dict(kind="entry_full" if blk % 2 == 0 else "entry_window", block=blk,
                                rows=(elo, ehi), commit=cm, token=tok))
        tr.committed += int(cm.sum())
        since = cm.sum(axis=1)
        hist_len = np.zeros(b, np.int32)
        dirty = [[] for _ in range(b)]
        while (y[:, bs:be] == mask).any():
            refresh = refreshes(int(since.max()), p.tau_upd)
            x = embed(weights["tok_emb"], weights["pos_emb"], y, bs, be)
            pkt_rows = dirty if refresh else [[] for _ in range(b)]
            pkt_x = [weights["tok_emb"][y[s, pkt_rows[s]]] + weights["pos_emb"][pkt_rows[s]] for s in range(b)]
            proxy = []                       # per layer: (drift per cluster, the proxy scores it measured)
            for li in range(L):
                w = weights["layers"][li]
                pl = layers[li]
                if refresh and any(len(rr) for rr in pkt_rows):
                    pl = patch(pl, pkt_rows, pkt_x, w, shape)
                # (X of the block rows is not kept: packets carry window rows only,
                # and the next block entry rewrites X of this block)
                r = layer_forward(x, bs, w, pl.st, mode="plain", block=(bs, p.block_len), shape=shape)
                pl = PacketLayer(r["state"], pl.x, pl.labels, pl.sums, pl.counts, pl.scores, pl.codec)
                if refresh:
                    pdrift, rows, sc = proxy_select(pl, w, shape, k_top)
                    proxy.append((pdrift, sc))
                    pl = PacketLayer(pl.st, pl.x, pl.labels, pl.sums, pl.counts, sc, pl.codec)
                    pkt_x = sparse_forward(pl, rows, w, shape)
                    pkt_rows = rows
                layers[li] = pl
                if li == L - 1:
                    att_new = pr.query_scores(block_queries(r["h"], w["w_q"], shape), pl.st.k)
                    delta = pr.attention_drift(att_new, att).astype(np.float32)
                    att = att_new
                x = r["x_out"]
            lg = logits(x, weights["w_lm"], dt)
            tok, conf = ref.confidence(lg, mask)
            masked = y[:, bs:be] == mask
            cm, hist, hist_len = ref.commit_rule(conf.astype(np.float32), delta, masked, hist, hist_len, p.h,
                                                 p.tau_s, p.alpha, p.force_one)
            y[:, bs:be] = np.where(cm, tok, y[:, bs:be])
            n_commit = cm.sum(axis=1)
            scm = None
            if p.suffix_commit and refresh and be < hi:
                n_s = hi - be
                el = np.zeros((b, n_s), bool)
                slg = np.zeros((b, n_s, shape.vocab))
                for s in range(b):
                    for i, pos in enumerate(pkt_rows[s]):
                        if be <= pos < hi:
                            el[s, pos - be] = True
                            slg[s, pos - be] = logits(pkt_x[s][i][None, None], weights["w_lm"], dt)[0, 0]
                stok, sconf = ref.confidence(slg, mask)
                smask = y[:, be:hi] == mask
                scm = ref.suffix_commit_rule(sconf.astype(np.float32), smask, el, p.tau_s)
                y[:, be:hi] = np.where(scm, stok, y[:, be:hi])
                n_commit = n_commit + scm.sum(axis=1)
            if refresh:      # F3-3: the rows this step's suffix commit changed go to the next layer-0 packet
                dirty = [[] for _ in range(b)] if scm is None else \
                    [[int(be + j) for j in np.flatnonzero(scm[s])] for s in range(b)]
            tr.forwards.append(dict(kind="refresh" if refresh else "plain", block=blk, rows=(bs, be),
                                    commit=cm, token=tok, suffix_commit=scm, proxy=proxy))
            tr.committed += int(n_commit.sum())
            since = n_commit if refresh else since + n_commit
    return y, tr
