"""The denoising loop of Alg. 1 on a whole pre-norm layer stack, driven from
the host through the library's entry points.

Every tensor operation is a call of libpolestar.so (embedding, RMSNorm, the
hot-path calls drift / select / refresh_kv / project_q / attend, the output
and FFN projections, SwiGLU, the residual add, the LM head, the commit
kernels); torch only provides device buffers and copies bookkeeping values
between host and device (the per-step commit flags, the masks).

Loop (Alg. 1 with per-token drift; Sec. 4.1 "Update Schedule", Sec. 4.2):
  block entry -- a full forward on even blocks, a forward of the local window
                 R = [start - prefix, end + suffix) against the cache on odd
                 ones; then the confidence-only commit of the block;
  each step   -- a refreshing step (more than tau_upd tokens committed since
                 the last refreshing forward) forwards R: per layer the drift
                 of R's rows against the cached hidden states, the top
                 ceil(|Omega|/2) window rows and the block get new K/V and
                 cached rows, and every row of R attends; a plain step
                 forwards the block only.  Then the block's logits, the
                 Polestar-Commit rule with delta = the last layer's drift of
                 the block rows, and the suffix commit of the suffix rows that
                 the last layer refreshed.
A layer's hidden state H (drifted, projected to K/V, cached) is the
normalised attention input RMSNorm(x); the residual stream x is fp32.
"""

from __future__ import annotations

import math
import time
from dataclasses import dataclass

import numpy as np
import torch

from paper_2607_14107_amd import polestar as P


@dataclass
class ModelShape:
    n_layers: int
    d: int
    n_heads: int
    head_dim: int
    ffn: int
    vocab: int
    seq: int

    @property
    def mask_id(self) -> int:
        return self.vocab - 1


@dataclass
class LoopConfig:
    prompt_len: int
    gen_len: int
    block_len: int = 32
    prefix: int = 64
    suffix: int = 32
    tau_upd: int = 3
    h: int = P.DEFAULT_HISTORY
    alpha: float = P.DEFAULT_ALPHA
    tau_s: float = P.DEFAULT_TAU_S
    force_one: bool = True
    suffix_commit: bool = True


def _view(buf: torch.Tensor, *shape) -> torch.Tensor:
    n = 1
    for s in shape:
        n *= s
    return buf.view(-1)[:n].view(*shape)


class Denoiser:
    """Buffers and the loop for one batch of sequences.

    weights: tok_emb [vocab][d], pos_emb [seq][d], w_lm [vocab][d] and
    layers[i] = dict(w_q, w_k, w_v [H*hd][d], w_o [d][H*hd],
    w_gu [2*ffn][d] (gate rows, then up rows), w_down [d][ffn]), all on the GPU
    in one dtype."""

    def __init__(self, weights: dict, shape: ModelShape, batch: int, cfg: LoopConfig):
        self.w, self.shape, self.b, self.cfg = weights, shape, batch, cfg
        sh, b = shape, batch
        if cfg.prompt_len + cfg.gen_len != sh.seq or cfg.gen_len % cfg.block_len:
            raise ValueError("prompt_len + gen_len must be seq and gen_len a multiple of block_len")
        dt = weights["tok_emb"].dtype
        dev = weights["tok_emb"].device
        self.dt, self.dev = dt, dev
        self.code = P.BF16 if dt == torch.bfloat16 else P.FP32
        S, d, H, hd, F, V = sh.seq, sh.d, sh.n_heads, sh.head_dim, sh.ffn, sh.vocab
        B = cfg.block_len
        nl = max(B, cfg.suffix)
        z = lambda *s, t=dt: torch.zeros(s, dtype=t, device=dev)
        self.k = [z(b, S, H, hd) for _ in range(sh.n_layers)]
        self.v = [z(b, S, H, hd) for _ in range(sh.n_layers)]
        self.hc = [z(b, S, d) for _ in range(sh.n_layers)]     # cached hidden states H per layer
        self.h_cur = z(b, S, d)
        self.x = z(b * S * d, t=torch.float32)
        self.q = z(b * S * H * hd)
        self.o = z(b * S * H * hd)
        self.t = z(b * S * d)
        self.g = z(b * S * d)
        self.gu = z(b * S * 2 * F)
        self.a = z(b * S * F)
        self.hf = z(b * nl * d)
        self.logits = z(b * nl * V)
        self.drift = z(b, S, t=torch.float32)
        self.stale_idx = z(b * S, t=torch.int32)
        self.stale_count = z(b, t=torch.int32)
        self.eligible = z(b, S, t=torch.uint8)
        self.hist = z(b, max(cfg.h, 1), B, t=torch.float32)
        self.hist_len = z(b, t=torch.int32)
        self.token = z(b * nl, t=torch.int32)
        self.conf = z(b * nl, t=torch.float32)
        self.commit = z(b * nl, t=torch.uint8)
        self.y = z(b, S, t=torch.int32)
        self.ws = torch.empty(self._workspace_bytes(), dtype=torch.uint8, device=dev)

    def _workspace_bytes(self) -> int:
        """The largest workspace of any call the loop makes (a GEMM plan's
        workspace is not monotonic in its row count, so every shape is asked)."""
        sh, cfg, b, c = self.shape, self.cfg, self.b, self.code
        S, d, H, hd, F, V, B = sh.seq, sh.d, sh.n_heads, sh.head_dim, sh.ffn, sh.vocab, cfg.block_len
        row_counts, tops, heads = {S, B}, {0}, {B}
        for blk in range(cfg.gen_len // B):
            bs = cfg.prompt_len + blk * B
            lo, hi = max(0, bs - cfg.prefix), min(S, bs + B + cfg.suffix)
            row_counts.add(hi - lo)
            tops.add(int(math.ceil((hi - lo - B) / 2)))
            if hi > bs + B:
                heads.add(hi - bs - B)
        sizes = [256]
        for m in row_counts:
            sizes += [P.refresh_kv_workspace_size(c, b, d, H, hd, 0, m), P.project_q_workspace_size(c, b, d, H, hd, m),
                      P.attend_workspace_size(c, b, S, d, H, H, hd, m),
                      P.linear_workspace_size(c, b, m, d, H * hd), P.linear_workspace_size(c, b, m, 2 * F, d),
                      P.linear_workspace_size(c, b, m, d, F)]
        for k in tops:
            sizes.append(P.refresh_kv_workspace_size(c, b, d, H, hd, k, B))
        for n in heads:
            sizes += [P.linear_workspace_size(c, b, n, V, d), P.commit_workspace_size(c, b, n, V)]
        return max(sizes)

    # -- one forward over rows [lo, hi) -------------------------------------------------

    def forward(self, lo: int, hi: int, mode: str, block: tuple[int, int], k_top: int = 0,
                trace=None, fwd: int = 0) -> None:
        """mode "all": every row of R rewritten; "refresh": drift-selected
        window rows and the block; "plain": the block only (R = block)."""
        sh, b, w = self.shape, self.b, self.w
        S, d, H, hd, F = sh.seq, sh.d, sh.n_heads, sh.head_dim, sh.ffn
        m = hi - lo
        bs, bl = block
        x = _view(self.x, b, m, d)
        P.embed(self.y, lo, m, w["tok_emb"], w["pos_emb"], x)
        q, o = _view(self.q, b, m, H, hd), _view(self.o, b, m, H, hd)
        t, g = _view(self.t, b, m, d), _view(self.g, b, m, d)
        gu, a = _view(self.gu, b, m, 2 * F), _view(self.a, b, m, F)
        for li in range(sh.n_layers):
            lw = w["layers"][li]
            before = None
            if trace is not None:
                before = dict(x=x.clone(), k=self.k[li].clone(), v=self.v[li].clone(), h=self.hc[li].clone())
            P.rmsnorm(x, 0, m, self.h_cur, lo)
            if mode == "refresh" or li == sh.n_layers - 1:
                P.drift(self.h_cur, self.hc[li], self.drift)
            if mode == "all":
                idx = cnt = None
                rb, rl = lo, m
            elif mode == "refresh":
                idx, cnt = _view(self.stale_idx, b, k_top), self.stale_count
                P.select(self.drift, k_top, bs, bl, self.eligible, idx, cnt)
                rb, rl = bs, bl
            else:
                idx = cnt = None
                rb, rl = bs, bl
            P.refresh_kv(self.h_cur, idx, cnt, rb, rl, lw["w_k"], lw["w_v"], self.k[li], self.v[li],
                         workspace=self.ws)
            P.copy_rows(self.h_cur, self.hc[li], idx, cnt, rb, rl)
            P.project_q(self.h_cur, lw["w_q"], lo, m, H, out=q, workspace=self.ws)
            P.attend(None, None, self.k[li], self.v[li], lo, m, H, q_buf=q, out=o, workspace=self.ws)
            P.linear(o.view(b, m, H * hd), 0, m, lw["w_o"], t, workspace=self.ws)
            P.residual_add(x, t)
            P.rmsnorm(x, 0, m, g, 0)
            P.linear(g, 0, m, lw["w_gu"], gu, workspace=self.ws)
            P.swiglu(gu, a)
            P.linear(a, 0, m, lw["w_down"], t, workspace=self.ws)
            P.residual_add(x, t)
            if trace is not None:
                trace(dict(event="layer", forward=fwd, layer=li, mode=mode, lo=lo, hi=hi, block=block,
                           k_top=k_top, before=before,
                           after=dict(x=x.clone(), k=self.k[li].clone(), v=self.v[li].clone(),
                                      h=self.hc[li].clone(), h_cur=self.h_cur.clone(), drift=self.drift.clone(),
                                      stale_idx=None if idx is None else idx.clone(),
                                      stale_count=None if cnt is None else cnt.clone())))

    def head(self, lo: int, r0: int, n: int) -> torch.Tensor:
        """Logits of rows [r0, r0 + n) of the last forward over [lo, ...)."""
        sh, b = self.shape, self.b
        hf = _view(self.hf, b, n, sh.d)
        x = _view(self.x, b, self.rows, sh.d)
        P.rmsnorm(x, r0 - lo, n, hf, 0)
        lg = _view(self.logits, b, n, sh.vocab)
        P.linear(hf, 0, n, self.w["w_lm"], lg, workspace=self.ws)
        return lg

    # -- the loop -----------------------------------------------------------------------

    def generate(self, prompt: np.ndarray, trace=None, capture=None, progress=None) -> tuple[np.ndarray, dict]:
        """Runs the loop; returns the token ids [batch][seq] and statistics.

        trace(event) receives, for every forward f of mode m ("all", "refresh",
        "plain") with capture(f, m) true (all forwards when capture is None),
        each layer's input, cache state before and after, drift and stale set,
        and the logits of each commit; for the other forwards only the commit
        decisions and their inputs.  progress(block, forwards) is called after
        every block."""
        sh, cfg, b = self.shape, self.cfg, self.b
        capture = (lambda f, m: True) if capture is None else capture
        captured = set()

        def full(f, m=None):
            if m is not None and capture(f, m):
                captured.add(f)
            return f in captured
        S, B, mask = sh.seq, cfg.block_len, sh.mask_id
        y = np.full((b, S), mask, np.int32)
        y[:, :cfg.prompt_len] = prompt
        self.y.copy_(torch.from_numpy(y))
        stats = dict(forwards=0, committed=0, refreshing_steps=0, plain_steps=0, full_entries=0,
                     window_entries=0, suffix_committed=0)
        gpu_ms = {"all": 0.0, "refresh": 0.0, "plain": 0.0}
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        fwd = 0
        for blk in range(cfg.gen_len // B):
            bs = cfg.prompt_len + blk * B
            be = bs + B
            lo, hi = max(0, bs - cfg.prefix), min(S, be + cfg.suffix)
            el = np.zeros((b, S), np.uint8)
            el[:, lo:bs] = 1
            el[:, be:hi] = 1
            self.eligible.copy_(torch.from_numpy(el))
            # block entry
            elo, ehi = (0, S) if blk % 2 == 0 else (lo, hi)
            self.rows = ehi - elo
            ev0.record()
            self.forward(elo, ehi, "all", (bs, B), trace=trace if full(fwd, "all") else None, fwd=fwd)
            ev1.record()
            stats["full_entries" if blk % 2 == 0 else "window_entries"] += 1
            lg = self.head(elo, bs, B)
            masked = torch.from_numpy((y[:, bs:be] == mask).astype(np.uint8)).to(self.dev)
            tok, conf, cm = P.commit(lg, masked, None, bs, None, None, mask, cfg.tau_s, cfg.alpha, False,
                                     _view(self.token, b, B), _view(self.conf, b, B), _view(self.commit, b, B),
                                     workspace=self.ws)
            n = self._apply(y, bs, tok, cm, trace, fwd, "entry", lg if full(fwd) else None, conf, masked)
            gpu_ms["all"] += ev0.elapsed_time(ev1)
            stats["committed"] += int(n.sum())
            fwd += 1
            since = n                       # per sequence; a batch refreshes when any sequence would
            self.hist_len.zero_()
            while (y[:, bs:be] == mask).any():
                refresh = int(since.max()) > cfg.tau_upd
                rlo, rhi = (lo, hi) if refresh else (bs, be)
                k_top = int(math.ceil((hi - lo - B) / 2)) if refresh else 0
                self.rows = rhi - rlo
                ev0.record()
                mode = "refresh" if refresh else "plain"
                self.forward(rlo, rhi, mode, (bs, B), k_top, trace=trace if full(fwd, mode) else None, fwd=fwd)
                ev1.record()
                stats["refreshing_steps" if refresh else "plain_steps"] += 1
                lg = self.head(rlo, bs, B)
                masked = torch.from_numpy((y[:, bs:be] == mask).astype(np.uint8)).to(self.dev)
                hist_in = (self.hist.clone(), self.hist_len.clone()) if trace is not None else None
                tok, conf, cm = P.commit(lg, masked, self.drift, bs, self.hist, self.hist_len, mask, cfg.tau_s,
                                         cfg.alpha, cfg.force_one, _view(self.token, b, B), _view(self.conf, b, B),
                                         _view(self.commit, b, B), workspace=self.ws)
                n = self._apply(y, bs, tok, cm, trace, fwd, "step", lg if full(fwd) else None, conf, masked, hist_in)
                gpu_ms["refresh" if refresh else "plain"] += ev0.elapsed_time(ev1)
                if cfg.suffix_commit and refresh and be < hi:
                    n_s = self._suffix(y, rlo, be, hi, k_top, trace, fwd, full(fwd))
                    stats["suffix_committed"] += int(n_s.sum())
                    n = n + n_s
                stats["committed"] += int(n.sum())
                fwd += 1
                since = n if refresh else since + n
            if progress is not None:
                progress(blk, fwd)
        torch.cuda.synchronize()
        stats["seconds"] = time.perf_counter() - t0
        stats["forwards"] = fwd
        stats["tpf"] = stats["committed"] / max(fwd * b, 1)      # tokens per forward pass, per sequence
        stats["forward_gpu_ms"] = {k: round(v, 3) for k, v in gpu_ms.items()}
        return y, stats

    def _apply(self, y, r0, tok, cm, trace, fwd, kind, lg, conf, masked, hist_in=None) -> int:
        """Copy the commit flags and tokens to the host, write committed
        tokens into y (host and device); returns the number committed per
        sequence."""
        n_rows = tok.shape[1]
        t = tok.cpu().numpy()
        c = cm.cpu().numpy().astype(bool)
        y[:, r0:r0 + n_rows] = np.where(c, t, y[:, r0:r0 + n_rows])
        self.y[:, r0:r0 + n_rows].copy_(torch.from_numpy(y[:, r0:r0 + n_rows]))
        if trace is not None:
            trace(dict(event="commit", forward=fwd, kind=kind, r0=r0, logits=None if lg is None else lg.clone(),
                       conf=conf.clone(),
                       token=tok.clone(), commit=cm.clone(), masked=masked.clone(), drift=self.drift.clone(),
                       hist_in=hist_in, hist_out=(self.hist.clone(), self.hist_len.clone())))
        return c.sum(axis=1)

    def _suffix(self, y, rlo, be, hi, k_top, trace, fwd, full=True) -> int:
        """Suffix commit of the suffix rows [be, hi) that the last layer refreshed."""
        b, mask = self.b, self.shape.mask_id
        n = hi - be
        idx = _view(self.stale_idx, b, k_top).cpu().numpy()
        cnt = self.stale_count.cpu().numpy()
        el = np.zeros((b, n), np.uint8)
        for s in range(b):
            for p in idx[s, :cnt[s]]:
                if be <= p < hi:
                    el[s, p - be] = 1
        if not el.any():
            return np.zeros(b, np.int64)
        lg = self.head(rlo, be, n)
        masked = torch.from_numpy((y[:, be:hi] == mask).astype(np.uint8)).to(self.dev)
        elig = torch.from_numpy(el).to(self.dev)
        tok, conf, cm = P.suffix_commit(lg, masked, elig, mask, self.cfg.tau_s, _view(self.token, b, n),
                                        _view(self.conf, b, n), _view(self.commit, b, n), workspace=self.ws)
        if trace is not None:
            trace(dict(event="suffix", forward=fwd, r0=be, eligible=elig.clone()))
        return self._apply(y, be, tok, cm, trace, fwd, "suffix", lg if full else None, conf, masked)
