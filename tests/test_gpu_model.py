"""GPU parity of the whole-stack loop: the glue calls (embedding, RMSNorm,
dense projections, SwiGLU, residual add, row copy) against their plain
definitions, and the denoising loop of a small stack replayed event by event
against the float64 oracle (oracle/model_ref.py).

Replay: every layer of every forward is recomputed by the oracle from the
GPU's layer input and the GPU's cache state before the layer, with the GPU's
stale set (itself checked bit-exactly against the oracle's selection on the
GPU's drift); outputs must agree to 2e-2 per row (bf16), the drift to 1e-4
relative on the rows the GPU normalised, decisions exactly."""

import numpy as np
import pytest

from oracle import codec_ref as cr
from oracle import model_ref as mr
from oracle import polestar_ref as ref
from paper_2607_14107_amd import inputs
from tests._util import assert_drift_close, assert_rows_close, ensure_built, from_dev, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    ensure_built()
    from paper_2607_14107_amd import polestar
    return polestar


def _torch():
    import torch
    return torch


def dec(t, dtype="bf16"):
    """GPU tensor -> float64 values."""
    a = from_dev(t)
    return ref.decode(a, dtype) if a.dtype == np.uint16 else np.asarray(a, dtype=np.float64)


# ---------------------------------------------------------------------------
# glue calls
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_embed_rmsnorm_swiglu_residual(P, dtype):
    torch = _torch()
    g = np.random.default_rng(1)
    b, seq, d, V, lo, n = 3, 40, 512, 77, 5, 29
    st = lambda a: inputs.store(a, dtype)
    tok, pos = st(g.standard_normal((V, d)).astype(np.float32)), st(g.standard_normal((seq, d)).astype(np.float32))
    ids = g.integers(0, V, size=(b, seq)).astype(np.int32)
    x = torch.empty((b, n, d), dtype=torch.float32, device="cuda")
    P.embed(torch.from_numpy(ids).cuda(), lo, n, to_dev(tok, dtype), to_dev(pos, dtype), x)
    want = ref.decode(tok, dtype)[ids[:, lo:lo + n]] + ref.decode(pos, dtype)[None, lo:lo + n]
    np.testing.assert_allclose(from_dev(x), want, rtol=1e-6, atol=1e-6)
    # RMSNorm into rows [7, 7 + n) of a wider buffer; other rows untouched
    out = to_dev(st(np.full((b, 50, d), 0.5, np.float32)), dtype)
    P.rmsnorm(x, 0, n, out, 7)
    got = dec(out, dtype)
    assert_rows_close(got[:, 7:7 + n], mr.rmsnorm(from_dev(x).astype(np.float64)), 1e-5 if dtype == "fp32" else 8e-3,
                      "rmsnorm")
    assert np.all(got[:, :7] == 0.5) and np.all(got[:, 7 + n:] == 0.5)
    # SwiGLU
    F = 96
    gu = st(g.standard_normal((b * n, 2 * F)).astype(np.float32) * 3)
    a = to_dev(st(np.zeros((b * n, F), np.float32)), dtype)
    P.swiglu(to_dev(gu, dtype), a)
    gud = ref.decode(gu, dtype)
    np.testing.assert_allclose(dec(a, dtype), ref.round_to(mr.silu(gud[:, :F]) * gud[:, F:], dtype),
                               rtol=1e-5 if dtype == "fp32" else 8e-3, atol=1e-6)
    # residual add
    y = st(g.standard_normal((b, n, d)).astype(np.float32))
    x0 = from_dev(x).astype(np.float64)
    P.residual_add(x, to_dev(y, dtype))
    np.testing.assert_allclose(from_dev(x), x0 + ref.decode(y, dtype), rtol=1e-6, atol=1e-6)


@pytest.mark.parametrize("dtype,b,seq,rs,n,K,N", [
    ("bf16", 3, 50, 4, 37, 384, 272),        # small-M kernel, ragged rows
    ("bf16", 2, 300, 10, 261, 256, 400),     # rows kernel, split K, ragged tiles
    ("fp32", 2, 90, 0, 90, 320, 144),
    ("bf16", 1, 700, 0, 700, 512, 1536),     # rows kernel, several row tiles
    ("bf16", 1, 400, 10, 385, 4096, 6480),    # 256x256-tile kernel: ragged rows and columns, K split 4
    ("bf16", 2, 1100, 30, 1000, 4096, 2000),  # 192x192-tile kernel: ragged rows and columns, K split 2
    ("bf16", 1, 1300, 20, 1250, 2048, 2512),  # 192x192-tile kernel: ragged rows and columns, K split 2
    ("bf16", 3, 320, 10, 300, 4096, 3008),    # 256x192-tile kernel: 900 rows of three sequences, K split 4
    ("bf16", 1, 460, 5, 450, 2048, 16736),    # 256x192-tile kernel, unsplit, ragged last column tile
    ("bf16", 2, 210, 3, 200, 4096, 2800),     # rows kernel, K split 6 (too short a split for two tile rows)
    ("bf16", 1, 4000, 0, 4000, 1024, 8000),   # tile kernel, no K split, ragged last column tile
    ("bf16", 1, 1100, 0, 1052, 3584, 1024),   # tile kernel, K split 7 (16 stages each)
    ("bf16", 2, 200, 20, 150, 4096, 1008),    # DMA kernel, two row tiles, ragged columns
])
def test_linear(P, dtype, b, seq, rs, n, K, N):
    torch = _torch()
    g = np.random.default_rng(2)
    x = inputs.store(g.standard_normal((b, seq, K)).astype(np.float32), dtype)
    w = inputs.store((g.standard_normal((N, K)) * 0.05).astype(np.float32), dtype)
    y = torch.empty((b, n, N), dtype=torch.bfloat16 if dtype == "bf16" else torch.float32, device="cuda")
    P.linear(to_dev(x, dtype), rs, n, to_dev(w, dtype), y)
    want = ref.decode(x, dtype)[:, rs:rs + n] @ ref.decode(w, dtype).T
    assert_rows_close(dec(y, dtype), want, 1e-4 if dtype == "fp32" else 2e-2, "linear")


def test_copy_rows(P):
    torch = _torch()
    g = np.random.default_rng(3)
    b, seq, d = 2, 30, 64
    src = inputs.store(g.standard_normal((b, seq, d)).astype(np.float32), "bf16")
    dst0 = inputs.store(g.standard_normal((b, seq, d)).astype(np.float32), "bf16")
    idx = np.array([[3, 7, 29, -1], [0, 40, 12, 5]], np.int32)     # 40: out of range, skipped
    cnt = np.array([3, 4], np.int32)
    dst = to_dev(dst0, "bf16")
    P.copy_rows(to_dev(src, "bf16"), dst, torch.from_numpy(idx).cuda(), torch.from_numpy(cnt).cuda(), 10, 4)
    want = dst0.copy()
    for s, rows in enumerate([[3, 7, 29], [0, 12, 5]]):
        for p in rows + list(range(10, 14)):
            want[s, p] = src[s, p]
    assert np.array_equal(from_dev(dst), want)


# ---------------------------------------------------------------------------
# the loop on a small stack, replayed against the oracle
# ---------------------------------------------------------------------------

def stack_weights(cfg, oracle_embeddings=True):
    names = ("tok_emb", "pos_emb", "w_lm")
    host = {n: inputs.stack_tensor(cfg, n) for n in names}
    host["layers"] = [{m: inputs.stack_tensor(cfg, m, li) for m in inputs.STACK_MATRICES} for li in range(cfg.n_layers)]
    devw = {n: to_dev(host[n], cfg.dtype) for n in names}
    devw["layers"] = [{m: to_dev(l[m], cfg.dtype) for m in l} for l in host["layers"]]
    ow = {n: ref.decode(host[n], cfg.dtype) for n in names if oracle_embeddings or n == "w_lm"}
    ow["layers"] = [{m: ref.decode(l[m], cfg.dtype) for m in l} for l in host["layers"]]
    return devw, ow


def run_stack(P, index, trace=True, capture=None, **loop):
    from paper_2607_14107_amd import model
    cfg = inputs.STACKS[index]
    devw, ow = stack_weights(cfg, oracle_embeddings=cfg.d <= 1024)
    shape = model.ModelShape(cfg.n_layers, cfg.d, cfg.n_heads, cfg.head_dim, cfg.ffn, cfg.vocab, cfg.seq)
    lc = model.LoopConfig(prompt_len=cfg.prompt_len, gen_len=cfg.gen_len, block_len=cfg.block_len, **loop)
    den = model.Denoiser(devw, shape, cfg.batch, lc)
    events = []
    y, stats = den.generate(inputs.stack_prompt(cfg), trace=events.append if trace else None, capture=capture)
    return cfg, lc, ow, y, stats, events


def replay(events, cfg, lc, ow, seqs=None):
    """Checks every traced event against the oracle.  Value parity (layer
    outputs, caches, logits, confidences) on the sequences in `seqs` (all by
    default); selections and decisions on every sequence.  Returns the
    number of layer events checked."""
    shape = mr.Shape(cfg.n_layers, cfg.d, cfg.n_heads, cfg.head_dim, cfg.ffn, cfg.vocab, cfg.seq, cfg.dtype)
    mask = shape.mask_id
    B = lc.block_len
    sq = np.arange(cfg.batch) if seqs is None else np.asarray(seqs)
    last_x, last_stale, suffix_elig = {}, {}, {}
    n_layer_checks = 0
    for ev in events:
        if ev["event"] == "layer":
            lo, hi, mode, li = ev["lo"], ev["hi"], ev["mode"], ev["layer"]
            bs, bl = ev["block"]
            bf, af = ev["before"], ev["after"]
            st = mr.LayerState(dec(bf["k"])[sq], dec(bf["v"])[sq], dec(bf["h"])[sq])
            x_in = from_dev(bf["x"])[sq].astype(np.float64)
            h_gpu = dec(af["h_cur"])[sq][:, lo:hi]
            assert_rows_close(h_gpu, ref.round_to(mr.rmsnorm(x_in), "bf16"), 2e-2, f"h rows, layer {li}")
            stale = None
            if mode == "refresh" or (li == cfg.n_layers - 1 and lc.flow != "packet"):
                gd = from_dev(af["drift"])[sq][:, lo:hi]
                assert_drift_close(gd, ref.drift(h_gpu, st.h[:, lo:hi]))
            if mode == "refresh":
                el = np.zeros((cfg.batch, cfg.seq), bool)
                el[:, lo:hi] = True
                el[:, bs:bs + bl] = False
                widx, wcnt = ref.select(from_dev(af["drift"]), ev["k_top"], bs, bl, el)
                gidx, gcnt = from_dev(af["stale_idx"]), from_dev(af["stale_count"])
                assert np.array_equal(gcnt, wcnt)
                assert np.array_equal(gidx, widx)
                stale = (gidx, gcnt)
            r = mr.layer_forward(x_in, lo, ow["layers"][li], st, mode=mode, block=(bs, bl), shape=shape,
                                 k_top=ev["k_top"], stale=None if stale is None else (stale[0][sq], stale[1][sq]))
            assert_rows_close(from_dev(af["x"])[sq], r["x_out"], 2e-2, f"x_out fwd {ev['forward']} layer {li}")
            for nm in ("k", "v"):
                assert_rows_close(dec(af[nm])[sq], getattr(r["state"], nm), 2e-2, f"{nm} cache")
            assert_rows_close(dec(af["h"])[sq], r["state"].h, 2e-2, "cached H")
            # rows the layer did not rewrite are bit-identical
            touched = np.zeros((cfg.batch, cfg.seq), bool)
            if mode == "all":
                touched[:, lo:hi] = True
            else:
                touched[:, bs:bs + bl] = True
                if stale is not None:
                    for s in range(cfg.batch):
                        touched[s, stale[0][s, :stale[1][s]]] = True
            for nm in ("k", "v", "h"):
                a, b0 = from_dev(af[nm]), from_dev(bf[nm])
                assert np.array_equal(a[~touched], b0[~touched]), f"{nm}: untouched rows changed"
            n_layer_checks += 1
            if li == cfg.n_layers - 1:
                last_x[ev["forward"]] = (lo, from_dev(af["x"])[sq].astype(np.float64))
                last_stale[ev["forward"]] = stale
        elif ev["event"] == "commit":
            r0 = ev["r0"]
            gconf = from_dev(ev["conf"])
            n = gconf.shape[1]
            if ev["logits"] is not None:
                lo, xf = last_x[ev["forward"]]
                lg = ref.decode(from_dev(ev["logits"])[sq], "bf16")
                assert_rows_close(lg, mr.logits(xf[:, r0 - lo:r0 - lo + n], ow["w_lm"], "bf16"), 2e-2, "logits")
                tok, conf = ref.confidence(lg, mask)
                assert np.array_equal(from_dev(ev["token"])[sq], tok)
                np.testing.assert_allclose(gconf[sq], conf, rtol=1e-4)
            masked = from_dev(ev["masked"]).astype(bool)
            gcm = from_dev(ev["commit"]).astype(bool)
            if ev["kind"] == "step" and lc.flow == "packet":
                hist, hl = (from_dev(t) for t in ev["hist_in"])
                delta = from_dev(ev["drift"])                     # the attention drift of the block rows
                wm, wh, wl = ref.commit_rule(gconf, delta, masked, hist, hl, lc.h, lc.tau_s, lc.alpha, lc.force_one)
                assert np.array_equal(gcm, wm)
            elif ev["kind"] == "entry":
                assert np.array_equal(gcm, masked & (gconf > np.float32(lc.tau_s)))
            elif ev["kind"] == "step":
                hist, hl = (from_dev(t) for t in ev["hist_in"])
                delta = from_dev(ev["drift"])[:, r0:r0 + B]
                wm, wh, wl = ref.commit_rule(gconf, delta, masked, hist, hl, lc.h, lc.tau_s, lc.alpha, lc.force_one)
                assert np.array_equal(gcm, wm)
                gh, gl = (from_dev(t) for t in ev["hist_out"])
                assert np.array_equal(gl, wl)
                for s in range(cfg.batch):
                    assert np.array_equal(gh[s, :gl[s]], wh[s, :wl[s]])
            else:
                el = suffix_elig[ev["forward"]]
                if ev["forward"] in last_stale:
                    gidx, gcnt = last_stale[ev["forward"]]
                    assert np.array_equal(ref.suffix_eligible(gidx, gcnt, r0, n), el)
                assert np.array_equal(gcm, ref.suffix_commit_rule(gconf, masked, el, lc.tau_s))
        elif ev["event"] == "suffix":           # precedes the suffix commit of its forward
            suffix_elig[ev["forward"]] = from_dev(ev["eligible"]).astype(bool)
    return n_layer_checks


def test_tiny_stack_loop_replay(P):
    cfg, lc, ow, y, stats, events = run_stack(P, 40)
    mask = cfg.vocab - 1
    # the loop finished: every generated position committed, the prompt intact
    assert not (y == mask).any()
    assert np.array_equal(y[:, :cfg.prompt_len], inputs.stack_prompt(cfg))
    assert stats["committed"] == cfg.batch * cfg.gen_len
    assert stats["refreshing_steps"] > 0 and stats["plain_steps"] > 0
    assert replay(events, cfg, lc, ow) == cfg.n_layers * stats["forwards"]


def test_llada_width_stack_replay(P):
    """The LLaDA-8B-shaped stack at full width and sequence length (d 4096,
    FFN 12288, vocab 126464, batch 16, seq 768) with two layers and two
    blocks: the first forward of each kind is traced and replayed on two of
    the sixteen sequences; every decision of the run is replayed."""
    firsts = set()

    def capture(f, mode):
        if mode in firsts:
            return False
        firsts.add(mode)
        return True

    cfg, lc, ow, y, stats, events = run_stack(P, 41, capture=capture)
    assert not (y == cfg.vocab - 1).any()
    assert stats["committed"] == cfg.batch * cfg.gen_len
    assert stats["full_entries"] == 1 and stats["window_entries"] == 1
    n = replay(events, cfg, lc, ow, seqs=[0, 11])
    assert n == cfg.n_layers * len(firsts) and firsts == {"all", "refresh", "plain"}


def test_tiny_stack_loop_schedule_and_determinism(P):
    cfg, lc, _, y, stats, events = run_stack(P, 40)
    _, _, _, y2, stats2, _ = run_stack(P, 40, trace=False)
    assert np.array_equal(y, y2) and stats["forwards"] == stats2["forwards"]
    # the kinds of forward follow the schedule rule on the GPU's own commits
    forwards = {}
    for ev in events:
        if ev["event"] == "layer" and ev["layer"] == 0:
            forwards[ev["forward"]] = dict(mode=ev["mode"], lo=ev["lo"], hi=ev["hi"], n=np.zeros(cfg.batch, int),
                                           entry=None)
        elif ev["event"] == "commit":
            f = forwards[ev["forward"]]
            f["n"] = f["n"] + from_dev(ev["commit"]).sum(axis=1)
            f["entry"] = f["entry"] or ev["kind"] == "entry"
    since = None
    n_blocks = 0
    for k in sorted(forwards):
        f = forwards[k]
        if f["entry"]:
            full = n_blocks % 2 == 0
            assert f["mode"] == "all" and ((f["lo"], f["hi"]) == (0, cfg.seq)) == full
            n_blocks += 1
            since = f["n"]
            continue
        assert (f["mode"] == "refresh") == mr.refreshes(int(since.max()), lc.tau_upd)
        since = f["n"] if f["mode"] == "refresh" else since + f["n"]
    assert n_blocks == cfg.gen_len // lc.block_len
    assert stats["tpf"] == pytest.approx(stats["committed"] / (stats["forwards"] * cfg.batch))


# ---------------------------------------------------------------------------
# the packet flow (update packets between layers, proxy drift per layer)
# ---------------------------------------------------------------------------

def _centroid_check(h, win, labels, sums, counts, cents, K):
    """GPU clustering of one sequence: labels are a nearest final centroid,
    counts and sums match the members."""
    hw = h[win]
    u = hw / np.linalg.norm(hw, axis=1, keepdims=True)
    cos = u @ cents.T
    lab = labels[win]
    assert np.all(cos[np.arange(len(win)), lab] >= cos.max(axis=1) - 1e-5)
    for k in range(K):
        m = hw[lab == k]
        assert counts[k] == len(m)
        np.testing.assert_allclose(sums[k], m.sum(axis=0), rtol=1e-5, atol=1e-5 * max(1.0, np.abs(m).max(initial=0)))
    assert np.all(labels[np.setdiff1d(np.arange(len(labels)), win)] == -1)


def _check_codes(fmt, X, means, labels, rows, gcodes, gscales):
    """Codes and scales of the listed rows of one sequence, bit-exact."""
    rows = [int(p) for p in rows]
    if not rows:
        return
    d = X.shape[1]
    mrows = np.stack([means[labels[p]] if labels[p] >= 0 else np.zeros(d, np.float32) for p in rows])
    c, e = cr.encode(X[rows], mrows, fmt)
    pc, pe = cr.pack(c, e, fmt)
    assert np.array_equal(gcodes[rows], pc) and np.array_equal(gscales[rows], pe), "codes differ"


def replay_packets(events, cfg, lc, ow):
    """The packet flow's own events against the oracle: clustering at block
    entry, the patch, proxy drift and selection, the packet rows, the commit
    drift and the suffix commit.  Returns the number of layer steps checked."""
    from oracle import proxy_ref as pr
    shape = mr.Shape(cfg.n_layers, cfg.d, cfg.n_heads, cfg.head_dim, cfg.ffn, cfg.vocab, cfg.seq, cfg.dtype)
    K, H = lc.n_clusters, cfg.n_heads
    n = 0
    last_pout = {}
    for ev in events:
        if ev["event"] == "cluster":
            h = dec(ev["h"])
            lab, sums, cnts, cents = (from_dev(ev[k]) for k in ("labels", "sums", "counts", "centroids"))
            for s in range(cfg.batch):
                _centroid_check(h[s], ev["win"], lab[s], sums[s], cnts[s], cents[s], K)
            if "codes" in ev:                 # the window's inputs encoded against the cluster means
                X, gm = from_dev(ev["X"]), from_dev(ev["means"])
                gcodes, gscales = from_dev(ev["codes"]), from_dev(ev["scales"])
                for s in range(cfg.batch):
                    np.testing.assert_allclose(gm[s], cr.cluster_means(X[s].astype(np.float64), lab[s], K),
                                               rtol=1e-5, atol=1e-6)
                    _check_codes(lc.codec, X[s], gm[s], lab[s], ev["win"], gcodes[s], gscales[s])
            want = pr.proxy_scores(pr.proxy_tokens(sums, cnts, "bf16"), ow["layers"][ev["layer"]]["w_q"],
                                   dec(ev["k"]), H, "bf16")
            assert_rows_close(from_dev(ev["pscores"]), want, 4e-3, "entry proxy scores")   # bf16 queries
        elif ev["event"] == "packet_layer":
            li = ev["layer"]
            w = ow["layers"][li]
            bf = ev["before"]
            labels = from_dev(bf["labels"]).astype(np.int64)
            counts = from_dev(bf["counts"]).astype(np.int64)
            pl = mr.PacketLayer(mr.LayerState(dec(bf["k"]), dec(bf["v"]), dec(bf["h"])),
                                from_dev(bf["X"]).astype(np.float64), labels,
                                from_dev(bf["sums"]).astype(np.float64), counts, from_dev(bf["pscores"]))
            if ev["pin"] is not None:
                idx, cnt, xin = (from_dev(t) for t in ev["pin"])
                rows = [list(idx[s, :cnt[s]]) for s in range(cfg.batch)]
                xs = [xin[s, :cnt[s]].astype(np.float64) for s in range(cfg.batch)]
                want = mr.patch(pl, rows, xs, w, shape)
                got = ev["patched"]
                np.testing.assert_array_equal(from_dev(got["X"]), want.x.astype(np.float32))
                for nm, a in (("k", want.st.k), ("v", want.st.v), ("h", want.st.h)):
                    assert_rows_close(dec(got[nm]), a, 2e-2, f"patched {nm}")
                # the sums move by the GPU's own new rows (whose bf16 rounding may
                # differ from the oracle's by an ulp; the rows are checked above)
                gh = dec(got["h"])
                wsums = from_dev(bf["sums"]).astype(np.float64)
                for s in range(cfg.batch):
                    for p in rows[s]:
                        if labels[s, p] >= 0:
                            wsums[s, labels[s, p]] += gh[s, p] - pl.st.h[s, p]
                np.testing.assert_allclose(from_dev(got["sums"]), wsums, rtol=1e-5, atol=1e-5 * np.abs(wsums).max())
                if "codes" in got:             # patched rows re-encoded against the block's means
                    X, gm = from_dev(got["X"]), from_dev(got["means"])
                    for s in range(cfg.batch):
                        _check_codes(lc.codec, X[s], gm[s], labels[s], rows[s], from_dev(got["codes"])[s],
                                     from_dev(got["scales"])[s])
            if ev["refresh"]:
                pr_ = ev["proxy"]
                sums = from_dev(pr_["sums"]).astype(np.float64)
                sc = pr.proxy_scores(pr.proxy_tokens(sums, counts, "bf16"), w["w_q"], dec(pr_["k"]), H, "bf16")
                # the proxy queries are rounded to bf16 on both sides from fp32 / fp64
                # arithmetic: an element can differ by an ulp, so the scores are
                # compared per (cluster, head) row at a bf16-derived tolerance, and
                # the drift is the KL of the GPU's own current and previous scores
                gsc = from_dev(pr_["pscores"])
                assert_rows_close(gsc, sc, 4e-3, "proxy scores")
                gd = from_dev(pr_["pdrift"])
                np.testing.assert_allclose(gd, pr.proxy_kl(gsc, from_dev(bf["pscores"])), rtol=2e-3, atol=1e-6)
                sel = pr.select_clusters(gd, lc.k_top)
                widx, wcnt = pr.cluster_members(labels, sel)
                oidx, ocnt, ox = (from_dev(t) for t in ev["pout"])
                assert np.array_equal(ocnt, wcnt)
                for s in range(cfg.batch):
                    assert np.array_equal(oidx[s, :ocnt[s]], widx[s, :wcnt[s]])
                rows = [list(oidx[s, :ocnt[s]]) for s in range(cfg.batch)]
                codec = None
                if pr_["codes"] is not None:   # the packet rows start from the GPU's codes, decoded
                    c, e = cr.unpack(from_dev(pr_["codes"]), from_dev(pr_["scales"]), lc.codec)
                    codec = dict(fmt=lc.codec, codes=c, exps=e, means=from_dev(pr_["means"]).astype(np.float64))
                cur = mr.PacketLayer(mr.LayerState(dec(pr_["k"]), dec(pr_["v"]), pl.st.h),
                                     from_dev(pr_["X"]).astype(np.float64), labels, sums, counts, sc, codec)
                out = mr.sparse_forward(cur, rows, w, shape)
                for s in range(cfg.batch):
                    assert_rows_close(ox[s, :ocnt[s]], out[s], 2e-2, "packet rows")
                last_pout[ev["forward"]] = (oidx, ocnt, ox)
            if "att" in ev:                   # the commit drift of the block's queries, last layer
                at = ev["att"]
                s1 = pr.query_scores(dec(at["q"]), dec(at["k"]))
                np.testing.assert_allclose(from_dev(at["scores_out"]), s1, rtol=1e-4, atol=1e-4 * np.abs(s1).max())
                np.testing.assert_allclose(from_dev(at["delta"]), pr.attention_drift(s1, from_dev(at["scores_in"])),
                                           rtol=2e-3, atol=1e-6)
            n += 1
        elif ev["event"] == "packet_suffix":
            gconf = from_dev(ev["conf"])
            el = from_dev(ev["eligible"]).astype(bool)
            masked = from_dev(ev["masked"]).astype(bool)
            oidx, ocnt, _ = last_pout[ev["forward"]]
            for s in range(cfg.batch):     # the last packet's rows in the suffix window, in order
                assert ev["positions"][s] == [int(p) for p in oidx[s, :ocnt[s]] if ev["be"] <= p < ev["hi"]]
                assert el[s].sum() == len(ev["positions"][s])
            if ev["logits"] is not None:
                xs = from_dev(ev["x"]).astype(np.float64)
                lg = ref.decode(from_dev(ev["logits"]), "bf16")
                for s in range(cfg.batch):
                    m = int(el[s].sum())
                    if m:
                        assert_rows_close(lg[s, :m], mr.logits(xs[s:s + 1, :m], ow["w_lm"], "bf16")[0], 2e-2, "suffix")
                tok, conf = ref.confidence(lg, cfg.vocab - 1)
                np.testing.assert_allclose(gconf[el], conf[el], rtol=1e-4)
            assert np.array_equal(from_dev(ev["commit"]).astype(bool), ref.suffix_commit_rule(gconf, masked, el, lc.tau_s))
    return n


def test_tiny_packet_stack_replay(P):
    cfg, lc, ow, y, stats, events = run_stack(P, 42, flow="packet")
    assert not (y == cfg.vocab - 1).any()
    assert np.array_equal(y[:, :cfg.prompt_len], inputs.stack_prompt(cfg))
    assert stats["committed"] == cfg.batch * cfg.gen_len
    assert stats["refreshing_steps"] > 0
    n = replay_packets(events, cfg, lc, ow)
    assert n == cfg.n_layers * (stats["refreshing_steps"] + stats["plain_steps"])
    # the block forwards and the decisions through the common replay
    assert replay(events, cfg, lc, ow) > 0


@pytest.mark.parametrize("codec", ["mxfp4", "mxfp8"])
def test_tiny_packet_stack_with_codec_replay(P, codec):
    cfg, lc, ow, y, stats, events = run_stack(P, 42, flow="packet", codec=codec)
    assert not (y == cfg.vocab - 1).any()
    assert stats["committed"] == cfg.batch * cfg.gen_len
    n = replay_packets(events, cfg, lc, ow)
    assert n == cfg.n_layers * (stats["refreshing_steps"] + stats["plain_steps"])
    assert replay(events, cfg, lc, ow) > 0
