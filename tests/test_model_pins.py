"""Pins of the whole-stack loop oracle (oracle/model_ref.py): closed forms of
its pieces, a brute-force layer written from the definitions with plain
loops, cache-consistency invariants of the sparse forwards, the schedule
rules and invariants of the free-running loop.  CPU only."""

import math

import numpy as np
import pytest

from oracle import model_ref as mr
from oracle import polestar_ref as ref
from oracle import proxy_ref as pr


def rand_weights(shape: mr.Shape, seed=0, std=0.3, lm_std=None):
    g = np.random.default_rng(seed)
    hdim = shape.n_heads * shape.head_dim

    def w(*s, sd=std):
        return ref.round_to(g.standard_normal(s) * sd, shape.dtype)

    layers = [dict(w_q=w(hdim, shape.d), w_k=w(hdim, shape.d), w_v=w(hdim, shape.d), w_o=w(shape.d, hdim),
                   w_gu=w(2 * shape.ffn, shape.d), w_down=w(shape.d, shape.ffn)) for _ in range(shape.n_layers)]
    return dict(tok_emb=w(shape.vocab, shape.d, sd=1.0), pos_emb=w(shape.seq, shape.d, sd=1.0), layers=layers,
                w_lm=w(shape.vocab, shape.d, sd=lm_std or std))


def empty_state(b, shape):
    return mr.LayerState(np.zeros((b, shape.seq, shape.n_heads, shape.head_dim)),
                         np.zeros((b, shape.seq, shape.n_heads, shape.head_dim)),
                         np.zeros((b, shape.seq, shape.d)))


def test_rmsnorm_and_silu_closed_forms():
    x = np.array([[3.0, 4.0]])
    assert np.allclose(mr.rmsnorm(x, eps=0.0), x / math.sqrt(12.5), rtol=1e-15)
    assert np.allclose(mr.rmsnorm(x), x / math.sqrt(12.5 + 1e-5), rtol=1e-15)
    assert mr.silu(np.array(0.0)) == 0.0
    assert mr.silu(np.array(math.log(3.0))) == pytest.approx(math.log(3.0) * 0.75, rel=1e-15)
    assert mr.silu(np.array(-50.0)) == pytest.approx(0.0, abs=1e-18)


def brute_layer_row(x_all, i, w, shape):
    """Row i of a full-sequence layer forward, from M-1..M-5 with plain loops
    (one sequence, fp64 throughout, rounding applied at the same points)."""
    S, d = len(x_all), shape.d
    H, hd, F = shape.n_heads, shape.head_dim, shape.ffn
    rnd = lambda v: float(ref.round_to(np.array(v), shape.dtype))

    def norm(vec):
        ms = sum(t * t for t in vec) / len(vec)
        return [rnd(t / math.sqrt(ms + mr.EPS)) for t in vec]

    def mat(wm, vec):
        return [sum(wm[r][c] * vec[c] for c in range(len(vec))) for r in range(len(wm))]

    h = [norm(list(x_all[j])) for j in range(S)]
    q = [rnd(t) for t in mat(w["w_q"], h[i])]
    keys = [[rnd(t) for t in mat(w["w_k"], h[j])] for j in range(S)]
    vals = [[rnd(t) for t in mat(w["w_v"], h[j])] for j in range(S)]
    o = []
    for hh in range(H):
        sl = slice(hh * hd, (hh + 1) * hd)
        sc = [sum(a * b for a, b in zip(q[sl], keys[j][sl])) / math.sqrt(hd) for j in range(S)]
        m = max(sc)
        e = [math.exp(s - m) for s in sc]
        z = sum(e)
        o += [rnd(sum(e[j] / z * vals[j][sl][c] for j in range(S))) for c in range(hd)]
    x = [x_all[i][c] + rnd(t) for c, t in enumerate(mat(w["w_o"], o))]
    g = norm(x)
    gu = [rnd(t) for t in mat(w["w_gu"], g)]
    a = [rnd(gu[f] / (1 + math.exp(-gu[f])) * gu[F + f]) for f in range(F)]
    return [x[c] + rnd(t) for c, t in enumerate(mat(w["w_down"], a))]


def test_embed_places_token_and_position_rows():
    """M-3: row r of sequence b is tok_emb[ids[b][lo + r]] + pos_emb[lo + r].
    Token v is encoded as v in channel 0 and position p as p in channel 1, so
    each output row reads back its (id, absolute position); a position table
    indexed from 0 instead of lo, or ids taken from the wrong offset, fail."""
    vocab, seq, d = 50, 12, 4
    tok = np.zeros((vocab, d))
    tok[:, 0] = np.arange(vocab)
    pos = np.zeros((seq, d))
    pos[:, 1] = np.arange(seq)
    ids = np.array([[3, 9, 14, 7, 1, 0, 22, 31, 45, 2, 8, 11],
                    [40, 41, 42, 43, 44, 45, 46, 47, 48, 49, 5, 6]])
    x = mr.embed(tok, pos, ids, 5, 9)
    assert x.shape == (2, 4, d)
    for b in range(2):
        for r in range(4):
            assert x[b, r].tolist() == [ids[b, 5 + r], 5 + r, 0.0, 0.0]


def test_logits_normalise_then_project():
    """M-6: logits = W_lm RMSNorm(x).  For x = c e_j (c > 0), RMSNorm gives
    e_j sqrt(d) / sqrt(1 + eps d / c^2), so the logits are that factor times
    column j of W_lm: independent of c up to eps (a dropped RMSNorm scales
    with c), and a column, not a row (a transposed W_lm reads row j)."""
    g = np.random.default_rng(15)
    d = 16
    w_lm = g.standard_normal((d, d))
    for c in (0.5, 3.0, 40.0):
        x = np.zeros((1, 1, d))
        x[0, 0, 9] = c
        got = mr.logits(x, w_lm, "fp32")[0, 0]
        scale = math.sqrt(d) / math.sqrt(1.0 + mr.EPS * d / (c * c))
        np.testing.assert_allclose(got, scale * w_lm[:, 9], rtol=1e-6)
    assert not np.allclose(got, scale * w_lm[9, :], rtol=1e-2)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_layer_matches_brute_force(dtype):
    shape = mr.Shape(n_layers=1, d=8, n_heads=2, head_dim=4, ffn=6, vocab=16, seq=5, dtype=dtype)
    wts = rand_weights(shape, seed=3)
    g = np.random.default_rng(4)
    x = g.standard_normal((1, shape.seq, shape.d))
    r = mr.layer_forward(x, 0, wts["layers"][0], empty_state(1, shape), mode="all", block=(0, shape.seq),
                         shape=shape)
    for i in range(shape.seq):
        want = brute_layer_row(x[0], i, wts["layers"][0], shape)
        np.testing.assert_allclose(r["x_out"][0, i], want, rtol=1e-9, atol=1e-12)


def test_zero_output_projections_leave_the_residual():
    shape = mr.Shape(n_layers=1, d=16, n_heads=2, head_dim=8, ffn=12, vocab=16, seq=6)
    wts = rand_weights(shape)
    w = dict(wts["layers"][0], w_o=np.zeros_like(wts["layers"][0]["w_o"]),
             w_down=np.zeros_like(wts["layers"][0]["w_down"]))
    x = np.random.default_rng(1).standard_normal((2, shape.seq, shape.d))
    r = mr.layer_forward(x, 0, w, empty_state(2, shape), mode="all", block=(0, shape.seq), shape=shape)
    assert np.array_equal(r["x_out"], x)


def _full_then(shape, mode, lo, hi, bs, bl, seed=5):
    """Full forward of a sequence, then a forward of rows [lo, hi) in `mode`
    against the cache it left, with the same inputs."""
    wts = rand_weights(shape, seed=seed)
    g = np.random.default_rng(seed + 1)
    x = g.standard_normal((2, shape.seq, shape.d))
    full = mr.layer_forward(x, 0, wts["layers"][0], empty_state(2, shape), mode="all", block=(bs, bl),
                            shape=shape)
    part = mr.layer_forward(x[:, lo:hi], lo, wts["layers"][0], full["state"], mode=mode, block=(bs, bl),
                            shape=shape, k_top=3)
    return full, part


@pytest.mark.parametrize("mode,lo,hi", [("all", 3, 15), ("refresh", 3, 15), ("plain", 8, 12)])
def test_sparse_forward_against_a_consistent_cache_reproduces_the_full_forward(mode, lo, hi):
    shape = mr.Shape(n_layers=1, d=16, n_heads=2, head_dim=8, ffn=12, vocab=16, seq=20)
    full, part = _full_then(shape, mode, lo, hi, 8, 4)
    np.testing.assert_array_equal(part["x_out"], full["x_out"][:, lo:hi])
    for a, b in ((part["state"].k, full["state"].k), (part["state"].v, full["state"].v),
                 (part["state"].h, full["state"].h)):
        np.testing.assert_array_equal(a, b)
    assert np.all(part["drift"] == 0.0)           # unchanged hidden states: zero drift


def test_refresh_mode_selects_from_the_window_only_and_rewrites_what_it_selects():
    shape = mr.Shape(n_layers=1, d=16, n_heads=2, head_dim=8, ffn=12, vocab=16, seq=20)
    wts = rand_weights(shape, seed=7)
    g = np.random.default_rng(8)
    x = g.standard_normal((1, shape.seq, shape.d))
    full = mr.layer_forward(x, 0, wts["layers"][0], empty_state(1, shape), mode="all", block=(8, 4),
                            shape=shape)
    x2 = x.copy()
    x2[0, [4, 6, 13]] += 3.0 * g.standard_normal((3, shape.d))     # perturb three window rows
    x2[0, 1] += 5.0                                                # and one outside the window
    r = mr.layer_forward(x2[:, 3:15], 3, wts["layers"][0], full["state"], mode="refresh", block=(8, 4),
                         shape=shape, k_top=3)
    assert r["stale_idx"][0].tolist() == [4, 6, 13] and r["stale_count"][0] == 3
    h_new = ref.round_to(mr.rmsnorm(x2[0]), shape.dtype)
    for p in (4, 6, 13, 8, 9, 10, 11):
        assert np.array_equal(r["state"].h[0, p], h_new[p])
    for p in (1, 3, 5, 7, 12, 14):
        assert np.array_equal(r["state"].h[0, p], full["state"].h[0, p])   # not refreshed


def test_window_and_schedule_rules():
    assert mr.block_bounds(512, 32, 0) == (512, 544)
    assert mr.window(512, 32, 768, 0, 64, 32) == (448, 576)
    assert mr.window(512, 32, 768, 7, 64, 32) == (672, 768)            # last block: no suffix
    assert mr.window(8, 32, 72, 0, 64, 32) == (0, 72)                  # clipped at both ends
    assert mr.window_top_k(448, 576, 32) == 48
    assert mr.window_top_k(672, 768, 32) == 32
    assert not mr.refreshes(3, 3) and mr.refreshes(4, 3) and mr.refreshes(1, 0)


def test_free_running_loop_invariants():
    shape = mr.Shape(n_layers=2, d=32, n_heads=2, head_dim=16, ffn=48, vocab=48, seq=40)
    wts = rand_weights(shape, seed=11, lm_std=0.6)
    g = np.random.default_rng(12)
    prompt = g.integers(0, shape.vocab - 1, size=(2, 8))
    p = mr.LoopParams(prompt_len=8, gen_len=32, block_len=8, prefix=16, suffix=8, tau_upd=1, h=2)
    y, tr = mr.generate(wts, prompt, shape, p)
    assert not (y == shape.mask_id).any()
    assert np.array_equal(y[:, :8], prompt)
    assert tr.committed == 2 * 32
    kinds = [f["kind"] for f in tr.forwards]
    entries = [f for f in tr.forwards if f["kind"].startswith("entry")]
    assert [e["kind"] for e in entries] == ["entry_full", "entry_window"] * 2
    assert kinds[0] == "entry_full"
    # schedule: a step refreshes iff more than tau_upd tokens were committed
    # since the last refreshing forward (entries included)
    since = None
    for f in tr.forwards:
        n = f["commit"].sum(axis=1) + (0 if f.get("suffix_commit") is None else f["suffix_commit"].sum(axis=1))
        if f["kind"].startswith("entry"):
            since = n
            continue
        # per-sequence counts; the batch refreshes when any sequence would
        assert (f["kind"] == "refresh") == mr.refreshes(int(since.max()), p.tau_upd)
        since = n if f["kind"] == "refresh" else since + n
        # force_one: every within-block step commits at least one token per unfinished sequence
        assert f["commit"].any(axis=1).sum() >= 1
    assert len(tr.forwards) < 2 * 32                 # some steps commit several tokens


# ---------------------------------------------------------------------------
# the update-packet flow (Alg. 1 per-layer loop)
# ---------------------------------------------------------------------------

def _packet_layer_from_full(shape, seed, lo, bs, be, hi, K=2):
    wts = rand_weights(shape, seed=seed)
    g = np.random.default_rng(seed + 1)
    x = g.standard_normal((1, shape.seq, shape.d))
    full = mr.layer_forward(x, 0, wts["layers"][0], empty_state(1, shape), mode="all", block=(bs, be - bs),
                            shape=shape)
    win = mr._window_positions(lo, bs, be, hi)
    labels, sums, counts = mr.cluster_layer(full["state"].h, win, K, 10)
    pl = mr.PacketLayer(full["state"], x.copy(), labels, sums, counts,
                        np.zeros((1, K, shape.n_heads, shape.seq)))
    return wts["layers"][0], x, full, pl


def test_packet_rows_forward_against_a_consistent_cache_reproduces_the_full_forward():
    shape = mr.Shape(n_layers=1, d=16, n_heads=2, head_dim=8, ffn=12, vocab=16, seq=20)
    w, x, full, pl = _packet_layer_from_full(shape, 21, 2, 8, 12, 16)
    rows = [[3, 9, 14, 17]]
    out = mr.sparse_forward(pl, rows, w, shape)
    np.testing.assert_array_equal(out[0], full["x_out"][0, rows[0]])


def test_patch_with_unchanged_inputs_changes_nothing_and_sums_track_the_window():
    shape = mr.Shape(n_layers=1, d=16, n_heads=2, head_dim=8, ffn=12, vocab=16, seq=20)
    w, x, full, pl = _packet_layer_from_full(shape, 23, 2, 8, 12, 16)
    same = mr.patch(pl, [[3, 13]], [x[0, [3, 13]]], w, shape)
    for a, b in ((same.st.k, pl.st.k), (same.st.v, pl.st.v), (same.st.h, pl.st.h), (same.x, pl.x), (same.sums, pl.sums)):
        np.testing.assert_array_equal(a, b)
    g = np.random.default_rng(5)
    new = x[0, [3, 13]] + g.standard_normal((2, shape.d))
    pt = mr.patch(pl, [[3, 13]], [new], w, shape)
    win = mr._window_positions(2, 8, 12, 16)
    lab_w = pl.labels[0, win]
    want, _ = pr.cluster_sums(pt.st.h[0, win], lab_w, 2)
    np.testing.assert_allclose(pt.sums[0], want, atol=1e-12)
    hn = ref.round_to(mr.rmsnorm(new), shape.dtype)
    np.testing.assert_array_equal(pt.st.h[0, [3, 13]], hn)
    np.testing.assert_array_equal(pt.st.k[0, 3].reshape(-1), ref.round_to(hn[0] @ w["w_k"].T, shape.dtype))


def test_proxy_select_with_unchanged_scores_picks_the_lowest_clusters():
    shape = mr.Shape(n_layers=1, d=16, n_heads=2, head_dim=8, ffn=12, vocab=16, seq=20)
    w, x, full, pl = _packet_layer_from_full(shape, 25, 2, 8, 12, 16, K=3)
    tok = pr.proxy_tokens(pl.sums, pl.counts, shape.dtype)
    pl.scores[:] = pr.proxy_scores(tok, w["w_q"], pl.st.k, shape.n_heads, shape.dtype)
    drift, rows, sc = mr.proxy_select(pl, w, shape, 2)
    assert np.all(drift == 0.0)
    members = sorted(int(p) for p in np.flatnonzero((pl.labels[0] == 0) | (pl.labels[0] == 1)))
    assert rows[0] == members


def test_packet_flow_selecting_every_cluster_equals_the_window_flow():
    # with every window row in every packet, a refreshing step of the packet
    # flow computes what the window flow's full-window forward does; drift
    # commits are off (their deltas are measured differently), so both loops
    # must decode the same tokens through the same forwards
    shape = mr.Shape(n_layers=2, d=32, n_heads=2, head_dim=16, ffn=48, vocab=48, seq=40)
    wts = rand_weights(shape, seed=31, lm_std=0.6)
    prompt = np.random.default_rng(32).integers(0, shape.vocab - 1, size=(2, 8))
    common = dict(prompt_len=8, gen_len=32, block_len=8, prefix=16, suffix=8, tau_upd=1, h=2, alpha=1e9)
    y1, t1 = mr.generate(wts, prompt, shape, mr.LoopParams(window_frac=1.0, **common))
    y2, t2 = mr.generate_packets(wts, prompt, shape, mr.LoopParams(**common), n_clusters=3, k_top=3)
    assert [f["kind"] for f in t1.forwards] == [f["kind"] for f in t2.forwards]
    assert np.array_equal(y1, y2)
    assert any(f["kind"] == "refresh" for f in t2.forwards)
    assert any(f.get("suffix_commit") is not None and f["suffix_commit"].any() for f in t2.forwards)


def test_packet_flow_loop_invariants():
    shape = mr.Shape(n_layers=2, d=32, n_heads=2, head_dim=16, ffn=48, vocab=48, seq=40)
    wts = rand_weights(shape, seed=11, lm_std=0.6)
    prompt = np.random.default_rng(12).integers(0, shape.vocab - 1, size=(2, 8))
    p = mr.LoopParams(prompt_len=8, gen_len=32, block_len=8, prefix=16, suffix=8, tau_upd=1, h=2)
    y, tr = mr.generate_packets(wts, prompt, shape, p, n_clusters=4, k_top=2)
    assert not (y == shape.mask_id).any() and np.array_equal(y[:, :8], prompt)
    assert tr.committed == 2 * 32
    assert [f["kind"] for f in tr.forwards if f["kind"].startswith("entry")] == ["entry_full", "entry_window"] * 2
    # D = KL(P(t) || P(t-1)): every refreshing step's drift is taken against the
    # proxy scores of the previous refreshing step of the same block
    prev = None
    n_checked = 0
    for f in tr.forwards:
        if f["kind"].startswith("entry"):
            prev = None
        elif f["kind"] == "refresh":
            if prev is not None:
                for li, (d, sc) in enumerate(f["proxy"]):
                    np.testing.assert_allclose(d, pr.proxy_kl(sc, prev[li][1]), rtol=1e-12, atol=1e-15)
                    n_checked += 1
            prev = f["proxy"]
    assert n_checked > 0


def test_codec_packet_rows_start_from_the_decoded_inputs():
    # with the codec on, a packet's forward equals the codec-free forward of
    # the decoded inputs; a patch re-encodes exactly the patched rows
    from oracle import codec_ref as cr
    shape = mr.Shape(n_layers=1, d=64, n_heads=2, head_dim=32, ffn=64, vocab=16, seq=20)
    w, x, full, pl = _packet_layer_from_full(shape, 41, 2, 8, 12, 16)
    win = mr._window_positions(2, 8, 12, 16)
    means = cr.cluster_means(pl.x[0], pl.labels[0], 2)[None]
    cd = dict(fmt="mxfp4", codes=np.zeros((1, 20, 64), np.int64), exps=np.zeros((1, 20, 2), np.int64), means=means)
    pc = mr.PacketLayer(pl.st, pl.x, pl.labels, pl.sums, pl.counts, pl.scores, mr.encode_rows(cd, pl.x, pl.labels, [win]))
    rows = [[3, 13, 15]]
    dec = mr.decoded_rows(pc, 0, rows[0])
    assert np.abs(dec - pl.x[0, rows[0]]).max() > 0                     # lossy
    plain = mr.PacketLayer(pl.st, pl.x.copy(), pl.labels, pl.sums, pl.counts, pl.scores)
    plain.x[0, rows[0]] = dec
    np.testing.assert_array_equal(mr.sparse_forward(pc, rows, w, shape)[0], mr.sparse_forward(plain, rows, w, shape)[0])
    new = x[0, [13]] + 0.5
    pt = mr.patch(pc, [[13]], [new], w, shape)
    c, e = cr.encode(new, means[0, [pc.labels[0, 13]]], "mxfp4")
    assert np.array_equal(pt.codec["codes"][0, 13], c[0]) and np.array_equal(pt.codec["exps"][0, 13], e[0])
    untouched = [p for p in win if p != 13]
    assert np.array_equal(pt.codec["codes"][0, untouched], pc.codec["codes"][0, untouched])


def test_packet_flow_with_codec_runs_to_completion():
    shape = mr.Shape(n_layers=2, d=64, n_heads=2, head_dim=32, ffn=64, vocab=48, seq=40)
    wts = rand_weights(shape, seed=13, lm_std=0.6)
    prompt = np.random.default_rng(14).integers(0, shape.vocab - 1, size=(1, 8))
    p = mr.LoopParams(prompt_len=8, gen_len=32, block_len=8, prefix=16, suffix=8, tau_upd=1, h=2)
    for fmt in ("mxfp4", "mxfp8"):
        y, tr = mr.generate_packets(wts, prompt, shape, p, n_clusters=3, k_top=2, codec=fmt)
        assert not (y == shape.mask_id).any() and tr.committed == 32
