"""Pins of the CPU oracle against what the paper and the mathematics fix.

These tests run on the CPU only.  Each one ties an oracle function to a fact
that does not come from the oracle itself: a hand-derived closed form
(tests/golden/closed_forms.json), an inequality or identity of the theory
(App. B: Proposition 1, Corollary 1, Proposition 2 / Pinsker), an invariance,
a special case, or the independent pure-Python path in `oracle.brute`.
"""

import math

import numpy as np
import pytest

from oracle import brute
from oracle import polestar_ref as ref
from paper_2607_14107_amd import inputs


def _expr(s):
    return eval(s, {"__builtins__": {}}, {"log": math.log, "sqrt": math.sqrt})


def _cfg0():
    cfg = inputs.CONFIGS[0]
    x = inputs.layer_inputs(cfg, 0)
    dec = {k: ref.decode(x[k], cfg.dtype) for k in ("h_prev", "h_cur", "w_q", "w_k", "w_v")}
    return cfg, x, dec


# --------------------------------------------------------------------------
# Step 1 -- drift
# --------------------------------------------------------------------------

def test_drift_closed_forms(golden):
    for name in ("kl_two_point", "kl_three_point"):
        g = golden[name]
        d = ref.drift(np.array([[g["h_cur"]]]), np.array([[g["h_prev"]]]))[0, 0]
        assert d == pytest.approx(_expr(g["expect"]), rel=1e-13)
    g = golden["kl_two_point"]
    rev = ref.drift(np.array([[g["h_prev"]]]), np.array([[g["h_cur"]]]))[0, 0]
    assert rev == pytest.approx(_expr(g["expect_reversed"]), rel=1e-13)
    # the direction matters: KL(p||q) != KL(q||p) here
    assert abs(rev - _expr(g["expect"])) > 1e-3


def test_drift_zero_on_identical_rows():
    g = np.random.default_rng(1)
    h = g.standard_normal((2, 7, 33))
    d = ref.drift(h, h.copy())
    assert np.all(d == 0.0)


def test_drift_nonnegative_and_shift_invariant():
    g = np.random.default_rng(2)
    a = g.standard_normal((3, 11, 64)) * 2
    b = g.standard_normal((3, 11, 64)) * 2
    d = ref.drift(a, b)
    assert np.all(d >= 0.0)
    # softmax is invariant to a per-row shift, so the drift is too
    shift = g.standard_normal((3, 11, 1)) * 5
    np.testing.assert_allclose(ref.drift(a + shift, b - shift), d, rtol=1e-10)


def test_drift_second_order_expansion():
    """For a small change delta = a - b, KL(p||q) = Var_p(delta)/2 + O(|delta|^3)."""
    g = np.random.default_rng(3)
    b = g.standard_normal((1, 20, 512))
    delta = g.standard_normal((1, 20, 512)) * 1e-3
    a = b + delta
    p = np.exp(ref.log_softmax(a))
    mean = np.sum(p * delta, axis=-1)
    var = np.sum(p * delta * delta, axis=-1) - mean ** 2
    np.testing.assert_allclose(ref.drift(a, b), 0.5 * var, rtol=1e-2)


def test_drift_pinsker_bound():
    """Prop. 2 rests on Pinsker: ||p - q||_1 <= sqrt(2 KL(p||q))."""
    g = np.random.default_rng(4)
    a = g.standard_normal((4, 30, 40)) * 1.5
    b = a + g.standard_normal((4, 30, 40)) * g.uniform(0.01, 1.0, size=(4, 30, 1))
    p = np.exp(ref.log_softmax(a))
    q = np.exp(ref.log_softmax(b))
    l1 = np.abs(p - q).sum(axis=-1)
    assert np.all(l1 <= np.sqrt(2 * ref.drift(a, b)) + 1e-12)


@pytest.mark.parametrize("delta", [100.0, -100.0, 1000.0, -1000.0, 1e-3])
def test_drift_one_channel_moved_closed_form(delta):
    """a = b + delta * e_c moves one channel.  With q = softmax(b), softmax(a)
    is q with q_c scaled by e^delta and renormalised, so
        KL(softmax(a) || q) = p_c * delta - log(1 - q_c + q_c e^delta),
    p_c = q_c e^delta / (1 - q_c + q_c e^delta); evaluated here through
    logaddexp so that e^1000 never forms.  Large moves of one channel (an
    outlier in the hidden state) must give this finite value."""
    g = np.random.default_rng(31)
    b = g.standard_normal((1, 6, 96)) * 2.0
    for c in (0, 17, int(np.argmax(b[0, 0]))):
        a = b.copy()
        a[..., c] += delta
        qc = np.exp(b[..., c] - np.log(np.sum(np.exp(b), axis=-1)))
        # log(1 - q_c + q_c e^delta) = logaddexp(log(1 - q_c), log(q_c) + delta)
        lz = np.logaddexp(np.log1p(-qc), np.log(qc) + delta)
        pc = np.exp(np.log(qc) + delta - lz)
        want = pc * delta - lz
        got = ref.drift(a, b)
        assert np.all(np.isfinite(got))
        np.testing.assert_allclose(got, want, rtol=1e-9, atol=1e-12)


def test_drift_matches_pure_python_on_tiny_config():
    cfg, x, dec = _cfg0()
    got = ref.drift(dec["h_cur"], dec["h_prev"])
    want = np.array(brute.drift(dec["h_cur"].tolist(), dec["h_prev"].tolist()))
    np.testing.assert_allclose(got, want, rtol=1e-9, atol=1e-15)


# --------------------------------------------------------------------------
# Step 2 -- select
# --------------------------------------------------------------------------

def test_select_matches_rank_count_with_ties():
    g = np.random.default_rng(5)
    vals = np.round(g.standard_normal((3, 57)), 1)          # many exact ties
    vals[0, 3] = -0.0
    vals[0, 4] = 0.0
    for k in (0, 1, 5, 13, 40, 57):
        idx, cnt = ref.select(vals, k, 20, 8)
        bidx, bcnt = brute.select(vals.tolist(), k, 20, 8)
        assert idx.tolist() == bidx
        assert cnt.tolist() == bcnt


def test_select_structure():
    g = np.random.default_rng(6)
    vals = g.standard_normal((2, 40))
    idx, cnt = ref.select(vals, 10, 30, 10)
    for b in range(2):
        chosen = idx[b, :cnt[b]]
        assert np.all(np.diff(chosen) > 0)                 # ascending
        assert np.all((chosen < 30) | (chosen >= 40))      # never the active block
        others = [i for i in range(30) if i not in chosen]
        assert vals[b, chosen].min() >= vals[b, others].max()
    # k = 0 -> empty; k beyond the candidates -> all of them, padded with -1
    idx0, cnt0 = ref.select(vals, 0, 30, 10)
    assert idx0.shape == (2, 0) and cnt0.tolist() == [0, 0]
    idx_all, cnt_all = ref.select(vals, 35, 30, 10)
    assert cnt_all.tolist() == [30, 30]
    assert idx_all[0, :30].tolist() == list(range(30)) and np.all(idx_all[:, 30:] == -1)
    # an eligibility mask narrows the candidates
    elig = np.zeros((2, 40), dtype=bool)
    elig[:, 5:9] = True
    idx_e, cnt_e = ref.select(vals, 10, 30, 10, elig)
    assert cnt_e.tolist() == [4, 4] and idx_e[0, :4].tolist() == [5, 6, 7, 8]


def test_select_recovers_planted_set_on_tiny_config():
    cfg, x, dec = _cfg0()
    d = ref.drift(dec["h_cur"], dec["h_prev"])
    idx, cnt = ref.select(d, x["k"], cfg.block_start, cfg.block_len)
    cached = np.ones(cfg.seq, dtype=bool)
    cached[cfg.block_start:cfg.block_start + cfg.block_len] = False
    planted = np.flatnonzero(x["planted"][0] & cached)
    assert idx[0, :cnt[0]].tolist() == planted.tolist()


def test_selection_agreement_with_paper_drift_and_staleness():
    """The criterion of the drift-policy ablation (Sec. 5.3): the selected
    positions should be the truly stale ones.  On the tiny workload the
    hidden-state drift, the paper's attention drift and the KV staleness E_i
    (App. C.2) all rank the planted positions on top."""
    cfg, x, dec = _cfg0()
    bs, bl = cfg.block_start, cfg.block_len
    cached = np.ones(cfg.seq, dtype=bool)
    cached[bs:bs + bl] = False
    planted = set(np.flatnonzero(x["planted"][0] & cached).tolist())
    k = len(planted)
    r2 = ref.drift(dec["h_cur"], dec["h_prev"])
    r1 = ref.drift_attention_exact(dec["h_cur"], dec["h_prev"], dec["w_q"], dec["w_k"],
                                   cfg.n_heads, cfg.n_kv_heads, cfg.head_dim)
    shape = (1, cfg.seq, cfg.n_kv_heads, cfg.head_dim)
    k_old = (dec["h_prev"] @ dec["w_k"].T).reshape(shape)
    v_old = (dec["h_prev"] @ dec["w_v"].T).reshape(shape)
    k_new = (dec["h_cur"] @ dec["w_k"].T).reshape(shape)
    v_new = (dec["h_cur"] @ dec["w_v"].T).reshape(shape)
    e = ref.staleness(k_old, v_old, k_new, v_new)
    for score in (r2, r1, e):
        idx, cnt = ref.select(score, k, bs, bl)
        assert set(idx[0, :cnt[0]].tolist()) == planted


def _sigmoid(x):
    return 1.0 / (1.0 + math.exp(-x))


def _bernoulli_kl(p, q):
    return p * math.log(p / q) + (1 - p) * math.log((1 - p) / (1 - q))


def test_drift_attention_exact_two_key_hand_case():
    """Two tokens, two heads of head_dim 2, W_q = W_k = I: head h of token i
    sees logits l_ij = x_i[h] . x_j[h] / sqrt(2) over the two keys, so its
    attention row is Bernoulli(sigmoid(l_i0 - l_i1)) and the drift of token i
    is the mean over heads of KL(Bernoulli(cur) || Bernoulli(prev)) (eq.
    drift, current || previous; heads averaged).  Worked by hand:
      prev x0 = (1,0 | 0,0), x1 = (0,1 | 0,0);  cur x0 = (2,0 | 1,0), x1 = (0,1 | 0,1)
      token 0: head 0 logits (4, 0)/sqrt2 vs (1, 0)/sqrt2, head 1 (1, 0)/sqrt2 vs (0, 0)
      token 1: head 0 (0, 1)/sqrt2 both steps, head 1 (0, 1)/sqrt2 vs (0, 0).
    A reversed KL, a missing 1/sqrt(d_h), or heads summed instead of averaged
    each change these values."""
    r2 = math.sqrt(2.0)
    prev = np.array([[[1.0, 0, 0, 0], [0, 1.0, 0, 0]]])
    cur = np.array([[[2.0, 0, 1.0, 0], [0, 1.0, 0, 1.0]]])
    eye = np.eye(4)
    got = ref.drift_attention_exact(cur, prev, eye, eye, 2, 2, 2)
    t0 = 0.5 * (_bernoulli_kl(_sigmoid(4 / r2), _sigmoid(1 / r2)) + _bernoulli_kl(_sigmoid(1 / r2), 0.5))
    t1 = 0.5 * (0.0 + _bernoulli_kl(_sigmoid(-1 / r2), 0.5))
    np.testing.assert_allclose(got, [[t0, t1]], rtol=1e-12)
    # the same hand case through the logits: l = x_i[h] . x_j[h] / sqrt(2)
    lg = ref.attention_logits(cur, eye, eye, 2, 2, 2)
    np.testing.assert_allclose(lg[0, 0], [[4 / r2, 0], [0, 1 / r2]], rtol=1e-14)
    np.testing.assert_allclose(lg[0, 1], [[1 / r2, 0], [0, 1 / r2]], rtol=1e-14)


def test_attention_logits_grouped_heads_share_their_kv_head():
    """GQA: with one KV head, both query heads read it, which equals MHA with
    that KV head's weights repeated; query head h uses rows h*d_h.. of W_q."""
    g = np.random.default_rng(14)
    h = g.standard_normal((1, 5, 6))
    w_q = g.standard_normal((2 * 3, 6))
    w_k = g.standard_normal((3, 6))
    gqa = ref.attention_logits(h, w_q, w_k, 2, 1, 3)
    mha = ref.attention_logits(h, w_q, np.vstack([w_k, w_k]), 2, 2, 3)
    np.testing.assert_allclose(gqa, mha, rtol=1e-14)
    q1 = h[0] @ w_q[3:6].T
    k = h[0] @ w_k.T
    np.testing.assert_allclose(gqa[0, 1], q1 @ k.T / math.sqrt(3), rtol=1e-12)


# --------------------------------------------------------------------------
# Step 3 -- sparse K/V refresh
# --------------------------------------------------------------------------

def _small_refresh_case(seed=7, batch=2, seq=12, d=10, kvh=2, hd=3):
    g = np.random.default_rng(seed)
    h = g.standard_normal((batch, seq, d))
    w_k = g.standard_normal((kvh * hd, d))
    w_v = g.standard_normal((kvh * hd, d))
    kc = g.standard_normal((batch, seq, kvh, hd))
    vc = g.standard_normal((batch, seq, kvh, hd))
    return h, w_k, w_v, kc, vc


def test_refresh_unit_vector_picks_weight_column():
    """K_r = W_K h_r: a unit hidden state e_j gives column j of W_K (a
    transposed weight would give row j instead)."""
    h, w_k, w_v, kc, vc = _small_refresh_case()
    h[:] = 0.0
    h[0, 2, 7] = 1.0
    idx = np.array([[2], [-1]], dtype=np.int32)
    cnt = np.array([1, 0], dtype=np.int32)
    k_new, v_new, rows = ref.refresh_kv(h, w_k, w_v, kc, vc, idx, cnt, 9, 0)
    assert rows == [[2], []]
    np.testing.assert_array_equal(k_new[0, 2].reshape(-1), w_k[:, 7])
    np.testing.assert_array_equal(v_new[0, 2].reshape(-1), w_v[:, 7])


def test_project_rows_is_w_times_h_on_a_square_weight():
    """project_rows(h, W, r) = W h_r (App. B setup: k = W_K x).  The weight
    is square, as W_K is on the LLaDA-8B layer (4096 x 4096), so a transposed
    product keeps every shape: a unit hidden state e_j must give column j of
    W, not row j; and the rows must agree with refresh_kv's."""
    g = np.random.default_rng(12)
    d = 8
    w = g.standard_normal((d, d))
    h = np.zeros((3, d))
    h[1, 5] = 1.0
    h[2] = g.standard_normal(d)
    got = ref.project_rows(h, w, [1, 2])
    np.testing.assert_array_equal(got[0], w[:, 5])
    assert not np.allclose(got[0], w[5, :])
    np.testing.assert_allclose(got[1], [sum(w[o, c] * h[2, c] for c in range(d)) for o in range(d)],
                               rtol=1e-12)
    kc = np.zeros((1, 3, 2, 4))
    idx = np.array([[1, 2]], dtype=np.int32)
    k_new, _, _ = ref.refresh_kv(h[None], w, w, kc, kc, idx, np.array([2], np.int32), 0, 0)
    np.testing.assert_array_equal(k_new[0, 1:].reshape(2, d), got)


def test_refresh_untouched_rows_and_empty_refresh():
    h, w_k, w_v, kc, vc = _small_refresh_case()
    idx = np.array([[1, 5, -1], [0, -1, -1]], dtype=np.int32)
    cnt = np.array([2, 1], dtype=np.int32)
    k_new, v_new, rows = ref.refresh_kv(h, w_k, w_v, kc, vc, idx, cnt, 8, 2)
    assert rows == [[1, 5, 8, 9], [0, 8, 9]]
    for b in range(2):
        keep = [i for i in range(12) if i not in rows[b]]
        np.testing.assert_array_equal(k_new[b, keep], kc[b, keep])
        np.testing.assert_array_equal(v_new[b, keep], vc[b, keep])
    # nothing stale and an empty block: the cache is left exactly as it was
    k0, v0, rows0 = ref.refresh_kv(h, w_k, w_v, kc, vc, idx, np.zeros(2, np.int32), 8, 0)
    assert rows0 == [[], []]
    np.testing.assert_array_equal(k0, kc)
    np.testing.assert_array_equal(v0, vc)


def test_refresh_is_linear_in_hidden_state():
    """Corollary 1: Delta K = W_K Delta H and Delta V = W_V Delta H."""
    h1, w_k, w_v, kc, vc = _small_refresh_case(8)
    h2 = np.random.default_rng(9).standard_normal(h1.shape)
    idx = np.array([[0, 3, 6], [2, 4, -1]], dtype=np.int32)
    cnt = np.array([3, 2], dtype=np.int32)
    zero = np.zeros_like(kc)
    ka, va, rows = ref.refresh_kv(h1, w_k, w_v, zero, zero, idx, cnt, 10, 2)
    kb, vb, _ = ref.refresh_kv(h2, w_k, w_v, zero, zero, idx, cnt, 10, 2)
    ks, vs, _ = ref.refresh_kv(h1 + 2.5 * h2, w_k, w_v, zero, zero, idx, cnt, 10, 2)
    np.testing.assert_allclose(ks, ka + 2.5 * kb, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(vs, va + 2.5 * vb, rtol=1e-12, atol=1e-12)


def test_refresh_change_obeys_corollary_bounds():
    """Corollary 1: sigma_min ||dH|| <= sqrt(||dK||^2 + ||dV||^2) <= ||[W_K;W_V]||_2 ||dH||."""
    h1, w_k, w_v, kc, vc = _small_refresh_case(10, d=4, kvh=2, hd=3)
    dh = np.random.default_rng(11).standard_normal(h1.shape)
    idx = np.tile(np.arange(12, dtype=np.int32), (2, 1))
    cnt = np.array([12, 12], dtype=np.int32)
    ka, va, _ = ref.refresh_kv(h1, w_k, w_v, kc, vc, idx, cnt, 0, 0)
    kb, vb, _ = ref.refresh_kv(h1 + dh, w_k, w_v, kc, vc, idx, cnt, 0, 0)
    sv = np.linalg.svd(np.vstack([w_k, w_v]), compute_uv=False)
    lhs = np.sqrt(((kb - ka) ** 2).sum(axis=(2, 3)) + ((vb - va) ** 2).sum(axis=(2, 3)))
    nh = np.linalg.norm(dh, axis=-1)
    assert np.all(lhs <= sv[0] * nh * (1 + 1e-12))
    assert np.all(lhs >= sv[-1] * nh * (1 - 1e-12))


def test_refresh_all_rows_matches_pure_python_projection():
    cfg, x, dec = _cfg0()
    seq = cfg.seq
    idx = np.arange(seq, dtype=np.int32)[None, :]
    cnt = np.array([seq], dtype=np.int32)
    zero = np.zeros((1, seq, cfg.n_kv_heads, cfg.head_dim))
    k_new, v_new, _ = ref.refresh_kv(dec["h_cur"], dec["w_k"], dec["w_v"], zero, zero,
                                     idx, cnt, cfg.block_start, cfg.block_len)
    wk, wv = dec["w_k"].tolist(), dec["w_v"].tolist()
    for r in (0, 17, 63, 64, 95):
        xr = dec["h_cur"][0, r].tolist()
        np.testing.assert_allclose(k_new[0, r].reshape(-1), brute.matvec(wk, xr), rtol=1e-10, atol=1e-13)
        np.testing.assert_allclose(v_new[0, r].reshape(-1), brute.matvec(wv, xr), rtol=1e-10, atol=1e-13)


# --------------------------------------------------------------------------
# Step 4 -- attention
# --------------------------------------------------------------------------

def test_attention_closed_form(golden):
    g = golden["attention_two_keys"]
    q = np.array(g["q"])[None, :, None, :]
    k = np.array(g["k"])[None, :, None, :]
    v = np.array(g["v"])[None, :, None, :]
    out, lse = ref.attend(q, k, v, scale=g["scale"])
    np.testing.assert_allclose(out[0, 0, 0], [_expr(e) for e in g["expect_out"]], rtol=1e-13)
    assert lse[0, 0, 0] == pytest.approx(_expr(g["expect_lse"]), rel=1e-13)


def test_attention_matches_pure_python_on_tiny_config():
    cfg, x, dec = _cfg0()
    g = np.random.default_rng(12)
    kc = g.standard_normal((1, cfg.seq, cfg.n_kv_heads, cfg.head_dim))
    vc = g.standard_normal((1, cfg.seq, cfg.n_kv_heads, cfg.head_dim))
    q = ref.q_project(dec["h_cur"], dec["w_q"], cfg.block_start, cfg.block_len,
                      cfg.n_heads, cfg.head_dim)
    out, lse = ref.attend(q, kc, vc)
    wq = dec["w_q"].tolist()
    for j in (0, 31):
        xr = dec["h_cur"][0, cfg.block_start + j].tolist()
        np.testing.assert_allclose(q[0, j].reshape(-1), brute.matvec(wq, xr), rtol=1e-10, atol=1e-13)
    for h in range(cfg.n_heads):
        o, l = brute.attention_head(q[0, :, h].tolist(), kc[0, :, h].tolist(), vc[0, :, h].tolist(),
                                    1.0 / math.sqrt(cfg.head_dim))
        np.testing.assert_allclose(out[0, :, h], o, rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(lse[0, h], l, rtol=1e-12)


def test_attention_key_order_invariance_and_special_cases():
    g = np.random.default_rng(13)
    q = g.standard_normal((2, 5, 4, 8))
    kc = g.standard_normal((2, 19, 2, 8))
    vc = g.standard_normal((2, 19, 2, 8))
    out, lse = ref.attend(q, kc, vc)
    perm = g.permutation(19)
    out_p, lse_p = ref.attend(q, kc[:, perm], vc[:, perm])
    np.testing.assert_allclose(out_p, out, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(lse_p, lse, rtol=1e-12)
    # a single key: the output is its value
    o1, _ = ref.attend(q, kc[:, :1], vc[:, :1])
    for h in range(4):
        np.testing.assert_allclose(o1[:, :, h], np.broadcast_to(vc[:, :1, h // 2], o1[:, :, h].shape))
    # equal scores (zero query): the output is the mean of the values
    o0, l0 = ref.attend(np.zeros_like(q), kc, vc)
    for h in range(4):
        np.testing.assert_allclose(o0[:, :, h], np.broadcast_to(vc[:, :, h // 2].mean(axis=1)[:, None],
                                                                 o0[:, :, h].shape), rtol=1e-12)
    np.testing.assert_allclose(l0, math.log(19), rtol=1e-12)


def test_attention_gqa_equals_mha_with_repeated_kv_heads():
    """Consecutive query heads share one KV head: query head h reads KV head
    h // (heads / kv_heads)."""
    g = np.random.default_rng(14)
    q = g.standard_normal((1, 6, 6, 4))
    kc = g.standard_normal((1, 9, 2, 4))
    vc = g.standard_normal((1, 9, 2, 4))
    out, lse = ref.attend(q, kc, vc)
    rep = [0, 0, 0, 1, 1, 1]
    out_m, lse_m = ref.attend(q, kc[:, :, rep], vc[:, :, rep])
    np.testing.assert_allclose(out, out_m, rtol=1e-13)
    np.testing.assert_allclose(lse, lse_m, rtol=1e-13)


def test_attention_first_order_perturbation_proposition_1():
    """Prop. 1 (App. B): changing position s's input by eta changes o_i by
    a_is W_V eta + a_is (q_i . W_K eta / sqrt(d_h)) (v_s - o_i) + O(|eta|^2)."""
    g = np.random.default_rng(15)
    d, hd, seq, s = 12, 6, 9, 4
    w_q = g.standard_normal((hd, d)) * 0.4
    w_k = g.standard_normal((hd, d)) * 0.4
    w_v = g.standard_normal((hd, d)) * 0.4
    x = g.standard_normal((seq, d))
    eta = g.standard_normal(d) * 1e-5

    def run(xx):
        q = (xx @ w_q.T)[None, :, None, :]
        k = (xx @ w_k.T)[None, :, None, :]
        v = (xx @ w_v.T)[None, :, None, :]
        return ref.attend(q, k, v)[0][0, :, 0, :]

    x2 = x.copy()
    x2[s] += eta
    diff = run(x2) - run(x)
    q = x @ w_q.T
    k = x @ w_k.T
    v = x @ w_v.T
    o = run(x)
    for i in range(seq):
        if i == s:
            continue
        logits = q[i] @ k.T / math.sqrt(hd)
        a = np.exp(logits - logits.max())
        a /= a.sum()
        pred = a[s] * (w_v @ eta) + a[s] * (q[i] @ (w_k @ eta) / math.sqrt(hd)) * (v[s] - o[i])
        np.testing.assert_allclose(diff[i], pred, rtol=1e-4, atol=1e-13)


# --------------------------------------------------------------------------
# Step 5 -- commit
# --------------------------------------------------------------------------

def test_confidence_closed_forms(golden):
    for name in ("confidence_two_level", "confidence_mask_excluded", "confidence_tie_lowest_id"):
        g = golden[name]
        tok, conf = ref.confidence(np.array([[g["logits"]]]), g["mask_token_id"])
        assert tok[0, 0] == g["token"]
        assert conf[0, 0] == pytest.approx(_expr(g["expect"]), rel=1e-13)
        bt, bc = brute.confidence_row(g["logits"], g["mask_token_id"])
        assert bt == g["token"] and bc == pytest.approx(_expr(g["expect"]), rel=1e-13)


def test_confidence_matches_pure_python_on_tiny_config():
    cfg, x, dec = _cfg0()
    lg = ref.decode(x["logits"], cfg.dtype)
    tok, conf = ref.confidence(lg, -1)
    tok_m, conf_m = ref.confidence(lg, 7)
    for j in range(cfg.block_len):
        t, c = brute.confidence_row(lg[0, j].tolist(), -1)
        assert tok[0, j] == t and conf[0, j] == pytest.approx(c, rel=1e-12)
        t, c = brute.confidence_row(lg[0, j].tolist(), 7)
        assert tok_m[0, j] == t and conf_m[0, j] == pytest.approx(c, rel=1e-12)


def test_commit_threshold_cases(golden):
    for case in golden["dynamic_threshold"]["cases"]:
        h = 1 if case["mu"] != 0.0 else 0
        hist = np.full((1, max(h, 1), 1), case["mu"], dtype=np.float32)
        commit, _, _ = ref.commit_rule(np.array([[case["conf"]]], np.float32),
                                       np.array([[case["delta"]]], np.float32),
                                       np.array([[True]]), hist, np.array([h], np.int32), h,
                                       case["tau_s"], case["alpha"], False)
        assert bool(commit[0, 0]) == case["commit"], case
        t = np.float32(case["tau_s"]) - np.float32(case["conf"])
        assert float(np.float32(np.float32(case["alpha"]) * t) * t) == pytest.approx(
            _expr(case["tau_d"]), rel=1e-5, abs=1e-7)


def test_commit_history_mean_push_and_raw_drift():
    # h = 0: no history, the delta is the raw drift
    c = np.array([[0.5, 0.5]], np.float32)
    dl = np.array([[1.7, 1.5]], np.float32)
    m = np.array([[True, True]])
    commit, hist, n = ref.commit_rule(c, dl, m, np.zeros((1, 0, 2), np.float32),
                                      np.array([0], np.int32), 0, 0.9, 10.0, False)
    assert commit.tolist() == [[True, False]] and n.tolist() == [0]
    # mean over the entries present, delta taken before the push
    hist = np.zeros((1, 3, 2), np.float32)
    hist[0, 0] = [1.0, 0.0]
    hist[0, 1] = [0.0, 0.0]
    dl2 = np.array([[2.0, 1.5]], np.float32)
    commit, h2, n2 = ref.commit_rule(c, dl2, m, hist, np.array([2], np.int32), 3, 0.9, 10.0, False)
    # 2.0 - (1 + 0) / 2 = 1.5 < 1.6 (a mean over all 3 slots would give 1.67 > 1.6)
    assert commit.tolist() == [[False, False]]
    assert n2.tolist() == [3] and h2[0, 2].tolist() == pytest.approx([2.0, 1.5])
    # full history: the oldest entry drops out
    commit, h3, n3 = ref.commit_rule(c, dl, m, h2, n2, 3, 0.9, 10.0, False)
    assert n3.tolist() == [3]
    assert h3[0, :, 0].tolist() == pytest.approx([0.0, 2.0, 1.7])


def test_commit_force_one_fallback():
    c = np.array([[0.3, 0.6, 0.6, 0.2], [0.95, 0.1, 0.2, 0.3]], np.float32)
    dl = np.zeros((2, 4), np.float32)
    m = np.array([[True, True, True, False], [True, True, False, False]])
    hist = np.zeros((2, 1, 4), np.float32)
    n = np.zeros(2, np.int32)
    commit, _, _ = ref.commit_rule(c, dl, m, hist, n, 1, 0.9, 10.0, True)
    # sequence 0: nothing qualifies -> the largest confidence, lower position on a tie
    assert commit[0].tolist() == [False, True, False, False]
    # sequence 1: token 0 qualifies; no extra commit
    assert commit[1].tolist() == [True, False, False, False]
    commit_off, _, _ = ref.commit_rule(c, dl, m, hist, n, 1, 0.9, 10.0, False)
    assert not commit_off[0].any()
    # no masked token: nothing is committed even with the fallback
    none, _, _ = ref.commit_rule(c, dl, np.zeros((2, 4), bool), hist, n, 1, 0.9, 10.0, True)
    assert not none.any()


def test_staleness_closed_forms(golden):
    g = np.random.default_rng(16)
    k = g.standard_normal((1, 3, 2, 5))
    v = g.standard_normal((1, 3, 2, 5))
    assert np.allclose(ref.staleness(k, v, k, v), _expr(golden["staleness"]["identical"]))
    assert np.allclose(ref.staleness(k, v, -k, -v), _expr(golden["staleness"]["negated"]))
    e1 = np.zeros((1, 1, 1, 2))
    e1[..., 0] = 1
    e2 = np.zeros((1, 1, 1, 2))
    e2[..., 1] = 1
    assert np.allclose(ref.staleness(e1, e1, e2, e2), _expr(golden["staleness"]["orthogonal"]))


# --------------------------------------------------------------------------
# Dtype helpers
# --------------------------------------------------------------------------

def test_bf16_rounding_definition():
    # exactly representable values stay; halfway cases go to the even significand
    one = 1.0
    ulp = 2.0 ** -7
    assert ref.round_to_bf16(np.array([one]))[0] == one
    assert ref.round_to_bf16(np.array([one + ulp / 2]))[0] == one              # tie -> even (1.0)
    assert ref.round_to_bf16(np.array([one + 1.5 * ulp]))[0] == one + 2 * ulp  # tie -> even
    assert ref.round_to_bf16(np.array([one + 0.51 * ulp]))[0] == one + ulp
    assert ref.round_to_bf16(np.array([-3.0 - 0.49 * 2 * ulp]))[0] == -3.0
    # agrees with the generator's integer rounding on float32 inputs
    x = np.random.default_rng(17).standard_normal(10000).astype(np.float32)
    bits = inputs.f32_to_bf16_bits(x)
    np.testing.assert_array_equal(ref.decode(bits, "bf16"), ref.round_to_bf16(x.astype(np.float64)))


# ---------------------------------------------------------------------------
# suffix-block commit (Sec. 4.2, "Suffix Block Commit")
# ---------------------------------------------------------------------------

def test_suffix_eligible_is_packet_within_suffix():
    # packet rows 3, 40, 41, 47, 48 of a sequence with suffix window [40, 48)
    idx = np.array([[3, 40, 41, 47, 48, -1], [44, -1, -1, -1, -1, -1]])
    cnt = np.array([5, 1])
    el = ref.suffix_eligible(idx, cnt, 40, 8)
    assert el[0].tolist() == [True, True, False, False, False, False, False, True]
    assert el[1].tolist() == [False] * 4 + [True] + [False] * 3
    # entries past stale_count are ignored
    assert not ref.suffix_eligible(idx, np.array([1, 0]), 40, 8).any()


def test_suffix_commit_closed_form():
    # two-token vocabularies with known softmax: conf = a / (a + 1) for logits (log a, 0)
    a = np.array([19.0, 4.0, 19.0, 19.0, 99.0])              # conf 0.95, 0.8, 0.95, 0.95, 0.99
    logits = np.stack([np.log(a), np.zeros_like(a)], axis=-1)[None]
    token, conf = ref.confidence(logits, -1)
    assert np.allclose(conf[0], a / (a + 1), rtol=1e-15) and (token == 0).all()
    masked = np.array([[1, 1, 0, 1, 1]], bool)
    eligible = np.array([[1, 1, 1, 0, 1]], bool)
    got = ref.suffix_commit_rule(conf.astype(np.float32), masked, eligible, 0.9)
    # conf high but unmasked (2) or not in the packet (3): no commit; low conf (1): no
    assert got[0].tolist() == [True, False, False, False, True]
    # strict comparison: conf equal to tau_s does not commit
    c = np.array([[np.float32(0.9)]])
    assert not ref.suffix_commit_rule(c, [[True]], [[True]], 0.9)[0, 0]
