"""GPU parity of the clustered proxy drift (polestar_cluster,
polestar_proxy_drift, polestar_cluster_select, polestar_cluster_update)
against the oracle in oracle/proxy_ref.py.

Inputs are seeded and built on the host; the oracle runs its own K-means,
caches and scores from them and never reads a GPU result.  Tolerances:
integer outputs (labels, counts, stale sets) exact; fp32 sums and centroids
1e-5 relative (fp32 accumulation over at most a few hundred exactly
representable terms); proxy scores 1e-4 relative and the drift 2e-3
relative + 1e-6 absolute (a KL of close distributions is a small
difference of fp32 terms).
"""

import numpy as np
import pytest

from oracle import polestar_ref as ref
from oracle import proxy_ref as pr
from paper_2607_14107_amd import inputs
from tests._util import assert_rows_close, ensure_built, from_dev, to_dev

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


def planted_window(batch, seq, d, win, K, dtype, seed, noise=0.1):
    """Hidden states whose window rows lie around K random directions, with
    norms spread over [0.5, 2] * sqrt(d); other rows N(0, 1).  Returns the
    stored array (bf16 bits or fp32) and the planted cluster of each window
    row."""
    g = np.random.default_rng(seed)
    h = g.standard_normal((batch, seq, d), dtype=np.float32)
    truth = np.zeros((batch, len(win)), dtype=np.int64)
    for b in range(batch):
        dirs = g.standard_normal((K, d))
        dirs /= np.linalg.norm(dirs, axis=1, keepdims=True)
        lab = g.integers(0, K, size=len(win))
        # the deterministic start points (window ranks floor(j*n/K)) fall in
        # distinct planted clusters, so K-means settles on the planted
        # partition with wide cosine margins (no fp32/fp64 near-ties)
        for j in range(K):
            lab[(j * len(win)) // K] = j
        x = dirs[lab] + noise * g.standard_normal((len(win), d)) / np.sqrt(d)
        x /= np.linalg.norm(x, axis=1, keepdims=True)
        x *= np.sqrt(d) * g.uniform(0.5, 2.0, size=(len(win), 1))
        h[b, win] = x.astype(np.float32)
        truth[b] = lab
    return inputs.store(h, dtype), truth


@pytest.mark.parametrize("dtype,batch,seq,d,K,block_start", [
    ("fp32", 1, 96, 256, 4, 64), ("bf16", 1, 768, 4096, 8, 512), ("bf16", 3, 300, 1024, 16, 100)])
def test_cluster_matches_oracle(P, dtype, batch, seq, d, K, block_start):
    torch = _torch()
    win = P.window_positions(seq, block_start, 32, 64, 32)
    hs, _ = planted_window(batch, seq, d, win, K, dtype, seed=seq + K)
    widx = torch.tensor([win] * batch, dtype=torch.int32, device="cuda")
    labels, sums, counts, cents = P.cluster(to_dev(hs, dtype), widx, K, iters=10)
    h = ref.decode(hs, dtype)
    lab_g, sums_g, cnt_g, z_g = from_dev(labels), from_dev(sums), from_dev(counts), from_dev(cents)
    for b in range(batch):
        lab_o, z_o = pr.spherical_kmeans(h[b, win], K, iters=10)
        s_o, c_o = pr.cluster_sums(h[b, win], lab_o, K)
        assert np.array_equal(lab_g[b], pr.labels_by_position(win, lab_o, seq))
        assert np.array_equal(cnt_g[b], c_o)
        np.testing.assert_allclose(sums_g[b], s_o, rtol=1e-5, atol=1e-5 * np.abs(s_o).max())
        np.testing.assert_allclose(z_g[b], z_o, rtol=0, atol=1e-5)


@pytest.mark.parametrize("n_win", [150, 176, 177, 192, 224, 225])
def test_cluster_window_sizes_match_oracle(P, n_win):
    """Windows of up to 224 positions run the K-means on the window's Gram
    matrix (its upper triangle in LDS), longer ones directly on the rows; both
    match the oracle (ragged tile counts, the largest Gram window, the first
    direct one)."""
    torch = _torch()
    seq, d, K = 400, 512, 12
    g = np.random.default_rng(n_win)
    win = sorted(g.choice(seq, size=n_win, replace=False).tolist())
    hs, _ = planted_window(2, seq, d, win, K, "bf16", seed=n_win)
    widx = torch.tensor([win, win], dtype=torch.int32, device="cuda")
    labels, sums, counts, cents = P.cluster(to_dev(hs, "bf16"), widx, K, iters=10)
    h = ref.decode(hs, "bf16")
    lab_g, sums_g, cnt_g, z_g = from_dev(labels), from_dev(sums), from_dev(counts), from_dev(cents)
    for b in range(2):
        lab_o, z_o = pr.spherical_kmeans(h[b, win], K, iters=10)
        s_o, c_o = pr.cluster_sums(h[b, win], lab_o, K)
        assert np.array_equal(lab_g[b], pr.labels_by_position(win, lab_o, seq))
        assert np.array_equal(cnt_g[b], c_o)
        np.testing.assert_allclose(sums_g[b], s_o, rtol=1e-5, atol=1e-5 * np.abs(s_o).max())
        np.testing.assert_allclose(z_g[b], z_o, rtol=0, atol=1e-5)


@pytest.mark.parametrize("n_win", [48, 65, 97, 177, 224])
def test_cluster_gram_over_workgroups_matches_oracle(P, n_win):
    """Windows longer than 64 positions whose packed Gram matrix fits the
    centroid output (K d >= n (n + 1) / 2) compute G over many workgroups in
    32 x 32 blocks (ragged last block row and column); 48 positions stay on
    the single-workgroup product."""
    torch = _torch()
    seq, d, K = 600, 2048, 16
    assert K * d >= n_win * (n_win + 1) // 2
    g = np.random.default_rng(1000 + n_win)
    win = sorted(g.choice(seq, size=n_win, replace=False).tolist())
    hs, _ = planted_window(2, seq, d, win, K, "bf16", seed=2000 + n_win)
    widx = torch.tensor([win, win], dtype=torch.int32, device="cuda")
    labels, sums, counts, cents = P.cluster(to_dev(hs, "bf16"), widx, K, iters=10)
    h = ref.decode(hs, "bf16")
    lab_g, sums_g, cnt_g, z_g = from_dev(labels), from_dev(sums), from_dev(counts), from_dev(cents)
    for b in range(2):
        lab_o, z_o = pr.spherical_kmeans(h[b, win], K, iters=10)
        s_o, c_o = pr.cluster_sums(h[b, win], lab_o, K)
        assert np.array_equal(lab_g[b], pr.labels_by_position(win, lab_o, seq))
        assert np.array_equal(cnt_g[b], c_o)
        np.testing.assert_allclose(sums_g[b], s_o, rtol=1e-5, atol=1e-5 * np.abs(s_o).max())
        np.testing.assert_allclose(z_g[b], z_o, rtol=0, atol=1e-5)


def test_cluster_dream_shape_window_matches_oracle(P):
    """The Dream-7B layer's block entry: batch 4, d 3584, K 8 over the window
    of 2B = 128 positions before the 64-position block and B after (192)."""
    torch = _torch()
    seq, d, K, bs, bl = 2048, 3584, 8, 1536, 64
    win = P.window_positions(seq, bs, bl, 2 * bl, bl)
    assert len(win) == 192
    hs, _ = planted_window(4, seq, d, win, K, "bf16", seed=77)
    widx = torch.tensor([win] * 4, dtype=torch.int32, device="cuda")
    labels, sums, counts, cents = P.cluster(to_dev(hs, "bf16"), widx, K, iters=10)
    h = ref.decode(hs, "bf16")
    lab_g, sums_g, cnt_g, z_g = from_dev(labels), from_dev(sums), from_dev(counts), from_dev(cents)
    for b in range(4):
        lab_o, z_o = pr.spherical_kmeans(h[b, win], K, iters=10)
        s_o, c_o = pr.cluster_sums(h[b, win], lab_o, K)
        assert np.array_equal(lab_g[b], pr.labels_by_position(win, lab_o, seq))
        assert np.array_equal(cnt_g[b], c_o)
        np.testing.assert_allclose(sums_g[b], s_o, rtol=1e-5, atol=1e-5 * np.abs(s_o).max())
        np.testing.assert_allclose(z_g[b], z_o, rtol=0, atol=1e-5)


def test_cluster_labels_are_nearest_final_centroids_on_noisy_data(P):
    """Heavy noise (clusters overlap): whatever the partition, every GPU label
    is a nearest GPU centroid by the float64 cosine, up to fp32 rounding."""
    torch = _torch()
    seq, d, K = 400, 512, 8
    win = list(range(0, 300))
    hs, _ = planted_window(1, seq, d, win, K, "bf16", seed=9, noise=3.0)
    widx = torch.tensor([win], dtype=torch.int32, device="cuda")
    labels, _, counts, cents = P.cluster(to_dev(hs, "bf16"), widx, K, iters=15)
    x = ref.decode(hs, "bf16")[0, win]
    x /= np.linalg.norm(x, axis=1, keepdims=True)
    cos = x @ from_dev(cents)[0].T
    lab = from_dev(labels)[0, win]
    assert np.all(cos[np.arange(len(win)), lab] >= cos.max(axis=1) - 1e-5)
    assert from_dev(counts)[0].sum() == len(win)


def _proxy_case(dtype, seed):
    """The batch-1 LLaDA-8B layer (the tiny fp32 layer for fp32) with planted clusters in the
    window of h_prev: weights, the prior cache, and a second cache whose 20
    random rows are re-projected from perturbed states."""
    cfg = inputs.CONFIGS[1] if dtype == "bf16" else inputs.CONFIGS[0]
    x = inputs.layer_inputs(cfg, 0)
    K = 8 if dtype == "bf16" else 4
    win = list(range(max(0, cfg.block_start - 2 * cfg.block_len), cfg.block_start)) + \
        list(range(cfg.block_start + cfg.block_len, min(cfg.seq, cfg.block_start + 2 * cfg.block_len)))
    hs, _ = planted_window(cfg.batch, cfg.seq, cfg.d, win, K, cfg.dtype, seed=seed)
    h_prev = ref.decode(hs, cfg.dtype)
    w_q, w_k = ref.decode(x["w_q"], cfg.dtype), ref.decode(x["w_k"], cfg.dtype)
    shape = (cfg.batch, cfg.seq, cfg.n_kv_heads, cfg.head_dim)
    k0 = ref.round_to((h_prev @ w_k.T).reshape(shape), cfg.dtype)
    g = np.random.default_rng(seed)
    rows = g.choice(cfg.seq, size=20, replace=False)
    moved = h_prev[:, rows] + 0.5 * g.standard_normal((cfg.batch, 20, cfg.d))
    k1 = k0.copy()
    k1[:, rows] = ref.round_to((moved @ w_k.T).reshape(cfg.batch, 20, cfg.n_kv_heads, cfg.head_dim), cfg.dtype)
    return cfg, x, hs, h_prev, w_q, K, win, k0, k1


def _bits(a, dtype):
    return inputs.store(a.astype(np.float32), dtype)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_proxy_drift_matches_oracle(P, dtype):
    torch = _torch()
    cfg, x, hs, h_prev, w_q, K, win, k0, k1 = _proxy_case(dtype, seed=3)
    widx = torch.tensor([win] * cfg.batch, dtype=torch.int32, device="cuda")
    labels, sums, counts, _ = P.cluster(to_dev(hs, cfg.dtype), widx, K)
    # the oracle's own clustering of the same states
    sums_o = np.zeros((cfg.batch, K, cfg.d))
    cnt_o = np.zeros((cfg.batch, K), dtype=np.int64)
    for b in range(cfg.batch):
        lab_o, _ = pr.spherical_kmeans(h_prev[b, win], K)
        sums_o[b], cnt_o[b] = pr.cluster_sums(h_prev[b, win], lab_o, K)
        assert np.array_equal(from_dev(labels)[b], pr.labels_by_position(win, lab_o, cfg.seq))
    tok = pr.proxy_tokens(sums_o, cnt_o, cfg.dtype)
    s0 = pr.proxy_scores(tok, w_q, k0, cfg.n_heads, cfg.dtype)
    s1 = pr.proxy_scores(tok, w_q, k1, cfg.n_heads, cfg.dtype)
    want = pr.proxy_kl(s1, s0)

    scores = torch.empty((cfg.batch, K, cfg.n_heads, cfg.seq), dtype=torch.float32, device="cuda")
    lse = torch.empty((cfg.batch, K, cfg.n_heads), dtype=torch.float32, device="cuda")
    wq = to_dev(x["w_q"], cfg.dtype)
    d0 = P.proxy_drift(sums, counts, wq, to_dev(_bits(k0, cfg.dtype), cfg.dtype), cfg.n_heads, scores, lse,
                       first=True)
    torch.cuda.synchronize()
    assert np.all(from_dev(d0) == 0.0)
    g0 = from_dev(scores)
    if dtype == "fp32":
        np.testing.assert_allclose(g0, s0, rtol=1e-4, atol=1e-4 * np.abs(s0).max())
        np.testing.assert_allclose(from_dev(lse), pr.log_sum_exp(s0), rtol=1e-4, atol=1e-5)
    else:
        # bf16 queries: an element on a rounding boundary may round the other
        # way under a different fp32 summation order, moving a score by
        # 2^-8 |q_j k_j| per such element
        assert_rows_close(g0, s0, 4e-3, "proxy scores")
        np.testing.assert_allclose(from_dev(lse), pr.log_sum_exp(g0), rtol=1e-5, atol=1e-5)
    d1 = P.proxy_drift(sums, counts, wq, to_dev(_bits(k1, cfg.dtype), cfg.dtype), cfg.n_heads, scores, lse,
                       first=False)
    torch.cuda.synchronize()
    g1 = from_dev(scores)
    assert want.max() > 1e-4                  # the changed rows do move the proxies
    if dtype == "fp32":
        np.testing.assert_allclose(from_dev(d1), want, rtol=2e-3, atol=1e-6)
        np.testing.assert_allclose(g1, s1, rtol=1e-4, atol=1e-4 * np.abs(s1).max())
    else:
        # Queries rounded to bf16 from K-means sums can differ from the
        # oracle's by one rounding step, which the KL of two close score rows
        # amplifies; the drift is compared with the KL of the GPU's own
        # scores here, and with the oracle's at the same bar in
        # test_proxy_drift_bf16_exact_queries_matches_oracle, where both
        # sides hold identical queries.
        assert_rows_close(g1, s1, 4e-3, "proxy scores")
        np.testing.assert_allclose(from_dev(d1), pr.proxy_kl(g1, g0), rtol=2e-3, atol=1e-6)
    # an unchanged cache gives zero drift
    d2 = P.proxy_drift(sums, counts, wq, to_dev(_bits(k1, cfg.dtype), cfg.dtype), cfg.n_heads, scores, lse,
                       first=False)
    torch.cuda.synchronize()
    assert np.abs(from_dev(d2)).max() < 1e-6


def test_proxy_drift_bf16_exact_queries_matches_oracle(P):
    """bf16 proxy drift on the batch-1 LLaDA-8B layer against the oracle at
    the fp32 arithmetic bar (2e-3 relative + 1e-6 absolute, the bound derived
    for a KL of two close fp32 score rows).  The inputs make the proxy queries
    identical on both sides: cluster sizes are powers of two and the members'
    mean lies on a 2^-6 grid in [-1, 1], so sums / count is exact; W_q lies on
    a 2^-10 grid in [-2^-4, 2^-4], so every fp32 partial sum of W_q . token is
    a multiple of 2^-16 below 2^8, exact in fp32 as in float64, and both round
    the same value to bf16.  What remains is fp32 rounding of the scores and
    of the KL itself."""
    torch = _torch()
    cfg, x, hs, h_prev, w_q_unused, K, win, k0, k1 = _proxy_case("bf16", seed=3)
    g = np.random.default_rng(77)
    counts = np.array([[1, 2, 4, 8, 16, 32, 8, 4]], dtype=np.int32)
    assert counts.shape == (cfg.batch, K)
    mean = g.integers(-64, 65, size=(cfg.batch, K, cfg.d)).astype(np.float64) / 64.0
    sums = mean * counts[..., None]
    w_q = g.integers(-64, 65, size=(cfg.n_heads * cfg.head_dim, cfg.d)).astype(np.float64) / 1024.0
    tok = pr.proxy_tokens(sums, counts, "bf16")
    assert np.array_equal(tok, mean)                 # the grid mean is exact in bf16
    s0 = pr.proxy_scores(tok, w_q, k0, cfg.n_heads, "bf16")
    s1 = pr.proxy_scores(tok, w_q, k1, cfg.n_heads, "bf16")
    want = pr.proxy_kl(s1, s0)
    assert want.min() > 1e-4                         # every proxy sees the moved rows

    dev_sums = torch.from_numpy(sums.astype(np.float32)).cuda()
    dev_cnt = torch.from_numpy(counts).cuda()
    wq = to_dev(_bits(w_q, "bf16"), "bf16")
    scores = torch.empty((cfg.batch, K, cfg.n_heads, cfg.seq), dtype=torch.float32, device="cuda")
    lse = torch.empty((cfg.batch, K, cfg.n_heads), dtype=torch.float32, device="cuda")
    P.proxy_drift(dev_sums, dev_cnt, wq, to_dev(_bits(k0, "bf16"), "bf16"), cfg.n_heads, scores, lse, first=True)
    torch.cuda.synchronize()
    assert_rows_close(from_dev(scores), s0, 1e-4, "proxy scores, step 0")
    np.testing.assert_allclose(from_dev(lse), pr.log_sum_exp(s0), rtol=1e-5, atol=1e-5)
    d1 = P.proxy_drift(dev_sums, dev_cnt, wq, to_dev(_bits(k1, "bf16"), "bf16"), cfg.n_heads, scores, lse,
                       first=False)
    torch.cuda.synchronize()
    assert_rows_close(from_dev(scores), s1, 1e-4, "proxy scores, step 1")
    np.testing.assert_allclose(from_dev(d1), want, rtol=2e-3, atol=1e-6)


@pytest.mark.parametrize("batch,seq,K,k_top,k_max", [(1, 768, 8, 4, 96), (3, 200, 16, 5, 40),
                                                       (2, 50, 4, 0, 10), (2, 300, 5, 9, 300),
                                                       (1, 100, 8, 8, 7)])
def test_cluster_select_bit_exact(P, batch, seq, K, k_top, k_max):
    torch = _torch()
    g = np.random.default_rng(seq + k_top)
    lab = np.full((batch, seq), -1, dtype=np.int32)
    for b in range(batch):
        win = g.choice(seq, size=min(seq, 96), replace=False)
        lab[b, win] = g.integers(0, K, size=len(win))
    drift = np.round(g.random((batch, K)), 1).astype(np.float32)    # ties on purpose
    idx, cnt = P.cluster_select(torch.from_numpy(lab).cuda(), torch.from_numpy(drift).cuda(), k_top, k_max)
    sel = pr.select_clusters(drift.astype(np.float64), k_top)
    want_idx, want_cnt = pr.cluster_members(lab, sel)
    want_cnt = np.minimum(want_cnt, k_max)
    got_idx, got_cnt = from_dev(idx), from_dev(cnt)
    assert np.array_equal(got_cnt, want_cnt)
    for b in range(batch):
        n = want_cnt[b]
        assert np.array_equal(got_idx[b, :n], want_idx[b, :n])
        assert np.all(got_idx[b, n:] == -1)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_cluster_update_matches_oracle(P, dtype):
    torch = _torch()
    g = np.random.default_rng(11)
    batch, seq, d, K = 2, 120, 256, 6
    win = list(range(30, 100))
    lab = np.stack([pr.labels_by_position(win, g.integers(0, K, size=len(win)), seq) for _ in range(batch)])
    h_old = inputs.store(g.standard_normal((batch, seq, d), dtype=np.float32), dtype)
    h_new = inputs.store(g.standard_normal((batch, seq, d), dtype=np.float32), dtype)
    stale = np.full((batch, 40), -1, dtype=np.int32)
    cnt = np.array([35, 12], dtype=np.int32)
    for b in range(batch):
        stale[b, :cnt[b]] = np.sort(g.choice(seq, size=cnt[b], replace=False))   # some outside the window
    sums0 = g.standard_normal((batch, K, d)).astype(np.float32)
    sums = torch.from_numpy(sums0.copy()).cuda()
    P.cluster_update(to_dev(h_new, dtype), to_dev(h_old, dtype), torch.from_numpy(lab.astype(np.int32)).cuda(),
                     torch.from_numpy(stale).cuda(), torch.from_numpy(cnt).cuda(), sums)
    want = pr.update_sums(sums0.astype(np.float64), lab, stale, cnt, ref.decode(h_new, dtype),
                          ref.decode(h_old, dtype))
    np.testing.assert_allclose(from_dev(sums), want, rtol=1e-5, atol=1e-5)


def test_proxy_pipeline_end_to_end(P):
    """Block entry (cluster, first proxy pass) then one step: the cache rows of
    two planted clusters' members change, so those clusters drift most; the
    selected rows are exactly their members, the refresh and the cluster
    update then match the oracle."""
    torch = _torch()
    cfg = inputs.CONFIGS[1]
    x = inputs.layer_inputs(cfg, 0)
    K, k_top = 8, 2
    win = P.window_positions(cfg.seq, cfg.block_start, cfg.block_len, 64, 32)
    hs, truth = planted_window(1, cfg.seq, cfg.d, win, K, "bf16", seed=21)
    h_prev = ref.decode(hs, "bf16")
    dec = {n: ref.decode(x[n], "bf16") for n in ("w_q", "w_k", "w_v")}
    lab_o, _ = pr.spherical_kmeans(h_prev[0, win], K)
    # h_cur: the members of the clusters started at window ranks 0 and
    # floor((K-1)n/K) move strongly, everything else stays
    moved = {int(lab_o[0]), int(lab_o[((K - 1) * len(win)) // K])}
    assert len(moved) == 2
    g = np.random.default_rng(22)
    h_cur = h_prev.copy()
    rows = [win[i] for i in range(len(win)) if lab_o[i] in moved]
    h_cur[0, rows] += 3.0 * g.standard_normal((len(rows), cfg.d))
    hc = inputs.store(h_cur.astype(np.float32), "bf16")
    h_cur = ref.decode(hc, "bf16")
    shape = (1, cfg.seq, cfg.n_kv_heads, cfg.head_dim)
    k0 = ref.round_to((h_prev @ dec["w_k"].T).reshape(shape), "bf16")
    v0 = ref.round_to((h_prev @ dec["w_v"].T).reshape(shape), "bf16")
    # the step's cache: rows of the moved clusters re-projected (what a refresh of
    # the previous layer's packet would carry), the rest as at block entry
    k1 = k0.copy()
    k1[:, rows] = ref.round_to((h_cur[:, rows] @ dec["w_k"].T).reshape(1, len(rows), cfg.n_kv_heads, cfg.head_dim),
                               "bf16")

    widx = torch.tensor([win], dtype=torch.int32, device="cuda")
    labels, sums, counts, _ = P.cluster(to_dev(hs, "bf16"), widx, K)
    scores = torch.empty((1, K, cfg.n_heads, cfg.seq), dtype=torch.float32, device="cuda")
    lse = torch.empty((1, K, cfg.n_heads), dtype=torch.float32, device="cuda")
    # W_q = W_k: a cluster's proxy query then attends to keys aligned with its
    # own members (with unrelated random W_q and W_k it would not), so moving
    # two clusters' members moves those clusters' proxy distributions most
    wq = to_dev(x["w_k"], "bf16")
    P.proxy_drift(sums, counts, wq, to_dev(_bits(k0, "bf16"), "bf16"), cfg.n_heads, scores, lse, first=True)
    drift = P.proxy_drift(sums, counts, wq, to_dev(_bits(k1, "bf16"), "bf16"), cfg.n_heads, scores, lse,
                          first=False)
    idx, cnt = P.cluster_select(labels, drift, k_top, len(win))
    torch.cuda.synchronize()
    top = set(np.argsort(-from_dev(drift)[0], kind="stable")[:k_top].tolist())
    assert top == moved
    n = int(from_dev(cnt)[0])
    assert from_dev(idx)[0, :n].tolist() == sorted(rows)
    # refresh those rows (and the block) from h_cur, then move the cluster sums
    kc, vc = to_dev(_bits(k1, "bf16"), "bf16"), to_dev(_bits(v0, "bf16"), "bf16")
    P.refresh_kv(to_dev(hc, "bf16"), idx, cnt, cfg.block_start, cfg.block_len, to_dev(x["w_k"], "bf16"),
                 to_dev(x["w_v"], "bf16"), kc, vc)
    P.cluster_update(to_dev(hc, "bf16"), to_dev(hs, "bf16"), labels, idx, cnt, sums)
    torch.cuda.synchronize()
    s_prev, _ = pr.cluster_sums(h_prev[0, win], lab_o, K)
    lab_pos = pr.labels_by_position(win, lab_o, cfg.seq)[None]
    want = pr.update_sums(s_prev[None], lab_pos, np.array([sorted(rows)]), np.array([len(rows)]), h_cur, h_prev)
    np.testing.assert_allclose(from_dev(sums), want, rtol=1e-5, atol=1e-5 * np.abs(want).max())
    kr = ref.decode(from_dev(kc), "bf16")
    k_want = ref.round_to((h_cur @ dec["w_k"].T).reshape(shape), "bf16")
    for r in rows:
        assert np.abs(kr[0, r] - k_want[0, r]).max() <= 2 ** -7 * np.abs(k_want[0, r]).max() + 1e-6


@pytest.mark.parametrize("dtype,b,seq,R,H,Hkv,hd", [
    ("bf16", 1, 768, 32, 32, 32, 128),     # the block's queries of the LLaDA-8B-shaped layer
    ("bf16", 4, 2048, 64, 28, 4, 128),     # Dream-7B GQA block of 64, long cache
    ("fp32", 2, 100, 5, 4, 2, 64),         # ragged key tile, few rows
])
def test_attention_drift_matches_oracle(P, dtype, b, seq, R, H, Hkv, hd):
    torch = _torch()
    g = np.random.default_rng(17)
    st = lambda a: inputs.store(a.astype(np.float32), dtype)
    q = st(g.standard_normal((b, R, H, hd)) * 0.5)
    k0 = st(g.standard_normal((b, seq, Hkv, hd)) * 0.5)
    k1f = ref.decode(k0, dtype).copy()
    rows = g.choice(seq, size=seq // 10, replace=False)
    k1f[:, rows] += g.standard_normal((b, len(rows), Hkv, hd)) * 0.3    # a refresh changed some keys
    k1 = st(k1f)
    qd, k0d, k1d = ref.decode(q, dtype), ref.decode(k0, dtype), ref.decode(k1, dtype)
    scores = torch.empty((b, R, H, seq), dtype=torch.float32, device="cuda")
    lse = torch.empty((b, R, H), dtype=torch.float32, device="cuda")
    qt = to_dev(q, dtype)
    d0 = P.attention_drift(qt, to_dev(k0, dtype), scores, lse, True)
    s0 = pr.query_scores(qd, k0d)
    assert np.all(from_dev(d0) == 0.0)
    np.testing.assert_allclose(from_dev(scores), s0, rtol=1e-4, atol=1e-4 * np.abs(s0).max())
    np.testing.assert_allclose(from_dev(lse), pr.log_sum_exp(s0), rtol=1e-4, atol=1e-5)
    d1 = P.attention_drift(qt, to_dev(k1, dtype), scores, lse, False)
    s1 = pr.query_scores(qd, k1d)
    want = pr.attention_drift(s1, s0)
    assert want.min() > 1e-5
    np.testing.assert_allclose(from_dev(d1), want, rtol=2e-3, atol=1e-6)
    np.testing.assert_allclose(from_dev(scores), s1, rtol=1e-4, atol=1e-4 * np.abs(s1).max())
    # an unchanged cache gives (numerically) zero drift
    d2 = P.attention_drift(qt, to_dev(k1, dtype), scores, lse, False)
    assert np.abs(from_dev(d2)).max() < 1e-5
