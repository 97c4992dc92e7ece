"""Pins of the clustered proxy-drift oracle (oracle/proxy_ref.py) against
what the paper and the mathematics fix: planted clusters, fixed-point
invariants of spherical K-means, closed forms of the proxy scores and of
KL, the head grouping, tie rules and the update-equals-recompute invariant.
CPU only."""

import math

import numpy as np
import pytest

from oracle import polestar_ref as ref
from oracle import proxy_ref as pr


def planted(n_clusters=4, per=10, d=64, seed=0, norm_lo=0.1, norm_hi=10.0, noise=0.05):
    """Points around n_clusters random directions with norms spread over two
    decades (Euclidean clustering would group by norm), shuffled."""
    g = np.random.default_rng(seed)
    dirs = g.standard_normal((n_clusters, d))
    dirs /= np.linalg.norm(dirs, axis=1, keepdims=True)
    truth = np.repeat(np.arange(n_clusters), per)
    x = dirs[truth] + noise * g.standard_normal((len(truth), d))
    x /= np.linalg.norm(x, axis=1, keepdims=True)
    x *= g.uniform(norm_lo, norm_hi, size=(len(truth), 1))
    perm = g.permutation(len(truth))
    return x[perm], truth[perm], dirs


def same_partition(a, b):
    pairs = {}
    for u, v in zip(a, b):
        if pairs.setdefault(u, v) != v:
            return False
    return len(set(pairs.values())) == len(pairs)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_kmeans_recovers_planted_directions_despite_norms(seed):
    x, truth, dirs = planted(seed=seed)
    labels, z = pr.spherical_kmeans(x, 4, iters=10)
    assert same_partition(labels, truth)
    for k in range(4):
        members = truth[labels == k]
        assert np.abs(z[k] @ dirs[members[0]]) > 0.99
        assert abs(np.linalg.norm(z[k]) - 1.0) < 1e-12


def test_kmeans_fixed_point_invariants():
    x, _, _ = planted(n_clusters=5, per=7, d=32, seed=4, noise=0.3)
    labels, z = pr.spherical_kmeans(x, 5, iters=50)
    u = x / np.linalg.norm(x, axis=1, keepdims=True)
    cos = u @ z.T
    # every point sits with a centroid of largest cosine
    assert np.all(cos[np.arange(len(x)), labels] >= cos.max(axis=1) - 1e-12)
    # every non-empty centroid is its members' normalised direction sum
    for k in range(5):
        m = u[labels == k]
        if len(m):
            s = m.sum(axis=0)
            assert np.allclose(z[k], s / np.linalg.norm(s), atol=1e-12)


def test_kmeans_deterministic_start_and_empty_cluster():
    # three identical directions: with K = 2 the start points are ranks 0 and 1
    # (same direction); the tie goes to cluster 0, cluster 1 stays empty and
    # keeps its start point
    x = np.array([[1.0, 0.0], [2.0, 0.0], [3.0, 0.0]])
    labels, z = pr.spherical_kmeans(x, 2, iters=3)
    assert labels.tolist() == [0, 0, 0]
    assert np.allclose(z[1], [1.0, 0.0])


def test_cluster_sums_partition_the_window():
    x, truth, _ = planted(seed=3)
    sums, counts = pr.cluster_sums(x, truth, 4)
    assert np.allclose(sums.sum(axis=0), x.sum(axis=0))
    assert counts.sum() == len(x) and counts.tolist() == [10, 10, 10, 10]
    assert np.allclose(sums[2], x[truth == 2].sum(axis=0))


def test_proxy_tokens_mean_rounding_and_empty():
    sums = np.array([[[3.0, 1.0]], [[0.0, 0.0]]]).reshape(1, 2, 2)
    counts = np.array([[3, 0]])
    tok = pr.proxy_tokens(sums, counts, "fp32")
    assert tok[0, 0].tolist() == [1.0, pytest.approx(1 / 3, abs=1e-7)]
    assert tok[0, 1].tolist() == [0.0, 0.0]
    # bf16: 1/3 -> 0.333984375 (8 significant bits, nearest)
    assert pr.proxy_tokens(sums, counts, "bf16")[0, 0, 1] == 0.333984375


def test_proxy_scores_closed_form_and_head_grouping():
    # hd = 2, H = 4 query heads over Hkv = 2 KV heads (heads 0,1 -> kv 0; 2,3 -> kv 1).
    # Token t = (1, 2, 0, 0); W_q gives head h the 2-vector (h+1) * (t0, t1).
    d, H, Hkv, hd, S = 4, 4, 2, 2, 3
    w_q = np.zeros((H * hd, d))
    for h in range(H):
        w_q[h * hd + 0, 0] = h + 1
        w_q[h * hd + 1, 1] = h + 1
    tokens = np.array([1.0, 2.0, 0.0, 0.0]).reshape(1, 1, d)
    k_cache = np.zeros((1, S, Hkv, hd))
    k_cache[0, :, 0, :] = [[1, 0], [0, 1], [1, 1]]        # kv head 0
    k_cache[0, :, 1, :] = [[0, 1], [1, 0], [0, 0]]        # kv head 1
    s = pr.proxy_scores(tokens, w_q, k_cache, H, "fp32")
    c = 1 / math.sqrt(hd)
    for h in range(H):
        q = (h + 1) * np.array([1.0, 2.0])
        keys = k_cache[0, :, h // 2, :]
        assert np.allclose(s[0, 0, h], c * keys @ q)
    assert np.allclose(s[0, 0, 0], c * np.array([1, 2, 3]))
    assert np.allclose(s[0, 0, 3], c * 4 * np.array([2, 1, 0]))


def test_proxy_kl_closed_forms():
    a, b = 0.7, 0.4
    cur = np.log([[a, 1 - a]])[None, None]         # [1][1][1 head][2 positions]
    prev = np.log([[b, 1 - b]])[None, None]
    want = a * math.log(a / b) + (1 - a) * math.log((1 - a) / (1 - b))
    assert pr.proxy_kl(cur.reshape(1, 1, 1, 2), prev.reshape(1, 1, 1, 2))[0, 0] == pytest.approx(want, rel=1e-12)
    # direction: KL(cur || prev), not the reverse
    rev = b * math.log(b / a) + (1 - b) * math.log((1 - b) / (1 - a))
    assert abs(want - rev) > 1e-3
    # identical and shifted scores give zero; averaging over heads
    g = np.random.default_rng(0)
    s = g.standard_normal((2, 3, 4, 9))
    assert np.allclose(pr.proxy_kl(s, s), 0.0, atol=1e-15)
    assert np.allclose(pr.proxy_kl(s + 5.0, s), 0.0, atol=1e-12)
    two = np.stack([np.log([a, 1 - a]), np.log([b, 1 - b])])[None, None]    # heads: (a), (b)
    ref = np.stack([np.log([b, 1 - b]), np.log([b, 1 - b])])[None, None]
    assert pr.proxy_kl(two, ref)[0, 0] == pytest.approx(want / 2, rel=1e-12)


def test_log_sum_exp_closed_form():
    s = np.array([math.log(2.0), math.log(3.0)]).reshape(1, 1, 1, 2)
    assert pr.log_sum_exp(s)[0, 0, 0] == pytest.approx(math.log(5.0), rel=1e-15)


def test_select_clusters_ties_and_overflow():
    d = np.array([[0.5, 0.9, 0.5, 0.1, 0.9]])
    assert pr.select_clusters(d, 2)[0].tolist() == [False, True, False, False, True]
    assert pr.select_clusters(d, 3)[0].tolist() == [True, True, False, False, True]   # tie 0 vs 2: lower
    assert pr.select_clusters(d, 9)[0].all()


def test_cluster_members_ascending_window_only():
    lab = np.array([[-1, 2, 0, 2, -1, 1, 0]])
    sel = np.array([[True, False, True]])
    idx, cnt = pr.cluster_members(lab, sel)
    assert cnt.tolist() == [4]
    assert idx[0].tolist() == [1, 2, 3, 6, -1, -1, -1]


def test_update_sums_equals_recomputing_the_window():
    g = np.random.default_rng(5)
    S, d, K = 12, 6, 3
    win = np.array([2, 3, 4, 5, 7, 8, 9])
    lab_w = np.array([0, 1, 1, 2, 0, 2, 1])
    lab = pr.labels_by_position(win, lab_w, S)[None]
    h_old = g.standard_normal((1, S, d))
    h_new = h_old.copy()
    stale = np.array([[3, 8, 9, 11, -1]])          # 11 is outside the window
    cnt = np.array([4])
    for p in (3, 8, 9, 11):
        h_new[0, p] += g.standard_normal(d)
    sums0, _ = pr.cluster_sums(h_old[0, win], lab_w, K)
    upd = pr.update_sums(sums0[None], lab, stale, cnt, h_new, h_old)
    want, _ = pr.cluster_sums(h_new[0, win], lab_w, K)
    assert np.allclose(upd[0], want, atol=1e-12)


def test_query_scores_closed_form_and_agreement_with_proxy_scores():
    # the proxy scores are the scores of the proxy tokens' rounded queries
    g = np.random.default_rng(9)
    b, K, d, H, Hkv, hd, S = 2, 3, 16, 4, 2, 4, 7
    tokens = g.standard_normal((b, K, d))
    w_q = g.standard_normal((H * hd, d)) * 0.3
    kc = g.standard_normal((b, S, Hkv, hd))
    q = ref.round_to(tokens @ w_q.T, "bf16").reshape(b, K, H, hd)
    assert np.allclose(pr.query_scores(q, kc), pr.proxy_scores(tokens, w_q, kc, H, "bf16"), rtol=1e-13)
    # one query, one head, two keys: scores are the scaled dot products
    q1 = np.array([1.0, 2.0]).reshape(1, 1, 1, 2)
    k1 = np.array([[3.0, 1.0], [0.0, -1.0]]).reshape(1, 2, 1, 2)
    assert np.allclose(pr.query_scores(q1, k1, scale=0.5)[0, 0, 0], [2.5, -1.0])


def test_attention_drift_is_the_head_averaged_kl_of_each_query_row():
    a, b = 0.7, 0.4
    cur = np.log([[a, 1 - a], [0.5, 0.5]])[None, :, None, :]         # [1 seq][2 rows][1 head][2 pos]
    prev = np.log([[b, 1 - b], [0.5, 0.5]])[None, :, None, :]
    d = pr.attention_drift(cur, prev)
    want = a * math.log(a / b) + (1 - a) * math.log((1 - a) / (1 - b))
    assert d.shape == (1, 2)
    assert d[0, 0] == pytest.approx(want, rel=1e-12) and d[0, 1] == 0.0
