"""GPU parity of every hot-path entry point against the CPU oracle.

Inputs come from the seeded generators (paper_2607_14107_amd.inputs) or are
built here from seeded random numbers; the oracle never sees a value produced
by the HIP path.  Tolerances: fp32 outputs 1e-4 relative, bf16 outputs 2e-2
relative per row (token x head), drift and confidence 1e-4 relative in every
dtype (their arithmetic is fp32 on exactly decoded inputs), integer outputs
and decisions exact.
"""

import math

import numpy as np
import pytest

from oracle import polestar_ref as ref
from paper_2607_14107_amd import inputs
from tests._util import RTOL, assert_drift_close, assert_rows_close, bits_of, ensure_built, from_dev, to_dev

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


_LAYER_CACHE = {}


def layer(cfg_index, subrun=0):
    """Generator inputs + decoded float64 copies + the oracle's prior cache."""
    key = (cfg_index, subrun)
    if key in _LAYER_CACHE:
        return _LAYER_CACHE[key]
    cfg = inputs.CONFIGS[cfg_index]
    x = inputs.layer_inputs(cfg, subrun)
    dec = {k: ref.decode(x[k], cfg.dtype) for k in ("h_prev", "h_cur", "w_q", "w_k", "w_v")}
    shape = (cfg.batch, cfg.seq, cfg.n_kv_heads, cfg.head_dim)
    if cfg_index in (0, 1):
        # prior cache = projection of the previous states, rounded to the cache dtype
        k0 = ref.round_to((dec["h_prev"] @ dec["w_k"].T).reshape(shape), cfg.dtype)
        v0 = ref.round_to((dec["h_prev"] @ dec["w_v"].T).reshape(shape), cfg.dtype)
        kc, vc = bits_of(k0, cfg.dtype), bits_of(v0, cfg.dtype)
    else:
        kc, vc = inputs.random_cache(cfg, subrun)
    out = dict(cfg=cfg, x=x, dec=dec, kc=kc, vc=vc,
               kc_dec=ref.decode(kc, cfg.dtype), vc_dec=ref.decode(vc, cfg.dtype))
    _LAYER_CACHE[key] = out
    return out


def planted_stale(L):
    """The planted cached positions of each sequence, ascending, padded with -1."""
    cfg, x = L["cfg"], L["x"]
    cached = np.ones(cfg.seq, dtype=bool)
    cached[cfg.block_start:cfg.block_start + cfg.block_len] = False
    rows = [np.flatnonzero(x["planted"][b] & cached) for b in range(cfg.batch)]
    k = max(len(r) for r in rows)
    idx = np.full((cfg.batch, k), -1, dtype=np.int32)
    cnt = np.zeros(cfg.batch, dtype=np.int32)
    for b, r in enumerate(rows):
        idx[b, :len(r)] = r
        cnt[b] = len(r)
    return idx, cnt


# ---------------------------------------------------------------------------
# drift
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("cfg_index", [0, 1, 2, 3])
def test_drift_matches_oracle(P, cfg_index):
    L = layer(cfg_index)
    cfg, x, dec = L["cfg"], L["x"], L["dec"]
    got = from_dev(P.drift(to_dev(x["h_cur"], cfg.dtype), to_dev(x["h_prev"], cfg.dtype)))
    want = ref.drift(dec["h_cur"], dec["h_prev"])
    assert_drift_close(got, want)


@pytest.mark.parametrize("rows", [(3, 37), (1, 2100)])
@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("d", [8, 256, 1000, 3584, 4096, 8192, 16384])
def test_drift_exact_zero_and_ragged_rows(P, dtype, d, rows):
    """A row per 256 threads (111 rows) and, from 2048 rows on, per wave or
    128 threads; ragged widths leave lanes or chunks without data."""
    if rows[1] > 1000 and d > 4096:
        pytest.skip("the wide rows are covered at 111 rows")
    g = np.random.default_rng(d + rows[1])
    h = inputs.store(g.standard_normal((*rows, d), dtype=np.float32), dtype)
    ht = to_dev(h, dtype)
    if dtype == "fp32" and d > 8192:
        # fp32 rows above 8192 are outside the register budget: refused on the
        # host before anything is enqueued
        with pytest.raises(P.PolestarError) as e:
            P.drift(ht, ht.clone())
        assert e.value.status == 2   # POLESTAR_ERR_UNSUPPORTED
        return
    zero = from_dev(P.drift(ht, ht.clone()))
    assert np.all(zero == 0.0) and not np.signbit(zero).any()
    h2 = inputs.store(inputs.load_f32(h, dtype) + 0.3 * g.standard_normal(h.shape, dtype=np.float32), dtype)
    got = from_dev(P.drift(to_dev(h2, dtype), ht))
    assert_drift_close(got, ref.drift(ref.decode(h2, dtype), ref.decode(h, dtype)))


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("d", [256, 4096])
def test_drift_outlier_channel(P, dtype, d):
    """One channel of the current state moved by +-100 or +-1000 (a large
    outlier between two steps), on an ordinary channel and on the row's
    maximal channel: the drift must stay finite and match the oracle."""
    g = np.random.default_rng(d + (1 if dtype == "bf16" else 0))
    rows = 16
    base = g.standard_normal((1, rows, d), dtype=np.float32)
    h_prev = inputs.store(base, dtype)
    prev = inputs.load_f32(h_prev, dtype)
    cur = prev + 0.01 * g.standard_normal(prev.shape, dtype=np.float32)
    moves = [100.0, -100.0, 1000.0, -1000.0]
    for r in range(rows - 1):
        c = 5 + 3 * r if r % 2 == 0 else int(np.argmax(prev[0, r]))
        cur[0, r, c] += moves[r % 4]
    h_cur = inputs.store(cur, dtype)        # the last row keeps only the light noise
    got = from_dev(P.drift(to_dev(h_cur, dtype), to_dev(h_prev, dtype)))
    assert np.all(np.isfinite(got))
    want = ref.drift(ref.decode(h_cur, dtype), ref.decode(h_prev, dtype))
    assert_drift_close(got, want)


# ---------------------------------------------------------------------------
# select
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seq,bs,bl", [(96, 64, 32), (768, 512, 32), (1536, 1024, 32),
                                       (2048, 1536, 64), (5000, 100, 64), (1, 0, 0), (33, 33, 0)])
def test_select_bit_exact(P, seq, bs, bl):
    torch = _torch()
    g = np.random.default_rng(seq)
    batch = 3
    vals = np.round(g.standard_normal((batch, seq)) * 3, 1).astype(np.float32)   # many ties
    vals[0, ::7] = -0.0
    vals[1, ::5] = 0.0
    vals[2] = np.abs(vals[2]) * 1e-6
    elig = (g.random((batch, seq)) < 0.8).astype(np.uint8)
    dv = torch.from_numpy(vals).cuda()
    ncand = seq - bl
    for k in sorted({0, 1, min(7, seq), ncand // 4, max(ncand - 1, 0), ncand, seq}):
        for e in (None, elig):
            idx, cnt = P.select(dv, k, bs, bl, None if e is None else torch.from_numpy(e).cuda())
            widx, wcnt = ref.select(vals.astype(np.float64), k, bs, bl, None if e is None else e.astype(bool))
            assert from_dev(cnt).tolist() == wcnt.tolist(), (k, e is None)
            if k > 0:
                assert np.array_equal(from_dev(idx), widx), (k, e is None)


def test_select_recovers_planted_set_from_gpu_drift(P):
    for cfg_index in (0, 1, 3):
        L = layer(cfg_index)
        cfg, x = L["cfg"], L["x"]
        d = P.drift(to_dev(x["h_cur"], cfg.dtype), to_dev(x["h_prev"], cfg.dtype))
        want_idx, want_cnt = planted_stale(L)
        k = want_idx.shape[1]
        idx, cnt = P.select(d, k, cfg.block_start, cfg.block_len)
        got_idx, got_cnt = from_dev(idx), from_dev(cnt)
        for b in range(cfg.batch):
            chosen = set(got_idx[b, :got_cnt[b]].tolist())
            assert set(want_idx[b, :want_cnt[b]].tolist()) <= chosen, (cfg_index, b)


# ---------------------------------------------------------------------------
# refresh
# ---------------------------------------------------------------------------

def _run_refresh(P, L, idx, cnt, bs, bl):
    cfg, x = L["cfg"], L["x"]
    torch = _torch()
    kc, vc = to_dev(L["kc"], cfg.dtype), to_dev(L["vc"], cfg.dtype)
    ti = torch.from_numpy(idx).cuda() if idx is not None and idx.shape[1] > 0 else None
    tc = torch.from_numpy(cnt).cuda() if ti is not None else None
    P.refresh_kv(to_dev(x["h_cur"], cfg.dtype), ti, tc, bs, bl, to_dev(x["w_k"], cfg.dtype),
                 to_dev(x["w_v"], cfg.dtype), kc, vc)
    return from_dev(kc), from_dev(vc)


def _check_refresh(L, kc_bits, vc_bits, idx, cnt, bs, bl, sample=None):
    cfg, dec = L["cfg"], L["dec"]
    rows = ref.refresh_rows(idx, cnt, bs, bl)
    shape = (cfg.n_kv_heads, cfg.head_dim)
    rtol = RTOL[cfg.dtype]
    for b in range(cfg.batch):
        r = np.asarray(rows[b], dtype=np.int64)
        keep = np.setdiff1d(np.arange(cfg.seq), r)
        assert np.array_equal(kc_bits[b, keep], L["kc"][b, keep]), "untouched K rows changed"
        assert np.array_equal(vc_bits[b, keep], L["vc"][b, keep]), "untouched V rows changed"
        if sample is not None and r.size > sample:
            r = np.random.default_rng(b).choice(r, size=sample, replace=False)
        if r.size == 0:
            continue
        kw = ref.project_rows(dec["h_cur"][b], dec["w_k"], r).reshape(r.size, *shape)
        vw = ref.project_rows(dec["h_cur"][b], dec["w_v"], r).reshape(r.size, *shape)
        kg = ref.decode(kc_bits[b, r], cfg.dtype)
        vg = ref.decode(vc_bits[b, r], cfg.dtype)
        assert_rows_close(kg, kw, rtol, f"K rows of sequence {b}")
        assert_rows_close(vg, vw, rtol, f"V rows of sequence {b}")
        if cfg.dtype == "bf16":
            # rounding of an fp32 accumulation: within one bf16 step of the exact value
            step = 2.0 ** (np.floor(np.log2(np.maximum(np.abs(kw), 1e-30))) - 7)
            assert np.mean(np.abs(kg - kw) <= step) > 0.999


@pytest.mark.parametrize("cfg_index,subrun", [(0, 0), (1, 0), (1, 1), (1, 2)])
def test_refresh_planted_rows_matches_oracle(P, cfg_index, subrun):
    L = layer(cfg_index, subrun)
    cfg = L["cfg"]
    idx, cnt = planted_stale(L)
    kb, vb = _run_refresh(P, L, idx, cnt, cfg.block_start, cfg.block_len)
    _check_refresh(L, kb, vb, idx, cnt, cfg.block_start, cfg.block_len)


@pytest.mark.parametrize("cfg_index", [0, 1])
def test_refresh_every_position_equals_full_recompute(P, cfg_index):
    L = layer(cfg_index)
    cfg = L["cfg"]
    idx = np.tile(np.arange(cfg.seq, dtype=np.int32), (cfg.batch, 1))
    cnt = np.full(cfg.batch, cfg.seq, dtype=np.int32)
    kb, vb = _run_refresh(P, L, idx, cnt, cfg.block_start, cfg.block_len)
    _check_refresh(L, kb, vb, idx, cnt, cfg.block_start, cfg.block_len)


def test_refresh_nothing_leaves_cache_untouched(P):
    L = layer(1)
    cfg = L["cfg"]
    idx = np.full((cfg.batch, 16), -1, dtype=np.int32)
    cnt = np.zeros(cfg.batch, dtype=np.int32)
    kb, vb = _run_refresh(P, L, idx, cnt, cfg.block_start, 0)
    assert np.array_equal(kb, L["kc"]) and np.array_equal(vb, L["vc"])
    kb, vb = _run_refresh(P, L, None, None, cfg.block_start, 0)
    assert np.array_equal(kb, L["kc"]) and np.array_equal(vb, L["vc"])


@pytest.mark.parametrize("cfg_index,subrun", [(2, 0), (2, 1), (2, 2), (3, 0)])
def test_refresh_large_configs_sampled(P, cfg_index, subrun):
    L = layer(cfg_index, subrun)
    cfg = L["cfg"]
    idx, cnt = planted_stale(L)
    kb, vb = _run_refresh(P, L, idx, cnt, cfg.block_start, cfg.block_len)
    _check_refresh(L, kb, vb, idx, cnt, cfg.block_start, cfg.block_len, sample=48)


@pytest.mark.parametrize("counts,k_max", [([33], 33), ([57], 100), ([128], 128), ([129], 129), ([40, 13], 40),
                                          ([300], 320), ([600, 250], 600), ([700], 735)])
def test_refresh_row_counts_around_one_tile(P, counts, k_max):
    """Refresh row sets on the LLaDA-8B-shaped weights: 65..160 rows (one row
    tile, the DMA-staged GEMM), the first two-tile case, and 352..1264 rows
    (192 x 256 tiles, unsplit or K split in 2 or 4, the last row tile
    ragged); slots
    past a sequence's count and an out-of-range index refresh nothing."""
    torch = _torch()
    L = layer(1)
    cfg, x, dec = L["cfg"], L["x"], L["dec"]
    batch = len(counts)
    bs, bl = cfg.block_start, cfg.block_len
    h_bits = np.concatenate([x["h_cur"], x["h_prev"]], axis=0)[:batch]
    h_dec = np.concatenate([dec["h_cur"], dec["h_prev"]], axis=0)[:batch]
    g = np.random.default_rng(k_max + batch)
    outside = np.setdiff1d(np.arange(cfg.seq), np.arange(bs, bs + bl))
    idx = np.full((batch, k_max), -1, dtype=np.int32)
    for b, c in enumerate(counts):
        idx[b, :c] = np.sort(g.choice(outside, size=c, replace=False))
    if batch > 1:
        idx[1, 5] = cfg.seq + 3                       # out of range: refreshes nothing
    cnt = np.asarray(counts, dtype=np.int32)
    shape = (batch, cfg.seq, cfg.n_kv_heads, cfg.head_dim)
    kc = torch.zeros(shape, dtype=torch.bfloat16, device="cuda")
    vc = torch.zeros(shape, dtype=torch.bfloat16, device="cuda")
    P.refresh_kv(to_dev(h_bits, cfg.dtype), torch.from_numpy(idx).cuda(), torch.from_numpy(cnt).cuda(), bs, bl,
                 to_dev(x["w_k"], cfg.dtype), to_dev(x["w_v"], cfg.dtype), kc, vc)
    kg, vg = from_dev(kc), from_dev(vc)
    for b in range(batch):
        valid = [int(i) for i in idx[b, :cnt[b]] if 0 <= i < cfg.seq]
        rows = np.asarray(sorted(set(valid) | set(range(bs, bs + bl))), dtype=np.int64)
        keep = np.setdiff1d(np.arange(cfg.seq), rows)
        assert not kg[b, keep].any() and not vg[b, keep].any(), "rows outside the refresh set were written"
        kw = ref.project_rows(h_dec[b], dec["w_k"], rows).reshape(rows.size, cfg.n_kv_heads, cfg.head_dim)
        vw = ref.project_rows(h_dec[b], dec["w_v"], rows).reshape(rows.size, cfg.n_kv_heads, cfg.head_dim)
        assert_rows_close(ref.decode(kg[b, rows], "bf16"), kw, RTOL["bf16"], f"K rows of sequence {b}")
        assert_rows_close(ref.decode(vg[b, rows], "bf16"), vw, RTOL["bf16"], f"V rows of sequence {b}")


# ---------------------------------------------------------------------------
# attend
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("cfg_index", [0, 1, 2, 3])
def test_attend_matches_oracle(P, cfg_index):
    torch = _torch()
    L = layer(cfg_index)
    cfg, x, dec = L["cfg"], L["x"], L["dec"]
    lse = torch.empty((cfg.batch, cfg.n_heads, cfg.block_len), dtype=torch.float32, device="cuda")
    out, q = P.attend(to_dev(x["h_cur"], cfg.dtype), to_dev(x["w_q"], cfg.dtype),
                      to_dev(L["kc"], cfg.dtype), to_dev(L["vc"], cfg.dtype),
                      cfg.block_start, cfg.block_len, cfg.n_heads, lse=lse)
    rtol = RTOL[cfg.dtype]
    q_want = ref.q_project(dec["h_cur"], dec["w_q"], cfg.block_start, cfg.block_len, cfg.n_heads, cfg.head_dim)
    assert_rows_close(ref.decode(from_dev(q), cfg.dtype), q_want, rtol, "Q")
    o_want, _ = ref.attend(q_want, L["kc_dec"], L["vc_dec"])
    assert_rows_close(ref.decode(from_dev(out), cfg.dtype), o_want, rtol, "attention output")
    # The GPU attends with Q as stored in the run dtype; the oracle does the
    # same with its own float64 projection rounded to that dtype.
    o_st, lse_st = ref.attend(ref.round_to(q_want, cfg.dtype), L["kc_dec"], L["vc_dec"])
    assert_rows_close(ref.decode(from_dev(out), cfg.dtype), o_st, rtol, "attention output (stored Q)")
    np.testing.assert_allclose(from_dev(lse), lse_st, rtol=rtol, atol=rtol)


@pytest.mark.parametrize("cfg_index", [0, 1, 2, 3])
def test_project_q_matches_oracle_and_attend(P, cfg_index):
    """The stand-alone projection equals the oracle's and, bit for bit, the
    projection polestar_attend makes itself (same kernels, same plan)."""
    L = layer(cfg_index)
    cfg, x, dec = L["cfg"], L["x"], L["dec"]
    h = to_dev(x["h_cur"], cfg.dtype)
    wq = to_dev(x["w_q"], cfg.dtype)
    q = P.project_q(h, wq, cfg.block_start, cfg.block_len, cfg.n_heads)
    want = ref.q_project(dec["h_cur"], dec["w_q"], cfg.block_start, cfg.block_len, cfg.n_heads, cfg.head_dim)
    assert_rows_close(ref.decode(from_dev(q), cfg.dtype), want, RTOL[cfg.dtype], "Q")
    _, q_att = P.attend(h, wq, to_dev(L["kc"], cfg.dtype), to_dev(L["vc"], cfg.dtype),
                        cfg.block_start, cfg.block_len, cfg.n_heads)
    assert np.array_equal(from_dev(q), from_dev(q_att))


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("batch,seq,bs,bl,d,H,hd", [(1, 40, 7, 33, 256, 2, 64), (3, 70, 60, 10, 512, 1, 128),
                                                    (5, 20, 0, 20, 1024, 4, 64),
                                                    (2, 70, 5, 48, 1280, 8, 128),     # bf16: splits of 10 stages
                                                    (1, 200, 50, 100, 1792, 4, 128)])  # bf16: splits of 14 stages
def test_project_q_ragged_shapes(P, dtype, batch, seq, bs, bl, d, H, hd):
    """Row tiles with a ragged tail, more than 64 rows (split-K path), and a
    block at the start of the sequence."""
    if dtype == "fp32" and d % 64:
        pytest.skip("fp32 rows need d % 64 == 0")
    g = np.random.default_rng(batch * 1000 + seq)
    h = inputs.store(g.standard_normal((batch, seq, d), dtype=np.float32), dtype)
    wq = inputs.store(0.05 * g.standard_normal((H * hd, d), dtype=np.float32), dtype)
    q = P.project_q(to_dev(h, dtype), to_dev(wq, dtype), bs, bl, H)
    want = ref.q_project(ref.decode(h, dtype), ref.decode(wq, dtype), bs, bl, H, hd)
    assert_rows_close(ref.decode(from_dev(q), dtype), want, RTOL[dtype], "Q")


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("batch,seq,bs,bl,H,Hkv,hd", [
    (2, 50, 10, 20, 4, 2, 64), (1, 300, 0, 45, 3, 1, 128), (3, 129, 97, 32, 2, 2, 128), (1, 1, 0, 1, 2, 1, 64),
    # bf16 with >= 4 (head, 32-query group) pairs per KV head: the grouped-head kernel
    (2, 130, 5, 40, 8, 2, 128),      # 8 pairs, one 8-wave workgroup per KV head and split
    (1, 77, 0, 64, 7, 1, 64),        # 14 pairs in two row blocks (two idle waves), ragged keys
    (3, 33, 1, 32, 4, 1, 128),       # 4 pairs, 4-wave workgroups
    (2, 2100, 0, 20, 6, 1, 128),     # 6 pairs (two idle waves), many key splits
    (1, 1, 0, 1, 8, 2, 64),          # a single key
])
def test_attend_small_shapes_with_given_queries(P, dtype, batch, seq, bs, bl, H, Hkv, hd):
    """Ragged key tiles and query groups, GQA grouping, a single key."""
    g = np.random.default_rng(seq * 7 + bl)
    q = inputs.store(g.standard_normal((batch, bl, H, hd), dtype=np.float32), dtype)
    kc = inputs.store(g.standard_normal((batch, seq, Hkv, hd), dtype=np.float32), dtype)
    vc = inputs.store(g.standard_normal((batch, seq, Hkv, hd), dtype=np.float32), dtype)
    torch = _torch()
    lse = torch.empty((batch, H, bl), dtype=torch.float32, device="cuda")
    out, _ = P.attend(None, None, to_dev(kc, dtype), to_dev(vc, dtype), bs, bl, H,
                      q_buf=to_dev(q, dtype), lse=lse)
    o_want, lse_want = ref.attend(ref.decode(q, dtype), ref.decode(kc, dtype), ref.decode(vc, dtype))
    assert_rows_close(ref.decode(from_dev(out), dtype), o_want, RTOL[dtype], "output")
    np.testing.assert_allclose(from_dev(lse), lse_want, rtol=RTOL[dtype], atol=RTOL[dtype])
    if seq == 1:   # a single key: the output is its value
        want = np.broadcast_to(ref.decode(vc, dtype)[:, :1, np.arange(H) // (H // Hkv)], o_want.shape)
        assert_rows_close(ref.decode(from_dev(out), dtype), want, RTOL[dtype], "single key")


@pytest.mark.parametrize("dtype,batch,seq,bl,H,Hkv,hd", [
    ("bf16", 2, 700, 32, 4, 4, 128),     # one (head, query group) pair per KV head: attend_kernel
    ("bf16", 2, 700, 64, 8, 2, 128),     # grouped-head kernel, 8 pairs per KV head
    ("bf16", 1, 2100, 32, 6, 1, 64),     # grouped, many key splits
    ("fp32", 1, 300, 20, 2, 1, 64),
])
def test_attend_late_dominant_keys(P, dtype, batch, seq, bl, H, Hkv, hd):
    """Keys late in the sequence whose scores exceed everything before them:
    one by about 4 nats (below the kernels' lazy rescale threshold of 8 in
    log2 units, so probabilities above 1 are accumulated against the old
    reference) and one by about 40 nats (the output and l are rescaled to a
    new reference).  Queries share one direction per head so that every
    query sees both jumps."""
    g = np.random.default_rng(seq + 31 * H + hd)
    u = g.standard_normal((batch, 1, H, hd)).astype(np.float32)
    u /= np.linalg.norm(u, axis=-1, keepdims=True)
    qf = 3.0 * u + 0.05 * g.standard_normal((batch, bl, H, hd)).astype(np.float32)
    kf = 0.2 * g.standard_normal((batch, seq, Hkv, hd)).astype(np.float32)
    vf = g.standard_normal((batch, seq, Hkv, hd)).astype(np.float32)
    G = H // Hkv
    ukv = u[:, 0].reshape(batch, Hkv, G, hd).mean(axis=2)             # the group's shared direction
    ukv /= np.linalg.norm(ukv, axis=-1, keepdims=True)
    # score = q.k / sqrt(hd) with |q| ~ 3: a key c * ukv scores about 3 c / sqrt(hd) * cos
    mid, late = int(seq * 0.4), int(seq * 0.85)
    kf[:, mid] = (4.0 * math.sqrt(hd) / 3.0) * ukv
    kf[:, late] = (40.0 * math.sqrt(hd) / 3.0) * ukv
    q, kc, vc = (inputs.store(a, dtype) for a in (qf, kf, vf))
    torch = _torch()
    lse = torch.empty((batch, H, bl), dtype=torch.float32, device="cuda")
    out, _ = P.attend(None, None, to_dev(kc, dtype), to_dev(vc, dtype), 0, bl, H, q_buf=to_dev(q, dtype), lse=lse)
    o_want, lse_want = ref.attend(ref.decode(q, dtype), ref.decode(kc, dtype), ref.decode(vc, dtype))
    assert_rows_close(ref.decode(from_dev(out), dtype), o_want, RTOL[dtype], "output")
    np.testing.assert_allclose(from_dev(lse), lse_want, rtol=RTOL[dtype], atol=RTOL[dtype])
    # the dominant key carries almost all of the weight
    vl = ref.decode(vc, dtype)[:, late][:, None, np.arange(H) // G]
    assert np.abs(o_want - vl).max() < 0.1 * np.abs(vl).max()


def test_attend_key_order_and_uniform_scores(P):
    torch = _torch()
    L = layer(1)
    cfg, x = L["cfg"], L["x"]
    kc, vc = L["kc"], L["vc"]
    q = to_dev(x["h_cur"], cfg.dtype)
    out, qb = P.attend(q, to_dev(x["w_q"], cfg.dtype), to_dev(kc, cfg.dtype), to_dev(vc, cfg.dtype),
                       cfg.block_start, cfg.block_len, cfg.n_heads)
    perm = np.random.default_rng(5).permutation(cfg.seq)
    out_p, _ = P.attend(None, None, to_dev(np.ascontiguousarray(kc[:, perm]), cfg.dtype),
                        to_dev(np.ascontiguousarray(vc[:, perm]), cfg.dtype), cfg.block_start,
                        cfg.block_len, cfg.n_heads, q_buf=qb.clone())
    a = ref.decode(from_dev(out), cfg.dtype)
    assert_rows_close(ref.decode(from_dev(out_p), cfg.dtype), a, 1e-2, "permuted keys")
    # zero queries: equal scores, the output is the mean of V
    zq = torch.zeros_like(qb)
    out0, _ = P.attend(None, None, to_dev(kc, cfg.dtype), to_dev(vc, cfg.dtype), cfg.block_start,
                       cfg.block_len, cfg.n_heads, q_buf=zq)
    mean_v = L["vc_dec"].mean(axis=1)                      # [b][Hkv][hd]
    want = np.broadcast_to(mean_v[:, None], (cfg.batch, cfg.block_len, cfg.n_heads, cfg.head_dim))
    assert_rows_close(ref.decode(from_dev(out0), cfg.dtype), want, RTOL[cfg.dtype], "mean of V")


# ---------------------------------------------------------------------------
# commit
# ---------------------------------------------------------------------------

TARGET_CONF = (0.97, 0.92, 0.88, 0.85, 0.80, 0.70)


def coverage_inputs(cfg, subrun=0):
    """Decision-coverage inputs: spiked logits on 25% of the tokens with
    confidences around tau_s, and drift/history placing delta - tau_d on both
    sides of zero with margin >= 1e-3.  Built with the oracle only."""
    x = inputs.layer_inputs(cfg, subrun) if cfg.index in (0, 1) else None
    lg = inputs.logits(cfg, subrun) if x is None else x["logits"]
    lgd = ref.decode(lg, cfg.dtype).copy()
    spikes = inputs.spike_rows(cfg, subrun)
    g = np.random.default_rng(inputs.seed_of(cfg.index, subrun, 6) + 1)

    def spike(b, j, c):
        v = int(np.argmax(lgd[b, j]))
        rest = np.delete(lgd[b, j], v)
        m = rest.max()
        lse_rest = m + math.log(np.exp(rest - m).sum())
        lgd[b, j, v] = lse_rest + math.log(c / (1.0 - c))

    n = 0
    for b in range(cfg.batch):
        for j in np.flatnonzero(spikes[b]):
            spike(b, j, TARGET_CONF[n % len(TARGET_CONF)])
            n += 1
    for _ in range(3):
        lg_bits = bits_of(ref.round_to(lgd, cfg.dtype), cfg.dtype)
        lgd = ref.decode(lg_bits, cfg.dtype)
        token, conf = ref.confidence(lgd, -1)
        conf32 = conf.astype(np.float32)
        near = np.argwhere(np.abs(conf32 - np.float32(cfg.tau_s)) <= 2e-3)
        if near.size == 0:
            break
        for b, j in near:          # keep every confidence clear of the threshold
            spike(b, j, 0.97)
    assert np.all(np.abs(conf32 - np.float32(cfg.tau_s)) > 1e-3)
    h = cfg.hist_depth
    hist = np.zeros((cfg.batch, h, cfg.block_len), dtype=np.float32)
    hist_len = np.full(cfg.batch, h, dtype=np.int32)
    hist_len[0] = 2 if cfg.batch > 1 else h
    mu = g.uniform(0.025, 0.05, size=(cfg.batch, cfg.block_len)).astype(np.float32)
    for b in range(cfg.batch):
        for r in range(hist_len[b]):
            hist[b, r] = mu[b]
    tau_d = np.float32(cfg.alpha) * (np.float32(cfg.tau_s) - conf32) ** 2
    sign = np.where(g.random((cfg.batch, cfg.block_len)) < 0.5, 1.0, -1.0).astype(np.float32)
    margin = g.uniform(0.002, 0.02, size=sign.shape).astype(np.float32)
    delta = (mu + tau_d + sign * margin).astype(np.float32)   # >= 0: mu >= margin
    drift = np.zeros((cfg.batch, cfg.seq), dtype=np.float32)
    drift[:, cfg.block_start:cfg.block_start + cfg.block_len] = delta
    masked = (g.random((cfg.batch, cfg.block_len)) < 0.9).astype(np.uint8)
    return lg_bits, token, conf, drift, hist, hist_len, masked


def _run_commit(P, cfg, lg_bits, drift, hist, hist_len, masked, force_one, mask_id=-1):
    torch = _torch()
    th = torch.from_numpy(hist.copy()).cuda() if hist is not None else None
    tl = torch.from_numpy(hist_len.copy()).cuda() if hist_len is not None else None
    td = torch.from_numpy(drift).cuda() if drift is not None else None
    tok, conf, cm = P.commit(to_dev(lg_bits, cfg.dtype), torch.from_numpy(masked).cuda(), td,
                             cfg.block_start, th, tl, mask_id, cfg.tau_s, cfg.alpha, force_one)
    return (from_dev(tok), from_dev(conf), from_dev(cm).astype(bool),
            None if th is None else from_dev(th), None if tl is None else from_dev(tl))


def _oracle_commit(cfg, conf, drift, hist, hist_len, masked, force_one):
    h = hist.shape[1] if hist is not None else 0
    delta = drift[:, cfg.block_start:cfg.block_start + cfg.block_len] if drift is not None \
        else np.zeros((cfg.batch, cfg.block_len), np.float32)
    hh = hist if hist is not None else np.zeros((cfg.batch, 0, cfg.block_len), np.float32)
    hl = hist_len if hist_len is not None else np.zeros(cfg.batch, np.int32)
    return ref.commit_rule(conf.astype(np.float32), delta.astype(np.float32), masked.astype(bool),
                           hh, hl, h, cfg.tau_s, cfg.alpha, force_one)


@pytest.mark.parametrize("cfg_index", [0, 1, 2, 3])
def test_commit_decision_coverage(P, cfg_index):
    cfg = inputs.CONFIGS[cfg_index]
    lg_bits, token, conf, drift, hist, hist_len, masked = coverage_inputs(cfg)
    for force_one in (False, True):
        gt, gc, gm, gh, gl = _run_commit(P, cfg, lg_bits, drift, hist, hist_len, masked, force_one)
        assert np.array_equal(gt, token)
        np.testing.assert_allclose(gc, conf, rtol=1e-4)
        wm, wh, wl = _oracle_commit(cfg, conf, drift, hist, hist_len, masked, force_one)
        assert np.array_equal(gm, wm)
        assert np.array_equal(gh, wh) and np.array_equal(gl, wl)
    # both branches of the rule and both outcomes occur
    assert gm.any() and (~gm & masked.astype(bool)).any()
    assert (conf > cfg.tau_s).any() and ((conf < cfg.tau_s) & gm).any()


@pytest.mark.parametrize("cfg_index", [0, 1])
def test_commit_plain_config_logits(P, cfg_index):
    """The configuration's own N(0, s) logits with the generator's history, a
    [MASK] id, the drift branch off and h = 0."""
    L = layer(cfg_index)
    cfg, x = L["cfg"], L["x"]
    lgd = ref.decode(x["logits"], cfg.dtype)
    drift = np.zeros((cfg.batch, cfg.seq), np.float32)
    drift[:, cfg.block_start:cfg.block_start + cfg.block_len] = np.float32(1e-4)
    for mask_id in (-1, 5):
        token, conf = ref.confidence(lgd, mask_id)
        gt, gc, gm, gh, gl = _run_commit(P, cfg, x["logits"], drift, x["hist"], x["hist_len"],
                                         x["masked"], True, mask_id)
        assert np.array_equal(gt, token)
        np.testing.assert_allclose(gc, conf, rtol=1e-4)
        wm, wh, wl = _oracle_commit(cfg, conf, drift, x["hist"], x["hist_len"], x["masked"], True)
        assert np.array_equal(gm, wm) and np.array_equal(gh, wh) and np.array_equal(gl, wl)
    # drift branch off: confidence rule only; no history
    token, conf = ref.confidence(lgd, -1)
    gt, gc, gm, gh, gl = _run_commit(P, cfg, x["logits"], None, None, None, x["masked"], False)
    assert np.array_equal(gt, token)
    assert np.array_equal(gm, (conf > cfg.tau_s) & x["masked"].astype(bool))


@pytest.mark.parametrize("cfg_index", [0, 1])
def test_commit_argmax_edges(P, cfg_index):
    """Argmax corner cases of the vocabulary scan against the oracle: ties
    (the lowest id wins, within one vocabulary slice and across slices), the
    [MASK] id holding the strict maximum, long -inf runs (so that a lane's
    and a slice's first elements are -inf), a row that is -inf except for its
    last element, -inf rows with a tie among their few finite entries, a
    maximum reached twice by one lane (16-byte chunks 256 apart), the [MASK]
    id tied with its neighbour, and a row that is -inf but for [MASK]."""
    L = layer(cfg_index)
    cfg, x = L["cfg"], L["x"]
    lg = x["logits"].copy()
    V = lg.shape[-1]
    mask_id = 5
    bf16 = cfg.dtype == "bf16"

    def val(v):
        return np.uint16(np.float32(v).view(np.uint32) >> 16) if bf16 else np.float32(v)

    lg[0, 0, 3] = lg[0, 0, V - 1] = val(60.0)                                    # tie: first and last id
    lg[0, 1, V // 3] = lg[0, 1, V // 3 + 1] = lg[0, 1, 2 * V // 3] = val(60.0)   # ties in two slices
    lg[0, 2, mask_id] = val(70.0)                                               # [MASK] is the maximum
    lg[0, 2, V // 2] = val(65.0)
    lg[0, 3, : V // 2] = val(-np.inf)                                           # -inf first half
    lg[0, 3, V - 7] = val(50.0)
    lg[0, 4, :] = val(-np.inf)                                                  # only the last id finite
    lg[0, 4, V - 1] = val(0.5)
    lg[0, 5, :] = val(-np.inf)                                                  # tie among three finite ids
    for pos in (V // 7, V // 2, V - 3):
        lg[0, 5, pos] = val(1.0)
    E = 8 if bf16 else 4                                                        # ids per 16-byte chunk
    lg[0, 6, 16] = val(55.0)                                                    # one lane, chunks 0 and 256 of it
    if 16 + 256 * E < V:
        lg[0, 6, 16 + 256 * E] = val(55.0)
    lg[0, 7, mask_id] = lg[0, 7, mask_id + 1] = val(80.0)                       # [MASK] tied with the next id
    lg[0, 8, :] = val(-np.inf)                                                  # only [MASK] finite
    lg[0, 8, mask_id] = val(3.0)
    token, conf = ref.confidence(ref.decode(lg, cfg.dtype), mask_id)
    assert token[0, :9].tolist() == [3, V // 3, V // 2, V - 7, V - 1, V // 7, 16, mask_id + 1, 0]
    gt, gc, _, _, _ = _run_commit(P, cfg, lg, None, None, None, x["masked"], False, mask_id)
    assert np.array_equal(gt, token)
    np.testing.assert_allclose(gc, conf, rtol=1e-4)


@pytest.mark.parametrize("cfg_index", [0, 1, 2, 3])
def test_suffix_commit(P, cfg_index):
    """Suffix-block commit: the coverage logits stand for the final-layer packet
    rows of the suffix window; the packet carries a seeded subset of it."""
    torch = _torch()
    cfg = inputs.CONFIGS[cfg_index]
    lg_bits, token, conf, _, _, _, masked = coverage_inputs(cfg)
    g = np.random.default_rng(inputs.seed_of(cfg.index, 0, 7))
    s0 = cfg.block_start + cfg.block_len
    n = cfg.block_len
    k = cfg.block_len
    idx = np.full((cfg.batch, 2 * k), -1, np.int64)
    cnt = np.zeros(cfg.batch, np.int64)
    hi = (conf > cfg.tau_s) & masked.astype(bool)
    for b in range(cfg.batch):
        # the packet: half of the confident masked suffix rows, a random third
        # of the others, and rows outside the suffix window
        h = np.flatnonzero(hi[b])
        lo = np.flatnonzero(~hi[b])
        inside = np.concatenate([h[: (len(h) + 1) // 2], g.choice(lo, size=len(lo) // 3, replace=False)])
        outside = g.choice(np.arange(max(0, s0 - n), s0), size=min(n // 4, s0), replace=False)
        rows = np.unique(np.concatenate([s0 + inside, outside]))
        idx[b, :len(rows)], cnt[b] = rows, len(rows)
    eligible = ref.suffix_eligible(idx, cnt, s0, n)
    assert eligible.any() and (~eligible).any()
    for mask_id in (-1, 3):
        want_tok, want_conf = ref.confidence(ref.decode(lg_bits, cfg.dtype), mask_id)
        gt, gc, gm = P.suffix_commit(to_dev(lg_bits, cfg.dtype), torch.from_numpy(masked).cuda(),
                                     torch.from_numpy(eligible.astype(np.uint8)).cuda(), mask_id, cfg.tau_s)
        gt, gc, gm = from_dev(gt), from_dev(gc), from_dev(gm).astype(bool)
        assert np.array_equal(gt, want_tok)
        np.testing.assert_allclose(gc, want_conf, rtol=1e-4)
        want = ref.suffix_commit_rule(want_conf.astype(np.float32), masked.astype(bool), eligible, cfg.tau_s)
        assert np.array_equal(gm, want)
    # both outcomes among eligible masked rows
    em = eligible & masked.astype(bool)
    assert gm.any() and (em & ~gm).any()


# ---------------------------------------------------------------------------
# whole step
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("cfg_index,subrun", [(0, 0), (1, 1)])
def test_layer_step_end_to_end_and_deterministic(P, cfg_index, subrun):
    torch = _torch()
    L = layer(cfg_index, subrun)
    cfg, x = L["cfg"], L["x"]
    dt = torch.float32 if cfg.dtype == "fp32" else torch.bfloat16
    step = P.Step(batch=cfg.batch, seq=cfg.seq, d=cfg.d, n_heads=cfg.n_heads, n_kv_heads=cfg.n_kv_heads,
                  head_dim=cfg.head_dim, block_start=cfg.block_start, block_len=cfg.block_len,
                  vocab=cfg.vocab, k=x["k"], dtype=dt)
    dev = {k: to_dev(x[k], cfg.dtype) for k in ("h_cur", "h_prev", "w_q", "w_k", "w_v", "logits")}
    results = []
    for _ in range(2):
        kc, vc = to_dev(L["kc"], cfg.dtype), to_dev(L["vc"], cfg.dtype)
        hist = torch.from_numpy(x["hist"].copy()).cuda()
        hl = torch.from_numpy(x["hist_len"].copy()).cuda()
        step.run(dev["h_cur"], dev["h_prev"], dev["w_q"], dev["w_k"], dev["w_v"], kc, vc, dev["logits"],
                 torch.from_numpy(x["masked"]).cuda(), hist, hl, force_one=True)
        torch.cuda.synchronize()
        results.append({k: from_dev(v) for k, v in dict(
            drift=step.drift, idx=step.stale_idx, cnt=step.stale_count, kc=kc, vc=vc, out=step.out,
            lse=step.lse, token=step.token, conf=step.conf, commit=step.commit, hist=hist).items()})
    a, b = results
    for k in a:
        assert np.array_equal(a[k], b[k]), f"run-to-run difference in {k}"
    w = ref.layer_step(L["dec"]["h_cur"], L["dec"]["h_prev"], L["dec"]["w_q"], L["dec"]["w_k"],
                       L["dec"]["w_v"], L["kc_dec"], L["vc_dec"], k=x["k"], block_start=cfg.block_start,
                       block_len=cfg.block_len, n_heads=cfg.n_heads, n_kv_heads=cfg.n_kv_heads,
                       head_dim=cfg.head_dim, cache_dtype=cfg.dtype)
    assert_drift_close(a["drift"], w["drift"])
    assert np.array_equal(a["idx"], w["stale_idx"]) and np.array_equal(a["cnt"], w["stale_count"])
    rtol = RTOL[cfg.dtype]
    assert_rows_close(ref.decode(a["kc"], cfg.dtype), w["k_exact"], rtol, "K cache")
    assert_rows_close(ref.decode(a["vc"], cfg.dtype), w["v_exact"], rtol, "V cache")
    assert_rows_close(ref.decode(a["out"], cfg.dtype), w["out"], rtol, "attention")
    token, conf = ref.confidence(ref.decode(x["logits"], cfg.dtype), -1)
    assert np.array_equal(a["token"], token)
    np.testing.assert_allclose(a["conf"], conf, rtol=1e-4)


# ---------------------------------------------------------------------------
# fused step == the six calls
# ---------------------------------------------------------------------------

def _step_inputs(cfg, x, kc, vc):
    torch = _torch()
    dev = {n: to_dev(x[n], cfg.dtype) for n in ("h_cur", "h_prev", "w_q", "w_k", "w_v", "logits")}
    dev["k_cache"], dev["v_cache"] = to_dev(kc, cfg.dtype), to_dev(vc, cfg.dtype)
    dev["masked"] = torch.from_numpy(x["masked"]).cuda()
    dev["hist"] = torch.from_numpy(x["hist"].copy()).cuda()
    dev["hist_len"] = torch.from_numpy(x["hist_len"].copy()).cuda()
    return dev


def _run_both(P, cfg, x, kc, vc, k, force_one=True):
    """Outputs of Step.run (polestar_step) and Step.run_calls on identical inputs."""
    torch = _torch()
    dt = torch.float32 if cfg.dtype == "fp32" else torch.bfloat16
    res = []
    for fused in (True, False):
        st = P.Step(batch=cfg.batch, seq=cfg.seq, d=cfg.d, n_heads=cfg.n_heads, n_kv_heads=cfg.n_kv_heads,
                    head_dim=cfg.head_dim, block_start=cfg.block_start, block_len=cfg.block_len,
                    vocab=cfg.vocab, k=k, dtype=dt)
        v = _step_inputs(cfg, x, kc, vc)
        run = st.run if fused else st.run_calls
        run(v["h_cur"], v["h_prev"], v["w_q"], v["w_k"], v["w_v"], v["k_cache"], v["v_cache"], v["logits"],
            v["masked"], v["hist"], v["hist_len"], force_one=force_one)
        torch.cuda.synchronize()
        out = dict(drift=st.drift, cnt=st.stale_count, q=st.q_buf, out=st.out, lse=st.lse, token=st.token,
                   conf=st.conf, commit=st.commit, kc=v["k_cache"], vc=v["v_cache"], hist=v["hist"],
                   hist_len=v["hist_len"])
        if k > 0:
            out["idx"] = st.stale_idx
        res.append({n: from_dev(t) for n, t in out.items()})
    return res


def _assert_same(a, b):
    for n in a:
        assert np.array_equal(a[n].view(np.uint8) if a[n].dtype != np.uint8 else a[n],
                              b[n].view(np.uint8) if b[n].dtype != np.uint8 else b[n]), f"fused step differs in {n}"


@pytest.mark.parametrize("cfg_index,subrun", [(0, 0), (1, 1), (2, 0), (2, 1), (3, 0)])
def test_step_fused_equals_calls_on_configs(P, cfg_index, subrun):
    """Configs 0-1 take the six fused launches with a Q projection of up to
    64 rows; 2-3 the front with two 128-row projection tiles (config 2's
    eight select workgroups overflow one round); config 2 at 10% stale also
    puts the Q reduction into its unsplit tile-kernel refresh (five launches).
    Either way the results equal the six calls bit for bit."""
    L = layer(cfg_index, subrun)
    a, b = _run_both(P, L["cfg"], L["x"], L["kc"], L["vc"], int(L["x"]["k"]))
    _assert_same(a, b)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("batch,seq,bs,bl,d,H,Hkv,hd,vocab,k", [
    (1, 100, 40, 30, 256, 2, 1, 64, 1000, 9),       # 1 key per thread, ragged block, GQA
    (2, 700, 600, 32, 256, 4, 4, 64, 2048, 70),     # 3 keys per thread, 64 query rows (MT 4)
    (1, 1500, 1400, 20, 512, 2, 2, 128, 4096, 0),   # 6 keys per thread, no stale rows
    (3, 2048, 0, 16, 256, 1, 1, 128, 512, 200),     # 8 keys per thread, block at the start
    # select and the Q projection as their own launches, the rest fused:
    (2, 3000, 100, 40, 256, 2, 1, 64, 1000, 50),    # 3000 positions (12 keys per thread), 80 query rows
    (1, 300, 10, 100, 256, 4, 2, 64, 512, 20),      # 100 query rows, grouped KV heads
    (2, 2048, 1500, 32, 256, 64, 64, 64, 512, 100),  # the ring attention kernel, head_dim 64, 2 key splits
])
def test_step_fused_equals_calls_small_shapes(P, dtype, batch, seq, bs, bl, d, H, Hkv, hd, vocab, k):
    from types import SimpleNamespace
    g = np.random.default_rng(seq + 31 * k)
    cfg = SimpleNamespace(dtype=dtype, batch=batch, seq=seq, d=d, n_heads=H, n_kv_heads=Hkv, head_dim=hd,
                          block_start=bs, block_len=bl, vocab=vocab)
    base = g.standard_normal((batch, seq, d), dtype=np.float32)
    hp = base.copy()
    hc = base.copy()
    heavy = g.random((batch, seq)) < 0.2
    hc[heavy] += 0.5 * g.standard_normal((int(heavy.sum()), d), dtype=np.float32)
    x = dict(h_cur=inputs.store(hc, dtype), h_prev=inputs.store(hp, dtype),
             w_q=inputs.store(0.03 * g.standard_normal((H * hd, d), dtype=np.float32), dtype),
             w_k=inputs.store(0.03 * g.standard_normal((Hkv * hd, d), dtype=np.float32), dtype),
             w_v=inputs.store(0.03 * g.standard_normal((Hkv * hd, d), dtype=np.float32), dtype),
             logits=inputs.store(3.0 * g.standard_normal((batch, bl, vocab), dtype=np.float32), dtype),
             masked=(g.random((batch, bl)) < 0.7).astype(np.uint8),
             hist=(1e-4 * g.random((batch, 5, bl))).astype(np.float32),
             hist_len=g.integers(0, 6, size=batch).astype(np.int32))
    kc = inputs.store(0.1 * g.standard_normal((batch, seq, Hkv, hd), dtype=np.float32), dtype)
    vc = inputs.store(0.1 * g.standard_normal((batch, seq, Hkv, hd), dtype=np.float32), dtype)
    a, b = _run_both(P, cfg, x, kc, vc, k, force_one=bool(k % 2))
    _assert_same(a, b)


def test_step_refresh_events_bracket_the_refresh(P):
    torch = _torch()
    L = layer(1, 1)
    cfg, x = L["cfg"], L["x"]
    st = P.Step(batch=cfg.batch, seq=cfg.seq, d=cfg.d, n_heads=cfg.n_heads, n_kv_heads=cfg.n_kv_heads,
                head_dim=cfg.head_dim, block_start=cfg.block_start, block_len=cfg.block_len, vocab=cfg.vocab,
                k=int(x["k"]), dtype=torch.bfloat16)
    v = _step_inputs(cfg, x, L["kc"], L["vc"])
    ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
    st.run(v["h_cur"], v["h_prev"], v["w_q"], v["w_k"], v["w_v"], v["k_cache"], v["v_cache"], v["logits"],
           v["masked"], v["hist"], v["hist_len"], refresh_events=ev)
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[1])
    assert 0.0 < ms < 50.0
