"""Seeded sweeps of random small shapes through the attention, Q-projection
and K/V-refresh entry points, each checked against the CPU oracle.

The shapes are drawn so that every launch plan gets exercised: per-head and
grouped-head attention (4 or 8 waves, idle waves, one or many key splits,
ragged key tiles and query groups; the ring kernel for long key ranges), and
the GEMM plans (small-M kernel, DMA kernel with up to eight row tiles and 8
to 16 stages per split, row kernel, and through polestar_linear the tile
kernel's 256- or 192-row by 256- or 192-column tiles) with ragged row tiles
and refresh row counts.  Tolerances as in
test_gpu_parity: fp32 1e-4, bf16 2e-2 relative per (row, head); rows the
refresh does not touch byte-identical.
"""

import numpy as np
import pytest

from oracle import polestar_ref as ref
from paper_2607_14107_amd import inputs
from tests._util import RTOL, assert_rows_close, ensure_built, from_dev, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    ensure_built()
    from paper_2607_14107_amd import polestar
    return polestar


def _i32(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()


def _attend_case(i):
    g = np.random.default_rng(7000 + i)
    dtype = "bf16" if i % 3 else "fp32"
    hkv = int(g.choice([1, 2, 4]))
    group = int(g.choice([1, 2, 3, 4, 7, 8]))
    hd = int(g.choice([64, 128]))
    batch = int(g.integers(1, 4))
    nq = int(g.integers(1, 97))
    seq = int(g.integers(nq, 700))
    bs = int(g.integers(0, seq - nq + 1))
    return dtype, batch, seq, bs, nq, hkv * group, hkv, hd


@pytest.mark.parametrize("case", range(24))
def test_attend_random_shapes(P, case):
    dtype, batch, seq, bs, nq, H, Hkv, hd = _attend_case(case)
    g = np.random.default_rng(9000 + case)
    q = inputs.store(g.standard_normal((batch, nq, H, hd), dtype=np.float32), dtype)
    kc = inputs.store(g.standard_normal((batch, seq, Hkv, hd), dtype=np.float32), dtype)
    vc = inputs.store(g.standard_normal((batch, seq, Hkv, hd), dtype=np.float32), dtype)
    torch = pytest.importorskip("torch")
    lse = torch.empty((batch, H, nq), dtype=torch.float32, device="cuda")
    out, _ = P.attend(None, None, to_dev(kc, dtype), to_dev(vc, dtype), bs, nq, H,
                      q_buf=to_dev(q, dtype), lse=lse)
    o_want, lse_want = ref.attend(ref.decode(q, dtype), ref.decode(kc, dtype), ref.decode(vc, dtype))
    shape = f"{dtype} b{batch} seq{seq} nq{nq} H{H}/{Hkv} hd{hd}"
    assert_rows_close(ref.decode(from_dev(out), dtype), o_want, RTOL[dtype], "output " + shape)
    np.testing.assert_allclose(from_dev(lse), lse_want, rtol=RTOL[dtype], atol=RTOL[dtype], err_msg=shape)


@pytest.mark.parametrize("batch,seq,nq,H,Hkv,hd", [
    (4, 2100, 32, 16, 16, 64),     # 66 key tiles (the last ragged) in 4 splits of 17: head_dim 64
    (4, 1600, 20, 24, 12, 128),    # two query heads per KV head, 20 queries, 2 splits of 25 tiles
    (1, 4200, 32, 64, 64, 128),    # 132 key tiles in 4 splits of 33: long walks per wave
])
def test_attend_ring_kernel_shapes(P, batch, seq, nq, H, Hkv, hd):
    """bf16 shapes whose plan takes the ring kernel (one workgroup per CU,
    at least four key tiles per wave), against the oracle."""
    dtype = "bf16"
    g = np.random.default_rng(seq + nq + H)
    bs = seq // 3
    q = inputs.store(g.standard_normal((batch, nq, H, hd), dtype=np.float32), dtype)
    kc = inputs.store(g.standard_normal((batch, seq, Hkv, hd), dtype=np.float32), dtype)
    vc = inputs.store(g.standard_normal((batch, seq, Hkv, hd), dtype=np.float32), dtype)
    torch = pytest.importorskip("torch")
    lse = torch.empty((batch, H, nq), dtype=torch.float32, device="cuda")
    out, _ = P.attend(None, None, to_dev(kc, dtype), to_dev(vc, dtype), bs, nq, H,
                      q_buf=to_dev(q, dtype), lse=lse)
    o_want, lse_want = ref.attend(ref.decode(q, dtype), ref.decode(kc, dtype), ref.decode(vc, dtype))
    shape = f"b{batch} seq{seq} nq{nq} H{H}/{Hkv} hd{hd}"
    assert_rows_close(ref.decode(from_dev(out), dtype), o_want, RTOL[dtype], "output " + shape)
    np.testing.assert_allclose(from_dev(lse), lse_want, rtol=RTOL[dtype], atol=RTOL[dtype], err_msg=shape)


def _gemm_dims(g, dtype):
    # d: K split into 8..16 stages per split for the DMA kernel at several of these
    d = int(g.choice([128, 256, 640, 1280, 1536, 1792, 2048])) if dtype == "bf16" else int(g.choice([128, 256, 512]))
    hd = int(g.choice([64, 128]))
    return d, hd


@pytest.mark.parametrize("case", range(12))
def test_linear_random_tile_shapes(P, case):
    """Row counts and widths where the tile kernel's plans compete (256- or
    192-row by 256- or 192-column tiles, unsplit or split K), ragged in both
    directions, bf16."""
    torch = pytest.importorskip("torch")
    g = np.random.default_rng(17000 + case)
    batch = int(g.integers(1, 4))
    n = int(g.integers(200, 1600)) // batch
    rs = int(g.integers(0, 40))
    seq = n + rs + int(g.integers(0, 30))
    K = int(g.choice([1024, 2048, 3072, 4096]))
    N = 16 * int(g.integers(16, 376))                      # 256 .. 6000 columns
    x = inputs.store(g.standard_normal((batch, seq, K)).astype(np.float32), "bf16")
    w = inputs.store((g.standard_normal((N, K)) * 0.05).astype(np.float32), "bf16")
    y = torch.empty((batch, n, N), dtype=torch.bfloat16, device="cuda")
    P.linear(to_dev(x, "bf16"), rs, n, to_dev(w, "bf16"), y)
    want = ref.decode(x, "bf16")[:, rs:rs + n] @ ref.decode(w, "bf16").T
    assert_rows_close(ref.decode(from_dev(y), "bf16"), want, RTOL["bf16"],
                      f"linear {batch}x{n} rows x {N} x K {K}")


@pytest.mark.parametrize("case", range(16))
def test_project_q_random_shapes(P, case):
    g = np.random.default_rng(11000 + case)
    dtype = "bf16" if case % 4 else "fp32"
    d, hd = _gemm_dims(g, dtype)
    H = int(g.integers(1, 9))
    batch = int(g.integers(1, 6))
    bl = int(g.integers(1, 70))
    seq = int(g.integers(bl, bl + 60))
    bs = int(g.integers(0, seq - bl + 1))
    h = inputs.store(g.standard_normal((batch, seq, d), dtype=np.float32), dtype)
    wq = inputs.store(0.05 * g.standard_normal((H * hd, d), dtype=np.float32), dtype)
    q = P.project_q(to_dev(h, dtype), to_dev(wq, dtype), bs, bl, H)
    want = ref.q_project(ref.decode(h, dtype), ref.decode(wq, dtype), bs, bl, H, hd)
    assert_rows_close(ref.decode(from_dev(q), dtype), want, RTOL[dtype],
                      f"Q {dtype} b{batch} rows {batch * bl} d{d} H{H} hd{hd}")


@pytest.mark.parametrize("case", range(16))
def test_refresh_random_shapes(P, case):
    g = np.random.default_rng(13000 + case)
    dtype = "bf16" if case % 4 else "fp32"
    d, hd = _gemm_dims(g, dtype)
    kvh = int(g.integers(1, 5))
    batch = int(g.integers(1, 4))
    seq = int(g.integers(40, 400))
    bl = int(g.integers(1, 40))
    bs = int(g.integers(0, seq - bl + 1))
    k_max = int(g.integers(0, min(seq, 120)))
    if case == 5:
        batch, bl, k_max = 1, 8, 6                         # at most 16 rows: the small-M kernel
        bs = min(bs, seq - bl)
    cached = np.setdiff1d(np.arange(seq), np.arange(bs, bs + bl))
    idx = np.full((batch, max(k_max, 1)), -1, dtype=np.int32)
    cnt = np.zeros(batch, dtype=np.int32)
    for b in range(batch):
        c = int(g.integers(0, min(k_max, cached.size) + 1))
        idx[b, :c] = np.sort(g.choice(cached, size=c, replace=False))
        cnt[b] = c
    h = inputs.store(g.standard_normal((batch, seq, d), dtype=np.float32), dtype)
    wk = inputs.store(0.05 * g.standard_normal((kvh * hd, d), dtype=np.float32), dtype)
    wv = inputs.store(0.05 * g.standard_normal((kvh * hd, d), dtype=np.float32), dtype)
    kc0 = inputs.store(g.standard_normal((batch, seq, kvh, hd), dtype=np.float32), dtype)
    vc0 = inputs.store(g.standard_normal((batch, seq, kvh, hd), dtype=np.float32), dtype)
    kc, vc = to_dev(kc0, dtype), to_dev(vc0, dtype)
    if k_max > 0:
        P.refresh_kv(to_dev(h, dtype), _i32(idx[:, :k_max]), _i32(cnt), bs, bl,
                     to_dev(wk, dtype), to_dev(wv, dtype), kc, vc)
    else:
        P.refresh_kv(to_dev(h, dtype), None, None, bs, bl, to_dev(wk, dtype), to_dev(wv, dtype), kc, vc)
    kg, vg = from_dev(kc), from_dev(vc)
    hdec, wkd, wvd = ref.decode(h, dtype), ref.decode(wk, dtype), ref.decode(wv, dtype)
    shape = f"{dtype} b{batch} seq{seq} k_max{k_max} bl{bl} d{d} kv{kvh}x{hd}"
    for b in range(batch):
        rows = np.asarray(sorted(set(idx[b, :cnt[b]].tolist()) | set(range(bs, bs + bl))), dtype=np.int64)
        keep = np.setdiff1d(np.arange(seq), rows)
        assert np.array_equal(kg[b, keep], kc0[b, keep]) and np.array_equal(vg[b, keep], vc0[b, keep]), \
            "untouched rows changed " + shape
        kw = ref.project_rows(hdec[b], wkd, rows).reshape(rows.size, kvh, hd)
        vw = ref.project_rows(hdec[b], wvd, rows).reshape(rows.size, kvh, hd)
        assert_rows_close(ref.decode(kg[b, rows], dtype), kw, RTOL[dtype], f"K rows b{b} " + shape)
        assert_rows_close(ref.decode(vg[b, rows], dtype), vw, RTOL[dtype], f"V rows b{b} " + shape)


@pytest.mark.parametrize("batch,seq,bs,bl,d,kvh,hd,k_max", [
    (2, 700, 600, 32, 3584, 4, 128, 603),   # 1270 rows x 1024 columns: eight 159-row DMA tiles, four K splits
    (1, 800, 400, 20, 640, 4, 128, 680),    # 700 rows x 1024 columns: five DMA tiles, K unsplit (5 steps)
])
def test_refresh_narrow_output_many_row_tiles(P, batch, seq, bs, bl, d, kvh, hd, k_max):
    """Outputs of at most 1024 columns keep the DMA kernel up to eight row
    tiles; every stale slot is filled, every refreshed row compared."""
    g = np.random.default_rng(d + k_max)
    dtype = "bf16"
    cached = np.setdiff1d(np.arange(seq), np.arange(bs, bs + bl))
    idx = np.stack([np.sort(g.choice(cached, size=k_max, replace=False)) for _ in range(batch)]).astype(np.int32)
    cnt = np.full(batch, k_max, dtype=np.int32)
    h = inputs.store(g.standard_normal((batch, seq, d), dtype=np.float32), dtype)
    wk = inputs.store(0.05 * g.standard_normal((kvh * hd, d), dtype=np.float32), dtype)
    wv = inputs.store(0.05 * g.standard_normal((kvh * hd, d), dtype=np.float32), dtype)
    kc0 = inputs.store(g.standard_normal((batch, seq, kvh, hd), dtype=np.float32), dtype)
    vc0 = inputs.store(g.standard_normal((batch, seq, kvh, hd), dtype=np.float32), dtype)
    kc, vc = to_dev(kc0, dtype), to_dev(vc0, dtype)
    P.refresh_kv(to_dev(h, dtype), _i32(idx), _i32(cnt), bs, bl, to_dev(wk, dtype), to_dev(wv, dtype), kc, vc)
    kg, vg = from_dev(kc), from_dev(vc)
    hdec, wkd, wvd = ref.decode(h, dtype), ref.decode(wk, dtype), ref.decode(wv, dtype)
    for b in range(batch):
        rows = np.asarray(sorted(set(idx[b].tolist()) | set(range(bs, bs + bl))), dtype=np.int64)
        keep = np.setdiff1d(np.arange(seq), rows)
        assert np.array_equal(kg[b, keep], kc0[b, keep]) and np.array_equal(vg[b, keep], vc0[b, keep])
        kw = ref.project_rows(hdec[b], wkd, rows).reshape(rows.size, kvh, hd)
        vw = ref.project_rows(hdec[b], wvd, rows).reshape(rows.size, kvh, hd)
        assert_rows_close(ref.decode(kg[b, rows], dtype), kw, RTOL[dtype], f"K rows b{b}")
        assert_rows_close(ref.decode(vg[b, rows], dtype), vw, RTOL[dtype], f"V rows b{b}")
