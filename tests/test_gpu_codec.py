"""GPU parity of the hidden-state residual codec against the oracle
(oracle/codec_ref.py): codes and scales bit-exact (both sides quantize the
same fp32 residuals), the fused gather's decoded rows within fp32 rounding of
the oracle's (one fp32 addition of the mean) and its RMSNorm within bf16
rounding, the cluster means within 1e-5."""

import numpy as np
import pytest

from oracle import codec_ref as cr
from oracle import model_ref as mr
from oracle import polestar_ref as ref
from tests._util import assert_rows_close, ensure_built, from_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    ensure_built()
    from paper_2607_14107_amd import polestar
    return polestar


def _case(b, seq, d, K, seed):
    """Rows with block magnitudes from 1e-30 to 1e3, exact zero residuals,
    rows outside every cluster; a window of ~1/3 of the positions."""
    g = np.random.default_rng(seed)
    win = np.sort(g.choice(seq, size=seq // 3, replace=False)).astype(np.int32)
    labels = np.full((b, seq), -1, np.int32)
    labels[:, win] = g.integers(0, K, size=(b, len(win)))
    labels[:, win[::7]] = -1                                   # a few window rows outside every cluster
    means = (g.standard_normal((b, K, d)) * 2).astype(np.float32)
    x = np.zeros((b, seq, d), np.float32)
    for s in range(b):
        for p in range(seq):
            m = means[s, labels[s, p]] if labels[s, p] >= 0 else np.zeros(d, np.float32)
            scale = 10.0 ** g.uniform(-30, 3, size=d // 32).repeat(32)
            x[s, p] = m + (g.standard_normal(d) * scale).astype(np.float32)
    x[0, win[1]] = means[0, labels[0, win[1]]] if labels[0, win[1]] >= 0 else 0.0     # zero residual
    return win, labels, means, x


@pytest.mark.parametrize("fmt", ["mxfp4", "mxfp8"])
@pytest.mark.parametrize("b,seq,d,K", [(2, 96, 4096, 8), (3, 50, 96, 3)])
def test_codec_encode_gather_match_oracle(P, fmt, b, seq, d, K):
    torch = pytest.importorskip("torch")
    f = P.CODECS[fmt]
    win, labels, means, x = _case(b, seq, d, K, 7)
    dev = "cuda"
    rb = P.codec_row_bytes(f, d)
    codes = torch.full((b, seq, rb), 0xAB, dtype=torch.uint8, device=dev)
    scales = torch.full((b, seq, d // 32), 0xCD, dtype=torch.uint8, device=dev)
    idx = torch.from_numpy(np.tile(win, (b, 1))).to(dev)
    cnt = torch.full((b,), len(win), dtype=torch.int32, device=dev)
    lab_t, x_t, m_t = torch.from_numpy(labels).to(dev), torch.from_numpy(x).to(dev), torch.from_numpy(means).to(dev)
    P.codec_encode(f, x_t, idx, cnt, lab_t, m_t, codes, scales)
    gc, gs = from_dev(codes), from_dev(scales)
    for s in range(b):
        mrows = np.stack([means[s, labels[s, p]] if labels[s, p] >= 0 else np.zeros(d, np.float32) for p in win])
        c, e = cr.encode(x[s, win], mrows, fmt)
        pc, pe = cr.pack(c, e, fmt)
        assert np.array_equal(gc[s, win], pc), "codes differ"
        assert np.array_equal(gs[s, win], pe), "scales differ"
        others = np.setdiff1d(np.arange(seq), win)
        assert np.all(gc[s, others] == 0xAB) and np.all(gs[s, others] == 0xCD)
    # fused gather + dequantisation + RMSNorm of a subset of rows, ragged counts
    k_max = len(win) // 2 + 3
    sel = np.full((b, k_max), -1, np.int32)
    counts = np.array([(k_max - 3 + s) % (k_max + 1) for s in range(b)], np.int32)
    for s in range(b):
        pick = win[s::2] if len(win[s::2]) >= counts[s] else win
        sel[s, :counts[s]] = pick[:counts[s]]
    xo = torch.empty((b, k_max, d), dtype=torch.float32, device=dev)
    ho = torch.empty((b, k_max, d), dtype=torch.bfloat16, device=dev)
    P.codec_gather(f, codes, scales, torch.from_numpy(sel).to(dev), torch.from_numpy(counts).to(dev), lab_t, m_t,
                   xo, ho)
    gx, gh = from_dev(xo), ref.decode(from_dev(ho), "bf16")
    for s in range(b):
        n = counts[s]
        rows = sel[s, :n]
        mrows = np.stack([means[s, labels[s, p]] if labels[s, p] >= 0 else np.zeros(d, np.float32) for p in rows]) \
            if n else np.zeros((0, d), np.float32)
        c, e = cr.encode(x[s, rows], mrows, fmt) if n else (np.zeros((0, d)), np.zeros((0, d // 32)))
        want = cr.decode(c, e, mrows, fmt) if n else np.zeros((0, d))
        np.testing.assert_allclose(gx[s, :n], want, rtol=1e-6, atol=1e-30)
        assert np.all(gx[s, n:] == 0.0)
        if n:
            assert_rows_close(gh[s, :n], ref.round_to(mr.rmsnorm(gx[s, :n].astype(np.float64)), "bf16"), 8e-3,
                              "fused RMSNorm")


def test_cluster_means_match_oracle(P):
    torch = pytest.importorskip("torch")
    b, seq, d, K = 2, 200, 512, 8
    win, labels, _, x = _case(b, seq, d, K, 11)
    x = np.random.default_rng(3).standard_normal((b, seq, d)).astype(np.float32)
    dev = "cuda"
    m = P.cluster_means(torch.from_numpy(x).to(dev), torch.from_numpy(np.tile(win, (b, 1))).to(dev),
                        torch.from_numpy(labels).to(dev), K)
    gm = from_dev(m)
    for s in range(b):
        lab = np.full(seq, -1)
        lab[win] = labels[s, win]
        want = cr.cluster_means(x[s].astype(np.float64), lab, K)
        np.testing.assert_allclose(gm[s], want, rtol=1e-5, atol=1e-6)
