"""Pins of the residual codec oracle (oracle/codec_ref.py) against the
definitions of the OCP microscaling formats: the element grids, rounding
to nearest even with saturation (E4M3 also against torch's own float8
conversion), the block-scale rule on worked examples, exact round trips,
the error bound, the byte layout and the cluster means.  CPU only."""

import math

import numpy as np
import pytest

from oracle import codec_ref as cr


def test_element_grids():
    v, c = cr._grid("mxfp4")
    assert v.tolist() == [0, 0.5, 1, 1.5, 2, 3, 4, 6] and c.tolist() == list(range(8))
    v8, c8 = cr._grid("mxfp8")
    assert len(v8) == 127 and v8[-1] == 448.0 and v8[1] == 2.0 ** -9
    assert c8[-1] == 0x7E                      # 0x7F is the NaN pattern of E4M3
    assert v8[c8.tolist().index(0x38)] == 1.0  # exponent 7 = bias


@pytest.mark.parametrize("v,want", [(0.25, 0.0), (0.75, 1.0), (1.25, 1.0), (1.75, 2.0), (2.5, 2.0), (3.5, 4.0),
                                    (5.0, 4.0), (5.5, 6.0), (7.0, 6.0), (100.0, 6.0), (-0.1, 0.0), (-2.6, -3.0),
                                    (0.74, 0.5), (0.76, 1.0)])
def test_fp4_rounding_ties_even_and_saturation(v, want):
    code, val = cr.quantize_element(v, "mxfp4")
    assert val == want
    if want == 0.0:
        assert code == 0                       # no negative zero
    assert (code >> 3) == (1 if want < 0 else 0)


def test_fp8_rounding_matches_torch_float8_e4m3fn():
    torch = pytest.importorskip("torch")
    g = np.random.default_rng(0)
    x = np.concatenate([g.standard_normal(3000) * s for s in (1e-3, 0.1, 1.0, 30.0, 200.0)])
    x = x[np.abs(x) < 448].astype(np.float32)
    want = torch.from_numpy(x).to(torch.float8_e4m3fn).to(torch.float64).numpy()
    got = np.array([cr.quantize_element(float(v), "mxfp8")[1] for v in x])
    assert np.array_equal(got, want)
    assert cr.quantize_element(1000.0, "mxfp8")[1] == 448.0     # saturates (torch would give NaN)


def test_block_exponent_rule():
    blk = np.zeros(32)
    assert cr.block_exponent(blk, "mxfp4") == -127
    blk[3] = 6.0
    assert cr.block_exponent(blk, "mxfp4") == 0          # floor(log2 6) = 2, minus emax 2
    blk[3] = -0.75
    assert cr.block_exponent(blk, "mxfp4") == -3         # 0.75 / 2^-3 = 6 exactly
    blk[3] = 7.0
    assert cr.block_exponent(blk, "mxfp4") == 0          # 7 saturates to 6 (the OCP rule's clamp)
    blk[3] = 448.0
    assert cr.block_exponent(blk, "mxfp8") == 0
    blk[3] = 1e-45
    assert cr.block_exponent(blk, "mxfp4") == -127       # clamped to the E8M0 range


@pytest.mark.parametrize("fmt", ["mxfp4", "mxfp8"])
def test_representable_rows_round_trip_exactly(fmt):
    vals, _ = cr._grid(fmt)
    g = np.random.default_rng(1)
    r = g.choice(np.concatenate([vals, -vals]), size=128) * 2.0 ** g.integers(-6, 6)
    r[0] = vals[-1] * 2.0 ** int(np.log2(np.abs(r).max() / vals[-1]) // 1) if np.abs(r).max() else 0
    codes, exps = cr.encode_row(r.astype(np.float32), fmt)
    assert np.array_equal(cr.decode_row(codes, exps, fmt), r)


@pytest.mark.parametrize("fmt,rel", [("mxfp4", 0.25), ("mxfp8", 1.0 / 16)])
def test_error_bound(fmt, rel):
    # |v - q(v)| <= half a grid step of v's binade (relative 2^-(m+1) of the binade
    # start) or, for the block's largest values, the saturation loss
    g = np.random.default_rng(2)
    r = (g.standard_normal(4096) * 0.05).astype(np.float32)
    codes, exps = cr.encode_row(r, fmt)
    dec = cr.decode_row(codes, exps, fmt)
    vmax = cr.FORMATS[fmt][4]
    for blk in range(len(r) // 32):
        seg = r[blk * 32:(blk + 1) * 32].astype(np.float64)
        d = dec[blk * 32:(blk + 1) * 32]
        x = 2.0 ** exps[blk]
        sub = 2.0 ** (1 - cr.FORMATS[fmt][2] - cr.FORMATS[fmt][1])     # subnormal step before scaling
        for v, q in zip(seg, d):
            bound = max(rel * abs(v), 0.5 * sub * x) + max(0.0, abs(v) - vmax * x)
            assert abs(v - q) <= bound * (1 + 1e-12)


def test_residual_codec_round_trip_and_zero_residual():
    g = np.random.default_rng(3)
    mean = g.standard_normal((1, 64)).astype(np.float32)
    codes, exps = cr.encode(mean, mean, "mxfp4")
    assert np.all(codes == 0) and np.all(exps == -127)
    assert np.array_equal(cr.decode(codes, exps, mean, "mxfp4"), mean.astype(np.float64))
    x = mean + (g.standard_normal((1, 64)) * 0.01).astype(np.float32)
    c8, e8 = cr.encode(x, mean, "mxfp8")
    assert np.abs(cr.decode(c8, e8, mean, "mxfp8") - x).max() <= np.abs(x - mean).max() / 16 + 1e-9


def test_pack_layout_and_cluster_means():
    codes = np.array([[1, 2, 15, 8]])
    b, e = cr.pack(codes, np.array([[-3]]), "mxfp4")
    assert b.tolist() == [[0x21, 0x8F]] and e.tolist() == [[124]]
    b8, _ = cr.pack(np.array([[0x7E, 0x81]]), np.array([[0]]), "mxfp8")
    assert b8.tolist() == [[0x7E, 0x81]]
    x = np.array([[1.0, 2.0], [3.0, 4.0], [10.0, 0.0], [7.0, 7.0]])
    m = cr.cluster_means(x, np.array([0, 0, 2, -1]), 3)
    assert m.tolist() == [[2.0, 3.0], [0.0, 0.0], [10.0, 0.0]]


@pytest.mark.parametrize("fmt", ["mxfp4", "mxfp8"])
def test_unpack_inverts_pack(fmt):
    g = np.random.default_rng(5)
    r = (g.standard_normal((3, 64)) * 0.1).astype(np.float32)
    c, e = cr.encode(r, np.zeros_like(r), fmt)
    b, e8 = cr.pack(c, e, fmt)
    c2, e2 = cr.unpack(b, e8, fmt)
    assert np.array_equal(c2, c) and np.array_equal(e2, e)
