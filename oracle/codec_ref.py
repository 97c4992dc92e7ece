"""CPU oracle of the cached hidden-state residual codec.

TEST INFRASTRUCTURE ONLY, like `polestar_ref`: the slow plain reference that
the HIP path is checked against; only the tests, the package's smoke check and
the benchmark's `cpu_baseline` leg may use it.

The paper caches the local window's hidden states as residuals to their
cluster's centroid, quantized along the channels in a 4-bit float format with
block scales (Sec. 4.1 "Cluster and Quantize Hidden States"; App. C
"Quantization Format"; the format ablation of App. D finds microscaling FP4
and FP8 residuals as accurate as the paper's choice).  The codec here uses the
OCP microscaling formats that MI355X supports natively:

  MXFP4: blocks of 32 consecutive channels share one E8M0 scale 2^e
         (one byte, e + 127); each value is FP4 E2M1 (sign, 2 exponent bits
         with bias 1, 1 mantissa bit: magnitudes 0, 0.5, 1, 1.5, 2, 3, 4, 6).
  MXFP8: the same blocks and scales, values in FP8 E4M3 (bias 7, no
         infinities, largest magnitude 448, subnormal step 2^-9).

Readings:
  Q-1  The block scale follows the OCP rule: e = floor(log2(amax)) - emax of
       the element format (2 for E2M1, 8 for E4M3), amax the block's largest
       magnitude, clamped to the E8M0 range [-127, 127]; a block of zeros
       gets e = -127.  Elements are v / 2^e
       rounded to nearest, ties to even, and saturated to the largest
       magnitude.
  Q-2  The residual is taken against the mean of the cluster's members'
       values (the same vector the proxy token is made of), computed once at
       block entry; rows outside every cluster use a zero mean.  Residuals are
       formed in fp32 (x - mean rounded to fp32), so that both sides quantize
       the same numbers.
  Q-3  Codes: MXFP4 packs two values per byte, the lower channel in the low
       nibble (sign in bit 3); MXFP8 stores one byte per value (sign in bit 7).
"""

from __future__ import annotations

import numpy as np

BLOCK = 32
FORMATS = {
    # name: (exponent bits, mantissa bits, exponent bias, emax of the block scale, largest magnitude)
    "mxfp4": (2, 1, 1, 2, 6.0),
    "mxfp8": (4, 3, 7, 8, 448.0),
}


def _grid(fmt: str) -> np.ndarray:
    """Every non-negative magnitude of the element format, ascending, with
    its code (the bit pattern without sign) at the same index."""
    eb, mb, bias, _, vmax = FORMATS[fmt]
    vals, codes = [], []
    for e in range(2 ** eb):
        for m in range(2 ** mb):
            if e == 0:
                v = (m / 2 ** mb) * 2.0 ** (1 - bias)                # subnormals and zero
            else:
                v = (1 + m / 2 ** mb) * 2.0 ** (e - bias)
            if v <= vmax:                                            # E4M3: drop the NaN pattern
                vals.append(v)
                codes.append((e << mb) | m)
    order = np.argsort(vals)
    return np.array(vals)[order], np.array(codes)[order]


def block_exponent(block: np.ndarray, fmt: str) -> int:
    """Q-1: floor(log2(amax)) - emax, or -127 for an all-zero block."""
    amax = float(np.max(np.abs(block)))
    if amax == 0.0:
        return -127
    _, e = np.frexp(amax)                                            # amax = f * 2^e, 0.5 <= f < 1
    return max(int(e - 1) - FORMATS[fmt][3], -127)                   # E8M0 holds 2^-127 .. 2^127


def quantize_element(v: float, fmt: str) -> tuple[int, float]:
    """Nearest grid magnitude of |v| (ties to the even code), saturated;
    returns (code with sign bit, value)."""
    vals, codes = _grid(fmt)
    eb, mb = FORMATS[fmt][0], FORMATS[fmt][1]
    sign_bit = 1 << (eb + mb)
    a = abs(v)
    if a >= vals[-1]:
        i = len(vals) - 1
    else:
        j = int(np.searchsorted(vals, a, side="right"))              # vals[j-1] <= a < vals[j]
        lo, hi = j - 1, j
        dlo, dhi = a - vals[lo], vals[hi] - a
        if dlo < dhi:
            i = lo
        elif dhi < dlo:
            i = hi
        else:
            i = lo if codes[lo] % 2 == 0 else hi                     # tie: even mantissa
    code = int(codes[i]) | (sign_bit if (v < 0 or (v == 0 and np.signbit(v))) and vals[i] != 0 else 0)
    val = -vals[i] if code & sign_bit else vals[i]
    return code, float(val)


def encode_row(r: np.ndarray, fmt: str):
    """One row of fp32 residuals -> (codes [d] ints, exponents [d / 32] ints)."""
    d = r.shape[0]
    codes = np.zeros(d, np.int64)
    exps = np.zeros(d // BLOCK, np.int64)
    for blk in range(d // BLOCK):
        seg = r[blk * BLOCK:(blk + 1) * BLOCK].astype(np.float64)
        e = block_exponent(seg, fmt)
        exps[blk] = e
        for i, v in enumerate(seg):
            codes[blk * BLOCK + i] = quantize_element(v / 2.0 ** e, fmt)[0]
    return codes, exps


def decode_row(codes: np.ndarray, exps: np.ndarray, fmt: str) -> np.ndarray:
    """Codes and block exponents -> values (float64, exact)."""
    vals, gcodes = _grid(fmt)
    lut = {int(c): v for c, v in zip(gcodes, vals)}
    eb, mb = FORMATS[fmt][0], FORMATS[fmt][1]
    sign_bit = 1 << (eb + mb)
    out = np.zeros(codes.shape[0])
    for i, c in enumerate(codes):
        v = lut[int(c) & (sign_bit - 1)]
        out[i] = (-v if int(c) & sign_bit else v) * 2.0 ** int(exps[i // BLOCK])
    return out


def residual(x: np.ndarray, mean: np.ndarray) -> np.ndarray:
    """Q-2: x - mean rounded to fp32."""
    return (np.asarray(x, np.float32) - np.asarray(mean, np.float32)).astype(np.float32)


def encode(x: np.ndarray, mean: np.ndarray, fmt: str):
    """Rows [n][d] against their means [n][d] -> (codes [n][d], exps [n][d/32])."""
    r = residual(x, mean)
    out = [encode_row(row, fmt) for row in r]
    return np.stack([o[0] for o in out]), np.stack([o[1] for o in out])


def decode(codes: np.ndarray, exps: np.ndarray, mean: np.ndarray, fmt: str) -> np.ndarray:
    """mean + the decoded residual, per row, in float64."""
    return np.stack([np.asarray(m, np.float64) + decode_row(c, e, fmt) for c, e, m in zip(codes, exps, mean)])


def cluster_means(x: np.ndarray, labels: np.ndarray, n_clusters: int) -> np.ndarray:
    """Q-2: per cluster the mean of its members' rows; x [S][d], labels [S]
    (-1 outside the window) -> [K][d]; an empty cluster gets zeros."""
    out = np.zeros((n_clusters, x.shape[1]))
    for k in range(n_clusters):
        m = x[labels == k]
        if len(m):
            out[k] = m.mean(axis=0)
    return out


def pack(codes: np.ndarray, exps: np.ndarray, fmt: str) -> tuple[np.ndarray, np.ndarray]:
    """Q-3: byte layout of a row set: codes [n][d] -> [n][d/2] (MXFP4, low
    nibble first) or [n][d] (MXFP8) uint8; exps -> E8M0 bytes e + 127."""
    c = np.asarray(codes, np.int64)
    if fmt == "mxfp4":
        b = (c[..., 0::2] & 0xF) | ((c[..., 1::2] & 0xF) << 4)
    else:
        b = c & 0xFF
    return b.astype(np.uint8), (np.asarray(exps, np.int64) + 127).astype(np.uint8)


def unpack(b: np.ndarray, e8: np.ndarray, fmt: str) -> tuple[np.ndarray, np.ndarray]:
    """Inverse of pack: bytes [n][d/2 or d] and E8M0 bytes [n][d/32] ->
    (codes [n][d], exponents [n][d/32])."""
    b = np.asarray(b, np.int64)
    if fmt == "mxfp4":
        c = np.empty(b.shape[:-1] + (2 * b.shape[-1],), np.int64)
        c[..., 0::2] = b & 0xF
        c[..., 1::2] = (b >> 4) & 0xF
    else:
        c = b
    return c, np.asarray(e8, np.int64) - 127
