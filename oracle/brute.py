"""Second, independent CPU path in pure-Python loops, for tiny inputs only.

TEST INFRASTRUCTURE ONLY (same rule as `polestar_ref`: only the test suite,
the smoke check and the benchmark's `cpu_baseline` leg may use it).  It takes
every step from its definition with explicit scalar loops and `math`, without
NumPy, so that the NumPy oracle is cross-checked by code that shares nothing
with it but the definitions:
  drift      -- eq. (drift), Sec. 3, with the per-token hidden-state reading
  select     -- TopK of Alg. 1 over the cached positions of Sec. 2
  projection -- q/k/v = W x of the App. B setup
  attention  -- l = q.k/sqrt(d_h), softmax, sum of a v (App. B setup, eq. 3)
  confidence -- eq. (1) argmax without [MASK], softmax probability of it
Inputs are nested Python lists of floats.
"""

from __future__ import annotations

import math


def softmax_list(x):
    m = max(x)
    e = [math.exp(v - m) for v in x]
    z = sum(e)
    return [v / z for v in e]


def drift_row(a, b):
    """KL(softmax(a) || softmax(b)) for two rows of equal length."""
    p = softmax_list(a)
    q = softmax_list(b)
    total = 0.0
    for pc, qc in zip(p, q):
        if pc > 0.0:
            total += pc * math.log(pc / qc)
    return total


def drift(h_cur, h_prev):
    return [[drift_row(h_cur[b][i], h_prev[b][i]) for i in range(len(h_cur[b]))]
            for b in range(len(h_cur))]


def select(drift_vals, k, block_start, block_len, eligible=None):
    """Per sequence: rank every candidate by counting how many candidates beat
    it (larger drift, or equal drift at a lower index), keep ranks < k."""
    out_idx, out_cnt = [], []
    for b, row in enumerate(drift_vals):
        cands = [i for i in range(len(row))
                 if not (block_start <= i < block_start + block_len)
                 and (eligible is None or eligible[b][i])]
        chosen = []
        for i in cands:
            rank = 0
            for j in cands:
                if row[j] > row[i] or (row[j] == row[i] and j < i):
                    rank += 1
            if rank < k:
                chosen.append(i)
        chosen.sort()
        out_cnt.append(len(chosen))
        out_idx.append(chosen + [-1] * (k - len(chosen)))
    return out_idx, out_cnt


def matvec(w, x):
    """y_o = sum_i w[o][i] x[i] for a weight stored output x input."""
    return [sum(w[o][i] * x[i] for i in range(len(x))) for o in range(len(w))]


def attention_head(q_rows, k_rows, v_rows, scale):
    """One head: out[j] = sum_s softmax_s(q_j.k_s * scale) v_s, plus lse[j]."""
    outs, lses = [], []
    for q in q_rows:
        logits = [scale * sum(qc * kc for qc, kc in zip(q, k)) for k in k_rows]
        m = max(logits)
        e = [math.exp(v - m) for v in logits]
        z = sum(e)
        o = [0.0] * len(v_rows[0])
        for s, vrow in enumerate(v_rows):
            w = e[s] / z
            for c in range(len(o)):
                o[c] += w * vrow[c]
        outs.append(o)
        lses.append(m + math.log(z))
    return outs, lses


def confidence_row(row, mask_token_id=-1):
    best = None
    for v, x in enumerate(row):
        if v == mask_token_id:
            continue
        if best is None or x > row[best]:
            best = v
    m = max(row)
    z = sum(math.exp(x - m) for x in row)
    return best, math.exp(row[best] - m) / z
