"""The whole layer step (polestar_step, the fused launches the benchmark
times) against the oracle on the batch-8 LLaDA-8B layer, run as three
chained steps, and on the Dream-7B GQA layer.

Chained steps (Alg. 1, the steps inside one block): step s runs on
h_prev := h_cur of step s-1, on the K/V cache step s-1 left behind and on
the drift history it pushed; heavy fractions 2%, 10%, 30%.  The GPU carries
its own cache and history from step to step; the oracle carries its own (its
exact projections rounded to bf16), so no GPU value enters the oracle's
state.  As the boundary fixes, the integer decisions are checked with the
oracle fed the GPU's drift values: the stale set is the oracle's select of
the GPU's drift, and the commit rule pushes the GPU's drift of the block.
Everything else (drift, refreshed and untouched cache rows, Q, attention
output and lse, tokens and confidences) is compared with the oracle's own
values at the stated bar.  The prior cache of the first step is the oracle's
projection of the base states, rounded to bf16.
"""

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


def _prior_cache(cfg, h_prev_dec, w_k, w_v):
    shape = (cfg.batch, cfg.seq, cfg.n_kv_heads, cfg.head_dim)
    k0 = ref.round_to((h_prev_dec @ w_k.T).reshape(shape), cfg.dtype)
    v0 = ref.round_to((h_prev_dec @ w_v.T).reshape(shape), cfg.dtype)
    return k0, v0


class _Chain:
    """One GPU run (cache and history on the device) beside one oracle run."""

    def __init__(self, P, cfg, x0):
        import torch
        self.P, self.cfg = P, cfg
        self.w = {n: ref.decode(x0[n], cfg.dtype) for n in ("w_q", "w_k", "w_v")}
        self.dev_w = {n: to_dev(x0[n], cfg.dtype) for n in ("w_q", "w_k", "w_v")}
        k0, v0 = _prior_cache(cfg, ref.decode(x0["h_prev"], cfg.dtype), self.w["w_k"], self.w["w_v"])
        self.kc = to_dev(bits_of(k0, cfg.dtype), cfg.dtype)
        self.vc = to_dev(bits_of(v0, cfg.dtype), cfg.dtype)
        self.k_o, self.v_o = k0, v0                       # the oracle's cache (bf16 values as float64)
        self.hist = torch.from_numpy(x0["hist"].copy()).cuda()
        self.hist_len = torch.from_numpy(x0["hist_len"].copy()).cuda()
        self.hist_o, self.hl_o = x0["hist"].copy(), x0["hist_len"].copy()

    def step(self, x, label):
        import torch
        P, cfg = self.P, self.cfg
        bs, bl, dt = cfg.block_start, cfg.block_len, cfg.dtype
        k = int(x["k"])
        st = P.Step(batch=cfg.batch, seq=cfg.seq, d=cfg.d, n_heads=cfg.n_heads, n_kv_heads=cfg.n_kv_heads,
                    head_dim=cfg.head_dim, block_start=bs, block_len=bl, vocab=cfg.vocab, k=k,
                    dtype=torch.bfloat16 if dt == "bf16" else torch.float32)
        kc_before, vc_before = from_dev(self.kc), from_dev(self.vc)
        st.run(to_dev(x["h_cur"], dt), to_dev(x["h_prev"], dt), self.dev_w["w_q"], self.dev_w["w_k"],
               self.dev_w["w_v"], self.kc, self.vc, to_dev(x["logits"], dt), torch.from_numpy(x["masked"]).cuda(),
               self.hist, self.hist_len, force_one=True)
        torch.cuda.synchronize()
        g = {n: from_dev(t) for n, t in dict(drift=st.drift, idx=st.stale_idx, cnt=st.stale_count, q=st.q_buf,
                                            out=st.out, lse=st.lse, token=st.token, conf=st.conf,
                                            commit=st.commit, kc=self.kc, vc=self.vc, hist=self.hist,
                                            hist_len=self.hist_len).items()}
        h_cur, h_prev = ref.decode(x["h_cur"], dt), ref.decode(x["h_prev"], dt)
        rtol = RTOL[dt]

        # drift and the stale set (the oracle's select of the GPU's drift)
        assert_drift_close(g["drift"], ref.drift(h_cur, h_prev))
        idx_o, cnt_o = ref.select(g["drift"].astype(np.float64), k, bs, bl)
        assert np.array_equal(g["idx"], idx_o) and np.array_equal(g["cnt"], cnt_o), f"{label}: stale set"

        # refresh: rows R re-projected, every other row keeps its bytes
        k_new, v_new, rows = ref.refresh_kv(h_cur, self.w["w_k"], self.w["w_v"], self.k_o, self.v_o,
                                            idx_o, cnt_o, bs, bl)
        for b in range(cfg.batch):
            r = np.asarray(rows[b], dtype=np.int64)
            keep = np.setdiff1d(np.arange(cfg.seq), r)
            assert np.array_equal(g["kc"][b, keep], kc_before[b, keep]), f"{label}: K rows outside R written"
            assert np.array_equal(g["vc"][b, keep], vc_before[b, keep]), f"{label}: V rows outside R written"
            assert_rows_close(ref.decode(g["kc"][b, r], dt), k_new[b, r], rtol, f"{label}: K rows of seq {b}")
            assert_rows_close(ref.decode(g["vc"][b, r], dt), v_new[b, r], rtol, f"{label}: V rows of seq {b}")
        self.k_o, self.v_o = ref.round_to(k_new, dt), ref.round_to(v_new, dt)

        # Q and attention over the oracle's own refreshed cache
        q_o = ref.q_project(h_cur, self.w["w_q"], bs, bl, cfg.n_heads, cfg.head_dim)
        assert_rows_close(ref.decode(g["q"], dt), q_o, rtol, f"{label}: Q")
        out_o, lse_o = ref.attend(ref.round_to(q_o, dt), self.k_o, self.v_o)
        assert_rows_close(ref.decode(g["out"], dt), out_o, rtol, f"{label}: attention output")
        np.testing.assert_allclose(g["lse"], lse_o, rtol=rtol, atol=rtol, err_msg=f"{label}: lse")

        # commit: tokens and confidences from the logits, the rule on the GPU's drift
        token_o, conf_o = ref.confidence(ref.decode(x["logits"], dt), -1)
        assert np.array_equal(g["token"], token_o), f"{label}: tokens"
        np.testing.assert_allclose(g["conf"], conf_o, rtol=1e-4, err_msg=f"{label}: confidence")
        conf32 = conf_o.astype(np.float32)
        for b in range(cfg.batch):   # the forced commit's argmax is not a near tie
            top = np.sort(conf32[b][x["masked"][b].astype(bool)])[::-1]
            assert top.size < 2 or top[0] - top[1] > 1e-4 * top[0], f"{label}: near tie in seq {b}"
        delta = g["drift"][:, bs:bs + bl].astype(np.float32)
        commit_o, self.hist_o, self.hl_o = ref.commit_rule(conf32, delta, x["masked"].astype(bool), self.hist_o,
                                                           self.hl_o, cfg.hist_depth, cfg.tau_s, cfg.alpha, True)
        assert np.array_equal(g["commit"].astype(bool), commit_o), f"{label}: commit decisions"
        assert np.array_equal(g["hist"], self.hist_o) and np.array_equal(g["hist_len"], self.hl_o), \
            f"{label}: drift history"
        return g


def test_step_chained_batch8_llada_layer(P):
    """Three consecutive steps of the batch-8 LLaDA-8B layer (seq 1536,
    block 32; 2%, 10%, 30% of the positions heavily perturbed)."""
    cfg = inputs.CONFIGS[2]
    assert cfg.chained
    xs = [inputs.layer_inputs(cfg, s) for s in range(len(cfg.heavy_fracs))]
    for s in range(1, len(xs)):        # the generator chains the states
        assert np.array_equal(xs[s]["h_prev"], xs[s - 1]["h_cur"])
    chain = _Chain(P, cfg, xs[0])
    for s, x in enumerate(xs):
        g = chain.step(x, f"step {s} ({cfg.heavy_fracs[s]:.0%} heavy)")
        assert (g["cnt"] == int(x["k"])).all()


def test_step_dream_gqa_layer(P):
    """One step of the batch-4 Dream-7B GQA layer (28 query / 4 KV heads,
    seq 2048, block 64, stale positions in contiguous runs)."""
    cfg = inputs.CONFIGS[3]
    x = inputs.layer_inputs(cfg, 0)
    _Chain(P, cfg, x).step(x, "dream step")
