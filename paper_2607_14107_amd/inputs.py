"""Seeded synthetic inputs for the Polestar layer step.

This module only draws random numbers and stores them in the run dtype; it
holds none of the method's arithmetic, so the HIP path and the CPU oracle can
both be fed from it.  Every array is generated on the host in float32 with
`numpy.random.default_rng(seed)` and rounded once to the run dtype (round to
nearest, ties to even).  bf16 arrays are returned as their uint16 bit
patterns, fp32 arrays as float32.

Seeds: seed = 1000 * config + 10 * subrun + stream, with streams
  0 weights, 1 base hidden states, 2 drift noise, 3 planted (heavy) set,
  4 logits, 5 drift history, 6 logit spikes, 7 stand-in K/V cache.
Weights and base hidden states depend on the configuration only.

The workloads follow the shapes of LLaDA-8B (d=4096, 32 MHA heads of 128,
vocab 126464) and Dream-7B (d=3584, 28 query / 4 KV heads of 128, vocab
152064) and the decoding structure of the paper: a prompt followed by the
generated region, the active block of B positions right after the prompt.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np


@dataclass(frozen=True)
class LayerConfig:
    """Shape and noise recipe of one synthetic single-layer workload."""
    index: int
    name: str
    dtype: str            # "fp32" or "bf16"
    batch: int
    d: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    prompt_len: int
    seq: int
    block_len: int
    vocab: int
    logit_std: float
    heavy_fracs: tuple    # heavy fraction of each sub-run (or chained step)
    chained: bool = False     # sub-runs are consecutive steps of one run
    clustered: bool = False   # heavy positions in contiguous runs
    weight_std: float = 0.02
    light_std: float = 0.01
    heavy_std: float = 0.5
    hist_depth: int = 5
    tau_s: float = 0.9
    alpha: float = 10.0
    extra: dict = field(default_factory=dict)

    @property
    def block_start(self) -> int:
        return self.prompt_len

    @property
    def cached_positions(self) -> int:
        return self.seq - self.block_len

    def tokens_per_step(self) -> int:
        return self.batch * self.block_len


CONFIGS = {
    0: LayerConfig(0, "tiny-fp32", "fp32", batch=1, d=256, n_heads=4, n_kv_heads=4,
                   head_dim=64, prompt_len=64, seq=96, block_len=32, vocab=1024,
                   logit_std=3.0, heavy_fracs=(0.10,)),
    1: LayerConfig(1, "llada8b-layer-b1-s768", "bf16", batch=1, d=4096, n_heads=32,
                   n_kv_heads=32, head_dim=128, prompt_len=512, seq=768, block_len=32,
                   vocab=126464, logit_std=4.0, heavy_fracs=(0.05, 0.15, 0.25)),
    2: LayerConfig(2, "llada8b-layer-b8-s1536", "bf16", batch=8, d=4096, n_heads=32,
                   n_kv_heads=32, head_dim=128, prompt_len=1024, seq=1536, block_len=32,
                   vocab=126464, logit_std=4.0, heavy_fracs=(0.02, 0.10, 0.30),
                   chained=True),
    3: LayerConfig(3, "dream7b-gqa-layer-b4-s2048", "bf16", batch=4, d=3584, n_heads=28,
                   n_kv_heads=4, head_dim=128, prompt_len=1536, seq=2048, block_len=64,
                   vocab=152064, logit_std=4.0, heavy_fracs=(0.10,), clustered=True),
}


def seed_of(config: int, subrun: int, stream: int) -> int:
    return 1000 * config + 10 * subrun + stream


def rng(config: int, subrun: int, stream: int) -> np.random.Generator:
    return np.random.default_rng(seed_of(config, subrun, stream))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns, round to nearest, ties to even.  In 32-bit
    integers: for every finite value (and the infinities) the sum below stays
    under 2^32 (the largest, -FLT_MAX, gives 0xFF807FFF)."""
    u = np.array(x, dtype=np.float32, copy=True).view(np.uint32)
    lsb = u >> np.uint32(16)
    lsb &= np.uint32(1)
    u += np.uint32(0x7FFF)
    u += lsb
    u >>= np.uint32(16)
    return u.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def store(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round a float32 array to the run dtype: uint16 bits for bf16."""
    if dtype == "fp32":
        return np.ascontiguousarray(x, dtype=np.float32)
    if dtype == "bf16":
        return f32_to_bf16_bits(x)
    raise ValueError(dtype)


def load_f32(x: np.ndarray, dtype: str) -> np.ndarray:
    """The float32 values of a stored array (exact for both dtypes)."""
    return bf16_bits_to_f32(x) if dtype == "bf16" else np.asarray(x, dtype=np.float32)


def normal(g: np.random.Generator, shape, std: float) -> np.ndarray:
    return g.standard_normal(size=shape, dtype=np.float32) * np.float32(std)


def planted_uniform(cfg: LayerConfig, subrun: int, frac: float) -> np.ndarray:
    """[batch][seq] bool: round(frac*seq) positions per sequence, uniform."""
    g = rng(cfg.index, subrun, 3)
    n = int(round(frac * cfg.seq))
    out = np.zeros((cfg.batch, cfg.seq), dtype=bool)
    for b in range(cfg.batch):
        out[b, g.choice(cfg.seq, size=n, replace=False)] = True
    return out


def planted_runs(cfg: LayerConfig, subrun: int, frac: float) -> np.ndarray:
    """[batch][seq] bool: non-overlapping contiguous runs of length U{8..64}
    placed uniformly among cached positions until they cover
    ceil(frac * cached) positions (the last run is truncated)."""
    g = rng(cfg.index, subrun, 3)
    bs, bl = cfg.block_start, cfg.block_len
    target = int(math.ceil(frac * cfg.cached_positions))
    out = np.zeros((cfg.batch, cfg.seq), dtype=bool)
    for b in range(cfg.batch):
        covered = 0
        while covered < target:
            length = int(g.integers(8, 65))
            start = int(g.integers(0, cfg.seq - length + 1))
            span = np.arange(start, start + length)
            if np.any((span >= bs) & (span < bs + bl)) or out[b, span].any():
                continue
            # keep a gap of one position so that runs stay separate
            lo, hi = max(0, start - 1), min(cfg.seq, start + length + 1)
            if out[b, lo:hi].any():
                continue
            take = min(length, target - covered)
            out[b, start:start + take] = True
            covered += take
    return out


def weights(cfg: LayerConfig) -> dict:
    """W_q [H*hd][d], W_k and W_v [Hkv*hd][d], N(0, weight_std)."""
    g = rng(cfg.index, 0, 0)
    qd = cfg.n_heads * cfg.head_dim
    kvd = cfg.n_kv_heads * cfg.head_dim
    w_q = normal(g, (qd, cfg.d), cfg.weight_std)
    w_k = normal(g, (kvd, cfg.d), cfg.weight_std)
    w_v = normal(g, (kvd, cfg.d), cfg.weight_std)
    return {k: store(v, cfg.dtype) for k, v in (("w_q", w_q), ("w_k", w_k), ("w_v", w_v))}


def base_states(cfg: LayerConfig) -> np.ndarray:
    """h_prev of the first step: [batch][seq][d], N(0, 1)."""
    g = rng(cfg.index, 0, 1)
    return store(normal(g, (cfg.batch, cfg.seq, cfg.d), 1.0), cfg.dtype)


def perturb(cfg: LayerConfig, h_prev: np.ndarray, subrun: int, planted: np.ndarray) -> np.ndarray:
    """h_cur = h_prev + N(0, light) everywhere + N(0, heavy) on planted rows."""
    g = rng(cfg.index, subrun, 2)
    base = load_f32(h_prev, cfg.dtype)
    light = normal(g, base.shape, cfg.light_std)
    heavy = normal(g, base.shape, cfg.heavy_std) * planted[:, :, None].astype(np.float32)
    return store(base + light + heavy, cfg.dtype)


def logits(cfg: LayerConfig, subrun: int) -> np.ndarray:
    g = rng(cfg.index, subrun, 4)
    return store(normal(g, (cfg.batch, cfg.block_len, cfg.vocab), cfg.logit_std), cfg.dtype)


def history(cfg: LayerConfig, subrun: int, light_kl: float = 5e-5) -> np.ndarray:
    """Drift history [batch][h][block_len] fp32: positive values around the
    drift that light noise gives (KL ~ light_std**2 / 2), spread 10%."""
    g = rng(cfg.index, subrun, 5)
    x = light_kl * (1.0 + 0.1 * g.standard_normal(
        size=(cfg.batch, cfg.hist_depth, cfg.block_len), dtype=np.float32))
    return np.abs(x).astype(np.float32)


def spike_rows(cfg: LayerConfig, subrun: int, fraction: float = 0.25) -> np.ndarray:
    """[batch][block_len] bool: which tokens receive a logit spike."""
    g = rng(cfg.index, subrun, 6)
    n = max(1, int(round(fraction * cfg.block_len)))
    out = np.zeros((cfg.batch, cfg.block_len), dtype=bool)
    for b in range(cfg.batch):
        out[b, g.choice(cfg.block_len, size=n, replace=False)] = True
    return out


def _step_inputs(cfg: LayerConfig, subrun: int, h_prev: np.ndarray, w: dict) -> dict:
    frac = cfg.heavy_fracs[subrun]
    planted = (planted_runs if cfg.clustered else planted_uniform)(cfg, subrun, frac)
    h_cur = perturb(cfg, h_prev, subrun, planted)
    bs, bl = cfg.block_start, cfg.block_len
    cached = np.ones(cfg.seq, dtype=bool)
    cached[bs:bs + bl] = False
    k = int((planted & cached[None, :]).sum(axis=1).max())
    out = dict(h_prev=h_prev, h_cur=h_cur, planted=planted, k=k,
               logits=logits(cfg, subrun), hist=history(cfg, subrun),
               hist_len=np.full(cfg.batch, cfg.hist_depth, dtype=np.int32),
               masked=np.ones((cfg.batch, cfg.block_len), dtype=np.uint8))
    out.update(w)
    return out


def layer_inputs(cfg: LayerConfig, subrun: int = 0) -> dict:
    """All inputs of one step of a single-layer workload.

    For a chained configuration, sub-run s is step s: its h_prev is the h_cur
    of step s-1 (step 0 starts from the base states)."""
    if cfg.chained:
        return chained_inputs(cfg, subrun)[-1]
    return _step_inputs(cfg, subrun, base_states(cfg), weights(cfg))


def chained_inputs(cfg: LayerConfig, last: int | None = None) -> list:
    """Steps 0..last of a chained configuration in one pass (the same arrays
    layer_inputs returns for each of them; weights shared)."""
    last = len(cfg.heavy_fracs) - 1 if last is None else last
    w = weights(cfg)
    h_prev = base_states(cfg)
    out = []
    for s in range(last + 1):
        out.append(_step_inputs(cfg, s, h_prev, w))
        h_prev = out[-1]["h_cur"]
    return out


def random_cache(cfg: LayerConfig, subrun: int = 0) -> tuple[np.ndarray, np.ndarray]:
    """A stand-in prior K/V cache [batch][seq][kv_heads][head_dim] with the
    spread of a projection of N(0,1) states by N(0, weight_std) weights
    (std weight_std * sqrt(d)), for workloads where re-projecting every row
    on the host would take minutes."""
    g = rng(cfg.index, subrun, 7)
    shape = (cfg.batch, cfg.seq, cfg.n_kv_heads, cfg.head_dim)
    std = cfg.weight_std * math.sqrt(cfg.d)
    return store(normal(g, shape, std), cfg.dtype), store(normal(g, shape, std), cfg.dtype)


# ---------------------------------------------------------------------------
# Whole-stack workloads: the denoising loop over a pre-norm layer stack
# ---------------------------------------------------------------------------

@dataclass(frozen=True)
class StackConfig:
    """Shape and weight recipe of a synthetic layer stack (random weights)."""
    index: int
    name: str
    dtype: str
    batch: int
    n_layers: int
    d: int
    n_heads: int
    head_dim: int
    ffn: int
    vocab: int
    prompt_len: int
    gen_len: int
    block_len: int = 32
    weight_std: float = 0.02
    embed_std: float = 0.02
    lm_std: float = 0.02

    @property
    def seq(self) -> int:
        return self.prompt_len + self.gen_len


STACKS = {
    # LLaDA-8B-shaped stack: 32 layers, d 4096, 32x128 MHA, SwiGLU FFN 12288,
    # vocab 126464 (mask id = vocab - 1), N(0, 0.02) weights everywhere,
    # batch 16, prompt 512, 256 generated tokens in blocks of 32
    4: StackConfig(4, "llada8b-stack-b16", "bf16", batch=16, n_layers=32, d=4096, n_heads=32, head_dim=128,
                   ffn=12288, vocab=126464, prompt_len=512, gen_len=256),
    # the 32-layer stack's width and sequence length with two layers and two blocks
    # (prompt 704 + 64 generated): the full-width parity case
    41: StackConfig(41, "llada8b-width-2layer-b16", "bf16", batch=16, n_layers=2, d=4096, n_heads=32,
                    head_dim=128, ffn=12288, vocab=126464, prompt_len=704, gen_len=64),
    # the same loop at sizes the float64 oracle replays in seconds; a wider
    # LM head makes the confidences spread so that the commit rule decides
    40: StackConfig(40, "tiny-stack-b2", "bf16", batch=2, n_layers=2, d=256, n_heads=4, head_dim=64, ffn=768,
                    vocab=512, prompt_len=64, gen_len=64, embed_std=1.0, lm_std=0.25),
    # the packet flow at replay size (the window K-means needs d % 512 == 0 in bf16)
    42: StackConfig(42, "tiny-packet-stack-b2", "bf16", batch=2, n_layers=2, d=512, n_heads=8, head_dim=64,
                    ffn=1024, vocab=512, prompt_len=64, gen_len=64, embed_std=1.0, lm_std=0.2),
}

STACK_MATRICES = ("w_q", "w_k", "w_v", "w_o", "w_gu", "w_down")


def _bf16_bits_fast(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bits, nearest, ties to even (finite values of modest
    magnitude, where the 32-bit sum cannot carry out)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    return ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)).astype(np.uint16)


def stack_tensor(cfg: StackConfig, name: str, layer: int = -1) -> np.ndarray:
    """One weight of the stack in the run dtype, from its own seed
    (config, layer, matrix).  Shapes: w_q/w_k/w_v [H*hd][d], w_o [d][H*hd],
    w_gu [2*ffn][d] (gate rows then up rows), w_down [d][ffn],
    tok_emb / w_lm [vocab][d], pos_emb [seq][d]."""
    hd = cfg.n_heads * cfg.head_dim
    shapes = dict(w_q=(hd, cfg.d), w_k=(hd, cfg.d), w_v=(hd, cfg.d), w_o=(cfg.d, hd), w_gu=(2 * cfg.ffn, cfg.d),
                  w_down=(cfg.d, cfg.ffn), tok_emb=(cfg.vocab, cfg.d), pos_emb=(cfg.seq, cfg.d),
                  w_lm=(cfg.vocab, cfg.d))
    std = dict(tok_emb=cfg.embed_std, pos_emb=cfg.embed_std, w_lm=cfg.lm_std).get(name, cfg.weight_std)
    names = STACK_MATRICES + ("tok_emb", "pos_emb", "w_lm")
    g = np.random.default_rng(np.random.SeedSequence([cfg.index, layer + 1, names.index(name)]))
    x = g.standard_normal(size=shapes[name], dtype=np.float32)
    x *= np.float32(std)
    return _bf16_bits_fast(x) if cfg.dtype == "bf16" else x


def stack_prompt(cfg: StackConfig) -> np.ndarray:
    """[batch][prompt_len] token ids in [0, vocab - 1) (never the mask id)."""
    g = np.random.default_rng(np.random.SeedSequence([cfg.index, 0, 99]))
    return g.integers(0, cfg.vocab - 1, size=(cfg.batch, cfg.prompt_len)).astype(np.int32)
