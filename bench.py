"""Benchmark of one Polestar layer step on one MI355X.

    python bench.py [--steps K] [--warmup W] [--config 1] [--subrun 1]

A step is the whole hot path over one batch: drift -> select -> sparse K/V
refresh -> Q projection + bidirectional attention -> commit, five C-ABI calls
on one stream.  The default workload is the LLaDA-8B-shaped layer (bf16,
batch 1, d=4096, 32 heads of 128, sequence 768 = prompt 512 + 256 generated,
active block 32, vocabulary 126464) with 15% of the positions heavily
perturbed.  Inputs are seeded synthetic data, resident in HBM before timing.

To measure HBM rather than the 256 MB Infinity Cache, every step reads one of
R independent copies of all inputs and weights (R * working set > 256 MB),
round robin.  Per-call durations come from HIP events recorded on the launch
stream around each call inside the timed region.  One JSON line is printed.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "denoise-step tokens/s per layer, LLaDA-8B shape; % of HBM/MFMA roofline"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # dense bf16 MFMA
FP32_PEAK_TFLOPS = 157.3
CALLS = ("drift", "select", "refresh_kv", "attend", "commit")


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--config", type=int, default=1)
    p.add_argument("--subrun", type=int, default=1)
    p.add_argument("--copies", type=int, default=0, help="input copies rotated (0: enough for 512 MB)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=20.0)
    return p.parse_args()


def algorithmic_cost(cfg, k, es):
    """Bytes each call must move and flops it must do (per step), counting
    the stale rows, the weights once, the cache once and the logits once."""
    b, S, d, B = cfg.batch, cfg.seq, cfg.d, cfg.block_len
    H, Hkv, hd, V = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.vocab
    kvd, qd = Hkv * hd, H * hd
    R = b * (k + B)                              # refreshed rows
    cost = {
        "drift": dict(bytes=2 * b * S * d * es + 4 * b * S, flops=0),
        "select": dict(bytes=4 * b * S + 4 * b * (k + 1), flops=0),
        "refresh_kv": dict(bytes=2 * kvd * d * es + R * d * es + R * 2 * kvd * es + 4 * b * (k + 1),
                           flops=2 * R * d * 2 * kvd),
        "attend": dict(bytes=qd * d * es + b * B * d * es + 2 * b * S * kvd * es + 2 * b * B * qd * es,
                       flops=2 * b * B * d * qd + 4 * b * H * B * S * hd),
        "commit": dict(bytes=b * B * V * es + b * B * (4 + 4 + 1 + 1) + 4 * b * (cfg.hist_depth + 1) * B,
                       flops=0),
    }
    return cost


def source_digest(files):
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_for(kernel_files, per_launch_units):
    """HBM bytes per launch from the committed counter summary, or None when
    the summary is missing or the kernel changed since it was taken."""
    path = os.path.join(ROOT, "profiles", "refresh_kv_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("source_digest") != source_digest(kernel_files):
        return None
    return t.get("bytes_per_launch")


def cpu_baseline(cfg, x, k, budget_s):
    """The oracle as it stands, timed on the host on whole steps of the same
    workload until about budget_s seconds of CPU work are done."""
    from oracle import polestar_ref as ref
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = len(os.sched_getaffinity(0))
    dec = {n: ref.decode(x[n], cfg.dtype) for n in ("h_cur", "h_prev", "w_q", "w_k", "w_v")}
    shape = (cfg.batch, cfg.seq, cfg.n_kv_heads, cfg.head_dim)
    kc = ref.round_to((dec["h_prev"] @ dec["w_k"].T).reshape(shape), cfg.dtype)
    vc = ref.round_to((dec["h_prev"] @ dec["w_v"].T).reshape(shape), cfg.dtype)
    logits = ref.decode(x["logits"], cfg.dtype)
    steps, t_total = 0, 0.0
    while t_total < budget_s and steps < 50:
        t0 = time.perf_counter()
        r = ref.layer_step(dec["h_cur"], dec["h_prev"], dec["w_q"], dec["w_k"], dec["w_v"], kc, vc,
                           k=k, block_start=cfg.block_start, block_len=cfg.block_len,
                           n_heads=cfg.n_heads, n_kv_heads=cfg.n_kv_heads, head_dim=cfg.head_dim,
                           cache_dtype=cfg.dtype)
        token, conf = ref.confidence(logits, -1)
        delta = r["drift"][:, cfg.block_start:cfg.block_start + cfg.block_len].astype(np.float32)
        ref.commit_rule(conf.astype(np.float32), delta, x["masked"].astype(bool), x["hist"],
                        x["hist_len"], cfg.hist_depth, cfg.tau_s, cfg.alpha, False)
        t_total += time.perf_counter() - t0
        steps += 1
    tok = cfg.batch * cfg.block_len
    return {"value": round(tok * steps / t_total, 3), "unit": "tokens/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{steps} whole oracle layer steps (drift, select, refresh, Q projection, "
                      f"attention, commit) of the benchmarked workload, {t_total:.1f} s"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the layer step shards over the batch with no exchange, see DESIGN.md)", file=sys.stderr)
        return 2

    import torch
    from paper_2607_14107_amd import inputs
    from paper_2607_14107_amd import polestar as P

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    if not os.path.exists(P.LIB_PATH):
        from paper_2607_14107_amd import build
        build.build(verbose=False)
    P.lib()

    cfg = inputs.CONFIGS[args.config]
    x = inputs.layer_inputs(cfg, args.subrun)
    k = int(x["k"])
    dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    es = 2 if cfg.dtype == "bf16" else 4
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)

    def up(a):
        if cfg.dtype == "bf16":
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)

    # working set of one copy; enough copies to exceed the Infinity Cache twice
    ws_bytes = sum(x[n].nbytes for n in ("h_cur", "h_prev", "w_q", "w_k", "w_v", "logits")) \
        + 2 * cfg.batch * cfg.seq * cfg.n_kv_heads * cfg.head_dim * es
    copies = args.copies or max(1, -(-512 * 2 ** 20 // ws_bytes))
    sets = []
    for c in range(copies):
        s = {n: up(x[n]) for n in ("h_cur", "h_prev", "w_q", "w_k", "w_v", "logits")}
        s["k_cache"] = torch.empty((cfg.batch, cfg.seq, cfg.n_kv_heads, cfg.head_dim), dtype=dt, device=dev)
        s["v_cache"] = torch.empty_like(s["k_cache"])
        # prior cache = projection of the previous states (setup, untimed)
        all_idx = torch.arange(cfg.seq, dtype=torch.int32, device=dev).repeat(cfg.batch, 1).contiguous()
        all_cnt = torch.full((cfg.batch,), cfg.seq, dtype=torch.int32, device=dev)
        P.refresh_kv(s["h_prev"], all_idx, all_cnt, cfg.block_start, 0, s["w_k"], s["w_v"],
                     s["k_cache"], s["v_cache"])
        s["masked"] = torch.from_numpy(x["masked"]).to(dev)
        s["hist"] = torch.from_numpy(x["hist"].copy()).to(dev)
        s["hist_len"] = torch.from_numpy(x["hist_len"].copy()).to(dev)
        sets.append(s)
    step = P.Step(batch=cfg.batch, seq=cfg.seq, d=cfg.d, n_heads=cfg.n_heads, n_kv_heads=cfg.n_kv_heads,
                  head_dim=cfg.head_dim, block_start=cfg.block_start, block_len=cfg.block_len,
                  vocab=cfg.vocab, k=k, dtype=dt, device=dev)
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()

    def run_step(i, ev=None):
        s = sets[i % copies]
        sh = step.shape
        if ev is not None:
            ev[0].record(stream)
        P.drift(s["h_cur"], s["h_prev"], out=step.drift)
        if ev is not None:
            ev[1].record(stream)
        if k > 0:
            P.select(step.drift, k, sh["block_start"], sh["block_len"], None, step.stale_idx, step.stale_count)
        if ev is not None:
            ev[2].record(stream)
        P.refresh_kv(s["h_cur"], step.stale_idx, step.stale_count, sh["block_start"], sh["block_len"],
                     s["w_k"], s["w_v"], s["k_cache"], s["v_cache"], workspace=step.ws_refresh)
        if ev is not None:
            ev[3].record(stream)
        P.attend(s["h_cur"], s["w_q"], s["k_cache"], s["v_cache"], sh["block_start"], sh["block_len"],
                 sh["n_heads"], q_buf=step.q_buf, out=step.out, lse=step.lse, workspace=step.ws_attend)
        if ev is not None:
            ev[4].record(stream)
        P.commit(s["logits"], s["masked"], step.drift, sh["block_start"], s["hist"], s["hist_len"], -1,
                 cfg.tau_s, cfg.alpha, False, step.token, step.conf, step.commit, workspace=step.ws_commit)
        if ev is not None:
            ev[5].record(stream)

    for i in range(args.warmup):
        run_step(i)
    torch.cuda.synchronize()

    # timed region: K whole steps, with events around each call
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        run_step(args.warmup + i, events[i])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    per_call = {c: [] for c in CALLS}
    for ev in events:
        for j, c in enumerate(CALLS):
            per_call[c].append(ev[j].elapsed_time(ev[j + 1]) * 1e3)   # us
    call_us = {c: float(np.mean(v)) for c, v in per_call.items()}

    tokens = cfg.batch * cfg.block_len
    value = tokens * args.steps / elapsed
    cost = algorithmic_cost(cfg, k, es)
    # dominant call: the longest one
    dom = max(call_us, key=call_us.get)
    dom_us = call_us[dom]
    c = cost[dom]
    flops_rate = c["flops"] / (dom_us * 1e-6) / 1e12
    bytes_rate = c["bytes"] / (dom_us * 1e-6) / 1e9
    peak_t = BF16_PEAK_TFLOPS if cfg.dtype == "bf16" else FP32_PEAK_TFLOPS
    mfma_bound = c["flops"] / (peak_t * 1e12) > c["bytes"] / (HBM_PEAK_GBS * 1e9)
    if mfma_bound:
        roof = {"bound": "mfma", "achieved": round(flops_rate, 3), "peak": peak_t, "unit": "TFLOP/s",
                "frac": round(flops_rate / peak_t, 4)}
    else:
        roof = {"bound": "hbm", "achieved": round(bytes_rate, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(bytes_rate / HBM_PEAK_GBS, 4)}
    roof["kernel"] = dom
    roof["traffic"] = traffic_for(["paper_2607_14107_amd/csrc/gemm.hip"], 1) if dom == "refresh_kv" else None

    calls = {}
    for name in CALLS:
        cc = cost[name]
        t = call_us[name] * 1e-6
        calls[name] = {"us": round(call_us[name], 3), "bytes": int(cc["bytes"]), "flops": int(cc["flops"]),
                       "GB_s": round(cc["bytes"] / t / 1e9, 1),
                       "hbm_frac": round(cc["bytes"] / t / 1e9 / HBM_PEAK_GBS, 4),
                       "TFLOP_s": round(cc["flops"] / t / 1e12, 3)}

    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: single {'LLaDA-8B' if cfg.n_heads == cfg.n_kv_heads else 'Dream-7B'}"
                               f"-shaped layer step, batch {cfg.batch}, seq {cfg.seq}, block {cfg.block_len}, "
                               f"d {cfg.d}, heads {cfg.n_heads}/{cfg.n_kv_heads}x{cfg.head_dim}, vocab {cfg.vocab}, "
                               f"{k} stale rows per sequence",
                   "global_batch": cfg.batch, "seq_len": cfg.seq, "block": cfg.block_len,
                   "stale_rows": k, "input_copies": copies},
        "roofline": roof,
        "calls_us": calls,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, x, k, args.cpu_seconds)
    print(json.dumps(out))
    return 0


if __name__ == "__main__":
    sys.exit(main())
