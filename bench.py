"""Benchmark of one Polestar layer step on one MI355X.

    python bench.py [--steps K] [--warmup W] [--config 1] [--subrun 1]

A step is the whole hot path over one batch: drift -> select -> sparse K/V
refresh -> Q projection of the active block -> bidirectional attention ->
commit, one polestar_step call on one stream (six launches: drift beside
the vocabulary scan, select beside the Q projection, the refresh GEMM, the
refresh's split-K reduction beside the Q projection's, attention, and the
attention merge beside the commit finalize).  The default workload is the LLaDA-8B-shaped layer (bf16,
batch 1, d=4096, 32 heads of 128, sequence 768 = prompt 512 + 256 generated,
active block 32, vocabulary 126464) with 15% of the positions heavily
perturbed.  Inputs are seeded synthetic data, resident in HBM before timing.

To measure HBM rather than the 256 MB Infinity Cache, every step reads one of
R independent copies of all inputs and weights (R * working set > 256 MB),
round robin.  After the warmup, an untimed diagnostic pass runs the six calls one
by one with HIP events around each (the per-call breakdown, "calls_us"); in
the timed region polestar_step records events on the launch stream around
its refresh launches, the dominant kernels, which gives the roofline's launch
duration.  One JSON line is printed.

Counter summaries (HBM traffic of the dominant call):

    python bench.py --copy-calibration      # a plain 1 GiB device copy, for the
                                            # FETCH_SIZE / WRITE_SIZE scale factor
    python bench.py --summarize-counters FETCH_DIR WRITE_DIR COPY_FETCH_DIR COPY_WRITE_DIR

read rocprofv3 --pmc output directories and write
profiles/<call>_<workload>_traffic.json.
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
CALLS = ("drift", "select", "refresh_kv", "project_q", "attend", "commit")


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
    p.add_argument("--copy-calibration", action="store_true",
                   help="run a plain 1 GiB device copy (counter scale factor) and exit")
    p.add_argument("--summarize-counters", nargs=4, metavar=("FETCH_DIR", "WRITE_DIR", "COPY_FETCH", "COPY_WRITE"),
                   help="write the traffic summary of the dominant call from rocprofv3 --pmc output")
    p.add_argument("--call", default="refresh_kv", help="call whose counters --summarize-counters reads")
    p.add_argument("--stack", type=int, default=None,
                   help="run the denoising loop of a whole layer stack (4: LLaDA-8B-shaped, 32 layers, batch 16) "
                        "once and print its tokens/s and tokens per forward instead of the layer-step benchmark")
    p.add_argument("--flow", default="window", choices=("window", "packet"),
                   help="--stack: window forwards with per-token drift, or the update-packet flow with proxy drift")
    p.add_argument("--codec", default=None, choices=("mxfp4", "mxfp8"),
                   help="--stack --flow packet: keep the window's cached inputs as quantized residuals")
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
        "project_q": dict(bytes=qd * d * es + b * B * d * es + b * B * qd * es, flops=2 * b * B * d * qd),
        "attend": dict(bytes=2 * b * S * kvd * es + 2 * b * B * qd * es, flops=4 * b * H * B * S * hd),
        "commit": dict(bytes=b * B * V * es + b * B * (4 + 4 + 1 + 1) + 4 * b * (cfg.hist_depth + 1) * B,
                       flops=0),
    }
    return cost


# Kernels launched by each call, and the sources they are built from.
CALL_KERNELS = {
    # polestar_step's refresh: the GEMM, then reduce2_kernel (the split-K
    # reduction, with the Q projection's beside it); the stand-alone call's
    # reduction is gemm_reduce_kernel
    "refresh_kv": ("gemm_dma_kernel", "gemm_reduce_kernel", "reduce2_kernel", "gemm_rows_kernel",
                   "gemm_small_kernel"),
    "project_q": ("gemm_dma_kernel", "gemm_small_kernel", "gemm_rows_kernel", "gemm_reduce_kernel"),
    "attend": ("attend_kernel", "attend_merge_kernel"),
    "drift": ("drift_kernel",),
    "select": ("select_kernel",),
    "commit": ("scan_kernel", "finalize_kernel"),
}
CALL_SOURCES = {
    "refresh_kv": ("gemm.hip", "gemm.hpp", "gemm_dev.hpp", "step.hip"),
    "project_q": ("attend.hip", "gemm.hip", "gemm.hpp", "gemm_dev.hpp"),
    "attend": ("attend.hip",),
    "drift": ("drift.hip", "drift_dev.hpp"),
    "select": ("select.hip",),
    "commit": ("commit.hip",),
}
COPY_BYTES = 1 << 30


def source_digest(call):
    """Digest of the sources a call's kernels are built from (changes when the
    kernels do, which retires a counter summary)."""
    h = hashlib.sha256()
    for f in CALL_SOURCES[call] + ("common.hpp", "host_common.hpp"):
        with open(os.path.join(ROOT, "paper_2607_14107_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_path(call, workload):
    return os.path.join(ROOT, "profiles", f"{call}_{workload}_traffic.json")


def traffic_for(call, workload):
    """HBM bytes per launch of `call` from the committed counter summary, or
    None when there is none or the kernels changed since it was taken."""
    path = traffic_path(call, workload)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("source_digest") != source_digest(call):
        return None
    return t.get("bytes_per_launch")


def copy_calibration():
    """A plain device-to-device copy of COPY_BYTES (the scale factor of the
    FETCH_SIZE / WRITE_SIZE counters: known bytes / counted bytes)."""
    import torch
    src = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1.0)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": COPY_BYTES, "launches": 3}))
    return 0


def _counter_rows(directory, counter):
    """(dispatch id, kernel name, value) per dispatch from the counter CSVs
    rocprofv3 --pmc wrote under `directory`."""
    import csv
    import glob
    out = {}
    for path in glob.glob(os.path.join(directory, "**", "*counter_collection.csv"), recursive=True):
        with open(path) as f:
            for r in csv.DictReader(f):
                if r.get("Counter_Name") != counter:
                    continue
                key = int(r["Dispatch_Id"])
                name = r["Kernel_Name"]
                prev = out.get(key, (name, 0.0))
                out[key] = (name, prev[1] + float(r["Counter_Value"]))
    return sorted((k, v[0], v[1]) for k, v in out.items())


def _call_launch_kib(rows, call):
    """Counter KiB per launch of `call`: the dispatches of its most frequent
    leading kernel, each with the dispatches of the same call that follow it."""
    names = CALL_KERNELS[call]
    lead = [n for _, n, _ in rows if names[0] in n]
    if not lead:
        lead = [n for _, n, _ in rows if any(k in n for k in names)]
    from collections import Counter
    main = Counter(lead).most_common(1)[0][0]
    per_launch = []
    i = 0
    while i < len(rows):
        _, name, v = rows[i]
        if name == main:
            tot = v
            j = i + 1
            while j < len(rows) and rows[j][1] != main and any(k in rows[j][1] for k in names[1:]):
                tot += rows[j][2]
                j += 1
            per_launch.append(tot)
            i = j
        else:
            i += 1
    return main, per_launch


def summarize_counters(fetch_dir, write_dir, copy_fetch_dir, copy_write_dir, call, workload):
    def copy_kib(d, counter):
        vals = [v for _, n, v in _counter_rows(d, counter) if "copy" in n.lower()]
        if not vals:
            raise SystemExit(f"no copy dispatch with {counter} under {d}")
        return float(np.median(vals))
    f_fetch = COPY_BYTES / (copy_kib(copy_fetch_dir, "FETCH_SIZE") * 1024)
    f_write = COPY_BYTES / (copy_kib(copy_write_dir, "WRITE_SIZE") * 1024)
    main, fetch = _call_launch_kib(_counter_rows(fetch_dir, "FETCH_SIZE"), call)
    _, write = _call_launch_kib(_counter_rows(write_dir, "WRITE_SIZE"), call)
    fetch_kib, write_kib = float(np.median(fetch)), float(np.median(write))
    t = {
        "call": call, "workload": workload, "lead_kernel": main,
        "launches_counted": [len(fetch), len(write)],
        "fetch_kib_per_launch": round(fetch_kib, 1), "write_kib_per_launch": round(write_kib, 1),
        "copy_scale_fetch": round(f_fetch, 4), "copy_scale_write": round(f_write, 4),
        "bytes_per_launch": int(fetch_kib * 1024 * f_fetch + write_kib * 1024 * f_write),
        "source_digest": source_digest(call),
        "commands": [
            "cd /tmp && export TMPDIR=/tmp",
            "rocprofv3 --pmc FETCH_SIZE -f csv -d $OUT/pmc_fetch -o c -- "
            "python3 $R/bench.py --no-cpu-baseline --steps 20 --warmup 2",
            "rocprofv3 --pmc WRITE_SIZE -f csv -d $OUT/pmc_write -o c -- "
            "python3 $R/bench.py --no-cpu-baseline --steps 20 --warmup 2",
            "rocprofv3 --pmc FETCH_SIZE -f csv -d $OUT/pmc_cfetch -o c -- python3 $R/bench.py --copy-calibration",
            "rocprofv3 --pmc WRITE_SIZE -f csv -d $OUT/pmc_cwrite -o c -- python3 $R/bench.py --copy-calibration",
            f"python3 $R/bench.py --summarize-counters $OUT/pmc_fetch $OUT/pmc_write "
            f"$OUT/pmc_cfetch $OUT/pmc_cwrite --call {call}",
        ],
        "note": "counter KiB per launch summed over the call's kernels (median over launches); "
                "bytes = KiB * 1024 * (copy bytes / copy counter bytes) for FETCH and WRITE; "
                "$R is the repository, $OUT any output directory",
    }
    with open(traffic_path(call, workload), "w") as f:
        json.dump(t, f, indent=1)
        f.write("\n")
    print(json.dumps(t))
    return 0


def measure_gather_scatter(P, torch, cfg, sets, idx, cnt, es, reps=50):
    """The row gather and scatter of an update packet on their own (untimed
    for the headline): the stale rows of h_cur into a compact [batch][k][d]
    buffer, and compact K rows back into the cache, rotating over the input
    copies.  Algorithmic bytes: every moved row read once and written once
    (the gather also writes the zero rows past a sequence's count).  Runs
    after everything else: the scatter overwrites cache rows."""
    if idx is None or idx.shape[1] == 0:
        return None
    b, k = idx.shape
    kvd = cfg.n_kv_heads * cfg.head_dim
    dev = idx.device
    dt = sets[0]["h_cur"].dtype
    rows = int(cnt.clamp(0, k).sum().item())
    packet = torch.empty((b, k, cfg.d), dtype=dt, device=dev)
    # one compact source per input copy, so that the scatter's reads come from HBM too
    krows = [torch.zeros((b, k, kvd), dtype=dt, device=dev) for _ in sets]
    out = {}
    for name in ("gather", "scatter"):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        torch.cuda._sleep(20_000_000)
        e0.record()
        for i in range(reps):
            c = sets[i % len(sets)]
            if name == "gather":
                P.gather_rows(c["h_cur"], idx, cnt, packet)
            else:
                P.scatter_rows(krows[i % len(sets)], idx, cnt, c["k_cache"].view(b, cfg.seq, kvd))
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / reps
        nbytes = (rows + b * k) * cfg.d * es if name == "gather" else 2 * rows * kvd * es
        out[name] = {"us": round(us, 3), "rows": rows, "bytes": int(nbytes), "GB_s": round(nbytes / us / 1e3, 1),
                     "hbm_frac": round(nbytes / us / 1e3 / HBM_PEAK_GBS, 4)}
    return out


def measure_proxy(P, torch, cfg, s, stream, es, n_clusters=8, k_top=4, reps=50):
    """The paper's clustered drift estimator on the same layer (untimed for
    the headline): block-entry K-means of the window (2B before the block, B
    after), then per step proxy drift + cluster select.  HIP events on the
    launch stream, behind a device spin so the GPU runs the calls back to back."""
    win = P.window_positions(cfg.seq, cfg.block_start, cfg.block_len, 2 * cfg.block_len, cfg.block_len)
    widx = torch.tensor([win] * cfg.batch, dtype=torch.int32, device=s["h_cur"].device)
    scores = torch.empty((cfg.batch, n_clusters, cfg.n_heads, cfg.seq), dtype=torch.float32, device=widx.device)
    lse = torch.empty((cfg.batch, n_clusters, cfg.n_heads), dtype=torch.float32, device=widx.device)
    dt = P.BF16 if cfg.dtype == "bf16" else P.FP32
    ws = torch.empty(P.proxy_drift_workspace_size(dt, cfg.batch, cfg.seq, cfg.d, cfg.n_heads, cfg.head_dim,
                                                  n_clusters), dtype=torch.uint8, device=widx.device)
    drift_c = torch.empty((cfg.batch, n_clusters), dtype=torch.float32, device=widx.device)
    idx = torch.empty((cfg.batch, len(win)), dtype=torch.int32, device=widx.device)
    cnt = torch.empty((cfg.batch,), dtype=torch.int32, device=widx.device)
    labels, sums, counts, _ = P.cluster(s["h_prev"], widx, n_clusters)
    P.proxy_drift(sums, counts, s["w_q"], s["k_cache"], cfg.n_heads, scores, lse, True, drift_c, workspace=ws)
    torch.cuda.synchronize()
    e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    torch.cuda._sleep(50_000_000)
    e[0].record(stream)
    for _ in range(5):
        P.cluster(s["h_prev"], widx, n_clusters)
    e[1].record(stream)
    for _ in range(reps):
        P.proxy_drift(sums, counts, s["w_q"], s["k_cache"], cfg.n_heads, scores, lse, False, drift_c, workspace=ws)
        P.cluster_select(labels, drift_c, k_top, len(win), idx, cnt)
    e[2].record(stream)
    torch.cuda.synchronize()
    step_us = e[1].elapsed_time(e[2]) * 1e3 / reps
    kv_bytes = cfg.batch * cfg.seq * cfg.n_kv_heads * cfg.head_dim * es
    sc_bytes = 3 * cfg.batch * n_clusters * cfg.n_heads * cfg.seq * 4
    alg = cfg.n_heads * cfg.head_dim * cfg.d * es + kv_bytes + sc_bytes
    return {"window": len(win), "clusters": n_clusters, "top_clusters": k_top,
            "block_entry_kmeans_us": round(e[0].elapsed_time(e[1]) * 1e3 / 5, 2),
            "step_us": round(step_us, 3), "step_bytes": int(alg),
            "step_GB_s": round(alg / (step_us * 1e-6) / 1e9, 1)}


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


def stack_bench(index, P, torch, flow="window", codec=None):
    """The loop of Alg. 1 on a whole stack with random weights: weights are
    drawn on the host (one thread per matrix) and uploaded as they complete,
    then one full generation is timed (wall clock around the loop, GPU time
    per forward kind from HIP events)."""
    import concurrent.futures as cf
    from paper_2607_14107_amd import inputs, model
    cfg = inputs.STACKS[index]
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    t0 = time.perf_counter()

    def up(a):
        if cfg.dtype == "bf16":
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(a).to(dev)

    jobs = [(n, -1) for n in ("tok_emb", "pos_emb", "w_lm")] + \
        [(m, li) for li in range(cfg.n_layers) for m in inputs.STACK_MATRICES]
    w = {"layers": [{} for _ in range(cfg.n_layers)]}
    with cf.ThreadPoolExecutor(max_workers=min(8, len(os.sched_getaffinity(0)))) as ex:
        futs = {ex.submit(inputs.stack_tensor, cfg, n, li): (n, li) for n, li in jobs}
        done = 0
        for f in cf.as_completed(futs):
            n, li = futs[f]
            t = up(f.result())
            if li < 0:
                w[n] = t
            else:
                w["layers"][li][n] = t
            done += 1
            if done % 24 == 0:
                print(f"weights {done}/{len(jobs)} ({time.perf_counter() - t0:.0f} s)", file=sys.stderr, flush=True)
    shape = model.ModelShape(cfg.n_layers, cfg.d, cfg.n_heads, cfg.head_dim, cfg.ffn, cfg.vocab, cfg.seq)
    lc = model.LoopConfig(prompt_len=cfg.prompt_len, gen_len=cfg.gen_len, block_len=cfg.block_len, flow=flow,
                          codec=codec)
    den = model.Denoiser(w, shape, cfg.batch, lc)
    print(f"weights ready ({time.perf_counter() - t0:.0f} s); generating", file=sys.stderr, flush=True)
    y, st = den.generate(inputs.stack_prompt(cfg), progress=lambda blk, f: print(
        f"block {blk} done, {f} forwards ({time.perf_counter() - t0:.0f} s)", file=sys.stderr, flush=True))
    assert not (y == shape.mask_id).any()
    kinds = {"all": st["full_entries"] + st["window_entries"], "refresh": st["refreshing_steps"],
             "plain": st["plain_steps"]}
    per_fwd = {k: round(st["forward_gpu_ms"][k] / n, 3) for k, n in kinds.items() if n}
    out = {"metric": "denoising-loop tokens/s, whole stack", "value": round(cfg.batch * cfg.gen_len / st["seconds"], 1),
           "unit": "tokens/s", "n_gpus": 1, "higher_is_better": True, "dtype": cfg.dtype, "data": "synthetic",
           "config": {"workload": f"{cfg.name}: {cfg.n_layers} layers, d {cfg.d}, {cfg.n_heads}x{cfg.head_dim} MHA, "
                                  f"SwiGLU {cfg.ffn}, vocab {cfg.vocab}, batch {cfg.batch}, prompt {cfg.prompt_len}, "
                                  f"{cfg.gen_len} generated in blocks of {cfg.block_len}, random N(0, 0.02) weights",
                      "flow": flow, "codec": codec,
                      "global_batch": cfg.batch, "seq_len": cfg.seq},
           "tpf": round(st["tpf"], 3), "forwards": st["forwards"], "committed": st["committed"],
           "suffix_committed": st["suffix_committed"], "seconds": round(st["seconds"], 3),
           "forwards_by_kind": kinds, "gpu_ms_per_forward": per_fwd,
           "gpu_ms_per_layer_forward": {k: round(v / cfg.n_layers, 4) for k, v in per_fwd.items()}}
    print(json.dumps(out), flush=True)
    return 0


def main():
    args = parse()
    if args.summarize_counters:
        from paper_2607_14107_amd import inputs
        return summarize_counters(*args.summarize_counters, args.call, inputs.CONFIGS[args.config].name)
    if args.copy_calibration:
        return copy_calibration()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the layer step shards over the batch with no exchange between GPUs)", file=sys.stderr)
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
    if args.stack is not None:
        return stack_bench(args.stack, P, torch, args.flow, args.codec)

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

    def call(name, s):
        sh = step.shape
        if name == "drift":
            P.drift(s["h_cur"], s["h_prev"], out=step.drift)
        elif name == "select":
            if k > 0:
                P.select(step.drift, k, sh["block_start"], sh["block_len"], None, step.stale_idx, step.stale_count)
        elif name == "refresh_kv":
            P.refresh_kv(s["h_cur"], step.stale_idx, step.stale_count, sh["block_start"], sh["block_len"],
                         s["w_k"], s["w_v"], s["k_cache"], s["v_cache"], workspace=step.ws_refresh)
        elif name == "project_q":
            P.project_q(s["h_cur"], s["w_q"], sh["block_start"], sh["block_len"], sh["n_heads"],
                        out=step.q_buf, workspace=step.ws_q)
        elif name == "attend":
            P.attend(None, None, s["k_cache"], s["v_cache"], sh["block_start"], sh["block_len"],
                     sh["n_heads"], q_buf=step.q_buf, out=step.out, lse=step.lse, workspace=step.ws_attend)
        else:
            P.commit(s["logits"], s["masked"], step.drift, sh["block_start"], s["hist"], s["hist_len"], -1,
                     cfg.tau_s, cfg.alpha, False, step.token, step.conf, step.commit, workspace=step.ws_commit)

    def run_serial(i, ev):
        """One step with every call on the launch stream and events around
        each (the per-call breakdown)."""
        s = sets[i % copies]
        for j, name in enumerate(CALLS):
            ev[j].record(stream)
            call(name, s)
        ev[len(CALLS)].record(stream)

    # the step as it runs in the timed region: polestar_step, with its
    # arguments built once per input copy
    prepared = [step.prepare(c["h_cur"], c["h_prev"], c["w_q"], c["w_k"], c["w_v"], c["k_cache"],
                             c["v_cache"], c["logits"], c["masked"], c["hist"], c["hist_len"],
                             tau_s=cfg.tau_s, alpha=cfg.alpha) for c in sets]

    def run_step(i, ev=None):
        step.launch(prepared[i % copies], ev)

    for i in range(args.warmup):
        run_step(i)
    torch.cuda.synchronize()

    # diagnostic pass (untimed): the six calls one by one with events around
    # each give the per-call breakdown
    # each give the per-call breakdown.  A device-side spin enqueued first
    # lets the host queue the whole pass ahead of the GPU, so the events time
    # the kernels back to back rather than the Python launch path.
    ndiag = max(1, min(args.steps, 50))
    dev_events = [[torch.cuda.Event(enable_timing=True) for _ in range(len(CALLS) + 1)] for _ in range(ndiag)]
    torch.cuda.synchronize()
    torch.cuda._sleep(100_000_000)
    for i in range(ndiag):
        run_serial(i, dev_events[i])
    torch.cuda.synchronize()
    call_us = {c: float(np.mean([ev[j].elapsed_time(ev[j + 1]) * 1e3 for ev in dev_events]))
               for j, c in enumerate(CALLS)}
    dom = "refresh_kv"   # the step's dominant launch group; polestar_step brackets it with events

    # timed region: K whole steps through polestar_step; its refresh launches
    # are bracketed by HIP events recorded on the launch stream
    events = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(args.steps)]
    for ev in events:             # create the events before timing
        ev[0].record(stream)
        ev[1].record(stream)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        run_step(args.warmup + i, events[i])
    enqueued = time.perf_counter() - t0
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    dom_us = float(np.mean([ev[0].elapsed_time(ev[1]) * 1e3 for ev in events]))

    proxy = measure_proxy(P, torch, cfg, sets[0], stream, es)

    tokens = cfg.batch * cfg.block_len
    value = tokens * args.steps / elapsed
    cost = algorithmic_cost(cfg, k, es)
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
    roof["launch_us"] = round(dom_us, 3)
    roof["traffic"] = traffic_for(dom, cfg.name)

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
        "proxy_drift": proxy,
        "host_enqueue_us_per_step": round(enqueued / args.steps * 1e6, 2),
        "calls_us": calls,
    }
    out["gather_scatter"] = measure_gather_scatter(P, torch, cfg, sets, step.stale_idx, step.stale_count, es)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, x, k, args.cpu_seconds)
    print(json.dumps(out))
    return 0


if __name__ == "__main__":
    sys.exit(main())
