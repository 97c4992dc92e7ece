"""Benchmark of one Polestar layer step on one MI355X.

    python bench.py [--steps K] [--warmup W] [--config 1] [--subrun 1]

A step is the whole hot path over one batch: drift -> select -> sparse K/V
refresh -> Q projection of the active block -> bidirectional attention ->
commit, one polestar_step call on one stream (its fused launches: drift
beside the vocabulary scan, select beside the Q projection, the refresh
GEMM, the split-K reductions, attention, and the attention merge beside the
commit finalize).  The default workload is the LLaDA-8B-shaped layer (bf16,
batch 1, d=4096, 32 heads of 128, sequence 768 = prompt 512 + 256 generated,
active block 32, vocabulary 126464) with 15% of the positions heavily
perturbed.  Inputs are seeded synthetic data, resident in HBM before timing.

To measure HBM rather than the 256 MB Infinity Cache, every step reads one of
R independent copies of all inputs and weights (R * working set > 256 MB),
round robin.  The JSON line holds, beside the contract's keys:
  - roofline: the dominant launch group (the refresh) from HIP events that
    polestar_step records on its launch stream around those launches, on
    every timed step;
  - step_us: median, p10 and p90 of per-step times over at least 50 steps
    (HIP events around each step, after the timed region);
All of these events are created with hipEventDisableSystemFence: recording
one then skips the system-scope release (an L2 write-back and invalidate
between two launches), which a default event performs and which added about
4 us per event to the step it sat in.
  - calls_us: the six calls one by one (median over 50 passes), each with its
    algorithmic bytes and flops, its fractions of HBM and MFMA peak and of its
    attainable roofline max(bytes / HBM peak, flops / MFMA peak);
  - copy_GB_s: a plain 1 GiB device copy, the achievable-bandwidth yardstick;
  - extra_configs: the same step summary on the batch-8 LLaDA-8B layer (10%
    stale, the middle of its three chained steps) and the Dream-7B GQA layer;
  - cpu_baseline: the oracle, per step function, with all host cores and with
    one thread.

Counters (rocprofv3 --pmc) come from a separate pass:

    python bench.py --counter-pass --record-digest DIR/digest.json   # under rocprofv3 --pmc
    python bench.py --copy-calibration                               # FETCH/WRITE scale factor
    python bench.py --summarize-counters FETCH_DIR WRITE_DIR COPY_FETCH_DIR COPY_WRITE_DIR [--mfma-dir DIR]

The counter pass runs each call (and the whole fused step) on its own,
separated by one-element fill kernels, so every dispatch after the opening
marker belongs to a known call; the summary (profiles/counters_<workload>.json)
holds HBM bytes per call and per fused kernel, MFMA operation counts and busy
cycles, and the source digest recorded when the counters were taken.
"""

from __future__ import annotations

import argparse
import ctypes
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
COUNTER_CALLS = CALLS + ("gather", "scatter", "step")
COPY_BYTES = 1 << 30
MARKER_RUN = 3                 # back-to-back marker fills that open the counter pass
EVENT_NO_SYSTEM_FENCE = 0x20000000   # hipEventDisableSystemFence (hip_runtime_api.h)


class TimingEvents:
    """HIP events for timing only, created with hipEventDisableSystemFence
    through the HIP runtime this process has already loaded (torch's): a
    default event's system-scope release writes back and invalidates the
    caches between the launches it separates, which both perturbs and
    lengthens what it times."""

    def __init__(self, torch):
        torch.cuda.init()
        path = None
        with open("/proc/self/maps") as f:
            for line in f:
                parts = line.split()
                if len(parts) >= 6 and os.path.basename(parts[-1]).startswith("libamdhip64"):
                    path = parts[-1]
                    break
        if path is None:
            raise RuntimeError("the HIP runtime is not loaded in this process")
        self.hip = ctypes.CDLL(path)
        self.hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        self.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.made = []

    def new(self) -> int:
        e = ctypes.c_void_p()
        if self.hip.hipEventCreateWithFlags(ctypes.byref(e), EVENT_NO_SYSTEM_FENCE) != 0:
            raise RuntimeError("hipEventCreateWithFlags failed")
        self.made.append(e.value)
        return e.value

    def record(self, ev: int, stream) -> None:
        if self.hip.hipEventRecord(ev, stream.cuda_stream) != 0:
            raise RuntimeError("hipEventRecord failed")

    def us(self, e0: int, e1: int) -> float:
        ms = ctypes.c_float()
        if self.hip.hipEventElapsedTime(ctypes.byref(ms), e0, e1) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value * 1e3

    def close(self) -> None:
        for e in self.made:
            self.hip.hipEventDestroy(e)
        self.made = []


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--config", type=int, default=1)
    p.add_argument("--subrun", type=int, default=1)
    p.add_argument("--copies", type=int, default=0, help="input copies rotated (0: enough for 512 MB)")
    p.add_argument("--stats-steps", type=int, default=100, help="steps timed one by one for the percentiles (>= 50)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-extras", action="store_true", help="skip the batch-8 and Dream-7B summaries")
    p.add_argument("--cpu-seconds", type=float, default=12.0)
    p.add_argument("--copy-calibration", action="store_true",
                   help="run a plain 1 GiB device copy (counter scale factor) and exit")
    p.add_argument("--counter-pass", action="store_true",
                   help="run every call on its own between marker kernels (for rocprofv3 --pmc) and exit")
    p.add_argument("--counter-rounds", type=int, default=12)
    p.add_argument("--record-digest", default=None, metavar="PATH",
                   help="write the digests of the sources the kernels are built from to PATH")
    p.add_argument("--summarize-counters", nargs=4, metavar=("FETCH_DIR", "WRITE_DIR", "COPY_FETCH", "COPY_WRITE"),
                   help="write profiles/counters_<workload>.json from rocprofv3 --pmc output of --counter-pass")
    p.add_argument("--mfma-dir", default=None, help="--summarize-counters: directory of the MFMA counter pass")
    p.add_argument("--stack", type=int, default=None,
                   help="run the denoising loop of a whole layer stack (4: LLaDA-8B-shaped, 32 layers, batch 16) "
                        "once and print its tokens/s and tokens per forward instead of the layer-step benchmark")
    p.add_argument("--flow", default="window", choices=("window", "packet"),
                   help="--stack: window forwards with per-token drift, or the update-packet flow with proxy drift")
    p.add_argument("--codec", default=None, choices=("mxfp4", "mxfp8"),
                   help="--stack --flow packet: keep the window's cached inputs as quantized residuals")
    return p.parse_args()


def workload_name(cfg, subrun):
    frac = cfg.heavy_fracs[subrun]
    return f"{cfg.name}-heavy{int(round(frac * 100)):02d}"


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
    cost["step"] = dict(bytes=sum(c["bytes"] for c in cost.values()), flops=sum(c["flops"] for c in cost.values()))
    return cost


def roofline_numbers(nbytes, flops, us, dtype):
    """Rates and fractions of one call: HBM and MFMA fractions of peak and
    the fraction of its attainable roofline max(bytes / HBM, flops / MFMA)."""
    t = us * 1e-6
    peak_t = BF16_PEAK_TFLOPS if dtype == "bf16" else FP32_PEAK_TFLOPS
    roof_us = max(nbytes / (HBM_PEAK_GBS * 1e9), flops / (peak_t * 1e12)) * 1e6
    return {"us": round(us, 3), "bytes": int(nbytes), "flops": int(flops),
            "GB_s": round(nbytes / t / 1e9, 1), "hbm_frac": round(nbytes / t / 1e9 / HBM_PEAK_GBS, 4),
            "TFLOP_s": round(flops / t / 1e12, 3), "mfma_frac": round(flops / t / 1e12 / peak_t, 4),
            "roofline_us": round(roof_us, 3), "roofline_frac": round(roof_us / us, 4),
            "bound": "mfma" if flops / (peak_t * 1e12) > nbytes / (HBM_PEAK_GBS * 1e9) else "hbm"}


# Sources each call's kernels are built from (a change retires its counters).
CALL_SOURCES = {
    "refresh_kv": ("gemm.hip", "gemm.hpp", "gemm_dev.hpp", "step.hip"),
    "project_q": ("attend.hip", "gemm.hip", "gemm.hpp", "gemm_dev.hpp"),
    "attend": ("attend.hip", "attend_dev.hpp", "attend_ring.hip"),
    "drift": ("drift.hip", "drift_dev.hpp"),
    "select": ("select.hip", "select_dev.hpp"),
    "commit": ("commit.hip", "commit_dev.hpp"),
    "gather": ("model.hip",),
    "scatter": ("model.hip",),
    "step": ("step.hip", "drift_dev.hpp", "select_dev.hpp", "gemm_dev.hpp", "gemm.hip", "attend_dev.hpp",
             "attend_ring.hip", "commit_dev.hpp"),
}


def source_digest(call):
    h = hashlib.sha256()
    for f in CALL_SOURCES[call] + ("common.hpp", "host_common.hpp"):
        with open(os.path.join(ROOT, "paper_2607_14107_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def source_digests():
    return {c: source_digest(c) for c in COUNTER_CALLS}


def counters_path(workload):
    return os.path.join(ROOT, "profiles", f"counters_{workload}.json")


def traffic_for(call_key, workload):
    """Counted HBM bytes per launch of `call_key` ("refresh_kv" in the fused
    step: its GEMM and reduction launches) from the committed counter summary,
    or None when there is none or the sources changed since it was taken."""
    path = counters_path(workload)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("source_digests", {}).get("step") != source_digest("step"):
        return None
    return t.get("step_kernels", {}).get(call_key, {}).get("bytes")


def copy_bandwidth(torch, reps=10):
    """A plain device copy of COPY_BYTES, median of `reps` (read + write bytes
    per second): the bandwidth a streaming kernel achieves on this GPU."""
    src = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1.0)
    dst.copy_(src)
    times = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        dst.copy_(src)
        e1.record()
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1) * 1e-3)
    del src, dst
    return round(2 * COPY_BYTES / float(np.median(times)) / 1e9, 1)


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


# ---------------------------------------------------------------------------
# Counter summaries
# ---------------------------------------------------------------------------

def _counter_rows(directory, counter):
    """(dispatch id, kernel name, value) per dispatch, in dispatch order, from
    the counter CSVs rocprofv3 --pmc wrote under `directory`."""
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


def _is_marker(name):
    # the counter pass's markers fill a float64 tensor; nothing else in the
    # process runs a float64 fill
    return "FillFunctor<double>" in name


def _segments(rows):
    """Split the dispatches after the opening run of markers into per-call
    segments: [(call, [(name, value), ...]), ...] in COUNTER_CALLS order."""
    start = None
    for i in range(len(rows) - MARKER_RUN + 1):
        if all(_is_marker(rows[i + j][1]) for j in range(MARKER_RUN)):
            start = i + MARKER_RUN
            break
    if start is None:
        raise SystemExit("no opening marker run: was the run made with --counter-pass?")
    while start < len(rows) and _is_marker(rows[start][1]):
        start += 1                    # the whole run; its last marker opens the first call
    start -= 1
    segs, cur = [], None
    for _, name, v in rows[start:]:
        if _is_marker(name):
            if cur is not None:
                segs.append(cur)
            cur = []
        elif cur is not None:
            cur.append((name, v))
    if cur:
        segs.append(cur)
    return [(COUNTER_CALLS[i % len(COUNTER_CALLS)], s) for i, s in enumerate(segs)]


# roles of the fused step's kernels, by name
STEP_ROLES = (("lead", ("lead_kernel",)), ("front", ("front_kernel", "front_dma_kernel", "select_kernel")),
              ("refresh_kv", ("gemm_", "reduce2_kernel", "tile_qred_kernel")), ("attend", ("attend_",)),
              ("back", ("back_kernel",)))


def _step_role(name):
    for role, pats in STEP_ROLES:
        if any(p in name for p in pats):
            return role
    return "other"


def _per_call(segs):
    """Median over rounds of the summed value per call, and per role of the
    fused step's kernels."""
    calls, roles = {}, {}
    for call, seg in segs:
        calls.setdefault(call, []).append(sum(v for _, v in seg))
        if call == "step":
            per = {}
            for name, v in seg:
                per[_step_role(name)] = per.get(_step_role(name), 0.0) + v
            for r, v in per.items():
                roles.setdefault(r, []).append(v)
    med = lambda xs: float(np.median(xs))
    return {c: med(v) for c, v in calls.items()}, {r: med(v) for r, v in roles.items()}


def summarize_counters(fetch_dir, write_dir, copy_fetch_dir, copy_write_dir, mfma_dir, cfg, subrun):
    from paper_2607_14107_amd import inputs
    x = inputs.layer_inputs(cfg, subrun)
    k = int(x["k"])
    cost = algorithmic_cost(cfg, k, 2 if cfg.dtype == "bf16" else 4)
    workload = workload_name(cfg, subrun)

    def copy_kib(d, counter):
        vals = [v for _, n, v in _counter_rows(d, counter) if "copy" in n.lower()]
        if not vals:
            raise SystemExit(f"no copy dispatch with {counter} under {d}")
        return float(np.median(vals))

    def digest_of(d):
        with open(os.path.join(d, "digest.json")) as f:
            return json.load(f)

    rec = digest_of(fetch_dir)
    if digest_of(write_dir)["source_digests"] != rec["source_digests"]:
        raise SystemExit("FETCH and WRITE passes ran on different sources")
    f_fetch = COPY_BYTES / (copy_kib(copy_fetch_dir, "FETCH_SIZE") * 1024)
    f_write = COPY_BYTES / (copy_kib(copy_write_dir, "WRITE_SIZE") * 1024)
    fetch, fetch_roles = _per_call(_segments(_counter_rows(fetch_dir, "FETCH_SIZE")))
    write, write_roles = _per_call(_segments(_counter_rows(write_dir, "WRITE_SIZE")))
    calls = {}
    for c in COUNTER_CALLS:
        if c not in fetch:
            continue
        nb = fetch[c] * 1024 * f_fetch + write[c] * 1024 * f_write
        calls[c] = {"fetch_bytes": int(fetch[c] * 1024 * f_fetch), "write_bytes": int(write[c] * 1024 * f_write),
                    "bytes": int(nb)}
        if c in cost:
            calls[c]["algorithmic_bytes"] = int(cost[c]["bytes"])
            calls[c]["ratio"] = round(nb / cost[c]["bytes"], 3)
    step_kernels = {r: {"fetch_bytes": int(fetch_roles[r] * 1024 * f_fetch),
                        "write_bytes": int(write_roles.get(r, 0.0) * 1024 * f_write),
                        "bytes": int(fetch_roles[r] * 1024 * f_fetch + write_roles.get(r, 0.0) * 1024 * f_write)}
                    for r in fetch_roles}
    t = {"workload": workload, "stale_rows": k, "calls": calls, "step_kernels": step_kernels,
         "copy_scale_fetch": round(f_fetch, 4), "copy_scale_write": round(f_write, 4),
         "source_digests": rec["source_digests"]}
    if mfma_dir:
        if digest_of(mfma_dir)["source_digests"] != rec["source_digests"]:
            raise SystemExit("the MFMA pass ran on different sources")
        mops, mops_roles = _per_call(_segments(_counter_rows(mfma_dir, "SQ_INSTS_VALU_MFMA_MOPS_BF16")))
        busy, busy_roles = _per_call(_segments(_counter_rows(mfma_dir, "SQ_VALU_MFMA_BUSY_CYCLES")))
        gui, gui_roles = _per_call(_segments(_counter_rows(mfma_dir, "GRBM_GUI_ACTIVE")))
        mf = {}
        for c in COUNTER_CALLS:
            if c in mops and mops[c] > 0:
                mf[c] = {"mfma_flops": int(mops[c] * 512), "mfma_busy_cycles": int(busy.get(c, 0)),
                         "gui_active_cycles": int(gui.get(c, 0))}
                if c in cost and cost[c]["flops"]:
                    mf[c]["algorithmic_flops"] = int(cost[c]["flops"])
        t["mfma"] = mf
        t["mfma_step_kernels"] = {r: {"mfma_flops": int(mops_roles[r] * 512),
                                      "mfma_busy_cycles": int(busy_roles.get(r, 0)),
                                      "gui_active_cycles": int(gui_roles.get(r, 0))}
                                  for r in mops_roles if mops_roles[r] > 0}
    t["commands"] = [
        "cd /tmp && export TMPDIR=/tmp",
        f"rocprofv3 --pmc FETCH_SIZE -f csv -d $OUT/f -o c -- python3 $R/bench.py --config {cfg.index} "
        f"--subrun {subrun} --counter-pass --record-digest $OUT/f/digest.json",
        f"rocprofv3 --pmc WRITE_SIZE -f csv -d $OUT/w -o c -- python3 $R/bench.py --config {cfg.index} "
        f"--subrun {subrun} --counter-pass --record-digest $OUT/w/digest.json",
        f"rocprofv3 --pmc SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE -f csv -d $OUT/m "
        f"-o c -- python3 $R/bench.py --config {cfg.index} --subrun {subrun} --counter-pass "
        f"--record-digest $OUT/m/digest.json",
        "rocprofv3 --pmc FETCH_SIZE -f csv -d $OUT/cf -o c -- python3 $R/bench.py --copy-calibration",
        "rocprofv3 --pmc WRITE_SIZE -f csv -d $OUT/cw -o c -- python3 $R/bench.py --copy-calibration",
        f"python3 $R/bench.py --config {cfg.index} --subrun {subrun} --summarize-counters $OUT/f $OUT/w "
        f"$OUT/cf $OUT/cw --mfma-dir $OUT/m",
    ]
    t["note"] = ("per call: median over the counter pass's rounds of the counter summed over the call's "
                 "dispatches (between marker fills); bytes = KiB * 1024 * (copy bytes / copy counter bytes); "
                 "mfma_flops = SQ_INSTS_VALU_MFMA_MOPS_BF16 * 512; $R is the repository, $OUT any directory")
    with open(counters_path(workload), "w") as f:
        json.dump(t, f, indent=1)
        f.write("\n")
    print(json.dumps(t))
    return 0


# ---------------------------------------------------------------------------
# One layer workload on the GPU
# ---------------------------------------------------------------------------

class Layer:
    """Inputs of one workload in HBM (R rotated copies), the Step buffers
    and the prepared polestar_step arguments of every copy."""

    def __init__(self, P, torch, cfg, subrun, copies=0):
        from paper_2607_14107_amd import inputs
        self.P, self.torch, self.cfg, self.subrun = P, torch, cfg, subrun
        self.events = TimingEvents(torch)
        x = inputs.layer_inputs(cfg, subrun)
        self.x = x
        self.k = k = int(x["k"])
        self.dt = dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
        self.es = es = 2 if cfg.dtype == "bf16" else 4
        dev = torch.device("cuda", 0)

        def up(a):
            if cfg.dtype == "bf16":
                return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)
            return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)

        # working set of one copy; enough copies to exceed the Infinity Cache twice
        ws_bytes = sum(x[n].nbytes for n in ("h_cur", "h_prev", "w_q", "w_k", "w_v", "logits")) \
            + 2 * cfg.batch * cfg.seq * cfg.n_kv_heads * cfg.head_dim * es
        self.copies = copies or max(1, -(-512 * 2 ** 20 // ws_bytes))
        self.sets = []
        for _ in range(self.copies):
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
            self.sets.append(s)
        self.step = P.Step(batch=cfg.batch, seq=cfg.seq, d=cfg.d, n_heads=cfg.n_heads, n_kv_heads=cfg.n_kv_heads,
                           head_dim=cfg.head_dim, block_start=cfg.block_start, block_len=cfg.block_len,
                           vocab=cfg.vocab, k=k, dtype=dt, device=dev)
        self.prepared = [self.step.prepare(c["h_cur"], c["h_prev"], c["w_q"], c["w_k"], c["w_v"], c["k_cache"],
                                           c["v_cache"], c["logits"], c["masked"], c["hist"], c["hist_len"],
                                           tau_s=cfg.tau_s, alpha=cfg.alpha) for c in self.sets]
        self.stream = torch.cuda.current_stream()
        self.cost = algorithmic_cost(cfg, k, es)
        if k > 0:   # packet buffers of the gather / scatter calls
            kvd = cfg.n_kv_heads * cfg.head_dim
            self.packet = torch.empty((cfg.batch, k, cfg.d), dtype=dt, device=dev)
            self.krows = [torch.zeros((cfg.batch, k, kvd), dtype=dt, device=dev) for _ in self.sets]
        torch.cuda.synchronize()

    def call(self, name, i):
        """One stand-alone call on input copy i % copies."""
        P, st, cfg, k = self.P, self.step, self.cfg, self.k
        s = self.sets[i % self.copies]
        sh = st.shape
        if name == "drift":
            P.drift(s["h_cur"], s["h_prev"], out=st.drift)
        elif name == "select":
            if k > 0:
                P.select(st.drift, k, sh["block_start"], sh["block_len"], None, st.stale_idx, st.stale_count)
        elif name == "refresh_kv":
            P.refresh_kv(s["h_cur"], st.stale_idx, st.stale_count, sh["block_start"], sh["block_len"],
                         s["w_k"], s["w_v"], s["k_cache"], s["v_cache"], workspace=st.ws_refresh)
        elif name == "project_q":
            P.project_q(s["h_cur"], s["w_q"], sh["block_start"], sh["block_len"], sh["n_heads"],
                        out=st.q_buf, workspace=st.ws_q)
        elif name == "attend":
            P.attend(None, None, s["k_cache"], s["v_cache"], sh["block_start"], sh["block_len"],
                     sh["n_heads"], q_buf=st.q_buf, out=st.out, lse=st.lse, workspace=st.ws_attend)
        elif name == "commit":
            P.commit(s["logits"], s["masked"], st.drift, sh["block_start"], s["hist"], s["hist_len"], -1,
                     cfg.tau_s, cfg.alpha, False, st.token, st.conf, st.commit, workspace=st.ws_commit)
        elif name == "gather":
            if k > 0:
                P.gather_rows(s["h_cur"], st.stale_idx, st.stale_count, self.packet)
        elif name == "scatter":
            if k > 0:
                kvd = cfg.n_kv_heads * cfg.head_dim
                P.scatter_rows(self.krows[i % self.copies], st.stale_idx, st.stale_count,
                               s["k_cache"].view(cfg.batch, cfg.seq, kvd))
        elif name == "step":
            self.run_step(i)
        else:
            raise ValueError(name)

    def run_step(self, i, ev=None):
        self.step.launch(self.prepared[i % self.copies], ev)

    def _spin(self):
        # a device-side spin ahead of a batch of launches lets the host queue
        # them all before the GPU starts, so events time the kernels back to
        # back rather than the Python launch path
        self.torch.cuda.synchronize()
        self.torch.cuda._sleep(100_000_000)

    def calls_us(self, n=50):
        """The six calls one by one with events around each: median µs."""
        torch, te = self.torch, self.events
        ev = [[te.new() for _ in range(len(CALLS) + 1)] for _ in range(n)]
        self._spin()
        for i in range(n):
            for j, name in enumerate(CALLS):
                te.record(ev[i][j], self.stream)
                self.call(name, i)
            te.record(ev[i][len(CALLS)], self.stream)
        torch.cuda.synchronize()
        out = {c: float(np.median([te.us(e[j], e[j + 1]) for e in ev])) for j, c in enumerate(CALLS)}
        te.close()
        return out

    def step_stats(self, n, first=0):
        """Per-step times (µs) of n consecutive steps, events between steps."""
        torch, te = self.torch, self.events
        ev = [te.new() for _ in range(n + 1)]
        self._spin()
        te.record(ev[0], self.stream)
        for i in range(n):
            self.run_step(first + i)
            te.record(ev[i + 1], self.stream)
        torch.cuda.synchronize()
        t = np.array([te.us(ev[i], ev[i + 1]) for i in range(n)])
        te.close()
        return {"n": n, "median": round(float(np.median(t)), 3), "p10": round(float(np.percentile(t, 10)), 3),
                "p90": round(float(np.percentile(t, 90)), 3), "mean": round(float(t.mean()), 3)}

    def calls_report(self, call_us):
        return {c: roofline_numbers(self.cost[c]["bytes"], self.cost[c]["flops"], call_us[c], self.cfg.dtype)
                for c in CALLS}

    def counter_pass(self, rounds):
        """Every call of COUNTER_CALLS on its own, `rounds` times, each preceded
        by a one-element float64 fill (the marker the counter summary splits
        on); the pass opens with MARKER_RUN fills back to back."""
        torch = self.torch
        marker = torch.zeros(1, dtype=torch.float64, device="cuda")
        torch.cuda.synchronize()
        for j in range(MARKER_RUN):
            marker.fill_(float(j))
        for r in range(rounds):
            for c in COUNTER_CALLS:
                marker.fill_(float(r))
                self.call(c, r)
        marker.fill_(-1.0)
        torch.cuda.synchronize()


def layer_summary(P, torch, cfg_index, subrun, n_steps=60):
    """The step of another workload: per-step percentiles and the calls
    against their rooflines (an extra key of the bench line)."""
    from paper_2607_14107_amd import inputs
    cfg = inputs.CONFIGS[cfg_index]
    L = Layer(P, torch, cfg, subrun)
    for i in range(5):
        L.run_step(i)
    stats = L.step_stats(n_steps, 5)
    calls = L.calls_report(L.calls_us(30))
    tokens = cfg.batch * cfg.block_len
    out = {"workload": workload_name(cfg, subrun),
           "shape": f"batch {cfg.batch}, seq {cfg.seq}, block {cfg.block_len}, d {cfg.d}, heads "
                    f"{cfg.n_heads}/{cfg.n_kv_heads}x{cfg.head_dim}, vocab {cfg.vocab}, {L.k} stale rows per sequence",
           "tokens_per_s": round(tokens / (stats["median"] * 1e-6), 1), "step_us": stats, "calls_us": calls}
    del L
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out


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
    """The oracle as it stands, timed on the host per step function on the
    benchmarked workload: median of at least 3 runs each, with the BLAS pool
    at every core this process may use and again with one thread; tokens/s
    = tokens of one step / the summed medians."""
    from oracle import polestar_ref as ref
    cores = len(os.sched_getaffinity(0))
    dec = {n: ref.decode(x[n], cfg.dtype) for n in ("h_cur", "h_prev", "w_q", "w_k", "w_v")}
    shape = (cfg.batch, cfg.seq, cfg.n_kv_heads, cfg.head_dim)
    kc = ref.round_to((dec["h_prev"] @ dec["w_k"].T).reshape(shape), cfg.dtype)
    vc = ref.round_to((dec["h_prev"] @ dec["w_v"].T).reshape(shape), cfg.dtype)
    logits = ref.decode(x["logits"], cfg.dtype)
    bs, bl = cfg.block_start, cfg.block_len
    st = {}

    def f_drift():
        st["d"] = ref.drift(dec["h_cur"], dec["h_prev"])

    def f_select():
        st["idx"], st["cnt"] = ref.select(st["d"], k, bs, bl)

    def f_refresh():
        kn, vn, _ = ref.refresh_kv(dec["h_cur"], dec["w_k"], dec["w_v"], kc, vc, st["idx"], st["cnt"], bs, bl)
        st["k"], st["v"] = ref.round_to(kn, cfg.dtype), ref.round_to(vn, cfg.dtype)

    def f_q():
        st["q"] = ref.q_project(dec["h_cur"], dec["w_q"], bs, bl, cfg.n_heads, cfg.head_dim)

    def f_attend():
        ref.attend(ref.round_to(st["q"], cfg.dtype), st["k"], st["v"])

    def f_commit():
        _, conf = ref.confidence(logits, -1)
        delta = st["d"][:, bs:bs + bl].astype(np.float32)
        ref.commit_rule(conf.astype(np.float32), delta, x["masked"].astype(bool), x["hist"], x["hist_len"],
                        cfg.hist_depth, cfg.tau_s, cfg.alpha, False)

    fns = (("drift", f_drift), ("select", f_select), ("refresh_kv", f_refresh), ("project_q", f_q),
           ("attend", f_attend), ("commit", f_commit))

    def run_all(per_fn_s):
        times = {n: [] for n, _ in fns}
        spent = 0.0
        while True:
            for n, f in fns:       # in step order: each function consumes the one before
                t0 = time.perf_counter()
                f()
                dt = time.perf_counter() - t0
                times[n].append(dt)
                spent += dt
            reps = len(times["drift"])
            if reps >= 3 and (spent >= per_fn_s * len(fns) or reps >= 50):
                break
        med = {n: float(np.median(v)) for n, v in times.items()}
        return med, reps, spent

    from threadpoolctl import threadpool_limits
    with threadpool_limits(limits=cores):
        multi, reps_m, spent_m = run_all(budget_s / len(fns) / 2)
    with threadpool_limits(limits=1):
        single, reps_s, spent_s = run_all(budget_s / len(fns) / 2)
    tok = cfg.batch * cfg.block_len
    return {"value": round(tok / sum(multi.values()), 3), "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "sample": f"{reps_m} oracle layer steps of the benchmarked workload timed per step function "
                      f"(drift, select, refresh, Q projection, attention, commit; median per function), "
                      f"{spent_m:.1f} s with {cores} BLAS threads; single-thread: {reps_s} steps, {spent_s:.1f} s",
            "per_call_s": {n: round(v, 5) for n, v in multi.items()},
            "single_thread": {"value": round(tok / sum(single.values()), 3), "cores": 1,
                              "per_call_s": {n: round(v, 5) for n, v in single.items()}}}


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
    from paper_2607_14107_amd import inputs
    if args.summarize_counters:
        return summarize_counters(*args.summarize_counters, args.mfma_dir, inputs.CONFIGS[args.config], args.subrun)
    if args.record_digest:
        os.makedirs(os.path.dirname(os.path.abspath(args.record_digest)), exist_ok=True)
        with open(args.record_digest, "w") as f:
            json.dump({"source_digests": source_digests(), "config": args.config, "subrun": args.subrun}, f)
    if args.copy_calibration:
        return copy_calibration()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the layer step shards over the batch with no exchange between GPUs)", file=sys.stderr)
        return 2

    import torch
    from paper_2607_14107_amd import polestar as P

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    if not os.path.exists(P.LIB_PATH):
        from paper_2607_14107_amd import build
        build.build(verbose=False)
    P.lib()
    torch.cuda.set_device(torch.device("cuda", 0))
    if args.stack is not None:
        return stack_bench(args.stack, P, torch, args.flow, args.codec)

    cfg = inputs.CONFIGS[args.config]
    L = Layer(P, torch, cfg, args.subrun, args.copies)
    if args.counter_pass:
        for i in range(3):
            L.run_step(i)
        L.counter_pass(args.counter_rounds)
        print(json.dumps({"counter_pass": workload_name(cfg, args.subrun), "rounds": args.counter_rounds}))
        return 0
    k, es, stream = L.k, L.es, L.stream

    dom = "refresh_kv"   # the step's dominant launch group; polestar_step brackets it with events
    # timed region: K whole steps through polestar_step right after the W
    # warm-up steps, each bracketing its refresh launches with the two timing
    # events it is given (recorded on its launch stream; without the
    # system-scope fence they cost no measurable step time: 60.6 against
    # 60.3 us per step at config 1 with events on every fifth step)
    te = L.events
    events = [(te.new(), te.new()) for _ in range(args.steps)]
    for i in range(args.warmup):
        L.run_step(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        L.run_step(args.warmup + i, events[i])
    enqueued = time.perf_counter() - t0
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    dom_us = float(np.mean([te.us(e0, e1) for e0, e1 in events]))
    te.close()

    # per-call breakdown (untimed for the headline)
    call_us = L.calls_us(max(1, min(args.steps, 50)))

    # per-step percentiles over at least 50 steps (after the timed region)
    stats = L.step_stats(max(50, args.stats_steps), args.warmup + args.steps)

    tokens = cfg.batch * cfg.block_len
    value = tokens * args.steps / elapsed
    c = L.cost[dom]
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
    roof["event_samples"] = len(events)   # every timed step
    roof["traffic"] = traffic_for(dom, workload_name(cfg, args.subrun))

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
        "config": {"workload": f"{workload_name(cfg, args.subrun)}: single "
                               f"{'LLaDA-8B' if cfg.n_heads == cfg.n_kv_heads else 'Dream-7B'}"
                               f"-shaped layer step, batch {cfg.batch}, seq {cfg.seq}, block {cfg.block_len}, "
                               f"d {cfg.d}, heads {cfg.n_heads}/{cfg.n_kv_heads}x{cfg.head_dim}, vocab {cfg.vocab}, "
                               f"{k} stale rows per sequence",
                   "global_batch": cfg.batch, "seq_len": cfg.seq, "block": cfg.block_len,
                   "stale_rows": k, "input_copies": L.copies},
        "roofline": roof,
        "step_us": stats,
        "tokens_per_s_median_step": round(tokens / (stats["median"] * 1e-6), 1),
        "host_enqueue_us_per_step": round(enqueued / args.steps * 1e6, 2),
        "calls_us": L.calls_report(call_us),
    }
    out["proxy_drift"] = measure_proxy(P, torch, cfg, L.sets[0], stream, es)
    out["gather_scatter"] = measure_gather_scatter(P, torch, cfg, L.sets, L.step.stale_idx, L.step.stale_count, es)
    x = L.x
    del L
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    out["copy_GB_s"] = copy_bandwidth(torch)
    if not args.no_extras and args.config == 1:
        out["extra_configs"] = {"llada8b_b8": layer_summary(P, torch, 2, 1), "dream7b_b4": layer_summary(P, torch, 3, 0)}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, x, k, args.cpu_seconds)
    print(json.dumps(out))
    return 0


if __name__ == "__main__":
    sys.exit(main())
