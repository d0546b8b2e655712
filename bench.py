"""Benchmark of the ARCHead packed LM-head forward on one MI355X.

Workload (N=1): the Qwen3-8B-shaped packed head (V=151936, d=4096, INT4
residual in groups of 128 with fp16 scales, core rank 64, correction rank 32,
INT8 factors), synthetic seeded inputs.  A step is one forward of the whole
hot path (stage-1 projections, head-streaming kernel with the fused rank-r
expansion, logit store) for one decode token (M=1), with every input already
resident in HBM.  The step rotates over three copies of the packed head
(3 x 336 MB > the 256 MB Infinity Cache), so each step streams its head from
HBM.  The headline value is decode GB/s over the packed bytes.  Secondary
lines: decode M=4, 16, 32 and 64, decode M=1 of the same head with 8-bit
residual scale codes, greedy decoding (the fused argmax, no logits written)
and top-10 selection at M=1 and 16, and the M=4096 prefill fused-CE pass
(tok/s and the many-token kernel's MFMA throughput).  The tiled kernel's
head-derived tables are prepared once per head copy (archead_prepare).

Before any timing, about 0.5 s of untimed decode steps bring the GPU's clocks
to their sustained-load state (--clock-warmup; a cold GPU runs the first
~100 ms of steps ~10% slower); then each line does its own --warmup steps
and times exactly --steps steps.

Prints one JSON line (rank 0, N=1).  --gpus N > 1 is refused: the
benchmark runs on one GPU.  --profile decode|prefill|topk (the M=1 top-10
selection) runs the same work without timing
or JSON, for rocprofv3 (the decode form first copies 256 MiB once, the
calibration kernel for the HBM byte counters).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "ARCHead head fwd: decode HBM GB/s (% peak) + prefill tok/s, V=151936 d=4096"
PEAK_HBM_GBS = 8000.0
PEAK_BF16_TFLOPS = 2500.0
N_COPIES = 3
CALIBRATION_BYTES = 256 << 20
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemv_qwen_decode_traffic.md")
SWEEP_PEAK_NOTE = "bf16 dense MFMA 2.5 PFLOP/s, HBM 8 TB/s"
# the decode GEMV's sources: the counters are valid while these are unchanged
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2608_02703_amd", "csrc", f)
                  for f in ("dev_common.cuh", "dev_gemv.cuh", "k_gemv.hip")]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def upload_copies(h, n):
    import torch
    from paper_2608_02703_amd import PackedHead
    base = PackedHead.from_arrays(h)
    heads = [base]
    for _ in range(n - 1):
        bufs = {k: (None if v is None else v.clone()) for k, v in base.buffers.items()}
        heads.append(PackedHead(h.V, h.d, h.g, h.rc, h.rr, bufs, h.gV, h.gB))
    torch.cuda.synchronize()
    return heads


def lib_packed_bytes(ph):
    """The packed head's persistent bytes as the library counts them
    (archead_packed_bytes: sum of element count x element size)."""
    from paper_2608_02703_amd import packed_bytes
    return packed_bytes(ph.desc)


def decode_algorithmic_bytes(pbytes, h, M):
    """Bytes one decode launch must move: the whole packed head once (pbytes:
    the residual codes and scales, the factors and their scales, V_c and B_w
    for the in-launch stage 1), x, and the fp32 logits it writes."""
    return pbytes + M * h.d * 2 + M * h.V * 4


def lanes_per_row(h):
    """Lanes per vocabulary row of the decode GEMV (the library's rule)."""
    chunks = h.d // 32
    lpr = 16
    while lpr > 1 and chunks % lpr:
        lpr //= 2
    r4 = (h.rc + h.rr) // 4
    while lpr < 64 and r4 > 2 * lpr and chunks % (2 * lpr) == 0:
        lpr *= 2
    return lpr


def mfma_algorithmic_flops(h, M):
    """Multiply-adds x 2 of one many-token pass: the residual contraction
    over d and the rank-r expansion over r_c + r_r."""
    return 2.0 * M * h.V * (h.d + h.rc + h.rr)


def source_sha256():
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic():
    """HBM bytes per decode launch from the committed counter summary, or
    None if it is missing or was taken on a different kernel source."""
    try:
        text = open(TRAFFIC_FILE).read()
    except OSError:
        return None
    h = re.search(r"source_sha256:\s*([0-9a-f]{64})", text)
    t = re.search(r"traffic_bytes_per_launch:\s*([0-9]+)", text)
    if not h or not t or h.group(1) != source_sha256():
        return None
    return int(t.group(1))


def _timed_loop(fn, steps):
    """ms per call of `steps` calls, bracketed by synchronize + events (no
    per-call instrumentation)."""
    import torch
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for i in range(steps):
        fn(i)
    t1.record()
    torch.cuda.synchronize()
    return t0.elapsed_time(t1) / steps


def _step_times(fn, steps):
    """Per-step durations (ms) from events recorded between consecutive
    steps on the stream (a separate pass from the unmarked timed loop)."""
    import torch
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    for i in range(steps):
        ev[i].record()
        fn(i)
    ev[steps].record()
    torch.cuda.synchronize()
    return [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]


def _pct(v, q):
    return float(np.percentile(np.asarray(v, dtype=np.float64), q))


def _kernel_times(heads, fn, steps):
    """Per-call durations (ms) of the head-streaming kernel: HIP events
    attached to its dispatch (a separate pass; the markers cost a few us per
    call, so the step time is measured without them)."""
    import torch
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    for a, b in ev:        # create the underlying HIP events
        a.record()
        b.record()
    torch.cuda.synchronize()
    for i in range(steps):
        heads[i % len(heads)].set_timing_events(*ev[i])
        fn(i)
    torch.cuda.synchronize()
    for hd in heads:
        hd.set_timing_events(None, None)
    return [a.elapsed_time(b) for a, b in ev]


def clock_warmup(heads, x, seconds):
    """Untimed decode steps for about `seconds` of wall time before any
    measurement.  The GPU's clocks ramp up over the first ~10-100 ms of
    sustained load (a step measured right after a cold start is ~10% slower
    than in steady state); a serving loop runs in the steady state."""
    import torch
    M = x.shape[0]
    outs = [torch.empty((M, heads[0].V), device="cuda") for _ in heads]
    wss = [hd.workspace(M, 0, x.device) for hd in heads]
    t0 = time.perf_counter()
    n = 0
    while time.perf_counter() - t0 < seconds:
        for _ in range(100):
            k = n % len(heads)
            heads[k].logits(x, out=outs[k], ws=wss[k])
            n += 1
        torch.cuda.synchronize()
    return n


def time_decode(heads, x, steps, warmup, ws=None, percentiles=False):
    """(ms per step, mean head-kernel ms, median head-kernel ms[, step-time
    percentiles p10 / p50 / p90 in ms])."""
    import torch
    M = x.shape[0]
    outs = [torch.empty((M, heads[0].V), device="cuda") for _ in heads]
    wss = [hd.workspace(M, 0, x.device) for hd in heads]

    def step(i):
        k = i % len(heads)
        heads[k].logits(x, out=outs[k], ws=wss[k])
    for i in range(warmup):
        step(i)
    ms = _timed_loop(step, steps)
    kern = _kernel_times(heads, step, min(steps, 100))
    out = (ms, float(np.mean(kern)), float(np.median(kern)))
    if percentiles:
        st = _step_times(step, steps)
        out += ({"p10": _pct(st, 10), "p50": _pct(st, 50), "p90": _pct(st, 90)},)
    return out


class ClockSampler:
    """Samples the GPU's current shader clock (the level marked '*' in the
    driver's pp_dpm_sclk table) from a host thread while the GPU runs the
    timed steps; None where the table is not readable."""

    def __init__(self, period=0.01):
        import glob
        import threading
        self.paths = sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk"))
        self.period = period
        self.samples = []
        self._stop = threading.Event()
        self._t = threading.Thread(target=self._run, daemon=True)

    def _read(self):
        for p in self.paths:
            try:
                for line in open(p):
                    if line.rstrip().endswith("*"):
                        m = re.search(r"(\d+)\s*[Mm][Hh]z", line)
                        if m:
                            return int(m.group(1))
            except OSError:
                continue
        return None

    def _run(self):
        while not self._stop.is_set():
            v = self._read()
            if v is not None:
                self.samples.append(v)
            self._stop.wait(self.period)

    def __enter__(self):
        if self.paths:
            self._t.start()
        return self

    def __exit__(self, *a):
        self._stop.set()
        if self.paths:
            self._t.join()

    def summary(self):
        if not self.samples:
            return {"sclk_mhz": None, "source": "pp_dpm_sclk not readable"}
        return {"sclk_mhz_median": _pct(self.samples, 50), "sclk_mhz_min": min(self.samples),
                "sclk_mhz_max": max(self.samples), "samples": len(self.samples),
                "source": "pp_dpm_sclk current level, sampled during the decode M=1 timing"}


def copy_bandwidth(nbytes=512 << 20, iters=20):
    """Device-to-device copy of nbytes (torch copy_): GB/s counting the bytes
    read and written, the HBM rate a plain streaming kernel reaches here."""
    import torch
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    ms = _timed_loop(lambda i: dst.copy_(src), iters)
    del src, dst
    torch.cuda.empty_cache()
    return {"bytes": nbytes, "ms": round(ms, 4), "gbs_read_plus_write": round(2 * nbytes / ms / 1e6, 1),
            "frac_of_8tbs": round(2 * nbytes / ms / 1e6 / PEAK_HBM_GBS, 4),
            "op": "torch copy_ of a 512 MiB device buffer"}


def time_argmax(heads, x, steps, warmup):
    """ms per greedy step (fused argmax, no logits written)."""
    M = x.shape[0]
    wss = [hd.workspace(M, 2, x.device) for hd in heads]

    def step(i):
        k = i % len(heads)
        heads[k].logits_argmax(x, ws=wss[k])
    for i in range(warmup):
        step(i)
    return _timed_loop(step, steps)


def time_topk(heads, x, k, steps, warmup):
    """ms per top-k selection step (fused into the GEMV pass at M = 1)."""
    import torch
    M = x.shape[0]
    wss = [hd.workspace(M, 3, x.device) for hd in heads]
    vals = torch.empty((M, k), dtype=torch.float32, device=x.device)
    idx = torch.empty((M, k), dtype=torch.int64, device=x.device)

    def step(i):
        j = i % len(heads)
        heads[j].logits_topk(x, k, vals=vals, idx=idx, ws=wss[j])
    for i in range(warmup):
        step(i)
    return _timed_loop(step, steps)


def time_prefill(heads, x, y, steps, warmup, prepared=True):
    """(ms per step, mean CE, median many-token kernel ms).  prepared: the
    heads keep the many-token kernel's head-derived tables across calls
    (built once, as a server or evaluation loop does at load time); else
    every step rebuilds them in its workspace first."""
    import torch
    for hd in heads:
        hd.prepare(prepared)
    torch.cuda.synchronize()
    try:
        return _time_prefill(heads, x, y, steps, warmup)
    finally:
        for hd in heads:
            hd.prepare(False)


def _time_prefill(heads, x, y, steps, warmup):
    import torch
    ws = [hd.workspace(x.shape[0], 1, x.device) for hd in heads]
    res = {}

    def step(i):
        k = i % len(heads)
        res["ce"] = heads[k].logits_ce(x, y, ws=ws[k])
    for i in range(warmup):
        step(i)
    ms = _timed_loop(step, steps)
    kern = _kernel_times(heads, step, steps)
    return ms, float(res["ce"][1].cpu()[0]), float(np.median(kern))


def ms1_for_dense(res):
    return res[1][0]


def _oracle_threads():
    cores = len(os.sched_getaffinity(0))
    return min(cores, int(os.environ.get("OMP_NUM_THREADS", cores)))


def cpu_baseline(h, pbytes, xb, min_sec=10.0, max_tokens=16, legs=True):
    """The fp64 oracle on the host cores (the oracle as it stands, never
    tuned): the headline leg runs decode steps of one token each over the
    full Qwen-shaped head (successive rows of xb) until at least min_sec of
    CPU work (at most max_tokens steps).  With legs, two bounded samples
    more: one decode token over the full Gemma-shaped head (logits), and the
    prefill / CE workload's first 256 tokens over the Qwen-shaped head (logits
    then CE), each timed around the oracle call alone."""
    from oracle import head as ohead
    n = 0
    t = time.perf_counter()
    while n < min(max_tokens, xb.shape[0]):
        ohead.logits(h, xb[n:n + 1])
        n += 1
        if time.perf_counter() - t >= min_sec:
            break
    sec = time.perf_counter() - t
    out = {"value": n * pbytes / sec / 1e9, "unit": "GB/s", "cores": _oracle_threads(),
           "kind": "oracle",
           "sample": f"fp64 numpy oracle, full Qwen-shaped head, {n} decode steps of 1 token: "
                     f"{sec:.2f} s ({n / sec:.3f} tok/s)"}
    if not legs:
        return out
    from oracle.bytes import head_bytes
    from synth import make_head, make_targets, make_x
    hg = make_head("gemma")
    xg = make_x("gemma", 1)
    t = time.perf_counter()
    ohead.logits(hg, xg)
    sg = time.perf_counter() - t
    out["gemma_decode_m1"] = {"sec": round(sg, 3), "tok_s": round(1 / sg, 4),
                              "gbs_packed": round(head_bytes(hg) / sg / 1e9, 4),
                              "sample": "1 token, full Gemma-shaped head (V=262144, d=2560), logits"}
    del hg
    Mc = 256
    xp = make_x("qwen_prefill", Mc)
    yp = make_targets("qwen_prefill", Mc)
    t = time.perf_counter()
    ce = ohead.cross_entropy(ohead.logits(h, xp), yp)
    sp = time.perf_counter() - t
    out["qwen_prefill_ce"] = {"sec": round(sp, 3), "tok_s": round(Mc / sp, 2),
                              "mean_ce_sample": round(float(ce.mean()), 6),
                              "sample": f"first {Mc} of the 4096 prefill tokens, full Qwen-shaped "
                                        "head, logits then CE"}
    return out


def profile_run(kind, steps):
    """The bench's work without timing markers, for rocprofv3: clock warm-up
    (decode steps), a few warm-up calls, then `steps` calls back to back;
    trace summaries take the last `steps` dispatches of the kernel."""
    import torch
    from synth import CONFIGS, make_head, make_targets, make_x
    h = make_head("qwen_decode")
    heads = upload_copies(h, N_COPIES)
    x1 = torch.from_numpy(make_x("qwen_decode", 1).view(np.int16)).view(torch.bfloat16).cuda()
    if kind == "topk":
        clock_warmup(heads, x1, 0.5)
        wss = [hd.workspace(1, 3, x1.device) for hd in heads]
        vals = torch.empty((1, 10), dtype=torch.float32, device="cuda")
        idx = torch.empty((1, 10), dtype=torch.int64, device="cuda")
        for i in range(5 + steps):
            k = i % len(heads)
            heads[k].logits_topk(x1, 10, vals=vals, idx=idx, ws=wss[k])
    elif kind == "decode":
        src = torch.empty(CALIBRATION_BYTES, dtype=torch.uint8, device="cuda").fill_(3)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        clock_warmup(heads, x1, 0.5)
        outs = [torch.empty((1, h.V), device="cuda") for _ in heads]
        wss = [hd.workspace(1, 0, x1.device) for hd in heads]
        for i in range(5 + steps):
            k = i % len(heads)
            heads[k].logits(x1, out=outs[k], ws=wss[k])
    else:
        Mp = CONFIGS["qwen_prefill"]["Ms"][0]
        x = torch.from_numpy(make_x("qwen_prefill", Mp).view(np.int16)).view(
            torch.bfloat16).cuda()
        y = torch.from_numpy(make_targets("qwen_prefill", Mp)).cuda()
        for hd in heads:
            hd.prepare()
        clock_warmup(heads, x1, 0.5)
        ws = [hd.workspace(Mp, 1, x.device) for hd in heads]
        for i in range(3 + steps):
            k = i % len(heads)
            heads[k].logits_ce(x, y, ws=ws[k])
    torch.cuda.synchronize()
    print(f"profile run {kind}: done", flush=True)


def trace_summary(csv_path, last, match=""):
    """Per-kernel durations from a rocprofv3 kernel-trace CSV over each
    kernel's last `last` dispatches (after the profile run's warm-up): count,
    mean, median, p10, p90 in us.  Prints one JSON line per kernel whose name
    contains `match`."""
    import csv
    per = {}
    with open(csv_path) as f:
        for r in csv.DictReader(f):
            name = r.get("Kernel_Name") or r.get("KernelName") or ""
            if match not in name:
                continue
            per.setdefault(name, []).append((int(r["Start_Timestamp"]), int(r["End_Timestamp"])))
    for name, ts in per.items():
        ts.sort()
        d = np.array([(e - b) / 1e3 for b, e in ts[-last:]])
        print(json.dumps({"kernel": name, "dispatches": len(ts), "summarised": int(d.size),
                          "mean_us": round(float(d.mean()), 2),
                          "median_us": round(float(np.median(d)), 2),
                          "p10_us": round(_pct(d, 10), 2), "p90_us": round(_pct(d, 90), 2)}))


def sweep(steps, cfg="sweep128k", Ms=None, paths=("auto", "dec", "mid", "gemv", "tiled")):
    """A head (default the 128k-vocabulary one: V=128256, d=8192, r_c=128,
    r_r=64) at every M of a list (default its workload's) through each
    kernel: step time, GB/s over the packed bytes and MFMA utilisation
    (algorithmic flops over the bf16 peak).  One JSON line per (M, kernel);
    "auto" is the library's own choice.  The heads keep the many-token
    kernel's head-derived tables across calls (archead_prepare)."""
    import torch
    from synth import CONFIGS, make_head, make_x
    h = make_head(cfg)
    heads = upload_copies(h, 3)
    pbytes = lib_packed_bytes(heads[0])
    if pbytes > 400e6:
        heads.pop().close()    # two copies already exceed the 256 MB Infinity Cache
    for hd in heads:
        hd.prepare()
    Ms = Ms or CONFIGS[cfg]["Ms"]
    xb = make_x(cfg, max(Ms))
    x_all = torch.from_numpy(xb.view(np.int16)).view(torch.bfloat16).cuda()
    clock_warmup(heads, x_all[:1], 0.5)
    for M in Ms:
        for path in paths:
            if path == "gemv" and M > 64:
                continue          # 4 tokens per pass: far off the crossover
            for hd in heads:
                hd.force_path(path)
            n = steps if M <= 64 else max(10, steps // 4)
            ms, kern, _ = time_decode(heads, x_all[:M], n, 3)
            flops = mfma_algorithmic_flops(h, M)
            print(json.dumps({"sweep": cfg, "M": M, "kernel": path,
                              "us_per_step": round(ms * 1e3, 2),
                              "gbs_packed": round(pbytes / ms / 1e6, 1),
                              "mfma_util": round(flops / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
                              "tok_s": round(M / ms * 1e3, 1)}), flush=True)
    for hd in heads:
        hd.force_path("auto")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--clock-warmup", type=float, default=0.5,
                    help="seconds of untimed decode steps before any timing (GPU clock ramp)")
    ap.add_argument("--prefill-steps", type=int, default=10)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-prefill", action="store_true")
    ap.add_argument("--no-u8", action="store_true",
                    help="skip the decode line of the head with 8-bit residual scale codes")
    ap.add_argument("--no-paper-storage", action="store_true",
                    help="skip the lines of the head in the paper's own storage (5-bit U_c, "
                         "r_c=10, r_r=6, g=64, 8-bit scale codes)")
    ap.add_argument("--no-dense", action="store_true",
                    help="skip the dense bf16 head context line")
    ap.add_argument("--profile", choices=["decode", "prefill", "topk"])
    ap.add_argument("--sweep", action="store_true",
                    help="M sweep of a head (default the 128k-vocabulary one) through each kernel")
    ap.add_argument("--sweep-cfg", default="sweep128k",
                    help="head of the sweep: sweep128k, qwen_decode or gemma")
    ap.add_argument("--sweep-ms", default="",
                    help="comma-separated M values of the sweep (default: the head's workload)")
    ap.add_argument("--sweep-paths", default="auto,dec,mid,gemv,tiled")
    ap.add_argument("--trace-summary", metavar="CSV",
                    help="summarise a rocprofv3 kernel-trace CSV (no GPU needed): the last "
                         "--trace-last dispatches of each kernel whose name contains --trace-match")
    ap.add_argument("--trace-last", type=int, default=200)
    ap.add_argument("--trace-match", default="")
    args = ap.parse_args()
    if args.trace_summary:
        trace_summary(args.trace_summary, args.trace_last, args.trace_match)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: runs on one GPU only; multi-GPU (vocab-parallel) "
              "runs are not implemented", file=sys.stderr)
        sys.exit(2)

    import torch
    from synth import CONFIGS, make_head, make_targets, make_x

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.profile:
        profile_run(args.profile, args.prefill_steps if args.profile == "prefill" else args.steps)
        return
    if args.sweep:
        sweep(min(args.steps, 40), args.sweep_cfg,
              [int(v) for v in args.sweep_ms.split(",") if v] or None,
              tuple(args.sweep_paths.split(",")))
        return
    cfg = "qwen_decode"
    log("generating the packed head ...")
    h = make_head(cfg)
    heads = upload_copies(h, N_COPIES)
    # the tiled kernel's head-derived tables, built once per head as a server
    # would at load time (used from M = 33 on: the decode M = 64 line)
    for hd in heads:
        hd.prepare()
    pbytes = lib_packed_bytes(heads[0])
    xb = make_x(cfg, 64)
    x_all = torch.from_numpy(xb.view(np.int16)).view(torch.bfloat16).cuda()

    n_clock = clock_warmup(heads, x_all[:1], args.clock_warmup)
    log(f"clock warm-up: {n_clock} untimed decode steps in {args.clock_warmup} s")
    res = {}
    pcts = None
    for M in (1, 4, 16, 32, 64):
        x = x_all[:M]
        if M == 1:
            with ClockSampler() as clk:
                ms, kern_ms, kern_med, pcts = time_decode(heads, x, args.steps, args.warmup,
                                                          percentiles=True)
        else:
            ms, kern_ms, kern_med = time_decode(heads, x, max(20, args.steps // 4), args.warmup)
        res[M] = (ms, kern_ms, kern_med)
        log(f"decode M={M}: {ms * 1e3:.1f} us/step, head kernel {kern_ms * 1e3:.1f} us "
            f"(median {kern_med * 1e3:.1f}), {pbytes / ms / 1e6:.0f} GB/s over packed bytes")

    # the same head with 8-bit residual scale codes (fp16 row scale): fewer
    # packed bytes per decode step
    u8 = None
    if not args.no_u8:
        h8 = make_head(cfg, scales="u8")
        heads8 = upload_copies(h8, N_COPIES)
        b8 = lib_packed_bytes(heads8[0])
        torch.cuda.synchronize()
        clock_warmup(heads8, x_all[:1], 0.2)
        ms8, _, k8 = time_decode(heads8, x_all[:1], args.steps, args.warmup)
        u8 = {"us_per_step": round(ms8 * 1e3, 2), "kernel_us_median": round(k8 * 1e3, 2),
              "packed_bytes": b8, "gbs_packed": round(b8 / ms8 / 1e6, 1)}
        log(f"decode M=1, 8-bit scale codes: {ms8 * 1e3:.1f} us/step, {b8 / 1e6:.1f} MB packed, "
            f"{b8 / ms8 / 1e6:.0f} GB/s")
        for hd in heads8:
            hd.close()
        del heads8
        torch.cuda.empty_cache()

    # the paper's own Qwen3-8B storage: r_c = 10 with 5-bit core-left words,
    # r_r = 6, residual groups of 64 with 8-bit scale codes
    paper = None
    if not args.no_paper_storage:
        hp = make_head(cfg, g=64, rc=10, rr=6, core_u="i5", scales="u8")
        headsp = upload_copies(hp, N_COPIES)
        bp = lib_packed_bytes(headsp[0])
        clock_warmup(headsp, x_all[:1], 0.2)
        msp, _, kp = time_decode(headsp, x_all[:1], args.steps, args.warmup)
        paper = {"config": "V=151936 d=4096 g=64 r_c=10 (5-bit ARCHEAD_I5) r_r=6, 8-bit scale codes",
                 "packed_bytes": bp, "packed_mib": round(bp / 2 ** 20, 2),
                 "decode_m1": {"us_per_step": round(msp * 1e3, 2), "kernel_us_median": round(kp * 1e3, 2),
                               "gbs_packed": round(bp / msp / 1e6, 1)}}
        log(f"paper storage head: {bp / 2 ** 20:.2f} MiB, decode M=1 {msp * 1e3:.1f} us/step, "
            f"{bp / msp / 1e6:.0f} GB/s")
        if not args.no_prefill:
            Mp = CONFIGS["qwen_prefill"]["Ms"][0]
            xpp = torch.from_numpy(make_x("qwen_prefill", Mp).view(np.int16)).view(
                torch.bfloat16).cuda()
            ypp = torch.from_numpy(make_targets("qwen_prefill", Mp)).cuda()
            ms_pp, ce_pp, k_pp = time_prefill(headsp, xpp, ypp, args.prefill_steps, 3)
            paper["prefill_m4096"] = {"ms_per_step": round(ms_pp, 4),
                                      "tok_s": round(Mp / ms_pp * 1e3, 1), "mean_ce": ce_pp,
                                      "kernel_ms_median": round(k_pp, 4)}
            log(f"paper storage head: prefill CE M={Mp} {ms_pp:.3f} ms/step")
            del xpp, ypp
        for hd in headsp:
            hd.close()
        del headsp
        torch.cuda.empty_cache()

    # greedy decoding: the fused argmax step (no [M, V] logits written)
    greedy = {}
    for M in (1, 16):
        gms = time_argmax(heads, x_all[:M], max(20, args.steps // 2), args.warmup)
        greedy[str(M)] = {"us_per_step": round(gms * 1e3, 2),
                          "gbs_packed": round(pbytes / gms / 1e6, 1)}
        log(f"greedy (fused argmax) M={M}: {gms * 1e3:.1f} us/step")
    # top-k selection (k = 10: the paper's largest top-k agreement; fused
    # into the head pass at M = 1, over the logits in the workspace above)
    topk = {}
    for M in (1, 16):
        tms = time_topk(heads, x_all[:M], 10, max(20, args.steps // 2), args.warmup)
        topk[str(M)] = {"k": 10, "us_per_step": round(tms * 1e3, 2),
                        "fused": M == 1}
        log(f"top-10 selection M={M}: {tms * 1e3:.1f} us/step")

    # context: the same decode step through a dense bf16 head of the same
    # shape (torch linear, random weights), the bytes the packed head avoids
    dense = None
    if not args.no_dense:
        import torch.nn.functional as F
        w = [torch.randn((h.V, h.d), device="cuda", dtype=torch.bfloat16) for _ in range(2)]
        x1 = x_all[:1]

        def dstep(i):
            F.linear(x1, w[i % 2])
        for i in range(50):
            dstep(i)
        dms = _timed_loop(dstep, args.steps)
        dbytes = h.V * h.d * 2
        dense = {"us_per_step": round(dms * 1e3, 2), "gbs": round(dbytes / dms / 1e6, 1),
                 "bytes": dbytes, "op": "torch.nn.functional.linear, bf16 [V, d] weight, M=1",
                 "packed_speedup": round(dms / ms1_for_dense(res), 2)}
        log(f"dense bf16 head M=1: {dms * 1e3:.1f} us/step ({dbytes / dms / 1e6:.0f} GB/s over "
            f"{dbytes / 1e9:.2f} GB)")
        del w
        torch.cuda.empty_cache()

    prefill = None
    if not args.no_prefill:
        pc = CONFIGS["qwen_prefill"]
        Mp = pc["Ms"][0]
        xp = torch.from_numpy(make_x("qwen_prefill", Mp).view(np.int16)).view(
            torch.bfloat16).cuda()
        yp = torch.from_numpy(make_targets("qwen_prefill", Mp)).cuda()
        ms_u, _, kern_u = time_prefill(heads, xp, yp, args.prefill_steps, 3, prepared=False)
        ms_p, mean_ce, kern_p = time_prefill(heads, xp, yp, args.prefill_steps, 3)
        flops = mfma_algorithmic_flops(h, Mp)
        tflops = flops / (kern_p * 1e-3) / 1e12
        prefill = {"M": Mp, "ms_per_step": round(ms_p, 4), "tok_s": round(Mp / ms_p * 1e3, 1),
                   "mean_ce": mean_ce,
                   "mfma_kernel": {"kernel": "k_mfma<true, 256, 8, 0>",
                                   "kernel_ms_median": round(kern_p, 4),
                                   "algorithmic_flops": flops,
                                   "achieved_tflops": round(tflops, 1),
                                   "peak_tflops": PEAK_BF16_TFLOPS,
                                   "frac": round(tflops / PEAK_BF16_TFLOPS, 4)},
                   "head_tables": "prepared once (archead_prepare)",
                   "prepared_bytes": heads[0].prepared_bytes(),
                   "packed_plus_prepared_bytes": pbytes + heads[0].prepared_bytes(),
                   "per_call_tables": {"ms_per_step": round(ms_u, 4),
                                       "tok_s": round(Mp / ms_u * 1e3, 1),
                                       "kernel_ms_median": round(kern_u, 4)}}
        log(f"prefill CE M={Mp}, head tables rebuilt per call: {ms_u:.3f} ms/step, "
            f"{Mp / ms_u * 1e3:.0f} tok/s")
        log(f"prefill CE M={Mp}: {ms_p:.3f} ms/step, {Mp / ms_p * 1e3:.0f} tok/s; "
            f"many-token kernel {kern_p:.3f} ms = {tflops:.0f} TFLOP/s "
            f"({100 * tflops / PEAK_BF16_TFLOPS:.1f}% of bf16 peak)")
        if not args.no_dense:
            # context: the logits of the same tokens through a dense bf16 head
            # of the same shape (hipBLASLt through torch, random weights; the
            # [M, V] logits are written, no softmax)
            import torch.nn.functional as F
            w = torch.randn((h.V, h.d), device="cuda", dtype=torch.bfloat16)
            for _ in range(2):
                F.linear(xp, w)
            dms = _timed_loop(lambda i: F.linear(xp, w), max(3, args.prefill_steps // 2))
            dfl = 2 * Mp * h.V * h.d
            prefill["dense_bf16_linear"] = {
                "ms_per_step": round(dms, 4), "tflops": round(dfl / dms / 1e9, 1),
                "frac": round(dfl / dms / 1e9 / PEAK_BF16_TFLOPS, 4),
                "op": "torch.nn.functional.linear, bf16 [M, d] x [V, d]^T, M=4096"}
            log(f"dense bf16 linear M={Mp}: {dms:.3f} ms/step = {dfl / dms / 1e9:.0f} TFLOP/s")
            # the fidelity metrics against that dense head inside the packed
            # head's tile pass (archead_logit_fidelity_head: fidelity pass,
            # merge, rank pass; no [M, V] array)
            hd0 = heads[0]
            wsf = hd0.workspace(Mp, 4, xp.device)
            for _ in range(2):
                hd0.logit_fidelity_head(xp, w, ws=wsf)
            fms = _timed_loop(lambda i: hd0.logit_fidelity_head(xp, w, ws=wsf),
                              max(3, args.prefill_steps // 2))
            kl, sqe, ridx, rk = hd0.logit_fidelity_head(xp, w, ws=wsf)
            prefill["fidelity_head"] = {
                "ms_per_step": round(fms, 4), "tok_s": round(Mp / fms * 1e3, 1),
                "mean_kl_random_dense": float(kl.mean()),
                "op": "archead_logit_fidelity_head vs the random dense bf16 head above, M=4096"}
            log(f"fidelity vs a dense head in the tile pass M={Mp}: {fms:.3f} ms/step, "
                f"{Mp / fms * 1e3:.0f} tok/s")
            del w, wsf
            torch.cuda.empty_cache()

    copy = copy_bandwidth()
    log(f"device copy: {copy['gbs_read_plus_write']} GB/s (read + write)")
    ms1, _, kern1 = res[1]
    value = pbytes / ms1 / 1e6          # GB/s
    alg = decode_algorithmic_bytes(pbytes, h, 1)
    kname = f"k_gemv<1, {lanes_per_row(h)}, false, false, 0, false>"
    # a decode step at M = 1 is one launch of the head kernel, so the HIP
    # events around the unmarked timed loop (on the stream the kernel is
    # launched on) give its average launch duration, launch gaps included;
    # events attached to every dispatch (the separate marked pass) slow the
    # kernel on some boxes and are reported beside it only
    achieved = alg / ms1 / 1e6
    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms1, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "qwen3-8b-shaped packed head decode, M=1",
                   "V": h.V, "d": h.d, "g": h.g, "r_c": h.rc, "r_r": h.rr,
                   "packed_bytes": pbytes, "head_copies_rotated": N_COPIES,
                   "parallelism": "none (1 GPU)"},
        "pct_peak_hbm": round(100 * value / PEAK_HBM_GBS, 2),
        "clock_warmup_s": args.clock_warmup,
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4),
                     "traffic": measured_traffic(), "kernel": kname,
                     "kernel_us_mean": round(ms1 * 1e3, 2), "algorithmic_bytes": alg,
                     "timing": f"HIP events on the launch stream around the timed loop of "
                               f"{args.steps} steps, one launch of the kernel per step "
                               f"(per-launch average, launch gaps included)",
                     "marked_pass_kernel_us_median": round(kern1 * 1e3, 2)},
        "step_us_percentiles": {k: round(v * 1e3, 2) for k, v in pcts.items()},
        "gpu_clock": clk.summary(),
        "hbm_copy": copy,
        "decode": {str(M): {"us_per_step": round(v[0] * 1e3, 2),
                            "kernel_us_median": round(v[2] * 1e3, 2),
                            "gbs_packed": round(pbytes / v[0] / 1e6, 1)}
                   for M, v in res.items()},
        "greedy_argmax": greedy,
        "topk_selection": topk,
        "decode_u8_scales": u8,
        "paper_storage_head": paper,
        "prefill": prefill,
        "dense_bf16_head": dense,
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle (1 token, full head) ...")
        out["cpu_baseline"] = cpu_baseline(h, pbytes, xb)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
