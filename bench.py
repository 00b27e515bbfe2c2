#!/usr/bin/env python3
"""Throughput of the ERASE detached-block training step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload ctr_mlp]

One "step" is one call of erase_step(): for each of the 6 detached CTR
subarchitectures (1677->512->256->128, local Linear(128->1) sigmoid-BCE head,
batch 4096, bf16 operands with fp32 accumulation) the forward, local loss,
weight/input gradients and Adam update.  Inputs are synthetic, seeded and
already resident in HBM (8 batches, cycled).

The headline value is samples/s of one ERASE schedule declared before the
run (--headline, default PIPELINE+worker: the ERASE order without the
end-of-step join, the backward streams' work enqueued by the library's worker
thread).  Every other schedule is reported beside it: OVERLAP, OVERLAP_GRAPH
(captured as a HIP graph), PIPELINE, OVERLAP+worker, and the same kernels in
the serial order (SERIAL, SERIAL_GRAPH); the speedups compare schedules with
identical kernels.  Per-step intervals (for the p90, the paper's statistic)
run from one step's start to the next step's start on the forward stream.
Per-kernel durations for the roofline and the backward/forward overlap come
from HIP events recorded by the library around each launch, on the stream of
that launch; the overlap is also derived from rocprofv3 kernel traces of each
ERASE schedule (--analyze-trace).  The CPU baseline times the float64 oracle
on the host on a bounded sample.  The CTR-DCNv2 workload (batch 16384) and
the small transformer are measured too.

A second measurement reproduces the paper's comparison of ERASE with
conventional backpropagation (one backward of the summed block losses at the
end of the step, gradients crossing every cut) on the 12-block chain, where
detachment removes the cross-cut input gradients; on the shared-input CTR
workload the two coincide.
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

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3     # MI355X fp32 vector/MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
METRIC = "train samples/s, 6-block CTR @1 MI355X; ERASE vs serial speedup; MFMA util %"
KIND_SYMBOL = {"prologue": "erase_prologue", "fwd_gemm": "erase_fwd_gemm", "head_bce": "erase_head_bce",
               "wgrad_gemm": "erase_wgrad_gemm", "dgrad_gemm": "erase_dgrad_gemm", "adam": "erase_adam",
               "bwd_gemm": "erase_bwd_gemm", "fwd_head_gemm": "erase_fwd_head_gemm", "fwd_gemm_kg2": "erase_fwd_gemm_kg2",
               "wgrad_gemm_kg2": "erase_wgrad_gemm_kg2", "wgrad_adam_kg2": "erase_wgrad_adam_kg2"}


def kernel_class(r, bf16=True):
    t = "bf16" if bf16 else "f32"
    if r["kind"] == "fwd_head_gemm" and bf16 and r["tile_m"] == 16:
        return "erase_fwd_head16"  # the bf16 16-row last layer + head kernel
    if r["kind"] in ("wgrad_adam_kg2", "wgrad_gemm_kg2") and bf16:
        # the bf16 first-layer weight gradient with its Adam update: four
        # waves per 64x64 tile, direct-to-LDS slices (one kernel for both)
        return "erase_wgrad_adam_w4"
    if r["tile_m"]:
        return f"{KIND_SYMBOL[r['kind']]}<{t},{r['tile_m']},{r['tile_n']}>"
    return f"{KIND_SYMBOL[r['kind']]}<{t}>"


TF_SOURCES = ("csrc/transformer.hip", "csrc/tf_api.cpp")


def kernel_source_hash(extra=()):
    """Hash of the kernel sources and build flags: counters taken from other
    sources are stale.  The transformer's figures also hash its own kernels
    and launch plan (`extra`)."""
    h = hashlib.sha256()
    for f in ("csrc/kernels.hip", "csrc/embed.hip", "csrc/internal.h", "build.py") + tuple(extra):
        with open(os.path.join(ROOT, "paper_2608_18469_amd", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "ctr_mlp_hbm_traffic.md")
MFMA_FILE = os.path.join(ROOT, "profiles", "mfma_busy_counters.md")


def mfma_kind(kind):
    """Kernel kinds whose launches run MFMA work (the GEMMs, and the first
    layer's weight gradient with the block's Adam in the same launch)."""
    return "gemm" in kind or kind == "wgrad_adam_kg2"


def roofline_of(flops, nbytes, dur_s, peak_mfma):
    """Roofline of one launch: the bound is the resource with the larger
    minimum time (flops at the MFMA peak against bytes at the HBM peak)."""
    t_mfma = flops / (peak_mfma * 1e12)
    t_hbm = nbytes / (PEAK_HBM_GBS * 1e9)
    if flops and t_mfma >= t_hbm:
        r = {"bound": "mfma", "achieved": flops / dur_s / 1e12, "peak": peak_mfma, "unit": "TFLOP/s"}
    else:
        r = {"bound": "hbm", "achieved": nbytes / dur_s / 1e9, "peak": PEAK_HBM_GBS, "unit": "GB/s"}
    r["frac"] = r["achieved"] / r["peak"]
    return r


def measured_mfma_busy(workload):
    """Counter-based MFMA utilisation over every MFMA launch of `workload`,
    from the committed summary of a rocprofv3 pass with
    SQ_VALU_MFMA_BUSY_CYCLES and GRBM_GUI_ACTIVE: busy SIMD cycles over
    (active cycles per XCD x 1024 SIMDs).  None when there is no summary or
    the kernels changed since it was taken."""
    try:
        with open(MFMA_FILE) as f:
            lines = f.read().splitlines()
    except OSError:
        return None
    src = kernel_source_hash(TF_SOURCES if workload.startswith("tf_") else ())
    for line in lines:
        parts = line.split()
        if len(parts) == 6 and parts[0] == "mfma_busy" and parts[1] == workload:
            if parts[2] != src:
                return None
            busy, simd_cycles, n = float(parts[3]), float(parts[4]), int(parts[5])
            return {"util": busy / simd_cycles, "busy_simd_cycles": busy, "active_simd_cycles": simd_cycles,
                    "dispatches": n, "source": src}
    return None


def measured_traffic(kernel_class, workload):
    """HBM bytes per launch of `kernel_class` from the committed byte-counter
    summary (rocprofv3 FETCH_SIZE and WRITE_SIZE passes, each scaled by the
    same counter's reading for a copy of known size), or None when there is
    no summary for this kernel and workload or the kernels changed since."""
    try:
        with open(TRAFFIC_FILE) as f:
            lines = f.read().splitlines()
    except OSError:
        return None
    src = kernel_source_hash()
    for line in lines:
        parts = line.split()
        if len(parts) == 6 and parts[0] == "traffic" and parts[1] == workload and parts[2] == kernel_class:
            if parts[3] != src:
                return None
            fetch, write = float(parts[4]), float(parts[5])
            return {"bytes": fetch + write, "fetch_bytes": fetch, "write_bytes": write, "source": src}
    return None


def overlap_fraction(recs):
    """Share of backward-stream kernel time (every backward stream) that runs
    while a forward-stream kernel is running (interval intersection on the
    device clock)."""
    fwd = sorted((r["start_ms"], r["end_ms"]) for r in recs if r["stream"] == 0)
    merged = []
    for a, b in fwd:
        if merged and a <= merged[-1][1]:
            merged[-1][1] = max(merged[-1][1], b)
        else:
            merged.append([a, b])
    tot = inter = 0.0
    for r in recs:
        if r["stream"] < 1:
            continue
        a, b = r["start_ms"], r["end_ms"]
        tot += b - a
        for c, d in merged:
            lo, hi = max(a, c), min(b, d)
            if hi > lo:
                inter += hi - lo
    return inter / tot if tot > 0 else 0.0


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_rate(cfg, params, batches, budget_s):
    """Full float64 oracle steps until budget_s has passed (at least one)."""
    import oracle
    from paper_2608_18469_amd import synth
    m = synth.zero_state(params)
    v = synth.zero_state(params)
    p, t = params, 0
    steps = 0
    t0 = time.perf_counter()
    while True:
        x, y = batches[steps % len(batches)]
        r = oracle.step(cfg, p, m, v, t, x, y)
        p, m, v, t = r["params"], r["m"], r["v"], r["t"]
        steps += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            return steps, el


def cpu_baseline(cfg, params, batches, budget_s, budget_1t_s):
    """Time the float64 oracle on the host (a reported baseline, not a
    target): with every BLAS thread, then with one thread."""
    from threadpoolctl import threadpool_info, threadpool_limits
    info = threadpool_info()
    threads = max([i.get("num_threads", 1) for i in info] or [1])
    blas = ", ".join(sorted({f"{i.get('internal_api', '?')} {i.get('version', '')}".strip() for i in info})) or "none"
    steps, el = _oracle_rate(cfg, params, batches, budget_s)
    with threadpool_limits(limits=1):
        steps1, el1 = _oracle_rate(cfg, params, batches, budget_1t_s)
    what = f"full float64 oracle steps of {cfg['name']} (batch {cfg['batch']}, {len(cfg['blocks'])} blocks)"
    return {"value": steps * cfg["batch"] / el, "unit": "samples/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{steps} {what} in {el:.1f} s on the host, {threads} BLAS threads",
            "single_thread": {"value": steps1 * cfg["batch"] / el1, "unit": "samples/s", "cores": 1,
                              "sample": f"{steps1} {what} in {el1:.1f} s, 1 BLAS thread"},
            "cpu_model": _cpu_model(), "blas": blas, "os_cpu_count": os.cpu_count()}


def tf_cpu_baseline(cfg, params, toks, budget_s):
    """The float64 transformer oracle on the host, on a bounded sample: whole
    steps of one layer (block 1, with the embedding) on one sequence of the
    full length; tokens/s of the 8-layer model = sample tokens / (time per
    one-layer step x layers)."""
    from threadpoolctl import threadpool_info
    from oracle import transformer_oracle
    from paper_2608_18469_amd import synth_tf
    info = threadpool_info()
    threads = max([i.get("num_threads", 1) for i in info] or [1])
    one = dict(cfg, batch=1, layers=1)
    p = [params[0]]
    m = synth_tf.zero_state(p)
    steps, t0 = 0, time.perf_counter()
    while True:
        r = transformer_oracle.tf_step(one, p, m, m, steps, toks[0][:1])
        steps += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    per = el / steps
    return {"value": cfg["seq"] / (per * cfg["layers"]), "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{steps} float64 oracle steps of one layer (with the embedding and its 32768-way head) on one "
                      f"sequence of {cfg['seq']} tokens in {el:.1f} s, {threads} BLAS threads; scaled to "
                      f"{cfg['layers']} layers",
            "cpu_model": _cpu_model()}


def time_schedules(tr, dev, scheds, steps, warmup, block, losses, M, log):
    """Warm every schedule up (graph capture and instantiation happen here),
    then time them interleaved in blocks of `block` steps so that clock and
    thermal drift affect every schedule alike.  One global step counter picks
    the batch, so every (batch, step parity) pair a graph schedule meets is
    one it has already captured.  Returns per-schedule throughput, the p90 and
    median of per-step samples/s (HIP events on the forward stream) and the
    host enqueue time, plus the step function for later passes.  Per-step
    intervals run from one step's start to the next step's start on the
    forward stream."""
    import torch
    gstep = 0
    mode = ["caller"]

    def one_step(s):
        # "<schedule>+worker": the library's worker thread enqueues the
        # backward streams' work (non-blocking dispatch)
        nonlocal gstep
        base, _, disp = s.partition("+")
        disp = disp or "caller"
        if disp != mode[0]:
            tr.set_dispatch(disp)
            mode[0] = disp
        x, y = dev[gstep % len(dev)]
        gstep += 1
        tr.step(x, y, base, losses, wait_current=False)

    for s in scheds:
        log(f"[bench] {s}: warmup {warmup}")
        for _ in range(warmup):
            one_step(s)
        tr.sync()
    acc = {s: {"el": 0.0, "per": [], "host": []} for s in scheds}
    nblk = (steps + block - 1) // block
    for bi in range(nblk):
        n = min(block, steps - bi * block)
        for s in scheds:
            # an event on the forward stream at the start of every step; a
            # step's interval is the time from its start to the next step's
            # start (steady state: it covers the step's whole work, also the
            # trailing backward of a PIPELINE step, which the next step's
            # forwards wait for); the last step of a block has no successor
            evs = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for i in range(n):
                evs[i].record(tr.sf)
                h0 = time.perf_counter()
                one_step(s)
                acc[s]["host"].append(time.perf_counter() - h0)
            tr.sync()  # waits for the worker's enqueues too, then for every stream
            torch.cuda.synchronize()
            acc[s]["el"] += time.perf_counter() - t0
            acc[s]["per"] += [evs[i].elapsed_time(evs[i + 1]) for i in range(n - 1)]  # ms, device clock
        log(f"[bench] block {bi + 1}/{nblk} ({n} steps per schedule) done")
    res = {}
    for s in scheds:
        el = acc[s]["el"]
        sps = M / (np.array(acc[s]["per"]) / 1e3)
        res[s] = {"samples_per_s": M * steps / el, "ms_per_step": el / steps * 1e3,
                  "p90_samples_per_s": float(np.percentile(sps, 90)), "median_samples_per_s": float(np.median(sps)),
                  "host_enqueue_us": float(np.median(acc[s]["host"]) * 1e6), "elapsed_s": el}
        log(f"[bench] {s}: {res[s]['samples_per_s']:.0f} samples/s, {res[s]['ms_per_step']:.3f} ms/step, "
            f"p90 {res[s]['p90_samples_per_s']:.0f}, enqueue {res[s]['host_enqueue_us']:.1f} us")
    return res, one_step


def timed_records(tr, one_step, sched, n):
    """Per-launch records (HIP events stamped at each kernel's own start and
    end) of n steps of one schedule."""
    tr.set_timing(True)
    out = []
    for _ in range(n):
        one_step(sched)
        tr.sync()
        out.append(tr.read_timing())
    tr.set_timing(False)
    return out


BWD_KINDS = ("wgrad_gemm", "wgrad_gemm_kg2", "wgrad_adam_kg2", "dgrad_gemm", "bwd_gemm", "adam")


def conventional_comparison(args, log):
    """ERASE against conventional backpropagation on the 12-block chain: the
    paper's comparison (one backward of the aggregate objective at the end of
    the step, gradients crossing every cut) beside the detached step run
    serially and the ERASE schedules.  On shared-input workloads nothing
    crosses a cut, so the conventional step is the serial one; the chain is
    where detachment changes the backward work."""
    import torch

    from paper_2608_18469_amd import erase, synth
    cfg = synth.config("deep_chain")
    M = cfg["batch"]
    params, batches = synth.make_workload(cfg, 0, 8)
    tr = erase.Trainer(cfg, params, keep_grads=True, bwd_streams=args.bwd_streams,
                       x_in_place=not args.x_copy and M % 128 == 0)
    dev = [tr.device_batch(x, y) for (x, y) in batches]
    losses = torch.zeros(len(cfg["blocks"]), device="cuda")
    scheds = ["undetached", "undetached_graph", "serial", "serial_graph", "overlap", "overlap_graph", "pipeline",
              "overlap+worker", "pipeline+worker"]
    log(f"[bench] conventional vs ERASE on deep_chain (batch {M}, {len(cfg['blocks'])} chained blocks)")
    res, one_step = time_schedules(tr, dev, scheds, args.steps, args.warmup, args.block, losses, M, log)
    bwd = {}
    tr.set_dispatch("caller")
    for s in ("undetached", "serial"):
        recs = [r[1:] for r in timed_records(tr, one_step, s, args.timing_steps)]
        bwd[s] = float(np.mean([sum(r["end_ms"] - r["start_ms"] for r in rs if r["kind"] in BWD_KINDS)
                                for rs in recs])) * 1e3
    tr.close()
    # the ERASE side is the declared headline schedule; the conventional side
    # takes the faster of its two schedules (the stronger baseline)
    best = args.headline if args.headline in res else "pipeline+worker"
    conv = max(("undetached", "undetached_graph"), key=lambda k: res[k]["samples_per_s"])
    det = max(("serial", "serial_graph"), key=lambda k: res[k]["samples_per_s"])
    return {
        "workload": f"deep_chain: {len(cfg['blocks'])} blocks chained through the stop-gradient, each "
                    f"256->256->256 + Linear(256->1) BCE head, batch {M}, bf16, Adam",
        "conventional": "the same network without the cuts, one backward of the sum of the block losses after the "
                        "last forward (gradients cross every cut); schedules 'undetached' (launched) and "
                        "'undetached_graph' (replayed HIP graph)",
        "schedules": res,
        "erase_schedule": best,
        "conventional_schedule": conv,
        "detached_serial_schedule": det,
        "erase_vs_conventional": res[best]["samples_per_s"] / res[conv]["samples_per_s"],
        "erase_vs_conventional_p90": res[best]["p90_samples_per_s"] / res[conv]["p90_samples_per_s"],
        "detached_serial_vs_conventional": res[det]["samples_per_s"] / res[conv]["samples_per_s"],
        "erase_vs_detached_serial": res[best]["samples_per_s"] / res[det]["samples_per_s"],
        "backward_kernel_us_per_step": {"conventional": bwd["undetached"], "detached": bwd["serial"],
                                        "reduction": 1.0 - bwd["serial"] / bwd["undetached"]},
    }


def input_stage(args, log, tr, cfg, head, labels, losses):
    """The CTR input stage on the device (erase_embed_bags: log1p dense
    features and 26 sum-pooled bags of the 100000 x 64 float32 tables) at the
    workload's batch: kernel time and algorithmic bytes per launch, and the
    headline schedule run from raw features (input stage then step, both
    enqueued on the forward stream)."""
    import torch

    from paper_2608_18469_amd import erase, synth
    M = cfg["batch"]
    rng = np.random.Generator(np.random.PCG64(1))
    tabs = synth.CtrTables(rng, rows=cfg.get("ctr_rows", synth.CTR_ROWS))
    raws = [synth.make_ctr_raw(tabs, M, rng) for _ in range(2)]
    tables = torch.from_numpy(np.stack(tabs.tables)).cuda()
    feats = [(torch.from_numpy(r["dense"].astype(np.float32)).cuda(), torch.from_numpy(r["offsets"]).cuda(),
              torch.from_numpy(r["indices"]).cuda()) for r in raws]
    xs = [torch.zeros((M, tr.ncfg.x_ld), dtype=tr.act_dtype, device="cuda") for _ in range(2)]
    status = torch.zeros(1, dtype=torch.int32, device="cuda")

    def emb(i):
        d, o, ix = feats[i % 2]
        erase.embed_bags(d, o, ix, tables, xs[i % 2], status, stream=tr.sf)

    for i in range(10):
        emb(i)
    torch.cuda.synchronize()
    n = 200
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(tr.sf)
    for i in range(n):
        emb(i)
    e1.record(tr.sf)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) / n * 1e3
    nnz = float(np.mean([r["indices"].size for r in raws]))
    T, dim, nd = synth.CTR_TABLES, synth.CTR_DIM, synth.CTR_DENSE
    esz = 2 if tr.act_dtype == torch.bfloat16 else 4
    nbytes = nnz * (dim * 4 + 4) + T * (M + 1) * 8 + M * nd * 4 + M * tr.ncfg.x_ld * esz
    # the headline schedule from raw features
    base, _, disp = head.partition("+")
    tr.set_dispatch(disp or "caller")
    for i in range(args.warmup):
        emb(i)
        tr.step(xs[i % 2], labels, base, losses, wait_current=False)
    tr.sync()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        emb(i)
        tr.step(xs[i % 2], labels, base, losses, wait_current=False)
    tr.sync()
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    tr.set_dispatch("caller")
    assert int(status.item()) == 0
    # its backward (table gradients from a gradient at x), for the same bags
    dx = torch.randn((M, tr.ncfg.x_ld), device="cuda").to(tr.act_dtype)
    d0, o0, ix0 = feats[0]
    tg = torch.empty((T, tabs.rows, dim), dtype=torch.float32, device="cuda")
    g_, scratch = erase.embed_bags_backward(o0, ix0, dx, nd, tabs.rows, dim, table_grad=tg, stream=tr.sf)
    torch.cuda.synchronize()
    e0.record(tr.sf)
    nb = 20
    for _ in range(nb):
        erase.embed_bags_backward(o0, ix0, dx, nd, tabs.rows, dim, table_grad=tg, stream=tr.sf)
    e1.record(tr.sf)
    torch.cuda.synchronize()
    us_b = e0.elapsed_time(e1) / nb * 1e3
    # algorithmic bytes: the offsets and ids read once, one dx row slice per
    # entry, and the dense table gradient written once (the bucketing's own
    # counters and lists are not counted)
    bytes_b = nnz * (4 + dim * esz) + T * (M + 1) * 8 + T * tabs.rows * dim * 4
    log(f"[bench] input stage: {us:.1f} us per batch, {nbytes / us / 1e3:.0f} GB/s algorithmic; "
        f"{head} from raw features {M * args.steps / el:.0f} samples/s; backward {us_b:.0f} us "
        f"({bytes_b / us_b / 1e3:.0f} GB/s algorithmic)")
    return {"kernel": "erase_embed_bags_k", "workload": f"{M} rows, {T} tables of {tabs.rows} x {dim} float32, "
                                                        f"bags of 1..20 Zipf(1.1) ids (mean nnz {nnz:.0f}), "
                                                        f"{nd} dense features, x in {tr.act_dtype}".replace("torch.", ""),
            "avg_launch_us": us, "algorithmic_bytes_per_launch": nbytes,
            "achieved_gbs": nbytes / us / 1e3, "peak_gbs": PEAK_HBM_GBS, "frac": nbytes / us / 1e3 / PEAK_HBM_GBS,
            "samples_per_s": M / (us * 1e-6),
            "step_from_raw_features": {"schedule": head, "samples_per_s": M * args.steps / el,
                                       "ms_per_step": el / args.steps * 1e3},
            "note": "bytes count every gathered table row once per use; Zipf-skewed ids hit the caches, so HBM "
                    "traffic is lower than the algorithmic bytes",
            "backward": {"entry": "erase_embed_bags_backward", "avg_us": us_b, "algorithmic_bytes": bytes_b,
                         "achieved_gbs": bytes_b / us_b / 1e3,
                         "note": "dense fp32 table gradient [26][100000][64] written in full (666 MB); eleven launches"}}


def _merge(iv):
    out = []
    for a, b in sorted(iv):
        if out and a <= out[-1][1]:
            out[-1][1] = max(out[-1][1], b)
        else:
            out.append([a, b])
    return out


def _concurrent(recs, sel):
    """Share of the time of the backward-stream records `sel` picks that a
    forward-stream kernel runs at the same time."""
    fwd = _merge([(r["start_ms"], r["end_ms"]) for r in recs if r["stream"] == 0 and r["kind"] != "empty"])
    tot = inter = 0.0
    for r in recs:
        if r["stream"] < 1 or not sel(r):
            continue
        a, b = r["start_ms"], r["end_ms"]
        tot += b - a
        for c, d in fwd:
            lo, hi = max(a, c), min(b, d)
            if hi > lo:
                inter += hi - lo
    return inter / tot if tot > 0 else None


def transformer_section(args, log):
    """The detached small transformer (vocabulary 32768, width 512, 8 heads,
    8 layers, sequences of 1024, batch 16): tokens/s of SERIAL and OVERLAP,
    per-kernel times, GEMM MFMA utilisation, and how much backward work runs
    beside forward work, for all of it and for the attention backward."""
    import torch

    from paper_2608_18469_amd import erase_tf, synth_tf
    cfg = synth_tf.tf_config("tf_c5")
    log(f"[bench] transformer tf_c5: V {cfg['vocab']}, d {cfg['d']}, {cfg['heads']} heads, {cfg['layers']} layers, "
        f"T {cfg['seq']}, B {cfg['batch']}")
    params, toks = synth_tf.make_workload(cfg, 0, 2)
    tr = erase_tf.TfTrainer(cfg, params, keep_grads=False)
    dev = [tr.device_tokens(t) for t in toks]
    ntok = cfg["batch"] * cfg["seq"]
    scheds = ["serial", "overlap"]
    times = {s: [] for s in scheds}
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    i = 0
    for s in scheds:
        for _ in range(args.tf_warmup):
            tr.step(dev[i % 2], s, wait_current=False)
            i += 1
    tr.sync()
    for blk in range(2):
        for s in scheds:
            tr.sync()
            t0 = time.perf_counter()
            for _ in range(args.tf_steps // 2):
                tr.step(dev[i % 2], s, wait_current=False)
                i += 1
            tr.sync()
            times[s].append((time.perf_counter() - t0) / (args.tf_steps // 2))
        log(f"[bench] transformer block {blk + 1}/2 done")
    res = {s: {"tokens_per_s": ntok / float(np.mean(v)), "ms_per_step": float(np.mean(v)) * 1e3} for s, v in times.items()}
    for s in scheds:
        log(f"[bench] transformer {s}: {res[s]['tokens_per_s']:.0f} tokens/s, {res[s]['ms_per_step']:.2f} ms/step")
    # per-launch timing
    tr.set_timing(True)
    recs = {}
    for s in scheds:
        recs[s] = []
        for _ in range(3):
            tr.step(dev[i % 2], s, wait_current=False)
            i += 1
            tr.sync()
            recs[s].append(tr.read_timing()[1:])
    tr.set_timing(False)
    tr.close()
    classes = {}
    for rs in recs["serial"]:
        for r in rs:
            name = r["kind"] + (":" + erase_tf.GEMM_NAMES[r["layer"]] if r["kind"].endswith("gemm") else
                                f":{r['layer']}" if r["kind"] == "attn_bwd" else "")
            c = classes.setdefault(name, {"ms": 0.0, "n": 0, "flops": 0.0, "bytes": 0.0})
            c["ms"] += r["end_ms"] - r["start_ms"]
            c["n"] += 1
            c["flops"] += r["flops"]
            c["bytes"] += r["bytes"]
    n = len(recs["serial"])
    kernels = {k: {"avg_us": v["ms"] / v["n"] * 1e3, "us_per_step": v["ms"] / n * 1e3,
                   "launches_per_step": v["n"] / n,
                   "tflops": v["flops"] / (v["ms"] / 1e3) / 1e12 if v["flops"] else None,
                   "gbs": v["bytes"] / (v["ms"] / 1e3) / 1e9 if v["bytes"] else None}
               for k, v in sorted(classes.items(), key=lambda kv: -kv[1]["ms"])}
    gm = [v for k, v in classes.items() if "gemm" in k]
    gemm_util = sum(v["flops"] for v in gm) / (sum(v["ms"] for v in gm) / 1e3) / 1e12 / PEAK_BF16_TFLOPS
    fl = synth_tf.flops_per_step(cfg)
    best = max(("overlap",), key=lambda s: res[s]["tokens_per_s"])
    ovl_all = float(np.mean([_concurrent(r, lambda x: True) for r in recs["overlap"]]))
    ovl_att = [_concurrent(r, lambda x: x["kind"] == "attn_bwd" and x["layer"] >= 2) for r in recs["overlap"]]
    ovl_voc = [_concurrent(r, lambda x: x["kind"].endswith("gemm") and x["layer"] == 4) for r in recs["overlap"]]
    dom = max(kernels.items(), key=lambda kv: kv[1]["us_per_step"])
    cpu = None
    if not args.no_cpu_baseline:
        log(f"[bench] transformer cpu baseline: oracle for ~{args.tf_cpu_budget:.0f} s")
        cpu = tf_cpu_baseline(cfg, params, toks, args.tf_cpu_budget)
    return {
        "workload": "tf_c5: detached small transformer, vocabulary 32768, d_model 512, 8 heads of 64, 8 layers "
                    "(causal attention + 4x GELU MLP, pre-RMSNorm), each layer with its own RMSNorm + "
                    "Linear(512->32768) next-token softmax-CE head; batch 16 x 1024 tokens, uniform random "
                    "token ids, bf16 operands, fp32 accumulation, Adam",
        "metric": "train tokens/s @1 MI355X",
        "value": res[best]["tokens_per_s"],
        "unit": "tokens/s",
        "schedule": best,
        "schedules": res,
        "overlap_vs_serial": res["overlap"]["tokens_per_s"] / res["serial"]["tokens_per_s"],
        "steps": args.tf_steps, "warmup": args.tf_warmup,
        "flops_per_step": fl["total"],
        "mfma_util": {"gemm_kernels": gemm_util,
                      "whole_step": fl["total"] / (res[best]["ms_per_step"] / 1e3) / 1e12 / PEAK_BF16_TFLOPS,
                      "counter_busy": (measured_mfma_busy("tf_c5") or {}).get("util"),
                      "counter_busy_detail": measured_mfma_busy("tf_c5") or
                      f"null: no MFMA busy counters of the current kernels ({kernel_source_hash(TF_SOURCES)})"},
        "bwd_fwd_overlap_fraction": ovl_all,
        "attention_bwd_overlap_fraction": float(np.mean([x for x in ovl_att if x is not None])) if any(
            x is not None for x in ovl_att) else None,
        "vocab_gemm_overlap_fraction": float(np.mean([x for x in ovl_voc if x is not None])) if any(
            x is not None for x in ovl_voc) else None,
        "dominant_kernel": dom[0],
        "kernels": kernels,
        "cpu_baseline": cpu,
    }


def normalized_entropy(losses, y):
    """Normalized entropy of each block's head (the paper's CTR metric,
    Section 3.2): the mean BCE divided by the entropy of the label base rate
    p of the batch, -(p log p + (1 - p) log(1 - p))."""
    p = float(np.mean(y))
    h = -(p * np.log(p) + (1.0 - p) * np.log1p(-p))
    return {"per_block": [float(l) / h for l in losses], "label_rate": p, "base_entropy": h}


def layer_kind(cfg, r):
    blk = cfg["blocks"][r["block"]] if r["block"] >= 0 else None
    if blk and 0 <= r["layer"] < len(blk["layers"]):
        return blk["layers"][r["layer"]][0]
    return None


def ctr_section(args, workload, log, scheds, headline, steps, warmup, timing_steps, cpu=True, inputs=True,
                n_batches=8):
    """One CTR-shaped workload: every schedule timed interleaved, per-kernel
    figures from a SERIAL timing pass, the overlap of backward with forward
    kernels from an OVERLAP timing pass, the dominant kernel's roofline, MFMA
    utilisation, the normalized entropy of the heads, and (optionally) the
    CPU baseline and the device input stage."""
    import torch

    from paper_2608_18469_amd import erase, synth
    cfg = synth.config(workload)
    bf16 = cfg["dtype"] == "bf16"
    log(f"[bench] generating {workload} (batch {cfg['batch']}, {len(cfg['blocks'])} blocks, {n_batches} batches)")
    # one more batch than the timed steps cycle over: held out, for the
    # normalized entropy of data the heads have not trained on
    params, batches = synth.make_workload(cfg, 0, n_batches + 1)
    held = batches.pop()
    in_place = not args.x_copy and cfg["batch"] % 128 == 0
    tr = erase.Trainer(cfg, params, keep_grads=True, bwd_streams=args.bwd_streams, x_in_place=in_place)
    dev = [tr.device_batch(x, y) for (x, y) in batches]
    losses = torch.zeros(len(cfg["blocks"]), device="cuda")
    flops_step = synth.gemm_flops_per_step(cfg)
    M = cfg["batch"]
    # the heads at initialisation: one serial step on batch 0
    tr.step(*dev[0], "serial", losses, wait_current=False)
    tr.sync()
    ne0 = normalized_entropy(losses.cpu().numpy(), batches[0][1])

    res, one_step = time_schedules(tr, dev, scheds, steps, warmup, args.block, losses, M, log)
    if timing_steps <= 0:  # schedules only (e.g. under a kernel-trace profiler)
        tr.close()
        return cfg, {"value": res[headline]["samples_per_s"], "ms_per_step": res[headline]["ms_per_step"],
                     "schedule": headline, "schedules": res}

    # Per-launch kernel times from HIP events the library records around each
    # launch on that launch's own stream: a SERIAL pass (each kernel alone on
    # the device: the kernel table and the roofline) and an OVERLAP pass (the
    # measured backward/forward overlap).
    tr.set_dispatch("caller")
    log(f"[bench] kernel timing: {timing_steps} serial + {timing_steps} overlap steps")
    recs_all = timed_records(tr, one_step, "serial", timing_steps)
    recs_ovl = timed_records(tr, one_step, "overlap", timing_steps)
    # an empty event pair per step (reported only: kernel events are stamped by the kernel dispatch)
    ev_cost_ms = float(np.median([r[0]["end_ms"] - r[0]["start_ms"] for r in recs_all]))
    recs_all = [r[1:] for r in recs_all]
    recs_ovl = [r[1:] for r in recs_ovl]
    classes = {}
    for recs in recs_all:
        for r in recs:
            name = kernel_class(r, bf16)
            if layer_kind(cfg, r) == "cross" and r["kind"].startswith("fwd_gemm"):
                name = name.replace("erase_fwd_gemm", "erase_fwd_cross_gemm")
            c = classes.setdefault(name, {"ms": 0.0, "n": 0, "flops": 0.0, "bytes": 0.0, "kind": r["kind"]})
            c["ms"] += r["end_ms"] - r["start_ms"]
            c["n"] += 1
            c["flops"] += r["flops"]
            c["bytes"] += r["bytes"]
    nsteps = len(recs_all)
    ovl = float(np.mean([overlap_fraction(r) for r in recs_ovl]))
    dom_name, dom = max(classes.items(), key=lambda kv: kv[1]["ms"])
    gemm_ms = sum(c["ms"] for c in classes.values() if mfma_kind(c["kind"]))
    gemm_flops = sum(c["flops"] for c in classes.values() if mfma_kind(c["kind"]))
    peak_mfma = PEAK_BF16_TFLOPS if bf16 else PEAK_F32_TFLOPS
    avg_dur_s = dom["ms"] / dom["n"] / 1e3
    roof = roofline_of(dom["flops"] / dom["n"], dom["bytes"] / dom["n"], avg_dur_s, peak_mfma)
    tr_meas = measured_traffic(dom_name, workload)
    roof["traffic"] = tr_meas["bytes"] if tr_meas else None  # HBM bytes per launch, counters
    roof["traffic_detail"] = tr_meas if tr_meas else f"null: no byte counters of the current kernels ({kernel_source_hash()})"
    roof["kernel"] = dom_name
    roof["algorithmic_bytes_per_launch"] = dom["bytes"] / dom["n"]
    roof["algorithmic_flops_per_launch"] = dom["flops"] / dom["n"]
    roof["avg_launch_us"] = avg_dur_s * 1e6
    roof["launches_per_step"] = dom["n"] / nsteps
    kernels = {k: {"avg_us": v["ms"] / v["n"] * 1e3, "launches_per_step": v["n"] / nsteps,
                   "us_per_step": v["ms"] / nsteps * 1e3,
                   "tflops": (v["flops"] / (v["ms"] / 1e3) / 1e12) if mfma_kind(v["kind"]) else None,
                   "gbs": v["bytes"] / (v["ms"] / 1e3) / 1e9}
               for k, v in sorted(classes.items(), key=lambda kv: -kv[1]["ms"])}
    # the heads after the run: the loss of a step is taken before its update,
    # so a step on batch 0 gives the training NE, one on the held-out batch
    # the NE on unseen data
    tr.step(*dev[0], "serial", losses, wait_current=False)
    tr.sync()
    ne1 = normalized_entropy(losses.cpu().numpy(), batches[0][1])
    tr.step(*tr.device_batch(*held), "serial", losses, wait_current=False)
    tr.sync()
    ne_held = normalized_entropy(losses.cpu().numpy(), held[1])
    best_serial = max((k for k in ("serial", "serial_graph") if k in res), key=lambda k: res[k]["samples_per_s"],
                      default=None)
    sp = lambda a, b: res[a]["samples_per_s"] / res[b]["samples_per_s"] if a in res and b in res else None
    out = {
        "value": res[headline]["samples_per_s"],
        "ms_per_step": res[headline]["ms_per_step"],
        "schedule": headline,
        "speedup_vs_serial": {
            "headline_vs_serial": sp(headline, "serial"),
            "headline_vs_best_serial": sp(headline, best_serial) if best_serial else None,
            "overlap_vs_serial": sp("overlap", "serial"),
            "overlap_graph_vs_serial_graph": sp("overlap_graph", "serial_graph"),
            "pipeline_vs_serial": sp("pipeline", "serial"),
            "pipeline_worker_vs_serial": sp("pipeline+worker", "serial")},
        "schedules": res,
        "mfma_util": {"gemm_kernels": gemm_flops / (gemm_ms / 1e3) / 1e12 / peak_mfma if gemm_ms else None,
                      "whole_step": flops_step / (res[headline]["ms_per_step"] / 1e3) / 1e12 / peak_mfma,
                      "counter_busy": (measured_mfma_busy(workload) or {}).get("util"),
                      "counter_busy_detail": measured_mfma_busy(workload) or
                      f"null: no MFMA busy counters of the current kernels ({kernel_source_hash()})"},
        "flops_per_step": flops_step,
        "x_layout": (f"read in place: [{M}][{tr.ncfg.x_ld}] with zero row tails (no per-step copy)" if in_place
                     else f"[{M}][{tr.ncfg.x_ld}], copied into a zero-padded workspace buffer every step"),
        "bwd_fwd_overlap_fraction": ovl,
        "bwd_fwd_overlap_trace": measured_trace_overlap(workload),
        "normalized_entropy": {"first_step": ne0, "after_run_train": ne1, "after_run_held_out": ne_held,
                               "note": "mean BCE of each head over the base-rate entropy of the batch's labels: batch "
                                       "0 at the first step and after the timed steps (the steps cycle over "
                                       f"{n_batches} synthetic batches, which the heads memorise: the labels are "
                                       "random), and a held-out batch after them"},
        "kernel_timing": "per-kernel figures from a SERIAL pass (kernels alone), HIP events stamped at each "
                         "kernel's own start and end; overlap fraction from an OVERLAP pass, over every "
                         "backward stream",
        "event_pair_cost_us": ev_cost_ms * 1e3,
        "roofline": roof,
        "kernels": kernels,
    }
    if cpu and not args.no_cpu_baseline:
        log(f"[bench] cpu baseline: oracle for ~{args.cpu_budget:.0f} s + ~{args.cpu_budget_1t:.0f} s on one thread")
        out["cpu_baseline"] = cpu_baseline(cfg, params, batches, args.cpu_budget, args.cpu_budget_1t)
    if inputs and cfg.get("input_kind") == "ctr" and not args.no_input_stage:
        out["input_stage"] = input_stage(args, log, tr, cfg, headline, dev[0][1], losses)
    tr.close()
    return cfg, out


TRACE_FILE = os.path.join(ROOT, "profiles", "ctr_mlp_overlap_trace.md")
FWD_PREFIXES = ("erase_prologue", "erase_fwd_")
BWD_PREFIXES = ("erase_bwd_gemm", "erase_wgrad_", "erase_dgrad_", "erase_adam", "erase_head_bce")


def _kernel_base(name):
    n = name.split("(")[0].split("<")[0].strip()
    for pre in ("void ", "erase::", "(anonymous namespace)::"):
        n = n.replace(pre, "")
    return n.strip()


def analyze_trace(path):
    """Overlap of backward with forward kernels from a rocprofv3 kernel trace
    (kernel_trace.csv) of one schedule: kernels are forward or backward work
    by name (prologue and forward GEMMs; backward GEMMs and Adam), which also
    holds for kernels replayed from a HIP graph; the fraction is the backward
    kernel time that intersects the union of forward kernel intervals.  Also
    the streams each class ran on and the device time per step."""
    import csv
    fwd, bwd, streams = [], [], {"fwd": set(), "bwd": set()}
    with open(path) as f:
        for row in csv.DictReader(f):
            base = _kernel_base(row["Kernel_Name"])
            a, b = int(row["Start_Timestamp"]), int(row["End_Timestamp"])
            if base.startswith(FWD_PREFIXES):
                fwd.append((a, b))
                streams["fwd"].add(row.get("Stream_Id"))
            elif base.startswith(BWD_PREFIXES):
                bwd.append((a, b))
                streams["bwd"].add(row.get("Stream_Id"))
    merged = _merge(fwd)
    tot = inter = 0
    j = 0
    for a, b in sorted(bwd):
        tot += b - a
        while j < len(merged) and merged[j][1] <= a:
            j += 1
        k = j
        while k < len(merged) and merged[k][0] < b:
            inter += max(0, min(b, merged[k][1]) - max(a, merged[k][0]))
            k += 1
    with open(path) as f:
        pro = sorted(int(r["Start_Timestamp"]) for r in csv.DictReader(f)
                     if _kernel_base(r["Kernel_Name"]).startswith("erase_prologue"))
    gaps = np.diff(pro) / 1e6 if len(pro) > 1 else np.array([])
    return {"overlap_fraction": inter / tot if tot else None, "bwd_kernel_ms": tot / 1e6,
            "fwd_kernels": len(fwd), "bwd_kernels": len(bwd), "steps": len(pro),
            "median_step_ms": float(np.median(gaps)) if gaps.size else None,
            "fwd_streams": sorted(str(x) for x in streams["fwd"]),
            "bwd_streams": sorted(str(x) for x in streams["bwd"])}


def measured_trace_overlap(workload):
    """Trace-derived overlap per schedule from the committed summary of
    rocprofv3 kernel traces (lines 'overlap_trace <workload> <schedule>
    <source hash> <fraction> <median step ms>'), while the kernels are the
    ones traced; None otherwise."""
    try:
        with open(TRACE_FILE) as f:
            lines = f.read().splitlines()
    except OSError:
        return None
    src = kernel_source_hash()
    out = {}
    for line in lines:
        parts = line.split()
        if len(parts) == 6 and parts[0] == "overlap_trace" and parts[1] == workload and parts[3] == src:
            out[parts[2]] = {"overlap_fraction": float(parts[4]), "median_step_ms": float(parts[5])}
    return out or None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="ctr_mlp")
    ap.add_argument("--block", type=int, default=50,
                    help="schedules are timed interleaved, this many steps at a time")
    ap.add_argument("--timing-steps", type=int, default=20)
    ap.add_argument("--cpu-budget", type=float, default=12.0,
                    help="seconds of oracle steps with every BLAS thread (then --cpu-budget-1t with one)")
    ap.add_argument("--cpu-budget-1t", type=float, default=6.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-input-stage", action="store_true",
                    help="skip the device embedding-bag input stage measurement")
    ap.add_argument("--no-conventional", action="store_true",
                    help="skip the ERASE vs conventional backpropagation comparison on the 12-block chain")
    ap.add_argument("--schedules", default="serial,overlap,serial_graph,overlap_graph,pipeline,overlap+worker,"
                                           "pipeline+worker")
    ap.add_argument("--headline", default="pipeline+worker",
                    help="the ERASE schedule whose throughput is the reported value (declared before the run)")
    ap.add_argument("--bwd-streams", type=int, default=2,
                    help="backward streams of the ERASE schedules (block b uses stream b %% n); 2 measured "
                         "fastest on ctr_mlp (1 leaves the backward chain serial, 3+ exceed the 4 hardware queues)")
    ap.add_argument("--x-copy", action="store_true",
                    help="hand x over in its plain layout, copied into a padded workspace buffer every step (by "
                         "default x is resident with rows of a multiple of 128 elements and zero tails, read in "
                         "place)")
    ap.add_argument("--no-dcn", action="store_true", help="skip the CTR-DCNv2 (batch 16384) measurement")
    ap.add_argument("--dcn-steps", type=int, default=40)
    ap.add_argument("--dcn-warmup", type=int, default=5)
    ap.add_argument("--dcn-schedules", default="serial,overlap,pipeline+worker")
    ap.add_argument("--no-transformer", action="store_true", help="skip the small-transformer measurement")
    ap.add_argument("--transformer-only", action="store_true",
                    help="only the small-transformer measurement (its JSON object on stdout)")
    ap.add_argument("--tf-steps", type=int, default=30)
    ap.add_argument("--tf-warmup", type=int, default=5)
    ap.add_argument("--tf-cpu-budget", type=float, default=10.0,
                    help="seconds of transformer oracle steps for its CPU baseline")
    ap.add_argument("--analyze-trace", nargs="+", metavar="KERNEL_TRACE_CSV",
                    help="no GPU run: print the backward/forward overlap of each rocprofv3 kernel trace")
    ap.add_argument("--verbose", action="store_true")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after the run, copy a buffer of this many MiB once (a plain copy kernel of known size "
                         "for scaling hardware byte counters)")
    args = ap.parse_args()

    if args.analyze_trace:
        for pth in args.analyze_trace:
            print(json.dumps({"trace": pth, "source": kernel_source_hash(), **analyze_trace(pth)}))
        return

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the detached-block step is built and timed on a single MI355X; "
              "multi-GPU runs are not part of this build.", file=sys.stderr)
        sys.exit(2)

    import torch

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    log = (lambda *a: print(*a, file=sys.stderr, flush=True))

    if args.transformer_only:
        print(json.dumps(transformer_section(args, log)))
        return

    scheds = args.schedules.split(",")
    if args.headline not in scheds:
        print(f"--headline {args.headline} is not among --schedules {args.schedules}", file=sys.stderr)
        sys.exit(2)
    cfg, sec = ctr_section(args, args.workload, log, scheds, args.headline, args.steps, args.warmup,
                           args.timing_steps, n_batches=8 if args.workload == "ctr_mlp" else 2)
    bf16 = cfg["dtype"] == "bf16"
    M = cfg["batch"]
    out = {
        "metric": METRIC,
        "value": sec["value"],
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": sec["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if bf16 else "f32",
        "data": "synthetic (seeded CTR-shaped input: 13 log1p-LogNormal dense + 26 Zipf(1.1) sum-pooled "
                "embedding bags of dim 64; random-init weights)",
        "config": {"workload": f"{args.workload}: 6 detached blocks 1677->512->256->128 + Linear(128->1) BCE head, "
                               f"batch {M}, Adam" if args.workload == "ctr_mlp" else args.workload,
                   "global_batch": M, "blocks": len(cfg["blocks"]), "schedule": args.headline,
                   "headline_declared": True, "bwd_streams": args.bwd_streams, "parallelism": "single GPU"},
    }
    out.update({k: v for k, v in sec.items() if k not in ("value", "ms_per_step", "schedule")})
    if args.workload == "ctr_mlp" and not args.no_dcn:
        dscheds = args.dcn_schedules.split(",")
        dhead = args.headline if args.headline in dscheds else dscheds[-1]
        _, dcn = ctr_section(args, "ctr_dcn", log, dscheds, dhead, args.dcn_steps, args.dcn_warmup,
                             max(2, args.timing_steps // 4), cpu=False, inputs=False, n_batches=2)
        dcn["workload"] = ("ctr_dcn: 6 detached blocks of 2 DCNv2 cross layers (1677) + 1677->1024->1024->512 "
                           "+ Linear(512->1) BCE head, batch 16384, bf16, Adam")
        dcn["unit"] = "samples/s"
        out["ctr_dcn"] = dcn
    if not args.no_transformer:
        out["transformer"] = transformer_section(args, log)
    if not args.no_conventional:
        out["erase_vs_conventional"] = conventional_comparison(args, log)
    if args.calib_copy_mib:
        n = args.calib_copy_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        out["calib_copy_bytes"] = 2 * n * 4
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
