#!/usr/bin/env python3
"""Update-throughput benchmark of the actor-critic learner on one MI355X.

Metric: update frames/s = batch rows fully processed per second, i.e. update
steps per second times the batch size (the paper's "network update frame rate",
Section 4.2, Tables 2 and 3). One step is the whole update: replay gather,
target action, target and online twin critics, critic loss and backward,
actor forward/backward through the critics, temperature, Adam and Polyak.

Default workload: the large-batch SAC case (obs 376, act 17, 3x1024 ReLU MLPs,
batch 131072, 4M-row ring, bf16 GEMM operands with fp32 accumulation and fp32
master weights / Adam). The ring is filled with synthetic rows before timing and
stays resident in HBM; nothing is transferred from the host in the timed region.

Prints one JSON line (rank 0). Also reports the dominant kernel against its
roofline (per-launch event timings taken by the library on the stream the kernel
runs on, during the timed region, where only that kernel's launches carry events,
in every TIMED_STRIDE-th step;
the kernel is picked, and the per-kernel table taken, in an untimed survey pass
before) and the CPU oracle's rate on a bounded sample of the same workload.
roofline.traffic (HBM bytes per launch) and roofline.mfma_busy (share of cycles the
matrix cores are busy, rocprofv3's MfmaUtil) come from the committed counter
summaries under profiles/, and are null once the kernel sources differ from the
ones the counters were taken on.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "actor-critic update frames/sec (batch rows/s) at 1 MI355X; MFMA util %"
PEAK_TFLOPS = {"bf16": 2500.0, "fp32": 157.3}   # MI355X dense matrix peaks
PEAK_HBM_GBS = 8000.0
GEMMS = ("gemm_fwd", "gemm_dgrad", "gemm_wgrad")
SURVEY_STEPS = 10   # untimed steps with every kernel launch timed (per-kernel table)
# In the timed region the dominant kernel's launches carry events in every
# TIMED_STRIDE-th step only (each event pair costs the GPU a few microseconds).
TIMED_STRIDE = 8
# Measured HBM traffic of the dominant kernel (rocprofv3 FETCH_SIZE / WRITE_SIZE,
# scaled by a plain copy of known size), valid while the kernel sources hash the same.
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemm_fwd_1024_sac_large_bf16_traffic.txt")
# Matrix-core busy share of the dominant kernel (rocprofv3 MfmaUtil), same validity rule.
MFMA_FILE = os.path.join(ROOT, "profiles", "gemm_mfma_util_sac_large_bf16.md")
KERNEL_SOURCES = ("gemm_big.hip", "gemm.hip", "internal.h")


def progress(msg: str):
    print("[bench] " + msg, file=sys.stderr, flush=True)


def frames_per_second(batch: int, steps: int, seconds: float) -> float:
    """Update frame rate = update frequency x batch size (rows per second)."""
    return batch * steps / seconds


def fill_ring(g, w, data_seed: int, rows: int):
    import synth
    chunk = 1 << 18
    t0 = time.time()
    for r0 in range(0, rows, chunk):
        n = min(chunk, rows - r0)
        g.buffer_push(*synth.workload_rows(w, r0, n, data_seed))
        if (r0 // chunk) % 4 == 3 or r0 + n >= rows:
            progress("ring %d / %d rows (%.1fs)" % (r0 + n, rows, time.time() - t0))


def kernel_source_hash() -> str:
    """Hash of the GEMM sources with comments and blank space removed (an edit to a
    comment leaves the counters valid; any change to the code does not)."""
    import hashlib
    import re
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2312_06126_amd", "csrc", f)) as fh:
            src = fh.read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        src = re.sub(r"//[^\n]*", "", src)
        h.update("\n".join(ln.strip() for ln in src.splitlines() if ln.strip()).encode())
    return h.hexdigest()[:16]


def profile_value(path: str, kernel: str, key: str):
    """A `key: value` entry of a committed counter summary, or None when there is none
    for this kernel or the kernel sources changed since the counters were taken."""
    try:
        kv = {}
        with open(path) as fh:
            for line in fh:
                if ":" in line and not line.startswith(("#", "|")):
                    k, v = line.split(":", 1)
                    kv[k.strip()] = v.strip()
        if kv.get("kernel") != kernel or kv.get("source_sha256") != kernel_source_hash():
            return None
        return float(kv[key])
    except (OSError, KeyError, ValueError):
        return None


def measured_traffic(kernel: str):
    """HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated)."""
    return profile_value(TRAFFIC_FILE, kernel, "traffic_bytes_per_launch")


def roofline(stats, prec: str):
    """The dominant kernel (largest total time) against its MI355X roofline."""
    top = stats[0]
    avg_s = top["avg_ms"] / 1e3
    if top["name"] in GEMMS:
        achieved = top["flops"] / avg_s / 1e12
        peak = PEAK_TFLOPS[prec]
        r = dict(bound="mfma", achieved=round(achieved, 2), peak=peak, unit="TFLOP/s")
    else:
        achieved = top["bytes"] / avg_s / 1e9
        peak = PEAK_HBM_GBS
        r = dict(bound="hbm", achieved=round(achieved, 1), peak=peak, unit="GB/s")
    r["frac"] = round(achieved / peak, 4)
    r["kernel"] = "%s M=%d N=%d K=%d" % (top["name"], top["M"], top["N"], top["K"])
    r["traffic"] = measured_traffic(r["kernel"])
    r["mfma_busy"] = profile_value(MFMA_FILE, r["kernel"], "mfma_busy") if top["name"] in GEMMS else None
    r["avg_launch_ms"] = round(top["avg_ms"], 5)
    r["launches"] = top["launches"]
    r["timed_every_steps"] = TIMED_STRIDE
    r["per_launch"] = top["flops"] if top["name"] in GEMMS else top["bytes"]
    return r


def sweep(g, w, stream, steps: int = 30, warm: int = 3):
    """Frame rate at the geometric batch sizes 16384 .. the workload's batch (the
    paper's batch-size enumeration, Section 3.4), on the timed context switched with
    spz_set_batch (its buffers are sized for the largest batch); the knee is the
    smallest batch within 5% of the best frame rate. Restores the workload's batch."""
    import torch
    out = []
    b = min(16384, w.batch)
    while True:
        g.set_batch(b)
        g.update(warm, stream)
        torch.cuda.synchronize()
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        g.update(steps, stream)
        t1.record(stream)
        torch.cuda.synchronize()
        ms = t0.elapsed_time(t1) / steps
        out.append(dict(batch=b, ms_per_step=round(ms, 4), value=round(frames_per_second(b, steps, ms * steps / 1e3), 1)))
        progress("sweep batch %d: %.3f ms/step" % (b, ms))
        if b >= w.batch:
            break
        b = min(2 * b, w.batch)
    g.set_batch(w.batch)
    best = max(r["value"] for r in out)
    knee = min(r["batch"] for r in out if r["value"] >= 0.95 * best)
    return dict(points=out, knee_batch=knee, steps=steps, note="one context created at the workload's batch, "
                "spz_set_batch between points, %d untimed steps before each" % warm)


def timed_rate(g, w, stream, steps: int, warmup: int):
    """ms per step and frame rate of `steps` update steps after `warmup` (events on stream)."""
    import torch
    g.update(warmup, stream)
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    g.update(steps, stream)
    t1.record(stream)
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    return dict(ms_per_step=round(ms, 4), value=round(frames_per_second(w.batch, steps, ms * steps / 1e3), 1),
                steps=steps, warmup=warmup)


def hbm_kernels(survey, names=("gather", "adam_polyak")):
    """Achieved HBM rate of the memory-bound kernels of the step (algorithmic bytes per
    launch over the mean event-measured duration in the survey pass) against 8 TB/s."""
    out = {}
    for s in survey:
        if s["name"] in names and s["name"] not in out and s["bytes"] > 0:
            gbs = s["bytes"] / (s["avg_ms"] / 1e3) / 1e9
            out[s["name"]] = dict(achieved=round(gbs, 1), peak=PEAK_HBM_GBS, unit="GB/s",
                                  frac=round(gbs / PEAK_HBM_GBS, 4), bytes_per_launch=s["bytes"],
                                  avg_launch_us=round(s["avg_ms"] * 1e3, 2))
    return out


def cpu_baseline(w, seed: int, data_seed: int, sample_batch: int):
    import numpy as np  # noqa: F401
    import synth
    from oracle import Oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = 1
    ws = w.replace(batch=sample_batch)
    o = Oracle(ws.obs_dim, ws.act_dim, ws.hidden, ws.batch, ws.hparams(), seed,
               row_source=lambda idx: synth.workload_rows_at(ws, idx, data_seed))
    o.set_virtual_size(ws.capacity)
    t0 = time.perf_counter()
    o.update(1)
    dt = time.perf_counter() - t0
    return dict(value=round(sample_batch / dt, 1), unit="rows/s", cores=threads, kind="oracle",
                sample="1 update step of %s at batch %d (full widths, %s operand emulation), %.1f s" %
                       (w.name, sample_batch, w.prec, dt))


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed steps (default: the workload's)")
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="sac_large_bf16")
    ap.add_argument("--batch", type=int, default=None, help="override the workload batch")
    ap.add_argument("--streams", type=int, default=1, choices=(1, 2),
                    help="2 runs the actor and critic halves on concurrent streams (per-kernel event "
                         "durations then overlap, so the roofline is taken from 1-stream runs)")
    ap.add_argument("--graphs", default="auto", choices=("auto", "0", "1"),
                    help="replay update steps from captured HIP graphs (auto: on for every workload but "
                         "the large one, whose roofline needs events on its kernels in the timed region)")
    ap.add_argument("--no-sweep", action="store_true",
                    help="skip the batch sweep 16384..batch (default on for the large workload)")
    ap.add_argument("--no-streams2", action="store_true",
                    help="skip the two-stream rate reported beside the one-stream headline")
    ap.add_argument("--autotune", action="store_true",
                    help="also run the library's adaptive batch-size controller (spz_autotune_batch) "
                         "from batch 16384 on a context created with the workload's batch")
    ap.add_argument("--seed", type=int, default=1)
    ap.add_argument("--data-seed", type=int, default=0)
    ap.add_argument("--cpu-sample-batch", type=int, default=32768)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true", help="skip per-kernel event timing")
    args = ap.parse_args()

    if args.gpus != 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path "
              "(--gpus %d requested)" % args.gpus, file=sys.stderr)
        sys.exit(2)
    if int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs as a single process on one GPU", file=sys.stderr)
        sys.exit(2)

    import torch

    import synth
    from paper_2312_06126_amd import Spz

    w = synth.workload(args.workload)
    if args.batch:
        w = w.replace(batch=args.batch)
    steps = args.steps if args.steps is not None else w.steps
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()

    large = w.name == "sac_large_bf16"
    graphs = (not large) if args.graphs == "auto" else args.graphs == "1"
    progress("workload %s batch %d ring %d prec %s streams %d graphs %d" % (w.name, w.batch, w.capacity, w.prec,
                                                                            args.streams, graphs))
    g = Spz(w.obs_dim, w.act_dim, w.hidden, w.batch, dict(w.hparams(), graphs=int(graphs)), args.seed,
            n_streams=args.streams)
    fill_ring(g, w, args.data_seed, w.capacity)

    g.update(args.warmup, stream)
    g.synchronize()
    torch.cuda.synchronize()
    progress("warmup %d steps done" % args.warmup)

    survey, top = [], None
    if not args.no_profile:
        # Untimed survey pass: every kernel launch of a few steps bracketed by events,
        # for the per-kernel table and to find the dominant kernel. In the timed
        # region only that kernel's launches carry events (events on every launch
        # cost the step several percent).
        g.profile_enable(True, reserve_launches=150 * SURVEY_STEPS)
        g.update(SURVEY_STEPS, stream)
        survey = g.profile_read()
        top = survey[0]
        if graphs:
            # Graph replays carry no per-kernel events: the timed region runs without
            # timing, and the roofline takes the dominant kernel's survey average.
            g.profile_enable(False, 0)
            progress("survey %d steps; timed region replays graphs, no kernel events" % SURVEY_STEPS)
        else:
            g.profile_enable(True, reserve_launches=40 * steps)
            g.profile_only(top["name"], top["M"], top["N"], top["K"])
            g.profile_stride(TIMED_STRIDE)
            progress("survey %d steps; timing %s M=%d N=%d K=%d in every %dth step of the timed region" %
                     (SURVEY_STEPS, top["name"], top["M"], top["N"], top["K"], TIMED_STRIDE))
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record(stream)
    g.update(steps, stream)
    t_end.record(stream)
    torch.cuda.synchronize()
    g.synchronize()
    elapsed_ms = t_start.elapsed_time(t_end)
    progress("timed %d steps: %.3f ms/step" % (steps, elapsed_ms / steps))

    stats = (g.profile_read() if not graphs else [dict(top)]) if top else []
    rec = g.read_losses(g.step() - steps + 1, steps)
    finite = bool((rec[:, 6] == 0).all())
    sweep_out = None
    if large and not args.no_sweep:
        g.profile_enable(False, 0)
        sweep_out = sweep(g, w, stream)
    g.close()
    streams2 = None
    if large and args.streams == 1 and not args.no_streams2:
        # The actor and critic halves on two concurrent streams (the one-GPU form of the
        # paper's two-GPU actor/critic split), same workload, another context.
        g2 = Spz(w.obs_dim, w.act_dim, w.hidden, w.batch, w.hparams(), args.seed, n_streams=2)
        fill_ring(g2, w, args.data_seed, w.capacity)
        streams2 = timed_rate(g2, w, stream, steps, args.warmup)
        g2.close()
        progress("two streams: %.3f ms/step" % streams2["ms_per_step"])

    value = frames_per_second(w.batch, steps, elapsed_ms / 1e3)
    prec = w.prec
    out = dict(metric=METRIC, value=round(value, 1), unit="rows/s", n_gpus=1, steps=steps, warmup=args.warmup,
               ms_per_step=round(elapsed_ms / steps, 4), higher_is_better=True, scaling="weak",
               vs_baseline=None, dtype=prec, data="synthetic",
               config=dict(workload=w.name, algo=w.algo, global_batch=w.batch, obs_dim=w.obs_dim,
                           act_dim=w.act_dim, hidden=list(w.hidden), replay_rows=w.capacity,
                           gemm_operands=prec, accumulate="fp32", master_weights="fp32",
                           streams=args.streams, seed=args.seed, data_seed=args.data_seed,
                           graphs=int(graphs),
                           parallelism="single GPU; " + ("actor and critic on concurrent streams"
                                                         if args.streams == 2 else "one stream")),
               losses_finite=finite)
    if not large:
        out["us_per_step"] = round(elapsed_ms / steps * 1e3, 1)
    if stats:
        gemm_ms = sum(s["total_ms"] for s in survey if s["name"] in GEMMS)
        gemm_flops = sum(s["flops"] * s["launches"] for s in survey if s["name"] in GEMMS)
        peak = PEAK_TFLOPS[prec] * 1e12
        out["mfma_util"] = dict(
            gemm_kernels=round(gemm_flops / (gemm_ms / 1e3) / peak, 4) if gemm_ms else None,
            whole_step=round(gemm_flops / SURVEY_STEPS / (elapsed_ms / steps / 1e3) / peak, 4),
            gemm_flops_per_step=gemm_flops / SURVEY_STEPS, peak_tflops=PEAK_TFLOPS[prec],
            note="gemm_kernels: GEMM flops / summed GEMM kernel time of the survey pass (events on every "
                 "launch; concurrent streams overlap); whole_step: GEMM flops per step / timed ms per step. "
                 "Both leave out the row-restricted input-gradient products of the SAC actor path "
                 "(gemm_dgrad_rows: a data-dependent number of rows, about half the batch per critic)")
        out["roofline"] = roofline(stats, prec)
        if graphs:
            out["roofline"]["timed_every_steps"] = None
            out["roofline"]["note"] = ("graph replays carry no kernel events: dominant kernel's mean event "
                                       "duration over the survey pass")
        out["hbm_kernels"] = hbm_kernels(survey)
        out["kernels"] = [dict(name=s["name"], M=s["M"], N=s["N"], K=s["K"], launches=s["launches"],
                               avg_ms=round(s["avg_ms"], 5), total_ms=round(s["total_ms"], 3))
                          for s in survey[:40]]
        out["kernels_note"] = "survey pass of %d untimed steps before the timed region" % SURVEY_STEPS
    if sweep_out:
        out["sweep"] = sweep_out
    if streams2:
        out["streams2"] = streams2
    if args.autotune:
        g = Spz(w.obs_dim, w.act_dim, w.hidden, w.batch, w.hparams(), args.seed, n_streams=args.streams)
        fill_ring(g, w, args.data_seed, w.capacity)
        chosen, probes = g.autotune_batch(min(16384, w.batch), 50, 0.05, stream)
        g.close()
        out["autotune"] = dict(chosen_batch=chosen, probe_steps=50, tolerance=0.05,
                               probes=[dict(batch=b, value=round(r, 1)) for b, r in probes])
        progress("autotune chose batch %d from %s" % (chosen, probes))
    if not args.no_cpu_baseline:
        progress("cpu baseline (oracle) at batch %d" % args.cpu_sample_batch)
        out["cpu_baseline"] = cpu_baseline(w, args.seed, args.data_seed, args.cpu_sample_batch)
        out["cpu_baseline"]["cpu"] = platform.processor() or platform.machine()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
