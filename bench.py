#!/usr/bin/env python3
"""Benchmark of the fused contraction + epilogue path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload C5] [--also C3,C4]

A step is one kf_fused_op call: the whole fused operation (contraction,
fused epilogue, row finishing kernel) on one batch of seeded synthetic input
already resident in device memory.  The headline workload (default C5, the
largest of the five: fp8 e4m3 GEMM 8192 x 8192 x 8192 with per-tensor scales
+ bias + hardtanh(-1, 1) + row softmax -> bf16 [8192, 8192]) fills the JSON
line; each workload named by --also (default the large bf16 ones, C3 and C4)
gets a block of the same fields under "also".  Per workload:

  value        whole-step throughput in TFLOP/s (2*M*N*K / mean step time
               over the K back-to-back steps)
  steps_us     per-step HIP-event times: median, min, p90, mean -- warm
               (back-to-back steps, a second loop of K steps) and cold (a
               read of a 512 MiB device buffer between steps, outside the
               events, evicts the L2s and the 256 MB Infinity Cache and
               leaves them clean)
  roofline     the main contraction kernel alone, timed live with HIP events
               recorded on its stream around each launch (achieved = the
               algorithmic FLOPs per launch / the mean launch time; median,
               min and p90 beside it), against the dense MFMA peak of its
               input dtype; `traffic` is the HBM bytes per launch from the
               committed rocprofv3 counter summary, or null if the kernel
               source changed since those counters were taken
  graph        the same step captured once in a HIP graph and replayed K
               times (median, min, p90 per replay): the step without the
               host's launch work
  unfused      the same operation as the library's own one-kernel-per-op
               chain, timed the same way; speedup = unfused / fused time
  cpu_baseline the fp64 oracle timed on the host cores over a bounded sample
               of rows (or images) of the same workload (every op in the
               chain is local to a row or an image, so a sample is the same
               computation per unit)
  tuning       the launch configuration kf_autotune kept before the timed
               steps (every candidate computes the same bits), or the one
               given with --tuning; for a GEMM also the modelled operand
               bytes its tile order makes the L2s fetch
  probe        the measured ceiling beside the datasheet peak: for bf16 /
               fp8 contractions kf_probe_mfma, the matrix cores' sustained
               rate with no memory traffic on this GPU in this run and the
               shader clock it ran at (the datasheet assumes 2.4 GHz); for
               the row-wise chains kf_probe_copy, a plain 512 MiB device
               copy (2 x 512 MiB, beyond the Infinity Cache); the roofline
               block carries achieved / that rate as frac_of_probe, and the
               cold kernel median's rate / that rate as frac_of_probe_cold
  clock_stamps (GEMMs) the shader clock inside the kernel, from its
               per-workgroup clock stamps (kf_set_clock_stamps) over 20
               launches, the tile time, the shares of prologue, K loop and
               epilogue in a tile's cycles, and the matrix cores' busy
               fraction within a tile and within its K loop at that clock
  diagnosis    kf_diagnose_counters on the measured kernel time and the
               committed counters (HBM bytes, matrix-core busy fraction, LDS
               bank conflicts) when they match the kernel source: compute and
               memory fractions, the bound and the recommendations
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# Dense peaks of one MI355X (256 CUs at 2.4 GHz), TFLOP/s.
PEAK_TFLOPS = {"bf16": 2516.6, "e4m3": 5033.2, "f32": 157.3}
HBM_PEAK_GBS = 8000.0
COLD_FLUSH_BYTES = 512 << 20
# rounds of 8 MFMAs per SIMD for the matrix-core probe: about 30 ms each at
# the clocks this GPU sustains under that load
PROBE_ITERS = {"bf16": 200000, "e4m3": 100000}
_probe_cache: dict = {}


PROBE_COPY_BYTES = 512 << 20


def _probe(dt: str):
    """The measured ceiling, once per process: the matrix-core rate probe for
    dtype dt, or (dt "hbm") the plain device copy of 512 MiB."""
    from paper_2605_30359_amd import kf
    if dt not in PROBE_ITERS and dt != "hbm":
        return None
    if dt not in _probe_cache:
        if dt == "hbm":
            r = kf.probe_copy(PROBE_COPY_BYTES, 10)
            _probe_cache[dt] = {"kind": "copy", "bytes": PROBE_COPY_BYTES, "gbps": round(r["gbps"], 1),
                                "frac_of_datasheet": round(r["gbps"] / HBM_PEAK_GBS, 4),
                                "ms": round(r["seconds"] * 1e3, 3)}
        else:
            r = kf.probe_mfma(dt, PROBE_ITERS[dt])
            _probe_cache[dt] = {"kind": "mfma", "dtype": dt, "tflops": round(r["tflops"], 1),
                                "clock_ghz": round(r["clock_ghz"], 3),
                                "frac_of_datasheet": round(r["tflops"] / PEAK_TFLOPS[dt], 4),
                                "ms": round(r["seconds"] * 1e3, 3)}
    return _probe_cache[dt]


def _hip():
    lib = ctypes.CDLL("libamdhip64.so")
    lib.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
    lib.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
    lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
    lib.hipEventDestroy.argtypes = [ctypes.c_void_p]
    lib.hipEventSynchronize.argtypes = [ctypes.c_void_p]
    lib.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    return lib


# Timing-only events: no system-scope fence (no cache writeback and
# invalidation around the kernel they bracket).
HIP_EVENT_DISABLE_SYSTEM_FENCE = 0x20000000


def _event(hip):
    e = ctypes.c_void_p()
    assert hip.hipEventCreateWithFlags(ctypes.byref(e), HIP_EVENT_DISABLE_SYSTEM_FENCE) == 0
    return e.value


def _elapsed_ms(hip, a, b) -> float:
    ms = ctypes.c_float()
    assert hip.hipEventElapsedTime(ctypes.byref(ms), ctypes.c_void_p(a), ctypes.c_void_p(b)) == 0
    return float(ms.value)


def _stats_us(ms_list) -> dict:
    """median, min, p90 and mean of a list of durations in ms, in us."""
    import numpy as np
    v = np.sort(np.asarray(ms_list, dtype=np.float64)) * 1e3
    return {"median": round(float(np.median(v)), 2), "min": round(float(v[0]), 2),
            "p90": round(float(np.percentile(v, 90)), 2), "mean": round(float(v.mean()), 2), "n": int(v.size)}


def _source_digest(kernel_files) -> str:
    """Digest of a kernel's sources (its files plus the shared device headers),
    so that a counter summary taken on other sources is not reported."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2605_30359_amd", "csrc")
    files = set(kernel_files) | {"kf_device.hpp", "kf_internal.hpp"}
    for name in sorted(os.listdir(csrc)):
        if name in files:
            h.update(open(os.path.join(csrc, name), "rb").read())
    return h.hexdigest()[:16]


KERNEL_FILES = {
    "kf_gemm_mfma_256x256": ["kf_gemm_mfma.hpp", "kf_gemm_epilogue.hpp", "kf_gemm_mfma.hip", "kf_gemm_mfma_bf16_nk.hip",
                             "kf_gemm_mfma_fp8_kn.hip", "kf_gemm_mfma_fp8_nk.hip"],
    "kf_gemm_mfma_pp128x256": ["kf_gemm_pp.hpp", "kf_gemm_epilogue.hpp", "kf_gemm_pp_bf16.hip", "kf_gemm_pp_fp8.hip"],
    "kf_gemm_f32_8x8": ["kf_gemm_f32.hip"],
    "kf_conv3x3_bf16_256x128": ["kf_conv_bf16.hip"],
    "kf_conv3x3_bf16_w8": ["kf_conv_bf16.hip"],
    "kf_conv3x3_bf16_gen": ["kf_conv_bf16.hip"],
    "kf_rowwise": ["kf_rowwise.hip"],
    "kf_rowwise_gn_panel": ["kf_rowwise.hip"],
    "kf_row_reduce_stream": ["kf_rowwise.hip"],
    "kf_conv3d_bf16_64x256": ["kf_conv3d_bf16.hip"],
    "kf_conv3d_bf16_gen": ["kf_conv3d_gen.hip"],
}


def _traffic_record(kernel: str, workload: str):
    """The committed counter summary of a kernel on a workload (HBM bytes per
    launch and the launch configuration they were counted with), if it was
    taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path)).get(f"{kernel}:{workload}")
    except Exception:
        return None
    if not rec or rec.get("source_digest") != _source_digest(KERNEL_FILES.get(kernel, [])):
        return None
    return rec


def _cpu_baseline(cfg, tensors, gpu_out, budget_s: float):
    """Time the fp64 oracle on the host cores over a bounded sample of the
    same workload: whole output rows (GEMM) or whole images (conv), drawn in
    a seeded random order and computed in chunks whose size adapts to the
    measured rate until about `budget_s` seconds of oracle work are done
    (wrapping round to the start if the whole workload takes less).  Every op
    of a chain is local to a row (GEMM) or an image (conv), so a chunk is the
    same per-unit computation as the full op.  The GPU output of the
    benchmarked op is checked against the oracle on every distinct unit of
    the sample."""
    import numpy as np

    import oracle
    from paper_2605_30359_amd import inputs

    ch = inputs.chain_for(cfg, tensors)
    rowwise = cfg["contraction"] == "rowwise"
    gemm = cfg["contraction"] == "gemm" or rowwise  # a sample is a set of rows
    units = cfg["M"] if gemm else cfg["batch"]
    work = inputs.rowwise_bytes(cfg) if rowwise else inputs.flops(cfg)
    work_unit = work / max(units, 1)
    unit_name = "output rows" if gemm else "images"

    import torch
    g_all = gpu_out.cpu()
    bf16_out = g_all.dtype == torch.bfloat16
    g_all = g_all.view(torch.int16).numpy().view(np.uint16) if bf16_out else g_all.numpy()
    names = [o[0] for o in cfg["ops"]]
    floor = (1.0 / cfg["N"] if names and names[-1] == "row_softmax" else
             1.0 / cfg["cout"] if "channel_softmax" in names else 1.0)

    perm = np.random.default_rng(0).permutation(units).astype(np.int64)
    pos, done, elapsed, err = 0, 0, 0.0, 0.0
    chunk = min(units, 64 if gemm else 2)
    while True:
        sel = perm[np.arange(pos, pos + chunk) % units]
        t0 = time.perf_counter()
        ref = oracle.run_chain(ch, tensors, **({"rows": sel} if gemm else {"images": sel}))
        dt = time.perf_counter() - t0
        if pos < units:
            fresh = np.arange(pos, pos + chunk) < units
            g = g_all[sel[fresh]]
            g = oracle.decode_bf16(g) if bf16_out else g.astype(np.float64)
            r = ref[fresh]
            e = np.abs(g - r) / np.maximum(np.abs(r), floor)
            err = max(err, float(np.max(e)) if np.all(np.isfinite(g)) else float("inf"))
        pos += chunk
        done += chunk
        elapsed += dt
        if elapsed >= budget_s:
            break
        rate = done / elapsed
        chunk = int(max(1, min(4 * chunk, units, rate * (budget_s - elapsed) + 1)))
    passes = done / units
    return {
        "value": done * work_unit / elapsed / (1e9 if rowwise else 1e12),
        "unit": "GB/s" if rowwise else "TFLOP/s",
        "cores": oracle.threads(),
        "kind": "oracle",
        "sample": (f"{done} {unit_name} ({passes:.2f} x the {units} of the full workload, seeded random order) "
                   f"of the same workload, fp64 plain C + OpenMP, {elapsed:.1f} s"),
        "seconds": round(elapsed, 2),
    }, err


def _timed_steps(hip, torch, run, steps, flush=None, kernel_events=True, step_events=True):
    """`steps` calls of run(ev_before, ev_after) on the current stream,
    bracketed by two events, each step between two step events if
    step_events; `flush` (a device tensor, written once beforehand) is read
    whole before every step, outside the events: the caches then hold its
    clean lines, and whatever the previous step left dirty in them is
    written back before the step starts.  run() records ev_before / ev_after around its main
    kernel when kernel_events is set.  Returns (total ms of the loop,
    per-step ms, per-kernel ms)."""
    stream = torch.cuda.current_stream()
    kev = [(_event(hip), _event(hip)) for _ in range(steps)] if kernel_events else []
    sev = [(_event(hip), _event(hip)) for _ in range(steps)] if step_events else []
    start, end = _event(hip), _event(hip)
    torch.cuda.synchronize()
    s = ctypes.c_void_p(stream.cuda_stream)
    hip.hipEventRecord(ctypes.c_void_p(start), s)
    for i in range(steps):
        if flush is not None:
            flush.view(torch.int32).sum()
        if step_events:
            hip.hipEventRecord(ctypes.c_void_p(sev[i][0]), s)
        run(*(kev[i] if kernel_events else (None, None)))
        if step_events:
            hip.hipEventRecord(ctypes.c_void_p(sev[i][1]), s)
    hip.hipEventRecord(ctypes.c_void_p(end), s)
    torch.cuda.synchronize()
    total = _elapsed_ms(hip, start, end)
    step_ms = [_elapsed_ms(hip, a, b) for a, b in sev]
    kern_ms = [_elapsed_ms(hip, a, b) for a, b in kev]
    for a, b in kev + sev + [(start, end)]:
        hip.hipEventDestroy(ctypes.c_void_p(a))
        hip.hipEventDestroy(ctypes.c_void_p(b))
    return total, step_ms, kern_ms


def run_workload(name: str, args, hip, cpu_budget: float) -> dict:
    """Time one workload; returns the fields of its JSON block."""
    import torch

    from paper_2605_30359_amd import inputs, kf

    print(f"[bench] {name}: generating inputs", file=sys.stderr, flush=True)
    cfg = inputs.config(name)
    tensors = inputs.generate(cfg)
    chain = inputs.chain_for(cfg, tensors)
    op = kf.FusedOp(chain, **kf.sizes_of(cfg))
    ins = op.device_inputs(tensors, "cuda:0")
    out = op.empty_output("cuda:0")

    # the plan's launch candidates, timed on these inputs; the fastest is kept,
    # or for a GEMM the fewest modelled L2 panel bytes within 2% of it (every
    # candidate computes the same bits)
    tuning = None
    if args.tuning:
        op.set_tuning(*(int(v) for v in args.tuning.split(",")))
        tuning = {"config": op.tuning(), "candidates": 0, "best_ms": None, "default_ms": None}
    elif not args.no_autotune:
        keys = ("raster_group", "xcd_remap", "wg_per_cu", "variant")
        plan_default = op.tuning()
        r = op.autotune(ins, out, reps=max(3, args.warmup // 2))
        default = [c for c in r["candidates"] if all(c[k] == plan_default[k] for k in keys)]
        tuning = {"config": {k: r["best"][k] for k in keys}, "candidates": len(r["candidates"]),
                  "best_ms": round(r["best"]["seconds"] * 1e3, 5),
                  "default_ms": round(default[0]["seconds"] * 1e3, 5) if default else None,
                  "panel_bytes_model": r["best"]["panel_bytes"] if r["best"]["panel_bytes"] >= 0 else None}

    print(f"[bench] {name}: timing", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        op(ins, out)
    torch.cuda.synchronize()

    K = args.steps
    fused = lambda e0, e1: op.timed(ins, out, e0, e1)  # noqa: E731
    # the timed steps: the main kernel bracketed by its own events, nothing
    # else recorded inside the loop (each event record costs the stream a few
    # microseconds)
    total_ms, _, kern_ms = _timed_steps(hip, torch, fused, K, step_events=False)
    ms_per_step = total_ms / K
    # per-step statistics from a second warm loop with step events only
    _, step_ms, _ = _timed_steps(hip, torch, lambda e0, e1: op(ins, out), K, kernel_events=False)
    # the same step recorded once in a HIP graph and replayed: the launch work
    # of the host (ctypes call, validation, kernel launches) leaves the loop
    graph = None
    if not args.no_graph:
        try:
            g = torch.cuda.CUDAGraph()
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                with torch.cuda.graph(g, stream=side):
                    op(ins, out)
            torch.cuda.current_stream().wait_stream(side)
            g.replay()
            torch.cuda.synchronize()
            g_total, g_step, _ = _timed_steps(hip, torch, lambda e0, e1: g.replay(), K, kernel_events=False)
            graph = {"ms_per_step": round(g_total / K, 5), "step_us": _stats_us(g_step)}
            del g
        except Exception as e:  # noqa: BLE001 -- reported, not fatal
            graph = {"error": str(e)}
    cold = None
    if args.cold_steps > 0:
        flush = torch.ones(COLD_FLUSH_BYTES, dtype=torch.uint8, device="cuda:0")
        _, c_step, c_kern = _timed_steps(hip, torch, fused, args.cold_steps, flush=flush)
        del flush
        cold = {"step_us": _stats_us(c_step), "kernel_us": _stats_us(c_kern)}

    # contraction chains are measured in FLOP/s against the MFMA (or fp32)
    # peak; the row-wise chains, which have no contraction, in bytes per
    # second against HBM bandwidth
    rowwise = cfg["contraction"] == "rowwise"
    dt = cfg["in_dtype"]
    work = inputs.rowwise_bytes(cfg) if rowwise else inputs.flops(cfg)
    peak = HBM_PEAK_GBS if rowwise else PEAK_TFLOPS[dt]
    scale = 1e9 if rowwise else 1e12
    kernel_ms = sum(kern_ms) / len(kern_ms)
    value = work / (ms_per_step * 1e-3) / scale
    achieved = work / (kernel_ms * 1e-3) / scale
    kname = op.kernel_name()

    unfused = None
    if not args.no_unfused:
        try:
            u_out = op.empty_output("cuda:0")
            for _ in range(max(2, args.warmup // 2)):
                op.unfused(ins, u_out)
            torch.cuda.synchronize()
            u_total, u_step, _ = _timed_steps(hip, torch, lambda e0, e1: op.unfused(ins, u_out), K,
                                              kernel_events=False)
            u_ms = u_total / K
            unfused = {"ms_per_step": round(u_ms, 5), "step_us": _stats_us(u_step),
                       "speedup": round(u_ms / ms_per_step, 3)}
            del u_out
        except kf.KFError as e:
            unfused = {"error": str(e)}

    probe = None if args.no_probe else _probe("hbm" if rowwise else dt)
    # the shader clock inside the GEMM kernel, from its per-workgroup clock
    # stamps; the shares of prologue, K loop and epilogue in a tile's cycles;
    # and the matrix cores' busy fraction within a tile and its K loop
    stamps = None
    if kname == "kf_gemm_mfma_256x256" and not args.no_stamps:
        tiles = -(-cfg["M"] // 256) * -(-cfg["N"] // 256)
        per_cycle = 2048 if dt == "e4m3" else 1024   # FLOP per clock per SIMD of a 32x32 MFMA stream
        mfma_cycles = 2.0 * 256 * 256 * cfg["K"] / 4 / per_cycle
        stamps = op.clock_stamps(lambda: op(ins, out), tiles, mfma_cycles=mfma_cycles)
        if "error" not in stamps:
            stamps = {k: (round(v, 4) if isinstance(v, float) else v) for k, v in stamps.items()}
    probe_rate = None if not probe else probe["gbps"] if rowwise else probe["tflops"]

    trec = _traffic_record(kname, cfg["workload"])
    traffic = trec.get("hbm_bytes_per_launch") if trec else None
    # the diagnosis from the live kernel time and, when the committed counter
    # summary matches the kernel source, its counted bytes, matrix-core busy
    # fraction and LDS bank conflicts
    diag = op.diagnose_counters(kernel_ms * 1e-3, float(traffic) if traffic else -1.0,
                                float(trec.get("mfma_busy", -1.0)) if trec else -1.0,
                                float(trec.get("lds_conflict", -1.0)) if trec else -1.0)
    diagnosis = {k: (round(v, 4) if isinstance(v, float) else v) for k, v in diag.items()
                 if k in ("bound", "compute_frac", "memory_frac", "intensity", "ridge", "workgroups", "compute_units",
                          "mfma_busy", "lds_conflict", "traffic_ratio", "hints")}

    cpu, err = (None, None)
    if cpu_budget > 0:
        print(f"[bench] {name}: cpu baseline", file=sys.stderr, flush=True)
        cpu, err = _cpu_baseline(cfg, tensors, out, cpu_budget)

    sizes = kf.sizes_of(cfg)
    block = {
        "value": round(value, 2),
        "unit": "GB/s" if rowwise else "TFLOP/s",
        "ms_per_step": round(ms_per_step, 5),
        "dtype": dt,
        "config": dict({"workload": cfg["workload"], "ops": "+".join(o[0] for o in cfg["ops"]),
                        "out_dtype": cfg["out_dtype"]}, **sizes),
        ("pct_hbm_peak" if rowwise else "pct_mfma_peak"): round(100.0 * value / peak, 2),
        "steps_us": {"warm": _stats_us(step_ms), "cold": cold["step_us"] if cold else None},
        "graph": graph,
        "speedup_vs_unfused": None if not unfused or "speedup" not in unfused else unfused["speedup"],
        "unfused": unfused,
        "roofline": {
            "bound": "hbm" if rowwise else "mfma",
            "kernel": kname,
            "achieved": round(achieved, 2),
            "peak": peak,
            "unit": "GB/s" if rowwise else "TFLOP/s",
            "frac": round(achieved / peak, 4),
            "frac_of_probe": round(achieved / probe_rate, 4) if probe_rate else None,
            # the cold kernels read from HBM like the probe copy (2 x 512 MiB,
            # larger than the Infinity Cache); warm row-wise launches may find
            # their input in that cache
            "frac_of_probe_cold": (round(work / (cold["kernel_us"]["median"] * 1e-6) / scale / probe_rate, 4)
                                   if probe_rate and cold else None),
            "kernel_us": round(kernel_ms * 1e3, 2),
            "kernel_us_stats": _stats_us(kern_ms),
            "kernel_us_cold": cold["kernel_us"] if cold else None,
            ("bytes_per_launch" if rowwise else "flops_per_launch"): work,
            "traffic": traffic,
            # the launch configuration the counters were taken with (the
            # raster order changes how often operand panels are re-fetched)
            "traffic_launch_config": trec.get("launch_config") if trec else None,
        },
        "probe": probe,
        "clock_stamps": stamps,
        "diagnosis": diagnosis,
        "tuning": tuning,
        "cpu_baseline": cpu,
        "parity_err_cpu_sample": err,
    }
    op.close()
    del ins, out, tensors
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    print(f"[bench] {name}: {block['value']} {block['unit']}, kernel {block['roofline']['kernel_us']} us",
          file=sys.stderr, flush=True)
    return block


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="C5", help="headline workload: C1..C5, F1..F6 (default C5)")
    ap.add_argument("--also", default="C3,C4",
                    help="comma-separated workloads timed after the headline, each reported under 'also' "
                         "(default C3,C4; empty for none)")
    ap.add_argument("--cold-steps", type=int, default=10,
                    help="steps timed with a 512 MiB device read before each (0: no cold timing)")
    ap.add_argument("--cpu-budget", type=float, default=12.0, help="seconds of oracle work for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-unfused", action="store_true")
    ap.add_argument("--no-autotune", action="store_true", help="keep the default launch configuration")
    ap.add_argument("--no-probe", action="store_true", help="skip the measured-ceiling probe")
    ap.add_argument("--no-graph", action="store_true", help="skip the HIP-graph replay timing")
    ap.add_argument("--no-stamps", action="store_true", help="skip the GEMM kernel's clock stamps")
    ap.add_argument("--tuning", default=None, metavar="RG,XR,WG[,V]",
                    help="use this launch configuration (raster group, XCD order, workgroups per CU, kernel variant) "
                         "instead of autotuning")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 256 MiB device copy 5 times (for scaling HBM byte counters)")
    args = ap.parse_args(argv)

    if args.copy_calibration:
        import torch
        src = torch.empty(256 << 20, dtype=torch.uint8, device="cuda:0")
        src.fill_(1)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": src.numel(), "launches": 5}))
        return 0

    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(sharded along rows or the batch, each GPU would run this same single-GPU kernel on its "
              "share with no cross-GPU exchange)",
              file=sys.stderr)
        return 2

    import torch

    torch.cuda.set_device(0)
    hip = _hip()
    budget = 0.0 if args.no_cpu_baseline else args.cpu_budget
    head = run_workload(args.workload, args, hip, budget)
    also = {}
    for name in [w for w in args.also.split(",") if w and w != args.workload]:
        also[name] = run_workload(name, args, hip, budget)

    rowwise = head["unit"] == "GB/s"
    line = {
        "metric": ("fused-op GB/s, % of HBM peak, speedup vs own unfused kernel chain" if rowwise else
                   "fused-op TFLOP/s, % of MFMA peak, speedup vs own unfused kernel chain"),
        "value": head["value"],
        "unit": head["unit"],
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": head["dtype"],
        "data": "synthetic",
    }
    line.update({k: v for k, v in head.items() if k not in line and k != "unit"})
    line["also"] = also
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
