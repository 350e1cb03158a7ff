"""Helpers for the GPU parity tests: run a workload through the C ABI and
compare with the fp64 oracle on the same seeded bits.

Comparison metric (max over compared elements):
    err = max |g - o| / max(|o|, floor)
with floor = 1 (absolute error below magnitude 1, relative above) except for
softmax outputs, whose floor is the uniform probability 1/N (1/cout for a
softmax over channels; values near it are compared relative to that
scale).  Any NaN / Inf in the GPU output
fails.  Tolerances per input dtype: fp32 1e-4, bf16 2e-2, fp8 6e-2, all with
fp32 accumulation.
"""
from __future__ import annotations

import numpy as np

import oracle
from paper_2605_30359_amd import inputs, kf

TOL = {"f32": 1e-4, "bf16": 2e-2, "e4m3": 6e-2}


def floor_for(cfg) -> float:
    names = [o[0] for o in cfg["ops"]]
    if names and names[-1] == "row_softmax":
        return 1.0 / cfg["N"]
    if "channel_softmax" in names:
        return 1.0 / cfg["cout"]
    return 1.0


def to_host_f64(t) -> np.ndarray:
    """Device output -> float64 (exact widening, no device compute)."""
    import torch
    if t.dtype == torch.bfloat16:
        bits = t.view(torch.int16).cpu().numpy().view(np.uint16)
        return oracle.decode_bf16(bits)
    return t.cpu().numpy().astype(np.float64)


def parity_error(gpu: np.ndarray, ref: np.ndarray, floor: float) -> float:
    if not np.all(np.isfinite(gpu)):
        return float("inf")
    if gpu.size == 0:
        return 0.0
    return float(np.max(np.abs(gpu - ref) / np.maximum(np.abs(ref), floor)))


def run_gpu(cfg, tensors, chain=None, unfused=False, tuning=None):
    """Plan the op (with launch configuration `tuning`, a (raster group, XCD
    order, workgroups per CU, variant) tuple, if given), copy inputs to the
    device, run, return (op, out tensor)."""
    import torch
    chain = chain if chain is not None else inputs.chain_for(cfg, tensors)
    op = kf.FusedOp(chain, **kf.sizes_of(cfg))
    if tuning is not None:
        op.set_tuning(*tuning)
    print(f"[gpu] {cfg.get('name')} {kf.sizes_of(cfg)} ops={[o[0] for o in chain['ops']]} unfused={unfused} "
          f"tuning={tuning}", flush=True)
    ins = op.device_inputs(tensors)
    out = op.empty_output("cuda")
    if unfused:
        op.unfused(ins, out)
    else:
        op(ins, out)
    torch.cuda.synchronize()
    return op, out


def sample_rows(M: int, n: int, seed: int = 0) -> np.ndarray:
    """First, last and random rows (sorted, unique)."""
    rng = np.random.default_rng(seed)
    rows = {0, M - 1, M // 2}
    rows.update(rng.integers(0, M, size=max(0, n - 3)).tolist())
    return np.array(sorted(rows), dtype=np.int64)


def check(cfg, tensors, gpu_out, rows=None, images=None, tol=None, chain=None, unfused=False, fused=None):
    """Compare a GPU output with the oracle: the fused chain's plain
    definition, or (unfused=True) the one-op-per-kernel evaluation that
    stores every intermediate in the chain's intermediate format, or
    (fused=p) the partly fused one: the contraction with its first p ops in
    one kernel, then one kernel per op."""
    chain = chain if chain is not None else inputs.chain_for(cfg, tensors)
    if fused is not None:
        ref = oracle.run_chain_unfused(chain, tensors, rows=rows, images=images, fused=fused)
    else:
        run = oracle.run_chain_unfused if unfused else oracle.run_chain
        ref = run(chain, tensors, rows=rows, images=images)
    g = to_host_f64(gpu_out)
    if rows is not None:
        g = g[rows]
    if images is not None:
        g = g[images]
    err = parity_error(g, ref, floor_for(cfg))
    tol = TOL[cfg["in_dtype"]] if tol is None else tol
    assert err <= tol, f"{cfg['name']}: parity error {err:.3e} > {tol:.1e}"
    return err
