"""kf_fused_op under HIP graph capture: a serving loop can record the fused
operation once (the contraction and, for a row softmax, its finishing
kernel) and replay it without host launch work.  The library's launch path
records kernels only -- no allocation, no memset, no host synchronisation --
once a first eager call has packed the conv weights and sized the grids.
Each replay is compared bit for bit with the eager result, with eager work
and synchronisations between the replays."""
import numpy as np
import pytest

from paper_2605_30359_amd import inputs, kf
from parity import check, sample_rows

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,kw", [
    ("C5", dict(M=1024, N=2048, K=512)),          # fp8 GEMM + row softmax: GEMM and finishing kernel
    ("C3", dict(M=512, N=8192, K=256)),           # GroupNorm (256-column groups) + swish + residual
    ("C4", dict(batch=2, H=16)),                  # conv + pool (weights packed by the eager call)
    ("F2", dict(batch=2, D=10, H=18, W=34)),      # conv3d + channel softmax + pools
    ("F3", dict(M=256, N=4096)),                  # row-wise GroupNorm chain
])
def test_graph_replay_matches_eager(name, kw):
    import torch
    cfg = inputs.config(name, **kw)
    t = inputs.generate(cfg, seed=61)
    op = kf.FusedOp(inputs.chain_for(cfg, t), **kf.sizes_of(cfg))
    ins = op.device_inputs(t)
    ref = op.empty_output("cuda")
    op(ins, ref)                      # eager: packs weights, sizes grids
    torch.cuda.synchronize()
    bits = (lambda x: x.view(torch.int16)) if ref.dtype == torch.bfloat16 else (lambda x: x)
    out = op.empty_output("cuda")
    print(f"[gpu] graph {name} {kw}", flush=True)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            op(ins, out)
    torch.cuda.current_stream().wait_stream(side)
    for rep in range(3):
        out.fill_(-1.0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(bits(ref), bits(out)), (name, rep)
        op(ins, ref)                  # eager work between replays
        torch.cuda.synchronize()
    if cfg["contraction"] in ("gemm", "rowwise"):
        check(cfg, t, out, rows=sample_rows(cfg["M"], 6))
    else:
        check(cfg, t, out, images=np.array([0]))


@pytest.mark.parametrize("name,kw", [
    ("C5", dict(M=1024, N=2048, K=512)),          # softmax partials in the static scratch
    ("C4", dict(batch=2, H=16)),                  # conv weights repacked into the scratch on every call
])
def test_graph_replay_of_the_entry_point_that_allocates_nothing(name, kw):
    """kf_fused_op_noalloc, the entry point for callers under HIP graph
    capture, recorded once (after a first eager call has looked up the
    scratch address) and replayed: every replay matches the eager result bit
    for bit."""
    import torch
    cfg = inputs.config(name, **kw)
    t = inputs.generate(cfg, seed=62)
    chain = inputs.chain_for(cfg, t)
    sizes = kf.sizes_of(cfg)
    op = kf.FusedOp(chain, **sizes)
    ins = op.device_inputs(t)
    ref = op.empty_output("cuda")
    kf.fused_op_noalloc(chain, ins, ref, **sizes)
    torch.cuda.synchronize()
    bits = (lambda x: x.view(torch.int16)) if ref.dtype == torch.bfloat16 else (lambda x: x)
    out = op.empty_output("cuda")
    print(f"[gpu] graph noalloc {name} {kw}", flush=True)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            kf.fused_op_noalloc(chain, ins, out, stream=side, **sizes)
    torch.cuda.current_stream().wait_stream(side)
    for rep in range(3):
        out.fill_(-1.0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(bits(ref), bits(out)), (name, rep)
        kf.fused_op_noalloc(chain, ins, ref, **sizes)   # eager work between replays
        torch.cuda.synchronize()
    if cfg["contraction"] == "gemm":
        check(cfg, t, out, rows=sample_rows(cfg["M"], 6))
    else:
        check(cfg, t, out, images=np.array([0]))
