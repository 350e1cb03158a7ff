"""kf_fused_op_noalloc, the entry point that allocates nothing, against
kf_create + kf_fused_op on the same inputs: the same kernels with the static
scratch in place of the descriptor's workspace, so the outputs must agree
bit for bit.  Two calls in a row per plan family that uses scratch (row
softmax / logsumexp partials, repacked conv weights), the second smaller, so
the second reuses scratch the first filled; and a plan with no scratch."""
import numpy as np
import pytest

from paper_2605_30359_amd import inputs, kf
from parity import check, run_gpu, sample_rows

pytestmark = pytest.mark.gpu


def _bits(t):
    import torch
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t


def _noalloc(cfg, seed):
    import torch
    t = inputs.generate(cfg, seed=seed)
    op, ref = run_gpu(cfg, t)
    ins = op.device_inputs(t)
    out = op.empty_output("cuda")
    out.fill_(float("nan") if out.dtype != torch.float32 else -1.0)
    print(f"[noalloc] {cfg['name']} {kf.sizes_of(cfg)}", flush=True)
    kf.fused_op_noalloc(inputs.chain_for(cfg, t), ins, out, **kf.sizes_of(cfg))
    torch.cuda.synchronize()
    assert torch.equal(_bits(ref), _bits(out)), cfg["name"]
    return t, out


@pytest.mark.parametrize("first,second", [
    (("C5", dict(M=1024, N=4096, K=256)), ("C5", dict(M=300, N=1040, K=208))),   # softmax partials
    (("C2", dict(M=2048, N=4096, K=256)), ("C2", dict(M=77, N=520, K=64))),      # logsumexp partials
    (("C4", dict(batch=4, H=16)), ("C4", dict(batch=1, H=8))),                    # repacked conv weights
    (("F2", dict(batch=2, D=10, H=18, W=34)), ("F2", dict(batch=1, D=6, H=10, W=18))),  # conv3d weights
    (("C3", dict(M=512, N=1024, K=128, ops=[("groupnorm", 4, 1e-5), ("swish",), ("residual_add",)])),
     ("C3", dict(M=100, N=256, K=64, ops=[("groupnorm", 1, 1e-5), ("swish",), ("residual_add",)]))),  # no scratch
])
def test_noalloc_matches_fused_op_twice(first, second):
    for (name, kw), seed in ((first, 5), (second, 6)):
        cfg = inputs.config(name, **kw)
        t, out = _noalloc(cfg, seed)
        if cfg["contraction"] in ("gemm", "rowwise"):
            check(cfg, t, out, rows=sample_rows(cfg["M"], 8))
        else:
            check(cfg, t, out, images=np.array([0]))


def test_noalloc_full_size_softmax():
    """The headline workload's plan (8192 rows x 32 tiles of partials = 2 MiB
    of scratch) through the entry point that allocates nothing."""
    cfg = inputs.config("C5")
    t, out = _noalloc(cfg, None)
    check(cfg, t, out, rows=sample_rows(cfg["M"], 4))


def test_noalloc_refuses_partly_fused_conv3d():
    """A Conv3d chain with a channel softmax outside the tiled kernel's
    family (here an NCDHW input) needs intermediate buffers: the entry point
    that allocates nothing refuses it before any launch."""
    import torch
    cfg = inputs.config("F2", batch=1, D=6, H=10, W=18)
    t = inputs.generate(cfg, seed=3)
    op = kf.FusedOp(inputs.chain_for(cfg, t), **kf.sizes_of(cfg))
    ins = op.device_inputs(t, conv3d_channels_last=False)
    out = op.empty_output("cuda")
    with pytest.raises(kf.KFError) as e:
        kf.fused_op_noalloc(inputs.chain_for(cfg, t), ins, out, **kf.sizes_of(cfg))
    assert e.value.status == kf.KF_ERR_UNSUPPORTED and "intermediate" in str(e.value)
    torch.cuda.synchronize()
