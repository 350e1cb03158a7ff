"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle on
the same seeded inputs.  Small and ragged shapes are compared element by
element; the full workload sizes are compared on sampled rows, plus a
bit-exact integer test of the contraction at full size."""
import numpy as np
import pytest

import oracle
from paper_2605_30359_amd import inputs, kf
from parity import TOL, check, parity_error, run_gpu, sample_rows, to_host_f64

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


# ------------------------------------------------------------ C1 (fp32)

def test_c1_full_config():
    _torch()
    cfg = inputs.config("C1")
    t = inputs.generate(cfg)
    _, out = run_gpu(cfg, t)
    err = check(cfg, t, out)
    print(f"C1 err {err:.3e}")


@pytest.mark.parametrize("M,N,K", [(1, 1, 1), (33, 65, 31), (100, 300, 257), (64, 512, 0)])
def test_c1_ragged(M, N, K):
    _torch()
    cfg = inputs.config("C1", M=M, N=N, K=K)
    t = inputs.generate(cfg, seed=M + N + K)
    _, out = run_gpu(cfg, t)
    check(cfg, t, out)


def test_c1_nk_layout_and_gelu_chain():
    _torch()
    cfg = inputs.config("C1", M=40, N=96, K=72, b_layout="nk",
                        ops=[("bias",), ("gelu_erf",), ("scale", -1.5), ("tanh",), ("swish",), ("sigmoid",), ("hardtanh", 0.55, 0.7)])
    t = inputs.generate(cfg, seed=3)
    _, out = run_gpu(cfg, t)
    check(cfg, t, out)


# ------------------------------------------------------------ bf16 GEMM

def test_bf16_contraction_bit_exact_full_size():
    """Integer-valued bf16 operands in [-8, 8]: every partial sum is an
    integer below 2^24, so the fp32 accumulator must equal the exact product."""
    torch = _torch()
    M = N = K = 4096
    rng = np.random.default_rng(11)
    a = rng.integers(-8, 9, size=(M, K)).astype(np.float32)
    b = rng.integers(-8, 9, size=(K, N)).astype(np.float32)
    t = {"a": inputs.f32_to_bf16_bits(a), "b": inputs.f32_to_bf16_bits(b)}
    cfg = inputs.config("C2", out_dtype="f32", ops=[])
    print("bit-exact 4096^3: launching", flush=True)
    _, out = run_gpu(cfg, t)
    g = out.cpu().numpy()
    # float64 BLAS is exact here: every partial sum is an integer < 2^53
    ref = a.astype(np.float64) @ b.astype(np.float64)
    print("bit-exact 4096^3: reference done", flush=True)
    assert np.array_equal(g.astype(np.float64), ref)


def test_bf16_contraction_bit_exact_c3_shape():
    """The integer test at C3's shape (8192 x 2048 times 2048 x 8192, 1024
    tiles: four per CU in the kept tile order and in both tile shapes),
    every output checked."""
    torch = _torch()
    M, N, K = 8192, 8192, 2048
    rng = np.random.default_rng(13)
    a = rng.integers(-8, 9, size=(M, K)).astype(np.float32)
    b = rng.integers(-8, 9, size=(K, N)).astype(np.float32)
    t = {"a": inputs.f32_to_bf16_bits(a), "b": inputs.f32_to_bf16_bits(b)}
    cfg = inputs.config("C3", out_dtype="f32", ops=[])
    ref = a.astype(np.float64) @ b.astype(np.float64)
    for tuning in ((2, 0, 2, 0), (4, 1, 2, 1)):
        print(f"bit-exact 8192x8192x2048 tuning {tuning}", flush=True)
        _, out = run_gpu(cfg, t, tuning=tuning)
        assert np.array_equal(out.cpu().numpy().astype(np.float64), ref), tuning
        del out


def test_fp8_contraction_bit_exact_c5_shape():
    """The integer test at C5's full 8192^3 (unit scales; 1024 sampled rows
    against float64 products, exact since every partial sum is an integer
    below 2^22)."""
    _torch()
    M = N = K = 8192
    rng = np.random.default_rng(32)
    a, qa = _int_e4m3(rng, (M, K))
    b, qb = _int_e4m3(rng, (K, N))
    t = {"a": qa, "b": qb, "scale_a": 1.0, "scale_b": 1.0}
    cfg = inputs.config("C5", out_dtype="f32", ops=[])
    print("fp8 bit-exact 8192^3", flush=True)
    _, out = run_gpu(cfg, t)
    rows = sample_rows(M, 1024, seed=5)
    ref = a[rows].astype(np.float64) @ b.astype(np.float64)
    assert np.array_equal(out.cpu().numpy()[rows].astype(np.float64), ref)


def test_bf16_contraction_bit_exact_nk_ragged():
    torch = _torch()
    M, N, K = 300, 264, 200
    rng = np.random.default_rng(12)
    a = rng.integers(-8, 9, size=(M, K)).astype(np.float32)
    b = rng.integers(-8, 9, size=(N, K)).astype(np.float32)
    t = {"a": inputs.f32_to_bf16_bits(a), "b": inputs.f32_to_bf16_bits(b)}
    cfg = inputs.config("C2", M=M, N=N, K=K, out_dtype="f32", ops=[], b_layout="nk")
    _, out = run_gpu(cfg, t)
    assert np.array_equal(out.cpu().numpy().astype(np.float64), a.astype(np.float64) @ b.astype(np.float64).T)


@pytest.mark.parametrize("M,N,K", [(300, 520, 136), (256, 256, 64), (1, 8, 8), (513, 776, 1000),
                                   (5, 16648, 40)])  # 66 column tiles: the row finish loops over them
def test_c2_ragged(M, N, K):
    _torch()
    cfg = inputs.config("C2", M=M, N=N, K=K)
    t = inputs.generate(cfg, seed=M * 7 + N + K)
    _, out = run_gpu(cfg, t)
    err = check(cfg, t, out)
    print(f"C2 {M}x{N}x{K} err {err:.3e}")


def test_c2_full_config_sampled_rows():
    _torch()
    cfg = inputs.config("C2")
    t = inputs.generate(cfg)
    _, out = run_gpu(cfg, t)
    rows = sample_rows(cfg["M"], 48)
    err = check(cfg, t, out, rows=rows)
    print(f"C2 full err {err:.3e}")
    # a property at every row: max_j s_ij <= lse_i <= max_j s_ij + ln N is
    # implied by the sampled parity; every row must at least be finite
    assert np.all(np.isfinite(to_host_f64(out)))


def test_c2_zero_weights_closed_form():
    _torch()
    cfg = inputs.config("C2", M=512, N=4096, K=64)
    t = inputs.generate(cfg, seed=5)
    t["b"] = np.zeros_like(t["b"])
    t["bias"] = np.zeros_like(t["bias"])
    _, out = run_gpu(cfg, t)
    g = to_host_f64(out)
    assert np.max(np.abs(g - np.log(4096.0))) < 1e-5


@pytest.mark.parametrize("M,N,K,G", [(300, 512, 136, 2), (256, 1024, 64, 8), (77, 256, 24, 1)])
def test_c3_ragged(M, N, K, G):
    _torch()
    cfg = inputs.config("C3", M=M, N=N, K=K, ops=[("groupnorm", G, 1e-5), ("swish",), ("residual_add",)])
    t = inputs.generate(cfg, seed=M + N * 3 + K)
    _, out = run_gpu(cfg, t)
    err = check(cfg, t, out)
    print(f"C3 {M}x{N}x{K} G={G} err {err:.3e}")


def test_c3_full_config_sampled_rows():
    _torch()
    cfg = inputs.config("C3")
    t = inputs.generate(cfg)
    _, out = run_gpu(cfg, t)
    rows = sample_rows(cfg["M"], 256)
    err = check(cfg, t, out, rows=rows)
    print(f"C3 full err {err:.3e}")


def test_c3_zero_weights_closed_form():
    _torch()
    cfg = inputs.config("C3", M=64, N=512, K=32, ops=[("groupnorm", 2, 1e-5), ("swish",), ("residual_add",)])
    t = inputs.generate(cfg, seed=9)
    t["b"] = np.zeros_like(t["b"])
    _, out = run_gpu(cfg, t)
    beta = t["beta"].astype(np.float64)
    expect = beta / (1 + np.exp(-beta)) + oracle.decode_bf16(t["residual"])
    assert parity_error(to_host_f64(out), expect, 1.0) < 1e-2


@pytest.mark.parametrize("M,N,K", [(300, 1032, 136), (64, 8192, 64)])
def test_bf16_row_softmax(M, N, K):
    _torch()
    cfg = inputs.config("C2", M=M, N=N, K=K, out_dtype="bf16",
                        ops=[("bias",), ("hardtanh", -1.0, 1.0), ("row_softmax",)])
    t = inputs.generate(cfg, seed=M + N)
    _, out = run_gpu(cfg, t)
    err = check(cfg, t, out)
    g = to_host_f64(out)
    assert np.allclose(g.sum(axis=1), 1.0, atol=2e-2)
    print(f"bf16 softmax err {err:.3e}")


def test_bf16_groupnorm_width_128_and_relu_chain():
    _torch()
    cfg = inputs.config("C3", M=130, N=384, K=96,
                        ops=[("scale", 2.0), ("groupnorm", 3, 1e-5), ("relu",), ("residual_add",)])
    t = inputs.generate(cfg, seed=21)
    _, out = run_gpu(cfg, t)
    check(cfg, t, out)


def test_empty_m_is_a_no_op():
    torch = _torch()
    cfg = inputs.config("C2", M=0, N=256, K=64)
    t = inputs.generate(cfg, seed=1)
    _, out = run_gpu(cfg, t)
    assert out.numel() == 0


@pytest.mark.parametrize("name,kw", [
    ("C1", dict(M=33, N=72, K=0)),
    ("C2", dict(M=70, N=296, K=0)),
    ("C3", dict(M=40, N=512, K=0, ops=[("groupnorm", 2, 1e-5), ("swish",), ("residual_add",)])),
    ("C5", dict(M=33, N=272, K=0)),
])
def test_empty_contraction_k0(name, kw):
    """K = 0: every pre-activation is exactly zero (an empty sum), so the
    output is the epilogue applied to zeros -- e.g. C2's rows are all
    LSE_j(0.5 gelu(b_j)), C3's GroupNorm sees zero variance."""
    _torch()
    cfg = inputs.config(name, **kw)
    t = inputs.generate(cfg, seed=3)
    _, out = run_gpu(cfg, t)
    err = check(cfg, t, out)
    g = to_host_f64(out)
    assert np.all(np.isfinite(g))
    if name == "C2":
        assert np.ptp(g) == 0.0  # every row computes the same bits
    print(f"{name} K=0 err {err:.3e}")


@pytest.mark.parametrize("M,out_dtype,ops", [
    ((1 << 21) + 37, "bf16", [("bias",), ("relu",)]),
    ((1 << 20) + 37, "f32", [("bias",), ("relu",)]),
    ((1 << 21) + 37, "bf16", [("bias",), ("hardtanh", -1.0, 1.0), ("row_softmax",)]),
])
def test_output_beyond_2gib(M, out_dtype, ops):
    """An output of more than 2^31 bytes (8193+ tile rows of 520 columns):
    tile bases are 64-bit, only offsets inside a tile are 32-bit, and the
    row finishing kernel addresses rows with 64-bit offsets.  Sampled rows,
    taken from the device output before the copy to the host."""
    torch = _torch()
    cfg = inputs.config("C2", M=M, N=520, K=40, out_dtype=out_dtype, ops=ops)
    t = inputs.generate(cfg, seed=11)
    _, out = run_gpu(cfg, t)
    es = 2 if out_dtype == "bf16" else 4
    assert out.numel() * es > (1 << 31)
    rows = sample_rows(M, 40, seed=3)
    sub = out[torch.as_tensor(rows, device=out.device)]
    chain = inputs.chain_for(cfg, t)
    ref = oracle.run_chain(chain, t, rows=rows)
    from parity import floor_for
    err = parity_error(to_host_f64(sub), ref, floor_for(cfg))
    assert err <= TOL[cfg["in_dtype"]], f"parity error {err:.3e}"
    print(f"M={M} {out_dtype} {[o[0] for o in ops]} err {err:.3e}")


def test_binding_reuses_descriptors_only_for_the_same_tensors():
    """The binding reuses the last call's tensor descriptors only when every
    tensor has the same address, dtype, shape and strides: new input values
    in a new buffer, and a new output buffer, are seen by the next call."""
    torch = _torch()
    cfg = inputs.config("C2", M=300, N=520, K=136)
    t1 = inputs.generate(cfg, seed=61)
    t2 = inputs.generate(cfg, seed=62)
    op = kf.FusedOp(inputs.chain_for(cfg, t1), **kf.sizes_of(cfg))
    ins1, ins2 = op.device_inputs(t1), op.device_inputs(t2)
    o1, o2 = op.empty_output("cuda"), op.empty_output("cuda")
    op(ins1, o1)
    op(ins1, o1)  # same tensors: the descriptors are reused
    op(ins2, o2)  # other buffers: new descriptors
    op(ins1, o2)  # same inputs as the first call, other output
    torch.cuda.synchronize()
    check(cfg, t1, o1)
    check(cfg, t1, o2)
    op(ins2, o2)
    torch.cuda.synchronize()
    check(cfg, t2, o2)
    assert not torch.equal(o1, o2)


def test_repeat_runs_bitwise_identical():
    torch = _torch()
    cfg = inputs.config("C3", M=512, N=512, K=256, ops=[("groupnorm", 2, 1e-5), ("swish",), ("residual_add",)])
    t = inputs.generate(cfg, seed=2)
    op = kf.FusedOp(inputs.chain(cfg), **kf.sizes_of(cfg))
    ins = op.device_inputs(t)
    o1, o2 = op(ins), op(ins)
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))


def test_shape_mismatch_rejected_on_device():
    torch = _torch()
    cfg = inputs.config("C2", M=64, N=64, K=64)
    t = inputs.generate(cfg, seed=1)
    op = kf.FusedOp(inputs.chain(cfg), **kf.sizes_of(cfg))
    ins = op.device_inputs(t)
    bad = torch.empty((63,), dtype=torch.float32, device="cuda")
    with pytest.raises(kf.KFError) as ei:
        op(ins, bad)
    assert ei.value.status == kf.KF_ERR_SHAPE


# ------------------------------------------------------------ fp8 (OCP e4m3)

def _int_e4m3(rng, shape):
    """Integers in [-16, 16]: all exactly representable in E4M3."""
    v = rng.integers(-16, 17, size=shape).astype(np.float32)
    return v, inputs.f32_to_e4m3_codes(v)


@pytest.mark.parametrize("layout", ["kn", "nk"])
def test_fp8_contraction_bit_exact(layout):
    """Every partial sum is an integer of magnitude < 8192 * 256 = 2^21, so the
    fp32 accumulator must equal the exact product (unit scales)."""
    _torch()
    M, N, K = 2048, 8192, 8192
    rng = np.random.default_rng(31)
    a, qa = _int_e4m3(rng, (M, K))
    b, qb = _int_e4m3(rng, (K, N) if layout == "kn" else (N, K))
    t = {"a": qa, "b": qb, "scale_a": 1.0, "scale_b": 1.0}
    cfg = inputs.config("C5", M=M, N=N, K=K, out_dtype="f32", ops=[], b_layout=layout)
    print(f"fp8 bit-exact {M}x{N}x{K} {layout}", flush=True)
    _, out = run_gpu(cfg, t)
    bb = b.astype(np.float64) if layout == "kn" else b.astype(np.float64).T
    ref = a.astype(np.float64) @ bb
    assert np.array_equal(out.cpu().numpy().astype(np.float64), ref)


@pytest.mark.parametrize("M,N,K,layout", [(300, 1040, 208, "kn"), (257, 272, 64, "nk"), (1, 16, 16, "kn"),
                                          (520, 4096, 1024, "kn")])
def test_c5_ragged(M, N, K, layout):
    _torch()
    cfg = inputs.config("C5", M=M, N=N, K=K, b_layout=layout)
    t = inputs.generate(cfg, seed=M + N + K)
    _, out = run_gpu(cfg, t)
    err = check(cfg, t, out)
    g = to_host_f64(out)
    assert np.allclose(g.sum(axis=1), 1.0, atol=3e-2)
    print(f"C5 {M}x{N}x{K} {layout} err {err:.3e}")


def test_c5_zero_weights_uniform_bit_exact():
    """W = 0, b = 0: every logit is 0, so every output is 1/8192 = 2^-13,
    exactly representable in bf16."""
    torch = _torch()
    cfg = inputs.config("C5", M=256, N=8192, K=256)
    t = inputs.generate(cfg, seed=4)
    t["b"] = np.zeros_like(t["b"])
    t["bias"] = np.zeros_like(t["bias"])
    _, out = run_gpu(cfg, t)
    bits = out.view(torch.int16).cpu().numpy().view(np.uint16)
    assert np.all(bits == inputs.f32_to_bf16_bits(np.array([2.0 ** -13], np.float32))[0])


def test_c5_full_config_sampled_rows():
    _torch()
    cfg = inputs.config("C5")
    t = inputs.generate(cfg)
    _, out = run_gpu(cfg, t)
    rows = sample_rows(cfg["M"], 128)
    err = check(cfg, t, out, rows=rows)
    g = to_host_f64(out)
    assert np.all(np.isfinite(g))
    assert np.allclose(g.sum(axis=1), 1.0, atol=3e-2)
    print(f"C5 full err {err:.3e}")



# ------------------------------------------------ GEMM + activation chain (F1)

@pytest.mark.parametrize("M,N,K,in_dtype", [(300, 520, 136, "bf16"), (1, 8, 8, "bf16"), (257, 272, 64, "e4m3"),
                                            (33, 65, 31, "f32")])
def test_f1_ragged(M, N, K, in_dtype):
    _torch()
    kw = dict(M=M, N=N, K=K, in_dtype=in_dtype)
    if in_dtype == "f32":
        kw["out_dtype"] = "f32"
    if in_dtype == "e4m3":
        kw["dist"] = dict(a=("normal", 1.0), b=("normal", 1.0), bias=("uniform", -0.1, 0.1))
    cfg = inputs.config("F1", **kw)
    t = inputs.generate(cfg, seed=M + N + K)
    _, out = run_gpu(cfg, t)
    err = check(cfg, t, out)
    print(f"F1 {M}x{N}x{K} {in_dtype} err {err:.3e}")


def test_f1_full_config_sampled_rows():
    _torch()
    cfg = inputs.config("F1")
    t = inputs.generate(cfg)
    _, out = run_gpu(cfg, t)
    err = check(cfg, t, out, rows=sample_rows(cfg["M"], 48))
    print(f"F1 full err {err:.3e}")


# ------------------------------------------ row-wise chains (no contraction)

_ROW_DIST = dict(a=("normal", 1.0), bias=("uniform", -0.1, 0.1), gamma=("uniform", 0.5, 1.5),
                 beta=("uniform", -0.1, 0.1), residual=("normal", 1.0))


@pytest.mark.parametrize("M,N,ops,in_dtype,out_dtype", [
    (37, 1024, [("groupnorm", 8, 1e-5), ("swish",), ("residual_add",)], "bf16", "bf16"),  # 128-column groups
    (5, 8192, [("groupnorm", 32, 1e-5), ("swish",), ("residual_add",)], "bf16", "bf16"),  # F3 rows
    (9, 2048, [("groupnorm", 1, 1e-5)], "f32", "f32"),                                    # one group per row
    (9, 2048, [("groupnorm", 256, 1e-5), ("relu",)], "bf16", "f32"),                      # 8-column groups
    (11, 1536, [("groupnorm", 4, 1e-5), ("swish",)], "bf16", "bf16"),                     # 48-chunk groups (LDS tree)
    (7, 8192, [("groupnorm", 8, 1e-5), ("residual_add",)], "bf16", "bf16"),               # 128-chunk groups (LDS tree)
    (33, 16384, [("row_softmax",)], "bf16", "bf16"),                                      # widest row
    (3, 8, [("row_softmax",)], "f32", "f32"),                                             # narrowest row
    (70, 3000, [("bias",), ("gelu_tanh",), ("scale", 0.5), ("row_logsumexp",)], "bf16", "f32"),
    (16, 4104, [("bias",), ("tanh",), ("residual_add",), ("hardtanh", -0.5, 0.5)], "f32", "bf16"),
    (2, 1024, [], "bf16", "bf16"),                                                        # a copy
])
def test_rowwise_chains(M, N, ops, in_dtype, out_dtype):
    _torch()
    cfg = inputs.config("F3", M=M, N=N, ops=ops, in_dtype=in_dtype, out_dtype=out_dtype, dist=_ROW_DIST)
    t = inputs.generate(cfg, seed=M + N)
    op, out = run_gpu(cfg, t)
    names = [o[0] for o in ops]
    streamed = bool(names) and names[-1] in ("row_logsumexp", "row_cross_entropy")
    assert op.kernel_name() in ("kf_rowwise", "kf_rowwise_gn_panel", "kf_row_reduce_stream")
    assert (op.kernel_name() == "kf_row_reduce_stream") == streamed
    tol = TOL["bf16"] if "bf16" in (in_dtype, out_dtype) else TOL["f32"]
    err = check(cfg, t, out, tol=tol)
    print(f"rowwise {M}x{N} {[o[0] for o in ops]} err {err:.3e}")


@pytest.mark.parametrize("name", ["F3", "F4"])
def test_rowwise_full_config_sampled_rows(name):
    _torch()
    cfg = inputs.config(name)
    t = inputs.generate(cfg)
    _, out = run_gpu(cfg, t)
    err = check(cfg, t, out, rows=sample_rows(cfg["M"], 64))
    print(f"{name} full err {err:.3e}")

# ------------------------------------------------------------ conv (C4)

@pytest.mark.parametrize("batch,H,ops", [
    (2, 8, [("bias",), ("relu",), ("maxpool2x2",)]),
    (1, 2, [("bias",), ("relu",), ("maxpool2x2",)]),
    (3, 6, [("bias",), ("relu",)]),
    (1, 4, [("bias",), ("gelu_tanh",), ("maxpool2x2",), ("scale", -2.0), ("swish",)]),
])
@pytest.mark.parametrize("variant", [0, 1, 2])
def test_c4_small(batch, H, ops, variant):
    _torch()
    cfg = inputs.config("C4", batch=batch, H=H, ops=ops)
    t = inputs.generate(cfg, seed=batch * 10 + H)
    _, out = run_gpu(cfg, t, tuning=(4, 1, 2, variant))
    err = check(cfg, t, out)
    print(f"C4 batch={batch} H={H} ops={[o[0] for o in ops]} err {err:.3e}")


def test_c4_integer_bit_exact():
    """Integer inputs in [-4, 4] and weights in [-2, 2]: every fp32 partial sum
    is an exact integer, so the GPU output (no ops) equals the oracle's exact
    sum rounded to bf16 (round to nearest even), bit for bit."""
    torch = _torch()
    cfg = inputs.config("C4", batch=2, H=6, ops=[])
    rng = np.random.default_rng(41)
    x = rng.integers(-4, 5, size=(2, 64, 6, 128)).astype(np.float32)
    w = rng.integers(-2, 3, size=(128, 64, 3, 3)).astype(np.float32)
    t = {"a": inputs.f32_to_bf16_bits(x), "b": inputs.f32_to_bf16_bits(w)}
    _, out = run_gpu(cfg, t)
    ref = oracle.conv2d_3x3(x.astype(np.float64), w.astype(np.float64))
    assert np.all(np.abs(ref) < 2 ** 24) and np.array_equal(ref, np.round(ref))
    ref_bits = inputs.f32_to_bf16_bits(ref.astype(np.float32))
    got_bits = out.view(torch.int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(got_bits, ref_bits)


def test_c4_integer_bit_exact_full_batch():
    """The integer test at C4's full size (64 images of 64 x 128 x 128, 4096
    row-pair tiles), eight images checked bit for bit."""
    torch = _torch()
    cfg = inputs.config("C4", ops=[])
    rng = np.random.default_rng(43)
    x = rng.integers(-4, 5, size=(64, 64, 128, 128)).astype(np.float32)
    w = rng.integers(-2, 3, size=(128, 64, 3, 3)).astype(np.float32)
    t = {"a": inputs.f32_to_bf16_bits(x), "b": inputs.f32_to_bf16_bits(w)}
    print("C4 integer bit-exact, full batch", flush=True)
    _, out = run_gpu(cfg, t)
    imgs = np.array([0, 9, 21, 32, 40, 51, 62, 63])
    ref = oracle.conv2d_3x3(x[imgs].astype(np.float64), w.astype(np.float64))
    ref_bits = inputs.f32_to_bf16_bits(ref.astype(np.float32))
    got_bits = out.view(torch.int16).cpu().numpy().view(np.uint16)[imgs]
    assert np.array_equal(got_bits, ref_bits)


def test_c4_zero_weights_and_centre_tap():
    _torch()
    cfg = inputs.config("C4", batch=1, H=4)
    t = inputs.generate(cfg, seed=3)
    z = dict(t, b=np.zeros_like(t["b"]))
    _, out = run_gpu(cfg, z)
    g = to_host_f64(out)
    expect = np.maximum(t["bias"].astype(np.float64), 0)[None, :, None, None]
    assert np.max(np.abs(g - expect)) <= 2.0 ** -8 * np.max(np.abs(expect))
    w = np.zeros((128, 64, 3, 3), np.float32)
    for c in range(64):
        w[c, c, 1, 1] = 1.0
    t2 = dict(t, b=inputs.f32_to_bf16_bits(w))
    _, out = run_gpu(cfg, t2)
    check(cfg, t2, out)


@pytest.mark.parametrize("variant", [0, 1])
def test_c4_full_config_sampled_images(variant):
    _torch()
    cfg = inputs.config("C4")
    t = inputs.generate(cfg)
    _, out = run_gpu(cfg, t, tuning=(4, 1, 2, variant))
    err = check(cfg, t, out, images=np.array([0, 5, 19, 26, 37, 44, 58, 63]))
    assert np.all(np.isfinite(to_host_f64(out)))
    print(f"C4 full err {err:.3e}")



@pytest.mark.parametrize("batch,H,ops", [
    (5, 120, [("bias",), ("relu",), ("maxpool2x2",)]),   # 300 row-pair tiles, 60 per image
    (3, 200, [("bias",), ("relu",)]),                    # unpooled
])
@pytest.mark.parametrize("variant", [0, 1])
def test_c4_tile_ranges(batch, H, ops, variant):
    """More tiles than workgroups: each workgroup walks a contiguous range of
    row pairs, reusing two halo rows from one tile to the next and reloading
    all four at the start of an image; ranges here cross image boundaries."""
    _torch()
    cfg = inputs.config("C4", batch=batch, H=H, ops=ops)
    t = inputs.generate(cfg, seed=batch + H)
    _, out = run_gpu(cfg, t, tuning=(4, 1, 2, variant))
    err = check(cfg, t, out, images=np.arange(batch))
    print(f"C4 batch={batch} H={H} err {err:.3e}")


@pytest.mark.parametrize("variant", [0, 1, 2])
def test_c4_integer_bit_exact_tile_ranges(variant):
    """The integer test of the contraction with several tiles per workgroup,
    on the 4-wave and the 8-wave tile and on the general kernel."""
    torch = _torch()
    batch, H = 3, 200
    cfg = inputs.config("C4", batch=batch, H=H, ops=[])
    rng = np.random.default_rng(43)
    x = rng.integers(-4, 5, size=(batch, 64, H, 128)).astype(np.float32)
    w = rng.integers(-2, 3, size=(128, 64, 3, 3)).astype(np.float32)
    t = {"a": inputs.f32_to_bf16_bits(x), "b": inputs.f32_to_bf16_bits(w)}
    _, out = run_gpu(cfg, t, tuning=(4, 1, 2, variant))
    got_bits = out.view(torch.int16).cpu().numpy().view(np.uint16)
    for n in range(batch):
        ref = oracle.conv2d_3x3(x[n:n + 1].astype(np.float64), w.astype(np.float64))
        assert np.array_equal(got_bits[n:n + 1], inputs.f32_to_bf16_bits(ref.astype(np.float32))), f"image {n}"

# ------------------------------------------------ conv, general shapes

@pytest.mark.parametrize("batch,cin,H,W,cout,ops", [
    (2, 3, 9, 50, 40, [("bias",), ("relu",)]),                       # odd height, ragged width, few channels
    (1, 32, 8, 64, 96, [("bias",), ("relu",), ("maxpool2x2",)]),      # cout not a multiple of 128
    (2, 16, 6, 34, 128, [("bias",), ("gelu_tanh",), ("maxpool2x2",)]),  # width not a multiple of 32
    (1, 64, 5, 33, 160, [("bias",)]),                                 # two channel tiles, the last partial
    (1, 130, 4, 20, 32, [("bias",), ("relu",), ("maxpool2x2",), ("scale", 0.5)]),  # cin not a multiple of 16
    (3, 1, 1, 1, 1, []),                                              # one pixel, one channel
])
def test_conv_general_shapes(batch, cin, H, W, cout, ops):
    """Shapes outside the tiled kernels' family run the general kernel."""
    _torch()
    cfg = inputs.config("C4", batch=batch, cin=cin, H=H, W=W, cout=cout, ops=ops)
    t = inputs.generate(cfg, seed=batch + cin + H + W + cout)
    op, out = run_gpu(cfg, t)
    assert op.kernel_name() == "kf_conv3x3_bf16_gen"
    err = check(cfg, t, out)
    print(f"conv general {batch}x{cin}x{H}x{W} -> {cout} err {err:.3e}")


def test_conv_general_integer_bit_exact():
    """Integer inputs and weights: every partial sum is exact, so the general
    kernel's output is the exact convolution rounded once to bf16."""
    torch = _torch()
    batch, cin, H, W, cout = 2, 48, 6, 40, 72
    cfg = inputs.config("C4", batch=batch, cin=cin, H=H, W=W, cout=cout, ops=[])
    rng = np.random.default_rng(44)
    x = rng.integers(-4, 5, size=(batch, cin, H, W)).astype(np.float32)
    w = rng.integers(-2, 3, size=(cout, cin, 3, 3)).astype(np.float32)
    t = {"a": inputs.f32_to_bf16_bits(x), "b": inputs.f32_to_bf16_bits(w)}
    _, out = run_gpu(cfg, t)
    ref = oracle.conv2d_3x3(x.astype(np.float64), w.astype(np.float64))
    got = out.view(torch.int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(got, inputs.f32_to_bf16_bits(ref.astype(np.float32)))


def test_conv_general_unfused_and_tuning():
    """The unfused chain of a general-shape conv, and the tuning rule: a
    general-shape plan runs only the general kernel (variant 2)."""
    _torch()
    cfg = inputs.config("C4", batch=2, cin=24, H=10, W=30, cout=64)
    t = inputs.generate(cfg, seed=12)
    op, out = run_gpu(cfg, t, unfused=True)
    check(cfg, t, out, unfused=True)
    assert op.tuning()["variant"] == 2
    with pytest.raises(kf.KFError):
        op.set_tuning(4, 1, 2, 1)


# ------------------------------------------- Conv3d, channel softmax, pools (F2)

_F2_OPS = [("bias",), ("channel_softmax",), ("maxpool3d2",), ("maxpool3d2",)]


@pytest.mark.parametrize("batch,D,H,W,ops", [
    (2, 7, 11, 20, _F2_OPS),            # ragged: 5 x 9 x 18 conv positions, 1 x 2 x 4 pooled cells
    (1, 6, 10, 18, _F2_OPS),            # one exact 4 x 8 x 16 tile
    (3, 9, 19, 35, _F2_OPS),            # 7 x 17 x 33: partial tiles in every axis
    (2, 7, 11, 20, []),                 # the conv alone, every position (ragged rows of 18)
    (1, 10, 12, 34, [("bias",), ("channel_softmax",)]),  # softmax, no pools, rows of 32
    (2, 7, 11, 20, [("bias",), ("sigmoid",), ("channel_softmax",), ("scale", 2.0), ("maxpool3d2",), ("maxpool3d2",)]),
])
def test_f2_small(batch, D, H, W, ops):
    _torch()
    cfg = inputs.config("F2", batch=batch, D=D, H=H, W=W, ops=ops)
    t = inputs.generate(cfg, seed=batch + D + H + W)
    _, out = run_gpu(cfg, t)
    assert tuple(out.shape) == inputs.conv3d_pooled_shape(cfg)
    err = check(cfg, t, out)
    print(f"F2 {batch}x{D}x{H}x{W} ops={[o[0] for o in ops]} err {err:.3e}")


_CONV3D_GEN_DIST = dict(a=("normal", 1.0), b=("normal_invk",), bias=("uniform", -0.1, 0.1))


@pytest.mark.parametrize("batch,cin,cout,D,H,W,ops,cl", [
    (2, 8, 32, 5, 9, 20, [("bias",)], True),                        # small channel counts, one partial tile
    (1, 24, 96, 4, 12, 40, [("bias",), ("gelu_erf",)], False),      # NCDHW input, cin past one 16-chunk
    (2, 40, 160, 3, 7, 35, [("bias",), ("relu",), ("scale", 0.5)], True),  # two channel tiles, ragged
    (1, 16, 64, 6, 10, 18, [("bias",), ("tanh",)], False),          # the tiled family's shape, NCDHW input
    (1, 3, 5, 3, 3, 3, [], False),                                  # one output position
])
def test_conv3d_general_shapes(batch, cin, cout, D, H, W, ops, cl):
    """The general Conv3d kernel: any channel counts and extents, input
    channels-last or contiguous NCDHW, bias and element-wise ops fused."""
    _torch()
    cfg = inputs.config("F2", batch=batch, cin=cin, cout=cout, D=D, H=H, W=W, ops=ops, dist=_CONV3D_GEN_DIST)
    t = inputs.generate(cfg, seed=cin + cout + D)
    op = kf.FusedOp(inputs.chain_for(cfg, t), **kf.sizes_of(cfg))
    if (cin, cout) != (16, 64):
        assert op.kernel_name() == "kf_conv3d_bf16_gen"
    ins = op.device_inputs(t, conv3d_channels_last=cl)
    out = op.empty_output("cuda")
    op(ins, out)
    err = check(cfg, t, out)
    out2 = op.empty_output("cuda")
    op.unfused(ins, out2)
    check(cfg, t, out2, unfused=True)
    print(f"conv3d general {batch}x{cin}->{cout} {D}x{H}x{W} cl={cl} err {err:.3e}")


@pytest.mark.parametrize("cl", [True, False])
def test_conv3d_general_integer_bit_exact(cl):
    """Integer inputs and weights: every partial sum is an exact integer, so
    the general kernel's output (no ops) is the exact sum rounded to bf16."""
    torch = _torch()
    batch, cin, cout, D, H, W = 2, 40, 136, 5, 11, 37
    cfg = inputs.config("F2", batch=batch, cin=cin, cout=cout, D=D, H=H, W=W, ops=[])
    rng = np.random.default_rng(45)
    x = rng.integers(-4, 5, size=(batch, cin, D, H, W)).astype(np.float32)
    w = rng.integers(-2, 3, size=(cout, cin, 3, 3, 3)).astype(np.float32)
    t = {"a": inputs.f32_to_bf16_bits(x), "b": inputs.f32_to_bf16_bits(w)}
    op = kf.FusedOp(inputs.chain_for(cfg, t), **kf.sizes_of(cfg))
    ins = op.device_inputs(t, conv3d_channels_last=cl)
    out = op.empty_output("cuda")
    op(ins, out)
    ref = oracle.conv3d_3x3x3(x.astype(np.float64), w.astype(np.float64))
    got = out.view(torch.int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(got, inputs.f32_to_bf16_bits(ref.astype(np.float32)))


def test_conv3d_family_layouts():
    """The tiled family's shape with the F2 chain: a channels-last input runs
    the tiled kernel, the whole chain fused; a contiguous NCDHW input runs
    partly fused (the general kernel with the bias, then the channel softmax
    and the pools one kernel each) and gives the partly fused oracle's
    result."""
    torch = _torch()
    cfg = inputs.config("F2", batch=1, D=6, H=10, W=18)
    t = inputs.generate(cfg, seed=5)
    op = kf.FusedOp(inputs.chain_for(cfg, t), **kf.sizes_of(cfg))
    out = op.empty_output("cuda")
    op(op.device_inputs(t), out)
    check(cfg, t, out)
    ins = op.device_inputs(t, conv3d_channels_last=False)
    assert ins[0].is_contiguous()
    out2 = op.empty_output("cuda")
    op(ins, out2)
    torch.cuda.synchronize()
    err = check(cfg, t, out2, fused=1)
    # and back: the tiled kernel's packed weights are restored
    out3 = op.empty_output("cuda")
    op(op.device_inputs(t), out3)
    assert torch.equal(out3.view(torch.int16), out.view(torch.int16))
    print(f"F2 NCDHW partly fused err {err:.3e}")


_F2_SPLIT = [("bias",), ("sigmoid",), ("channel_softmax",), ("scale", 2.0), ("maxpool3d2",), ("maxpool3d2",)]


@pytest.mark.parametrize("batch,cin,cout,D,H,W,ops,cl,prefix", [
    (2, 24, 96, 7, 11, 20, _F2_OPS, True, 1),          # general shape, channels-last
    (1, 40, 160, 7, 9, 37, _F2_SPLIT, False, 2),       # two channel tiles, NCDHW, ragged pools
    (2, 8, 32, 4, 6, 9, [("channel_softmax",)], True, 0),  # the softmax straight after the conv
    (1, 16, 64, 6, 10, 18, _F2_SPLIT, False, 2),       # the tiled family's shape, NCDHW input
])
def test_conv3d_partly_fused_chains(batch, cin, cout, D, H, W, ops, cl, prefix):
    """Outside the tiled kernel's family a Conv3d chain with a channel softmax
    or pools runs partly fused: the general kernel with the leading bias and
    element-wise ops, then one kernel per remaining op through bf16
    intermediates.  Compared with the oracle of that evaluation, and the
    unfused chain with the unfused oracle."""
    torch = _torch()
    cfg = inputs.config("F2", batch=batch, cin=cin, cout=cout, D=D, H=H, W=W, ops=ops, dist=_CONV3D_GEN_DIST)
    t = inputs.generate(cfg, seed=cin + D)
    op = kf.FusedOp(inputs.chain_for(cfg, t), **kf.sizes_of(cfg))
    ins = op.device_inputs(t, conv3d_channels_last=cl)
    print(f"[gpu] conv3d partly fused {batch}x{cin}->{cout} {D}x{H}x{W} cl={cl} prefix={prefix}", flush=True)
    out = op.empty_output("cuda")
    op(ins, out)
    torch.cuda.synchronize()
    assert tuple(out.shape) == inputs.conv3d_pooled_shape(cfg)
    err = check(cfg, t, out, fused=prefix)
    out2 = op.empty_output("cuda")
    op.unfused(ins, out2)
    check(cfg, t, out2, unfused=True)
    print(f"conv3d partly fused err {err:.3e}")


def test_f2_degenerate_shapes():
    """3x3x3 volumes (one conv position: no pooled cell) and an empty batch
    produce empty outputs without a launch."""
    _torch()
    for batch, D in [(2, 3), (0, 8)]:
        cfg = inputs.config("F2", batch=batch, D=D, H=8, W=8)
        t = inputs.generate(cfg, seed=5)
        _, out = run_gpu(cfg, t)
        assert out.numel() == 0


def test_f2_integer_bit_exact_many_tiles():
    """Integer inputs in [-4, 4] and weights in [-2, 2], no ops: every fp32
    partial sum is an exact integer (|sum| <= 432 * 8), so the stored conv
    output equals the oracle's exact sum rounded to bf16, bit for bit; 512
    tiles, two per workgroup, across image boundaries."""
    torch = _torch()
    batch, D, H, W = 8, 18, 34, 66
    cfg = inputs.config("F2", batch=batch, D=D, H=H, W=W, ops=[])
    rng = np.random.default_rng(45)
    x = rng.integers(-4, 5, size=(batch, 16, D, H, W)).astype(np.float32)
    w = rng.integers(-2, 3, size=(64, 16, 3, 3, 3)).astype(np.float32)
    t = {"a": inputs.f32_to_bf16_bits(x), "b": inputs.f32_to_bf16_bits(w)}
    _, out = run_gpu(cfg, t)
    ref = oracle.conv3d_3x3x3(x.astype(np.float64), w.astype(np.float64))
    assert np.all(np.abs(ref) < 2 ** 24) and np.array_equal(ref, np.round(ref))
    ref_bits = inputs.f32_to_bf16_bits(ref.astype(np.float32))
    got_bits = out.view(torch.int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(got_bits, ref_bits)


def test_f2_zero_weights_uniform_bit_exact():
    """W = 0, b = 0: every softmax is uniform, so every pooled cell is 1/64
    exactly."""
    torch = _torch()
    cfg = inputs.config("F2", batch=2, D=10, H=18, W=34)
    t = inputs.generate(cfg, seed=9)
    z = dict(t, b=np.zeros_like(t["b"]), bias=np.zeros_like(t["bias"]))
    _, out = run_gpu(cfg, z)
    assert torch.all(out.float() == 1.0 / 64).item()


def test_f2_full_config_sampled_images():
    _torch()
    cfg = inputs.config("F2")
    t = inputs.generate(cfg)
    _, out = run_gpu(cfg, t)
    assert np.all(np.isfinite(to_host_f64(out)))
    err = check(cfg, t, out, images=np.array([0, 7, 15]))
    print(f"F2 full err {err:.3e}")


# ------------------------------------------------------------ unfused chain

@pytest.mark.parametrize("name,kw", [
    ("C1", {}),
    ("C2", dict(M=300, N=520, K=136)),
    ("C3", dict(M=300, N=512, K=136, ops=[("groupnorm", 2, 1e-5), ("swish",), ("residual_add",)])),
    ("C4", dict(batch=2, H=8)),
    ("C5", dict(M=300, N=1040, K=208)),
    ("F1", dict(M=300, N=520, K=136)),
    ("F3", dict(M=37, N=1024, ops=[("groupnorm", 8, 1e-5), ("swish",), ("residual_add",)])),
    ("F4", dict(M=9, N=2048)),
    ("F2", dict(batch=2, D=7, H=11, W=20)),
    ("F5", dict(M=37, N=2056)),
    ("F6", dict(M=300, N=1040, K=136)),
])
def test_unfused_chain_parity(name, kw):
    """The one-kernel-per-op comparator computes the same chain with every
    intermediate stored in bf16 (fp32 for fp32 chains), as an eager chain
    stores it; it is held to the same tolerance as the fused kernels against
    the oracle's evaluation that rounds the intermediates at the same
    places."""
    _torch()
    cfg = inputs.config(name, **kw)
    t = inputs.generate(cfg, seed=77)
    _, out = run_gpu(cfg, t, unfused=True)
    err = check(cfg, t, out, unfused=True)
    print(f"unfused {name} err {err:.3e}")


@pytest.mark.parametrize("name,kw", [
    ("C3", dict(M=300, N=2048, K=136, ops=[("groupnorm", 8, 1e-5), ("swish",), ("residual_add",)])),
    ("C5", dict(M=300, N=1040, K=208)),
    ("F1", dict(M=77, N=1024, K=64)),
    ("F2", dict(batch=2, D=10, H=11, W=34)),
    ("F2", dict(batch=3, D=7, H=13, W=34)),   # 1760 positions: a partial last tile of the channel softmax
    ("F3", dict(M=40, N=8192)),
])
def test_unfused_chain_vector_kernels(name, kw):
    """Shapes whose intermediates take the vectorised per-op kernels (rows of
    whole 16-byte chunks, group-aligned GroupNorm, pooled rows of 16 columns)
    -- the paths the full-size workloads run -- against the same oracle."""
    _torch()
    cfg = inputs.config(name, **kw)
    t = inputs.generate(cfg, seed=78)
    _, out = run_gpu(cfg, t, unfused=True)
    err = check(cfg, t, out, unfused=True)
    print(f"unfused {name} err {err:.3e}")


@pytest.mark.parametrize("name", ["C2", "C3", "C5"])
def test_unfused_full_config_sampled_rows(name):
    _torch()
    cfg = inputs.config(name)
    t = inputs.generate(cfg)
    _, out = run_gpu(cfg, t, unfused=True)
    err = check(cfg, t, out, rows=sample_rows(cfg["M"], 16), unfused=True)
    print(f"unfused {name} full err {err:.3e}")


def test_unfused_c4_full_config_sampled_images():
    _torch()
    cfg = inputs.config("C4")
    t = inputs.generate(cfg)
    _, out = run_gpu(cfg, t, unfused=True)
    err = check(cfg, t, out, images=np.array([0, 63]), unfused=True)
    print(f"unfused C4 full err {err:.3e}")


# ------------------------------------------------- epilogue operand paths

_ALL_DIST = dict(a=("normal", 1.0), b=("normal_invk",), bias=("uniform", -0.1, 0.1),
                 gamma=("uniform", 0.5, 1.5), beta=("uniform", -0.1, 0.1), residual=("normal", 1.0))


@pytest.mark.parametrize("name,kw,res_f32", [
    # residual in a plain epilogue, ragged M and N (tile tails), bf16 and fp32 residual
    ("C2", dict(M=300, N=520, K=136, out_dtype="bf16", ops=[("bias",), ("residual_add",), ("relu",)]), False),
    ("C2", dict(M=300, N=520, K=136, out_dtype="bf16", ops=[("bias",), ("residual_add",), ("relu",)]), True),
    # residual before the GroupNorm statistics, 256-wide groups across both waves
    ("C3", dict(M=260, N=512, K=64, ops=[("bias",), ("residual_add",), ("groupnorm", 2, 1e-5), ("swish",)]), False),
    # residual feeding a row softmax, columns past N masked out
    ("C2", dict(M=77, N=520, K=40, out_dtype="bf16", ops=[("bias",), ("residual_add",), ("row_softmax",)]), False),
    # fp8 contraction with a residual
    ("C5", dict(M=300, N=528, K=160, ops=[("bias",), ("residual_add",), ("hardtanh", -1.0, 1.0)]), False),
    # NK layout with every column vector present
    ("C3", dict(M=100, N=256, K=48, b_layout="nk", ops=[("bias",), ("groupnorm", 1, 1e-5), ("residual_add",)]), False),
])
def test_epilogue_operand_paths(name, kw, res_f32):
    _torch()
    cfg = inputs.config(name, dist=_ALL_DIST, residual_dtype="f32" if res_f32 else "bf16", **kw)
    t = inputs.generate(cfg, seed=21)
    if res_f32:
        t["residual"] = oracle.decode_bf16(t["residual"]).astype(np.float32) * np.float32(1.25)
    _, out = run_gpu(cfg, t)
    err = check(cfg, t, out)
    print(f"{name} {kw['ops']} err {err:.3e}")


@pytest.mark.parametrize("name,kw", [
    # K-step counts that are multiples of four (the pipeline's four stages
    # end aligned): nk = 4 fills every stage once, nk = 12 loops
    ("C3", dict(M=300, N=512, K=128, ops=[("groupnorm", 2, 1e-5), ("swish",), ("residual_add",)])),
    ("C3", dict(M=300, N=1024, K=384, ops=[("groupnorm", 8, 1e-5), ("swish",), ("residual_add",)])),
    # interpreted plain epilogue, ragged N (a last column tile of 8 columns)
    ("C2", dict(M=300, N=520, K=256, out_dtype="bf16", ops=[("bias",), ("residual_add",), ("relu",)])),
    # residual before the GroupNorm statistics
    ("C3", dict(M=260, N=512, K=256, ops=[("bias",), ("residual_add",), ("groupnorm", 2, 1e-5), ("swish",)])),
    # residual feeding a row softmax
    ("C2", dict(M=77, N=520, K=128, out_dtype="bf16", ops=[("bias",), ("residual_add",), ("row_softmax",)])),
    # fp8 (64 k per K-step): nk = 4
    ("C5", dict(M=300, N=528, K=256, ops=[("bias",), ("residual_add",), ("hardtanh", -1.0, 1.0)])),
    # B in NK layout
    ("C3", dict(M=100, N=256, K=128, b_layout="nk", ops=[("bias",), ("groupnorm", 1, 1e-5), ("residual_add",)])),
])
def test_residual_aligned_k_steps(name, kw):
    """A bf16 residual with a K-step count that is a multiple of four (no
    partial pipeline round at the end) gives the oracle's result on ragged
    tiles, and the same bits under both store paths of the 256x256 tile and
    with the 128x256 tile."""
    torch = _torch()
    cfg = inputs.config(name, dist=_ALL_DIST, residual_dtype="bf16", **kw)
    t = inputs.generate(cfg, seed=33)
    op = kf.FusedOp(inputs.chain_for(cfg, t), **kf.sizes_of(cfg))
    ins = op.device_inputs(t)
    ref = op.empty_output("cuda")
    op.set_tuning(4, 1, 2, 0)
    op(ins, ref)
    torch.cuda.synchronize()
    err = check(cfg, t, ref)
    print(f"{name} {kw['ops']} K={kw['K']} err {err:.3e}")
    variants = (2, 1) if cfg.get("b_layout", "kn") == "kn" else (2,)
    for v in variants:
        op.set_tuning(4, 1, 2, v)
        out = op.empty_output("cuda")
        op(ins, out)
        torch.cuda.synchronize()
        assert torch.equal(ref.view(torch.int16), out.view(torch.int16)), (name, v)


@pytest.mark.parametrize("ops,tol", [
    ([("tanh",), ("gelu_erf",)], 1e-6),   # input from a tanh: the polynomial form
    ([("gelu_erf",)], 3e-6),              # general input: the rational erf approximation
    ([("tanh",), ("relu",), ("gelu_erf",)], 3e-6),  # not right after the tanh: general form
])
def test_gelu_erf_accuracy_on_device(ops, tol):
    """The epilogue's GELU(erf) against the exact function of the device's own
    fp32 contraction output: the same inputs run once with no ops and once
    with the ops, and the exact (fp64, math.erf) ops applied to the first
    output must match the second to `tol` (fp32 rounding of tanh and GELU)."""
    import math
    _torch()
    cfg0 = inputs.config("F1", M=256, N=512, K=64, out_dtype="f32", ops=[])
    t = inputs.generate(cfg0, seed=71)
    _, h = run_gpu(cfg0, t)
    cfg1 = inputs.config("F1", M=256, N=512, K=64, out_dtype="f32", ops=ops)
    _, y = run_gpu(cfg1, {k: t[k] for k in ("a", "b")})
    x = to_host_f64(h)
    for o in ops:
        if o[0] == "tanh":
            x = np.tanh(x)
        elif o[0] == "relu":
            x = np.maximum(x, 0.0)
        else:
            x = 0.5 * x * (1.0 + np.vectorize(math.erf)(x / math.sqrt(2.0)))
    err = float(np.max(np.abs(to_host_f64(y) - x)))
    print(f"[gpu] gelu_erf {[o[0] for o in ops]} max |err| {err:.3e} (|h| up to {np.max(np.abs(to_host_f64(h))):.2f})")
    assert err < tol, err


@pytest.mark.parametrize("name,kw", [
    # a row reduction right after a HARDTANH with bounds at most 64 apart takes
    # the upper bound as the row offset (one pass, no max exchange)
    ("C5", dict(M=300, N=1040, K=128, ops=[("bias",), ("hardtanh", -30.0, 30.0), ("row_softmax",)])),
    ("C5", dict(M=300, N=1040, K=128, ops=[("bias",), ("hardtanh", -0.25, 0.5), ("row_softmax",)])),
    # wider bounds: planned on the interpreted epilogue with the tile-row max
    ("C5", dict(M=300, N=1040, K=128, ops=[("bias",), ("hardtanh", -100.0, 100.0), ("row_softmax",)])),
    # interpreted chains with the bounded offset
    ("C5", dict(M=300, N=1040, K=128, ops=[("bias",), ("scale", 4.0), ("hardtanh", -2.0, 2.0), ("row_softmax",)])),
    ("C2", dict(M=200, N=1040, K=96, ops=[("bias",), ("hardtanh", -4.0, 4.0), ("row_logsumexp",)])),
    ("F6", dict(M=200, N=1040, K=96, ops=[("bias",), ("hardtanh", -3.0, 3.0), ("row_cross_entropy",)])),
])
def test_row_reduction_after_hardtanh(name, kw):
    """Row softmax / logsumexp / cross-entropy after a HARDTANH, with bounds
    narrow enough for the one-pass offset and too wide for it, compiled and
    interpreted, ragged N: the oracle's result."""
    _torch()
    cfg = inputs.config(name, **kw)
    t = inputs.generate(cfg, seed=77)
    _, out = run_gpu(cfg, t)
    err = check(cfg, t, out)
    print(f"[gpu] {name} {kw['ops']} err {err:.3e}")


# ------------------------------------- specialised vs interpreted epilogues

@pytest.mark.parametrize("name,kw", [
    ("C2", dict(M=300, N=520, K=136)),                                     # bias, GELU(tanh), scale, logsumexp
    ("C3", dict(M=300, N=512, K=136, ops=[("groupnorm", 2, 1e-5), ("swish",), ("residual_add",)])),
    ("C5", dict(M=300, N=528, K=160)),                                     # fp8, bias, hardtanh, softmax
    ("C4", dict(batch=2, H=10)),                                           # conv, bias, ReLU, pool (pool first)
    ("F1", dict(M=300, N=520, K=136)),                                     # bias, swish, tanh, GELU(erf), hardtanh
    ("F3", dict(M=37, N=2048)),                                            # rows: GroupNorm, swish, residual
    ("F4", dict(M=37, N=4104)),                                            # rows: softmax
    ("F2", dict(batch=2, D=7, H=11, W=20)),                                # conv3d, bias, softmax, pools
    ("F5", dict(M=37, N=4104)),                                            # rows: cross-entropy
    ("F6", dict(M=300, N=1040, K=136)),                                    # GEMM, bias, cross-entropy
])
def test_specialised_chain_matches_interpreted(name, kw):
    """The benchmarked op lists run an epilogue generated for that exact
    chain; prefixing a scale by 1.0 (exact) makes the same list run through
    the interpreted epilogue.  Both must agree bit for bit, and the conv one
    shows that pooling before the monotone bias and ReLU changes nothing."""
    torch = _torch()
    cfg = inputs.config(name, **kw)
    t = inputs.generate(cfg, seed=31)
    _, out_spec = run_gpu(cfg, t)
    cfg2 = dict(cfg, ops=[("scale", 1.0)] + list(cfg["ops"]))
    _, out_gen = run_gpu(cfg2, t)
    a, b = out_spec, out_gen
    if a.dtype == torch.bfloat16:
        a, b = a.view(torch.int16), b.view(torch.int16)
    assert torch.equal(a, b), f"{name}: specialised and interpreted epilogues differ"
    check(cfg, t, out_spec)


# ------------------------------------------------- launch tuning, diagnosis

@pytest.mark.parametrize("name,kw", [
    ("C3", dict(M=1024, N=1024, K=136, ops=[("groupnorm", 4, 1e-5), ("swish",), ("residual_add",)])),  # 16 tiles
    ("C5", dict(M=1024, N=2048, K=128)),                                  # fp8, softmax rows across 8 column tiles
    ("F2", dict(batch=3, D=9, H=19, W=35)),                               # conv3d, partial tiles
    ("C4", dict(batch=3, H=10)),                                          # conv: 4- and 8-wave tiles
    ("C4", dict(batch=2, H=8, ops=[("bias",), ("swish",)])),              # unpooled, interpreted epilogue
    ("C2", dict(M=300, N=1040, K=200)),                                   # ragged GEMM, logsumexp rows
    ("F1", dict(M=520, N=776, K=136)),                                    # activation chain
    ("F6", dict(M=260, N=1040, K=72)),                                    # cross-entropy rows
    ("C3", dict(M=300, N=512, K=72, ops=[("groupnorm", 2, 1e-5), ("swish",), ("residual_add",)])),
    ("C2", dict(M=600, N=520, K=64, ops=[("bias",), ("sigmoid",), ("row_softmax",)], out_dtype="bf16")),  # interpreted
    ("F1", dict(M=300, N=520, K=64, out_dtype="f32")),                    # fp32 tile: variant 2 stores from registers
    ("C5", dict(M=520, N=1040, K=128, b_layout="nk")),                    # B in NK layout: variants 0 and 2 only
    ("C3", dict(M=260, N=512, K=64, b_layout="nk",
                ops=[("groupnorm", 2, 1e-5), ("swish",), ("residual_add",)])),  # staged stores over the residual rows
])
def test_tuning_candidates_bit_identical(name, kw):
    """Every launch configuration the tuner may pick computes the same bits:
    the fields only reorder independent tiles, resize a persistent grid, or
    change the tile shape (GEMM 256x256 or 128x256, conv 4 or 8 waves) with
    each output's sum over k in the same order, or the path of the stores
    (GEMM variant 2: through LDS)."""
    torch = _torch()
    cfg = inputs.config(name, **kw)
    t = inputs.generate(cfg, seed=51)
    op = kf.FusedOp(inputs.chain_for(cfg, t), **kf.sizes_of(cfg))
    ins = op.device_inputs(t)
    ref = op.empty_output("cuda")
    op(ins, ref)
    kn = cfg.get("b_layout", "kn") == "kn"
    configs = ([(4, r, w, 0) for r in (1, 0) for w in (2, 1)] if name == "F2" else
               [(4, 1, 2, v) for v in (1, 0)] if name == "C4" else
               [(g, r, 2, v) for v in (0, 2) for r in (1, 0) for g in (1, 2, 4, 8, 16, 32, 64)] +
               ([(4, 1, 2, 1)] if kn else []))
    for g, r, w, v in configs:
        op.set_tuning(g, r, w, v)
        out = op.empty_output("cuda")
        op(ins, out)
        a, b = (ref, out) if ref.dtype != torch.bfloat16 else (ref.view(torch.int16), out.view(torch.int16))
        assert torch.equal(a, b), (name, g, r, w, v)
    check(cfg, t, ref)


@pytest.mark.parametrize("name", ["C2", "C3", "C4", "C5", "F1", "F2"])
def test_full_size_tuned_launch_bit_identical(name):
    """At the full workload size, the launch configuration the bench keeps
    (by autotuning, as the bench does) and every other candidate compute the
    same bits as the default configuration, whose output is compared with the
    oracle on sampled rows (or images) here and in the full-size tests."""
    torch = _torch()
    cfg = inputs.config(name)
    t = inputs.generate(cfg)
    op = kf.FusedOp(inputs.chain_for(cfg, t), **kf.sizes_of(cfg))
    ins = op.device_inputs(t)
    ref = op.empty_output("cuda")
    op(ins, ref)
    bits = (lambda x: x.view(torch.int16)) if ref.dtype == torch.bfloat16 else (lambda x: x)
    out = op.empty_output("cuda")
    r = op.autotune(ins, out, reps=1)
    assert torch.equal(bits(ref), bits(out)), (name, r["best"])
    for c in r["candidates"]:
        op.set_tuning(c["raster_group"], c["xcd_remap"], c["wg_per_cu"], c["variant"])
        out.zero_()
        op(ins, out)
        assert torch.equal(bits(ref), bits(out)), (name, c)
    if cfg["contraction"] in ("conv3d_3x3x3", "conv2d_3x3"):
        check(cfg, t, ref, images=np.array([0, cfg["batch"] - 1]))
    else:
        check(cfg, t, ref, rows=sample_rows(cfg["M"], 8, seed=4))
    print(f"{name}: {len(r['candidates'])} candidates bit-identical at full size, kept {r['best']}")


@pytest.mark.parametrize("name,kw,n", [
    ("C2", dict(M=1024, N=2048, K=512), 29),
    ("F2", dict(batch=2, D=10, H=18, W=34), 4),
    ("F4", dict(M=256, N=2048), 1),
    ("C4", dict(batch=8, H=16), 2),
])
def test_autotune_keeps_the_fastest_candidate(name, kw, n):
    _torch()
    cfg = inputs.config(name, **kw)
    t = inputs.generate(cfg, seed=52)
    op = kf.FusedOp(inputs.chain_for(cfg, t), **kf.sizes_of(cfg))
    ins = op.device_inputs(t)
    out = op.empty_output("cuda")
    r = op.autotune(ins, out, reps=3)
    assert len(r["candidates"]) == n
    assert all(c["seconds"] > 0 for c in r["candidates"])
    fastest = min(c["seconds"] for c in r["candidates"])
    if name in ("C2", "C3", "C5", "F1"):
        # GEMMs: the fewest modelled panel bytes among the candidates within 2% of the fastest
        near = [c for c in r["candidates"] if c["seconds"] <= fastest * 1.02]
        assert r["best"]["seconds"] <= fastest * 1.02
        assert r["best"]["panel_bytes"] == min(c["panel_bytes"] for c in near)
    else:
        assert r["best"]["seconds"] == fastest
        assert all(c["panel_bytes"] == -1 for c in r["candidates"])
    best = {k: r["best"][k] for k in ("raster_group", "xcd_remap", "wg_per_cu", "variant")}
    assert op.tuning() == best
    check(cfg, t, out)
    out2 = op.empty_output("cuda")
    op(ins, out2)
    check(cfg, t, out2)
    with pytest.raises(kf.KFError):
        op.set_tuning(0, 1, 2)


def test_gemm_tuning_variants_validated():
    """GEMM plans take variants 0 and 2 for either B layout and the 128x256
    tile (variant 1) for B in KN layout only; nothing else."""
    _torch()
    for layout, ok in (("kn", (0, 1, 2)), ("nk", (0, 2))):
        op = kf.FusedOp.from_config(inputs.config("C2", M=512, N=512, K=64, b_layout=layout))
        for v in range(4):
            if v in ok:
                op.set_tuning(4, 1, 2, v)
                assert op.tuning()["variant"] == v
            else:
                with pytest.raises(kf.KFError) as e:
                    op.set_tuning(4, 1, 2, v)
                assert e.value.status == kf.KF_ERR_INVALID_ARG
        op.close()


def test_autotune_picks_the_tile_shape():
    """A short GEMM (256 x 8192 x 4096: 32 tiles of 256 x 256 for 256 CUs)
    runs faster with 128 x 256 tiles (64 tiles, two workgroups per CU): the
    tuner keeps that shape there, and the 256 x 256 tile at C2's size."""
    _torch()
    kept = {}
    for tag, kw in (("short", dict(M=256, N=8192, K=4096)), ("C2", {})):
        cfg = inputs.config("F6", **kw) if tag == "short" else inputs.config("C2")
        t = inputs.generate(cfg, seed=9)
        op = kf.FusedOp(inputs.chain_for(cfg, t), **kf.sizes_of(cfg))
        ins = op.device_inputs(t)
        out = op.empty_output("cuda")
        r = op.autotune(ins, out, reps=3)
        kept[tag] = r["best"]["variant"]
        times = {c["variant"]: c["seconds"] for c in r["candidates"] if c["variant"] == 1}
        print(tag, r["best"], times)
        check(cfg, t, out, rows=sample_rows(cfg["M"], 8, seed=2))
    # C2 stores no tile (its output is one logsumexp per row): both store
    # paths of the 256x256 kernel are the same work there
    assert kept["short"] == 1 and kept["C2"] in (0, 2), kept


def test_panel_traffic_model():
    """The tuner's L2 traffic model at C2's 16 x 16 tiles (one round of 256
    workgroups, 2 MiB panels): a 2-row raster in hardware order gives each XCD
    8 tile rows x 4 tile columns (12 panels), XCD-contiguous 1-row rasters 2
    rows x 16 columns (18 panels), XCD-contiguous 4-row rasters 4 x 8 (12)."""
    _torch()
    cfg = inputs.config("C2")
    t = inputs.generate(cfg, seed=3)
    op = kf.FusedOp(inputs.chain_for(cfg, t), **kf.sizes_of(cfg))
    ins = op.device_inputs(t)
    out = op.empty_output("cuda")
    r = op.autotune(ins, out, reps=1)
    by = {(c["raster_group"], c["xcd_remap"]): c["panel_bytes"] for c in r["candidates"] if c["variant"] == 0}
    assert all(c["panel_bytes"] == by[(c["raster_group"], c["xcd_remap"])] for c in r["candidates"]
               if c["variant"] == 2)
    panel = 256 * 4096 * 2
    assert by[(2, 0)] == 8 * 12 * panel
    assert by[(1, 1)] == 8 * 18 * panel
    assert by[(4, 1)] == 8 * 12 * panel
    assert by[(1, 0)] == 8 * (16 + 2) * panel   # one tile row per 16 workgroups: 16 rows x 2 columns per XCD


@pytest.mark.parametrize("name,bound", [("C1", "latency"), ("C2", "instruction"), ("F4", "memory"),
                                        ("F2", "instruction")])
def test_diagnosis_of_reference_workloads(name, bound):
    """The diagnosis rule on measured times: the 32 x 512 fp32 linear layer is
    latency-bound, the 4096^3 bf16 GEMM instruction-bound, and the softmax
    over stored 8192 x 8192 bf16 rows memory-bound."""
    torch = _torch()
    cfg = inputs.config(name)
    t = inputs.generate(cfg)
    op = kf.FusedOp(inputs.chain_for(cfg, t), **kf.sizes_of(cfg))
    ins = op.device_inputs(t)
    out = op.empty_output("cuda")
    for _ in range(3):
        op(ins, out)
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(10):
        op(ins, out)
    e.record()
    torch.cuda.synchronize()
    sec = s.elapsed_time(e) * 1e-3 / 10
    g = op.diagnose(sec)
    print(f"{name}: {g['bound']} compute {g['compute_frac']:.3f} memory {g['memory_frac']:.3f}")
    assert g["bound"] == bound
    assert g["flops"] == inputs.flops(cfg)


def test_unfused_rejects_padded_rows():
    """The unfused chain's per-op kernels index [M, N] tensors densely: a
    residual or output with a padded row stride is refused, not misread."""
    torch = _torch()
    cfg = inputs.config("C2", M=64, N=256, K=64, out_dtype="bf16", ops=[("bias",), ("residual_add",), ("relu",)],
                        dist=_ALL_DIST)
    t = inputs.generate(cfg, seed=3)
    op = kf.FusedOp.from_config(cfg)
    ins = op.device_inputs(t)
    wide = torch.empty((64, 264), dtype=torch.bfloat16, device="cuda")[:, :256]
    with pytest.raises(kf.KFError) as e:
        op.unfused(ins, wide)
    assert e.value.status == kf.KF_ERR_UNSUPPORTED and "row stride" in str(e.value)
    ins[3] = torch.empty((64, 264), dtype=torch.bfloat16, device="cuda")[:, :256].copy_(ins[3])
    with pytest.raises(kf.KFError) as e:
        op.unfused(ins, op.empty_output("cuda"))
    assert e.value.status == kf.KF_ERR_UNSUPPORTED and "residual" in str(e.value)
    out = op.empty_output("cuda")
    op(ins, out)                          # the fused kernel takes any row stride
    torch.cuda.synchronize()
    check(cfg, t, out)


# ------------------------------------------------------- cross-entropy rows

@pytest.mark.parametrize("M,N", [(37, 1032), (64, 4104), (5, 16384), (1, 8), (3, 131072), (2, 100008)])
def test_f5_rows_cross_entropy(M, N):
    _torch()
    cfg = inputs.config("F5", M=M, N=N)
    t = inputs.generate(cfg, seed=M + N)
    _, out = run_gpu(cfg, t)
    err = check(cfg, t, out)
    print(f"F5 {M}x{N} err {err:.3e}")


_STREAM_DIST = dict(a=("normal", 2.0), bias=("uniform", -0.5, 0.5), targets=("classes",))


@pytest.mark.parametrize("ops,N", [
    ([("scale", 0.5), ("tanh",), ("row_logsumexp",)], 4104),
    ([("bias",), ("gelu_erf",), ("row_cross_entropy",)], 1032),
    ([("bias",), ("hardtanh", -1.0, 1.0), ("row_cross_entropy",)], 40000),
    ([("row_logsumexp",)], 65536),
])
def test_streamed_row_reductions(ops, N):
    """Row logsumexp / cross-entropy after element-wise ops and a bias
    (interpreted list, rows streamed, widths past the held-row limit)."""
    _torch()
    cfg = inputs.config("F5", M=19, N=N, ops=ops, dist=_STREAM_DIST)
    t = inputs.generate(cfg, seed=N + len(ops))
    _, out = run_gpu(cfg, t)
    err = check(cfg, t, out)
    print(f"streamed {[o[0] for o in ops]} {N} err {err:.3e}")


def test_cross_entropy_targets_out_of_range():
    """A target outside [0, N) gives NaN for its row and leaves the others."""
    _torch()
    for name, kw in (("F5", dict(M=6, N=1032)), ("F6", dict(M=6, N=1032, K=64))):
        cfg = inputs.config(name, **kw)
        t = inputs.generate(cfg, seed=5)
        t["targets"] = t["targets"].copy()
        t["targets"][[1, 4]] = [-1, kw["N"]]
        _, out = run_gpu(cfg, t)
        g = to_host_f64(out)
        assert np.isnan(g[[1, 4]]).all(), (name, g)
        keep = np.array([0, 2, 3, 5])
        ref = oracle.run_chain(inputs.chain_for(cfg, t), t, rows=keep)
        assert np.isnan(oracle.run_chain(inputs.chain_for(cfg, t), t, rows=np.array([1, 4]))).all()
        assert parity_error(g[keep], ref, 1.0) <= TOL["bf16"], name


@pytest.mark.parametrize("M,N,K,layout", [(300, 1040, 136, "kn"), (77, 16384, 64, "kn"), (129, 776, 200, "nk"),
                                          (1, 8, 8, "kn")])
def test_f6_gemm_cross_entropy(M, N, K, layout):
    """The target logit is left by whichever lane of whichever tile holds it:
    ragged last column tiles, many tiles per row, both B layouts."""
    _torch()
    cfg = inputs.config("F6", M=M, N=N, K=K, b_layout=layout)
    t = inputs.generate(cfg, seed=M + N + K)
    _, out = run_gpu(cfg, t)
    err = check(cfg, t, out)
    print(f"F6 {M}x{N}x{K} {layout} err {err:.3e}")


@pytest.mark.parametrize("name", ["F5", "F6"])
def test_cross_entropy_full_config_sampled_rows(name):
    _torch()
    cfg = inputs.config(name)
    t = inputs.generate(cfg)
    _, out = run_gpu(cfg, t)
    g = to_host_f64(out)
    assert np.all(np.isfinite(g)) and np.all(g >= -1e-3)   # a loss is >= 0 up to rounding
    err = check(cfg, t, out, rows=sample_rows(cfg["M"], 24))
    print(f"{name} full err {err:.3e}")


@pytest.mark.parametrize("name,kw", [("F5", dict(M=6, N=1024)), ("F6", dict(M=6, N=1040, K=64))])
def test_cross_entropy_every_target_column_and_out_of_range(name, kw):
    """Targets on the first and last column, on every lane position of a
    tile, and outside [0, N): the fused kernels give NaN for the latter,
    like the oracle, and the exact loss elsewhere; so does the unfused chain."""
    _torch()
    cfg = inputs.config(name, **kw)
    t = inputs.generate(cfg, seed=8)
    N = cfg["N"]
    t["targets"] = np.array([0, N - 1, 255, 256, -3, N], dtype=np.int32)
    for unfused in (False, True):
        _, out = run_gpu(cfg, t, unfused=unfused)
        g = to_host_f64(out)
        assert np.all(np.isnan(g[4:])) and np.all(np.isfinite(g[:4]))
        ref = (oracle.run_chain_unfused if unfused else oracle.run_chain)(inputs.chain_for(cfg, t), t)
        assert parity_error(g[:4], ref[:4], 1.0) <= TOL["bf16"]
    cfg = inputs.config(name, **dict(kw, M=64))
    t = inputs.generate(cfg, seed=9)
    t["targets"] = np.arange(64, dtype=np.int32) * 16 % N   # lanes of every position across tiles
    _, out = run_gpu(cfg, t)
    check(cfg, t, out)


def test_diagnosis_from_counters():
    """kf_diagnose_counters on counter values of the kind the committed
    profiles hold: a bf16 GEMM whose matrix cores are busy half the time and
    whose operand panels are fetched 4.5x is instruction-bound with the
    overlap and reuse hints; the softmax rows moving their algorithmic bytes
    are memory-bound with no hint; LDS bank conflicts set the layout hint; a
    busy fraction above 0.75 drops the overlap hint."""
    _torch()
    c2 = kf.FusedOp.from_config(inputs.config("C2"))
    g = c2.diagnose_counters(115e-6, 303.8e6, 0.51, 0.0)
    assert g["bound"] == "instruction" and sorted(g["hints"]) == ["overlap", "reuse"]
    assert g["compute_frac"] == 0.51 and abs(g["traffic_ratio"] - 303.8e6 / 67141632) < 1e-9
    g = c2.diagnose_counters(115e-6, 70e6, 0.8, 0.12)
    assert g["bound"] == "instruction" and g["hints"] == ["lds_layout"]
    f4 = kf.FusedOp.from_config(inputs.config("F4"))
    g = f4.diagnose_counters(40e-6, 268.6e6)
    assert g["bound"] == "memory" and g["hints"] == [] and g["mfma_busy"] == -1.0
    g = f4.diagnose_counters(400e-6, 268.6e6)
    assert g["bound"] == "latency" and g["hints"] == ["pipeline"]


@pytest.mark.parametrize("dt,peak", [("bf16", 2516.6), ("e4m3", 5033.2)])
def test_mfma_probe(dt, peak):
    """The matrix-core probe: one workgroup per compute unit; its rate is a
    positive fraction of the datasheet peak, and it cannot exceed what the
    matrix cores deliver at the clock it measured (the datasheet peak
    scaled by clock / 2.4 GHz), so rate and clock check each other."""
    torch = _torch()
    r = kf.probe_mfma(dt, 20000)
    print(f"[gpu] probe {dt}: {r}", flush=True)
    assert r["workgroups"] == torch.cuda.get_device_properties(0).multi_processor_count
    assert r["seconds"] > 0 and 0.5 < r["clock_ghz"] < 2.6
    assert 0.2 * peak < r["tflops"] < 1.02 * peak * r["clock_ghz"] / 2.4


def test_copy_probe():
    """The copy probe moves its bytes: 64 MiB copied at a rate between a
    tenth of the datasheet HBM bandwidth and the datasheet itself (the
    64 MiB buffers fit the 256 MB Infinity Cache, hence the loose bound)."""
    _torch()
    r = kf.probe_copy(64 << 20, 5)
    print(f"[gpu] copy probe: {r}", flush=True)
    assert r["seconds"] > 0 and 800 < r["gbps"] < 2 * 8000


@pytest.mark.parametrize("name,kw", [("C2", dict(M=520, N=776, K=256)), ("C5", dict(M=512, N=1024, K=512))])
def test_gemm_clock_stamps(name, kw):
    """kf_set_clock_stamps: every workgroup of the 256x256 kernel writes its
    six counters, in order (start, end of the prologue, end of the K loop,
    end), the shader clock they give is a clock the device can run at, the
    output bits do not change, and NULL turns the stamps off; other plans
    refuse them."""
    torch = _torch()
    cfg = inputs.config(name, **kw)
    t = inputs.generate(cfg, seed=63)
    op = kf.FusedOp(inputs.chain_for(cfg, t), **kf.sizes_of(cfg))
    ins = op.device_inputs(t)
    ref = op.empty_output("cuda")
    op(ins, ref)
    tiles = -(-cfg["M"] // 256) * -(-cfg["N"] // 256)
    buf = torch.zeros(6 * tiles + 6, dtype=torch.int64, device="cuda")
    op.set_clock_stamps(buf)
    out = op.empty_output("cuda")
    op(ins, out)
    torch.cuda.synchronize()
    bits = (lambda x: x.view(torch.int16)) if ref.dtype == torch.bfloat16 else (lambda x: x)
    assert torch.equal(bits(ref), bits(out))
    a = buf.cpu().numpy().reshape(-1, 6)
    assert np.all(a[:tiles, 1] > a[:tiles, 0]) and np.all(a[:tiles, 3] > a[:tiles, 2])
    c0, c1, cp, ck = a[:tiles, 0], a[:tiles, 1], a[:tiles, 4], a[:tiles, 5]
    assert np.all(c0 < cp) and np.all(cp < ck) and np.all(ck < c1)
    assert np.all(a[tiles:] == 0)           # room for one more workgroup than launched: untouched
    hz = kf.lib().kf_wall_clock_hz()
    ghz = (a[:tiles, 1] - a[:tiles, 0]) / ((a[:tiles, 3] - a[:tiles, 2]) / hz) * 1e-9
    assert 0.3 < np.median(ghz) < 2.6, ghz
    op.set_clock_stamps(None)
    buf.zero_()
    op(ins, out)
    torch.cuda.synchronize()
    assert int(buf.abs().sum().item()) == 0
    mfma = 2.0 * 256 * 256 * cfg["K"] / 4 / (2048 if cfg["in_dtype"] == "e4m3" else 1024)
    st = op.clock_stamps(lambda: op(ins, out), tiles, calls=3, mfma_cycles=mfma)
    print(f"[gpu] {name} stamps {st}", flush=True)
    assert st["workgroups"] == tiles and 0.3 < st["clock_ghz_median"] < 2.6
    shares = st["prologue_share"] + st["k_loop_share"] + st["epilogue_share"]
    assert 0.9 < shares < 1.1, st
    # the matrix cores cannot be busy for more cycles than the K loop has
    assert 0 < st["mfma_busy_in_tile"] < st["mfma_busy_in_k_loop"] <= 1.02, st
    rows = kf.FusedOp.from_config(inputs.config("F4", M=64, N=2048))
    with pytest.raises(kf.KFError) as e:
        rows.set_clock_stamps(buf)
    assert e.value.status == kf.KF_ERR_UNSUPPORTED
