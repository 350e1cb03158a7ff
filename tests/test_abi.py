"""Boundary tests that need no GPU: libkf.so loads, exports every function
include/kf.h declares, links no vendor math library, and rejects malformed
op descriptors on the host with the documented status codes."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2605_30359_amd import inputs, kf

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kf.h")


def _gpu_present():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kf_[a-z_]+)\s*\(", text)))


def test_header_declares_expected_api():
    names = declared_functions()
    for required in ("kf_create", "kf_fused_op", "kf_destroy", "kf_status_string", "kf_last_error"):
        assert required in names
    assert set(names) == set(kf.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = kf.lib()
    out = subprocess.run(["nm", "-D", "--defined-only", kf.LIB_PATH], capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r" T (kf_\w+)", out))
    for name in declared_functions():
        assert name in exported, name
        assert hasattr(lib, name)


def test_library_links_no_vendor_math_or_torch():
    out = subprocess.run(["ldd", kf.LIB_PATH], capture_output=True, text=True).stdout.lower()
    for bad in ("rocblas", "hipblas", "miopen", "torch", "rocsolver"):
        assert bad not in out, out


def test_status_strings():
    for st in range(7):
        assert kf.status_string(st).startswith("KF_")
    assert kf.status_string(99) == "unknown kf_status"


def test_ctypes_struct_layout_matches_header():
    # kf_op 16 B; kf_op_spec: 4 ints, 8 int64, 2 floats, 2 ints, 8 ops
    assert ctypes.sizeof(kf.KfOp) == 16
    assert ctypes.sizeof(kf.KfOpSpec) == 16 + 72 + 8 + 8 + 8 * 16
    assert ctypes.sizeof(kf.KfTensor) == 8 + 4 + 4 + 40 + 40


def _create(spec):
    h = ctypes.c_void_p()
    st = kf.lib().kf_create(ctypes.byref(spec), ctypes.byref(h))
    return st, h


def _spec(name, **kw):
    cfg = inputs.config(name, **kw)
    return kf.make_spec(inputs.chain(cfg), **kf.sizes_of(cfg))


def test_conv_validation():
    """Any conv shape plans (the tiled kernels' family or the general
    kernel); a 2x2 pool needs an even height and width; the op and dtype
    rules hold for both."""
    ok = kf.KF_ERR_NO_DEVICE if not _gpu_present() else kf.KF_OK
    for kw, status in [(dict(cin=32), ok), (dict(cin=3, cout=40, W=50), ok), (dict(H=7, ops=[("bias",)]), ok),
                       (dict(H=7), kf.KF_ERR_UNSUPPORTED), (dict(W=9), kf.KF_ERR_UNSUPPORTED),
                       (dict(ops=[("groupnorm", 2, 1e-5)]), kf.KF_ERR_UNSUPPORTED),
                       (dict(out_dtype="f32"), kf.KF_ERR_UNSUPPORTED), (dict(in_dtype="f32"), kf.KF_ERR_UNSUPPORTED)]:
        st, h = _create(_spec("C4", **kw))
        assert st == status, (kw, st, kf.last_error())
        if h.value:
            kf.lib().kf_destroy(h)


def test_create_null_arguments():
    lib = kf.lib()
    h = ctypes.c_void_p()
    assert lib.kf_create(None, ctypes.byref(h)) == kf.KF_ERR_INVALID_ARG
    assert "NULL" in kf.last_error()
    spec = _spec("C2")
    assert lib.kf_create(ctypes.byref(spec), None) == kf.KF_ERR_INVALID_ARG
    lib.kf_destroy(None)  # NULL-safe


@pytest.mark.parametrize("mutate,status,msg", [
    (lambda s: setattr(s, "contraction", 7), kf.KF_ERR_INVALID_ARG, "contraction"),
    (lambda s: setattr(s, "in_dtype", 9), kf.KF_ERR_INVALID_ARG, "in_dtype"),
    (lambda s: setattr(s, "out_dtype", kf.KF_FP8_E4M3), kf.KF_ERR_INVALID_ARG, "out_dtype"),
    (lambda s: setattr(s, "n_ops", 9), kf.KF_ERR_INVALID_ARG, "n_ops"),
    (lambda s: setattr(s, "K", 100), kf.KF_ERR_UNSUPPORTED, "K % 8"),
    (lambda s: setattr(s, "N", 4100), kf.KF_ERR_UNSUPPORTED, "N % 8"),
    (lambda s: setattr(s, "M", -1), kf.KF_ERR_SHAPE, "M >= 0"),
    (lambda s: setattr(s, "b_layout", 5), kf.KF_ERR_INVALID_ARG, "b_layout"),
    (lambda s: (setattr(s, "in_dtype", kf.KF_FP8_E4M3), setattr(s, "scale_a", 0.0)), kf.KF_ERR_INVALID_ARG, "scale"),
    (lambda s: (setattr(s, "in_dtype", kf.KF_FP8_E4M3), setattr(s, "K", 4104)), kf.KF_ERR_UNSUPPORTED, "K % 16"),
])
def test_create_rejects_bad_specs(mutate, status, msg):
    spec = _spec("C2")
    mutate(spec)
    st, h = _create(spec)
    assert st == status, (st, kf.last_error())
    assert not h.value
    assert msg in kf.last_error()


def test_row_op_must_be_last():
    cfg = inputs.config("C2", ops=[("bias",), ("row_logsumexp",), ("relu",)])
    spec = kf.make_spec(inputs.chain(cfg), **kf.sizes_of(cfg))
    st, _ = _create(spec)
    assert st == kf.KF_ERR_UNSUPPORTED and "last" in kf.last_error()


def test_row_reductions_reject_more_rows_than_one_launch_covers():
    """Row softmax / logsumexp finishing kernels and the row-wise chains run
    one 256-thread workgroup per row: 2^24 rows would exceed the 2^32
    work-items of one launch, so the plan refuses them on the host."""
    for name, ops in (("C2", None), ("C5", None), ("F4", None)):
        cfg = inputs.config(name, M=1 << 24, K=64, **({"ops": ops} if ops else {}))
        ch = inputs.chain(cfg)
        ch.update(scale_a=1.0, scale_b=1.0)
        st, _ = _create(kf.make_spec(ch, **kf.sizes_of(cfg)))
        assert st == kf.KF_ERR_UNSUPPORTED and "M < 16777216" in kf.last_error(), (name, kf.last_error())
    # a plain GEMM epilogue has no per-row launch
    cfg = inputs.config("C2", M=1 << 24, K=64, out_dtype="bf16", ops=[("bias",), ("relu",)])
    st, _ = _create(kf.make_spec(inputs.chain(cfg), **kf.sizes_of(cfg)))
    assert st != kf.KF_ERR_UNSUPPORTED, kf.last_error()


def test_logsumexp_needs_f32_output():
    cfg = inputs.config("C2", out_dtype="bf16")
    st, _ = _create(kf.make_spec(inputs.chain(cfg), **kf.sizes_of(cfg)))
    assert st == kf.KF_ERR_UNSUPPORTED


def test_groupnorm_validation():
    cfg = inputs.config("C3", ops=[("groupnorm", 3, 1e-5)])
    st, _ = _create(kf.make_spec(inputs.chain(cfg), **kf.sizes_of(cfg)))
    assert st == kf.KF_ERR_SHAPE and "divisible" in kf.last_error()
    cfg = inputs.config("C3", ops=[("groupnorm", 256, 1e-5)])   # width 32: not fused
    st, _ = _create(kf.make_spec(inputs.chain(cfg), **kf.sizes_of(cfg)))
    assert st == kf.KF_ERR_UNSUPPORTED
    cfg = inputs.config("C3", ops=[("groupnorm", 32, -1.0)])
    st, _ = _create(kf.make_spec(inputs.chain(cfg), **kf.sizes_of(cfg)))
    assert st == kf.KF_ERR_INVALID_ARG


def test_maxpool_needs_conv_and_fp32_limits():
    cfg = inputs.config("C2", ops=[("maxpool2x2",)], out_dtype="f32")
    st, _ = _create(kf.make_spec(inputs.chain(cfg), **kf.sizes_of(cfg)))
    assert st == kf.KF_ERR_UNSUPPORTED and "CONV" in kf.last_error()
    cfg = inputs.config("C1", ops=[("row_softmax",)])
    st, _ = _create(kf.make_spec(inputs.chain(cfg), **kf.sizes_of(cfg)))
    assert st == kf.KF_ERR_UNSUPPORTED


def test_hardtanh_bounds_validated():
    cfg = inputs.config("C5", ops=[("hardtanh", 1.0, -1.0)], in_dtype="bf16")
    st, _ = _create(kf.make_spec(inputs.chain(cfg), **kf.sizes_of(cfg)))
    assert st == kf.KF_ERR_INVALID_ARG


@pytest.mark.skipif(_gpu_present(), reason="checks the no-device path")
def test_valid_spec_without_device_reports_no_device():
    for name in ("C1", "C2", "C3", "C4", "C5"):
        st, h = _create(_spec(name, **({"scale_a": 0.01, "scale_b": 0.01} if name == "C5" else {})))
        assert st == kf.KF_ERR_NO_DEVICE, (name, st, kf.last_error())
        assert not h.value


def test_binding_raises_kferror():
    cfg = inputs.config("C2", K=100)
    with pytest.raises(kf.KFError) as ei:
        kf.FusedOp.from_config(cfg)
    assert ei.value.status == kf.KF_ERR_UNSUPPORTED


def test_input_slot_order():
    ch = inputs.chain(inputs.config("C3"))
    assert kf.input_names(ch) == ["a", "b", "gamma", "beta", "residual"]
    ch = inputs.chain(inputs.config("C2"))
    assert kf.input_names(ch) == ["a", "b", "bias"]


def test_struct_offsets_match_c_compiler(tmp_path):
    # the ctypes mirror against what a C compiler makes of include/kf.h
    import shutil
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    structs = [("kf_op", kf.KfOp), ("kf_op_spec", kf.KfOpSpec), ("kf_tensor", kf.KfTensor),
               ("kf_diagnosis", kf.KfDiagnosis), ("kf_tuning", kf.KfTuning), ("kf_tune_result", kf.KfTuneResult),
               ("kf_counters", kf.KfCounters), ("kf_mfma_probe", kf.KfMfmaProbe),
               ("kf_copy_probe", kf.KfCopyProbe)]
    lines, want = [], []
    for cname, py in structs:
        for f in py._fields_:
            lines.append(f'  printf("%zu\\n", offsetof({cname}, {f[0]}));\n')
            want.append(getattr(py, f[0]).offset)
        lines.append(f'  printf("%zu\\n", sizeof({cname}));\n')
        want.append(ctypes.sizeof(py))
    src = tmp_path / "off.c"
    src.write_text('#include <stdio.h>\n#include <stddef.h>\n#include "kf.h"\nint main(void) {\n'
                   + "".join(lines) + "  return 0;\n}\n")
    exe = tmp_path / "off"
    subprocess.check_call([cc, "-std=c99", f"-I{os.path.join(ROOT, 'include')}", str(src), "-o", str(exe)])
    got = [int(x) for x in subprocess.check_output([str(exe)]).split()]
    assert got == want



def test_probe_argument_checks():
    """The matrix-core and copy probes check their arguments before touching
    a device."""
    r = kf.KfMfmaProbe()
    lib = kf.lib()
    assert lib.kf_probe_mfma(kf.KF_BF16, 100, None) == kf.KF_ERR_INVALID_ARG
    assert lib.kf_probe_mfma(kf.KF_F32, 100, ctypes.byref(r)) == kf.KF_ERR_UNSUPPORTED
    assert lib.kf_probe_mfma(kf.KF_BF16, 0, ctypes.byref(r)) == kf.KF_ERR_INVALID_ARG
    assert lib.kf_probe_mfma(kf.KF_FP8_E4M3, (1 << 24) + 1, ctypes.byref(r)) == kf.KF_ERR_INVALID_ARG
    if not _gpu_present():
        assert lib.kf_probe_mfma(kf.KF_BF16, 100, ctypes.byref(r)) == kf.KF_ERR_NO_DEVICE
    c = kf.KfCopyProbe()
    assert lib.kf_probe_copy(1 << 20, 1, None) == kf.KF_ERR_INVALID_ARG
    assert lib.kf_probe_copy(1000, 1, ctypes.byref(c)) == kf.KF_ERR_INVALID_ARG      # not a multiple of 16
    assert lib.kf_probe_copy(1 << 20, 0, ctypes.byref(c)) == kf.KF_ERR_INVALID_ARG
    assert lib.kf_probe_copy((1 << 34) + 16, 1, ctypes.byref(c)) == kf.KF_ERR_INVALID_ARG
    if not _gpu_present():
        assert lib.kf_probe_copy(1 << 20, 1, ctypes.byref(c)) == kf.KF_ERR_NO_DEVICE


def test_clock_stamp_argument_checks():
    lib = kf.lib()
    assert lib.kf_set_clock_stamps(None, None, 0) == kf.KF_ERR_INVALID_ARG
    if not _gpu_present():
        assert lib.kf_wall_clock_hz() == -1


def test_rowwise_validation():
    base = dict(M=64, N=1024)
    cases = [
        (dict(N=1020), kf.KF_ERR_UNSUPPORTED),                              # N % 8
        (dict(N=16392), kf.KF_ERR_UNSUPPORTED),                             # too wide
        (dict(ops=[("groupnorm", 3, 1e-5)]), kf.KF_ERR_UNSUPPORTED),        # N % groups
        (dict(ops=[("groupnorm", 256, 1e-5)]), kf.KF_ERR_UNSUPPORTED),      # 4-column groups
        (dict(ops=[("maxpool2x2",)]), kf.KF_ERR_UNSUPPORTED),
        (dict(ops=[("row_softmax",), ("relu",)]), kf.KF_ERR_UNSUPPORTED),   # row op not last
        (dict(in_dtype="e4m3"), kf.KF_ERR_UNSUPPORTED),
        (dict(M=-1), kf.KF_ERR_SHAPE),
    ]
    for kw, status in cases:
        cfg = inputs.config("F3", **dict(base, **kw))
        st, _ = _create(kf.make_spec(inputs.chain(cfg), **kf.sizes_of(cfg)))
        assert st == status, (kw, st, kf.last_error())


def test_rowwise_width_limits():
    """Rows held in registers stop at 16384 columns; a row logsumexp or
    cross-entropy after element-wise ops streams its rows, any width."""
    ok = kf.KF_ERR_NO_DEVICE if not _gpu_present() else kf.KF_OK
    for name, ops, N, status in [
        ("F4", [("row_softmax",)], 16392, kf.KF_ERR_UNSUPPORTED),
        ("F5", [("row_cross_entropy",)], 131072, ok),
        ("F5", [("bias",), ("tanh",), ("row_logsumexp",)], 1 << 20, ok),
        ("F5", [("groupnorm", 2, 1e-5), ("row_logsumexp",)], 32768, kf.KF_ERR_UNSUPPORTED),
        ("F5", [("row_cross_entropy",)], 131076, kf.KF_ERR_UNSUPPORTED),  # N % 8
    ]:
        cfg = inputs.config(name, M=4, N=N, ops=ops)
        st, h = _create(kf.make_spec(inputs.chain(cfg), **kf.sizes_of(cfg)))
        assert st == status, (name, ops, N, st, kf.last_error())
        if h.value:
            kf.lib().kf_destroy(h)


def test_rowwise_input_slots():
    ch = inputs.chain(inputs.config("F3"))
    assert kf.input_names(ch) == ["a", "gamma", "beta", "residual"]
    assert kf.input_names(inputs.chain(inputs.config("F4"))) == ["a"]


def test_conv3d_validation():
    ok = kf.KF_ERR_NO_DEVICE if not _gpu_present() else kf.KF_OK
    # outside the tiled kernel's shape family the whole op family runs, partly fused
    for kw, status in [(dict(cin=32), ok), (dict(cout=32), ok),
                       (dict(cin=32, ops=[("bias",), ("relu",)]), ok),      # the general kernel
                       (dict(cin=3, cout=200, D=3, H=3, W=3, ops=[]), ok),
                       (dict(cout=32, ops=[("bias",), ("channel_softmax",)]), ok),
                       (dict(D=2), kf.KF_ERR_SHAPE), (dict(W=2), kf.KF_ERR_SHAPE),
                       (dict(out_dtype="f32"), kf.KF_ERR_UNSUPPORTED), (dict(in_dtype="f32"), kf.KF_ERR_UNSUPPORTED),
                       (dict(ops=[("bias",), ("channel_softmax",), ("maxpool3d2",)]), kf.KF_ERR_UNSUPPORTED),
                       (dict(ops=[("maxpool3d2",), ("maxpool3d2",), ("channel_softmax",)]), kf.KF_ERR_UNSUPPORTED),
                       (dict(ops=[("maxpool3d2",), ("relu",), ("maxpool3d2",)]), kf.KF_ERR_UNSUPPORTED),
                       (dict(ops=[("channel_softmax",), ("channel_softmax",)]), kf.KF_ERR_UNSUPPORTED),
                       (dict(ops=[("groupnorm", 2, 1e-5)]), kf.KF_ERR_UNSUPPORTED),
                       (dict(ops=[("row_softmax",)]), kf.KF_ERR_UNSUPPORTED),
                       (dict(ops=[("maxpool2x2",)]), kf.KF_ERR_UNSUPPORTED),
                       (dict(D=2000, H=2000, W=20), kf.KF_ERR_UNSUPPORTED)]:
        st, h = _create(_spec("F2", **kw))
        assert st == status, (kw, st, kf.last_error())
        assert bool(h.value) == (st == kf.KF_OK)
        if h.value:
            kf.lib().kf_destroy(h)
    # the conv3d ops on other contractions
    for name, ops in [("C2", [("channel_softmax",)]), ("C4", [("maxpool3d2",), ("maxpool3d2",)]),
                      ("F4", [("channel_softmax",)])]:
        st, _ = _create(_spec(name, ops=ops))
        assert st == kf.KF_ERR_UNSUPPORTED, (name, ops)
    if not _gpu_present():
        for kw in [{}, dict(ops=[]), dict(ops=[("bias",), ("channel_softmax",)])]:
            st, _ = _create(_spec("F2", **kw))
            assert st == kf.KF_ERR_NO_DEVICE, (kw, kf.last_error())


# ------------------------------------------------------------ diagnosis rule

def test_classify_bounds():
    """The three classes of the diagnosis rule on hand-computed cases
    (MI355X bf16 peak 2516.6 TFLOP/s, HBM 8000 GB/s, 256 compute units)."""
    P, B, CU = 2516.6, 8000.0, 256
    # 4096^3 bf16 GEMM in 100 us: 1374 TFLOP/s = 54.6 % of peak, 0.67 GB/ms -> instruction-bound
    g = kf.classify(2 * 4096 ** 3, 3 * 4096 * 4096 * 2, 100e-6, P, B, 256, CU)
    assert g["bound"] == "instruction"
    assert abs(g["tflops"] - 2 * 4096 ** 3 / 100e-6 / 1e12) < 1e-6 and abs(g["compute_frac"] - g["tflops"] / P) < 1e-12
    assert abs(g["ridge"] - P * 1e12 / (B * 1e9)) < 1e-9
    # 256 MiB streamed in 50 us (5369 GB/s, 67 %), no FLOPs -> memory-bound
    g = kf.classify(0.0, 2 * 2 ** 27, 50e-6, P, B, 8192, CU)
    assert g["bound"] == "memory" and abs(g["memory_frac"] - 2 ** 28 / 50e-6 / 1e9 / B) < 1e-12
    # tiny fp32 op: 8.4 MFLOP and 0.6 MB in 6 us -> far below both roofs -> latency-bound
    g = kf.classify(8388608, 624640, 6e-6, 157.3, B, 256, CU)
    assert g["bound"] == "latency" and g["compute_frac"] < 0.25 and g["memory_frac"] < 0.25
    # a launch with fewer workgroups than compute units is latency-bound whatever the rates
    assert kf.classify(2 * 4096 ** 3, 1e8, 100e-6, P, B, 64, CU)["bound"] == "latency"
    # ties between the roofs go to memory
    assert kf.classify(P * 1e12 * 0.5, B * 1e9 * 0.5, 1.0, P, B, 1000, CU)["bound"] == "memory"
    with pytest.raises(kf.KFError):
        kf.classify(1.0, 1.0, 0.0, P, B, 1, CU)


def test_noalloc_rejects_before_any_device_call():
    """kf_fused_op_noalloc plans on the host first: a malformed spec, and an
    op whose workspace exceeds the 4 MiB static scratch, are rejected before
    any device call (so also here, with no GPU); a valid small spec then
    needs a device."""
    ch = inputs.chain(inputs.config("C5"))
    ch.update(scale_a=1.0, scale_b=1.0)
    # 16384 rows x 64 column tiles of (max, sum) partials = 8 MiB > 4 MiB
    st, msg = kf.fused_op_noalloc_status(ch, M=16384, N=16384, K=64)
    assert st == kf.KF_ERR_UNSUPPORTED and "static scratch holds 4194304" in msg, msg
    bad = dict(ch, ops=[("row_softmax",), ("relu",)])
    st, msg = kf.fused_op_noalloc_status(bad, M=64, N=64, K=64)
    assert st == kf.KF_ERR_UNSUPPORTED and "last op" in msg, msg
    # exactly at the limit: 8192 rows x 64 tiles = 4 MiB is accepted by the planner
    st, msg = kf.fused_op_noalloc_status(ch, M=8192, N=16384, K=64)
    if not _gpu_present():
        assert st == kf.KF_ERR_NO_DEVICE, msg
    else:
        assert st in (kf.KF_ERR_INVALID_ARG, kf.KF_ERR_SHAPE), msg  # the empty tensors are refused


def test_classify_sets_latency_hints():
    """Latency-bound launches carry a hint: too few workgroups -> more
    parallelism, enough workgroups but far from both roofs -> pipelining."""
    few = kf.classify(1e9, 1e6, 1e-3, 2516.6, 8000.0, 100, 256)
    assert few["bound"] == "latency" and few["hints"] == ["parallelism"]
    slow = kf.classify(1e9, 1e6, 1e-3, 2516.6, 8000.0, 1000, 256)
    assert slow["bound"] == "latency" and slow["hints"] == ["pipeline"]
    busy = kf.classify(2e12, 1e9, 1e-3, 2516.6, 8000.0, 1000, 256)
    assert busy["bound"] == "instruction" and busy["hints"] == []
    assert busy["mfma_busy"] == -1.0 and busy["traffic_ratio"] == -1.0
