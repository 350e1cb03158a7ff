"""Seeded synthetic inputs for the fused chains, shared by the tests, the
benchmark and the oracle checks.

This module holds no arithmetic of the fused chains themselves: it draws
random tensors, rounds them once into the storage formats the kernels consume
(bfloat16, OCP FP8 E4M3 with a per-tensor scale) and describes each workload
as plain data.  Both the HIP path and the oracle receive the exact same bits.

The paper evaluates on a public benchmark suite of PyTorch operators
(Evaluation, Benchmark); none of its items are reproduced here.  The five
workloads below are synthetic stand-ins, one per fused-operator category of
the paper's category table (Table 2: matmul-centred, conv-centred, mixed
reduction), with the shapes and value distributions stated per workload.

Normal draws N(0, v) give the variance v (so W ~ N(0, 1/K) keeps x@W at unit
scale).  Tensors are drawn in float32 in the order x, W, b, gamma, beta,
residual from ``numpy.random.Generator(PCG64(SeedSequence(seed)))``; the
default seed of workload k (1..5) is 260530359 + k.
"""
from __future__ import annotations

import copy

import numpy as np

# ---------------------------------------------------------------------------
# Workloads (plain data)
# ---------------------------------------------------------------------------

CONFIGS = {
    "C1": dict(
        workload="linear_bias_relu_f32",
        contraction="gemm", in_dtype="f32", out_dtype="f32", b_layout="kn",
        M=32, N=512, K=256,
        ops=[("bias",), ("relu",)],
        dist=dict(a=("normal", 1.0), b=("normal_invk",), bias=("uniform", -0.1, 0.1)),
    ),
    "C2": dict(
        workload="gemm_bias_gelutanh_scale_logsumexp_bf16",
        contraction="gemm", in_dtype="bf16", out_dtype="f32", b_layout="kn",
        M=4096, N=4096, K=4096,
        ops=[("bias",), ("gelu_tanh",), ("scale", 0.5), ("row_logsumexp",)],
        dist=dict(a=("normal", 1.0), b=("normal_invk",), bias=("uniform", -0.1, 0.1)),
    ),
    "C3": dict(
        workload="gemm_groupnorm_swish_residual_bf16",
        contraction="gemm", in_dtype="bf16", out_dtype="bf16", b_layout="kn",
        M=8192, N=8192, K=2048,
        ops=[("groupnorm", 32, 1e-5), ("swish",), ("residual_add",)],
        residual_dtype="bf16",
        dist=dict(a=("normal", 1.0), b=("normal_invk",), gamma=("uniform", 0.5, 1.5),
                  beta=("uniform", -0.1, 0.1), residual=("normal", 1.0)),
    ),
    "C4": dict(
        workload="conv3x3_bias_relu_maxpool2_bf16",
        contraction="conv2d_3x3", in_dtype="bf16", out_dtype="bf16",
        batch=64, cin=64, H=128, W=128, cout=128,
        ops=[("bias",), ("relu",), ("maxpool2x2",)],
        dist=dict(a=("normal", 1.0), b=("normal_invk",), bias=("uniform", -0.1, 0.1)),
    ),
    "C5": dict(
        workload="fp8_gemm_scales_bias_hardtanh_softmax",
        contraction="gemm", in_dtype="e4m3", out_dtype="bf16", b_layout="kn",
        M=8192, N=8192, K=8192,
        ops=[("bias",), ("hardtanh", -1.0, 1.0), ("row_softmax",)],
        dist=dict(a=("normal", 1.0), b=("normal", 1.0), bias=("uniform", -0.1, 0.1)),
    ),
    # the paper's worked matmul + activation fusion (Appendix C): a GEMM
    # followed by bias, swish, tanh, exact GELU and hardtanh, at the C2 size
    "F1": dict(
        workload="gemm_bias_swish_tanh_geluerf_hardtanh_bf16",
        contraction="gemm", in_dtype="bf16", out_dtype="bf16", b_layout="kn",
        M=4096, N=4096, K=4096,
        ops=[("bias",), ("swish",), ("tanh",), ("gelu_erf",), ("hardtanh", -1.0, 1.0)],
        dist=dict(a=("normal", 1.0), b=("normal_invk",), bias=("uniform", -0.1, 0.1)),
    ),
    # the Conv3d -> channel softmax -> MaxPool3d -> MaxPool3d operator of the
    # paper's case study (Appendix C), with the conv's bias; the paper gives
    # no sizes, so these are chosen for one GPU: 16 volumes of 16 channels,
    # each 34 x 66 x 66, and 64 output channels
    "F2": dict(
        workload="conv3d_bias_channelsoftmax_maxpool3d_x2_bf16",
        contraction="conv3d_3x3x3", in_dtype="bf16", out_dtype="bf16",
        batch=16, cin=16, D=34, H=66, W=66, cout=64,
        ops=[("bias",), ("channel_softmax",), ("maxpool3d2",), ("maxpool3d2",)],
        dist=dict(a=("normal", 1.0), b=("normal_invk",), bias=("uniform", -0.1, 0.1)),
    ),
    # memory-bound reduction chains with no contraction (the paper's
    # reduction-dominated category, Table 2): C3's epilogue and C5's softmax
    # over stored [8192, 8192] bf16 activations
    "F3": dict(
        workload="rows_groupnorm_swish_residual_bf16",
        contraction="rowwise", in_dtype="bf16", out_dtype="bf16",
        M=8192, N=8192,
        ops=[("groupnorm", 32, 1e-5), ("swish",), ("residual_add",)],
        residual_dtype="bf16",
        dist=dict(a=("normal", 1.0), gamma=("uniform", 0.5, 1.5), beta=("uniform", -0.1, 0.1),
                  residual=("normal", 1.0)),
    ),
    "F4": dict(
        workload="rows_softmax_bf16",
        contraction="rowwise", in_dtype="bf16", out_dtype="bf16",
        M=8192, N=8192,
        ops=[("row_softmax",)],
        dist=dict(a=("normal", 1.0)),
    ),
    # the loss operators of the reduction categories (Table 2): per-row
    # cross-entropy against class-index targets, over stored bf16 logits
    # [8192, 16384], and fused behind a GEMM + bias that produces the logits
    # (x [4096, 4096] times W [4096, 16384]: a classifier head) so that the
    # logits never reach memory
    "F5": dict(
        workload="rows_cross_entropy_bf16",
        contraction="rowwise", in_dtype="bf16", out_dtype="f32",
        M=8192, N=16384,
        ops=[("row_cross_entropy",)],
        dist=dict(a=("normal", 1.0), targets=("classes",)),
    ),
    "F6": dict(
        workload="gemm_bias_cross_entropy_bf16",
        contraction="gemm", in_dtype="bf16", out_dtype="f32", b_layout="kn",
        M=4096, N=16384, K=4096,
        ops=[("bias",), ("row_cross_entropy",)],
        dist=dict(a=("normal", 1.0), b=("normal_invk",), bias=("uniform", -0.1, 0.1), targets=("classes",)),
    ),
}

BASE_SEED = 260530359


def default_seed(name: str) -> int:
    # C1..C5: BASE_SEED + k; the F workloads (the next chains) from + 100
    return BASE_SEED + int(name[1:]) + (100 if name.startswith("F") else 0)


def conv3d_pooled_shape(cfg: dict) -> tuple:
    """Output shape of a conv3d chain: [batch, cout, D', H', W'] after the
    valid 3x3x3 conv and each MaxPool3d(2) (floor mode) of the op list."""
    d, h, w = cfg["D"] - 2, cfg["H"] - 2, cfg["W"] - 2
    for op in cfg["ops"]:
        if op[0] == "maxpool3d2":
            d, h, w = d // 2, h // 2, w // 2
    return (cfg["batch"], cfg["cout"], d, h, w)


def config(name: str, **overrides) -> dict:
    """A copy of workload `name` with shape fields overridden (M, N, K, batch,
    cin, H, W, cout, ops, b_layout, ...)."""
    cfg = copy.deepcopy(CONFIGS[name])
    cfg.update(overrides)
    cfg["name"] = name
    return cfg


def chain(cfg: dict) -> dict:
    """The chain description consumed by both the binding and the oracle."""
    keys = ("contraction", "in_dtype", "out_dtype", "b_layout", "ops",
            "residual_dtype", "scale_a", "scale_b")
    return {k: copy.deepcopy(cfg[k]) for k in keys if k in cfg}


def flops(cfg: dict) -> int:
    """Algorithmic FLOPs: 2 per multiply-add of the contraction only (conv:
    at every pre-pool output position).  Epilogue arithmetic is not counted
    (a row-wise chain has none)."""
    if cfg["contraction"] == "rowwise":
        return 0
    if cfg["contraction"] == "gemm":
        return 2 * cfg["M"] * cfg["N"] * cfg["K"]
    if cfg["contraction"] == "conv3d_3x3x3":
        outs = cfg["batch"] * (cfg["D"] - 2) * (cfg["H"] - 2) * (cfg["W"] - 2)
        return 2 * outs * cfg["cout"] * cfg["cin"] * 27
    return 2 * cfg["batch"] * cfg["H"] * cfg["W"] * cfg["cout"] * cfg["cin"] * 9


# ---------------------------------------------------------------------------
# Storage-format rounding (applied once, before anything is timed)
# ---------------------------------------------------------------------------

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    nan = np.isnan(np.asarray(x, dtype=np.float32))
    return np.where(nan, np.uint16(0x7FC0), rounded).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


E4M3_MAX = 448.0


def f32_to_e4m3_codes(v: np.ndarray) -> np.ndarray:
    """float32 -> OCP E4M3 codes (uint8): round to nearest even, saturating
    to +-448 (finite inputs only).

    Every step is exact in float32: the quantum of a value in [2^E, 2^(E+1))
    is 2^(E-3) (2^-9 below the normal range), so dividing by it, rounding
    half to even (np.rint) and multiplying back only rescales by powers of 2.
    """
    v = np.asarray(v, dtype=np.float32)
    sign = np.signbit(v)
    a = np.minimum(np.abs(v), np.float32(E4M3_MAX))
    _, e = np.frexp(a)                           # a = m * 2^e, m in [0.5, 1)
    E = np.maximum(e - 1, -6)                    # floor(log2 a), clamped to the subnormal range
    q = np.ldexp(np.rint(np.ldexp(a, 3 - E)), E - 3).astype(np.float32)
    q = np.minimum(q, np.float32(E4M3_MAX))
    m2, e2 = np.frexp(q)
    E2 = e2 - 1
    normal = q >= np.float32(2.0 ** -6)
    # normal: q = (1 + f/8) * 2^E2, f = 16 m2 - 8; subnormal: q = f * 2^-9
    mant = np.where(normal, np.rint(m2 * 16 - 8), np.rint(np.ldexp(q, 9))).astype(np.int32)
    e_field = np.where(normal, E2 + 7, 0).astype(np.int32)
    code = (e_field << 3) | mant
    return (code | np.where(sign & (q > 0), 0x80, 0)).astype(np.uint8)


def quantize_e4m3(x: np.ndarray):
    """Per-tensor amax scaling: s = amax|x| / 448 (float32), codes = E4M3(x / s)."""
    x = np.asarray(x, dtype=np.float32)
    amax = np.float32(np.max(np.abs(x))) if x.size else np.float32(0)
    s = np.float32(amax / np.float32(E4M3_MAX)) if amax > 0 else np.float32(1.0)
    return f32_to_e4m3_codes(x / s), float(s)


# ---------------------------------------------------------------------------
# Generation
# ---------------------------------------------------------------------------

def _draw(rng, spec, shape, k_fan_in):
    kind = spec[0]
    if kind == "normal":
        return (rng.standard_normal(shape, dtype=np.float32) * np.float32(np.sqrt(spec[1])))
    if kind == "normal_invk":
        return rng.standard_normal(shape, dtype=np.float32) * np.float32(1.0 / np.sqrt(max(k_fan_in, 1)))  # K = 0: an empty draw
    if kind == "uniform":
        return rng.uniform(spec[1], spec[2], size=shape).astype(np.float32)
    if kind == "classes":  # class indices, uniform over the N columns
        return rng.integers(0, shape[1], size=shape[0]).astype(np.int32)
    raise ValueError(kind)


def rowwise_bytes(cfg: dict) -> int:
    """Algorithmic HBM bytes of a row-wise chain: A and each tensor input read
    once, the output written once."""
    M, N = cfg["M"], cfg["N"]
    es = {"f32": 4, "bf16": 2}
    names = [op[0] for op in cfg["ops"]]
    b = M * N * es[cfg["in_dtype"]]
    b += 4 * N * (("bias" in names) + 2 * ("groupnorm" in names))
    if "residual_add" in names:
        b += M * N * es[cfg.get("residual_dtype", "bf16")]
    if "row_cross_entropy" in names:
        b += 4 * M  # int32 targets
    b += 4 * M if names and names[-1] in ("row_logsumexp", "row_cross_entropy") else M * N * es[cfg["out_dtype"]]
    return b


def shapes(cfg: dict) -> dict:
    if cfg["contraction"] == "rowwise":
        M, N = cfg["M"], cfg["N"]
        return dict(a=(M, N), bias=(N,), gamma=(N,), beta=(N,), residual=(M, N), fan_in=N)
    if cfg["contraction"] == "gemm":
        M, N, K = cfg["M"], cfg["N"], cfg["K"]
        b = (K, N) if cfg.get("b_layout", "kn") == "kn" else (N, K)
        return dict(a=(M, K), b=b, bias=(N,), gamma=(N,), beta=(N,), residual=(M, N), fan_in=K)
    nb, ci, H, W, co = cfg["batch"], cfg["cin"], cfg["H"], cfg["W"], cfg["cout"]
    if cfg["contraction"] == "conv3d_3x3x3":
        D = cfg["D"]
        return dict(a=(nb, ci, D, H, W), b=(co, ci, 3, 3, 3), bias=(co,), fan_in=ci * 27)
    return dict(a=(nb, ci, H, W), b=(co, ci, 3, 3), bias=(co,), gamma=(co,), beta=(co,),
                residual=(nb, co, H // 2, W // 2), fan_in=ci * 9)


def generate(cfg: dict, seed: int | None = None) -> dict:
    """Draw the raw input tensors of a workload.

    Returns a dict with "a", "b" in the storage format of cfg["in_dtype"]
    (float32 array, uint16 bf16 bits, or uint8 e4m3 codes), the float32
    vectors "bias" / "gamma" / "beta" that the ops need, "residual" (bf16
    bits) when the chain has a residual add, and "scale_a" / "scale_b" for
    e4m3 operands.
    """
    seed = default_seed(cfg["name"]) if seed is None else seed
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed)))
    shp = shapes(cfg)
    dist = cfg["dist"]
    names = [op[0] for op in cfg["ops"]]
    out = {}
    raw_a = _draw(rng, dist["a"], shp["a"], shp["fan_in"])
    raw_b = _draw(rng, dist["b"], shp["b"], shp["fan_in"]) if "b" in shp else None
    if "bias" in names:
        out["bias"] = _draw(rng, dist["bias"], shp["bias"], shp["fan_in"])
    if "groupnorm" in names:
        out["gamma"] = _draw(rng, dist["gamma"], shp["gamma"], shp["fan_in"])
        out["beta"] = _draw(rng, dist["beta"], shp["beta"], shp["fan_in"])
    if "residual_add" in names:
        out["residual"] = f32_to_bf16_bits(_draw(rng, dist["residual"], shp["residual"], shp["fan_in"]))
    if "row_cross_entropy" in names:
        out["targets"] = _draw(rng, dist["targets"], (shp["residual"][0], shp["residual"][1]), shp["fan_in"])
    dt = cfg["in_dtype"]
    if raw_b is None:  # a row-wise chain: A only
        if dt not in ("f32", "bf16"):
            raise ValueError(dt)
        out["a"] = raw_a if dt == "f32" else f32_to_bf16_bits(raw_a)
    elif dt == "f32":
        out["a"], out["b"] = raw_a, raw_b
    elif dt == "bf16":
        out["a"], out["b"] = f32_to_bf16_bits(raw_a), f32_to_bf16_bits(raw_b)
    elif dt == "e4m3":
        out["a"], out["scale_a"] = quantize_e4m3(raw_a)
        out["b"], out["scale_b"] = quantize_e4m3(raw_b)
    else:
        raise ValueError(dt)
    return out


def chain_for(cfg: dict, tensors: dict) -> dict:
    """chain(cfg) with the per-tensor fp8 scales of `tensors` filled in."""
    ch = chain(cfg)
    if "scale_a" in tensors:
        ch["scale_a"] = tensors["scale_a"]
        ch["scale_b"] = tensors["scale_b"]
    return ch
