"""fp64 CPU oracle for the fused contraction + epilogue chains.

TEST INFRASTRUCTURE ONLY.  Only the test suite, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this package.  The product path
(the HIP library and its Python binding) never imports, links or calls it, and
this package imports nothing from the product path.

What it computes.  The paper (Methodology, Overview; Evaluation, Metrics) takes
as its task a PyTorch operator given as a reference computation, and accepts a
candidate kernel when its outputs are numerically equivalent to that reference.
The operators in scope are the fusion patterns named in Appendix A ("Operator
Fusion": matmul + activation, normalisation + activation, softmax; "Algorithmic
Optimization": online softmax, reduced precision): a dense contraction (GEMM,
a 3x3 convolution, or the 3x3x3 convolution of the Conv3d -> channel softmax ->
max-pool operator of the Appendix C case study) followed by an ordered list of
epilogue ops.  The method
reaches the plain result of that reference, so this oracle is the plain
definition of each step, applied in the listed order, in float64:

* inputs are the exact bit patterns the GPU receives (fp32, bf16, OCP e4m3),
  widened exactly to float64 (``to_f64``);
* the contraction is plain C with ascending-index sums (``kf_oracle.c``);
* each epilogue op below is the textbook / PyTorch definition of that op.

Where the paper is silent the readings are: GEMM operands x[M,K] and W[K,N]
(layout "kn") or W[N,K] (layout "nk"); GroupNorm on a 2-D [rows, C] tensor
follows nn.GroupNorm with C channels per row (biased variance, eps inside the
square root); softmax and logsumexp run over the last axis; swish is x*sigmoid(x);
GELU(tanh) is the tanh approximation; fp8 operands are dequantised by their
per-tensor fp32 scale before the contraction.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_SRC = os.path.join(_HERE, "kf_oracle.c")


def build(force: bool = True) -> str:
    """Compile ``kf_oracle.c`` to ``liboracle.so`` (gcc, OpenMP)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(
            ["gcc", "-O3", "-march=x86-64-v3", "-fopenmp", "-fPIC", "-shared",
             "-o", tmp, _SRC])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=False)
        lib = ctypes.CDLL(_LIB_PATH)
        p = ctypes.c_void_p
        i64 = ctypes.c_int64
        lib.kfo_gemm_rows.argtypes = [p, p, i64, i64, i64, ctypes.c_int, p, i64, p]
        lib.kfo_gemm_rows.restype = None
        lib.kfo_conv2d_3x3.argtypes = [p, p, i64, i64, i64, i64, i64, p, i64, p]
        lib.kfo_conv2d_3x3.restype = None
        lib.kfo_conv3d_3x3x3.argtypes = [p, p, i64, i64, i64, i64, i64, i64, p, i64, p]
        lib.kfo_conv3d_3x3x3.restype = None
        lib.kfo_max_threads.argtypes = []
        lib.kfo_max_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def threads() -> int:
    """OpenMP threads the contraction uses."""
    return int(_load().kfo_max_threads())


# --------------------------------------------------------------------------
# Exact widening of the input encodings
# --------------------------------------------------------------------------

def decode_bf16(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> float64.  bf16 is the upper half of
    an IEEE binary32, so the value is the binary32 whose low 16 bits are 0."""
    bits = np.asarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def decode_e4m3(codes: np.ndarray) -> np.ndarray:
    """OCP FP8 E4M3 ("e4m3fn") codes (uint8) -> float64, from the format
    definition: 1 sign bit, 4 exponent bits with bias 7, 3 mantissa bits;
    exponent field 0 is subnormal (m/8 * 2^-6); S.1111.111 is NaN; there are no
    infinities, so the largest finite magnitude is 1.75 * 2^8 = 448."""
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    sign = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 0xF
    m = (c & 0x7).astype(np.float64)
    normal = (1.0 + m / 8.0) * np.exp2((e - 7).astype(np.float64))
    sub = (m / 8.0) * 2.0 ** (1 - 7)
    v = sign * np.where(e == 0, sub, normal)
    return np.where((e == 15) & ((c & 0x7) == 7), np.nan, v)


def to_f64(arr: np.ndarray, dtype: str) -> np.ndarray:
    """Widen raw input storage to float64 exactly."""
    if dtype == "f32":
        return np.asarray(arr, dtype=np.float32).astype(np.float64)
    if dtype == "bf16":
        return decode_bf16(arr)
    if dtype == "e4m3":
        return decode_e4m3(arr)
    if dtype == "f64":
        return np.asarray(arr, dtype=np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


# --------------------------------------------------------------------------
# Contractions (plain C, ascending sums)
# --------------------------------------------------------------------------

def gemm(a: np.ndarray, b: np.ndarray, layout: str = "kn", rows=None) -> np.ndarray:
    """h = a @ b for a[M,K] and b[K,N] ("kn") or b[N,K] ("nk", h = a @ b^T),
    restricted to the selected rows of a (all rows by default)."""
    a = np.ascontiguousarray(a, dtype=np.float64)
    b = np.ascontiguousarray(b, dtype=np.float64)
    M, K = a.shape
    if layout == "kn":
        assert b.shape[0] == K
        N = b.shape[1]
    elif layout == "nk":
        assert b.shape[1] == K
        N = b.shape[0]
    else:
        raise ValueError(layout)
    rows = np.arange(M, dtype=np.int64) if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
    assert rows.size == 0 or (rows.min() >= 0 and rows.max() < M)
    out = np.empty((rows.size, N), dtype=np.float64)
    if rows.size and N:
        _load().kfo_gemm_rows(a.ctypes.data, b.ctypes.data, M, N, K,
                              1 if layout == "nk" else 0, rows.ctypes.data,
                              rows.size, out.ctypes.data)
    elif rows.size:
        pass
    return out


def conv2d_3x3(x: np.ndarray, w: np.ndarray, images=None) -> np.ndarray:
    """PyTorch Conv2d (cross-correlation) with a 3x3 kernel, stride 1, zero
    padding 1, no bias: x[Nb,Cin,H,W], w[Cout,Cin,3,3] -> [n_sel,Cout,H,W]."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    w = np.ascontiguousarray(w, dtype=np.float64)
    Nb, Cin, H, W = x.shape
    Cout = w.shape[0]
    assert w.shape == (Cout, Cin, 3, 3)
    images = np.arange(Nb, dtype=np.int64) if images is None else np.ascontiguousarray(images, dtype=np.int64)
    out = np.empty((images.size, Cout, H, W), dtype=np.float64)
    if images.size:
        _load().kfo_conv2d_3x3(x.ctypes.data, w.ctypes.data, Nb, Cin, H, W, Cout,
                               images.ctypes.data, images.size, out.ctypes.data)
    return out


def conv3d_3x3x3(x: np.ndarray, w: np.ndarray, images=None) -> np.ndarray:
    """PyTorch Conv3d (cross-correlation) with a 3x3x3 kernel, stride 1, no
    padding, no bias: x[Nb,Cin,D,H,W], w[Cout,Cin,3,3,3] ->
    [n_sel,Cout,D-2,H-2,W-2]."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    w = np.ascontiguousarray(w, dtype=np.float64)
    Nb, Cin, D, H, W = x.shape
    Cout = w.shape[0]
    assert w.shape == (Cout, Cin, 3, 3, 3) and min(D, H, W) >= 3
    images = np.arange(Nb, dtype=np.int64) if images is None else np.ascontiguousarray(images, dtype=np.int64)
    out = np.empty((images.size, Cout, D - 2, H - 2, W - 2), dtype=np.float64)
    if images.size:
        _load().kfo_conv3d_3x3x3(x.ctypes.data, w.ctypes.data, Nb, Cin, D, H, W, Cout,
                                 images.ctypes.data, images.size, out.ctypes.data)
    return out


# --------------------------------------------------------------------------
# Epilogue ops (each the plain definition; float64 throughout)
# --------------------------------------------------------------------------

def _channel_shape(h: np.ndarray) -> tuple:
    # Per-channel parameters broadcast along axis 1 of an NCHW / NCDHW
    # tensor, and along the last axis (output features) of a 2-D GEMM output.
    return (1, -1) + (1,) * (h.ndim - 2) if h.ndim >= 4 else (1, -1)


def op_bias(h, bias):
    """h + b, b per output feature (GEMM column) or per output channel (conv)."""
    return h + np.asarray(bias, np.float64).reshape(_channel_shape(h))


def op_relu(h):
    """max(h, 0)."""
    return np.maximum(h, 0.0)


def op_gelu_tanh(h):
    """Tanh-approximate GELU: 0.5 h (1 + tanh(sqrt(2/pi) (h + 0.044715 h^3)))."""
    return 0.5 * h * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (h + 0.044715 * h ** 3)))


def op_gelu_erf(h):
    """Exact GELU: h * Phi(h) = 0.5 h (1 + erf(h / sqrt 2))."""
    from scipy.special import erf
    return 0.5 * h * (1.0 + erf(h / math.sqrt(2.0)))


def op_sigmoid(h):
    """1 / (1 + e^-h), evaluated without overflow."""
    from scipy.special import expit
    return expit(h)


def op_swish(h):
    """Swish with beta = 1: h * sigmoid(h)."""
    return h * op_sigmoid(h)


def op_tanh(h):
    return np.tanh(h)


def op_hardtanh(h, lo=-1.0, hi=1.0):
    """clamp(h, lo, hi)."""
    return np.minimum(np.maximum(h, lo), hi)


def op_scale(h, c):
    return h * c


def op_groupnorm(h, groups, eps, gamma=None, beta=None):
    """nn.GroupNorm: channels (axis 1) split into `groups` contiguous groups;
    per (sample, group): mean mu and biased variance v over the group's
    channels (and spatial positions for 4-D input), then
    (h - mu) / sqrt(v + eps), then the per-channel affine gamma, beta."""
    shp = h.shape
    C = shp[1]
    assert C % groups == 0
    g = h.reshape(shp[0], groups, -1)
    mu = g.mean(axis=2, keepdims=True)
    var = ((g - mu) ** 2).mean(axis=2, keepdims=True)
    n = ((g - mu) / np.sqrt(var + eps)).reshape(shp)
    if gamma is not None:
        n = n * np.asarray(gamma, np.float64).reshape(_channel_shape(h))
    if beta is not None:
        n = n + np.asarray(beta, np.float64).reshape(_channel_shape(h))
    return n


def op_residual_add(h, r):
    return h + np.asarray(r, np.float64).reshape(h.shape)


def op_maxpool2x2(h):
    """MaxPool2d(kernel 2, stride 2, no padding, floor mode) on NCHW."""
    n, c, H, W = h.shape
    Ho, Wo = H // 2, W // 2
    v = h[:, :, :2 * Ho, :2 * Wo].reshape(n, c, Ho, 2, Wo, 2)
    return v.max(axis=(3, 5))


def op_channel_softmax(h):
    """Softmax over the channel axis (axis 1) at every position of an NCDHW
    tensor, as torch.softmax(h, dim=1): e^(h - m) / sum_c e^(h - m), m the
    maximum over the channels at that position."""
    m = h.max(axis=1, keepdims=True)
    e = np.exp(h - m)
    return e / e.sum(axis=1, keepdims=True)


def op_maxpool3d2(h):
    """MaxPool3d(kernel 2, stride 2, no padding, floor mode) on NCDHW."""
    n, c, D, H, W = h.shape
    Do, Ho, Wo = D // 2, H // 2, W // 2
    v = h[:, :, :2 * Do, :2 * Ho, :2 * Wo].reshape(n, c, Do, 2, Ho, 2, Wo, 2)
    return v.max(axis=(3, 5, 7))


def op_row_softmax(h):
    """Softmax over the last axis: e^(h - m) / sum e^(h - m), m the row max."""
    m = h.max(axis=-1, keepdims=True)
    e = np.exp(h - m)
    return e / e.sum(axis=-1, keepdims=True)


def op_row_logsumexp(h):
    """log sum_j e^h_j over the last axis, as m + log sum e^(h - m)."""
    m = h.max(axis=-1, keepdims=True)
    return (m + np.log(np.exp(h - m).sum(axis=-1, keepdims=True)))[..., 0]


def op_row_cross_entropy(h, targets):
    """Cross-entropy of each row against its class index, as
    nn.CrossEntropyLoss(reduction='none') defines it: the row's logsumexp
    minus the row's entry at the target column.  A target outside [0, N)
    gives NaN (the GPU path's documented answer for it)."""
    t = np.asarray(targets, dtype=np.int64)
    N = h.shape[-1]
    ok = (t >= 0) & (t < N)
    picked = np.take_along_axis(h, np.clip(t, 0, N - 1)[:, None], axis=-1)[:, 0]
    return np.where(ok, op_row_logsumexp(h) - picked, np.nan)


# --------------------------------------------------------------------------
# Chains
# --------------------------------------------------------------------------

def _apply_ops(chain: dict, tensors: dict, h: np.ndarray, sel, store=None, first_store: int = 1) -> np.ndarray:
    """The op list of `chain`, in order, on the float64 contraction result h
    (rows / images `sel` of the full result, or all of it).  `store`, if
    given, is applied to the input of every op from index `first_store` on
    (the storage rounding of an intermediate that is written to memory)."""
    ops = chain["ops"]
    for i, op in enumerate(ops):
        if store is not None and i >= first_store:
            h = store(h)
        name, params = op[0], op[1:]
        if name == "bias":
            h = op_bias(h, to_f64(tensors["bias"], "f32"))
        elif name == "relu":
            h = op_relu(h)
        elif name == "gelu_tanh":
            h = op_gelu_tanh(h)
        elif name == "gelu_erf":
            h = op_gelu_erf(h)
        elif name == "swish":
            h = op_swish(h)
        elif name == "sigmoid":
            h = op_sigmoid(h)
        elif name == "tanh":
            h = op_tanh(h)
        elif name == "hardtanh":
            h = op_hardtanh(h, *params)
        elif name == "scale":
            h = op_scale(h, params[0])
        elif name == "groupnorm":
            groups, eps = params[0], params[1]
            h = op_groupnorm(h, groups, eps, to_f64(tensors["gamma"], "f32"),
                             to_f64(tensors["beta"], "f32"))
        elif name == "residual_add":
            r = to_f64(tensors["residual"], chain.get("residual_dtype", "bf16"))
            if sel is not None:
                r = r[np.asarray(sel, dtype=np.int64)]
            h = op_residual_add(h, r)
        elif name == "maxpool2x2":
            h = op_maxpool2x2(h)
        elif name == "channel_softmax":
            h = op_channel_softmax(h)
        elif name == "maxpool3d2":
            h = op_maxpool3d2(h)
        elif name == "row_softmax":
            h = op_row_softmax(h)
        elif name == "row_logsumexp":
            h = op_row_logsumexp(h)
        elif name == "row_cross_entropy":
            t = np.asarray(tensors["targets"], dtype=np.int64)
            if sel is not None:
                t = t[np.asarray(sel, dtype=np.int64)]
            h = op_row_cross_entropy(h, t)
        else:
            raise ValueError(f"unknown op {name!r}")
    return h


# --------------------------------------------------------------------------
# Storage rounding of intermediates (the unfused chain)
# --------------------------------------------------------------------------

def round_bf16(x: np.ndarray) -> np.ndarray:
    """float64 -> the nearest bfloat16 value (round half to even), as float64.

    bfloat16 keeps 8 significant bits and binary32's exponent range: a finite
    value in [2^E, 2^(E+1)) is a multiple of 2^(E-7), and below the normal
    range (E < -126) of 2^-133.  Dividing by that quantum, rounding half to
    even (np.rint) and multiplying back only rescales by powers of two, so
    every step is exact in float64.  Magnitudes that round past the largest
    finite value, (2 - 2^-7) 2^127, become infinite."""
    x = np.asarray(x, dtype=np.float64)
    ax = np.abs(x)
    _, e = np.frexp(ax)                        # ax = m 2^e, m in [0.5, 1)
    E = np.maximum(e - 1, -126)                # floor(log2 ax), clamped to the normal range
    q = np.ldexp(np.rint(np.ldexp(ax, 7 - E)), E - 7)
    q = np.where(q > (2.0 - 2.0 ** -7) * 2.0 ** 127, np.inf, q)
    q = np.where(np.isnan(x), np.nan, q)
    return np.copysign(q, x)


def round_f32(x: np.ndarray) -> np.ndarray:
    """float64 -> the nearest binary32 value (IEEE round half to even)."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def intermediate_dtype(chain: dict) -> str:
    """Storage format of the unfused chain's intermediates: what an eager
    chain of one operator per kernel stores in the operands' precision --
    bfloat16 for bf16 and e4m3 contractions (and bf16 row-wise chains),
    binary32 for fp32 ones."""
    return "f32" if chain["in_dtype"] == "f32" else "bf16"


def run_chain_unfused(chain: dict, tensors: dict, rows=None, images=None, fused: int = 0) -> np.ndarray:
    """The chain as a one-operator-per-kernel evaluation computes it -- the
    unfused form that operator fusion removes (Appendix A, "Operator
    Fusion"): the contraction's result and the result of every op but the
    last are written to memory, so each is rounded to the intermediate
    storage format (``intermediate_dtype``) before the next op reads it.
    Each op itself is the same plain float64 definition as in ``run_chain``,
    applied to the stored values.  A chain with no ops writes the
    contraction's result directly (no intermediate); a row-wise chain's first
    op reads A itself.  The last op's result is returned unrounded, like
    ``run_chain``'s.

    fused > 0: the partly fused evaluation -- the contraction and its first
    `fused` ops run as one kernel (nothing stored between them), the result
    of op fused - 1 is stored, then one kernel per remaining op as above.
    fused = len(ops) is ``run_chain``."""
    store = round_f32 if intermediate_dtype(chain) == "f32" else round_bf16
    h, sel = _contraction(chain, tensors, rows, images)
    if fused == 0 and chain["ops"] and chain["contraction"] != "rowwise":
        h = store(h)
    return _apply_ops(chain, tensors, h, sel, store, first_store=max(fused, 1))


def _contraction(chain: dict, tensors: dict, rows=None, images=None):
    """The float64 contraction result of a chain (A itself for "rowwise"),
    restricted to the selected rows / images, and the selection."""
    dt = chain["in_dtype"]
    a = to_f64(tensors["a"], dt)
    if chain["contraction"] == "rowwise":
        h = a if rows is None else a[np.asarray(rows, dtype=np.int64)]
        return h, rows
    b = to_f64(tensors["b"], dt)
    if dt == "e4m3":
        a = a * float(np.float32(chain["scale_a"]))
        b = b * float(np.float32(chain["scale_b"]))
    if chain["contraction"] == "gemm":
        return gemm(a, b, chain.get("b_layout", "kn"), rows), rows
    if chain["contraction"] == "conv2d_3x3":
        return conv2d_3x3(a, b, images), images
    if chain["contraction"] == "conv3d_3x3x3":
        return conv3d_3x3x3(a, b, images), images
    raise ValueError(chain["contraction"])


def run_chain(chain: dict, tensors: dict, rows=None, images=None) -> np.ndarray:
    """Evaluate one fused chain in float64.

    chain:   {"contraction": "gemm" | "conv2d_3x3" | "conv3d_3x3x3" | "rowwise",
              "in_dtype": "f32" | "bf16"
              | "e4m3", "b_layout": "kn" | "nk", "scale_a": s_x, "scale_b": s_w,
              "ops": [(name, *params), ...]}
    tensors: raw storage: "a", "b" (in_dtype; no "b" for "rowwise", whose h is
             A itself), "bias", "gamma", "beta" (f32),
             "residual" (its own dtype given by chain["residual_dtype"]),
             "targets" (int class indices, one per row).
    rows / images: evaluate only these output rows (GEMM) or batch entries
             (conv); every op in scope is local to a row (GEMM) or to one
             image (conv), so the selected slice is exact.
    """
    h, sel = _contraction(chain, tensors, rows, images)
    return _apply_ops(chain, tensors, h, sel)
