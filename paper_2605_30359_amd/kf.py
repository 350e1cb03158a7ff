"""ctypes binding of libkf.so (include/kf.h): argument marshalling only.

Every step of the fused operation runs in the library's HIP kernels; this
module converts a chain description and torch tensors into the C structs and
passes ``tensor.data_ptr()`` plus the current HIP stream.  torch is used only
for device memory and streams.  If the library has not been built the first
call raises: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libkf.so")

# ---------------------------------------------------------------- C mirror

KF_OK, KF_ERR_INVALID_ARG, KF_ERR_SHAPE, KF_ERR_UNSUPPORTED, KF_ERR_NO_DEVICE, KF_ERR_OOM, KF_ERR_HIP = range(7)
KF_GEMM, KF_CONV2D_3X3, KF_ROWWISE, KF_CONV3D_3X3X3 = 0, 1, 2, 3
CONTRACTIONS = {"gemm": KF_GEMM, "conv2d_3x3": KF_CONV2D_3X3, "rowwise": KF_ROWWISE,
                "conv3d_3x3x3": KF_CONV3D_3X3X3}
KF_F32, KF_BF16, KF_FP8_E4M3, KF_I32 = 0, 1, 2, 3
KF_LAYOUT_KN, KF_LAYOUT_NK = 0, 1
KF_MAX_OPS = 8
KF_MAX_DIMS = 5

OP_KINDS = {
    "bias": 1, "relu": 2, "gelu_tanh": 3, "gelu_erf": 4, "swish": 5, "sigmoid": 6,
    "tanh": 7, "hardtanh": 8, "scale": 9, "groupnorm": 10, "residual_add": 11,
    "maxpool2x2": 12, "row_softmax": 13, "row_logsumexp": 14, "channel_softmax": 15,
    "maxpool3d2": 16, "row_cross_entropy": 17,
}
DTYPES = {"f32": KF_F32, "bf16": KF_BF16, "e4m3": KF_FP8_E4M3, "i32": KF_I32}
DTYPE_NAMES = {v: k for k, v in DTYPES.items()}

EXPORTED = ("kf_create", "kf_fused_op", "kf_fused_op_timed", "kf_unfused_op", "kf_destroy", "kf_num_inputs",
            "kf_input_info", "kf_output_info", "kf_workspace_bytes", "kf_kernel_name",
            "kf_status_string", "kf_last_error", "kf_classify", "kf_diagnose", "kf_get_tuning", "kf_set_tuning",
            "kf_autotune", "kf_weights_changed", "kf_fused_op_noalloc", "kf_diagnose_counters", "kf_probe_mfma",
            "kf_probe_copy", "kf_set_clock_stamps", "kf_wall_clock_hz")
BOUNDS = {0: "memory", 1: "instruction", 2: "latency"}
HINTS = {1: "reuse", 2: "parallelism", 4: "pipeline", 8: "overlap", 16: "lds_layout"}
KF_MAX_TUNE_CANDIDATES = 32


class KfOp(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("groups", ctypes.c_int32),
                ("p0", ctypes.c_float), ("p1", ctypes.c_float)]


class KfOpSpec(ctypes.Structure):
    _fields_ = [("contraction", ctypes.c_int32), ("in_dtype", ctypes.c_int32),
                ("out_dtype", ctypes.c_int32), ("b_layout", ctypes.c_int32),
                ("M", ctypes.c_int64), ("N", ctypes.c_int64), ("K", ctypes.c_int64),
                ("batch", ctypes.c_int64), ("cin", ctypes.c_int64), ("height", ctypes.c_int64),
                ("width", ctypes.c_int64), ("cout", ctypes.c_int64), ("depth", ctypes.c_int64),
                ("scale_a", ctypes.c_float), ("scale_b", ctypes.c_float),
                ("residual_dtype", ctypes.c_int32), ("n_ops", ctypes.c_int32),
                ("ops", KfOp * KF_MAX_OPS)]


class KfTensor(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("dtype", ctypes.c_int32), ("ndim", ctypes.c_int32),
                ("shape", ctypes.c_int64 * KF_MAX_DIMS), ("stride", ctypes.c_int64 * KF_MAX_DIMS)]


class KfDiagnosis(ctypes.Structure):
    _fields_ = [(n, ctypes.c_double) for n in ("flops", "bytes", "seconds", "tflops", "gbps", "peak_tflops",
                                               "peak_gbps", "compute_frac", "memory_frac", "intensity", "ridge")] + \
               [("workgroups", ctypes.c_int64), ("compute_units", ctypes.c_int32), ("bound", ctypes.c_int32),
                ("mfma_busy", ctypes.c_double), ("lds_conflict", ctypes.c_double), ("traffic_ratio", ctypes.c_double),
                ("hints", ctypes.c_uint32), ("reserved", ctypes.c_int32)]

    def as_dict(self) -> dict:
        d = {n: getattr(self, n) for n, _ in self._fields_ if n != "reserved"}
        d["bound"] = BOUNDS[self.bound]
        d["hints"] = [name for bit, name in HINTS.items() if self.hints & bit]
        return d


class KfCounters(ctypes.Structure):
    _fields_ = [(n, ctypes.c_double) for n in ("kernel_seconds", "hbm_bytes", "mfma_busy", "lds_conflict")]


class KfTuning(ctypes.Structure):
    _fields_ = [("raster_group", ctypes.c_int32), ("xcd_remap", ctypes.c_int32), ("wg_per_cu", ctypes.c_int32),
                ("variant", ctypes.c_int32)]

    def as_dict(self) -> dict:
        return {"raster_group": self.raster_group, "xcd_remap": self.xcd_remap, "wg_per_cu": self.wg_per_cu,
                "variant": self.variant}


class KfTuneResult(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("best", ctypes.c_int32), ("config", KfTuning * KF_MAX_TUNE_CANDIDATES),
                ("seconds", ctypes.c_double * KF_MAX_TUNE_CANDIDATES),
                ("panel_bytes", ctypes.c_double * KF_MAX_TUNE_CANDIDATES)]


class KfMfmaProbe(ctypes.Structure):
    _fields_ = [("tflops", ctypes.c_double), ("seconds", ctypes.c_double), ("clock_ghz", ctypes.c_double),
                ("workgroups", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class KfCopyProbe(ctypes.Structure):
    _fields_ = [("gbps", ctypes.c_double), ("seconds", ctypes.c_double)]


class KFError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{status_string(status)} -- {message}")
        self.status = status


_lib = None


def lib():
    """Load libkf.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2605_30359_amd.build` (there is no fallback path)")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32 = ctypes.c_void_p, ctypes.c_int32
        L.kf_create.argtypes = [ctypes.POINTER(KfOpSpec), ctypes.POINTER(vp)]
        L.kf_create.restype = i32
        L.kf_fused_op.argtypes = [vp, ctypes.POINTER(KfTensor), ctypes.POINTER(KfTensor), vp]
        L.kf_fused_op.restype = i32
        L.kf_fused_op_timed.argtypes = [vp, ctypes.POINTER(KfTensor), ctypes.POINTER(KfTensor), vp, vp, vp]
        L.kf_fused_op_timed.restype = i32
        L.kf_unfused_op.argtypes = [vp, ctypes.POINTER(KfTensor), ctypes.POINTER(KfTensor), vp]
        L.kf_unfused_op.restype = i32
        L.kf_weights_changed.argtypes = [vp]
        L.kf_weights_changed.restype = None
        L.kf_fused_op_noalloc.argtypes = [ctypes.POINTER(KfOpSpec), ctypes.POINTER(KfTensor),
                                          ctypes.POINTER(KfTensor), vp]
        L.kf_fused_op_noalloc.restype = i32
        L.kf_destroy.argtypes = [vp]
        L.kf_destroy.restype = None
        L.kf_num_inputs.argtypes = [vp]
        L.kf_num_inputs.restype = i32
        L.kf_input_info.argtypes = [vp, i32, ctypes.POINTER(i32), ctypes.POINTER(i32), ctypes.c_int64 * KF_MAX_DIMS]
        L.kf_input_info.restype = i32
        L.kf_output_info.argtypes = [vp, ctypes.POINTER(i32), ctypes.POINTER(i32), ctypes.c_int64 * KF_MAX_DIMS]
        L.kf_output_info.restype = i32
        L.kf_workspace_bytes.argtypes = [vp]
        L.kf_workspace_bytes.restype = ctypes.c_size_t
        L.kf_kernel_name.argtypes = [vp]
        L.kf_kernel_name.restype = ctypes.c_char_p
        L.kf_status_string.argtypes = [i32]
        L.kf_status_string.restype = ctypes.c_char_p
        L.kf_last_error.argtypes = []
        L.kf_last_error.restype = ctypes.c_char_p
        dbl = ctypes.c_double
        L.kf_classify.argtypes = [dbl, dbl, dbl, dbl, dbl, ctypes.c_int64, i32, ctypes.POINTER(KfDiagnosis)]
        L.kf_classify.restype = i32
        L.kf_diagnose.argtypes = [vp, dbl, dbl, ctypes.POINTER(KfDiagnosis)]
        L.kf_diagnose.restype = i32
        L.kf_diagnose_counters.argtypes = [vp, ctypes.POINTER(KfCounters), ctypes.POINTER(KfDiagnosis)]
        L.kf_diagnose_counters.restype = i32
        L.kf_probe_mfma.argtypes = [i32, ctypes.c_int64, ctypes.POINTER(KfMfmaProbe)]
        L.kf_probe_mfma.restype = i32
        L.kf_probe_copy.argtypes = [ctypes.c_int64, i32, ctypes.POINTER(KfCopyProbe)]
        L.kf_probe_copy.restype = i32
        L.kf_set_clock_stamps.argtypes = [vp, vp, ctypes.c_int64]
        L.kf_set_clock_stamps.restype = i32
        L.kf_wall_clock_hz.argtypes = []
        L.kf_wall_clock_hz.restype = ctypes.c_int64
        L.kf_get_tuning.argtypes = [vp, ctypes.POINTER(KfTuning)]
        L.kf_get_tuning.restype = i32
        L.kf_set_tuning.argtypes = [vp, ctypes.POINTER(KfTuning)]
        L.kf_set_tuning.restype = i32
        L.kf_autotune.argtypes = [vp, ctypes.POINTER(KfTensor), ctypes.POINTER(KfTensor), vp, i32,
                                  ctypes.POINTER(KfTuneResult)]
        L.kf_autotune.restype = i32
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().kf_status_string(status).decode()


def last_error() -> str:
    return lib().kf_last_error().decode()


def _check(status: int):
    if status != KF_OK:
        raise KFError(status, last_error())


def classify(flops: float, bytes_: float, seconds: float, peak_tflops: float, peak_gbps: float,
             workgroups: int, compute_units: int) -> dict:
    """kf_classify: the bound of a kernel from its work, time and launch."""
    g = KfDiagnosis()
    _check(lib().kf_classify(flops, bytes_, seconds, peak_tflops, peak_gbps, workgroups, compute_units,
                             ctypes.byref(g)))
    return g.as_dict()


# ------------------------------------------------------------ spec building

def make_spec(chain: dict, *, M=0, N=0, K=0, batch=0, cin=0, D=0, H=0, W=0, cout=0) -> KfOpSpec:
    """Fill a kf_op_spec from a chain description (see paper_2605_30359_amd.inputs)."""
    s = KfOpSpec()
    s.contraction = CONTRACTIONS[chain["contraction"]]
    s.in_dtype = DTYPES[chain["in_dtype"]]
    s.out_dtype = DTYPES[chain.get("out_dtype", "f32")]
    s.b_layout = KF_LAYOUT_NK if chain.get("b_layout", "kn") == "nk" else KF_LAYOUT_KN
    s.M, s.N, s.K = M, N, K
    s.batch, s.cin, s.height, s.width, s.cout = batch, cin, H, W, cout
    s.depth = D
    s.scale_a = float(chain.get("scale_a", 1.0))
    s.scale_b = float(chain.get("scale_b", 1.0))
    s.residual_dtype = DTYPES[chain.get("residual_dtype", "bf16")]
    ops = chain["ops"]
    if len(ops) > KF_MAX_OPS:
        raise ValueError(f"at most {KF_MAX_OPS} ops")
    s.n_ops = len(ops)
    for i, op in enumerate(ops):
        name, params = op[0], op[1:]
        s.ops[i].kind = OP_KINDS[name]
        if name == "hardtanh":
            s.ops[i].p0, s.ops[i].p1 = float(params[0]), float(params[1])
        elif name == "scale":
            s.ops[i].p0 = float(params[0])
        elif name == "groupnorm":
            s.ops[i].groups = int(params[0])
            s.ops[i].p0 = float(params[1])
    return s


def input_names(chain: dict) -> list:
    """Input slot order: A, B (no B for a row-wise chain), then the tensors
    the ops need, in op order."""
    names = ["a"] if chain["contraction"] == "rowwise" else ["a", "b"]
    for op in chain["ops"]:
        if op[0] == "bias":
            names.append("bias")
        elif op[0] == "groupnorm":
            names += ["gamma", "beta"]
        elif op[0] == "residual_add":
            names.append("residual")
        elif op[0] == "row_cross_entropy":
            names.append("targets")
    return names


def sizes_of(cfg: dict) -> dict:
    if cfg["contraction"] == "gemm":
        return dict(M=cfg["M"], N=cfg["N"], K=cfg["K"])
    if cfg["contraction"] == "rowwise":
        return dict(M=cfg["M"], N=cfg["N"])
    if cfg["contraction"] == "conv3d_3x3x3":
        return dict(batch=cfg["batch"], cin=cfg["cin"], D=cfg["D"], H=cfg["H"], W=cfg["W"], cout=cfg["cout"])
    return dict(batch=cfg["batch"], cin=cfg["cin"], H=cfg["H"], W=cfg["W"], cout=cfg["cout"])


# ------------------------------------------------------------ tensors

def _torch():
    import torch
    return torch


def torch_dtype(code: int):
    torch = _torch()
    return {KF_F32: torch.float32, KF_BF16: torch.bfloat16, KF_FP8_E4M3: torch.float8_e4m3fn, KF_I32: torch.int32}[code]


def device_tensor(arr: np.ndarray, dtype: str, device="cuda", channels_last=False):
    """Copy raw storage (float32 / bf16 bits as uint16 / e4m3 codes as uint8)
    to the device as a tensor of the matching torch dtype.  channels_last: a
    5-D [N, C, D, H, W] array is stored as [N][D][H][W][C] (the strides of
    torch.channels_last_3d), transposed on the host."""
    torch = _torch()
    if channels_last:
        t = device_tensor(np.ascontiguousarray(np.moveaxis(arr, 1, -1)), dtype, device)
        return t.permute(0, 4, 1, 2, 3)
    arr = np.ascontiguousarray(arr)
    if dtype == "f32":
        return torch.from_numpy(arr.astype(np.float32, copy=False)).to(device)
    if dtype == "bf16":
        return torch.from_numpy(arr.view(np.int16)).to(device).view(torch.bfloat16)
    if dtype == "e4m3":
        return torch.from_numpy(arr.view(np.uint8)).to(device).view(torch.float8_e4m3fn)
    if dtype == "i32":
        return torch.from_numpy(arr.astype(np.int32, copy=False)).to(device)
    raise ValueError(dtype)


def to_kf_tensor(t) -> KfTensor:
    torch = _torch()
    codes = {torch.float32: KF_F32, torch.bfloat16: KF_BF16, torch.float8_e4m3fn: KF_FP8_E4M3, torch.int32: KF_I32}
    if t.dtype not in codes:
        raise TypeError(f"unsupported tensor dtype {t.dtype}")
    if t.dim() < 1 or t.dim() > KF_MAX_DIMS:
        raise ValueError(f"tensors must have 1..{KF_MAX_DIMS} dimensions")
    k = KfTensor()
    k.data = t.data_ptr()
    k.dtype = codes[t.dtype]
    k.ndim = t.dim()
    for i in range(t.dim()):
        k.shape[i] = t.shape[i]
        k.stride[i] = t.stride(i)
    return k


class FusedOp:
    """One planned fused operation (kf_create / kf_fused_op / kf_destroy)."""

    def __init__(self, chain: dict, **sizes):
        self.chain = chain
        self.sizes = sizes
        self._spec = make_spec(chain, **sizes)
        self._marshalled = None  # (key, inputs array, output array) of the last call
        h = ctypes.c_void_p()
        _check(lib().kf_create(ctypes.byref(self._spec), ctypes.byref(h)))
        self._h = h

    @classmethod
    def from_config(cls, cfg: dict, chain: dict | None = None):
        from . import inputs
        return cls(chain if chain is not None else inputs.chain(cfg), **sizes_of(cfg))

    def close(self):
        if getattr(self, "_h", None):
            lib().kf_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def num_inputs(self) -> int:
        return lib().kf_num_inputs(self._h)

    def input_info(self, slot: int):
        dt, nd, shp = ctypes.c_int32(), ctypes.c_int32(), (ctypes.c_int64 * KF_MAX_DIMS)()
        _check(lib().kf_input_info(self._h, slot, ctypes.byref(dt), ctypes.byref(nd), shp))
        return DTYPE_NAMES[dt.value], tuple(shp[i] for i in range(nd.value))

    def output_info(self):
        dt, nd, shp = ctypes.c_int32(), ctypes.c_int32(), (ctypes.c_int64 * KF_MAX_DIMS)()
        _check(lib().kf_output_info(self._h, ctypes.byref(dt), ctypes.byref(nd), shp))
        return DTYPE_NAMES[dt.value], tuple(shp[i] for i in range(nd.value))

    def workspace_bytes(self) -> int:
        return int(lib().kf_workspace_bytes(self._h))

    def kernel_name(self) -> str:
        return lib().kf_kernel_name(self._h).decode()

    def empty_output(self, device="cuda"):
        torch = _torch()
        dt, shp = self.output_info()
        return torch.empty(shp, dtype=torch_dtype(DTYPES[dt]), device=device)

    def _call(self, fn, inputs, out, stream, events=None):
        torch = _torch()
        if out is None:
            out = self.empty_output(inputs[0].device)
        # The descriptors of the last call are reused when every tensor has
        # the same address, dtype, shape and strides (a loop over the same
        # buffers): building them costs more host time than a small launch.
        key = tuple((t.data_ptr(), t.dtype, t.shape, t.stride()) for t in (*inputs, out))
        if self._marshalled is not None and self._marshalled[0] == key:
            arr, o = self._marshalled[1], self._marshalled[2]
        else:
            arr = (KfTensor * max(1, len(inputs)))(*[to_kf_tensor(t) for t in inputs])
            o = (KfTensor * 1)(to_kf_tensor(out))
            self._marshalled = (key, arr, o)
        if stream is None:
            stream = torch.cuda.current_stream(out.device).cuda_stream
        elif not isinstance(stream, int):
            stream = stream.cuda_stream
        if events is None:
            _check(fn(self._h, arr, o, ctypes.c_void_p(stream)))
        else:
            _check(fn(self._h, arr, o, ctypes.c_void_p(stream), ctypes.c_void_p(events[0]), ctypes.c_void_p(events[1])))
        return out

    def __call__(self, inputs, out=None, stream=None):
        return self._call(lib().kf_fused_op, inputs, out, stream)

    def timed(self, inputs, out, ev_before: int, ev_after: int, stream=None):
        """Like __call__, recording two caller-created hipEvent_t handles
        around the main contraction kernel."""
        return self._call(lib().kf_fused_op_timed, inputs, out, stream, (ev_before, ev_after))

    def unfused(self, inputs, out=None, stream=None):
        return self._call(lib().kf_unfused_op, inputs, out, stream)

    def set_clock_stamps(self, stamps=None):
        """kf_set_clock_stamps with a device int64 tensor of 6 x workgroups
        values (None: off)."""
        if stamps is None:
            _check(lib().kf_set_clock_stamps(self._h, None, 0))
        else:
            _check(lib().kf_set_clock_stamps(self._h, ctypes.c_void_p(stamps.data_ptr()), stamps.numel() // 6))
        self._stamps = stamps

    def clock_stamps(self, launch, workgroups: int, calls: int = 20, mfma_cycles: float = 0.0) -> dict:
        """Run launch() `calls` times with clock stamps on (a fresh device
        buffer for `workgroups` workgroups), then turn them off; returns, over
        the workgroups of the last call, the median shader clock (GHz) and
        tile time (us), and the median shares of prologue, K loop and
        epilogue in a tile's shader cycles, from kf_set_clock_stamps'
        counters.  With mfma_cycles (the matrix-core issue cycles of one tile)
        also the matrix cores' busy share of the tile and of its K loop."""
        torch = _torch()
        import numpy as np
        buf = torch.zeros(6 * workgroups, dtype=torch.int64, device="cuda")
        self.set_clock_stamps(buf)
        try:
            for _ in range(calls):
                launch()
            torch.cuda.synchronize()
        finally:
            self.set_clock_stamps(None)
        a = buf.view(workgroups, 6).cpu().numpy()
        a = a[(a[:, 3] > a[:, 2]) & (a[:, 1] > a[:, 0])]
        hz = float(lib().kf_wall_clock_hz())
        if a.size == 0 or hz <= 0:
            return {"error": "no stamps recorded"}
        secs = (a[:, 3] - a[:, 2]) / hz
        ghz = (a[:, 1] - a[:, 0]) / secs * 1e-9
        cyc = (a[:, 1] - a[:, 0]).astype(np.float64)
        kloop = (a[:, 5] - a[:, 4]).astype(np.float64)
        r = {"workgroups": int(a.shape[0]), "clock_ghz_median": float(np.median(ghz)),
             "clock_ghz_min": float(ghz.min()), "clock_ghz_max": float(ghz.max()),
             "tile_us_median": float(np.median(secs) * 1e6),
             "tile_cycles_median": float(np.median(cyc)),
             "prologue_share": float(np.median((a[:, 4] - a[:, 0]) / cyc)),
             "k_loop_share": float(np.median(kloop / cyc)),
             "epilogue_share": float(np.median((a[:, 1] - a[:, 5]) / cyc))}
        if mfma_cycles > 0:
            r["mfma_busy_in_tile"] = float(mfma_cycles / np.median(cyc))
            r["mfma_busy_in_k_loop"] = float(mfma_cycles / np.median(kloop))
        return r

    def weights_changed(self):
        """kf_weights_changed: B was rewritten in place; the next call repacks it."""
        lib().kf_weights_changed(self._h)

    def diagnose(self, kernel_seconds: float, hbm_bytes: float = 0.0) -> dict:
        g = KfDiagnosis()
        _check(lib().kf_diagnose(self._h, kernel_seconds, hbm_bytes or 0.0, ctypes.byref(g)))
        return g.as_dict()

    def diagnose_counters(self, kernel_seconds: float, hbm_bytes: float = -1.0, mfma_busy: float = -1.0,
                          lds_conflict: float = -1.0) -> dict:
        """kf_diagnose_counters: the diagnosis from a launch's counters."""
        g = KfDiagnosis()
        c = KfCounters(kernel_seconds, hbm_bytes, mfma_busy, lds_conflict)
        _check(lib().kf_diagnose_counters(self._h, ctypes.byref(c), ctypes.byref(g)))
        return g.as_dict()

    def tuning(self) -> dict:
        t = KfTuning()
        _check(lib().kf_get_tuning(self._h, ctypes.byref(t)))
        return t.as_dict()

    def set_tuning(self, raster_group: int, xcd_remap: int, wg_per_cu: int, variant: int = 0):
        t = KfTuning(raster_group, xcd_remap, wg_per_cu, variant)
        _check(lib().kf_set_tuning(self._h, ctypes.byref(t)))

    def autotune(self, inputs, out, reps: int = 5, stream=None) -> dict:
        """kf_autotune: time the plan's launch candidates, keep the fastest."""
        torch = _torch()
        arr = (KfTensor * max(1, len(inputs)))(*[to_kf_tensor(t) for t in inputs])
        o = (KfTensor * 1)(to_kf_tensor(out))
        if stream is None:
            stream = torch.cuda.current_stream(out.device).cuda_stream
        elif not isinstance(stream, int):
            stream = stream.cuda_stream
        r = KfTuneResult()
        _check(lib().kf_autotune(self._h, arr, o, ctypes.c_void_p(stream), reps, ctypes.byref(r)))
        cands = [dict(r.config[i].as_dict(), seconds=r.seconds[i], panel_bytes=r.panel_bytes[i]) for i in range(r.n)]
        return {"best": cands[r.best], "candidates": cands}

    def device_inputs(self, tensors: dict, device="cuda", conv3d_channels_last=True) -> list:
        """Marshal raw generated storage into the slot order of this op (a
        conv3d input channels-last unless conv3d_channels_last is False)."""
        out = []
        for name in input_names(self.chain):
            if name in ("a", "b"):
                dt = self.chain["in_dtype"]
            elif name == "residual":
                dt = self.chain.get("residual_dtype", "bf16")
            elif name == "targets":
                dt = "i32"
            else:
                dt = "f32"
            cl = name == "a" and self.chain["contraction"] == "conv3d_3x3x3" and conv3d_channels_last
            out.append(device_tensor(tensors[name], dt, device, channels_last=cl))
        return out


def fused_op_noalloc(chain: dict, inputs, out, stream=None, **sizes):
    """kf_fused_op_noalloc: plan `chain` on the stack and run it with the
    library's static device scratch -- no allocation anywhere, for callers
    that cannot allocate.  `inputs` / `out` are device tensors in the slot
    order of FusedOp.device_inputs; returns `out`."""
    torch = _torch()
    spec = make_spec(chain, **sizes)
    arr = (KfTensor * max(1, len(inputs)))(*[to_kf_tensor(t) for t in inputs])
    o = (KfTensor * 1)(to_kf_tensor(out))
    if stream is None:
        stream = torch.cuda.current_stream(out.device).cuda_stream
    elif not isinstance(stream, int):
        stream = stream.cuda_stream
    _check(lib().kf_fused_op_noalloc(ctypes.byref(spec), arr, o, ctypes.c_void_p(stream)))
    return out


def fused_op_noalloc_status(chain: dict, **sizes) -> tuple:
    """(status, message) of kf_fused_op_noalloc for `chain` with no tensors
    bound (NULL-free empty descriptors): the host-side planning and scratch
    size checks, which run before any device call."""
    spec = make_spec(chain, **sizes)
    arr = (KfTensor * 8)()
    o = (KfTensor * 1)()
    st = lib().kf_fused_op_noalloc(ctypes.byref(spec), arr, o, None)
    return st, last_error()


def probe_mfma(in_dtype: str, iters: int) -> dict:
    """kf_probe_mfma: the matrix cores' sustained rate for "bf16" or "e4m3"
    MFMAs with no memory traffic, and the shader clock they ran at."""
    r = KfMfmaProbe()
    _check(lib().kf_probe_mfma(DTYPES[in_dtype], int(iters), ctypes.byref(r)))
    return {"dtype": in_dtype, "tflops": r.tflops, "seconds": r.seconds, "clock_ghz": r.clock_ghz,
            "workgroups": r.workgroups}


def probe_copy(nbytes: int, reps: int) -> dict:
    """kf_probe_copy: a plain device copy of nbytes, GB/s counting read and
    write."""
    r = KfCopyProbe()
    _check(lib().kf_probe_copy(int(nbytes), int(reps), ctypes.byref(r)))
    return {"gbps": r.gbps, "seconds": r.seconds, "bytes": int(nbytes)}
