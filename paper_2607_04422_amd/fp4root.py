"""ctypes binding of libfp4root.so (argument marshalling only).

Every function here checks its tensors, passes raw device pointers, sizes and
the current HIP stream to the C entry point of the same name, and raises
``Fp4RootError`` on a non-zero return code.  Device memory for outputs and the
workspace comes from PyTorch; all computation happens in the library's
kernels.  There is no CPU path: without the built library or a GPU every call
raises.
"""
from __future__ import annotations

import ctypes
import os
import re

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libfp4root.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "fp4root.h")

OK = 0
F_CLIP = 1
F_HADAMARD = 2
F_ADAPTIVE46 = 4
F_BF16_PATH = 8
F_STOCHASTIC = 16
F_FP32_ACCUM = 32   # products accumulate in binary32 (MFMA order) instead of exactly
F_DEFAULT = 7


class Fp4RootError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__(f"{where}: {status_string(code)} ({code})")


class Matrix(ctypes.Structure):
    _fields_ = [("in_", ctypes.c_void_p), ("out", ctypes.c_void_p), ("rows", ctypes.c_int64),
                ("cols", ctypes.c_int64), ("ld_in", ctypes.c_int64), ("ld_out", ctypes.c_int64)]


class NsConfig(ctypes.Structure):
    _fields_ = [("steps", ctypes.c_int32), ("coeffs", ctypes.POINTER(ctypes.c_float)),
                ("flags", ctypes.c_uint32), ("clip_quantile", ctypes.c_float),
                ("eps", ctypes.c_float), ("seed", ctypes.c_uint64)]


class Param(ctypes.Structure):
    _fields_ = [("w", ctypes.c_void_p), ("g", ctypes.c_void_p), ("m", ctypes.c_void_p),
                ("m_codes", ctypes.c_void_p), ("m_scales", ctypes.c_void_p), ("m_tensor_scale", ctypes.c_void_p),
                ("rows", ctypes.c_int64), ("cols", ctypes.c_int64), ("scale", ctypes.c_float)]


class RootConfig(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("wd", ctypes.c_float), ("beta", ctypes.c_float),
                ("momentum_flags", ctypes.c_uint32), ("momentum_seed", ctypes.c_uint64), ("step", ctypes.c_int32)]


class NsTrace(ctypes.Structure):
    _fields_ = [(name, ctypes.c_void_p) for name in (
        "qx_codes", "qx_scales", "qx_sg", "qxt_codes", "qxt_scales", "qxt_sg", "A",
        "qa_codes", "qa_scales", "qa_sg", "B", "qb_codes", "qb_scales", "qb_sg")]


_lib = None


def load(path: str = None) -> ctypes.CDLL:
    """Load the library (once): `path`, else $FP4ROOT_LIBRARY, else the in-tree build.
    Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    path = path or os.environ.get("FP4ROOT_LIBRARY") or LIB_PATH
    if not os.path.exists(path):
        raise RuntimeError(f"libfp4root.so not built at {path}; run __graft_entry__.build()")
    lib = ctypes.CDLL(path)
    i64, u32, u64, f32, vp, i32 = (ctypes.c_int64, ctypes.c_uint32, ctypes.c_uint64,
                                   ctypes.c_float, ctypes.c_void_p, ctypes.c_int32)
    sz = ctypes.c_size_t
    lib.fp4root_quantize_workspace.argtypes = [i64, i64, i64, u32]
    lib.fp4root_quantize_workspace.restype = sz
    lib.fp4root_ns_step_workspace.argtypes = [i64, i64, i64, u32]
    lib.fp4root_ns_step_workspace.restype = sz
    lib.fp4root_orthogonalize_workspace.argtypes = [ctypes.POINTER(Matrix), i64, ctypes.POINTER(NsConfig)]
    lib.fp4root_orthogonalize_workspace.restype = sz
    lib.fp4root_quantize.argtypes = [vp, i64, i64, i64, i64, i64, ctypes.c_int, u32, f32, u64, i32,
                                     vp, vp, vp, vp, vp, sz, vp]
    lib.fp4root_quantize.restype = ctypes.c_int
    lib.fp4root_quantize_noalloc.argtypes = [vp, i64, i64, i64, i64, i64, ctypes.c_int, u32, f32, u64, i32,
                                             vp, vp, vp, vp, vp, vp]
    lib.fp4root_quantize_noalloc.restype = ctypes.c_int
    lib.fp4root_ns_step.argtypes = [vp, i64, i64, i64, i64, f32, f32, f32, u32, u64, i32,
                                    ctypes.POINTER(NsTrace), vp, sz, vp]
    lib.fp4root_ns_step.restype = ctypes.c_int
    lib.fp4root_orthogonalize.argtypes = [ctypes.POINTER(Matrix), i64, ctypes.POINTER(NsConfig), vp, sz, vp]
    lib.fp4root_orthogonalize.restype = ctypes.c_int
    lib.fp4root_momentum_workspace.argtypes = [i64, i64, i64]
    lib.fp4root_momentum_workspace.restype = sz
    lib.fp4root_momentum_update.argtypes = [vp, vp, i64, i64, i64, vp, vp, vp, f32, u32, u64, i32, vp, sz, vp]
    lib.fp4root_momentum_update.restype = ctypes.c_int
    lib.fp4root_qadamw_workspace.argtypes = [i64]
    lib.fp4root_qadamw_workspace.restype = sz
    lib.fp4root_qadamw_update.argtypes = [vp, vp, vp, i64, vp, vp, vp, vp, vp, vp, f32, f32, f32, f32, f32,
                                          u32, u64, i32, vp, sz, vp]
    lib.fp4root_qadamw_update.restype = ctypes.c_int
    lib.fp4root_apply_update.argtypes = [vp, vp, i64, f32, f32, f32, vp]
    lib.fp4root_apply_update.restype = ctypes.c_int
    lib.fp4root_root_step_workspace.argtypes = [ctypes.POINTER(Param), i64, ctypes.POINTER(NsConfig)]
    lib.fp4root_root_step_workspace.restype = sz
    lib.fp4root_root_step.argtypes = [ctypes.POINTER(Param), i64, ctypes.POINTER(RootConfig),
                                      ctypes.POINTER(NsConfig), vp, sz, vp]
    lib.fp4root_root_step.restype = ctypes.c_int
    lib.fp4root_default_coeffs.argtypes = [i64, i64, i32, ctypes.POINTER(ctypes.c_float)]
    lib.fp4root_default_coeffs.restype = ctypes.c_int
    lib.fp4root_device_status.argtypes = [vp, vp]
    lib.fp4root_device_status.restype = ctypes.c_int
    lib.fp4root_status_string.argtypes = [ctypes.c_int]
    lib.fp4root_status_string.restype = ctypes.c_char_p
    lib.fp4root_version.argtypes = []
    lib.fp4root_version.restype = ctypes.c_int
    lib.fp4root_set_product_tiling.argtypes = [ctypes.c_int]
    lib.fp4root_set_product_tiling.restype = ctypes.c_int
    lib.fp4root_timer_enable.argtypes = [ctypes.c_int]
    lib.fp4root_timer_enable.restype = ctypes.c_int
    lib.fp4root_timer_read.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_double),
                                       ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_double)]
    lib.fp4root_timer_read.restype = ctypes.c_int
    lib.fp4root_timer_reset.argtypes = []
    lib.fp4root_timer_reset.restype = ctypes.c_int
    _lib = lib
    return lib


def header_symbols(path: str = HEADER) -> list[str]:
    """Names of the functions include/fp4root.h declares."""
    text = open(path).read()
    return sorted(set(re.findall(r"^\s*(?:const char\*|int|size_t)\s+(fp4root_\w+)\s*\(", text, re.M)))


def status_string(code: int) -> str:
    return load().fp4root_status_string(code).decode()


def _check(code: int, where: str):
    if code != OK:
        raise Fp4RootError(code, where)


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _need_gpu_f32(x: torch.Tensor, name: str):
    if not isinstance(x, torch.Tensor) or not x.is_cuda:
        raise TypeError(f"{name} must be a GPU tensor")
    if x.dtype != torch.float32:
        raise TypeError(f"{name} must be float32")


def workspace(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


def fp4root_version() -> int:
    return load().fp4root_version()


def fp4root_set_product_tiling(mode: int) -> int:
    """0: tile form chosen per launch, 1: narrow (32 x 64 per wave), 2: wide (64 x 64)
    for the Gram of qX and the update product; returns the previous mode.  Outputs are
    the same bits in every mode."""
    code = load().fp4root_set_product_tiling(int(mode))
    if code < 0:
        raise Fp4RootError(code, "fp4root_set_product_tiling")
    return code


def fp4root_timer_enable(on: bool = True):
    _check(load().fp4root_timer_enable(1 if on else 0), "fp4root_timer_enable")


def fp4root_timer_read(kernel: int = -1):
    """(total kernel ms, launches, algorithmic FLOP) of the recorded product launches."""
    ms, n, fl = ctypes.c_double(), ctypes.c_int64(), ctypes.c_double()
    _check(load().fp4root_timer_read(kernel, ctypes.byref(ms), ctypes.byref(n), ctypes.byref(fl)),
           "fp4root_timer_read")
    return ms.value, n.value, fl.value


def fp4root_timer_reset():
    _check(load().fp4root_timer_reset(), "fp4root_timer_reset")


def fp4root_default_coeffs(rows: int, cols: int, steps: int = 5):
    buf = (ctypes.c_float * (3 * steps))()
    _check(load().fp4root_default_coeffs(rows, cols, steps, buf), "fp4root_default_coeffs")
    return [(buf[3 * k], buf[3 * k + 1], buf[3 * k + 2]) for k in range(steps)]


def fp4root_device_status(ws: torch.Tensor, stream=None) -> int:
    return load().fp4root_device_status(_ptr(ws), _stream(stream))


def fp4root_quantize(x: torch.Tensor, axis: int = 1, flags: int = F_HADAMARD | F_ADAPTIVE46,
                     clip_quantile: float = 0.99, seed: int = 0, step: int = 0, ws=None, stream=None):
    """NVFP4-quantise a matrix or a batch (B, rows, cols) of float32 matrices.

    Returns (codes, scales, tensor_scale, clip_threshold, ws); codes hold two
    4-bit codes per byte.  See fp4root_quantize in include/fp4root.h.
    """
    _need_gpu_f32(x, "x")
    lib = load()
    xb = x if x.dim() == 3 else x.unsqueeze(0)
    if xb.stride(-1) != 1:
        raise ValueError("x rows must be contiguous")
    B, R, C = xb.shape
    ld = xb.stride(1)
    bstride = xb.stride(0) if B > 1 else R * ld
    dev = x.device
    if axis == 1:
        codes = torch.empty((B, R, C // 2), dtype=torch.uint8, device=dev)
        scales = torch.empty((B, R, C // 16), dtype=torch.uint8, device=dev)
    else:
        codes = torch.empty((B, C, R // 2), dtype=torch.uint8, device=dev)
        scales = torch.empty((B, C, R // 16), dtype=torch.uint8, device=dev)
    sg = torch.empty(B, dtype=torch.float32, device=dev)
    tau = torch.empty(B, dtype=torch.float32, device=dev)
    need = lib.fp4root_quantize_workspace(B, R, C, flags)
    if ws is None or ws.numel() < need:
        ws = workspace(need, dev)
    _check(lib.fp4root_quantize(_ptr(xb), B, R, C, ld, bstride, axis, flags, clip_quantile, seed,
                                step, _ptr(codes), _ptr(scales), _ptr(sg), _ptr(tau), _ptr(ws),
                                ws.numel(), _stream(stream)), "fp4root_quantize")
    if x.dim() == 2:
        codes, scales = codes[0], scales[0]
    return codes, scales, sg, tau, ws


def fp4root_quantize_noalloc(x: torch.Tensor, out, axis: int = 1, flags: int = F_HADAMARD | F_ADAPTIVE46,
                             clip_quantile: float = 0.99, seed: int = 0, step: int = 0, stream=None):
    """fp4root_quantize into caller-owned outputs without a workspace (the library's
    fixed scratch; at most 256 matrices).  out = (codes, scales, tensor_scale,
    clip_threshold or None, status or None), shaped as fp4root_quantize returns them
    (batch first); status is an int32 device tensor of one element."""
    _need_gpu_f32(x, "x")
    codes, scales, sg, tau, status = out
    xb = x if x.dim() == 3 else x.unsqueeze(0)
    if xb.stride(-1) != 1:
        raise ValueError("x rows must be contiguous")
    B, R, C = xb.shape
    ld = xb.stride(1)
    bstride = xb.stride(0) if B > 1 else R * ld
    _check(load().fp4root_quantize_noalloc(_ptr(xb), B, R, C, ld, bstride, axis, flags, clip_quantile, seed, step,
                                           _ptr(codes), _ptr(scales), _ptr(sg),
                                           _ptr(tau) if tau is not None else None,
                                           _ptr(status) if status is not None else None, _stream(stream)),
           "fp4root_quantize_noalloc")


def fp4root_ns_step(x: torch.Tensor, a: float, b: float, c: float,
                    flags: int = F_HADAMARD | F_ADAPTIVE46, seed: int = 0, step: int = 0,
                    trace: bool = False, ws=None, stream=None):
    """One NS step in place on x (m, n) or (B, m, n).  With trace=True returns a dict of
    the step's intermediates (qX, qXt, A, qA, B, qB), else None."""
    _need_gpu_f32(x, "x")
    if not x.is_contiguous():
        raise ValueError("x must be contiguous")
    lib = load()
    xb = x if x.dim() == 3 else x.unsqueeze(0)
    B, m, n = xb.shape
    need = lib.fp4root_ns_step_workspace(B, m, n, flags)
    if ws is None or ws.numel() < need:
        ws = workspace(need, x.device)
    tr = None
    out = None
    if trace:
        dev = x.device
        u8 = dict(dtype=torch.uint8, device=dev)
        f32 = dict(dtype=torch.float32, device=dev)
        out = {
            "qx_codes": torch.empty((B, m, n // 2), **u8), "qx_scales": torch.empty((B, m, n // 16), **u8),
            "qx_sg": torch.empty(B, **f32),
            "qxt_codes": torch.empty((B, n, m // 2), **u8), "qxt_scales": torch.empty((B, n, m // 16), **u8),
            "qxt_sg": torch.empty(B, **f32),
            "A": torch.empty((B, m, m), **f32),
            "qa_codes": torch.empty((B, m, m // 2), **u8), "qa_scales": torch.empty((B, m, m // 16), **u8),
            "qa_sg": torch.empty(B, **f32),
            "B": torch.empty((B, m, m), **f32),
            "qb_codes": torch.empty((B, m, m // 2), **u8), "qb_scales": torch.empty((B, m, m // 16), **u8),
            "qb_sg": torch.empty(B, **f32),
        }
        tr = NsTrace(**{k: v.data_ptr() for k, v in out.items()})
    _check(lib.fp4root_ns_step(_ptr(xb), B, m, n, m * n, a, b, c, flags, seed, step,
                               ctypes.byref(tr) if tr is not None else None, _ptr(ws), ws.numel(),
                               _stream(stream)), "fp4root_ns_step")
    return out


class MomentumState:
    """NVFP4 first-moment state of a batch of rows x cols matrices (device tensors):
    codes (B, rows, cols/2), scales (B, rows, cols/16), tensor_scale (B,)."""

    def __init__(self, batch: int, rows: int, cols: int, device="cuda"):
        self.codes = torch.zeros((batch, rows, cols // 2), dtype=torch.uint8, device=device)
        self.scales = torch.zeros((batch, rows, cols // 16), dtype=torch.uint8, device=device)
        self.tensor_scale = torch.zeros(batch, dtype=torch.float32, device=device)
        self.ws = workspace(load().fp4root_momentum_workspace(batch, rows, cols), device)


def fp4root_momentum_update(g: torch.Tensor, state: MomentumState, beta: float, step: int,
                            flags: int = F_HADAMARD | F_ADAPTIVE46 | F_STOCHASTIC, seed: int = 0,
                            m: torch.Tensor = None, stream=None) -> torch.Tensor:
    """One first-moment step: returns m_t (FP32, shape of g) and re-encodes `state`.
    g: (rows, cols) or (B, rows, cols) contiguous float32.  See include/fp4root.h."""
    _need_gpu_f32(g, "g")
    if not g.is_contiguous():
        raise ValueError("g must be contiguous")
    gb = g if g.dim() == 3 else g.unsqueeze(0)
    B, R, C = gb.shape
    if tuple(state.codes.shape) != (B, R, C // 2):
        raise ValueError("state shape does not match g")
    if m is None:
        m = torch.empty_like(g)
    _need_gpu_f32(m, "m")
    if m.shape != g.shape or not m.is_contiguous():
        raise ValueError("m must be a contiguous tensor of g's shape")
    _check(load().fp4root_momentum_update(_ptr(gb), _ptr(m), B, R, C, _ptr(state.codes), _ptr(state.scales),
                                          _ptr(state.tensor_scale), beta, flags, seed, step, _ptr(state.ws),
                                          state.ws.numel(), _stream(stream)), "fp4root_momentum_update")
    return m


def fp4root_apply_update(w: torch.Tensor, o: torch.Tensor, lr: float, wd: float, scale: float, stream=None):
    """W <- bf16(fl32(fl32(W c1) - fl32(c2 O))) in place on a contiguous bfloat16 tensor w."""
    if w.dtype != torch.bfloat16 or not w.is_cuda or not w.is_contiguous():
        raise TypeError("w must be a contiguous bfloat16 GPU tensor")
    _need_gpu_f32(o, "o")
    if o.shape != w.shape or not o.is_contiguous():
        raise ValueError("o must be a contiguous float32 tensor of w's shape")
    _check(load().fp4root_apply_update(_ptr(w), _ptr(o), w.numel(), lr, wd, scale, _stream(stream)),
           "fp4root_apply_update")


class QAdamWState:
    """Both quantized AdamW moments of a flat parameter of n elements (device tensors)."""

    def __init__(self, n: int, device="cuda", keep_m: bool = False):
        if n <= 0 or n % 256:
            raise ValueError("n must be a positive multiple of 256")
        self.n = n
        # this step's binary32 first moment, written only when kept (diagnostics)
        self.m = torch.empty(n, dtype=torch.float32, device=device) if keep_m else None
        self.m_codes = torch.zeros(n // 2, dtype=torch.uint8, device=device)
        self.m_scales = torch.zeros(n // 16, dtype=torch.uint8, device=device)
        self.m_tensor_scale = torch.zeros(1, dtype=torch.float32, device=device)
        self.v_codes = torch.zeros(n // 2, dtype=torch.uint8, device=device)
        self.v_scales = torch.zeros(n // 16, dtype=torch.int16, device=device)
        self.v_means = torch.zeros(n // 256, dtype=torch.int16, device=device)
        self.ws = workspace(load().fp4root_qadamw_workspace(n), device)


def fp4root_qadamw_update(w: torch.Tensor, g: torch.Tensor, state: QAdamWState, step: int, lr: float,
                          wd: float = 0.1, beta1: float = 0.9, beta2: float = 0.95, eps: float = 1e-8,
                          flags: int = F_HADAMARD | F_ADAPTIVE46 | F_STOCHASTIC, seed: int = 0, stream=None):
    """One quantized-state AdamW step on a flat contiguous bfloat16 parameter w with FP32 gradient g."""
    if w.dtype != torch.bfloat16 or not w.is_cuda or not w.is_contiguous():
        raise TypeError("w must be a contiguous bfloat16 GPU tensor")
    _need_gpu_f32(g, "g")
    if g.numel() != w.numel() or not g.is_contiguous() or w.numel() != state.n:
        raise ValueError("g and state must match w")
    _check(load().fp4root_qadamw_update(
        _ptr(w), _ptr(g), _ptr(state.m), state.n, _ptr(state.m_codes), _ptr(state.m_scales),
        _ptr(state.m_tensor_scale), _ptr(state.v_codes), _ptr(state.v_scales), _ptr(state.v_means),
        lr, wd, beta1, beta2, eps, flags, seed, step, _ptr(state.ws), state.ws.numel(), _stream(stream)),
        "fp4root_qadamw_update")


class RootStep:
    """Reusable fp4root_root_step over a fixed list of (BF16 weight, FP32 gradient) pairs.

    Holds the descriptors, each parameter's first-moment state and FP32 scratch,
    the configurations and the workspace; each call is one C call.
    """

    def __init__(self, weights, grads, lr: float, wd: float = 0.1, beta: float = 0.9, steps: int = 5,
                 coeffs=None, ns_flags: int = F_DEFAULT, momentum_flags: int = F_HADAMARD | F_ADAPTIVE46 | F_STOCHASTIC,
                 clip_quantile: float = 0.99, eps: float = 1e-7, seed: int = 0, momentum_seed: int = 0,
                 scales=None):
        lib = load()
        self.weights, self.grads = list(weights), list(grads)
        n = len(self.weights)
        self.scratch, self.states = [], []
        self.params = (Param * max(n, 1))()
        for i, (w, g) in enumerate(zip(self.weights, self.grads)):
            if w.dtype != torch.bfloat16 or not w.is_cuda or not w.is_contiguous() or w.dim() != 2:
                raise TypeError(f"weights[{i}] must be a contiguous 2-D bfloat16 GPU tensor")
            _need_gpu_f32(g, f"grads[{i}]")
            if g.shape != w.shape or not g.is_contiguous():
                raise ValueError(f"grads[{i}] must be contiguous with the weight's shape")
            r, c = w.shape
            m = torch.empty_like(g)
            st = MomentumState(1, r, c, device=w.device)
            self.scratch.append(m)
            self.states.append(st)
            sc = scales[i] if scales is not None else 0.0   # 0: the library's default scale
            self.params[i] = Param(w.data_ptr(), g.data_ptr(), m.data_ptr(), st.codes.data_ptr(),
                                   st.scales.data_ptr(), st.tensor_scale.data_ptr(), r, c, sc)
        self.count = n
        if coeffs is not None:
            flat = [float(v) for row in coeffs for v in row]
            if len(flat) != 3 * steps:
                raise ValueError("coeffs must hold steps rows of (a, b, c)")
            self._coeffs = (ctypes.c_float * len(flat))(*flat)
            cptr = ctypes.cast(self._coeffs, ctypes.POINTER(ctypes.c_float))
        else:
            self._coeffs, cptr = None, None
        self.ns = NsConfig(steps, cptr, ns_flags, clip_quantile, eps, seed)
        self.cfg = RootConfig(lr, wd, beta, momentum_flags, momentum_seed, 0)
        need = lib.fp4root_root_step_workspace(self.params, n, ctypes.byref(self.ns))
        if need == 0:
            raise ValueError("invalid parameters or configuration")
        self.ws = workspace(need, self.weights[0].device if n else torch.device("cuda"))

    def __call__(self, step: int, stream=None):
        self.cfg.step = step
        _check(load().fp4root_root_step(self.params, self.count, ctypes.byref(self.cfg), ctypes.byref(self.ns),
                                        _ptr(self.ws), self.ws.numel(), _stream(stream)), "fp4root_root_step")

    def status(self, stream=None) -> int:
        return fp4root_device_status(self.ws, stream)


class Orthogonalizer:
    """Reusable call of fp4root_orthogonalize over a fixed list of matrices.

    Holds the descriptor array, the configuration and the workspace so that a
    timed loop makes exactly one C call per invocation.
    """

    def __init__(self, inputs, outputs=None, steps: int = 5, coeffs=None, flags: int = F_DEFAULT,
                 clip_quantile: float = 0.99, eps: float = 1e-7, seed: int = 0):
        lib = load()
        self.inputs = list(inputs)
        self.outputs = list(outputs) if outputs is not None else [torch.empty_like(t) for t in self.inputs]
        n = len(self.inputs)
        self.mats = (Matrix * max(n, 1))()
        for i, (a, o) in enumerate(zip(self.inputs, self.outputs)):
            _need_gpu_f32(a, f"inputs[{i}]")
            _need_gpu_f32(o, f"outputs[{i}]")
            if a.dim() != 2 or a.stride(1) != 1 or o.stride(1) != 1 or o.shape != a.shape:
                raise ValueError(f"matrix {i}: need 2-D row-contiguous input and output of equal shape")
            self.mats[i] = Matrix(a.data_ptr(), o.data_ptr(), a.shape[0], a.shape[1], a.stride(0), o.stride(0))
        self.count = n
        if coeffs is not None:
            flat = [float(v) for row in coeffs for v in row]
            if len(flat) != 3 * steps:
                raise ValueError("coeffs must hold steps rows of (a, b, c)")
            self._coeffs = (ctypes.c_float * len(flat))(*flat)
            cptr = ctypes.cast(self._coeffs, ctypes.POINTER(ctypes.c_float))
        else:
            self._coeffs = None
            cptr = None
        self.cfg = NsConfig(steps, cptr, flags, clip_quantile, eps, seed)
        need = lib.fp4root_orthogonalize_workspace(self.mats, n, ctypes.byref(self.cfg))
        if need == 0:
            raise ValueError("invalid matrices or configuration")
        dev = self.inputs[0].device if n else torch.device("cuda")
        self.ws = workspace(need, dev)

    def __call__(self, stream=None):
        _check(load().fp4root_orthogonalize(self.mats, self.count, ctypes.byref(self.cfg),
                                            _ptr(self.ws), self.ws.numel(), _stream(stream)),
               "fp4root_orthogonalize")
        return self.outputs

    def capture(self):
        """Record one call into a HIP graph (the library allocates nothing and clears
        its scalars with kernels, so the whole call can be captured); returns the graph,
        whose replay() repeats the call on the same buffers."""
        graph = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            self()                       # warm call outside the capture
        torch.cuda.current_stream().wait_stream(side)
        with torch.cuda.graph(graph, stream=side):
            self()
        torch.cuda.synchronize()
        return graph

    def status(self, stream=None) -> int:
        return fp4root_device_status(self.ws, stream)


def fp4root_orthogonalize(inputs, outputs=None, steps: int = 5, coeffs=None, flags: int = F_DEFAULT,
                          clip_quantile: float = 0.99, eps: float = 1e-7, seed: int = 0, stream=None):
    """Orthogonalise a list of float32 GPU matrices; returns the outputs (new tensors unless given)."""
    return Orthogonalizer(inputs, outputs, steps, coeffs, flags, clip_quantile, eps, seed)(stream)
