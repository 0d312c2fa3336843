"""Python binding of the LR-QAT C ABI (include/lrqat.h).

Argument marshalling only: every step of the layer runs in the HIP library
liblrqat.so.  torch provides device memory (tensors) and the current stream.
The functions keep the C names; tensors must be contiguous and on the GPU.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblrqat.so")

LRQAT_OK, LRQAT_EINVAL, LRQAT_EUNSUPPORTED, LRQAT_EWORKSPACE, LRQAT_EHIP = range(5)
PHI_FIXED_Q8, PHI_INT_PACKED2 = 0, 1
FP32, BF16 = 0, 1
_FMT = {"q8": PHI_FIXED_Q8, "int_packed2": PHI_INT_PACKED2}
_DT = {"fp32": FP32, "bf16": BF16}


class _Layer(ctypes.Structure):
    _fields_ = [("out_features", ctypes.c_int64), ("in_features", ctypes.c_int64),
                ("rank", ctypes.c_int32), ("alpha", ctypes.c_float), ("bits", ctypes.c_int32),
                ("phi_format", ctypes.c_int32), ("group_size", ctypes.c_int64),
                ("act_bits", ctypes.c_int32), ("act_dtype", ctypes.c_int32)]


class _ParamGroup(ctypes.Structure):
    _fields_ = [("param", ctypes.c_void_p), ("grad", ctypes.c_void_p), ("exp_avg", ctypes.c_void_p),
                ("exp_avg_sq", ctypes.c_void_p), ("n", ctypes.c_int64), ("lr_max", ctypes.c_float),
                ("weight_decay", ctypes.c_float)]


class _AdamWConfig(ctypes.Structure):
    _fields_ = [("beta1", ctypes.c_float), ("beta2", ctypes.c_float), ("eps", ctypes.c_float),
                ("max_grad_norm", ctypes.c_float), ("total_steps", ctypes.c_int64), ("warmup_steps", ctypes.c_int64)]


@dataclass(frozen=True)
class LayerSpec:
    """Hyper-parameters of one LR-QAT linear (mirrors the C struct lrqat_layer)."""
    out_features: int
    in_features: int
    rank: int
    alpha: float
    bits: int
    phi_format: str = "q8"        # "q8" or "int_packed2"
    group_size: int = 0
    act_bits: int = 0
    act_dtype: str = "bf16"       # "bf16" or "fp32"

    def c_struct(self) -> _Layer:
        return _Layer(self.out_features, self.in_features, self.rank, self.alpha, self.bits,
                      _FMT[self.phi_format], self.group_size, self.act_bits, _DT[self.act_dtype])

    @property
    def torch_dtype(self):
        return torch.bfloat16 if self.act_dtype == "bf16" else torch.float32

    def scale_shape(self):
        m, k, g = self.out_features, self.in_features, self.group_size
        return (m,) if g == 0 else (m, k // g)

    def phi_shape(self):
        m, k = self.out_features, self.in_features
        return (m, k) if self.phi_format == "q8" else (m, k // 2)

    @property
    def phi_dtype(self):
        return torch.int8 if self.phi_format == "q8" else torch.uint8


class LRQATError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{_lib().lrqat_status_string(status).decode()}: {message}")
        self.status = status


_LIB = None


def _lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2406_06385_amd.build`")
        lib = ctypes.CDLL(LIB_PATH)
        P, I64, SZ, F = ctypes.c_void_p, ctypes.c_int64, ctypes.c_size_t, ctypes.POINTER(_Layer)
        lib.lrqat_forward_workspace_size.argtypes = [F, I64]
        lib.lrqat_forward_workspace_size.restype = SZ
        lib.lrqat_backward_workspace_size.argtypes = [F, I64]
        lib.lrqat_backward_workspace_size.restype = SZ
        lib.lrqat_init_from_weights.argtypes = [F, P, P, P, P, P]
        lib.lrqat_infer_workspace_size.argtypes = [F, I64]
        lib.lrqat_infer_workspace_size.restype = SZ
        lib.lrqat_infer_forward.argtypes = [F, I64, P, P, P, P, P, P, SZ, P]
        lib.lrqat_forward.argtypes = [F, I64, P, P, P, P, P, P, P, P, SZ, P]
        lib.lrqat_backward.argtypes = [F, I64, P, P, P, P, P, P, P, P, P, P, P, ctypes.c_int, P, SZ, P]
        lib.lrqat_backward_static.argtypes = [F, I64, P, P, P, P, P, P, P, P, P, P, P, ctypes.c_int, P]
        lib.lrqat_backward_static_capacity.argtypes = []
        lib.lrqat_backward_static_capacity.restype = SZ
        lib.lrqat_merge_to_int4.argtypes = [F, P, P, P, P, P]
        for fn in ("lrqat_init_from_weights", "lrqat_forward", "lrqat_backward", "lrqat_backward_static",
                   "lrqat_merge_to_int4", "lrqat_infer_forward"):
            getattr(lib, fn).restype = ctypes.c_int
        lib.lrqat_init_lp.argtypes = [F, P, ctypes.c_float, ctypes.c_int, P, P, P]
        lib.lrqat_init_lp.restype = ctypes.c_int
        lib.lrqat_init_loftq_workspace_size.argtypes = [F]
        lib.lrqat_init_loftq_workspace_size.restype = SZ
        lib.lrqat_init_loftq.argtypes = [F, P, P, ctypes.c_int, P, P, P, P, P, SZ, P]
        lib.lrqat_init_loftq.restype = ctypes.c_int
        PG = ctypes.POINTER(_ParamGroup)
        lib.lrqat_adamw_workspace_size.argtypes = [ctypes.c_int, PG]
        lib.lrqat_adamw_workspace_size.restype = SZ
        lib.lrqat_adamw_step.argtypes = [ctypes.POINTER(_AdamWConfig), I64, ctypes.c_int, PG, P, P, SZ, P]
        lib.lrqat_adamw_step.restype = ctypes.c_int
        lib.lrqat_status_string.argtypes = [ctypes.c_int]
        lib.lrqat_status_string.restype = ctypes.c_char_p
        lib.lrqat_last_error.restype = ctypes.c_char_p
        lib.lrqat_timing_enable.argtypes = [ctypes.c_int]
        lib.lrqat_timing_read.argtypes = [ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(I64),
                                          ctypes.POINTER(ctypes.c_double), ctypes.c_int]
        lib.lrqat_timing_read.restype = ctypes.c_int
        _LIB = lib
    return _LIB


def load_library() -> str:
    """Load liblrqat.so (raises if it is missing) and return its path."""
    _lib()
    return LIB_PATH


def _check(status: int):
    if status != LRQAT_OK:
        raise LRQATError(status, _lib().lrqat_last_error().decode())


def _ptr(t):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError("expected a torch.Tensor")
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError("tensors passed to the LR-QAT library must be contiguous GPU tensors")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _torch_stream(stream):
    return torch.cuda.current_stream() if stream is None else stream


def _expect(t, shape, dtype, name, device=None):
    """Reject a tensor whose shape, dtype, layout or device the C ABI would
    misread (the library sees only a pointer)."""
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name}: expected a torch.Tensor, got {type(t).__name__}")
    if tuple(t.shape) != tuple(shape) or t.dtype != dtype:
        raise ValueError(f"{name}: expected {tuple(shape)} {dtype}, got {tuple(t.shape)} {t.dtype}")
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError(f"{name}: must be a contiguous GPU tensor")
    if device is not None and t.device != device:
        raise ValueError(f"{name}: on {t.device}, expected {device}")


def _weights(spec: "LayerSpec", phi0, s, A, B, device, z=None):
    m, k, r = spec.out_features, spec.in_features, spec.rank
    _expect(phi0, spec.phi_shape(), spec.phi_dtype, "phi0", device)
    _expect(s, spec.scale_shape(), torch.float32, "s", device)
    if z is not None:
        _expect(z, spec.scale_shape(), torch.int32, "z", device)
    _expect(A, (m, r), torch.float32, "A", device)
    _expect(B, (r, k), torch.float32, "B", device)


def lrqat_forward_workspace_size(spec: LayerSpec, tokens: int) -> int:
    L = spec.c_struct()
    n = _lib().lrqat_forward_workspace_size(ctypes.byref(L), tokens)
    if n == 0:
        raise LRQATError(LRQAT_EINVAL, _lib().lrqat_last_error().decode())
    return n


def lrqat_backward_workspace_size(spec: LayerSpec, tokens: int) -> int:
    L = spec.c_struct()
    n = _lib().lrqat_backward_workspace_size(ctypes.byref(L), tokens)
    if n == 0:
        raise LRQATError(LRQAT_EINVAL, _lib().lrqat_last_error().decode())
    return n


def workspace(nbytes: int, device="cuda") -> torch.Tensor:
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


def lrqat_init_from_weights(spec: LayerSpec, W0: torch.Tensor, stream=None, asymmetric=False):
    """-> (s0 float32, Phi0) computed on the GPU from W0 [m][k] float32, or
    (s0, z0 int32, Phi0) with asymmetric=True (Phi0 then carries z0)."""
    _expect(W0, (spec.out_features, spec.in_features), torch.float32, "W0")
    st = _torch_stream(stream)
    with torch.cuda.stream(st):
        s0 = torch.empty(spec.scale_shape(), dtype=torch.float32, device=W0.device)
        z0 = torch.empty(spec.scale_shape(), dtype=torch.int32, device=W0.device) if asymmetric else None
        phi0 = torch.empty(spec.phi_shape(), dtype=spec.phi_dtype, device=W0.device)
    L = spec.c_struct()
    _check(_lib().lrqat_init_from_weights(ctypes.byref(L), _ptr(W0), _ptr(s0), _ptr(z0), _ptr(phi0), _stream(st)))
    return (s0, z0, phi0) if asymmetric else (s0, phi0)


def lrqat_init_lp(spec: LayerSpec, W0: torch.Tensor, p: float, n_grid: int = 100, stream=None):
    """-> (s0, Phi0) with s0 from the L^p-norm range search over n_grid clipping ratios."""
    _expect(W0, (spec.out_features, spec.in_features), torch.float32, "W0")
    st = _torch_stream(stream)
    with torch.cuda.stream(st):
        s0 = torch.empty(spec.scale_shape(), dtype=torch.float32, device=W0.device)
        phi0 = torch.empty(spec.phi_shape(), dtype=spec.phi_dtype, device=W0.device)
    L = spec.c_struct()
    _check(_lib().lrqat_init_lp(ctypes.byref(L), _ptr(W0), float(p), int(n_grid), _ptr(s0), _ptr(phi0), _stream(st)))
    return s0, phi0


def lrqat_init_loftq(spec: LayerSpec, W0: torch.Tensor, s0: torch.Tensor, n_iter: int = 32, stream=None):
    """-> (Phi0 packed INT-b, A, B, sigma) of the LoftQ (T = 1) initialisation for the given scale."""
    m, k, r = spec.out_features, spec.in_features, spec.rank
    _expect(W0, (m, k), torch.float32, "W0")
    dev = W0.device
    _expect(s0, spec.scale_shape(), torch.float32, "s0", dev)
    L = spec.c_struct()
    n = _lib().lrqat_init_loftq_workspace_size(ctypes.byref(L))
    if n == 0:
        raise LRQATError(LRQAT_EINVAL, _lib().lrqat_last_error().decode())
    st = _torch_stream(stream)
    with torch.cuda.stream(st):
        phi0 = torch.empty(spec.phi_shape(), dtype=spec.phi_dtype, device=dev)
        A = torch.empty((m, r), dtype=torch.float32, device=dev)
        B = torch.empty((r, k), dtype=torch.float32, device=dev)
        sigma = torch.empty(r, dtype=torch.float32, device=dev)
        ws = workspace(n, dev)
    _check(_lib().lrqat_init_loftq(ctypes.byref(L), _ptr(W0), _ptr(s0), int(n_iter), _ptr(phi0), _ptr(A), _ptr(B),
                                   _ptr(sigma), _ptr(ws), ws.numel(), _stream(st)))
    return phi0, A, B, sigma


def lrqat_forward(spec: LayerSpec, X, phi0, s, A, B, Y=None, ws=None, stream=None, z=None):
    """Y = X_hat W_hat^T.  X [T][k] in the layer's activation dtype; z (int32,
    shaped like s) is the zero offset of asymmetric quantisation."""
    T = X.shape[0] if X.dim() == 2 else -1
    _expect(X, (T, spec.in_features), spec.torch_dtype, "X")
    dev = X.device
    _weights(spec, phi0, s, A, B, dev, z)
    st = _torch_stream(stream)
    with torch.cuda.stream(st):  # buffers made here belong to the stream the kernels run on
        if Y is None:
            Y = torch.empty((T, spec.out_features), dtype=spec.torch_dtype, device=dev)
        if ws is None:
            ws = workspace(lrqat_forward_workspace_size(spec, T), dev)
    _expect(Y, (T, spec.out_features), spec.torch_dtype, "Y", dev)
    _expect(ws, (ws.numel(),), torch.uint8, "ws", dev)
    L = spec.c_struct()
    _check(_lib().lrqat_forward(ctypes.byref(L), T, _ptr(X), _ptr(phi0), _ptr(s), _ptr(z), _ptr(A), _ptr(B),
                                _ptr(Y), _ptr(ws), ws.numel(), _stream(st)))
    return Y


def _backward_args(spec, X, phi0, s, A, B, dY, dX, dA, dB, want_dx, ds, want_ds, z, stream):
    T = X.shape[0] if X.dim() == 2 else -1
    m, k, r = spec.out_features, spec.in_features, spec.rank
    _expect(X, (T, k), spec.torch_dtype, "X")
    dev = X.device
    _weights(spec, phi0, s, A, B, dev, z)
    _expect(dY, (T, m), spec.torch_dtype, "dY", dev)
    st = _torch_stream(stream)
    with torch.cuda.stream(st):  # buffers made here belong to the stream the kernels run on
        if dX is None and want_dx:
            dX = torch.empty((T, k), dtype=spec.torch_dtype, device=dev)
        if dA is None:
            dA = torch.empty((m, r), dtype=torch.float32, device=dev)
        if dB is None:
            dB = torch.empty((r, k), dtype=torch.float32, device=dev)
        if ds is None and want_ds:
            ds = torch.empty(spec.scale_shape(), dtype=torch.float32, device=dev)
    if dX is not None:
        _expect(dX, (T, k), spec.torch_dtype, "dX", dev)
    _expect(dA, (m, r), torch.float32, "dA", dev)
    _expect(dB, (r, k), torch.float32, "dB", dev)
    if ds is not None:
        _expect(ds, spec.scale_shape(), torch.float32, "ds", dev)
    return T, dev, st, dX, dA, dB, ds


def lrqat_backward(spec: LayerSpec, X, phi0, s, A, B, dY, dX=None, dA=None, dB=None, want_dx=True,
                   accumulate=False, ws=None, stream=None, z=None, ds=None, want_ds=False):
    """-> (dX or None, dA, dB) with the straight-through estimator; W_hat is
    recomputed.  With want_ds (or a ds tensor) -> (dX, dA, dB, ds)."""
    T, dev, st, dX, dA, dB, ds = _backward_args(spec, X, phi0, s, A, B, dY, dX, dA, dB, want_dx, ds, want_ds, z,
                                                stream)
    if ws is None:
        with torch.cuda.stream(st):
            ws = workspace(lrqat_backward_workspace_size(spec, T), dev)
    _expect(ws, (ws.numel(),), torch.uint8, "ws", dev)
    L = spec.c_struct()
    _check(_lib().lrqat_backward(ctypes.byref(L), T, _ptr(X), _ptr(phi0), _ptr(s), _ptr(z), _ptr(A), _ptr(B),
                                 _ptr(dY), _ptr(dX), _ptr(dA), _ptr(dB), _ptr(ds), int(bool(accumulate)), _ptr(ws),
                                 ws.numel(), _stream(st)))
    return (dX, dA, dB, ds) if ds is not None else (dX, dA, dB)


def lrqat_backward_static(spec: LayerSpec, X, phi0, s, A, B, dY, dX, dA, dB, accumulate=False, stream=None,
                          z=None, ds=None):
    """lrqat_backward on the library's device-resident scratch array: every
    output tensor is the caller's, nothing is allocated."""
    T, dev, st, dX, dA, dB, ds = _backward_args(spec, X, phi0, s, A, B, dY, dX, dA, dB, dX is not None, ds,
                                                False, z, stream)
    L = spec.c_struct()
    _check(_lib().lrqat_backward_static(ctypes.byref(L), T, _ptr(X), _ptr(phi0), _ptr(s), _ptr(z), _ptr(A),
                                        _ptr(B), _ptr(dY), _ptr(dX), _ptr(dA), _ptr(dB), _ptr(ds),
                                        int(bool(accumulate)), _stream(st)))
    return (dX, dA, dB, ds) if ds is not None else (dX, dA, dB)


def lrqat_backward_static_capacity() -> int:
    return int(_lib().lrqat_backward_static_capacity())


def lrqat_merge_to_int4(spec: LayerSpec, phi0, A, B, out=None, stream=None):
    """W_Z = clip(round(Phi0 + (alpha/r) A B)) double-packed, uint8 [m][k/2]."""
    m, k, r = spec.out_features, spec.in_features, spec.rank
    dev = A.device
    _expect(phi0, spec.phi_shape(), spec.phi_dtype, "phi0", dev)
    _expect(A, (m, r), torch.float32, "A", dev)
    _expect(B, (r, k), torch.float32, "B", dev)
    st = _torch_stream(stream)
    if out is None:
        with torch.cuda.stream(st):
            out = torch.empty((m, k // 2), dtype=torch.uint8, device=dev)
    _expect(out, (m, k // 2), torch.uint8, "out", dev)
    L = spec.c_struct()
    _check(_lib().lrqat_merge_to_int4(ctypes.byref(L), _ptr(phi0), _ptr(A), _ptr(B), _ptr(out), _stream(st)))
    return out


def lrqat_infer_workspace_size(spec: LayerSpec, tokens: int) -> int:
    L = spec.c_struct()
    n = _lib().lrqat_infer_workspace_size(ctypes.byref(L), tokens)
    if n == 0:
        raise LRQATError(LRQAT_EINVAL, _lib().lrqat_last_error().decode())
    return n


def lrqat_infer_forward(spec: LayerSpec, X, W_int4, s, z=None, Y=None, ws=None, stream=None):
    """Y = X_hat (s (W_Z - z))^T on the merged packed int4 weights uint8 [m][k/2]."""
    T = X.shape[0] if X.dim() == 2 else -1
    m, k = spec.out_features, spec.in_features
    _expect(X, (T, k), spec.torch_dtype, "X")
    dev = X.device
    _expect(W_int4, (m, k // 2), torch.uint8, "W_int4", dev)
    _expect(s, spec.scale_shape(), torch.float32, "s", dev)
    if z is not None:
        _expect(z, spec.scale_shape(), torch.int32, "z", dev)
    st = _torch_stream(stream)
    with torch.cuda.stream(st):
        if Y is None:
            Y = torch.empty((T, m), dtype=spec.torch_dtype, device=dev)
        if ws is None:
            ws = workspace(lrqat_infer_workspace_size(spec, T), dev)
    _expect(Y, (T, m), spec.torch_dtype, "Y", dev)
    _expect(ws, (ws.numel(),), torch.uint8, "ws", dev)
    L = spec.c_struct()
    _check(_lib().lrqat_infer_forward(ctypes.byref(L), T, _ptr(X), _ptr(W_int4), _ptr(s), _ptr(z), _ptr(Y),
                                      _ptr(ws), ws.numel(), _stream(st)))
    return Y


def _groups(groups):
    arr = (_ParamGroup * max(1, len(groups)))()
    dev = None
    for i, g in enumerate(groups):
        p = g["param"]
        dev = dev or p.device
        n = p.numel()
        for key in ("param", "grad", "exp_avg", "exp_avg_sq"):
            _expect(g[key], tuple(p.shape), torch.float32, key, dev)
        arr[i] = _ParamGroup(g["param"].data_ptr(), g["grad"].data_ptr(), g["exp_avg"].data_ptr(),
                             g["exp_avg_sq"].data_ptr(), n, float(g["lr_max"]), float(g.get("weight_decay", 0.0)))
    return arr, dev


def lrqat_adamw_step(groups, step, total_steps, warmup_steps, beta1=0.9, beta2=0.95, eps=1e-8, max_grad_norm=1.0,
                     grad_norm=None, ws=None, stream=None):
    """AdamW with global L2 clipping and the linear warm-up/decay schedule, in place.
    groups: list of dicts with float32 tensors param, grad, exp_avg, exp_avg_sq (same
    shape) and floats lr_max, weight_decay.  grad_norm: optional float32 [1] tensor
    receiving the norm before clipping."""
    arr, dev = _groups(groups)
    cfg = _AdamWConfig(beta1, beta2, eps, max_grad_norm, int(total_steps), int(warmup_steps))
    st = _torch_stream(stream)
    if ws is None:
        n = _lib().lrqat_adamw_workspace_size(len(groups), arr)
        if n == 0:
            raise LRQATError(LRQAT_EINVAL, _lib().lrqat_last_error().decode())
        with torch.cuda.stream(st):
            ws = workspace(n, dev or "cuda")
    if grad_norm is not None:
        _expect(grad_norm, (1,), torch.float32, "grad_norm", dev)
    _check(_lib().lrqat_adamw_step(ctypes.byref(cfg), int(step), len(groups), arr, _ptr(grad_norm), _ptr(ws),
                                   ws.numel(), _stream(st)))


def lrqat_timing_enable(on: bool = True):
    _lib().lrqat_timing_enable(int(bool(on)))


def lrqat_timing_reset():
    _lib().lrqat_timing_reset()


def lrqat_timing_read() -> dict:
    """{kernel name: (launches, total milliseconds)} since the last reset."""
    n = 32
    names = (ctypes.c_char_p * n)()
    launches = (ctypes.c_int64 * n)()
    ms = (ctypes.c_double * n)()
    cnt = _lib().lrqat_timing_read(names, launches, ms, n)
    if cnt < 0:
        raise LRQATError(LRQAT_EHIP, "timing read failed")
    return {names[i].decode(): (int(launches[i]), float(ms[i])) for i in range(cnt)}
