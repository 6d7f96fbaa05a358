"""CurvaDion optimizer step on AMD Instinct MI355X: Python binding.

A thin ctypes layer over ``libcurvadion.so`` (the C ABI in
``include/curvadion.h``).  It only marshals arguments: every step of the method
runs in the library's HIP kernels.  PyTorch supplies device memory and the
current HIP stream.  There is no fallback path: if the library is missing the
import succeeds but every call raises ``LibraryNotBuilt``.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Sequence, Tuple

__all__ = [
    "LibraryNotBuilt", "CurvaDionError", "Layer", "Group", "lib", "library_path",
    "POLICY_RMMC", "POLICY_ALWAYS_SYNC", "POLICY_NEVER_SYNC", "POLICY_EVERY_H",
    "F32", "BF16", "EXPORTED_SYMBOLS", "PointerArray", "check_operand", "step_static",
    "STATIC_SCRATCH_BYTES",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
library_path = os.path.join(_HERE, "libcurvadion.so")

CD_OK, CD_EINVAL, CD_ENOMEM, CD_EHIP, CD_ENONFINITE, CD_ERANKDEF = 0, -1, -2, -3, -4, -5
F32, BF16 = 0, 1
POLICY_RMMC, POLICY_ALWAYS_SYNC, POLICY_NEVER_SYNC, POLICY_EVERY_H = 0, 1, 2, 3
_STATUS = {0: "CD_OK", -1: "CD_EINVAL", -2: "CD_ENOMEM", -3: "CD_EHIP",
           -4: "CD_ENONFINITE", -5: "CD_ERANKDEF"}

#: every function the header declares
EXPORTED_SYMBOLS = (
    "cd_layer_create", "cd_step", "cd_destroy", "cd_group_create", "cd_group_step",
    "cd_group_destroy", "cd_layer_get_state", "cd_layer_set_state",
    "cd_layer_last_factors", "cd_layer_rank_deficient", "cd_group_set_timing",
    "cd_group_kernel_times", "cd_group_set_timing_kinds", "cd_last_error", "cd_abi_version",
    "cd_step_static", "cd_group_last_result", "cd_layer_last_result",
)


class LibraryNotBuilt(RuntimeError):
    pass


class CurvaDionError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{_STATUS.get(status, status)}: {msg}")
        self.status = status


class LayerDesc(ctypes.Structure):
    _fields_ = [("m", ctypes.c_int), ("n", ctypes.c_int), ("r_max", ctypes.c_int),
                ("grad_dtype", ctypes.c_int), ("tau", ctypes.c_double),
                ("eps", ctypes.c_double), ("eta_local_scale", ctypes.c_double),
                ("policy", ctypes.c_int), ("H", ctypes.c_int), ("weight_decay", ctypes.c_double)]


class Result(ctypes.Structure):
    _fields_ = [("rmmc", ctypes.c_double), ("sync_flag", ctypes.c_int)]


class KernelTime(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 32), ("launches", ctypes.c_int),
                ("total_ms", ctypes.c_double), ("bytes", ctypes.c_double),
                ("flops", ctypes.c_double)]


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library (raises LibraryNotBuilt if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(library_path):
        raise LibraryNotBuilt(
            f"{library_path} is missing; build it with `python -m paper_2512_13728_amd.build`")
    L = ctypes.CDLL(library_path)
    vp, i, f, d = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_double
    L.cd_layer_create.argtypes = [ctypes.POINTER(LayerDesc), ctypes.POINTER(vp)]
    L.cd_step.argtypes = [vp, vp, vp, vp, vp, f, f, i, vp, ctypes.POINTER(Result)]
    L.cd_destroy.argtypes = [vp]
    L.cd_step_static.argtypes = [ctypes.POINTER(LayerDesc), vp, ctypes.POINTER(ctypes.c_longlong), vp, vp,
                                 vp, vp, f, f, i, vp, ctypes.POINTER(Result)]
    L.cd_group_create.argtypes = [ctypes.POINTER(vp), i, ctypes.POINTER(vp)]
    L.cd_group_step.argtypes = [vp, ctypes.POINTER(vp), ctypes.POINTER(vp), ctypes.POINTER(vp),
                                ctypes.POINTER(vp), f, f, i, vp, ctypes.POINTER(d),
                                ctypes.POINTER(Result)]
    L.cd_group_destroy.argtypes = [vp]
    L.cd_group_last_result.argtypes = [vp, ctypes.POINTER(d), ctypes.POINTER(Result)]
    L.cd_layer_last_result.argtypes = [vp, ctypes.POINTER(Result)]
    L.cd_layer_get_state.argtypes = [vp, ctypes.POINTER(d), ctypes.POINTER(ctypes.c_longlong)]
    L.cd_layer_set_state.argtypes = [vp, d, ctypes.c_longlong]
    L.cd_layer_last_factors.argtypes = [vp, ctypes.POINTER(vp), ctypes.POINTER(vp)]
    L.cd_layer_rank_deficient.argtypes = [vp, ctypes.POINTER(i)]
    L.cd_group_set_timing.argtypes = [vp, i]
    L.cd_group_set_timing_kinds.argtypes = [vp, ctypes.c_char_p]
    L.cd_group_kernel_times.argtypes = [vp, ctypes.POINTER(KernelTime), i, ctypes.POINTER(i)]
    L.cd_last_error.restype = ctypes.c_char_p
    L.cd_last_error.argtypes = []
    L.cd_abi_version.restype = i
    for name in EXPORTED_SYMBOLS:
        if name not in ("cd_last_error", "cd_abi_version"):
            getattr(L, name).restype = i
    _lib = L
    return L


def _check(st: int, allow=(CD_OK,)) -> int:
    if st not in allow:
        raise CurvaDionError(st, lib().cd_last_error().decode(errors="replace"))
    return st


def _ptr(t) -> int:
    """Device address of a tensor (or an int address)."""
    if isinstance(t, int):
        return t
    return t.data_ptr()


def check_operand(t, role: str, m: int, n: int, r: int, grad_dtype: str, device=None) -> None:
    """Raise ValueError unless tensor `t` can be handed to the library as
    operand `role` ("G", "M", "X" or "Q") of an m x n layer stepped at rank r:
    G, M, X are m x n and Q is n x r, row-major contiguous, on a GPU (the
    layer's, when `device` is given); M, X, Q fp32 and G of the layer's
    gradient dtype.  The kernels index these buffers by (m, n, r) alone, so a
    tensor of another shape or layout would be read out of bounds.  A plain
    int is a raw device address and is passed through unchecked."""
    if isinstance(t, int):
        return
    want_shape = (n, r) if role == "Q" else (m, n)
    shape = tuple(t.shape)
    if shape != want_shape:
        raise ValueError(f"{role}: expected shape {want_shape}, got {shape}")
    want_dtype = ("bfloat16" if grad_dtype == "bf16" else "float32") if role == "G" else "float32"
    if str(t.dtype) != "torch." + want_dtype:
        raise ValueError(f"{role}: expected {want_dtype}, got {str(t.dtype).replace('torch.', '')}")
    if not t.is_contiguous():
        raise ValueError(f"{role}: must be contiguous (row-major, leading dimension = columns)")
    if t.device.type != "cuda":
        raise ValueError(f"{role}: must be a GPU tensor, got device {t.device}")
    if device is not None and t.device.index != device:
        raise ValueError(f"{role}: on GPU {t.device.index}, the layer lives on GPU {device}")


def _stream_handle(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


class Layer:
    """One weight matrix under CurvaDion (m x n, rank up to r_max)."""

    def __init__(self, m: int, n: int, r_max: int, *, grad_dtype: str = "f32",
                 tau: float = 0.5, eps: float = 1e-8, eta_local_scale: float = 1.0,
                 policy: int = POLICY_RMMC, H: int = 1, weight_decay: float = 0.0):
        self._h = None
        desc = LayerDesc(m, n, r_max, BF16 if grad_dtype == "bf16" else F32, tau, eps,
                         eta_local_scale, policy, H, weight_decay)
        h = ctypes.c_void_p()
        _check(lib().cd_layer_create(ctypes.byref(desc), ctypes.byref(h)))
        self._h = h
        self.m, self.n, self.r_max = m, n, r_max
        self.grad_dtype = grad_dtype
        import torch
        self.device = torch.cuda.current_device()   # the device cd_layer_create used

    def check(self, t, role: str, r: int) -> None:
        """check_operand for this layer."""
        check_operand(t, role, self.m, self.n, r, self.grad_dtype, self.device)

    @property
    def handle(self) -> ctypes.c_void_p:
        return self._h

    def step(self, G, M, X, Q, mu: float, eta: float, r: Optional[int] = None,
             stream=None, wait: bool = True):
        """One CurvaDion step; returns (rmmc, sync_flag, status).  wait=False
        enqueues the whole step without reading its outcome (the asynchronous
        step) and returns None; last_result() reads it later."""
        r = Q.shape[1] if r is None and hasattr(Q, "shape") else r
        for t, role in ((G, "G"), (M, "M"), (X, "X"), (Q, "Q")):
            self.check(t, role, r)
        res = Result()
        st = lib().cd_step(self._h, _ptr(G), _ptr(M), _ptr(X), _ptr(Q), mu, eta, r,
                           _stream_handle(stream), ctypes.byref(res) if wait else None)
        _check(st, allow=(CD_OK, CD_ENONFINITE))
        return (res.rmmc, bool(res.sync_flag), st) if wait else None

    def last_result(self) -> Tuple[float, bool, int]:
        """(rmmc, sync_flag, status) of the last step, once its work has
        finished; status CD_OK, CD_ENONFINITE or CD_ERANKDEF."""
        res = Result()
        st = lib().cd_layer_last_result(self._h, ctypes.byref(res))
        _check(st, allow=(CD_OK, CD_ENONFINITE, CD_ERANKDEF))
        return res.rmmc, bool(res.sync_flag), st

    def get_state(self) -> Tuple[float, int]:
        p, s = ctypes.c_double(), ctypes.c_longlong()
        _check(lib().cd_layer_get_state(self._h, ctypes.byref(p), ctypes.byref(s)))
        return p.value, s.value

    def set_state(self, prev_norm: float, step: int) -> None:
        _check(lib().cd_layer_set_state(self._h, prev_norm, step))

    def last_factors(self) -> Tuple[int, int]:
        """Device addresses of the last sync step's P (m x r) and R (n x r)."""
        P, R = ctypes.c_void_p(), ctypes.c_void_p()
        _check(lib().cd_layer_last_factors(self._h, ctypes.byref(P), ctypes.byref(R)))
        return P.value, R.value

    def rank_deficient(self) -> bool:
        f = ctypes.c_int()
        _check(lib().cd_layer_rank_deficient(self._h, ctypes.byref(f)))
        return bool(f.value)

    def close(self) -> None:
        if self._h is not None and _lib is not None:
            lib().cd_destroy(self._h)
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


#: size of the per-device workspace of cd_step_static (CD_STATIC_SCRATCH_BYTES)
STATIC_SCRATCH_BYTES = 64 << 20


def step_static(m: int, n: int, r_max: int, prev_norm, step: int, G, M, X, Q, mu: float, eta: float,
                r: Optional[int] = None, *, grad_dtype: str = "f32", tau: float = 0.5, eps: float = 1e-8,
                eta_local_scale: float = 1.0, policy: int = POLICY_RMMC, H: int = 1,
                weight_decay: float = 0.0, stream=None) -> Tuple[float, bool, int, int]:
    """One step of one layer through cd_step_static, the entry point that
    allocates nothing (its workspace is a fixed per-device array).  The
    caller owns the layer state: `prev_norm` is a one-element fp64 GPU tensor
    (or a device address), `step` the steps taken so far.  Returns
    (rmmc, sync_flag, status, step + 1)."""
    r = Q.shape[1] if r is None and hasattr(Q, "shape") else r
    for t, role in ((G, "G"), (M, "M"), (X, "X"), (Q, "Q")):
        check_operand(t, role, m, n, r, grad_dtype)
    if not isinstance(prev_norm, int):
        if str(prev_norm.dtype) != "torch.float64" or prev_norm.numel() != 1 or prev_norm.device.type != "cuda":
            raise ValueError("prev_norm: expected one float64 element on a GPU")
    desc = LayerDesc(m, n, r_max, BF16 if grad_dtype == "bf16" else F32, tau, eps, eta_local_scale,
                     policy, H, weight_decay)
    st_c = ctypes.c_longlong(step)
    res = Result()
    st = lib().cd_step_static(ctypes.byref(desc), _ptr(prev_norm), ctypes.byref(st_c), _ptr(G), _ptr(M),
                              _ptr(X), _ptr(Q), mu, eta, r, _stream_handle(stream), ctypes.byref(res))
    _check(st, allow=(CD_OK, CD_ENONFINITE))
    return res.rmmc, bool(res.sync_flag), st, st_c.value


class PointerArray:
    """One device address per layer, marshalled once (Group.pack); keeps the
    tensors alive so the addresses stay valid."""

    def __init__(self, array, keep):
        self.array = array
        self._keep = list(keep)
        self._checked = set()      # (role, r) pairs the tensors were checked for

    def __len__(self):
        return len(self.array)


class Group:
    """Layers stepped together: the gate takes the max of RMMC over all of them."""

    def __init__(self, layers: Sequence[Layer]):
        self._h = None
        self.layers = list(layers)
        arr = (ctypes.c_void_p * len(layers))(*[L.handle.value for L in layers])
        h = ctypes.c_void_p()
        _check(lib().cd_group_create(arr, len(layers), ctypes.byref(h)))
        self._h = h

    def _check_all(self, tensors, role: str, r: int) -> None:
        if len(tensors) != len(self.layers):
            raise ValueError(f"{role}: expected {len(self.layers)} tensors, got {len(tensors)}")
        for L, t in zip(self.layers, tensors):
            L.check(t, role, r)

    def pack(self, tensors, role: Optional[str] = None, r: Optional[int] = None) -> "PointerArray":
        """The device addresses of one tensor per layer, marshalled once: pass
        the result to step() in place of the list while those tensors live.
        With `role` ("G", "M", "X" or "Q"; Q also takes its rank r, by default
        its column count) the tensors are checked here, once; otherwise on the
        first step() that uses the array."""
        n = len(self.layers)
        if len(tensors) != n:
            raise ValueError(f"expected {n} tensors, got {len(tensors)}")
        pa = PointerArray((ctypes.c_void_p * n)(*[_ptr(t) for t in tensors]), tensors)
        if role is not None:
            if role == "Q" and r is None:
                r = next((t.shape[1] for t in tensors if not isinstance(t, int)), None)
            key = r if role == "Q" else None
            self._check_all(tensors, role, r if r is not None else 1)
            pa._checked.add((role, key))
        return pa

    def step(self, G, M, X, Q, mu: float, eta: float, r: int, stream=None, wait: bool = True):
        """One step over every layer; returns (rmmc_max, sync_flag, rmmc_per_layer, status).
        G, M, X, Q are lists with one tensor (or address) per layer, or pack() results.
        wait=False: the asynchronous step (returns None; see last_result)."""
        n = len(self.layers)

        def mk(ts, role):
            # a packed array is checked once (per rank, for Q), a list on every call
            if isinstance(ts, PointerArray):
                key = (role, r if role == "Q" else None)
                if key not in ts._checked:
                    self._check_all(ts._keep, role, r)
                    ts._checked.add(key)
                return ts.array
            self._check_all(ts, role, r)
            return (ctypes.c_void_p * n)(*[_ptr(t) for t in ts])

        arrays = [mk(G, "G"), mk(M, "M"), mk(X, "X"), mk(Q, "Q")]
        if not wait:
            _check(lib().cd_group_step(self._h, *arrays, mu, eta, r, _stream_handle(stream), None, None))
            return None
        per = (ctypes.c_double * n)()
        res = Result()
        st = lib().cd_group_step(self._h, *arrays, mu, eta, r,
                                 _stream_handle(stream), per, ctypes.byref(res))
        _check(st, allow=(CD_OK, CD_ENONFINITE))
        return res.rmmc, bool(res.sync_flag), list(per), st

    def last_result(self):
        """(rmmc_max, sync_flag, rmmc_per_layer, status) of the last step, once
        its work has finished; status CD_OK, CD_ENONFINITE or CD_ERANKDEF."""
        n = len(self.layers)
        per = (ctypes.c_double * n)()
        res = Result()
        st = lib().cd_group_last_result(self._h, per, ctypes.byref(res))
        _check(st, allow=(CD_OK, CD_ENONFINITE, CD_ERANKDEF))
        return res.rmmc, bool(res.sync_flag), list(per), st

    def set_timing(self, enable: bool, kinds=None) -> None:
        """Bracket kernel launches with HIP events (see kernel_times): every
        launch, or only those of the kernel kinds named in `kinds`."""
        spec = None if not kinds else ",".join(kinds).encode()
        _check(lib().cd_group_set_timing_kinds(self._h, spec))
        _check(lib().cd_group_set_timing(self._h, 1 if enable else 0))

    def kernel_times(self) -> dict:
        """{kind: dict(launches, total_ms, bytes, flops)} since timing was
        switched on or since the previous call (which clears the records)."""
        buf = (KernelTime * 32)()
        n = ctypes.c_int()
        _check(lib().cd_group_kernel_times(self._h, buf, 32, ctypes.byref(n)))
        return {buf[k].name.decode(): dict(launches=buf[k].launches, total_ms=buf[k].total_ms,
                                           bytes=buf[k].bytes, flops=buf[k].flops)
                for k in range(min(n.value, 32))}

    def close(self) -> None:
        if self._h is not None and _lib is not None:
            lib().cd_group_destroy(self._h)
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
