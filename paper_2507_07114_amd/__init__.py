"""Python binding of liblossy.so, the HIP library of the lossy data-parallel step.

Argument marshalling only: every function forwards device pointers, sizes
and torch's current HIP stream to the C entry point of the same name
(declared in include/lossy.h) and raises on a non-zero return code.  All
computation happens in the library's HIP kernels; there is no fallback.

torch is imported before the library is loaded so that both share the one
HIP runtime already in the process.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

__all__ = [
    # entry points of include/lossy.h
    "ll_masks", "ll_ages_update", "lossy_aggregate", "shard_step", "lossy_broadcast",
    "drift_stats", "lossy_step_fused", "ll_workspace_bytes", "ll_masks_workspace_bytes",
    "ll_last_error",
    # argument structs and their builders
    "LossSpec", "OptSpec", "Ext", "bernoulli", "gilbert_elliott", "sgd", "sgd_momentum", "adam",
    "ext", "ESTIMATORS",
    # helpers
    "drift_buffer", "read_drift", "library_path", "LossyError",
    "LL_F32", "LL_BF16", "LL_DIR_GRAD", "LL_DIR_BCAST",
]

LL_OK, LL_EINVAL, LL_EALIGN, LL_EHIP = 0, -1, -2, -3
LL_F32, LL_BF16 = 0, 1
LL_LOSS_BERNOULLI, LL_LOSS_GILBERT_ELLIOTT = 0, 1
LL_SGD, LL_SGD_MOMENTUM, LL_ADAM = 0, 1, 2
LL_DIR_GRAD, LL_DIR_BCAST = 0, 1
LL_EST_ARRIVED_MEAN, LL_EST_HORVITZ_THOMPSON, LL_EST_STALE_FILL = 0, 1, 2
ESTIMATORS = {"arrived_mean": LL_EST_ARRIVED_MEAN, "horvitz_thompson": LL_EST_HORVITZ_THOMPSON,
              "stale_fill": LL_EST_STALE_FILL}

_PKG = os.path.dirname(os.path.abspath(__file__))


def library_path() -> str:
    return os.path.join(_PKG, "liblossy.so")


class LossyError(RuntimeError):
    def __init__(self, func: str, code: int, msg: str):
        super().__init__(f"{func} failed with code {code}: {msg}")
        self.code = code


class LossSpec(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("p", ctypes.c_double), ("p_gb", ctypes.c_double),
                ("p_bg", ctypes.c_double), ("loss_good", ctypes.c_double),
                ("loss_bad", ctypes.c_double), ("seed", ctypes.c_uint64)]


class OptSpec(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("lr", ctypes.c_float), ("momentum", ctypes.c_float),
                ("beta1", ctypes.c_float), ("beta2", ctypes.c_float), ("eps", ctypes.c_float),
                ("fallback_lambda", ctypes.c_float)]


class Ext(ctypes.Structure):
    """ll_ext: variants of the step (see include/lossy.h).  Built by ext(),
    which also keeps the tensors behind its device pointers alive."""
    _fields_ = [("estimator", ctypes.c_int32), ("owner", ctypes.c_int32),
                ("reliable", ctypes.c_void_p), ("g_prev", ctypes.c_void_p),
                ("ages", ctypes.c_void_p), ("arrival_prob", ctypes.c_double),
                ("parity_group", ctypes.c_int32)]


def ext(estimator: str = "arrived_mean", owner: int = -1,
        reliable: Optional[torch.Tensor] = None, g_prev: Optional[torch.Tensor] = None,
        ages: Optional[torch.Tensor] = None, arrival_prob: float = 0.0,
        parity_group: int = 0) -> Ext:
    if estimator not in ESTIMATORS:
        raise ValueError(f"unknown estimator {estimator!r}")
    e = Ext(ESTIMATORS[estimator], owner, _flat(reliable, "reliable", torch.uint8),
            None if g_prev is None else _rows(g_prev, "g_prev")[0],
            _flat(ages, "ages", torch.int16), arrival_prob, parity_group)
    e._tensors = (reliable, g_prev, ages)  # the pointers above stay valid while e lives
    return e


def _ext_ref(e: Optional[Ext]):
    return None if e is None else ctypes.byref(e)


def bernoulli(p: float, seed: int = 0) -> LossSpec:
    return LossSpec(LL_LOSS_BERNOULLI, p, 0.0, 0.0, 0.0, 0.0, seed)


def gilbert_elliott(p_gb: float, p_bg: float, loss_good: float, loss_bad: float,
                    seed: int = 0) -> LossSpec:
    return LossSpec(LL_LOSS_GILBERT_ELLIOTT, 0.0, p_gb, p_bg, loss_good, loss_bad, seed)


def sgd(lr: float, fallback_lambda: float = 0.0) -> OptSpec:
    return OptSpec(LL_SGD, lr, 0.0, 0.0, 0.0, 0.0, fallback_lambda)


def sgd_momentum(lr: float, momentum: float, fallback_lambda: float = 0.0) -> OptSpec:
    return OptSpec(LL_SGD_MOMENTUM, lr, momentum, 0.0, 0.0, 0.0, fallback_lambda)


def adam(lr: float, beta1: float, beta2: float, eps: float,
         fallback_lambda: float = 0.0) -> OptSpec:
    return OptSpec(LL_ADAM, lr, 0.0, beta1, beta2, eps, fallback_lambda)


_lib = None
_vp = ctypes.c_void_p
_i32, _i64, _u64, _f32 = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_float
_SIGNATURES = {
    "ll_masks": (ctypes.c_int, [_i32, _i64, _u64, _i32, ctypes.POINTER(LossSpec), _vp, _vp, _vp,
                                ctypes.c_size_t, ctypes.POINTER(Ext), _vp]),
    "ll_ages_update": (ctypes.c_int, [_i32, _i64, _vp, _vp, _vp]),
    "ll_masks_workspace_bytes": (ctypes.c_size_t, [_i32, _i64]),
    "lossy_aggregate": (ctypes.c_int, [_i32, _i64, _i64, _i32, _vp, _i64, _vp, _f32, _vp, _vp,
                                       _vp, ctypes.POINTER(Ext), _vp]),
    "shard_step": (ctypes.c_int, [ctypes.POINTER(OptSpec), _i64, _u64, _vp, _vp, _vp, _vp, _vp]),
    "lossy_broadcast": (ctypes.c_int, [_i32, _i64, _i64, _vp, _i32, _vp, _i64, _vp, _vp]),
    "drift_stats": (ctypes.c_int, [_i32, _i64, _i64, _i32, _vp, _i64, _vp, _vp, _vp,
                                   ctypes.c_size_t, _vp, _vp]),
    "lossy_step_fused": (ctypes.c_int, [_i32, _i64, _i64, _u64, ctypes.POINTER(LossSpec),
                                        ctypes.POINTER(LossSpec), _vp, _vp, _i32, _vp, _i64,
                                        ctypes.POINTER(OptSpec), _vp, _vp, _vp, _i32, _vp, _i64,
                                        _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp,
                                        ctypes.POINTER(Ext), _vp]),
    "ll_workspace_bytes": (ctypes.c_size_t, [_i32, _i64, _i64]),
    "ll_last_error": (ctypes.c_char_p, []),
}


def _load():
    global _lib
    if _lib is None:
        path = library_path()
        if not os.path.exists(path):
            raise RuntimeError(f"HIP library {path} is not built; run "
                               "`python -m paper_2507_07114_amd.build` first")
        lib = ctypes.CDLL(path)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def ll_last_error() -> str:
    return _load().ll_last_error().decode()


def ll_workspace_bytes(n: int, d: int, packet: int) -> int:
    return int(_load().ll_workspace_bytes(n, d, packet))


def _check(name: str, code: int):
    if code != LL_OK:
        raise LossyError(name, code, ll_last_error())


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def _dev(t: Optional[torch.Tensor], name: str, dtype=None) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must have dtype {dtype}, got {t.dtype}")
    return t.data_ptr()


def _rows(t: torch.Tensor, name: str):
    """(pointer, ld, dtype code) of a [n][ld] row-major device tensor."""
    if t.dim() != 2:
        raise ValueError(f"{name} must be 2-D")
    if t.numel() and t.stride(1) != 1:
        raise ValueError(f"{name} must have unit column stride")
    if t.dtype == torch.float32:
        code = LL_F32
    elif t.dtype == torch.bfloat16:
        code = LL_BF16
    else:
        raise ValueError(f"{name} must be float32 or bfloat16, got {t.dtype}")
    if t.numel() == 0:
        return None, 8, code
    return _dev(t, name), t.stride(0), code


def _flat(t: Optional[torch.Tensor], name: str, dtype) -> Optional[int]:
    if t is not None and not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return _dev(t, name, dtype)


def ll_masks(n: int, num_packets: int, step: int, direction: int, loss: LossSpec,
             arrived: torch.Tensor, ge_state: Optional[torch.Tensor] = None,
             workspace: Optional[torch.Tensor] = None, ext: Optional[Ext] = None) -> None:
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check("ll_masks", _load().ll_masks(
        n, num_packets, step, direction, ctypes.byref(loss),
        _flat(ge_state, "ge_state", torch.uint8), _flat(arrived, "arrived", torch.uint8),
        _dev(workspace, "workspace"), ws_bytes, _ext_ref(ext), _stream()))


def ll_ages_update(arrived_bc: torch.Tensor, ages: torch.Tensor) -> None:
    """ages (int16 storage of uint16 counts) [n][P] after a broadcast."""
    n, P = arrived_bc.shape
    _check("ll_ages_update", _load().ll_ages_update(
        n, P, _flat(arrived_bc, "arrived_bc", torch.uint8), _flat(ages, "ages", torch.int16),
        _stream()))


def ll_masks_workspace_bytes(n: int, num_packets: int) -> int:
    return int(_load().ll_masks_workspace_bytes(n, num_packets))


def lossy_aggregate(grads: torch.Tensor, arrived: torch.Tensor, *, d: int, packet: int,
                    g_hat: torch.Tensor, fallback_lambda: float = 0.0,
                    theta: Optional[torch.Tensor] = None,
                    counts: Optional[torch.Tensor] = None, ext: Optional[Ext] = None) -> None:
    gp, ld, gt = _rows(grads, "grads")
    _check("lossy_aggregate", _load().lossy_aggregate(
        grads.shape[0], d, packet, gt, gp, ld, _flat(arrived, "arrived", torch.uint8),
        fallback_lambda, _flat(theta, "theta", torch.float32),
        _flat(g_hat, "g_hat", torch.float32), _flat(counts, "counts", torch.int32),
        _ext_ref(ext), _stream()))


def shard_step(opt: OptSpec, step: int, theta: torch.Tensor, g_hat: torch.Tensor,
               m: Optional[torch.Tensor] = None, v: Optional[torch.Tensor] = None,
               d: Optional[int] = None) -> None:
    d = theta.numel() if d is None else d
    _check("shard_step", _load().shard_step(
        ctypes.byref(opt), d, step, _flat(theta, "theta", torch.float32),
        _flat(m, "m", torch.float32), _flat(v, "v", torch.float32),
        _flat(g_hat, "g_hat", torch.float32), _stream()))


def lossy_broadcast(theta: torch.Tensor, replicas: torch.Tensor, arrived_bc: torch.Tensor, *,
                    d: int, packet: int) -> None:
    rp, ld, rt = _rows(replicas, "replicas")
    _check("lossy_broadcast", _load().lossy_broadcast(
        replicas.shape[0], d, packet, _flat(theta, "theta", torch.float32), rt, rp, ld,
        _flat(arrived_bc, "arrived_bc", torch.uint8), _stream()))


def drift_buffer(device="cuda") -> torch.Tensor:
    """Device storage for one ll_drift record (4 doubles + 2 uint64)."""
    return torch.zeros(6, dtype=torch.float64, device=device)


def read_drift(buf: torch.Tensor) -> dict:
    """Copy an ll_drift record to the host (synchronises with its stream)."""
    h = buf.detach().cpu()
    ints = h.view(torch.int64)
    return dict(max_abs=float(h[0]), mean_sq=float(h[1]), rms=float(h[2]),
                mean_abs_to_master=float(h[3]), stale_packets=int(ints[4]),
                empty_packets=int(ints[5]))


def drift_stats(replicas: torch.Tensor, *, d: int, packet: int, workspace: torch.Tensor,
                out: torch.Tensor, theta: Optional[torch.Tensor] = None,
                arrived_bc: Optional[torch.Tensor] = None) -> None:
    rp, ld, rt = _rows(replicas, "replicas")
    _check("drift_stats", _load().drift_stats(
        replicas.shape[0], d, packet, rt, rp, ld, _flat(theta, "theta", torch.float32),
        _flat(arrived_bc, "arrived_bc", torch.uint8), _dev(workspace, "workspace"),
        workspace.numel() * workspace.element_size(), _dev(out, "out", torch.float64),
        _stream()))


def lossy_step_fused(*, d: int, packet: int, step: int, loss_g: LossSpec, loss_b: LossSpec,
                     grads: torch.Tensor, opt: OptSpec, theta: torch.Tensor,
                     replicas: torch.Tensor, m: Optional[torch.Tensor] = None,
                     v: Optional[torch.Tensor] = None,
                     ge_state_g: Optional[torch.Tensor] = None,
                     ge_state_b: Optional[torch.Tensor] = None,
                     arrived_g: Optional[torch.Tensor] = None,
                     arrived_b: Optional[torch.Tensor] = None,
                     counts: Optional[torch.Tensor] = None,
                     workspace: Optional[torch.Tensor] = None,
                     drift: Optional[torch.Tensor] = None, ext: Optional[Ext] = None) -> None:
    gp, ldg, gt = _rows(grads, "grads")
    rp, ldr, rt = _rows(replicas, "replicas")
    if replicas.shape[0] != grads.shape[0]:
        raise ValueError("grads and replicas must have the same number of rows")
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check("lossy_step_fused", _load().lossy_step_fused(
        grads.shape[0], d, packet, step, ctypes.byref(loss_g), ctypes.byref(loss_b),
        _flat(ge_state_g, "ge_state_g", torch.uint8), _flat(ge_state_b, "ge_state_b", torch.uint8),
        gt, gp, ldg, ctypes.byref(opt), _flat(theta, "theta", torch.float32),
        _flat(m, "m", torch.float32), _flat(v, "v", torch.float32), rt, rp, ldr,
        _flat(arrived_g, "arrived_g", torch.uint8), _flat(arrived_b, "arrived_b", torch.uint8),
        _flat(counts, "counts", torch.int32), _dev(workspace, "workspace"), ws_bytes,
        _dev(drift, "drift", torch.float64), _ext_ref(ext), _stream()))
