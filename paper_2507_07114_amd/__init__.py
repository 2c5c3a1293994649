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
    "drift_stats", "lossy_step_fused", "lossy_step_fused_noalloc", "ll_workspace_bytes",
    "ll_masks_workspace_bytes", "LL_NOALLOC_SCRATCH_BYTES",
    "ll_last_error", "ll_set_pacing", "ll_get_pacing",
    # argument structs and their builders
    "LossSpec", "OptSpec", "Ext", "ExtArgs", "Pacing", "bernoulli", "gilbert_elliott", "sgd", "sgd_momentum", "adam",
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
LL_NOALLOC_SCRATCH_BYTES = 16 << 20
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


class ExtArgs:
    """Variants of the step as tensors and numbers (see ext()); turned into
    an ll_ext only when a call has checked them against its other arguments."""

    def __init__(self, estimator: int, owner: int, reliable, g_prev, ages, arrival_prob: float,
                 parity_group: int):
        self.estimator = estimator
        self.owner = owner
        self.reliable = reliable
        self.g_prev = g_prev
        self.ages = ages
        self.arrival_prob = arrival_prob
        self.parity_group = parity_group

    def check(self, n: int, num_packets: int, grads: Optional[torch.Tensor]):
        if self.reliable is not None:
            _need_numel(self.reliable, "reliable", num_packets, torch.uint8)
        if self.ages is not None:
            _need_shape(self.ages, "ages", (n, num_packets), torch.int16)
        if self.g_prev is not None and grads is not None:
            g = self.g_prev
            if (g.dim() != 2 or tuple(g.shape) != tuple(grads.shape) or g.dtype != grads.dtype
                    or (g.numel() and g.stride() != grads.stride())):
                raise ValueError(
                    f"g_prev must match grads in shape, row stride and dtype: got "
                    f"{tuple(g.shape)} stride {g.stride()} {g.dtype}, grads "
                    f"{tuple(grads.shape)} stride {grads.stride()} {grads.dtype}")

    def as_struct(self) -> "Ext":
        e = Ext(self.estimator, self.owner, _flat(self.reliable, "reliable", torch.uint8),
                None if self.g_prev is None else _rows(self.g_prev, "g_prev")[0],
                _flat(self.ages, "ages", torch.int16), self.arrival_prob, self.parity_group)
        e._tensors = (self.reliable, self.g_prev, self.ages)  # pointers stay valid while e lives
        return e


def ext(estimator: str = "arrived_mean", owner: int = -1,
        reliable: Optional[torch.Tensor] = None, g_prev: Optional[torch.Tensor] = None,
        ages: Optional[torch.Tensor] = None, arrival_prob: float = 0.0,
        parity_group: int = 0) -> ExtArgs:
    if estimator not in ESTIMATORS:
        raise ValueError(f"unknown estimator {estimator!r}")
    return ExtArgs(ESTIMATORS[estimator], owner, reliable, g_prev, ages, arrival_prob,
                   parity_group)


def _ext_ref(e, n: int = 0, num_packets: int = 0, grads: Optional[torch.Tensor] = None):
    """ll_ext* for a call: None, a raw Ext as given, or an ExtArgs checked
    against the call's sizes and then marshalled."""
    if e is None:
        return None
    if isinstance(e, ExtArgs):
        e.check(n, num_packets, grads)
        e = e.as_struct()
    return ctypes.byref(e)


def _num_packets(d: int, packet: int) -> int:
    return (d + packet - 1) // packet if packet >= 1 and d >= 0 else 0


def _need_numel(t: Optional[torch.Tensor], name: str, numel: int, dtype=None):
    if t is None:
        return
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must have dtype {dtype}, got {t.dtype}")
    if t.numel() < numel:
        raise ValueError(f"{name} has {t.numel()} elements, needs at least {numel}")


def _need_shape(t: Optional[torch.Tensor], name: str, shape, dtype=None):
    if t is None:
        return
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must have dtype {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")


def _need_rows(t: torch.Tensor, name: str, d: int):
    if t.dim() != 2:
        raise ValueError(f"{name} must be 2-D")
    if t.shape[1] < d:
        raise ValueError(f"{name} rows hold {t.shape[1]} elements, fewer than d={d}")


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
    "lossy_step_fused_noalloc": (ctypes.c_int, [_i32, _i64, _i64, _u64, ctypes.POINTER(LossSpec),
                                                ctypes.POINTER(LossSpec), _vp, _vp, _i32, _vp,
                                                _i64, ctypes.POINTER(OptSpec), _vp, _vp, _vp,
                                                _i32, _vp, _i64, _vp, _vp, _vp, _vp,
                                                ctypes.POINTER(Ext), _vp]),
    "ll_workspace_bytes": (ctypes.c_size_t, [_i32, _i64, _i64]),
    "ll_last_error": (ctypes.c_char_p, []),
    "ll_set_pacing": (ctypes.c_int, [ctypes.c_void_p]),
    "ll_get_pacing": (ctypes.c_int, [ctypes.c_void_p]),
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


class Pacing(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int32), ("bytes_per_s", ctypes.c_double),
                ("gap_us", ctypes.c_double), ("lead_us", ctypes.c_double),
                ("overlap", ctypes.c_int32), ("resident", ctypes.c_int32),
                ("headroom", ctypes.c_double), ("tail_us", ctypes.c_double),
                ("persistent", ctypes.c_int32), ("bytes_per_s_f32", ctypes.c_double)]


PACE_MODES = {"auto": 0, "always": 1, "never": 2}


def ll_set_pacing(mode: str = "auto", bytes_per_s: float = 6.3e12, gap_us: float = 2.0,
                  lead_us: float = 4.0, overlap: int = 1, resident: int = 1,
                  headroom: float = 1.0, tail_us: float = 3.0, persistent: int = 0,
                  bytes_per_s_f32: float = 5.9e12) -> None:
    """Process-wide pacing of lossy_step_fused (a performance setting; see
    include/lossy.h)."""
    if mode not in PACE_MODES:
        raise ValueError(f"unknown pacing mode {mode!r}")
    cfg = Pacing(PACE_MODES[mode], bytes_per_s, gap_us, lead_us, overlap, resident, headroom,
                 tail_us, persistent, bytes_per_s_f32)
    _check("ll_set_pacing", _load().ll_set_pacing(ctypes.byref(cfg)))


def ll_get_pacing() -> dict:
    cfg = Pacing()
    _check("ll_get_pacing", _load().ll_get_pacing(ctypes.byref(cfg)))
    mode = {v: k for k, v in PACE_MODES.items()}[cfg.mode]
    return dict(mode=mode, bytes_per_s=cfg.bytes_per_s, gap_us=cfg.gap_us, lead_us=cfg.lead_us,
                overlap=cfg.overlap, resident=cfg.resident, headroom=cfg.headroom,
                tail_us=cfg.tail_us, persistent=cfg.persistent,
                bytes_per_s_f32=cfg.bytes_per_s_f32)


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
             workspace: Optional[torch.Tensor] = None, ext=None) -> None:
    _need_shape(arrived, "arrived", (n, num_packets), torch.uint8)
    _need_numel(ge_state, "ge_state", n, torch.uint8)
    ref = _ext_ref(ext, n, num_packets)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check("ll_masks", _load().ll_masks(
        n, num_packets, step, direction, ctypes.byref(loss),
        _flat(ge_state, "ge_state", torch.uint8), _flat(arrived, "arrived", torch.uint8),
        _dev(workspace, "workspace"), ws_bytes, ref, _stream()))


def ll_ages_update(arrived_bc: torch.Tensor, ages: torch.Tensor) -> None:
    """ages (int16 storage of uint16 counts) [n][P] after a broadcast."""
    n, P = arrived_bc.shape
    _need_shape(ages, "ages", (n, P), torch.int16)
    _check("ll_ages_update", _load().ll_ages_update(
        n, P, _flat(arrived_bc, "arrived_bc", torch.uint8), _flat(ages, "ages", torch.int16),
        _stream()))


def ll_masks_workspace_bytes(n: int, num_packets: int) -> int:
    return int(_load().ll_masks_workspace_bytes(n, num_packets))


def lossy_aggregate(grads: torch.Tensor, arrived: torch.Tensor, *, d: int, packet: int,
                    g_hat: torch.Tensor, fallback_lambda: float = 0.0,
                    theta: Optional[torch.Tensor] = None,
                    counts: Optional[torch.Tensor] = None, ext=None) -> None:
    _need_rows(grads, "grads", d)
    n, P = grads.shape[0], _num_packets(d, packet)
    _need_shape(arrived, "arrived", (n, P), torch.uint8)
    _need_numel(g_hat, "g_hat", d, torch.float32)
    _need_numel(theta, "theta", d, torch.float32)
    _need_numel(counts, "counts", P, torch.int32)
    ref = _ext_ref(ext, n, P, grads)
    gp, ld, gt = _rows(grads, "grads")
    _check("lossy_aggregate", _load().lossy_aggregate(
        n, d, packet, gt, gp, ld, _flat(arrived, "arrived", torch.uint8),
        fallback_lambda, _flat(theta, "theta", torch.float32),
        _flat(g_hat, "g_hat", torch.float32), _flat(counts, "counts", torch.int32),
        ref, _stream()))


def shard_step(opt: OptSpec, step: int, theta: torch.Tensor, g_hat: torch.Tensor,
               m: Optional[torch.Tensor] = None, v: Optional[torch.Tensor] = None,
               d: Optional[int] = None) -> None:
    d = theta.numel() if d is None else d
    for t, name in ((theta, "theta"), (g_hat, "g_hat"), (m, "m"), (v, "v")):
        _need_numel(t, name, d, torch.float32)
    _check("shard_step", _load().shard_step(
        ctypes.byref(opt), d, step, _flat(theta, "theta", torch.float32),
        _flat(m, "m", torch.float32), _flat(v, "v", torch.float32),
        _flat(g_hat, "g_hat", torch.float32), _stream()))


def lossy_broadcast(theta: torch.Tensor, replicas: torch.Tensor, arrived_bc: torch.Tensor, *,
                    d: int, packet: int) -> None:
    _need_rows(replicas, "replicas", d)
    _need_numel(theta, "theta", d, torch.float32)
    _need_shape(arrived_bc, "arrived_bc", (replicas.shape[0], _num_packets(d, packet)),
                torch.uint8)
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
    _need_rows(replicas, "replicas", d)
    _need_numel(theta, "theta", d, torch.float32)
    _need_shape(arrived_bc, "arrived_bc", (replicas.shape[0], _num_packets(d, packet)),
                torch.uint8)
    _need_numel(out, "out", 6, torch.float64)
    rp, ld, rt = _rows(replicas, "replicas")
    _check("drift_stats", _load().drift_stats(
        replicas.shape[0], d, packet, rt, rp, ld, _flat(theta, "theta", torch.float32),
        _flat(arrived_bc, "arrived_bc", torch.uint8), _dev(workspace, "workspace"),
        workspace.numel() * workspace.element_size(), _dev(out, "out", torch.float64),
        _stream()))


def _fused_args(d, packet, step, loss_g, loss_b, grads, opt, theta, replicas, m, v,
                ge_state_g, ge_state_b, arrived_g, arrived_b, counts, drift, ext):
    """Checked, marshalled arguments of the fused step, in C order up to (and
    without) the workspace, and the tail after it."""
    _need_rows(grads, "grads", d)
    _need_rows(replicas, "replicas", d)
    if replicas.shape[0] != grads.shape[0]:
        raise ValueError("grads and replicas must have the same number of rows")
    n, P = grads.shape[0], _num_packets(d, packet)
    for t, name in ((theta, "theta"), (m, "m"), (v, "v")):
        _need_numel(t, name, d, torch.float32)
    _need_shape(arrived_g, "arrived_g", (n, P), torch.uint8)
    _need_shape(arrived_b, "arrived_b", (n, P), torch.uint8)
    _need_numel(counts, "counts", P, torch.int32)
    _need_numel(ge_state_g, "ge_state_g", n, torch.uint8)
    _need_numel(ge_state_b, "ge_state_b", n, torch.uint8)
    _need_numel(drift, "drift", 6, torch.float64)
    ref = _ext_ref(ext, n, P, grads)
    gp, ldg, gt = _rows(grads, "grads")
    rp, ldr, rt = _rows(replicas, "replicas")
    head = (grads.shape[0], d, packet, step, ctypes.byref(loss_g), ctypes.byref(loss_b),
            _flat(ge_state_g, "ge_state_g", torch.uint8),
            _flat(ge_state_b, "ge_state_b", torch.uint8),
            gt, gp, ldg, ctypes.byref(opt), _flat(theta, "theta", torch.float32),
            _flat(m, "m", torch.float32), _flat(v, "v", torch.float32), rt, rp, ldr,
            _flat(arrived_g, "arrived_g", torch.uint8), _flat(arrived_b, "arrived_b", torch.uint8),
            _flat(counts, "counts", torch.int32))
    tail = (_dev(drift, "drift", torch.float64), ref, _stream())
    return head, tail


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
                     drift: Optional[torch.Tensor] = None, ext=None) -> None:
    head, tail = _fused_args(d, packet, step, loss_g, loss_b, grads, opt, theta, replicas, m, v,
                             ge_state_g, ge_state_b, arrived_g, arrived_b, counts, drift, ext)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check("lossy_step_fused", _load().lossy_step_fused(
        *head, _dev(workspace, "workspace"), ws_bytes, *tail))


def lossy_step_fused_noalloc(*, d: int, packet: int, step: int, loss_g: LossSpec,
                             loss_b: LossSpec, grads: torch.Tensor, opt: OptSpec,
                             theta: torch.Tensor, replicas: torch.Tensor,
                             m: Optional[torch.Tensor] = None, v: Optional[torch.Tensor] = None,
                             ge_state_g: Optional[torch.Tensor] = None,
                             ge_state_b: Optional[torch.Tensor] = None,
                             arrived_g: Optional[torch.Tensor] = None,
                             arrived_b: Optional[torch.Tensor] = None,
                             counts: Optional[torch.Tensor] = None,
                             drift: Optional[torch.Tensor] = None, ext=None) -> None:
    """lossy_step_fused with the library's static device scratch instead of a
    workspace (for callers that cannot allocate)."""
    head, tail = _fused_args(d, packet, step, loss_g, loss_b, grads, opt, theta, replicas, m, v,
                             ge_state_g, ge_state_b, arrived_g, arrived_b, counts, drift, ext)
    _check("lossy_step_fused_noalloc", _load().lossy_step_fused_noalloc(*head, *tail))
