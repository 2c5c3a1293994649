"""Python binding of libhbmprobe.so, the HBM bandwidth probes declared in
include/hbm_probe.h (measurement only; not part of the lossy step).

Argument marshalling only: each function forwards device pointers and sizes
of torch tensors and torch's current HIP stream to the C entry point of the
same name and raises on a non-zero return code.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

__all__ = ["hbm_probe_copy", "hbm_probe_read", "hbm_probe_write", "hbm_probe_rows",
           "probe_library_path", "SINK_BYTES"]

SINK_BYTES = 4096
_PKG = os.path.dirname(os.path.abspath(__file__))
_lib = None
_vp, _i32, _i64, _sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
_SIGNATURES = {
    "hbm_probe_copy": [_vp, _vp, _sz, _vp],
    "hbm_probe_read": [_vp, _sz, _vp, _vp],
    "hbm_probe_write": [_vp, _sz, _vp],
    "hbm_probe_rows": [_vp, _i32, _vp, _i32, _i64, _i64, _vp, _vp],
}


def probe_library_path() -> str:
    return os.path.join(_PKG, "libhbmprobe.so")


def _load():
    global _lib
    if _lib is None:
        path = probe_library_path()
        if not os.path.exists(path):
            raise RuntimeError(f"HIP library {path} is not built; run "
                               "`python -m paper_2507_07114_amd.build` first")
        lib = ctypes.CDLL(path)
        for name, args in _SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = ctypes.c_int
            fn.argtypes = args
        _lib = lib
    return _lib


def _check(name: str, code: int):
    if code != 0:
        raise RuntimeError(f"{name} failed with code {code}")


def _ptr(t: Optional[torch.Tensor], name: str) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous device tensor")
    return t.data_ptr()


def _nbytes(t: torch.Tensor) -> int:
    return t.numel() * t.element_size()


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def hbm_probe_copy(src: torch.Tensor, dst: torch.Tensor) -> int:
    """Copy src into dst (same byte size); returns the bytes moved."""
    n = _nbytes(src)
    if _nbytes(dst) < n:
        raise ValueError("dst is smaller than src")
    _check("hbm_probe_copy", _load().hbm_probe_copy(_ptr(src, "src"), _ptr(dst, "dst"), n,
                                                    _stream()))
    return 2 * n


def hbm_probe_read(src: torch.Tensor, sink: torch.Tensor) -> int:
    if _nbytes(sink) < SINK_BYTES:
        raise ValueError(f"sink needs {SINK_BYTES} bytes")
    n = _nbytes(src)
    _check("hbm_probe_read", _load().hbm_probe_read(_ptr(src, "src"), n, _ptr(sink, "sink"),
                                                    _stream()))
    return n


def hbm_probe_write(dst: torch.Tensor) -> int:
    n = _nbytes(dst)
    _check("hbm_probe_write", _load().hbm_probe_write(_ptr(dst, "dst"), n, _stream()))
    return n


def hbm_probe_rows(src: Optional[torch.Tensor], n_read: int, dst: Optional[torch.Tensor],
                   n_write: int, row_bytes: int, sink: torch.Tensor) -> int:
    """The many-row shape over [rows][ld] tensors (row stride from src or dst,
    which must agree); returns the bytes moved."""
    ref = src if src is not None else dst
    if ref is None or ref.dim() != 2:
        raise ValueError("src or dst must be a 2-D device tensor")
    ld_bytes = ref.stride(0) * ref.element_size()
    for t, rows, name in ((src, n_read, "src"), (dst, n_write, "dst")):
        if t is None:
            if rows:
                raise ValueError(f"{name} is missing")
            continue
        if t.dim() != 2 or t.stride(0) * t.element_size() != ld_bytes or t.stride(1) != 1:
            raise ValueError(f"{name} must be [rows][ld] with the same row stride")
        if t.shape[0] < rows or t.shape[1] * t.element_size() < row_bytes:
            raise ValueError(f"{name} is smaller than {rows} rows of {row_bytes} bytes")
    if _nbytes(sink) < SINK_BYTES:
        raise ValueError(f"sink needs {SINK_BYTES} bytes")
    _check("hbm_probe_rows", _load().hbm_probe_rows(
        None if src is None else src.data_ptr(), n_read,
        None if dst is None else dst.data_ptr(), n_write, row_bytes, ld_bytes,
        _ptr(sink, "sink"), _stream()))
    return (n_read + n_write) * row_bytes
