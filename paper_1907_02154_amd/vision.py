"""Thin Python binding over the vision operators of libmiconv.so
(``include/mivision.h``): the three-stage prefix sum, segmented argsort and
box_nms of the paper's Sec. 3.1.1.

Argument marshalling only, as in ``miconv``: dtype / device / shape checks,
raw device pointers, torch's current HIP stream, and a workspace tensor
allocated here when the caller passes none (the C entry points never
allocate).  All arithmetic runs in the library's HIP kernels.
"""
from __future__ import annotations

import ctypes
from typing import Optional

import torch

from . import miconv
from .miconv import _check, _dev, _ptr, _stream

NMS_MAX_CANDIDATES = 4096   # MIVISION_NMS_MAX_CANDIDATES

_bound = False


def lib() -> ctypes.CDLL:
    """libmiconv.so with the argument types of the vision entry points set."""
    global _bound
    L = miconv.lib()
    if not _bound:
        i, p, l, f, sz = ctypes.c_int, ctypes.c_void_p, ctypes.c_long, ctypes.c_float, ctypes.c_size_t
        L.vision_scan_workspace_bytes.argtypes = [i, l]
        L.vision_scan_workspace_bytes.restype = l
        L.vision_scan_i32.argtypes = [i, l, p, p, i, p, sz, p]
        L.vision_scan_i32.restype = i
        L.vision_argsort_workspace_bytes.argtypes = [l, i]
        L.vision_argsort_workspace_bytes.restype = l
        L.vision_segmented_argsort.argtypes = [l, i, p, p, i, p, p, sz, p]
        L.vision_segmented_argsort.restype = i
        L.vision_box_nms_workspace_bytes.argtypes = [i, i, i, i]
        L.vision_box_nms_workspace_bytes.restype = l
        L.vision_box_nms.argtypes = [i, i, i, p, p, f, f, i, i, i, i, i, p, sz, p]
        L.vision_box_nms.restype = i
        _bound = True
    return L


def _bytes(rc: int, what: str) -> int:
    if rc < 0:
        _check(int(rc), what)
    return int(rc)


def _ws(nbytes: int, ws: Optional[torch.Tensor], device) -> Optional[torch.Tensor]:
    if nbytes == 0:
        return None
    if ws is None:
        return miconv.workspace(nbytes, device)
    if ws.device.type != "cuda" or ws.numel() * ws.element_size() < nbytes or ws.data_ptr() % 256:
        raise ValueError(f"workspace must be a 256-byte aligned device tensor of at least {nbytes} bytes")
    return ws


def scan_workspace_bytes(rows: int, n: int) -> int:
    return _bytes(lib().vision_scan_workspace_bytes(rows, n), "vision_scan_workspace_bytes")


def scan_i32(x: torch.Tensor, y: Optional[torch.Tensor] = None, exclusive: bool = False,
             ws: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Prefix sum of each row of x (int32 [rows][n], or [n] as one row)."""
    _dev(x, torch.int32, "x")
    rows, n = (1, x.shape[0]) if x.dim() == 1 else tuple(x.shape)
    if x.dim() not in (1, 2):
        raise ValueError("x must be [n] or [rows][n]")
    if y is None:
        y = torch.empty_like(x)
    _dev(y, torch.int32, "y")
    if y.shape != x.shape:
        raise ValueError("y must have x's shape")
    w = _ws(scan_workspace_bytes(rows, n), ws, x.device)
    _check(lib().vision_scan_i32(rows, n, _ptr(x), _ptr(y), int(exclusive), _ptr(w),
                                 0 if w is None else w.numel(), _stream(stream)), "vision_scan_i32")
    return y


def argsort_workspace_bytes(n: int, segments: int) -> int:
    return _bytes(lib().vision_argsort_workspace_bytes(n, segments), "vision_argsort_workspace_bytes")


def segmented_argsort(keys: torch.Tensor, offsets: torch.Tensor, descending: bool = True,
                      out: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                      stream=None) -> torch.Tensor:
    """keys fp32 [n], offsets int32 [segments + 1] (device) -> int32 [n] of
    indices local to each segment, in rank order."""
    _dev(keys, torch.float32, "keys", 1)
    _dev(offsets, torch.int32, "offsets", 1)
    n, segments = keys.shape[0], offsets.shape[0] - 1
    if out is None:
        out = torch.empty(n, dtype=torch.int32, device=keys.device)
    _dev(out, torch.int32, "out", 1)
    if out.shape[0] != n:
        raise ValueError("out must have n elements")
    w = _ws(argsort_workspace_bytes(n, segments), ws, keys.device)
    _check(lib().vision_segmented_argsort(n, segments, _ptr(keys), _ptr(offsets), int(descending), _ptr(out),
                                          _ptr(w), 0 if w is None else w.numel(), _stream(stream)),
           "vision_segmented_argsort")
    return out


def box_nms_workspace_bytes(batch: int, num: int, width: int, topk: int = -1) -> int:
    return _bytes(lib().vision_box_nms_workspace_bytes(batch, num, width, topk), "vision_box_nms_workspace_bytes")


def box_nms(data: torch.Tensor, overlap_thresh: float = 0.5, valid_thresh: float = 0.0, topk: int = -1,
            id_index: int = 0, score_index: int = 1, coord_start: int = 2, force_suppress: bool = False,
            out: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """data fp32 [batch][num][width] -> out of the same shape: kept rows first
    in rank order, every other value -1."""
    _dev(data, torch.float32, "data", 3)
    B, N, W = data.shape
    if out is None:
        out = torch.empty_like(data)
    _dev(out, torch.float32, "out", 3)
    if out.shape != data.shape:
        raise ValueError("out must have data's shape")
    w = _ws(box_nms_workspace_bytes(B, N, W, topk), ws, data.device)
    _check(lib().vision_box_nms(B, N, W, _ptr(data), _ptr(out), float(overlap_thresh), float(valid_thresh),
                                int(topk), int(id_index), int(score_index), int(coord_start), int(force_suppress),
                                _ptr(w), 0 if w is None else w.numel(), _stream(stream)), "vision_box_nms")
    return out
