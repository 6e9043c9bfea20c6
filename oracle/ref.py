"""numpy wrapper around the C oracle (``ref_conv.c``).

TEST INFRASTRUCTURE ONLY (tests, smoke check, CPU baseline).  Every function
takes and returns host numpy arrays; nothing here touches a GPU.

Operator definitions follow the standard Conv2D of CNN inference that the
paper optimises (Sec. 3.2.2) and its claim that optimised schedules keep the
model semantics (Sec. 4.2, Sec. 5); the readings taken where the paper is
silent (no flip, symmetric zero padding, floor output size, fp64
accumulation) are written at the top of ``ref_conv.c``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ref_conv.c")
_LIB = os.path.join(_HERE, "libref_conv.so")
_lock = threading.Lock()
_lib = None

_CFLAGS = ["-O2", "-fopenmp", "-fno-fast-math", "-ffp-contract=off", "-std=c11",
           "-Wall", "-Wextra", "-shared", "-fPIC"]


def lib_path() -> str:
    return _LIB


def build(force: bool = True) -> str:
    """Compile ``ref_conv.c`` into ``libref_conv.so`` next to it (gcc)."""
    global _lib
    with _lock:
        if force or not os.path.exists(_LIB):
            tmp = _LIB + ".tmp%d" % os.getpid()
            subprocess.run(["gcc", *_CFLAGS, "-o", tmp, _SRC, "-lm"], check=True)
            os.replace(tmp, _LIB)
            _lib = None
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        with _lock:
            if _lib is None:
                lib = ctypes.CDLL(_LIB)
                i, p, v = ctypes.c_int, ctypes.c_void_p, ctypes.c_long
                lib.ref_out_dims.argtypes = [i] * 6 + [ctypes.POINTER(i)] * 2
                sig = [i] * 10 + [p, p, p, p, i]
                lib.ref_conv2d_f32.argtypes = sig
                lib.ref_conv2d_bf16.argtypes = sig
                lib.ref_conv2d_res.argtypes = [i] * 11 + [p, p, p, p, p, i]
                lib.ref_dwconv2d_f32.argtypes = [i] * 8 + [p, p, p, p, i]
                lib.ref_maxpool2d_f32.argtypes = [i] * 8 + [p, p]
                lib.ref_add_act_f32.argtypes = [v, p, p, p, i]
                lib.ref_f32_to_bf16.argtypes = [v, p, p]
                lib.ref_num_threads.argtypes = []
                for f in ("ref_num_threads", "ref_out_dims", "ref_conv2d_f32", "ref_conv2d_bf16",
                          "ref_conv2d_res",
                          "ref_dwconv2d_f32", "ref_maxpool2d_f32", "ref_add_act_f32",
                          "ref_f32_to_bf16"):
                    getattr(lib, f).restype = i
                _lib = lib
    return _lib


def num_threads() -> int:
    """OpenMP threads the oracle's parallel loops use."""
    return int(_load().ref_num_threads())


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    a = np.asarray(a)
    if a.dtype != dtype:
        raise TypeError(f"expected {dtype}, got {a.dtype}")
    return np.ascontiguousarray(a)


def out_dims(H, W, R, S, stride, pad):
    """Output height/width: floor((H + 2*pad - R)/stride) + 1 (and likewise for W)."""
    P, Q = ctypes.c_int(), ctypes.c_int()
    rc = _load().ref_out_dims(H, W, R, S, stride, pad, ctypes.byref(P), ctypes.byref(Q))
    if rc != 0:
        raise ValueError("bad geometry")
    return P.value, Q.value


def _conv(fn, x, w, bias, stride, pad, groups, relu, xdtype, res=None):
    x = _c(x, xdtype)
    w = _c(w, xdtype)
    N, C, H, W = x.shape
    K, Cg, R, S = w.shape
    if groups <= 0 or C % groups or K % groups or Cg * groups != C:
        raise ValueError("groups does not match the tensor shapes")
    b = None if bias is None else _c(bias, np.float32)
    if b is not None and b.shape != (K,):
        raise ValueError("bias must have shape (K,)")
    P, Q = out_dims(H, W, R, S, stride, pad)
    if P <= 0 or Q <= 0:
        raise ValueError("empty output")
    y = np.empty((N, K, P, Q), np.float32)
    if res is not None:
        r = _c(res, np.float32)
        if r.shape != y.shape:
            raise ValueError("res must have the output's shape")
        rc = _load().ref_conv2d_res(N, C, H, W, K, R, S, stride, pad, groups,
                                    1 if xdtype == np.uint16 else 0, _ptr(x), _ptr(w), _ptr(b),
                                    _ptr(r), _ptr(y), 1 if relu else 0)
        if rc != 0:
            raise RuntimeError(f"oracle conv failed ({rc})")
        return y
    rc = fn(N, C, H, W, K, R, S, stride, pad, groups, _ptr(x), _ptr(w), _ptr(b), _ptr(y),
            1 if relu else 0)
    if rc != 0:
        raise RuntimeError(f"oracle conv failed ({rc})")
    return y


def conv2d(x, w, bias=None, stride=1, pad=0, groups=1, relu=False, res=None):
    """Conv2D on fp32 arrays: x [N][C][H][W], w [K][C/groups][R][S] -> y [N][K][P][Q].

    With ``res`` (fp32, y's shape): the fused residual join of a bottleneck
    block (operator fusion, Sec. 3.2.3), act(conv + bias + res) summed in fp64."""
    return _conv(_load().ref_conv2d_f32, x, w, bias, stride, pad, groups, relu, np.float32, res)


def conv2d_bf16(x_bits, w_bits, bias=None, stride=1, pad=0, groups=1, relu=False, res=None):
    """Conv2D with x and w given as bf16 bit patterns (uint16); bias, res and y are fp32."""
    return _conv(_load().ref_conv2d_bf16, x_bits, w_bits, bias, stride, pad, groups, relu,
                 np.uint16, res)


def dwconv2d(x, w, bias=None, stride=1, pad=0, relu=False):
    """Depthwise conv: w [C][1][R][S]; the grouped conv with groups = C = K."""
    x = _c(x, np.float32)
    w = _c(w, np.float32)
    N, C, H, W = x.shape
    if w.shape[0] != C or w.shape[1] != 1:
        raise ValueError("depthwise weights must be [C][1][R][S]")
    R, S = w.shape[2], w.shape[3]
    b = None if bias is None else _c(bias, np.float32)
    P, Q = out_dims(H, W, R, S, stride, pad)
    y = np.empty((N, C, P, Q), np.float32)
    rc = _load().ref_dwconv2d_f32(N, C, H, W, R, S, stride, pad, _ptr(x), _ptr(w), _ptr(b),
                                  _ptr(y), 1 if relu else 0)
    if rc != 0:
        raise RuntimeError(f"oracle dwconv failed ({rc})")
    return y


def maxpool2d(x, R, S, stride, pad=0):
    """Max-pool; padded positions never win."""
    x = _c(x, np.float32)
    N, C, H, W = x.shape
    P, Q = out_dims(H, W, R, S, stride, pad)
    y = np.empty((N, C, P, Q), np.float32)
    rc = _load().ref_maxpool2d_f32(N, C, H, W, R, S, stride, pad, _ptr(x), _ptr(y))
    if rc != 0:
        raise RuntimeError(f"oracle maxpool failed ({rc})")
    return y


def add_act(a, b, relu=True):
    """Residual join: act(a + b) elementwise in fp32."""
    a = _c(a, np.float32)
    b = _c(b, np.float32)
    if a.shape != b.shape:
        raise ValueError("shape mismatch")
    y = np.empty_like(a)
    rc = _load().ref_add_act_f32(a.size, _ptr(a), _ptr(b), _ptr(y), 1 if relu else 0)
    if rc != 0:
        raise RuntimeError("oracle add failed")
    return y


def f32_to_bf16(x):
    """fp32 -> bf16 bit patterns, round to nearest even."""
    x = _c(x, np.float32)
    y = np.empty(x.shape, np.uint16)
    rc = _load().ref_f32_to_bf16(x.size, _ptr(x), _ptr(y))
    if rc != 0:
        raise RuntimeError("oracle bf16 rounding failed")
    return y


def bf16_to_f32(bits):
    """bf16 bit patterns -> exact fp32 values (bf16 is the upper half of fp32)."""
    bits = _c(bits, np.uint16)
    return (bits.astype(np.uint32) << 16).view(np.float32)


def conv2d_bf16_cl(x_bits, w_bits, bias=None, stride=1, pad=0, groups=1, relu=False, res_bits=None):
    """One layer of a network whose activations stay bf16 and channel-last
    between layers (the graph-level layout choice and operator fusion of
    Sec. 3.2.3): x bf16 bits [N][H][W][C], w bf16 bits [K][C/groups][R][S],
    bias fp32 [K], res bf16 bits [N][P][Q][K] or None; returns bf16 bits
    [N][P][Q][K].

    Reading: the layer's value is the definition above, act(conv + bias +
    res) summed in fp64 and rounded once to fp32 (conv2d_bf16 with the
    residual widened exactly), then rounded to bf16, nearest even
    (f32_to_bf16).  The layout change is a transpose, no arithmetic."""
    x = np.ascontiguousarray(np.transpose(_c(x_bits, np.uint16), (0, 3, 1, 2)))
    res = None
    if res_bits is not None:
        res = bf16_to_f32(np.ascontiguousarray(np.transpose(_c(res_bits, np.uint16), (0, 3, 1, 2))))
    y = conv2d_bf16(x, w_bits, bias, stride, pad, groups, relu, res=res)
    return f32_to_bf16(np.ascontiguousarray(np.transpose(y, (0, 2, 3, 1))))


def maxpool2d_bf16_cl(x_bits, R, S, stride, pad=0):
    """Max-pool of bf16 channel-last bits [N][H][W][C] -> [N][P][Q][C]: the
    maxima of the exactly widened values are input values, so they convert
    back to bf16 without rounding."""
    x = bf16_to_f32(np.ascontiguousarray(np.transpose(_c(x_bits, np.uint16), (0, 3, 1, 2))))
    y = maxpool2d(x, R, S, stride, pad)
    return f32_to_bf16(np.ascontiguousarray(np.transpose(y, (0, 2, 3, 1))))
