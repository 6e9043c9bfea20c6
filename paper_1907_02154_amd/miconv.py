"""Thin Python binding over libmiconv.so (``include/miconv.h``).

Argument marshalling only: every function checks dtype / device / layout,
reads the extents off the tensor shapes and passes raw device pointers plus
torch's current HIP stream to the C entry point of the same name.  PyTorch
provides device memory and streams; all arithmetic runs in the library's HIP
kernels.  If the library is missing the import of any entry point raises.
"""
from __future__ import annotations

import ctypes
import os
import re
from typing import Optional

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmiconv.so")
HEADER = os.path.join(os.path.dirname(_PKG), "include", "miconv.h")
HEADERS = [HEADER, os.path.join(os.path.dirname(_PKG), "include", "mivision.h")]

OK = 0
(ERR_NULL, ERR_SHAPE, ERR_GROUPS, ERR_UNSUPPORTED, ERR_TOO_LARGE, ERR_ALIGN, ERR_HIP,
 ERR_WORKSPACE) = range(-1, -9, -1)
ALGO_AUTO, ALGO_DIRECT, ALGO_IGEMM, ALGO_WAVE = 0, 1, 2, 3
# enum miconv_plan_mode: which entry point a plan is made for
PLAN_PLAIN, PLAN_WS, PLAN_PACKED, PLAN_STACK = 0, 1, 2, 3
_PLAN = {"plain": PLAN_PLAIN, "ws": PLAN_WS, "packed": PLAN_PACKED, "stack": PLAN_STACK}

_lib = None


class MiconvError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        extra = ""
        if status == ERR_HIP:
            extra = f", hipError {lib().miconv_last_hip_error()}"
        super().__init__(f"{what}: {strerror(status)} ({status}{extra})")


def lib() -> ctypes.CDLL:
    """Load libmiconv.so (built by ``paper_1907_02154_amd.build``); raise if absent."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() first")
        L = ctypes.CDLL(LIB_PATH)
        i, p, l = ctypes.c_int, ctypes.c_void_p, ctypes.c_long
        conv = [i] * 10 + [p, p, p, p, i, p]
        L.conv2d_fwd.argtypes = conv
        L.conv2d_fwd_bf16.argtypes = conv
        L.dwconv2d_fwd.argtypes = conv
        L.conv2d_fwd_algo.argtypes = [i] * 10 + [p, p, p, p, i, i, p]
        L.conv2d_fwd_bf16_algo.argtypes = [i] * 10 + [p, p, p, p, i, i, p]
        L.miconv_out_dims.argtypes = [i] * 6 + [ctypes.POINTER(i)] * 2
        L.maxpool2d_fwd.argtypes = [i] * 8 + [p, p, p]
        L.add_act_fwd.argtypes = [l, p, p, p, i, p]
        L.cast_f32_to_bf16.argtypes = [l, p, p, p]
        L.conv2d_fwd_res.argtypes = [i] * 12 + [p, p, p, p, p, i, p]
        L.conv2d_fwd_ex.argtypes = [i] * 12 + [p, p, p, p, p, l, i, p]
        L.conv2d_packed_weight_bytes.argtypes = [i] * 11
        L.conv2d_packed_weight_bytes.restype = l
        L.conv2d_pack_weights.argtypes = [i] * 11 + [p, p, p]
        L.conv2d_pack_weights.restype = i
        L.conv2d_fwd_packed.argtypes = [i] * 11 + [p, p, p, p, i, p]
        L.conv2d_fwd_packed.restype = i
        L.conv2d_describe.argtypes = [i] * 13 + [ctypes.c_char_p, i, ctypes.POINTER(i)]
        L.conv2d_workspace_bytes.argtypes = [i] * 12
        L.conv2d_workspace_bytes.restype = l
        L.conv2d_fwd_ws.argtypes = [i] * 12 + [p, p, p, p, p, l, i, p, ctypes.c_size_t, p]
        L.conv2d_fwd_ws.restype = i
        L.conv2d_fwd_noalloc.argtypes = [i] * 12 + [p, p, p, p, p, l, i, p]
        L.conv2d_fwd_noalloc.restype = i
        L.conv2d_cl_workspace_bytes.argtypes = [i] * 11
        L.conv2d_cl_workspace_bytes.restype = l
        L.conv2d_fwd_cl.argtypes = [i] * 11 + [p, p, p, p, p, i, p, ctypes.c_size_t, p]
        L.conv2d_fwd_cl.restype = i
        L.conv2d_cl_describe.argtypes = [i] * 11 + [ctypes.c_char_p, i, ctypes.POINTER(i)]
        L.conv2d_cl_describe.restype = i
        L.maxpool2d_nhwc_bf16.argtypes = [i] * 8 + [p, p, p]
        L.maxpool2d_nhwc_bf16.restype = i
        L.conv2d_describe.restype = i
        L.miconv_stack_create.argtypes = [p, i, ctypes.POINTER(p)]
        L.miconv_stack_size.argtypes = [p]
        L.miconv_stack_describe.argtypes = [p, i, ctypes.c_char_p, i]
        L.miconv_stack_launch.argtypes = [p, p]
        L.miconv_stack_launches.argtypes = [p]
        L.miconv_stack_launch_info.argtypes = [p, i, ctypes.c_char_p, i]
        L.miconv_stack_capture.argtypes = [p, i, i, p]
        L.miconv_stack_launch_timed.argtypes = [p, i, p]
        L.miconv_stack_replay.argtypes = [p, p]
        L.miconv_stack_times.argtypes = [p, p, l]
        L.miconv_stack_destroy.argtypes = [p]
        L.miconv_stack_overlap.argtypes = [p, i]
        for f in ("miconv_stack_create", "miconv_stack_size", "miconv_stack_describe",
                  "miconv_stack_launches", "miconv_stack_launch_info",
                  "miconv_stack_launch", "miconv_stack_launch_timed", "miconv_stack_capture", "miconv_stack_replay",
                  "miconv_stack_times", "miconv_stack_destroy", "miconv_stack_overlap"):
            getattr(L, f).restype = i
        L.miconv_strerror.argtypes = [i]
        L.miconv_strerror.restype = ctypes.c_char_p
        L.miconv_last_hip_error.argtypes = []
        L.miconv_version.argtypes = []
        for f in ("conv2d_fwd", "conv2d_fwd_bf16", "dwconv2d_fwd", "conv2d_fwd_algo",
                  "conv2d_fwd_bf16_algo",
                  "miconv_out_dims", "maxpool2d_fwd", "add_act_fwd", "cast_f32_to_bf16",
                  "miconv_last_hip_error", "miconv_version"):
            getattr(L, f).restype = i
        _lib = L
    return _lib


def header_functions() -> list:
    """Names of the functions ``include/miconv.h`` and ``include/mivision.h`` declare."""
    names = set()
    for h in HEADERS:
        with open(h) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names |= set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M))
    return sorted(names)


def strerror(status: int) -> str:
    return lib().miconv_strerror(status).decode()


def _check(rc: int, what: str):
    if rc != OK:
        raise MiconvError(rc, what)


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else t.data_ptr()


def _dev(t: torch.Tensor, dtype, name: str, ndim: Optional[int] = None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims")


def _image_strided(t: torch.Tensor, name: str) -> int:
    """Checks that a 4-d fp32 device tensor is dense within each image (a
    channel range of a wider NCHW tensor qualifies) and returns its image
    stride in elements."""
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda" or t.dtype != torch.float32 \
            or t.dim() != 4:
        raise TypeError(f"{name} must be a 4-d float32 device tensor")
    N, K, P, Q = t.shape
    if t.stride()[1:] != (P * Q, Q, 1) and K * P * Q > 1:
        raise ValueError(f"{name} must be dense within each image")
    if N > 1 and t.stride(0) < K * P * Q:
        # e.g. an expanded view: images would overlap in memory
        raise ValueError(f"{name}: images overlap (image stride {t.stride(0)} < {K * P * Q})")
    return t.stride(0) if N > 1 else K * P * Q


def out_dims(H: int, W: int, R: int, S: int, stride: int, pad: int):
    P, Q = ctypes.c_int(), ctypes.c_int()
    rc = lib().miconv_out_dims(H, W, R, S, stride, pad, ctypes.byref(P), ctypes.byref(Q))
    _check(rc, "miconv_out_dims")
    return P.value, Q.value


def _conv_common(fn, x, w, bias, y, stride, pad, groups, relu, stream, xdtype, extra=()):
    _dev(x, xdtype, "x", 4)
    _dev(w, xdtype, "w", 4)
    _dev(y, torch.float32, "y", 4)
    if bias is not None:
        _dev(bias, torch.float32, "bias", 1)
    N, C, H, W = x.shape
    K, Cg, R, S = w.shape
    if groups <= 0 or Cg * groups != C:
        raise ValueError("w.shape[1] * groups must equal C")
    if bias is not None and bias.shape[0] != K:
        raise ValueError("bias must have K entries")
    P, Q = out_dims(H, W, R, S, stride, pad)
    if tuple(y.shape) != (N, K, P, Q):
        raise ValueError(f"y must have shape {(N, K, P, Q)}, got {tuple(y.shape)}")
    rc = fn(N, C, H, W, K, R, S, stride, pad, groups, _ptr(x), _ptr(w), _ptr(bias), _ptr(y),
            1 if relu else 0, *extra, _stream(stream))
    _check(rc, fn.__name__)
    return y


def conv2d_fwd(x, w, bias, y, stride=1, pad=0, groups=1, relu=False, stream=None):
    """fp32 conv2d: x [N][C][H][W], w [K][C/groups][R][S], bias [K] or None -> y [N][K][P][Q]."""
    return _conv_common(lib().conv2d_fwd, x, w, bias, y, stride, pad, groups, relu, stream,
                        torch.float32)


def conv2d_fwd_algo(x, w, bias, y, stride=1, pad=0, groups=1, relu=False, algo=ALGO_AUTO,
                    stream=None):
    """conv2d_fwd with an explicit algorithm (ALGO_AUTO / ALGO_DIRECT / ALGO_IGEMM / ALGO_WAVE)."""
    f = lib().conv2d_fwd_algo
    _dev(x, torch.float32, "x", 4)
    return _conv_common(f, x, w, bias, y, stride, pad, groups, relu, stream, torch.float32,
                        extra=(int(algo),))


def conv2d_fwd_res(x, w, bias, res, y, stride=1, pad=0, groups=1, relu=False, algo=ALGO_AUTO,
                   stream=None):
    """y = act(conv(x, w) + bias + res) with the join in the conv's epilogue.

    x and w fp32 or bf16 (the dtype selects conv2d_fwd or conv2d_fwd_bf16),
    res fp32 shaped like y, or None; res may be y itself."""
    xdt = torch.bfloat16 if x.dtype == torch.bfloat16 else torch.float32
    if res is not None:
        _dev(res, torch.float32, "res", 4)
        if tuple(res.shape) != tuple(y.shape):
            raise ValueError("res must have y's shape")
    f = lib().conv2d_fwd_res

    def call(N, C, H, W, K, R, S, stride_, pad_, groups_, px, pw, pb, py, relu_, stream_):
        return f(N, C, H, W, K, R, S, stride_, pad_, groups_, 1 if xdt == torch.bfloat16 else 0,
                 int(algo), px, pw, pb, _ptr(res), py, relu_, stream_)
    call.__name__ = "conv2d_fwd_res"
    return _conv_common(call, x, w, bias, y, stride, pad, groups, relu, stream, xdt)


def conv2d_fwd_ex(x, w, bias, y, stride=1, pad=0, groups=1, relu=False, res=None, algo=ALGO_AUTO,
                  stream=None):
    """y = act(conv(x, w) + bias [+ res]) where y (and res, with the same
    strides) may be a channel range of a wider NCHW tensor, e.g. big[:, 64:128]:
    its image stride is passed to the library."""
    xdt = torch.bfloat16 if x.dtype == torch.bfloat16 else torch.float32
    _dev(x, xdt, "x", 4)
    _dev(w, xdt, "w", 4)
    if bias is not None:
        _dev(bias, torch.float32, "bias", 1)
    ys = _image_strided(y, "y")
    if res is not None:
        if _image_strided(res, "res") != ys or tuple(res.shape) != tuple(y.shape):
            raise ValueError("res must have y's shape and strides")
    N, C, H, W = x.shape
    K, Cg, R, S = w.shape
    if groups <= 0 or Cg * groups != C:
        raise ValueError("w.shape[1] * groups must equal C")
    P, Q = out_dims(H, W, R, S, stride, pad)
    if tuple(y.shape) != (N, K, P, Q):
        raise ValueError(f"y must have shape {(N, K, P, Q)}, got {tuple(y.shape)}")
    rc = lib().conv2d_fwd_ex(N, C, H, W, K, R, S, stride, pad, groups, 1 if xdt == torch.bfloat16 else 0,
                             int(algo), _ptr(x), _ptr(w), _ptr(bias), _ptr(res), _ptr(y), ys,
                             1 if relu else 0, _stream(stream))
    _check(rc, "conv2d_fwd_ex")
    return y


def conv2d_workspace_bytes(N, C, H, W, K, R, S, stride, pad, groups=1, dtype="f32",
                           algo=ALGO_AUTO) -> int:
    """Bytes of workspace conv2d_fwd_ws needs for this shape (any pointer alignment)."""
    n = lib().conv2d_workspace_bytes(N, C, H, W, K, R, S, stride, pad, groups,
                                     1 if dtype == "bf16" else 0, int(algo))
    if n < 0:
        raise MiconvError(int(n), "conv2d_workspace_bytes")
    return n


def workspace(nbytes: int, device="cuda") -> Optional[torch.Tensor]:
    """A 256-byte aligned device buffer of at least nbytes (torch's caching
    allocator returns such blocks), or None for 0."""
    if nbytes <= 0:
        return None
    t = torch.empty(nbytes, dtype=torch.uint8, device=device)
    if t.data_ptr() % 256:
        raise RuntimeError("workspace not 256-byte aligned")
    return t


def conv2d_fwd_ws(x, w, bias, y, stride=1, pad=0, groups=1, relu=False, res=None, algo=ALGO_AUTO,
                  ws=None, stream=None):
    """conv2d_fwd_ex with a caller workspace: the fastest single-call plans
    (split reductions, channel-last staging, per-call filter packing).  ws is
    a uint8 device tensor of at least conv2d_workspace_bytes bytes; None
    allocates one from torch's caching allocator (the library never
    allocates)."""
    xdt = torch.bfloat16 if x.dtype == torch.bfloat16 else torch.float32
    _dev(x, xdt, "x", 4)
    _dev(w, xdt, "w", 4)
    if bias is not None:
        _dev(bias, torch.float32, "bias", 1)
    ys = _image_strided(y, "y")
    if res is not None:
        if _image_strided(res, "res") != ys or tuple(res.shape) != tuple(y.shape):
            raise ValueError("res must have y's shape and strides")
    N, C, H, W = x.shape
    K, Cg, R, S = w.shape
    if groups <= 0 or Cg * groups != C:
        raise ValueError("w.shape[1] * groups must equal C")
    P, Q = out_dims(H, W, R, S, stride, pad)
    if tuple(y.shape) != (N, K, P, Q):
        raise ValueError(f"y must have shape {(N, K, P, Q)}, got {tuple(y.shape)}")
    dt = 1 if xdt == torch.bfloat16 else 0
    if ws is None:
        ws = workspace(conv2d_workspace_bytes(N, C, H, W, K, R, S, stride, pad, groups,
                                              "bf16" if dt else "f32", algo), x.device)
    elif ws.device.type != "cuda" or ws.dtype != torch.uint8 or not ws.is_contiguous():
        raise TypeError("ws must be a contiguous uint8 device tensor")
    rc = lib().conv2d_fwd_ws(N, C, H, W, K, R, S, stride, pad, groups, dt, int(algo), _ptr(x), _ptr(w),
                             _ptr(bias), _ptr(res), _ptr(y), ys, 1 if relu else 0, _ptr(ws),
                             0 if ws is None else ws.numel(), _stream(stream))
    _check(rc, "conv2d_fwd_ws")
    return y


NOALLOC_SCRATCH_BYTES = 32 << 20   # MICONV_NOALLOC_SCRATCH_BYTES


def conv2d_fwd_noalloc(x, w, bias, y, stride=1, pad=0, groups=1, relu=False, res=None, algo=ALGO_AUTO,
                       stream=None):
    """conv2d_fwd_ws on the library's fixed per-GPU scratch (nothing is
    allocated by anyone); plans needing more than NOALLOC_SCRATCH_BYTES fail
    with ERR_WORKSPACE.  Calls that may overlap on one GPU race on the scratch."""
    xdt = torch.bfloat16 if x.dtype == torch.bfloat16 else torch.float32
    _dev(x, xdt, "x", 4)
    _dev(w, xdt, "w", 4)
    if bias is not None:
        _dev(bias, torch.float32, "bias", 1)
    ys = _image_strided(y, "y")
    if res is not None:
        if _image_strided(res, "res") != ys or tuple(res.shape) != tuple(y.shape):
            raise ValueError("res must have y's shape and strides")
    N, C, H, W = x.shape
    K, Cg, R, S = w.shape
    if groups <= 0 or Cg * groups != C:
        raise ValueError("w.shape[1] * groups must equal C")
    P, Q = out_dims(H, W, R, S, stride, pad)
    if tuple(y.shape) != (N, K, P, Q):
        raise ValueError(f"y must have shape {(N, K, P, Q)}, got {tuple(y.shape)}")
    rc = lib().conv2d_fwd_noalloc(N, C, H, W, K, R, S, stride, pad, groups,
                                  1 if xdt == torch.bfloat16 else 0, int(algo), _ptr(x), _ptr(w),
                                  _ptr(bias), _ptr(res), _ptr(y), ys, 1 if relu else 0, _stream(stream))
    _check(rc, "conv2d_fwd_noalloc")
    return y


class PackedFilters:
    """Filters packed once for repeated calls of one layer shape
    (conv2d_pack_weights); ``forward`` runs conv2d_fwd_packed.  Holds the
    packed device buffer (or, when the kernel reads w as given, w itself)."""

    def __init__(self, w, x_shape, stride=1, pad=0, groups=1, stream=None):
        dtype = 1 if w.dtype == torch.bfloat16 else 0
        _dev(w, torch.bfloat16 if dtype else torch.float32, "w", 4)
        N, C, H, W = x_shape
        K, Cg, R, S = w.shape
        if groups <= 0 or Cg * groups != C:
            raise ValueError("w.shape[1] * groups must equal C")
        self.shape = (N, C, H, W, K, R, S, stride, pad, groups, dtype)
        nbytes = lib().conv2d_packed_weight_bytes(*self.shape)
        if nbytes < 0:
            raise MiconvError(int(nbytes), "conv2d_packed_weight_bytes")
        self.nbytes = nbytes
        if nbytes == 0:
            self.buf = w
        else:
            self.buf = torch.empty(nbytes, dtype=torch.uint8, device=w.device)
            _check(lib().conv2d_pack_weights(*self.shape, _ptr(w), _ptr(self.buf), _stream(stream)),
                   "conv2d_pack_weights")

    def forward(self, x, bias, y, relu=False, stream=None):
        N, C, H, W, K, R, S, stride, pad, groups, dtype = self.shape
        _dev(x, torch.bfloat16 if dtype else torch.float32, "x", 4)
        _dev(y, torch.float32, "y", 4)
        if bias is not None:
            _dev(bias, torch.float32, "bias", 1)
        if tuple(x.shape) != (N, C, H, W):
            raise ValueError(f"x must have shape {(N, C, H, W)}")
        P, Q = out_dims(H, W, R, S, stride, pad)
        if tuple(y.shape) != (N, K, P, Q):
            raise ValueError(f"y must have shape {(N, K, P, Q)}")
        _check(lib().conv2d_fwd_packed(*self.shape, _ptr(x), _ptr(self.buf), _ptr(bias), _ptr(y),
                                       1 if relu else 0, _stream(stream)), "conv2d_fwd_packed")
        return y


def conv2d_fwd_bf16(x, w, bias, y, stride=1, pad=0, groups=1, relu=False, stream=None):
    """bf16 x and w (torch.bfloat16), fp32 bias and y."""
    return _conv_common(lib().conv2d_fwd_bf16, x, w, bias, y, stride, pad, groups, relu, stream,
                        torch.bfloat16)


def conv2d_fwd_bf16_algo(x, w, bias, y, stride=1, pad=0, groups=1, relu=False, algo=ALGO_AUTO,
                         stream=None):
    """conv2d_fwd_bf16 with an explicit algorithm (ALGO_AUTO / ALGO_IGEMM / ALGO_DIRECT)."""
    return _conv_common(lib().conv2d_fwd_bf16_algo, x, w, bias, y, stride, pad, groups, relu, stream,
                        torch.bfloat16, extra=(int(algo),))


def dwconv2d_fwd(x, w, bias, y, stride=1, pad=1, relu=False, stream=None):
    """Depthwise conv: w [C][1][R][S], groups = C = K."""
    C = x.shape[1]
    return _conv_common(lib().dwconv2d_fwd, x, w, bias, y, stride, pad, C, relu, stream,
                        torch.float32)


def maxpool2d_fwd(x, y, R, S, stride, pad=0, stream=None):
    _dev(x, torch.float32, "x", 4)
    _dev(y, torch.float32, "y", 4)
    N, C, H, W = x.shape
    P, Q = out_dims(H, W, R, S, stride, pad)
    if tuple(y.shape) != (N, C, P, Q):
        raise ValueError(f"y must have shape {(N, C, P, Q)}")
    _check(lib().maxpool2d_fwd(N, C, H, W, R, S, stride, pad, _ptr(x), _ptr(y), _stream(stream)),
           "maxpool2d_fwd")
    return y


def add_act_fwd(a, b, y, relu=True, stream=None):
    for t, n in ((a, "a"), (b, "b"), (y, "y")):
        _dev(t, torch.float32, n)
    if a.shape != b.shape or a.shape != y.shape:
        raise ValueError("a, b, y must have one shape")
    _check(lib().add_act_fwd(a.numel(), _ptr(a), _ptr(b), _ptr(y), 1 if relu else 0,
                             _stream(stream)), "add_act_fwd")
    return y


def cast_f32_to_bf16(x, y, stream=None):
    _dev(x, torch.float32, "x")
    _dev(y, torch.bfloat16, "y")
    if x.shape != y.shape:
        raise ValueError("x and y must have one shape")
    _check(lib().cast_f32_to_bf16(x.numel(), _ptr(x), _ptr(y), _stream(stream)), "cast_f32_to_bf16")
    return y


def conv2d_describe(N, C, H, W, K, R, S, stride, pad, groups=1, dtype="f32", algo=ALGO_AUTO,
                    mode="ws"):
    """(kernel names, launch count) the library would use for this conv shape
    through the entry point of `mode`: "plain" (conv2d_fwd & co, no
    workspace), "ws" (conv2d_fwd_ws), "packed" (conv2d_fwd_packed) or
    "stack" (a miconv_stack layer)."""
    buf = ctypes.create_string_buffer(256)
    n = ctypes.c_int()
    rc = lib().conv2d_describe(N, C, H, W, K, R, S, stride, pad, groups,
                               1 if dtype == "bf16" else 0, int(algo), _PLAN[mode], buf, 256,
                               ctypes.byref(n))
    _check(rc, "conv2d_describe")
    return buf.value.decode(), n.value


OP_CONV_F32, OP_CONV_BF16, OP_DWCONV_F32, OP_MAXPOOL_BF16_NHWC, OP_MAXPOOL_F32 = 0, 1, 2, 3, 4
# enum miconv_layout flags
LAYOUT_NCHW, LAYOUT_X_NHWC, LAYOUT_Y_NHWC_BF16 = 0, 1, 2


class ConvDesc(ctypes.Structure):
    _fields_ = [("op", ctypes.c_int)] + [(n, ctypes.c_int) for n in
                                         ("N", "C", "H", "W", "K", "R", "S", "stride", "pad",
                                          "groups", "relu")] + \
               [("x", ctypes.c_void_p), ("w", ctypes.c_void_p), ("bias", ctypes.c_void_p),
                ("y", ctypes.c_void_p), ("res", ctypes.c_void_p), ("y_image_stride", ctypes.c_long),
                ("layout", ctypes.c_int)]


def _cl_shapes(x, w, y, stride, pad, groups, layout):
    """Extents of a channel-last bf16 layer from its tensors: x [N][H][W][C]
    (MICONV_LAYOUT_X_NHWC) or [N][C][H][W] bf16, y [N][P][Q][K] bf16
    (MICONV_LAYOUT_Y_NHWC_BF16) or [N][K][P][Q] fp32; checks y's shape."""
    _dev(x, torch.bfloat16, "x", 4)
    _dev(w, torch.bfloat16, "w", 4)
    if layout & LAYOUT_X_NHWC:
        N, H, W, C = x.shape
    else:
        N, C, H, W = x.shape
    K, Cg, R, S = w.shape
    if groups <= 0 or Cg * groups != C:
        raise ValueError("w.shape[1] * groups must equal C")
    P, Q = out_dims(H, W, R, S, stride, pad)
    if layout & LAYOUT_Y_NHWC_BF16:
        _dev(y, torch.bfloat16, "y", 4)
        want = (N, P, Q, K)
    else:
        _dev(y, torch.float32, "y", 4)
        want = (N, K, P, Q)
    if tuple(y.shape) != want:
        raise ValueError(f"y must have shape {want}, got {tuple(y.shape)}")
    return N, C, H, W, K, R, S


def conv2d_cl_workspace_bytes(N, C, H, W, K, R, S, stride, pad, groups=1, layout=LAYOUT_X_NHWC | LAYOUT_Y_NHWC_BF16):
    n = lib().conv2d_cl_workspace_bytes(N, C, H, W, K, R, S, stride, pad, groups, int(layout))
    if n < 0:
        raise MiconvError(int(n), "conv2d_cl_workspace_bytes")
    return n


def conv2d_fwd_cl(x, w, bias, y, stride=1, pad=0, groups=1, relu=False, res=None,
                  layout=LAYOUT_X_NHWC | LAYOUT_Y_NHWC_BF16, ws=None, stream=None):
    """bf16 conv with channel-last x and/or y (conv2d_fwd_cl); res like y.
    ws None: a workspace from torch's caching allocator."""
    N, C, H, W, K, R, S = _cl_shapes(x, w, y, stride, pad, groups, layout)
    if bias is not None:
        _dev(bias, torch.float32, "bias", 1)
    if res is not None:
        _dev(res, y.dtype, "res", 4)
        if tuple(res.shape) != tuple(y.shape):
            raise ValueError("res must have y's shape")
    if ws is None:
        ws = workspace(conv2d_cl_workspace_bytes(N, C, H, W, K, R, S, stride, pad, groups, layout), x.device)
    rc = lib().conv2d_fwd_cl(N, C, H, W, K, R, S, stride, pad, groups, int(layout), _ptr(x), _ptr(w),
                             _ptr(bias), _ptr(res), _ptr(y), 1 if relu else 0, _ptr(ws),
                             0 if ws is None else ws.numel(), _stream(stream))
    _check(rc, "conv2d_fwd_cl")
    return y


def conv2d_cl_describe(N, C, H, W, K, R, S, stride, pad, groups=1,
                       layout=LAYOUT_X_NHWC | LAYOUT_Y_NHWC_BF16):
    """(kernel names, launch count) of conv2d_fwd_cl for this shape and layout."""
    buf = ctypes.create_string_buffer(256)
    n = ctypes.c_int()
    _check(lib().conv2d_cl_describe(N, C, H, W, K, R, S, stride, pad, groups, int(layout), buf, 256,
                                    ctypes.byref(n)), "conv2d_cl_describe")
    return buf.value.decode(), n.value


def maxpool2d_nhwc_bf16(x, y, R, S, stride, pad=0, stream=None):
    """Max-pool on bf16 channel-last tensors: x [N][H][W][C] -> y [N][P][Q][C]."""
    _dev(x, torch.bfloat16, "x", 4)
    _dev(y, torch.bfloat16, "y", 4)
    N, H, W, C = x.shape
    P, Q = out_dims(H, W, R, S, stride, pad)
    if tuple(y.shape) != (N, P, Q, C):
        raise ValueError(f"y must have shape {(N, P, Q, C)}")
    _check(lib().maxpool2d_nhwc_bf16(N, C, H, W, R, S, stride, pad, _ptr(x), _ptr(y), _stream(stream)),
           "maxpool2d_nhwc_bf16")
    return y


class Stack:
    """A list of conv layers planned once by the library's stack executor.

    ``layers`` holds tuples ``(op, x, w, bias, y, stride, pad, groups, relu)``
    of device tensors (bias may be None), optionally with a tenth element
    ``res``: a residual shaped like y joined before the activation (or None).
    y (and res, with the same strides) may be a channel range of a wider NCHW
    tensor.  The tensors are kept referenced for the executor's lifetime.
    """

    def __init__(self, layers):
        self._keep = []
        descs = (ConvDesc * len(layers))()
        for d, layer in zip(descs, layers):
            if layer[0] == "maxpool":
                # ("maxpool", x, y, R, S, stride, pad): glue, bf16 channel-last
                # ([N][H][W][C] tensors) or fp32 NCHW
                _, x, y, R, S, stride, pad = layer
                cl = x.dtype == torch.bfloat16
                _dev(x, x.dtype if cl else torch.float32, "x", 4)
                _dev(y, x.dtype, "y", 4)
                if cl:
                    N, H, W, C = x.shape
                else:
                    N, C, H, W = x.shape
                P, Q = out_dims(H, W, R, S, stride, pad)
                want = (N, P, Q, C) if cl else (N, C, P, Q)
                if tuple(y.shape) != want:
                    raise ValueError(f"y must have shape {want}")
                d.op = OP_MAXPOOL_BF16_NHWC if cl else OP_MAXPOOL_F32
                d.N, d.C, d.H, d.W, d.K, d.R, d.S = N, C, H, W, C, R, S
                d.stride, d.pad, d.groups, d.relu = stride, pad, 1, 0
                d.x, d.y = x.data_ptr(), y.data_ptr()
                self._keep.append((x, y))
                continue
            op, x, w, bias, y, stride, pad, groups, relu = layer[:9]
            res = layer[9] if len(layer) > 9 else None
            layout = layer[10] if len(layer) > 10 else 0
            if layout:
                # a channel-last bf16 layer (conv2d_fwd_cl)
                if op != OP_CONV_BF16:
                    raise ValueError("a layout applies to bf16 convolutions only")
                N, C, H, W, K, R, S = _cl_shapes(x, w, y, stride, pad, groups, layout)
                if bias is not None:
                    _dev(bias, torch.float32, "bias", 1)
                if res is not None:
                    _dev(res, y.dtype, "res", 4)
                    if tuple(res.shape) != tuple(y.shape):
                        raise ValueError("res must have y's shape")
                d.op, d.N, d.C, d.H, d.W, d.K, d.R, d.S = op, N, C, H, W, K, R, S
                d.stride, d.pad, d.groups, d.relu = stride, pad, groups, 1 if relu else 0
                d.x, d.w, d.bias, d.y = x.data_ptr(), w.data_ptr(), _ptr(bias), y.data_ptr()
                d.res = _ptr(res)
                d.layout = int(layout)
                self._keep.append((x, w, bias, y, res))
                continue
            ys = _image_strided(y, "y")
            if res is not None:
                if _image_strided(res, "res") != ys or tuple(res.shape) != tuple(y.shape):
                    raise ValueError("res must have y's shape and strides")
            xdt = torch.bfloat16 if op == OP_CONV_BF16 else torch.float32
            _dev(x, xdt, "x", 4)
            _dev(w, xdt, "w", 4)
            if bias is not None:
                _dev(bias, torch.float32, "bias", 1)
            N, C, H, W = x.shape
            K, _, R, S = w.shape
            d.op, d.N, d.C, d.H, d.W, d.K, d.R, d.S = op, N, C, H, W, K, R, S
            d.stride, d.pad, d.groups, d.relu = stride, pad, groups, 1 if relu else 0
            d.x, d.w, d.bias, d.y = x.data_ptr(), w.data_ptr(), _ptr(bias), y.data_ptr()
            d.res = _ptr(res)
            d.y_image_stride = ys
            self._keep.append((x, w, bias, y, res))
        self.n = len(layers)
        self.steps = 0
        h = ctypes.c_void_p()
        _check(lib().miconv_stack_create(descs, self.n, ctypes.byref(h)), "miconv_stack_create")
        self._h = h
        self.launches = lib().miconv_stack_launches(h)

    def launch_info(self, j: int):
        """(layer index, kernel name) of kernel launch j of a pass."""
        buf = ctypes.create_string_buffer(256)
        layer = lib().miconv_stack_launch_info(self._h, j, buf, 256)
        if layer < 0:
            _check(layer, "miconv_stack_launch_info")
        return layer, buf.value.decode()

    def describe(self, i: int) -> str:
        buf = ctypes.create_string_buffer(256)
        rc = lib().miconv_stack_describe(self._h, i, buf, 256)
        if rc < 0:
            _check(rc, "miconv_stack_describe")
        return buf.value.decode()

    def launch(self, stream=None):
        _check(lib().miconv_stack_launch(self._h, _stream(stream)), "miconv_stack_launch")

    def launch_timed(self, steps: int, stream=None):
        _check(lib().miconv_stack_launch_timed(self._h, steps, _stream(stream)),
               "miconv_stack_launch_timed")
        self.steps = steps

    def overlap(self, enable: bool) -> int:
        """Overlap independent layers on a second stream in the next untimed
        capture (off by default); returns how many layers run there."""
        rc = lib().miconv_stack_overlap(self._h, 1 if enable else 0)
        if rc < 0:
            _check(rc, "miconv_stack_overlap")
        return rc

    def capture(self, steps: int, timed: bool, stream=None):
        _check(lib().miconv_stack_capture(self._h, steps, 1 if timed else 0, _stream(stream)),
               "miconv_stack_capture")
        self.steps = steps

    def replay(self, stream=None):
        _check(lib().miconv_stack_replay(self._h, _stream(stream)), "miconv_stack_replay")

    def times(self):
        import numpy as np
        out = np.empty(self.steps * self.launches, np.float32)
        _check(lib().miconv_stack_times(self._h, out.ctypes.data, out.size), "miconv_stack_times")
        return out.reshape(self.steps, self.launches)

    def close(self):
        if getattr(self, "_h", None):
            lib().miconv_stack_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# Allocating conveniences (output buffers come from torch's caching allocator).

def conv2d(x, w, bias=None, stride=1, pad=0, groups=1, relu=False, algo=ALGO_AUTO, stream=None,
           mode="ws"):
    """y = act(conv(x, w) + bias) into a new tensor.  mode "ws": conv2d_fwd_ws
    with a workspace from torch's caching allocator (the fastest plan);
    "plain": conv2d_fwd / conv2d_fwd_bf16 (and *_algo), no workspace."""
    N, _, H, W = x.shape
    K, _, R, S = w.shape
    P, Q = out_dims(H, W, R, S, stride, pad)
    y = torch.empty((N, K, P, Q), device=x.device, dtype=torch.float32)
    if mode == "ws":
        return conv2d_fwd_ws(x, w, bias, y, stride, pad, groups, relu, algo=algo, stream=stream)
    if mode != "plain":
        raise ValueError(f"mode must be 'ws' or 'plain', got {mode!r}")
    if x.dtype == torch.bfloat16:
        if algo == ALGO_AUTO:
            return conv2d_fwd_bf16(x, w, bias, y, stride, pad, groups, relu, stream)
        return conv2d_fwd_bf16_algo(x, w, bias, y, stride, pad, groups, relu, algo, stream)
    if algo == ALGO_AUTO:
        return conv2d_fwd(x, w, bias, y, stride, pad, groups, relu, stream)
    return conv2d_fwd_algo(x, w, bias, y, stride, pad, groups, relu, algo, stream)


def dwconv2d(x, w, bias=None, stride=1, pad=1, relu=False, stream=None):
    N, C, H, W = x.shape
    P, Q = out_dims(H, W, w.shape[2], w.shape[3], stride, pad)
    y = torch.empty((N, C, P, Q), device=x.device, dtype=torch.float32)
    return dwconv2d_fwd(x, w, bias, y, stride, pad, relu, stream)
