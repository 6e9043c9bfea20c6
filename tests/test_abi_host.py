"""Host-side checks of the C-ABI library (no GPU needed).

The library must load, export every function ``include/miconv.h`` declares,
and reject invalid arguments before any HIP call (so these run on a machine
without a GPU).  The fake pointers below are never dereferenced: every call
here fails validation first.
"""
import ctypes

import pytest

from paper_1907_02154_amd import miconv

FAKE = 4096   # aligned, non-null, never touched


@pytest.fixture(scope="module")
def L():
    return miconv.lib()


def test_exports_every_declared_symbol(L):
    names = miconv.header_functions()
    for expected in ("conv2d_fwd", "conv2d_fwd_bf16", "dwconv2d_fwd", "conv2d_fwd_algo",
                     "miconv_out_dims", "maxpool2d_fwd", "add_act_fwd", "cast_f32_to_bf16",
                     "miconv_strerror", "miconv_last_hip_error", "miconv_version"):
        assert expected in names
    for n in names:
        assert hasattr(L, n), n


def test_out_dims(L):
    assert miconv.out_dims(224, 224, 7, 7, 2, 3) == (112, 112)
    assert miconv.out_dims(112, 112, 3, 3, 2, 1) == (56, 56)
    assert miconv.out_dims(14, 14, 1, 1, 2, 0) == (7, 7)
    assert miconv.out_dims(5, 6, 3, 2, 2, 0) == (2, 3)
    P, Q = ctypes.c_int(), ctypes.c_int()
    assert L.miconv_out_dims(2, 2, 3, 3, 1, 0, ctypes.byref(P), ctypes.byref(Q)) == miconv.ERR_SHAPE
    assert L.miconv_out_dims(2, 2, 3, 3, 0, 0, ctypes.byref(P), ctypes.byref(Q)) == miconv.ERR_SHAPE
    assert L.miconv_out_dims(2, 2, 3, 3, 1, 0, None, None) == miconv.ERR_NULL


def _call(L, fn, N=1, C=4, H=8, W=8, K=4, R=3, S=3, stride=1, pad=1, groups=1,
          x=FAKE, w=FAKE, b=None, y=FAKE):
    return getattr(L, fn)(N, C, H, W, K, R, S, stride, pad, groups, x, w, b, y, 0, None)


@pytest.mark.parametrize("fn", ["conv2d_fwd", "conv2d_fwd_bf16", "dwconv2d_fwd"])
def test_validation_errors(L, fn):
    assert _call(L, fn, x=None) == miconv.ERR_NULL
    assert _call(L, fn, w=None) == miconv.ERR_NULL
    assert _call(L, fn, y=None) == miconv.ERR_NULL
    for bad in (dict(N=0), dict(C=-1), dict(H=0), dict(W=0), dict(K=0), dict(R=0), dict(S=0),
                dict(stride=0), dict(pad=-1), dict(H=2, W=2, pad=0)):
        assert _call(L, fn, **bad) == miconv.ERR_SHAPE, bad
    assert _call(L, fn, groups=3) == miconv.ERR_GROUPS
    assert _call(L, fn, groups=0) == miconv.ERR_GROUPS
    assert _call(L, fn, N=70000, C=1024, H=64, W=64, K=4, groups=1) == miconv.ERR_TOO_LARGE
    assert _call(L, fn, x=FAKE + 1) == miconv.ERR_ALIGN
    assert _call(L, fn, y=FAKE + 2) == miconv.ERR_ALIGN


def test_depthwise_specific_errors(L):
    assert _call(L, "dwconv2d_fwd", groups=1) == miconv.ERR_GROUPS
    assert _call(L, "dwconv2d_fwd", C=4, K=8, groups=4) == miconv.ERR_GROUPS
    assert _call(L, "dwconv2d_fwd", C=4, K=4, groups=4, R=9, S=9, pad=4) == miconv.ERR_UNSUPPORTED


def test_algo_and_glue_errors(L):
    assert L.conv2d_fwd_algo(1, 4, 8, 8, 4, 3, 3, 1, 1, 1, FAKE, FAKE, None, FAKE, 0, 7, None) == \
        miconv.ERR_UNSUPPORTED
    assert L.maxpool2d_fwd(1, 1, 4, 4, 2, 2, 2, 2, FAKE, FAKE, None) == miconv.ERR_SHAPE   # pad >= R
    assert L.maxpool2d_fwd(1, 1, 4, 4, 2, 2, 2, 0, None, FAKE, None) == miconv.ERR_NULL
    assert L.add_act_fwd(-1, FAKE, FAKE, FAKE, 1, None) == miconv.ERR_SHAPE
    assert L.add_act_fwd(4, None, FAKE, FAKE, 1, None) == miconv.ERR_NULL
    assert L.cast_f32_to_bf16(4, FAKE, FAKE + 1, None) == miconv.ERR_ALIGN


def test_strerror_and_version(L):
    for s in range(0, -8, -1):
        assert miconv.strerror(s)
    assert miconv.strerror(-99) == "unknown status"
    assert L.miconv_version() >= 100
    assert L.miconv_last_hip_error() == 0


def test_packed_weight_sizes(L):
    """Packed filter sizes follow the layout of the kernel each shape takes:
    wave order (fp32: [groups][K/32][Kred/8][64 lanes][4]), KRSC (bf16 3x3),
    tap pairs (bf16 7x7 stem: [K][28][8]); 0 when the kernel reads w as given."""
    f = L.conv2d_packed_weight_bytes
    assert f(1, 64, 56, 56, 64, 3, 3, 1, 1, 1, 0) == 2 * 72 * 256 * 4          # fp32 wave, Kred 576
    assert f(1, 64, 56, 56, 256, 1, 1, 1, 0, 1, 0) == 8 * 8 * 256 * 4          # fp32 wave, Kred 64
    assert f(64, 64, 56, 56, 64, 3, 3, 1, 1, 1, 1) == 64 * 64 * 9 * 2          # bf16 KRSC
    assert f(64, 3, 224, 224, 64, 7, 7, 2, 3, 1, 1) == 64 * 28 * 8 * 2         # bf16 stem
    assert f(64, 256, 56, 56, 64, 1, 1, 1, 0, 1, 1) == 0                       # bf16 1x1: w as given
    assert f(1, 32, 56, 56, 32, 3, 3, 1, 1, 32, 0) == 0                        # depthwise
    assert f(1, 64, 56, 56, 64, 3, 3, 1, 1, 1, 2) == miconv.ERR_UNSUPPORTED    # no such dtype
    assert f(0, 64, 56, 56, 64, 3, 3, 1, 1, 1, 0) == miconv.ERR_SHAPE
    assert f(1, 64, 56, 56, 64, 3, 3, 1, 1, 3, 0) == miconv.ERR_GROUPS


def test_packed_entry_points_validate_first(L):
    shape = (1, 64, 56, 56, 64, 3, 3, 1, 1, 1, 0)
    assert L.conv2d_pack_weights(*shape, None, FAKE, None) == miconv.ERR_NULL
    assert L.conv2d_pack_weights(*shape, FAKE, None, None) == miconv.ERR_NULL
    assert L.conv2d_pack_weights(*shape[:-1], 5, FAKE, FAKE, None) == miconv.ERR_UNSUPPORTED
    assert L.conv2d_fwd_packed(*shape, None, FAKE, None, FAKE, 0, None) == miconv.ERR_NULL
    assert L.conv2d_fwd_packed(*shape, FAKE, None, None, FAKE, 0, None) == miconv.ERR_NULL
    assert L.conv2d_fwd_packed(*shape[:-1], 7, FAKE, FAKE, None, FAKE, 0, None) == miconv.ERR_UNSUPPORTED
    assert L.conv2d_fwd_packed(1, 64, 56, 56, 64, 3, 3, 0, 1, 1, 0, FAKE, FAKE, None, FAKE, 0,
                               None) == miconv.ERR_SHAPE


def test_residual_entry_point_validates_first(L):
    """conv2d_fwd_res checks dtype, pointers, the residual's alignment and the
    operator kind before anything is launched (no GPU needed)."""
    shape = (1, 64, 56, 56, 64, 3, 3, 1, 1, 1)
    A = miconv.ALGO_AUTO
    assert L.conv2d_fwd_res(*shape, 2, A, FAKE, FAKE, None, FAKE, FAKE, 0, None) == miconv.ERR_UNSUPPORTED
    assert L.conv2d_fwd_res(*shape, 0, A, None, FAKE, None, FAKE, FAKE, 0, None) == miconv.ERR_NULL
    assert L.conv2d_fwd_res(*shape, 1, A, FAKE, FAKE, None, FAKE, None, 0, None) == miconv.ERR_NULL
    assert L.conv2d_fwd_res(*shape, 0, 9, FAKE, FAKE, None, FAKE, FAKE, 0, None) == miconv.ERR_UNSUPPORTED
    for off in (2, 4, 8, 12):   # not at y's offset modulo 16 bytes
        assert L.conv2d_fwd_res(*shape, 0, A, FAKE, FAKE, None, FAKE + off, FAKE, 0,
                                None) == miconv.ERR_ALIGN, off
    dw = (1, 32, 28, 28, 32, 3, 3, 1, 1, 32)
    assert L.conv2d_fwd_res(*dw, 0, A, FAKE, FAKE, None, FAKE, FAKE, 0, None) == miconv.ERR_UNSUPPORTED


def test_output_stride_validation(L):
    """conv2d_fwd_ex: the image stride of y must keep images apart, fit 32-bit
    offsets, and is refused for depthwise shapes; checked before any launch."""
    shape = (2, 64, 56, 56, 64, 3, 3, 1, 1, 1)
    A = miconv.ALGO_AUTO
    dense = 64 * 56 * 56
    assert L.conv2d_fwd_ex(*shape, 0, A, FAKE, FAKE, None, None, FAKE, dense - 1, 0, None) == miconv.ERR_SHAPE
    assert L.conv2d_fwd_ex(*shape, 0, A, FAKE, FAKE, None, None, FAKE, 1 << 31, 0, None) == miconv.ERR_TOO_LARGE
    dw = (2, 32, 28, 28, 32, 3, 3, 1, 1, 32)
    assert L.conv2d_fwd_ex(*dw, 0, A, FAKE, FAKE, None, None, FAKE, 64 * 28 * 28, 0, None) == miconv.ERR_UNSUPPORTED
    assert L.conv2d_fwd_ex(*shape, 3, A, FAKE, FAKE, None, None, FAKE, 0, 0, None) == miconv.ERR_UNSUPPORTED
