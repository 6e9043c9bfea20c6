"""GPU: bf16 channel-last layers (conv2d_fwd_cl, maxpool2d_nhwc_bf16, stack
layers with a layout) against the oracle.

A layer of a channel-last network reads x as bf16 [N][H][W][C] and writes y
(and reads the residual) as bf16 [N][P][Q][K]: the oracle's reading is the
fp64 sum rounded to fp32, then to bf16 (oracle.conv2d_bf16_cl).  On small
integers every fp32 sum is exact, so both sides round the same value and
must agree bit for bit, for every kernel instantiation (1x1 and 3x3
direct-to-LDS tiles, the halo kernel, strided 1x1 and 3x3, split reductions
with their channel-last reduce, groups, ragged tiles, the one-stage 1x1
tiles, the 7x7 stem).
"""
import numpy as np
import pytest
import torch

from paper_1907_02154_amd import miconv
from paper_1907_02154_amd import workloads as wl

pytestmark = pytest.mark.gpu

XY = miconv.LAYOUT_X_NHWC | miconv.LAYOUT_Y_NHWC_BF16
X = miconv.LAYOUT_X_NHWC
Y = miconv.LAYOUT_Y_NHWC_BF16


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    miconv.lib()


def bf(bits):
    """bf16 bit patterns (numpy uint16) -> a bf16 device tensor of that shape."""
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)


def bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def nhwc(a):
    return np.ascontiguousarray(np.transpose(a, (0, 2, 3, 1)))


# (N, C, H, W, K, R, S, stride, pad, groups, layout, kernel the call must use)
CL_CASES = [
    (4, 64, 28, 28, 256, 1, 1, 1, 0, 1, XY, "igemm_bf16_dma_cl_kernel<1, 1, 64, 64, 2, 2, 3, 0, 64>"),
    (16, 64, 28, 28, 256, 1, 1, 1, 0, 1, XY, "igemm_bf16_dma_cl_kernel<1, 1, 128, 64, 2, 2, 1, 0, 64>"),   # one stage
    (17, 128, 28, 28, 256, 1, 1, 1, 0, 1, XY, "igemm_bf16_dma_cl_kernel<1, 1, 128, 64, 2, 2, 1, 0, 64>"),  # 2 chunks, ragged M
    (42, 64, 28, 28, 64, 1, 1, 1, 0, 1, XY, "igemm_bf16_dma_cl_kernel<1, 1, 64, 64, 2, 2, 1, 0, 64>"),     # one stage, 64 x 64
    (32, 64, 56, 56, 256, 1, 1, 1, 0, 1, XY, "igemm_bf16_dma_cl_kernel<1, 1, 128, 64, 2, 2, 1, 0, 64>"),   # 3136 tiles
    (128, 64, 28, 28, 64, 1, 1, 1, 0, 1, XY, "igemm_bf16_dma_cl_kernel<1, 1, 64, 64, 2, 2, 1, 0, 64>"),    # 1568 tiles
    (16, 128, 28, 28, 256, 1, 1, 1, 0, 2, XY, "igemm_bf16_dma_cl_kernel<1, 1, 128, 64, 2, 2, 1, 0, 64>"),  # two groups
    (64, 256, 28, 28, 200, 1, 1, 2, 0, 1, XY, "igemm_bf16_dma_cl_kernel<1, 1, 128, 64, 2, 2, 1, 0, 64>"),  # stride 2, ragged K
    (32, 64, 30, 30, 136, 1, 1, 1, 0, 1, XY, "igemm_bf16_dma_cl_kernel<1, 1, 128, 64, 2, 2, 1, 0, 64>"),   # K = 136: a partial filter tile
    (16, 256, 28, 28, 128, 1, 1, 1, 0, 1, XY, "igemm_bf16_dma_cl_kernel<1, 1, 64, 64, 2, 2, 3, 0, 64>"),
    (64, 512, 28, 28, 256, 1, 1, 1, 0, 1, XY, "igemm_bf16_dma_cl_kernel<1, 1, 128, 128, 2, 2, 2, 0, 64>"),
    (4, 256, 28, 28, 64, 1, 1, 1, 0, 1, XY, "igemm_bf16_dma_cl_kernel<1, 1, "),
    (8, 256, 28, 28, 128, 1, 1, 2, 0, 1, XY, "igemm_bf16_dma_cl_kernel<1, 1, "),                # stride 2
    (3, 64, 9, 11, 72, 1, 1, 1, 0, 1, XY, "igemm_bf16_dma_cl_kernel<1, 1, "),                   # ragged M, K
    (64, 128, 28, 28, 128, 3, 3, 1, 1, 1, XY, "igemm_bf16_halo_cl_kernel<128, 128, 2, 2, 192, 2>"),
    (21, 64, 56, 56, 64, 3, 3, 1, 1, 1, XY, "igemm_bf16_halo_cl_kernel<128, 64, 2, 2, 256, 1>"),
    (32, 64, 14, 14, 128, 3, 3, 1, 1, 1, XY, "igemm_bf16_dma_cl_kernel<3, 3, "),
    (4, 64, 15, 15, 128, 3, 3, 2, 1, 1, XY, "igemm_bf16_dma_cl_kernel<3, 3, "),                 # 3x3 stride 2
    (1, 512, 7, 7, 512, 3, 3, 1, 1, 1, XY, "splitk_reduce_cl_kernel"),                          # split
    (2, 2048, 7, 7, 512, 1, 1, 1, 0, 1, XY, "splitk_reduce_cl_kernel"),                         # 1x1 split
    (4, 128, 14, 14, 128, 3, 3, 1, 1, 2, XY, "_cl_kernel<"),                                    # two groups
    (4, 64, 28, 28, 256, 1, 1, 1, 0, 1, X, "igemm_bf16_dma_kernel<1, 1, 64, 64, 2, 2, 3, 0, 64>"),
    (64, 128, 28, 28, 128, 3, 3, 1, 1, 1, X, "igemm_bf16_halo_kernel<128, 128, 2, 2, 192, 2>"),
    (2, 3, 224, 224, 64, 7, 7, 2, 3, 1, Y, "stem7_bf16_kernel"),
]


def _ids(c):
    return "x".join(map(str, c[:10])) + f"-L{c[10]}"


def _case_data(case, seed):
    N, C, H, W, K, R, S, st, pad, g, layout = case[:11]
    x = wl.to_bf16_bits(wl.small_ints((N, C, H, W), -4, 4, seed))          # NCHW bits
    w = wl.to_bf16_bits(wl.small_ints((K, C // g, R, S), -4, 4, seed + 1))
    b = wl.small_ints((K,), -8, 8, seed + 2)
    P, Q = miconv.out_dims(H, W, R, S, st, pad)
    res = wl.to_bf16_bits(wl.small_ints((N, P, Q, K), -60, 60, seed + 3))  # NHWC bits
    return x, w, b, res, P, Q


def _oracle(oracle_lib, case, x, w, b, res, relu):
    """Expected output in the call's own layout: bf16 bits [N][P][Q][K], or
    fp32 [N][K][P][Q] for an fp32 NCHW y."""
    st, pad, g, layout = case[7], case[8], case[9], case[10]
    if layout & Y:
        return oracle_lib.conv2d_bf16_cl(nhwc(x), w, b, st, pad, g, relu, res)
    return oracle_lib.conv2d_bf16(x, w, b, st, pad, g, relu)


@pytest.mark.parametrize("case", CL_CASES, ids=_ids)
def test_channel_last_small_int_bitwise(oracle_lib, case):
    N, C, H, W, K, R, S, st, pad, g, layout, kernel = case
    x, w, b, res, P, Q = _case_data(case, 8100 + sum(case[:10]))
    tx = bf(nhwc(x)) if layout & X else bf(x)
    tw, tb = bf(w), dev(b)
    s = None
    for relu, with_res in ((True, False), (False, False), (True, True), (False, True)):
        if with_res and not layout & Y or (with_res and R == 7):
            continue
        ref = _oracle(oracle_lib, case, x, w, b, res if with_res else None, relu)
        if layout & Y:
            y = torch.full((N, P, Q, K), float("nan"), device="cuda", dtype=torch.bfloat16)
        else:
            y = torch.full((N, K, P, Q), float("nan"), device="cuda")
        miconv.conv2d_fwd_cl(tx, tw, tb, y, st, pad, g, relu, res=bf(res) if with_res else None,
                             layout=layout)
        torch.cuda.synchronize()
        got = bits(y) if layout & Y else y.cpu().numpy()
        np.testing.assert_array_equal(got, ref, err_msg=f"relu={relu} res={with_res}")
        if s is None:
            # the same layer in a stack: names the kernel, packs filters once
            s = miconv.Stack([(miconv.OP_CONV_BF16, tx, tw, tb, y, st, pad, g, relu, None, layout)])
            assert kernel in s.describe(0), s.describe(0)
            y.fill_(float("nan"))
            s.launch()
            torch.cuda.synchronize()
            got = bits(y) if layout & Y else y.cpu().numpy()
            np.testing.assert_array_equal(got, ref, err_msg="stack")
            s.close()
    if layout & Y and R != 7:
        # in place: the residual is the output buffer itself
        y = bf(res)
        miconv.conv2d_fwd_cl(tx, tw, tb, y, st, pad, g, True, res=y, layout=layout)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(bits(y), _oracle(oracle_lib, case, x, w, b, res, True), err_msg="in place")


def test_channel_last_maxpool_bitwise(oracle_lib):
    """ResNet's stem pool (3x3, stride 2, pad 1), a 2x2/2 pool, and 3x3 pools
    on odd planes (windows cut by the padding on every side) on bf16
    channel-last data: every output is the oracle's maximum, bit for bit."""
    for (N, C, H, W, R, st, pad) in ((4, 64, 112, 112, 3, 2, 1), (2, 32, 15, 17, 2, 2, 0), (1, 8, 7, 9, 3, 1, 1),
                                     (3, 24, 13, 11, 3, 2, 1)):
        xb = wl.to_bf16_bits(wl.normal((N, H, W, C), 1.0, 8300 + C))
        P, Q = miconv.out_dims(H, W, R, R, st, pad)
        y = torch.empty((N, P, Q, C), device="cuda", dtype=torch.bfloat16)
        miconv.maxpool2d_nhwc_bf16(bf(xb), y, R, R, st, pad)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(bits(y), oracle_lib.maxpool2d_bf16_cl(xb, R, R, st, pad))


def test_channel_last_rejections():
    x = torch.zeros((2, 8, 8, 48), device="cuda", dtype=torch.bfloat16)     # C/groups % 64 != 0
    w = torch.zeros((64, 48, 3, 3), device="cuda", dtype=torch.bfloat16)
    y = torch.zeros((2, 8, 8, 64), device="cuda", dtype=torch.bfloat16)
    with pytest.raises(miconv.MiconvError) as e:
        miconv.conv2d_fwd_cl(x, w, None, y, 1, 1, layout=XY)
    assert e.value.status == miconv.ERR_UNSUPPORTED
    x = torch.zeros((2, 8, 8, 64), device="cuda", dtype=torch.bfloat16)
    w = torch.zeros((36, 64, 1, 1), device="cuda", dtype=torch.bfloat16)    # K % 8 != 0
    y = torch.zeros((2, 8, 8, 36), device="cuda", dtype=torch.bfloat16)
    with pytest.raises(miconv.MiconvError) as e:
        miconv.conv2d_fwd_cl(x, w, None, y, 1, 0, layout=XY)
    assert e.value.status == miconv.ERR_UNSUPPORTED
    # x NCHW with a channel-last y: only the 7x7 stem
    x = torch.zeros((2, 64, 8, 8), device="cuda", dtype=torch.bfloat16)
    w = torch.zeros((64, 64, 1, 1), device="cuda", dtype=torch.bfloat16)
    y = torch.zeros((2, 8, 8, 64), device="cuda", dtype=torch.bfloat16)
    with pytest.raises(miconv.MiconvError) as e:
        miconv.conv2d_fwd_cl(x, w, None, y, 1, 0, layout=Y)
    assert e.value.status == miconv.ERR_UNSUPPORTED
