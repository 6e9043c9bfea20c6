"""GPU: the residual join fused into the conv epilogue, y = act(conv + bias + res).

ResNet's bottleneck blocks add the shortcut before their last ReLU; the
library joins it in the conv's own epilogue (operator fusion, paper
Sec. 3.2.3) instead of a separate add kernel.  Small-integer data keep every
sum exact, so each kernel family's epilogue (and the split-K reduction that
finishes a split layer) must reproduce the oracle bit for bit, in place
(res = y) and out of place, with the join before the activation.
"""
import numpy as np
import pytest
import torch

from paper_1907_02154_amd import miconv
from paper_1907_02154_amd import workloads as wl

pytestmark = pytest.mark.gpu

A, D, I = miconv.ALGO_AUTO, miconv.ALGO_DIRECT, miconv.ALGO_IGEMM


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    miconv.lib()


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def dev_bf16_bits(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)


# (N, C, H, W, K, R, S, stride, pad, groups, dtype, algo, kernel conv2d_fwd_ws must use)
RES_CASES = [
    (1, 64, 56, 56, 64, 3, 3, 1, 1, 1, "f32", A, "igemm_wave_f32_kcrs_kernel<3, 3, 8, 1, 0, false, 1>"),
    (2, 64, 15, 13, 130, 1, 1, 1, 0, 1, "f32", A, "igemm_wave_f32_kcrs_kernel<1, 1, 8, 1, 1, false, 1>"),
    (1, 512, 8, 8, 96, 3, 3, 1, 1, 1, "f32", A, "splitk_reduce_kernel"),        # 16-byte reduce
    (1, 1024, 7, 7, 40, 3, 3, 1, 1, 1, "f32", A, "splitk_reduce_kernel"),       # scalar reduce
    (8, 3, 224, 224, 64, 3, 3, 1, 1, 1, "f32", A, "igemm_wave_f32_kcrs_kernel<3, 3, 4, 2, 2, true, 2>"),
    (1, 3, 45, 47, 40, 7, 7, 2, 3, 1, "f32", A, "igemm_wave_f32_kcrs_kernel<7, 7, 8, 1, 2, false, 2>"),
    (2, 64, 15, 13, 130, 1, 1, 1, 0, 1, "f32", I, "igemm_f32_kernel<1, 1, 32, 64, 1, 2, 64>"),
    (1, 12, 9, 9, 18, 3, 3, 1, 1, 3, "f32", A, "conv_direct_kernel<float>"),
    # named without the residual; with it the two-stage tile runs (test_residual_plan_keeps_two_stage_tile)
    (4, 64, 56, 56, 256, 1, 1, 1, 0, 1, "bf16", A, "igemm_bf16_dma_kernel<1, 1, 128, 64, 2, 2, 1, 1, 64>"),
    (64, 64, 14, 14, 256, 1, 1, 1, 0, 1, "bf16", A, "igemm_bf16_dma_kernel<1, 1, 128, 64, 2, 2, 3, 2, 64>"),
    (8, 64, 28, 28, 128, 1, 1, 2, 0, 1, "bf16", A, "igemm_bf16_dma_kernel<1, 1, 64, 64, 2, 2, 3, 0, 64>"),
    (32, 64, 14, 14, 128, 3, 3, 1, 1, 1, "bf16", A, "igemm_bf16_dma_kernel<3, 3, 64, 64, 2, 2, 3, 0, 64>"),
    (21, 64, 56, 56, 64, 3, 3, 1, 1, 1, "bf16", A, "igemm_bf16_halo_kernel<128, 64, 2, 2, 256, 1>"),
    (64, 128, 28, 28, 128, 3, 3, 1, 1, 1, "bf16", A, "igemm_bf16_halo_kernel<128, 128, 2, 2, 192, 2>"),
    (1, 512, 7, 7, 512, 3, 3, 1, 1, 1, "bf16", A, "splitk_reduce_kernel"),
    (64, 96, 14, 14, 96, 3, 3, 1, 1, 1, "bf16", A, "igemm_bf16_nhwc_kernel<3, 3, 64, 64, 32>"),
    (2, 64, 15, 13, 130, 1, 1, 1, 0, 1, "bf16", I, "igemm_bf16_kernel<1, 1, 64, 64, 64, false, true, false>"),
    (1, 40, 19, 19, 70, 3, 3, 1, 1, 1, "bf16", A, "splitk_reduce_kernel"),
    (1, 3, 224, 224, 64, 7, 7, 2, 3, 1, "bf16", A, "stem7_bf16_kernel"),
    (1, 12, 9, 9, 18, 3, 3, 1, 1, 3, "bf16", D, "conv_direct_kernel<unsigned short>"),
    (4, 384, 56, 56, 200, 1, 1, 1, 0, 1, "bf16", A, "igemm_bf16_dma_kernel<1, 1, 128, 64, 2, 2, 2, 1, 64>"),   # six chunks: pipelined
]


def _inputs(case, seed):
    N, C, H, W, K, R, S, st, pad, g, dt = case[:11]
    x = wl.small_ints((N, C, H, W), -4, 4, seed)
    w = wl.small_ints((K, C // g, R, S), -4, 4, seed + 1)
    b = wl.small_ints((K,), -8, 8, seed + 2)
    P, Q = miconv.out_dims(H, W, R, S, st, pad)
    res = wl.small_ints((N, K, P, Q), -60, 60, seed + 3)
    if dt == "bf16":
        x, w = wl.to_bf16_bits(x), wl.to_bf16_bits(w)
        tx, tw = dev_bf16_bits(x), dev_bf16_bits(w)
    else:
        tx, tw = dev(x), dev(w)
    return x, w, b, res, tx, tw


def _oracle(oracle_lib, case, x, w, b, res, relu):
    st, pad, g, dt = case[7], case[8], case[9], case[10]
    f = oracle_lib.conv2d_bf16 if dt == "bf16" else oracle_lib.conv2d
    return f(x, w, b, st, pad, g, relu, res=res)


def _join(tx, tw, tb, res, y, st, pad, g, relu, algo, mode):
    if mode == "ws":
        miconv.conv2d_fwd_ws(tx, tw, tb, y, st, pad, g, relu, res=res, algo=algo)
    elif mode == "stack":   # a one-layer stack: filters packed at create
        op = miconv.OP_CONV_BF16 if tx.dtype == torch.bfloat16 else miconv.OP_CONV_F32
        s = miconv.Stack([(op, tx, tw, tb, y, st, pad, g, relu, res)])
        s.launch()
        torch.cuda.synchronize()
        s.close()
    else:
        miconv.conv2d_fwd_res(tx, tw, tb, res, y, st, pad, g, relu, algo=algo)


@pytest.mark.parametrize("case", RES_CASES, ids=lambda c: "x".join(map(str, c[:10])) + "-" + c[10])
@pytest.mark.parametrize("mode", ["ws", "plain", "stack"])
def test_residual_join_small_int_bitwise(oracle_lib, case, mode):
    """conv2d_fwd_ws (the kernel named in the case), conv2d_fwd_res (the
    plan without a workspace) and a one-layer stack (packed filters) with the
    join in the epilogue."""
    N, C, H, W, K, R, S, st, pad, g, dt, algo, kernel = case
    name = miconv.conv2d_describe(N, C, H, W, K, R, S, st, pad, g, dt, algo, mode=mode)[0]
    if mode == "ws":
        assert kernel in name, name
    x, w, b, res, tx, tw = _inputs(case, 6000 + sum(case[:10]))
    tres = dev(res)
    for relu in (True, False):
        ref = _oracle(oracle_lib, case, x, w, b, res, relu)
        y = torch.full(res.shape, float("nan"), device="cuda")
        _join(tx, tw, dev(b), tres, y, st, pad, g, relu, algo, mode)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(y.cpu().numpy(), ref, err_msg=f"{name} relu={relu}")
    # in place: the residual is the output buffer itself
    y = tres.clone()
    _join(tx, tw, dev(b), y, y, st, pad, g, True, algo, mode)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(y.cpu().numpy(), _oracle(oracle_lib, case, x, w, b, res, True),
                                  err_msg=f"{name} in place")
    # no residual: the plain operator
    y = torch.empty(res.shape, device="cuda")
    _join(tx, tw, dev(b), None, y, st, pad, g, True, algo, mode)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(y.cpu().numpy(), _oracle(oracle_lib, case, x, w, b, np.zeros_like(res), True))


def test_residual_plan_keeps_two_stage_tile():
    """A 1x1 layer reading NCHW x with few reduction chunks takes the
    one-stage tile alone, but with a residual the planner keeps the two-stage
    one: the one-stage kernel's residual epilogue leaves room for two
    work-groups per CU only."""
    x = torch.zeros((4, 64, 56, 56), dtype=torch.bfloat16, device="cuda")
    w = torch.zeros((256, 64, 1, 1), dtype=torch.bfloat16, device="cuda")
    y = torch.zeros((4, 256, 56, 56), device="cuda")
    res = torch.zeros_like(y)
    names = []
    for r in (None, res):
        s = miconv.Stack([(miconv.OP_CONV_BF16, x, w, None, y, 1, 0, 1, True, r)])
        names.append(s.describe(0))
        s.close()
    assert names[0] == "igemm_bf16_dma_kernel<1, 1, 128, 64, 2, 2, 1, 1, 64>", names[0]
    assert names[1] == "igemm_bf16_dma_res_kernel<1, 1, 128, 64, 2, 2, 2, 1, 64>", names[1]


@pytest.mark.parametrize("case", [c for c in RES_CASES if c[-1] in (
    "igemm_wave_f32_kcrs_kernel<1, 1, 8, 1, 1, false, 1>", "splitk_reduce_kernel",
    "igemm_bf16_dma_kernel<1, 1, 128, 64, 2, 2, 1, 1, 64>")][:4],
    ids=lambda c: "x".join(map(str, c[:10])) + "-" + c[10])
def test_residual_offset_pointers(oracle_lib, case):
    """y and res one float past a 16-byte boundary (same offset): the kernels
    take their element-by-element epilogue paths and write nothing outside y."""
    N, C, H, W, K, R, S, st, pad, g, dt, algo, kernel = case
    x, w, b, res, tx, tw = _inputs(case, 6500 + sum(case[:10]))
    n = res.size
    yb = torch.full((n + 8,), float("nan"), device="cuda")
    rb = torch.zeros(n + 8, device="cuda")
    y = yb[1:1 + n].view(res.shape)
    r = rb[1:1 + n].view(res.shape)
    r.copy_(dev(res))
    assert y.data_ptr() % 16 == 4 and r.data_ptr() % 16 == 4
    miconv.conv2d_fwd_ws(tx, tw, dev(b), y, st, pad, g, True, res=r, algo=algo)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(y.cpu().numpy(), _oracle(oracle_lib, case, x, w, b, res, True))
    assert torch.isnan(yb[0]) and torch.isnan(yb[1 + n:]).all()


def test_residual_rejections():
    x = torch.zeros((1, 8, 6, 6), device="cuda")
    w = torch.zeros((8, 8, 3, 3), device="cuda")
    y = torch.zeros((1, 8, 6, 6), device="cuda")
    rb = torch.zeros(8 * 36 + 4, device="cuda")
    with pytest.raises(miconv.MiconvError) as e:      # res at another offset modulo 16 bytes
        miconv.conv2d_fwd_res(x, w, None, rb[1:1 + 288].view(1, 8, 6, 6), y, 1, 1)
    assert e.value.status == miconv.ERR_ALIGN
    with pytest.raises(miconv.MiconvError) as e:      # depthwise
        miconv.conv2d_fwd_res(x, torch.zeros((8, 1, 3, 3), device="cuda"), None, y, y, 1, 1, groups=8)
    assert e.value.status == miconv.ERR_UNSUPPORTED
    with pytest.raises(ValueError):
        miconv.conv2d_fwd_res(x, w, None, torch.zeros((1, 8, 5, 5), device="cuda"), y, 1, 1)


def test_residual_random_bf16_bottleneck_join(oracle_lib):
    """The join layer of a ResNet-50 stage-3 block at batch 64 (1x1, 128 -> 512
    channels on 28 x 28) with random data: within the bf16 gate on two
    sampled images, computed by the oracle exactly."""
    N, C, H, W, K = 64, 128, 28, 28, 512
    rng_x = wl.uniform01((N, C, H, W), 7100)
    w = wl.normal((K, C, 1, 1), np.sqrt(2.0 / C), 7101)
    b = wl.normal((K,), 0.01, 7102)
    res = wl.normal((N, K, H, W), 1.0, 7103)
    xb, wb = wl.to_bf16_bits(rng_x), wl.to_bf16_bits(w)
    y = torch.empty((N, K, H, W), device="cuda")
    miconv.conv2d_fwd_res(dev_bf16_bits(xb), dev_bf16_bits(wb), dev(b), dev(res), y, 1, 0, 1, True)
    torch.cuda.synchronize()
    got = y.cpu().numpy()
    for i in (0, N - 1):
        ref = oracle_lib.conv2d_bf16(xb[i:i + 1], wb, b, 1, 0, 1, True, res=res[i:i + 1])
        e = np.max(np.abs(got[i:i + 1] - ref)) / np.max(np.abs(ref))
        assert e <= 2e-2, (i, e)


def test_stack_layers_with_residual(oracle_lib):
    """A stack whose layers carry residuals (one of them in place) gives, on
    eager passes and on every graph replay, the oracle's exact results."""
    picks = [RES_CASES[1], RES_CASES[2], RES_CASES[9], RES_CASES[12]]
    ops, want, inplace = [], [], []
    for j, case in enumerate(picks):
        N, C, H, W, K, R, S, st, pad, g, dt, algo, kernel = case
        x, w, b, res, tx, tw = _inputs(case, 6800 + j)
        op = miconv.OP_CONV_BF16 if dt == "bf16" else miconv.OP_CONV_F32
        y = torch.empty(res.shape, device="cuda")
        r = y if j == 1 else dev(res)
        ops.append((op, tx, tw, dev(b), y, st, pad, g, True, r))
        inplace.append((y, res) if j == 1 else None)
        want.append(_oracle(oracle_lib, case, x, w, b, res, True))
    s = miconv.Stack(ops)
    # layers with a residual and no reduction split run the epilogue-join kernels
    assert "igemm_bf16_dma_res_kernel<1, 1, 128, 64, 2, 2, 3, 2, 64>" in s.describe(2), s.describe(2)
    assert "igemm_bf16_halo_res_kernel<128, 64, 2, 2, 256, 1>" in s.describe(3), s.describe(3)

    def reset():
        for o, ip in zip(ops, inplace):
            if ip is None:
                o[4].fill_(float("nan"))
            else:
                ip[0].copy_(dev(ip[1]))

    reset()
    s.launch()
    torch.cuda.synchronize()
    for o, ref in zip(ops, want):
        np.testing.assert_array_equal(o[4].cpu().numpy(), ref)
    s.capture(1, timed=False)
    for rep in range(3):
        reset()
        torch.cuda.synchronize()
        s.replay()
        torch.cuda.synchronize()
        for i, (o, ref) in enumerate(zip(ops, want)):
            np.testing.assert_array_equal(o[4].cpu().numpy(), ref, err_msg=f"replay {rep} layer {i}")
    s.close()


@pytest.mark.parametrize("case", RES_CASES, ids=lambda c: "x".join(map(str, c[:10])) + "-" + c[10])
def test_output_image_stride(oracle_lib, case):
    """y (and res) as a channel range of a wider NCHW tensor at batch >= 2
    (conv2d_fwd_ex): every kernel writes image n at n * stride, joins the
    residual read with the same strides, and leaves the other channels alone."""
    N, C, H, W, K, R, S, st, pad, g, dt, algo, kernel = case
    case2 = (max(N, 2),) + case[1:]
    x, w, b, res, tx, tw = _inputs(case2, 7300 + sum(case[:10]))
    n2, _, P, Q = res.shape
    for off, extra, mode in ((4, 8, "ws"), (3, 5, "ws"), (4, 8, "plain")):   # y 16-byte aligned or not
        big = torch.full((n2, K + extra, P, Q), float("nan"), device="cuda")
        rbig = torch.zeros((n2, K + extra, P, Q), device="cuda")
        y, r = big[:, off:off + K], rbig[:, off:off + K]
        r.copy_(dev(res))
        if mode == "ws":
            miconv.conv2d_fwd_ws(tx, tw, dev(b), y, st, pad, g, True, res=r, algo=algo)
        else:
            miconv.conv2d_fwd_ex(tx, tw, dev(b), y, st, pad, g, True, res=r, algo=algo)
        torch.cuda.synchronize()
        name = miconv.conv2d_describe(n2, C, H, W, K, R, S, st, pad, g, dt, algo, mode=mode)[0]
        np.testing.assert_array_equal(y.cpu().numpy(), _oracle(oracle_lib, case2, x, w, b, res, True),
                                      err_msg=f"{name} offset {off}")
        assert torch.isnan(big[:, :off]).all() and torch.isnan(big[:, off + K:]).all()


VEC_Y_CASES = [c for c in RES_CASES if c[-1] in (
    "igemm_bf16_dma_kernel<1, 1, 128, 64, 2, 2, 1, 1, 64>",
    "igemm_bf16_dma_kernel<1, 1, 128, 64, 2, 2, 2, 1, 64>",
    "igemm_bf16_halo_kernel<128, 64, 2, 2, 256, 1>",
    "igemm_bf16_halo_kernel<128, 128, 2, 2, 192, 2>",
    "igemm_wave_f32_kcrs_kernel<3, 3, 8, 1, 0, false, 1>")]


@pytest.mark.parametrize("case", VEC_Y_CASES, ids=lambda c: "x".join(map(str, c[:10])) + "-" + c[10])
def test_output_stride_misaligned_vector_planes(oracle_lib, case):
    """y and res as channel ranges of a wider tensor whose base sits one float
    past a 16-byte boundary, on planes (P*Q % 4 == 0) where the epilogues
    would otherwise store 16 bytes at a time: the strided, misaligned rows
    take the element-wise path, exactly, and the guard channels stay NaN."""
    N, C, H, W, K, R, S, st, pad, g, dt, algo, kernel = case
    case2 = (max(N, 2),) + case[1:]
    x, w, b, res, tx, tw = _inputs(case2, 7600 + sum(case[:10]))
    n2, _, P, Q = res.shape
    assert (P * Q) % 4 == 0
    extra = 6
    flat = torch.full((n2 * (K + extra) * P * Q + 1,), float("nan"), device="cuda")
    rflat = torch.zeros_like(flat)
    big = flat[1:].view(n2, K + extra, P, Q)
    rbig = rflat[1:].view(n2, K + extra, P, Q)
    y, r = big[:, 2:2 + K], rbig[:, 2:2 + K]
    assert y.data_ptr() % 16 != 0 and (y.data_ptr() - r.data_ptr()) % 16 == 0
    r.copy_(dev(res))
    miconv.conv2d_fwd_ws(tx, tw, dev(b), y, st, pad, g, True, res=r, algo=algo)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(y.cpu().numpy(), _oracle(oracle_lib, case2, x, w, b, res, True))
    assert torch.isnan(big[:, :2]).all() and torch.isnan(big[:, 2 + K:]).all() and torch.isnan(flat[0])
