"""GPU parity: the HIP kernels behind the C ABI against the CPU oracle.

* Small-integer data (|x|, |w| <= 4, |bias| <= 8) keep every partial sum
  exact in fp32, so any summation order must reproduce the oracle bit for
  bit: this checks indexing, padding, strides, groups, tiling edges and the
  split-K reduction of every kernel independently of rounding.
* Random data at the layer shapes of the five evaluation configurations are
  held to the gate e = max|y - y_ref| / max|y_ref| <= 1e-4 (fp32 path) and
  <= 2e-2 (bf16 inputs, fp32 accumulation), with the GPU running the full
  batch in the same launch configuration the bench times.  Where the oracle
  would take minutes (VGG-16 at batch 8, ResNet-50 at batch 64) it is run on
  a sample that it computes exactly: a few images and a subset of output
  channels (each output channel depends only on its own filter and each
  image only on itself).
"""
import numpy as np
import pytest
import torch

from paper_1907_02154_amd import miconv
from paper_1907_02154_amd import workloads as wl

pytestmark = pytest.mark.gpu

TOL_F32 = 1e-4
TOL_BF16 = 2e-2


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    miconv.lib()   # fails loudly if the library is missing


def dev(a, dtype=torch.float32):
    return torch.from_numpy(np.ascontiguousarray(a)).to(device="cuda", dtype=dtype)


def dev_bf16_bits(bits):
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda()
    return t.view(torch.bfloat16)


def gpu_conv(x, w, b, stride, pad, groups, relu, algo, mode="ws"):
    y = miconv.conv2d(dev(x), dev(w), None if b is None else dev(b), stride, pad, groups, relu,
                      algo=algo, mode=mode)
    torch.cuda.synchronize()
    return y.cpu().numpy()


def err_inf(y, ref):
    d = np.max(np.abs(y.astype(np.float64) - ref.astype(np.float64)))
    s = np.max(np.abs(ref.astype(np.float64)))
    return d / s if s > 0 else d


def ints(shape, lo, hi, seed):
    return wl.small_ints(shape, lo, hi, seed)


# (N, C, H, W, K, R, S, stride, pad, groups): several tiles and ragged tails
DENSE_CASES = [
    (1, 1, 1, 1, 1, 1, 1, 1, 0, 1),
    (1, 3, 5, 7, 2, 3, 3, 1, 1, 1),
    (2, 3, 17, 19, 70, 7, 7, 2, 3, 1),       # stem-like, ragged M and K
    (1, 40, 19, 19, 70, 3, 3, 1, 1, 1),      # Kred 360, several chunks
    (2, 64, 15, 13, 130, 1, 1, 1, 0, 1),     # 1x1, ragged tiles
    (1, 96, 14, 14, 200, 1, 1, 2, 0, 1),     # 1x1 stride 2
    (1, 512, 7, 7, 96, 3, 3, 1, 1, 1),       # small M, long reduction -> split-K
    (3, 33, 9, 11, 65, 3, 3, 2, 1, 1),
    (1, 16, 10, 10, 24, 3, 5, 1, 2, 1),      # R != S, generic path
    (1, 12, 9, 9, 18, 3, 3, 1, 1, 3),        # grouped
    (2, 32, 8, 8, 64, 3, 3, 1, 1, 2),        # grouped with Cg >= 8
    (1, 8, 6, 6, 4, 3, 3, 1, 4, 1),          # padding wider than the filter
    (1, 130, 130, 1, 3, 1, 1, 1, 0, 1),      # W = 1
    (1, 1024, 7, 7, 40, 3, 3, 1, 1, 1),      # Kred 9216: wave split + work-group split
    (2, 250, 9, 9, 33, 1, 1, 1, 0, 1),       # Kred not a multiple of 4
    (1, 64, 60, 60, 64, 3, 3, 1, 1, 1),      # M >= 2048: two pixel blocks per tile
    (1, 3, 45, 47, 40, 7, 7, 2, 3, 1),       # C <= 4 stem: reduction over (r, s, 4 channels), odd R*S
    (2, 2, 19, 17, 33, 3, 3, 2, 1, 1),       # two channels padded to four
    (1, 4, 13, 13, 20, 5, 5, 1, 2, 1),       # four channels, generic 5x5
    (1, 8, 12, 10, 64, 3, 2, 1, 1, 2),       # C/groups = 4 in each of two groups, R != S
    (4, 512, 7, 7, 64, 3, 3, 1, 1, 1),       # split over four images: the reduction's pixel quads span images
]


@pytest.mark.parametrize("case", DENSE_CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("algo", [miconv.ALGO_DIRECT, miconv.ALGO_IGEMM, miconv.ALGO_WAVE,
                                  miconv.ALGO_AUTO])
@pytest.mark.parametrize("mode", ["ws", "plain"])
def test_dense_small_int_bitwise(oracle_lib, case, algo, mode):
    """Every fp32 algorithm through conv2d_fwd_ws (split reductions allowed)
    and through the plain entry point (no workspace: filters read as given,
    no split)."""
    N, C, H, W, K, R, S, st, pad, g = case
    seed = 1000 + sum(case)
    x = ints((N, C, H, W), -4, 4, seed)
    w = ints((K, C // g, R, S), -4, 4, seed + 1)
    b = ints((K,), -8, 8, seed + 2)
    for relu in (False, True):
        ref = oracle_lib.conv2d(x, w, b, st, pad, g, relu)
        y = gpu_conv(x, w, b, st, pad, g, relu, algo, mode)
        np.testing.assert_array_equal(y, ref, err_msg=f"{case} relu={relu} algo={algo}")
    y = gpu_conv(x, w, None, st, pad, g, False, algo, mode)
    np.testing.assert_array_equal(y, oracle_lib.conv2d(x, w, None, st, pad, g, False))


DW_CASES = [  # (N, C, H, W, R, stride, pad)
    (1, 32, 112, 112, 3, 1, 1), (1, 64, 112, 112, 3, 2, 1), (2, 128, 28, 28, 3, 2, 1),
    (2, 5, 14, 14, 3, 1, 1), (1, 7, 7, 7, 3, 1, 1), (1, 3, 14, 14, 3, 2, 1),
    (1, 4, 130, 130, 3, 1, 1),          # row wider than one lane group: several segments
    (1, 4, 9, 13, 3, 1, 1), (2, 3, 11, 10, 3, 2, 1),   # odd sizes
    (1, 6, 12, 12, 5, 3, 2), (1, 2, 8, 8, 7, 1, 3), (1, 3, 6, 6, 1, 1, 0), (1, 2, 5, 5, 3, 1, 0),
    # whole-plane run kernel: every plane size and stride it is built for, with
    # a partial last run (and, for 7x7, runs that end inside a 16-byte vector)
    (3, 37, 7, 7, 3, 1, 1), (2, 41, 7, 7, 3, 2, 1), (5, 61, 14, 14, 3, 1, 1),
    (3, 53, 14, 14, 3, 2, 1), (2, 23, 28, 28, 3, 1, 1), (1, 19, 28, 28, 3, 2, 1),
    (1, 9, 56, 56, 3, 1, 1), (1, 7, 56, 56, 3, 2, 1),
    # ... and with more runs than work-groups, so work-groups loop over runs
    (133, 1024, 7, 7, 3, 1, 1), (37, 1024, 14, 14, 3, 1, 1), (10, 1000, 28, 28, 3, 2, 1),
    (9, 250, 56, 56, 3, 1, 1),
    # 112x112 band kernel (enough bands to fill the grid; a few work-groups take two)
    (4, 130, 112, 112, 3, 1, 1), (2, 260, 112, 112, 3, 2, 1),
]


@pytest.mark.parametrize("case", DW_CASES, ids=lambda c: "x".join(map(str, c)))
def test_depthwise_small_int_bitwise(oracle_lib, case):
    N, C, H, W, R, st, pad = case
    seed = 2000 + sum(case)
    x = ints((N, C, H, W), -4, 4, seed)
    w = ints((C, 1, R, R), -4, 4, seed + 1)
    b = ints((C,), -8, 8, seed + 2)
    for relu in (False, True):
        ref = oracle_lib.dwconv2d(x, w, b, st, pad, relu)
        y = miconv.dwconv2d(dev(x), dev(w), dev(b), st, pad, relu)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(y.cpu().numpy(), ref, err_msg=f"{case} relu={relu}")
        # conv2d_fwd with groups == C == K reaches the same kernel
        y2 = gpu_conv(x, w, b, st, pad, C, relu, miconv.ALGO_AUTO)
        np.testing.assert_array_equal(y2, ref)


BF16_CASES = DENSE_CASES[:9] + [
    (2, 64, 15, 15, 70, 3, 3, 2, 1, 1),      # channel-last path, 3x3 stride 2, ragged tiles
    (1, 64, 9, 9, 48, 3, 3, 1, 1, 2),        # channel-last path, grouped (C/groups = 32)
    (3, 96, 13, 11, 130, 1, 1, 1, 0, 1),     # channel-last 1x1, chunk of 32 channels
    (1, 256, 7, 7, 520, 3, 3, 1, 1, 1),      # long reduction: split across work-groups
    (2, 64, 14, 14, 128, 1, 1, 2, 0, 1),     # 1x1 stride 2: only the sampled pixels are copied (whole-plane copy)
    (3, 64, 7, 9, 72, 1, 1, 2, 0, 1),        # sampled whole-plane copy, odd plane, P x Q = 4 x 5
    (1, 128, 28, 28, 64, 1, 1, 3, 0, 1),     # sampled copy, stride 3, scalar reads
    (2, 96, 10, 10, 64, 1, 1, 2, 0, 1),      # sampled whole-plane copy, a 32-channel block
    (2, 64, 9, 9, 64, 1, 1, 2, 1, 1),        # 1x1 stride 2 with padding: full (whole-plane) copy
    (5, 64, 7, 7, 64, 1, 1, 1, 0, 1),        # 49-pixel planes (whole-plane copy)
    (3, 64, 14, 14, 96, 3, 3, 1, 1, 1),      # 196-pixel planes: 4-pixel copy reads
    (2, 64, 15, 17, 64, 3, 3, 1, 1, 1),      # 255-pixel planes: the largest whole-plane copy
    (2, 64, 17, 16, 64, 3, 3, 1, 1, 1),      # 272-pixel planes: 8-pixel copy reads
    (3, 160, 7, 7, 64, 1, 1, 1, 0, 1),       # whole-plane copy with a last block of 32 channels
    (2, 64, 15, 17, 64, 1, 1, 2, 0, 1),      # sampled whole-plane copy, 255-pixel planes, P x Q = 8 x 9
    (10, 256, 62, 62, 16, 1, 1, 1, 0, 1),    # large copy: 256-pixel tiles, 4-pixel reads
    (32, 256, 63, 63, 16, 1, 1, 2, 0, 1),    # large sampled copy: 256-pixel tiles
    (24, 256, 45, 45, 16, 1, 1, 1, 0, 1),    # large copy of odd planes: 256-pixel tiles, scalar reads
    (2, 64, 21, 23, 64, 3, 3, 1, 1, 1),      # 483-pixel planes: whole-plane copy in 32-channel blocks
    (3, 96, 56, 56, 40, 1, 1, 2, 0, 1),      # stride-2 copy, 4 sampled pixels per 16-byte load, ragged channels
    (2, 64, 28, 28, 72, 1, 1, 2, 0, 1),      # stride-2 copy, 2 sampled pixels per 8-byte load (Q = 14)
    (2, 64, 20, 36, 64, 1, 1, 2, 0, 1),      # 10 x 18 sampled rows: 8-byte loads
    (2, 64, 30, 30, 64, 1, 1, 2, 0, 1),      # odd Q = 15: sampled copy reads pixel by pixel
    (4, 512, 7, 7, 256, 3, 3, 1, 1, 1),      # split over four images: the reduction's pixel quads span images
]


@pytest.mark.parametrize("case", BF16_CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("algo", [miconv.ALGO_AUTO, miconv.ALGO_IGEMM, miconv.ALGO_DIRECT])
@pytest.mark.parametrize("mode", ["ws", "plain"])
def test_bf16_small_int_bitwise(oracle_lib, case, algo, mode):
    N, C, H, W, K, R, S, st, pad, g = case
    seed = 3000 + sum(case)
    x = wl.to_bf16_bits(ints((N, C, H, W), -4, 4, seed))
    w = wl.to_bf16_bits(ints((K, C // g, R, S), -4, 4, seed + 1))
    b = ints((K,), -8, 8, seed + 2)
    ref = oracle_lib.conv2d_bf16(x, w, b, st, pad, g, True)
    y = miconv.conv2d(dev_bf16_bits(x), dev_bf16_bits(w), dev(b), st, pad, g, True, algo=algo, mode=mode)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(y.cpu().numpy(), ref)


OFFSET_CASES = [  # (N, C, H, W, K, R, S, stride, pad, groups) run on x and y at odd element offsets
    (2, 64, 7, 7, 64, 1, 1, 1, 0, 1),
    (2, 64, 14, 14, 96, 3, 3, 1, 1, 1),
    (2, 64, 14, 14, 64, 1, 1, 2, 0, 1),
    (1, 64, 16, 16, 128, 1, 1, 1, 0, 1),
    (2, 64, 28, 28, 64, 1, 1, 2, 0, 1),      # stride-2 copy: the grouped loads need an aligned x
]


def _offset_bf16(bits, shape):
    """A bf16 device tensor holding `bits` one element past a 16-byte boundary."""
    buf = torch.empty(bits.size + 8, dtype=torch.int16, device="cuda")
    buf[1:1 + bits.size] = torch.from_numpy(bits.reshape(-1).view(np.int16)).cuda()
    t = buf[1:1 + bits.size].view(torch.bfloat16).view(shape)
    assert t.data_ptr() % 16 == 2
    return t


@pytest.mark.parametrize("case", OFFSET_CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("which", ["xy", "w"])
@pytest.mark.parametrize("mode", ["ws", "plain"])
def test_bf16_offset_pointers_small_int_bitwise(oracle_lib, case, which, mode):
    """x one bf16 element and y one float past a 16-byte boundary: the
    channel-last copy falls back to reads that need no alignment, the 1x1
    layer that would read x in NCHW takes the copy, and the epilogue stores
    element by element.  w one element past a 16-byte boundary: a 1x1 layer,
    whose kernels read w as given with 16-byte loads, takes the gather kernel
    instead.  Results stay exact on small integers, nothing is written
    outside y."""
    N, C, H, W, K, R, S, st, pad, g = case
    seed = 3900 + sum(case)
    x = wl.to_bf16_bits(ints((N, C, H, W), -4, 4, seed))
    w = wl.to_bf16_bits(ints((K, C // g, R, S), -4, 4, seed + 1))
    b = ints((K,), -8, 8, seed + 2)
    ref = oracle_lib.conv2d_bf16(x, w, b, st, pad, g, True)
    tx = _offset_bf16(x, (N, C, H, W)) if which == "xy" else dev_bf16_bits(x)
    tw = _offset_bf16(w, w.shape) if which == "w" else dev_bf16_bits(w)
    P, Q = miconv.out_dims(H, W, R, S, st, pad)
    o = 1 if which == "xy" else 0
    yb = torch.full((N * K * P * Q + 4,), float("nan"), device="cuda")
    ty = yb[o:o + N * K * P * Q].view(N, K, P, Q)
    if mode == "ws":
        miconv.conv2d_fwd_ws(tx, tw, dev(b), ty, st, pad, g, True)
    else:
        miconv.conv2d_fwd_bf16(tx, tw, dev(b), ty, st, pad, g, True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(ty.cpu().numpy(), ref, err_msg=str(case))
    assert torch.isnan(yb[:o]).all() and torch.isnan(yb[o + N * K * P * Q:]).all()   # nothing outside y


HALO_CASES = [  # (N, C, H, W, K, groups): bf16 3x3 stride-1 layers that take the halo-patch kernel
    (64, 128, 28, 28, 128, 1),   # ResNet-50 s3 at batch 64: two channel blocks
    (63, 128, 27, 29, 128, 1),   # odd plane: tiles and patches cross rows and images, ragged last tile
    (64, 192, 28, 28, 128, 1),   # three channel blocks
    (42, 256, 28, 28, 256, 2),   # two groups of 128 channels
    (1, 512, 7, 7, 512, 1),      # reduction split across work-groups
    (1, 256, 9, 31, 130, 1),     # widest plane (a 192-row patch), ragged filter tile, split
    (21, 64, 56, 56, 64, 1),     # one 64-channel block: 128 x 64 tiles, one 242-row patch
    (12, 128, 55, 53, 128, 2),   # two groups of 64 channels, odd 55 x 53 planes
]


@pytest.mark.parametrize("case", HALO_CASES, ids=lambda c: "x".join(map(str, c)))
def test_bf16_halo_small_int_bitwise(oracle_lib, case):
    """bf16 3x3 layers whose pixel operand is staged once per 64-channel block
    for all nine taps (padding taps zeroed after the read) against the
    oracle on small integers, bias and ReLU included."""
    N, C, H, W, K, g = case
    name = miconv.conv2d_describe(N, C, H, W, K, 3, 3, 1, 1, g, "bf16")[0]
    assert "igemm_bf16_halo_kernel" in name, name
    seed = 3800 + sum(case)
    x = wl.to_bf16_bits(ints((N, C, H, W), -4, 4, seed))
    w = wl.to_bf16_bits(ints((K, C // g, 3, 3), -4, 4, seed + 1))
    b = ints((K,), -8, 8, seed + 2)
    ref = oracle_lib.conv2d_bf16(x, w, b, 1, 1, g, True)
    y = miconv.conv2d(dev_bf16_bits(x), dev_bf16_bits(w), dev(b), 1, 1, g, True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(y.cpu().numpy(), ref, err_msg=str(case))


NCHW_1X1_CASES = [  # (N, C, H, W, K, groups, loads): 1x1 stride-1 layers whose pixel operand comes from NCHW x
    (3, 64, 56, 56, 520, 1, 1),     # image boundaries inside pixel tiles, ragged M and K (one-stage 128 x 64 tiles)
    (4, 64, 56, 56, 512, 1, 1),     # one-stage tiles
    (2, 192, 64, 64, 256, 1, 1),    # three reduction chunks, one stage
    (8, 128, 64, 64, 256, 2, 1),    # two groups of 64 channels
    (8, 384, 56, 56, 256, 1, 1),    # six chunks: pipelined 128 x 128 tiles
    (4, 384, 56, 56, 200, 1, 1),    # six chunks: pipelined 128 x 64 tiles, ragged K
    (64, 64, 14, 14, 256, 1, 2),    # 196-pixel planes: 8-pixel groups straddle images, 4-byte loads
    (64, 256, 14, 14, 1024, 1, 2),  # ResNet-50 s4 expansion layer, 128 x 128 tiles
    (200, 64, 10, 13, 256, 1, 2),   # 130-pixel planes, ragged last tile
    (64, 128, 14, 14, 256, 2, 2),   # two groups, 4-byte loads (three LDS stages)
    (340, 64, 14, 14, 64, 1, 2),    # 128 x 64 tiles, two LDS stages
]


@pytest.mark.parametrize("case", NCHW_1X1_CASES, ids=lambda c: "x".join(map(str, c)))
def test_bf16_1x1_nchw_operand_small_int_bitwise(oracle_lib, case):
    """bf16 1x1 layers that skip the channel-last copy (pixel operand read from
    NCHW x through LDS transpose reads; 16-byte loads of 8 pixels, or 4-byte
    loads of 2 pixels when 8-pixel groups can straddle images) against the
    oracle on small integers."""
    N, C, H, W, K, g, mode = case
    name = miconv.conv2d_describe(N, C, H, W, K, 1, 1, 1, 0, g, "bf16")[0]
    assert "nchw_to_nhwc" not in name and name.endswith(f", {mode}, 64>"), name
    seed = 3700 + sum(case)
    x = wl.to_bf16_bits(ints((N, C, H, W), -4, 4, seed))
    w = wl.to_bf16_bits(ints((K, C // g, 1, 1), -4, 4, seed + 1))
    b = ints((K,), -8, 8, seed + 2)
    ref = oracle_lib.conv2d_bf16(x, w, b, 1, 0, g, True)
    y = miconv.conv2d(dev_bf16_bits(x), dev_bf16_bits(w), dev(b), 1, 0, g, True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(y.cpu().numpy(), ref, err_msg=str(case))


STEM_CASES = [  # (N, C, H, W, K): 7x7 stride-2 pad-3 stems with 112 output columns
    (2, 3, 224, 224, 64),     # ResNet's stem
    (1, 1, 224, 224, 32),     # one channel, half a filter tile
    (1, 4, 223, 223, 96),     # odd width (scalar row loads), two filter tiles, the second partial
]


@pytest.mark.parametrize("case", STEM_CASES, ids=lambda c: "x".join(map(str, c)))
def test_bf16_stem_small_int_bitwise(oracle_lib, case):
    """The dedicated bf16 stem kernel (tap-pair reduction order, packed
    filters per call) against the oracle on small integers, with and without
    ReLU and bias."""
    N, C, H, W, K = case
    assert miconv.conv2d_describe(N, C, H, W, K, 7, 7, 2, 3, 1, "bf16")[0].endswith("stem7_bf16_kernel")
    seed = 3500 + sum(case)
    x = wl.to_bf16_bits(ints((N, C, H, W), -4, 4, seed))
    w = wl.to_bf16_bits(ints((K, C, 7, 7), -4, 4, seed + 1))
    b = ints((K,), -8, 8, seed + 2)
    for relu, bias in ((True, b), (False, None)):
        ref = oracle_lib.conv2d_bf16(x, w, bias, 2, 3, 1, relu)
        y = miconv.conv2d(dev_bf16_bits(x), dev_bf16_bits(w), None if bias is None else dev(bias), 2, 3, 1,
                          relu)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(y.cpu().numpy(), ref, err_msg=f"{case} relu={relu}")


def _layers(config):
    """Unique layer shapes of a config with the index of their first use."""
    seen, out = set(), []
    for i, l in enumerate(wl.workload(config).layers):
        key = (l.N, l.C, l.H, l.W, l.K, l.R, l.S, l.stride, l.pad, l.groups, l.relu)
        if key not in seen:
            seen.add(key)
            out.append((i, l))
    return out


def _layer_ids(config):
    return [f"c{config}-{i}-{l.name}" for i, l in _layers(config)]


def _check_layer(oracle_lib, config, i, l, images=None, kmax=None, tol=TOL_F32):
    x, w, b = wl.layer_tensors(config, i, l)
    bf16 = wl.workload(config).dtype == "bf16"
    if bf16:
        xb, wb = wl.to_bf16_bits(x), wl.to_bf16_bits(w)
        y = miconv.conv2d(dev_bf16_bits(xb), dev_bf16_bits(wb), dev(b), l.stride, l.pad, l.groups, l.relu)
    elif l.kind == "dw":
        y = miconv.dwconv2d(dev(x), dev(w), dev(b), l.stride, l.pad, l.relu)
    else:
        y = miconv.conv2d(dev(x), dev(w), dev(b), l.stride, l.pad, l.groups, l.relu)
    torch.cuda.synchronize()
    y = y.cpu().numpy()
    imgs = list(range(l.N)) if images is None else images
    if kmax is None or l.groups != 1 or kmax >= l.K:
        ks = np.arange(l.K)
    else:   # first, last and evenly spread output channels
        ks = np.unique(np.concatenate([np.linspace(0, l.K - 1, kmax).astype(int), [0, l.K - 1]]))
    for n in imgs:
        if bf16:
            ref = oracle_lib.conv2d_bf16(xb[n:n + 1], wb[ks], b[ks], l.stride, l.pad, l.groups, l.relu)
        elif l.kind == "dw":
            ref = oracle_lib.dwconv2d(x[n:n + 1], w, b, l.stride, l.pad, l.relu)
        else:
            ref = oracle_lib.conv2d(x[n:n + 1], w[ks], b[ks], l.stride, l.pad, l.groups, l.relu)
        got = y[n:n + 1, ks] if l.kind != "dw" else y[n:n + 1]
        e = err_inf(got, ref)
        assert e <= tol, f"config {config} layer {i} {l.name} image {n}: e={e:.3e}"
    return y


@pytest.mark.parametrize("config", [1, 2, 3, 6])
def test_configs_full_oracle(oracle_lib, config):
    """Configs 1-3 (batch 1, fp32): every layer against the whole oracle output."""
    for i, l in _layers(config):
        print(f"config {config} layer {i} {l.name}", flush=True)
        _check_layer(oracle_lib, config, i, l)


def test_config4_vgg_sampled(oracle_lib):
    """VGG-16 at batch 8: images 0 and 7, 24 output channels per layer."""
    for i, l in _layers(4):
        print(f"config 4 layer {i} {l.name}", flush=True)
        _check_layer(oracle_lib, 4, i, l, images=[0, l.N - 1], kmax=24)


def test_config5_resnet_bf16_sampled(oracle_lib):
    """ResNet-50 at batch 64 with bf16 x and w: images 0 and 63, 24 channels."""
    for i, l in _layers(5):
        print(f"config 5 layer {i} {l.name}", flush=True)
        _check_layer(oracle_lib, 5, i, l, images=[0, l.N - 1], kmax=24, tol=TOL_BF16)


def _stack_layer(config, i, l):
    """One layer through a one-layer stack (filters packed at create, a
    workspace of its own): the kernels the bench's layer-by-layer passes run.
    Returns (kernel names, y on the host, the oracle's x, w, bias)."""
    x, w, b = wl.layer_tensors(config, i, l)
    bf16 = wl.workload(config).dtype == "bf16"
    if bf16:
        x, w = wl.to_bf16_bits(x), wl.to_bf16_bits(w)
        tx, tw, op = dev_bf16_bits(x), dev_bf16_bits(w), miconv.OP_CONV_BF16
    else:
        tx, tw, op = dev(x), dev(w), miconv.OP_CONV_F32
    P, Q = miconv.out_dims(l.H, l.W, l.R, l.S, l.stride, l.pad)
    y = torch.full((l.N, l.K, P, Q), float("nan"), device="cuda")
    st = miconv.Stack([(op, tx, tw, dev(b), y, l.stride, l.pad, l.groups, l.relu)])
    name = st.describe(0)
    st.launch()
    torch.cuda.synchronize()
    st.close()
    return name, y.cpu().numpy(), x, w, b


def test_config5_stack_whole_layer_per_kernel(oracle_lib):
    """ResNet-50 at batch 64, bf16 x and w, as the bench's layer-by-layer stack
    runs it: for every distinct kernel sequence the stack picks, its first
    layer checked on the whole output (all 64 images, every channel) against
    the oracle, e <= 2e-2."""
    picked = {}
    for i, l in _layers(5):
        N, C, H, W, K, R, S = l.N, l.C, l.H, l.W, l.K, l.R, l.S
        name = miconv.conv2d_describe(N, C, H, W, K, R, S, l.stride, l.pad, l.groups, "bf16", mode="stack")[0]
        picked.setdefault(name, (i, l))
    assert len(picked) >= 8, sorted(picked)
    for name, (i, l) in picked.items():
        print(f"config 5 layer {i} {l.name}: {name}", flush=True)
        got_name, y, x, w, b = _stack_layer(5, i, l)
        assert got_name == name, (got_name, name)
        ref = oracle_lib.conv2d_bf16(x, w, b, l.stride, l.pad, l.groups, l.relu)
        e = err_inf(y, ref)
        assert e <= TOL_BF16, f"layer {i} {l.name} ({name}): e={e:.3e}"


def test_config4_vgg_batch32_stack_sampled(oracle_lib):
    """VGG-16 at batch 32 (the bench's --batch 32 run) through one-layer
    stacks: images 0, 13 and 31, 24 output channels per layer, e <= 1e-4."""
    for i, l in _layers(4):
        l = l.with_batch(32)
        name, y, x, w, b = _stack_layer(4, i, l)
        print(f"config 4 b32 layer {i} {l.name}: {name}", flush=True)
        ks = np.unique(np.linspace(0, l.K - 1, 24).astype(int))
        for n in (0, 13, 31):
            ref = oracle_lib.conv2d(x[n:n + 1], w[ks], b[ks], l.stride, l.pad, l.groups, l.relu)
            e = err_inf(y[n:n + 1, ks], ref)
            assert e <= TOL_F32, f"layer {i} {l.name} image {n}: e={e:.3e}"


ERROR_BOUND_CASES = [  # (config, layer index): layers on seeded random data
    (1, 0),     # 64 -> 64 3x3 at 56x56, batch 1
    (2, 0),     # ResNet-50 stem, 7x7 over 3 channels
    (2, 51),    # ResNet-50 s5 3x3: reduction of 4608 split across work-groups
    (3, 26),    # MobileNet's last pointwise layer, split
    (4, 0),     # VGG-16's first layer at batch 8, one tile per wavefront
    (5, 16),    # ResNet-50 s3 3x3 at batch 64, bf16 (halo-patch kernel)
    (5, 30),    # ResNet-50 s4 expansion at batch 64, bf16 (4-byte NCHW loads)
]


@pytest.mark.parametrize("config,idx", ERROR_BOUND_CASES, ids=lambda v: str(v))
def test_elementwise_error_bound(oracle_lib, config, idx):
    """Every output element within the a priori bound of recursive summation:
    |y - y_ref| <= (gamma_n + u) * (sum |w x| + |b|), n = C/groups*R*S + 1,
    gamma_n = n u / (1 - n u), with u = 2^-23 (twice fp32's unit roundoff:
    room for accumulators that round toward zero), sum |w x| + |b| computed by
    the oracle on |x|, |w|, |b|, and u |ref| covering the oracle's own final
    rounding.  Rounding the inputs or products to bf16 inside an fp32 layer
    would break it by orders of magnitude.  ReLU is 1-Lipschitz, so it keeps
    the bound."""
    l = wl.workload(config).layers[idx]
    x, w, b = wl.layer_tensors(config, idx, l)
    bf16 = wl.workload(config).dtype == "bf16"
    if bf16:
        x, w = wl.to_bf16_bits(x), wl.to_bf16_bits(w)
        y = miconv.conv2d(dev_bf16_bits(x), dev_bf16_bits(w), dev(b), l.stride, l.pad, l.groups, l.relu)
        ref = oracle_lib.conv2d_bf16(x, w, b, l.stride, l.pad, l.groups, l.relu)
        # |x|, |w| in bf16: the sign bit cleared
        mag = oracle_lib.conv2d_bf16(x & 0x7FFF, w & 0x7FFF, np.abs(b), l.stride, l.pad, l.groups, False)
    else:
        y = miconv.conv2d(dev(x), dev(w), dev(b), l.stride, l.pad, l.groups, l.relu)
        ref = oracle_lib.conv2d(x, w, b, l.stride, l.pad, l.groups, l.relu)
        mag = oracle_lib.conv2d(np.abs(x), np.abs(w), np.abs(b), l.stride, l.pad, l.groups, False)
    torch.cuda.synchronize()
    mag = mag.astype(np.float64) * (1 + 2.0 ** -23)   # the oracle rounds it to fp32 once
    n = (l.C // l.groups) * l.R * l.S + 1
    u = 2.0 ** -23
    gamma = n * u / (1 - n * u)
    err = np.abs(y.cpu().numpy().astype(np.float64) - ref.astype(np.float64))
    bound = (gamma + u) * mag
    worst = np.max(err - bound)
    assert worst <= 0, f"config {config} layer {idx} {l.name}: max excess {worst:.3e}"
    # typical error sits far below the worst case (about sqrt(n) u)
    assert np.median(err / np.maximum(mag, 1e-30)) < 8 * np.sqrt(n) * 2.0 ** -24


def test_dense_deterministic():
    l = wl.workload(2).layers[-2]      # s5 3x3: small M, split-K
    x, w, b = wl.layer_tensors(2, 51, l)
    X, Wt, B = dev(x), dev(w), dev(b)
    y1 = miconv.conv2d(X, Wt, B, l.stride, l.pad, 1, l.relu)
    y2 = miconv.conv2d(X, Wt, B, l.stride, l.pad, 1, l.relu)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)


IND_CASES = [  # (N, C, H, W, K, stride): C <= 4 3x3 layers with one tile per wavefront
    (3, 3, 224, 224, 64, 1),     # VGG-16's first layer at batch 3
    (3, 3, 223, 221, 40, 1),     # ragged pixel and filter tiles
    (12, 3, 224, 224, 64, 2),    # stride 2 (MobileNet's stem at batch 12)
    (3, 2, 224, 224, 64, 1),     # two channels, padded to four
]


@pytest.mark.parametrize("case", IND_CASES, ids=lambda c: "x".join(map(str, c)))
def test_wave_independent_tiles_small_int_bitwise(oracle_lib, case):
    """Short reductions over many tiles run one tile per wavefront, the
    epilogue stored straight from the accumulators: exact against the oracle
    on small integers."""
    N, C, H, W, K, st = case
    name = miconv.conv2d_describe(N, C, H, W, K, 3, 3, st, 1, 1, "f32", mode="stack")[0]
    assert name.endswith("igemm_wave_f32_kernel<3, 3, 4, 2, 2, true>"), name
    name = miconv.conv2d_describe(N, C, H, W, K, 3, 3, st, 1, 1, "f32", mode="plain")[0]
    assert name.endswith("igemm_wave_f32_kcrs_kernel<3, 3, 4, 2, 2, true, 2>"), name
    seed = 4800 + sum(case)
    x = ints((N, C, H, W), -4, 4, seed)
    w = ints((K, C, 3, 3), -4, 4, seed + 1)
    b = ints((K,), -8, 8, seed + 2)
    P, Q = miconv.out_dims(H, W, 3, 3, st, 1)
    for relu, bias in ((True, b), (False, None)):
        ref = oracle_lib.conv2d(x, w, bias, st, 1, 1, relu)
        np.testing.assert_array_equal(gpu_conv(x, w, bias, st, 1, 1, relu, miconv.ALGO_AUTO, "plain"), ref,
                                      err_msg=f"{case} relu={relu}")
        # packed filters (a one-layer stack)
        y = torch.full((N, K, P, Q), float("nan"), device="cuda")
        s = miconv.Stack([(miconv.OP_CONV_F32, dev(x), dev(w), None if bias is None else dev(bias), y,
                           st, 1, 1, relu)])
        s.launch()
        torch.cuda.synchronize()
        s.close()
        np.testing.assert_array_equal(y.cpu().numpy(), ref, err_msg=f"{case} relu={relu} stack")


PACKED_CASES = [  # (N, C, H, W, K, R, S, stride, pad, groups, dtype): filters packed once
    (1, 64, 20, 20, 48, 3, 3, 1, 1, 1, 0),     # fp32 wave kernel, (r, s, c) order
    (2, 32, 15, 15, 40, 1, 1, 2, 0, 1, 0),     # fp32 1x1 stride 2
    (1, 32, 10, 10, 48, 3, 3, 1, 1, 2, 0),     # fp32 grouped
    (1, 3, 40, 40, 32, 7, 7, 2, 3, 1, 0),      # fp32 stem, (r, s, c4) order
    (1, 512, 7, 7, 512, 3, 3, 1, 1, 1, 0),     # fp32 split reduction
    (2, 64, 14, 14, 64, 3, 3, 1, 1, 1, 1),     # bf16 channel-last, KRSC
    (1, 3, 224, 224, 64, 7, 7, 2, 3, 1, 1),    # bf16 stem, tap pairs
    (2, 64, 16, 16, 128, 1, 1, 1, 0, 1, 1),    # bf16 1x1: w read as given (0 packed bytes)
    (1, 32, 12, 12, 32, 3, 3, 1, 1, 32, 0),    # depthwise: w read as given
]


@pytest.mark.parametrize("case", PACKED_CASES, ids=lambda c: "x".join(map(str, c)))
def test_packed_filters_match_plain_calls(oracle_lib, case):
    """conv2d_pack_weights + conv2d_fwd_packed (filters packed once, no
    workspace): bitwise the output of the workspace entry point, exact against
    the oracle on small integers, for two calls on one packing."""
    N, C, H, W, K, R, S, st, pad, g, dtype = case
    seed = 4600 + sum(case)
    x = ints((N, C, H, W), -4, 4, seed)
    w = ints((K, C // g, R, S), -4, 4, seed + 1)
    b = ints((K,), -8, 8, seed + 2)
    if dtype:
        x, w = wl.to_bf16_bits(x), wl.to_bf16_bits(w)
        tx, tw = dev_bf16_bits(x), dev_bf16_bits(w)
        ref = oracle_lib.conv2d_bf16(x, w, b, st, pad, g, True)
    else:
        tx, tw = dev(x), dev(w)
        ref = oracle_lib.conv2d(x, w, b, st, pad, g, True)
    plain = miconv.conv2d(tx, tw, dev(b), st, pad, g, True)
    pk = miconv.PackedFilters(tw, (N, C, H, W), st, pad, g)
    assert (pk.nbytes == 0) == ((R == 1 and dtype == 1) or g == C), pk.nbytes
    for _ in range(2):
        y = torch.full_like(plain, float("nan"))
        pk.forward(tx, dev(b), y, relu=True)
        torch.cuda.synchronize()
        assert torch.equal(y, plain)
    np.testing.assert_array_equal(y.cpu().numpy(), ref)


def test_packed_filters_reject_a_kernel_change():
    """The bf16 stem kernel needs y at a 16-byte boundary; with y one float
    off, the layer would take a kernel that reads w unpacked, so the call on
    stem-packed filters fails instead of reading them wrongly."""
    N, C, H, W, K = 1, 3, 224, 224, 64
    tx = dev_bf16_bits(wl.to_bf16_bits(ints((N, C, H, W), -4, 4, 4700)))
    tw = dev_bf16_bits(wl.to_bf16_bits(ints((K, C, 7, 7), -4, 4, 4701)))
    pk = miconv.PackedFilters(tw, (N, C, H, W), 2, 3, 1)
    assert pk.nbytes > 0
    yb = torch.zeros(N * K * 112 * 112 + 1, device="cuda")
    with pytest.raises(miconv.MiconvError) as e:
        pk.forward(tx, None, yb[1:].view(N, K, 112, 112))
    assert e.value.status == miconv.ERR_ALIGN


SPLIT_CASES = [  # batch-1 layers whose reduction the wave planner splits (ResNet-50 s3/s4/s5)
    (1, 128, 28, 28, 128, 3, 3, 1, 1, 1),
    (1, 1024, 14, 14, 256, 1, 1, 1, 0, 1),
    (1, 512, 7, 7, 512, 3, 3, 1, 1, 1),
]


def test_split_reduction_shared_workspace(oracle_lib):
    """Split layers write their partials into one caller workspace, which
    channel-last bf16 calls in between also use (for x's copy, their packed
    filters and their own partials): calls of different shapes, repeated and
    interleaved on one stream, must all stay exact on small integers."""
    data, need = [], 0
    for i, (N, C, H, W, K, R, S, st, pad, g) in enumerate(SPLIT_CASES):
        x = ints((N, C, H, W), -3, 3, 4100 + i)
        w = ints((K, C // g, R, S), -3, 3, 4200 + i)
        b = ints((K,), -8, 8, 4300 + i)
        name, launches = miconv.conv2d_describe(N, C, H, W, K, R, S, st, pad, g, "f32")
        assert "igemm_wave_f32_kcrs_kernel" in name and "splitk_reduce" in name, name
        need = max(need, miconv.conv2d_workspace_bytes(N, C, H, W, K, R, S, st, pad, g))
        data.append((x, w, b, st, pad, g, oracle_lib.conv2d(x, w, b, st, pad, g, True)))
    bx = wl.to_bf16_bits(ints((2, 64, 30, 30), -4, 4, 4400))
    bw = wl.to_bf16_bits(ints((64, 64, 3, 3), -4, 4, 4401))
    bb = ints((64,), -8, 8, 4402)
    bref = oracle_lib.conv2d_bf16(bx, bw, bb, 1, 1, 1, True)
    need = max(need, miconv.conv2d_workspace_bytes(2, 64, 30, 30, 64, 3, 3, 1, 1, 1, "bf16"))
    ws = miconv.workspace(need)
    for order in ([0, 1, 2, 0], [2, 1, 0, 2, 2]):
        for j in order:
            x, w, b, st, pad, g, ref = data[j]
            P, Q = miconv.out_dims(x.shape[2], x.shape[3], w.shape[2], w.shape[3], st, pad)
            y = torch.empty((x.shape[0], w.shape[0], P, Q), device="cuda")
            miconv.conv2d_fwd_ws(dev(x), dev(w), dev(b), y, st, pad, g, True, ws=ws)
            yb = torch.empty((2, 64, 30, 30), device="cuda")
            miconv.conv2d_fwd_ws(dev_bf16_bits(bx), dev_bf16_bits(bw), dev(bb), yb, 1, 1, 1, True, ws=ws)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(y.cpu().numpy(), ref, err_msg=f"case {j}")
            np.testing.assert_array_equal(yb.cpu().numpy(), bref)


# Kernel families for the graph-capture test: (N, C, H, W, K, R, S, stride, pad, groups, dtype)
CAPTURE_CASES = [
    (1, 64, 20, 20, 48, 3, 3, 1, 1, 1, "f32"),     # wave, (r, s, c) filter reads
    (2, 64, 15, 13, 130, 1, 1, 1, 0, 1, "f32"),    # wave 1x1, 16-byte filter reads
    (1, 3, 45, 47, 40, 7, 7, 2, 3, 1, "f32"),      # wave stem, (r, s, c4)
    (3, 3, 224, 224, 64, 3, 3, 1, 1, 1, "f32"),    # one tile per wavefront
    (1, 512, 7, 7, 512, 3, 3, 1, 1, 1, "f32"),     # split reduction (ws)
    (1, 12, 9, 9, 18, 3, 3, 1, 1, 3, "f32"),       # direct
    (2, 32, 12, 12, 32, 3, 3, 1, 1, 32, "f32"),    # depthwise
    (4, 64, 56, 56, 256, 1, 1, 1, 0, 1, "bf16"),   # NCHW-operand 1x1
    (8, 64, 28, 28, 128, 1, 1, 2, 0, 1, "bf16"),   # channel-last copy (ws) / gather (plain)
    (21, 64, 56, 56, 64, 3, 3, 1, 1, 1, "bf16"),   # halo kernel (ws)
    (1, 512, 7, 7, 512, 3, 3, 1, 1, 1, "bf16"),    # split (ws)
    (1, 3, 224, 224, 64, 7, 7, 2, 3, 1, "bf16"),   # stem (ws: filters packed per call)
]


@pytest.mark.parametrize("case", CAPTURE_CASES, ids=lambda c: "x".join(map(str, c[:10])) + "-" + c[10])
@pytest.mark.parametrize("mode", ["plain", "ws"])
def test_first_call_captured_in_a_graph(oracle_lib, case, mode):
    """The very first call of a shape (nothing warmed up, nothing allocated
    by the library) captured into a HIP graph, replayed three times with
    eager work and synchronisation in between: every replay exact against
    the oracle on small integers."""
    N, C, H, W, K, R, S, st, pad, g, dt = case
    seed = 5100 + sum(case[:10]) + (7 if mode == "ws" else 0)
    x = ints((N, C, H, W), -4, 4, seed)
    w = ints((K, C // g, R, S), -4, 4, seed + 1)
    b = ints((K,), -8, 8, seed + 2)
    if dt == "bf16":
        x, w = wl.to_bf16_bits(x), wl.to_bf16_bits(w)
        tx, tw = dev_bf16_bits(x), dev_bf16_bits(w)
        ref = oracle_lib.conv2d_bf16(x, w, b, st, pad, g, True)
    else:
        tx, tw = dev(x), dev(w)
        ref = oracle_lib.conv2d(x, w, b, st, pad, g, True)
    tb = dev(b)
    P, Q = miconv.out_dims(H, W, R, S, st, pad)
    y = torch.empty((N, K, P, Q), device="cuda")
    ws = None
    if mode == "ws":
        ws = miconv.workspace(miconv.conv2d_workspace_bytes(N, C, H, W, K, R, S, st, pad, g, dt))
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    with torch.cuda.graph(graph, stream=side):
        if mode == "ws":
            miconv.conv2d_fwd_ws(tx, tw, tb, y, st, pad, g, True, ws=ws, stream=side)
        elif dt == "bf16":
            miconv.conv2d_fwd_bf16(tx, tw, tb, y, st, pad, g, True, stream=side)
        else:
            miconv.conv2d_fwd(tx, tw, tb, y, st, pad, g, True, stream=side)
    for rep in range(3):
        y.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(y.cpu().numpy(), ref, err_msg=f"replay {rep}")


def test_workspace_too_small_launches_nothing():
    N, C, H, W, K = 1, 512, 7, 7, 512
    need = miconv.conv2d_workspace_bytes(N, C, H, W, K, 3, 3, 1, 1)
    assert need > 0
    x = torch.ones((N, C, H, W), device="cuda")
    w = torch.ones((K, C, 3, 3), device="cuda")
    y = torch.full((N, K, H, W), float("nan"), device="cuda")
    ws = miconv.workspace(need)
    with pytest.raises(miconv.MiconvError) as e:
        miconv.conv2d_fwd_ws(x, w, None, y, 1, 1, ws=ws[:need - 256])
    assert e.value.status == miconv.ERR_WORKSPACE
    torch.cuda.synchronize()
    assert torch.isnan(y).all()


def test_maxpool_add_cast(oracle_lib):
    rng = np.random.default_rng(0)
    for (N, C, H, W, R, st, pad) in [(1, 64, 112, 112, 3, 2, 1), (2, 64, 224, 224, 2, 2, 0), (1, 3, 7, 9, 3, 2, 1)]:
        x = rng.standard_normal((N, C, H, W)).astype(np.float32)
        P, Q = oracle_lib.out_dims(H, W, R, R, st, pad)
        y = torch.empty((N, C, P, Q), device="cuda")
        miconv.maxpool2d_fwd(dev(x), y, R, R, st, pad)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(y.cpu().numpy(), oracle_lib.maxpool2d(x, R, R, st, pad))
    for n in (1, 7, 4096, 1 << 20):
        a = rng.standard_normal(n).astype(np.float32)
        b = rng.standard_normal(n).astype(np.float32)
        for relu in (True, False):
            y = torch.empty(n, device="cuda")
            miconv.add_act_fwd(dev(a), dev(b), y, relu)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(y.cpu().numpy(), oracle_lib.add_act(a, b, relu))
    bits = rng.integers(0, 2 ** 32, 1 << 18, dtype=np.uint64).astype(np.uint32)
    f = bits.view(np.float32)
    f = f[np.isfinite(f)]
    y = torch.empty(f.shape, device="cuda", dtype=torch.bfloat16)
    miconv.cast_f32_to_bf16(dev(f), y)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(y.view(torch.int16).cpu().numpy().view(np.uint16), oracle_lib.f32_to_bf16(f))


def test_cast_bf16_rounding_every_class(oracle_lib):
    """The device's bf16 rounding (one conversion instruction for a pair of
    values, used by every bf16 epilogue) against the oracle's on the cases
    that decide rounding: signed zeros, infinities, quiet and signalling NaNs
    of both signs and several payloads, denormals, the largest finite values
    (which round to infinity), every exponent with a dropped half of exactly
    0x8000 (ties, both parities of the kept bit) and its neighbours, and 2^22
    random bit patterns; odd and even lengths."""
    specials = [0x00000000, 0x80000000, 0x7F800000, 0xFF800000, 0x7FC00000, 0xFFC00000, 0x7F800001,
                0xFF800001, 0x7FBFFFFF, 0xFFFFFFFF, 0x7FFF8000, 0x00000001, 0x80000001, 0x007FFFFF,
                0x00008000, 0x00018000, 0x80008000, 0x7F7FFFFF, 0xFF7FFFFF, 0x7F7F8000, 0x7F7F7FFF]
    e = np.arange(256, dtype=np.uint32) << 23
    ties = np.concatenate([e | 0x8000, e | 0x18000, e | 0x7FFF, e | 0x8001, e | 0x17FFF, e | 0x18001])
    ties = np.concatenate([ties, ties | 0x80000000])
    rng = np.random.default_rng(7)
    rand = rng.integers(0, 2 ** 32, 1 << 22, dtype=np.uint64).astype(np.uint32)
    bits = np.concatenate([np.uint32(specials), ties, rand])
    for n in (bits.size, bits.size - 1, 1, 3):
        f = bits[:n].view(np.float32)
        y = torch.empty(f.shape, device="cuda", dtype=torch.bfloat16)
        miconv.cast_f32_to_bf16(dev(f), y)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(y.view(torch.int16).cpu().numpy().view(np.uint16), oracle_lib.f32_to_bf16(f))


def test_rejects_wrong_shapes_from_python():
    x = torch.zeros((1, 4, 8, 8), device="cuda")
    w = torch.zeros((4, 4, 3, 3), device="cuda")
    with pytest.raises(ValueError):
        miconv.conv2d_fwd(x, w, None, torch.zeros((1, 4, 7, 7), device="cuda"), 1, 1)
    with pytest.raises(TypeError):
        miconv.conv2d_fwd(x.double(), w, None, torch.zeros((1, 4, 8, 8), device="cuda"), 1, 1)
    # an expanded y (image stride 0) would make every image land on one buffer
    x4 = torch.zeros((4, 4, 8, 8), device="cuda")
    y1 = torch.full((1, 4, 8, 8), float("nan"), device="cuda")
    res = torch.zeros((4, 4, 8, 8), device="cuda")
    for f in (miconv.conv2d_fwd_ex, miconv.conv2d_fwd_ws):
        with pytest.raises(ValueError):
            f(x4, w, None, y1.expand(4, 4, 8, 8), 1, 1)
        with pytest.raises(ValueError):
            f(x4, w, None, torch.empty((4, 4, 8, 8), device="cuda"), 1, 1, res=y1.expand(4, 4, 8, 8))
    with pytest.raises(ValueError):
        miconv.Stack([(miconv.OP_CONV_F32, x4, w, None, y1.expand(4, 4, 8, 8), 1, 1, 1, False)])
    torch.cuda.synchronize()
    assert torch.isnan(y1).all()


def test_depthwise_batch64_sampled(oracle_lib):
    """Depthwise at the bandwidth-sweep batch (64 images): images 0 and 63 of
    every MobileNet depthwise shape against the oracle."""
    for i, l in _layers(3):
        if l.kind != "dw":
            continue
        l = l.with_batch(64)
        x, w, b = wl.layer_tensors(3, i, l)
        y = miconv.dwconv2d(dev(x), dev(w), dev(b), l.stride, l.pad, l.relu)
        torch.cuda.synchronize()
        y = y.cpu().numpy()
        for n in (0, 63):
            ref = oracle_lib.dwconv2d(x[n:n + 1], w, b, l.stride, l.pad, l.relu)
            e = err_inf(y[n:n + 1], ref)
            assert e <= TOL_F32, (l.name, n, e)
