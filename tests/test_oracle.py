"""Pins for the CPU oracle (runs without a GPU).

The oracle is the plain Conv2D definition (paper Sec. 3.2.2 names the operator;
Sec. 4.2 and Sec. 5 state that the optimised schedules keep its semantics).
These tests tie it to things other than itself: hand-worked examples,
closed forms (delta kernel, all-ones counts, zero input), identities
(1x1 conv = matrix product, linearity, batch independence, channel
permutation, depthwise = block-diagonal dense conv) and brute force against
independent library routines (torch float64 conv2d / max_pool2d, numpy
float64 matmul) over a grid of tiny shapes.
"""
import itertools
import json
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

GOLD = os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")


@pytest.fixture(scope="module")
def gold():
    with open(GOLD) as f:
        return json.load(f)


def _f32(a):
    return np.asarray(a, dtype=np.float32)


def test_hand_examples(oracle_lib, gold):
    x = _f32(gold["x_1to9"]).reshape(1, 1, 3, 3)
    for case in gold["cases"]:
        w = _f32(case["w"])
        w = w.reshape(1, 1, *w.shape)
        b = _f32([case["bias"]])
        y = oracle_lib.conv2d(x, w, b, case["stride"], case["pad"], 1, case["relu"])
        np.testing.assert_array_equal(y[0, 0], _f32(case["y"]), err_msg=case["id"])


def test_hand_depthwise(oracle_lib, gold):
    d = gold["depthwise"]
    x = _f32(d["x"])[None]
    w = _f32(d["w"])[:, None]
    y = oracle_lib.dwconv2d(x, w, None, d["stride"], d["pad"])
    np.testing.assert_array_equal(y[0], _f32(d["y"]))
    # The same operator through the grouped dense entry.
    y2 = oracle_lib.conv2d(x, w, None, d["stride"], d["pad"], groups=2)
    np.testing.assert_array_equal(y2, y)


def test_out_dims_closed_form(oracle_lib):
    # floor((H + 2 pad - R)/stride) + 1, worked by hand for the shapes of the networks
    assert oracle_lib.out_dims(224, 224, 7, 7, 2, 3) == (112, 112)
    assert oracle_lib.out_dims(112, 112, 3, 3, 2, 1) == (56, 56)
    assert oracle_lib.out_dims(56, 56, 1, 1, 2, 0) == (28, 28)
    assert oracle_lib.out_dims(7, 7, 3, 3, 1, 1) == (7, 7)
    assert oracle_lib.out_dims(5, 6, 3, 2, 2, 0) == (2, 3)
    assert oracle_lib.out_dims(2, 2, 3, 3, 1, 0) == (0, 0)


@pytest.mark.parametrize("r0,s0", [(0, 0), (0, 2), (1, 1), (2, 0), (2, 1)])
@pytest.mark.parametrize("stride", [1, 2])
def test_delta_kernel_shifts(oracle_lib, r0, s0, stride):
    """w[k][c][r][s] = [k==c][r==r0][s==s0] moves x by (r0-pad, s0-pad): no flip."""
    rng = np.random.default_rng(7)
    C, H, W, pad = 3, 7, 6, 1
    x = rng.standard_normal((2, C, H, W)).astype(np.float32)
    w = np.zeros((C, C, 3, 3), np.float32)
    for k in range(C):
        w[k, k, r0, s0] = 1.0
    y = oracle_lib.conv2d(x, w, None, stride, pad)
    P, Q = y.shape[2:]
    expect = np.zeros_like(y)
    for p in range(P):
        for q in range(Q):
            h, ww = p * stride - pad + r0, q * stride - pad + s0
            if 0 <= h < H and 0 <= ww < W:
                expect[:, :, p, q] = x[:, :, h, ww]
    np.testing.assert_array_equal(y, expect)


@pytest.mark.parametrize("stride", [1, 2])
def test_1x1_is_matmul(oracle_lib, stride):
    rng = np.random.default_rng(11)
    N, C, H, W, K = 2, 13, 9, 7, 5
    x = rng.standard_normal((N, C, H, W)).astype(np.float32)
    w = rng.standard_normal((K, C, 1, 1)).astype(np.float32)
    b = rng.standard_normal(K).astype(np.float32)
    y = oracle_lib.conv2d(x, w, b, stride, 0)
    xs = x[:, :, ::stride, ::stride].astype(np.float64)
    ref = np.matmul(w[:, :, 0, 0].astype(np.float64), xs.reshape(N, C, -1)).reshape(N, K, *xs.shape[2:])
    ref = ref + b.astype(np.float64)[None, :, None, None]
    np.testing.assert_allclose(y, ref.astype(np.float32), rtol=2.0 ** -23, atol=0)


def test_linearity_exact(oracle_lib):
    """conv(a*x1 + b*x2) = a*conv(x1) + b*conv(x2) and the same in w; small
    integers and power-of-two scales keep every value exact."""
    rng = np.random.default_rng(3)
    x1 = rng.integers(-4, 5, (2, 3, 6, 5)).astype(np.float32)
    x2 = rng.integers(-4, 5, (2, 3, 6, 5)).astype(np.float32)
    w1 = rng.integers(-4, 5, (4, 3, 3, 3)).astype(np.float32)
    w2 = rng.integers(-4, 5, (4, 3, 3, 3)).astype(np.float32)
    c = lambda x, w: oracle_lib.conv2d(x, w, None, 2, 1)
    np.testing.assert_array_equal(c(2 * x1 - 0.5 * x2, w1), 2 * c(x1, w1) - 0.5 * c(x2, w1))
    np.testing.assert_array_equal(c(x1, 4 * w1 + w2), 4 * c(x1, w1) + c(x1, w2))


def test_batch_independence_and_channel_permutation(oracle_lib):
    rng = np.random.default_rng(5)
    x = rng.standard_normal((3, 6, 8, 8)).astype(np.float32)
    w = rng.standard_normal((4, 6, 3, 3)).astype(np.float32)
    b = rng.standard_normal(4).astype(np.float32)
    y = oracle_lib.conv2d(x, w, b, 1, 1, relu=True)
    for n in range(3):
        np.testing.assert_array_equal(oracle_lib.conv2d(x[n:n + 1], w, b, 1, 1, relu=True)[0], y[n])
    # Permuting the input channels of x and w together changes only the order of
    # the terms, so compare within rounding.
    perm = rng.permutation(6)
    y2 = oracle_lib.conv2d(x[:, perm], w[:, perm], b, 1, 1, relu=True)
    np.testing.assert_allclose(y2, y, rtol=1e-6, atol=1e-6)


def test_zero_input_and_all_ones_counts(oracle_lib):
    N, C, H, W, K, R, S, st, pad = 1, 3, 5, 4, 2, 3, 3, 2, 2
    b = np.array([0.25, -0.5], np.float32)
    y0 = oracle_lib.conv2d(np.zeros((N, C, H, W), np.float32), np.ones((K, C, R, S), np.float32),
                           b, st, pad, relu=True)
    np.testing.assert_array_equal(y0, np.maximum(b, 0)[None, :, None, None] * np.ones_like(y0))
    y1 = oracle_lib.conv2d(np.ones((N, C, H, W), np.float32), np.ones((K, C, R, S), np.float32),
                           b, st, pad)
    P, Q = y1.shape[2:]
    for p in range(P):
        rows = sum(1 for r in range(R) if 0 <= p * st - pad + r < H)
        for q in range(Q):
            cols = sum(1 for s in range(S) if 0 <= q * st - pad + s < W)
            for k in range(K):
                assert y1[0, k, p, q] == np.float32(C * rows * cols + float(b[k]))


def test_depthwise_is_block_diagonal_dense(oracle_lib):
    rng = np.random.default_rng(9)
    N, C, H, W = 2, 5, 9, 8
    x = rng.standard_normal((N, C, H, W)).astype(np.float32)
    w = rng.standard_normal((C, 1, 3, 3)).astype(np.float32)
    b = rng.standard_normal(C).astype(np.float32)
    for st in (1, 2):
        y = oracle_lib.dwconv2d(x, w, b, st, 1, relu=True)
        wbd = np.zeros((C, C, 3, 3), np.float32)
        for c in range(C):
            wbd[c, c] = w[c, 0]
        yd = oracle_lib.conv2d(x, wbd, b, st, 1, relu=True)
        # block-diagonal adds exact zeros only, so the two agree bitwise
        np.testing.assert_array_equal(y, yd)


def _tiny_grid():
    for N, C, Kmul, H, W, R, S, st, pad in itertools.product(
            (1, 2), (1, 2, 3), (1, 2), range(1, 7), range(1, 7), (1, 2, 3), (1, 2, 3), (1, 2), (0, 1, 2)):
        for groups in sorted({1, C}):
            K = Kmul * groups
            if (H + 2 * pad - R) < 0 or (W + 2 * pad - S) < 0:
                continue
            yield N, C, K, H, W, R, S, st, pad, groups


def test_brute_force_against_torch_float64(oracle_lib):
    """Oracle vs torch.nn.functional.conv2d in float64 (an independent
    implementation) on a seeded sample of the tiny-shape grid."""
    cases = list(_tiny_grid())
    rng = np.random.default_rng(2019)
    idx = rng.choice(len(cases), size=1500, replace=False)
    for i in idx:
        N, C, K, H, W, R, S, st, pad, groups = cases[i]
        x = rng.standard_normal((N, C, H, W)).astype(np.float32)
        w = rng.standard_normal((K, C // groups, R, S)).astype(np.float32)
        b = rng.standard_normal(K).astype(np.float32)
        relu = bool(rng.integers(0, 2))
        y = oracle_lib.conv2d(x, w, b, st, pad, groups, relu)
        ref = F.conv2d(torch.from_numpy(x).double(), torch.from_numpy(w).double(),
                       torch.from_numpy(b).double(), stride=st, padding=pad, groups=groups)
        if relu:
            ref = torch.relu(ref)
        ref = ref.numpy()
        assert y.shape == ref.shape, cases[i]
        np.testing.assert_allclose(y, ref.astype(np.float32), rtol=2.0 ** -22, atol=1e-12,
                                   err_msg=str(cases[i]))


def test_brute_force_small_integers_exact(oracle_lib):
    """Small-integer data make every sum exact, so the oracle must equal an
    independent numpy im2col + float64 matmul bit for bit."""
    rng = np.random.default_rng(42)
    for N, C, K, H, W, R, S, st, pad, groups in [(2, 3, 6, 6, 5, 3, 3, 2, 1, 3), (1, 2, 4, 5, 6, 2, 3, 1, 2, 1),
                                                 (2, 3, 3, 4, 4, 1, 1, 2, 0, 1), (1, 3, 3, 6, 6, 3, 2, 1, 0, 3)]:
        x = rng.integers(-4, 5, (N, C, H, W)).astype(np.float32)
        w = rng.integers(-4, 5, (K, C // groups, R, S)).astype(np.float32)
        b = rng.integers(-8, 9, K).astype(np.float32)
        y = oracle_lib.conv2d(x, w, b, st, pad, groups)
        xp = np.pad(x.astype(np.float64), ((0, 0), (0, 0), (pad, pad), (pad, pad)))
        P = (H + 2 * pad - R) // st + 1
        Q = (W + 2 * pad - S) // st + 1
        Cg, Kg = C // groups, K // groups
        ref = np.zeros((N, K, P, Q))
        for g in range(groups):
            cols = np.empty((N, Cg * R * S, P * Q))
            for c in range(Cg):
                for r in range(R):
                    for s in range(S):
                        patch = xp[:, g * Cg + c, r:r + st * (P - 1) + 1:st, s:s + st * (Q - 1) + 1:st]
                        cols[:, (c * R + r) * S + s] = patch.reshape(N, -1)
            wm = w[g * Kg:(g + 1) * Kg].reshape(Kg, -1).astype(np.float64)
            ref[:, g * Kg:(g + 1) * Kg] = np.matmul(wm, cols).reshape(N, Kg, P, Q)
        ref += b[None, :, None, None]
        np.testing.assert_array_equal(y, ref.astype(np.float32))


def test_bf16_entry_matches_widened_fp32(oracle_lib):
    """The bf16 entry widens its inputs exactly: on values that bf16 holds it
    must agree bitwise with the fp32 entry."""
    rng = np.random.default_rng(1)
    x = rng.standard_normal((2, 4, 7, 7)).astype(np.float32)
    w = rng.standard_normal((3, 4, 3, 3)).astype(np.float32)
    b = rng.standard_normal(3).astype(np.float32)
    xb = torch.from_numpy(x).to(torch.bfloat16)
    wb = torch.from_numpy(w).to(torch.bfloat16)
    xbits = xb.view(torch.int16).numpy().view(np.uint16)
    wbits = wb.view(torch.int16).numpy().view(np.uint16)
    y16 = oracle_lib.conv2d_bf16(xbits, wbits, b, 2, 1, relu=True)
    y32 = oracle_lib.conv2d(xb.float().numpy(), wb.float().numpy(), b, 2, 1, relu=True)
    np.testing.assert_array_equal(y16, y32)


def test_bf16_rounding_hand_cases(oracle_lib, gold):
    for src, dst in gold["bf16_rounding"]["cases"]:
        f = np.array([int(src, 16)], np.uint32).view(np.float32)
        assert oracle_lib.f32_to_bf16(f)[0] == int(dst, 16), src
    nan = np.array([0x7fc00001], np.uint32).view(np.float32)
    out = oracle_lib.f32_to_bf16(nan)[0]
    assert (out & 0x7f80) == 0x7f80 and (out & 0x7f) != 0


def test_bf16_rounding_matches_torch(oracle_lib):
    rng = np.random.default_rng(4)
    bits = rng.integers(0, 2 ** 32, 200000, dtype=np.uint64).astype(np.uint32)
    f = bits.view(np.float32)
    f = f[np.isfinite(f)]
    ref = torch.from_numpy(f).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(oracle_lib.f32_to_bf16(f), ref)
    np.testing.assert_array_equal(oracle_lib.bf16_to_f32(ref), torch.from_numpy(ref.view(np.int16)).view(
        torch.bfloat16).float().numpy())


@pytest.mark.parametrize("R,stride,pad", [(2, 2, 0), (3, 2, 1), (3, 1, 1)])
def test_maxpool_against_torch(oracle_lib, R, stride, pad):
    rng = np.random.default_rng(R * 10 + pad)
    x = rng.standard_normal((2, 3, 9, 8)).astype(np.float32)
    y = oracle_lib.maxpool2d(x, R, R, stride, pad)
    ref = F.max_pool2d(torch.from_numpy(x).double(), R, stride, pad).float().numpy()
    np.testing.assert_array_equal(y, ref)


def test_add_act(oracle_lib):
    a = np.array([1.5, -2.0, 0.25, -0.0], np.float32)
    b = np.array([-3.0, 1.0, 0.5, 0.0], np.float32)
    np.testing.assert_array_equal(oracle_lib.add_act(a, b, True), np.array([0, 0, 0.75, 0], np.float32))
    np.testing.assert_array_equal(oracle_lib.add_act(a, b, False), np.array([-1.5, -1.0, 0.75, 0], np.float32))


def test_rejects_bad_arguments(oracle_lib):
    x = np.zeros((1, 3, 4, 4), np.float32)
    with pytest.raises(ValueError):
        oracle_lib.conv2d(x, np.zeros((2, 2, 3, 3), np.float32), groups=2)   # C % groups
    with pytest.raises(ValueError):
        oracle_lib.conv2d(x, np.zeros((2, 3, 5, 5), np.float32))             # empty output


def test_hand_residual(oracle_lib, gold):
    """The fused residual join, act(conv + bias + res), on a hand-worked 1x1
    example; the activation comes after the join (relu before it gives a
    different, wrong, answer on this example)."""
    d = gold["residual"]
    x = _f32(d["x"])[None, None]
    w = _f32([[[[d["w"]]]]])
    b = _f32([d["bias"]])
    res = _f32(d["res"])[None, None]
    y = oracle_lib.conv2d(x, w, b, relu=True, res=res)
    np.testing.assert_array_equal(y[0, 0], _f32(d["y_relu"]))
    np.testing.assert_array_equal(oracle_lib.conv2d(x, w, b, relu=False, res=res)[0, 0],
                                  _f32(d["y_linear"]))
    wrong = oracle_lib.conv2d(x, w, b, relu=True) + res
    np.testing.assert_array_equal(wrong[0, 0], _f32(d["y_relu_before_join"]))
    assert not np.array_equal(wrong, y)
    # bf16 entry: the same values are exact in bf16
    xb, wb = oracle_lib.f32_to_bf16(x), oracle_lib.f32_to_bf16(w)
    np.testing.assert_array_equal(oracle_lib.conv2d_bf16(xb, wb, b, relu=True, res=res), y)


def test_residual_brute_force_against_torch_float64(oracle_lib):
    """act(conv + bias + res) against torch float64 conv2d plus the residual,
    on random tiny shapes (strides, padding, groups)."""
    rng = np.random.default_rng(77)
    cases = list(_tiny_grid())
    for i in rng.choice(len(cases), size=300, replace=False):
        N, C, K, H, W, R, S, st, pad, groups = cases[i]
        x = rng.standard_normal((N, C, H, W)).astype(np.float32)
        w = rng.standard_normal((K, C // groups, R, S)).astype(np.float32)
        b = rng.standard_normal(K).astype(np.float32)
        ref = F.conv2d(torch.from_numpy(x).double(), torch.from_numpy(w).double(),
                       torch.from_numpy(b).double(), stride=st, padding=pad, groups=groups)
        res = rng.standard_normal(tuple(ref.shape)).astype(np.float32)
        relu = bool(rng.integers(0, 2))
        ref = ref + torch.from_numpy(res).double()
        if relu:
            ref = torch.relu(ref)
        y = oracle_lib.conv2d(x, w, b, st, pad, groups, relu, res=res)
        np.testing.assert_allclose(y, ref.numpy().astype(np.float32), rtol=2.0 ** -22, atol=1e-12,
                                   err_msg=str(cases[i]))


def test_residual_small_integers_exact(oracle_lib):
    """On small integers every sum is exact: the fused join equals the plain
    conv plus the residual, and res = 0 gives the plain conv."""
    rng = np.random.default_rng(5)
    x = rng.integers(-4, 5, (2, 6, 7, 5)).astype(np.float32)
    w = rng.integers(-4, 5, (4, 3, 3, 3)).astype(np.float32)
    b = rng.integers(-8, 9, 4).astype(np.float32)
    plain = oracle_lib.conv2d(x, w, b, 2, 1, 2)
    res = rng.integers(-50, 51, plain.shape).astype(np.float32)
    np.testing.assert_array_equal(oracle_lib.conv2d(x, w, b, 2, 1, 2, res=res), plain + res)
    np.testing.assert_array_equal(oracle_lib.conv2d(x, w, b, 2, 1, 2, True, res=res),
                                  np.maximum(plain + res, 0))
    np.testing.assert_array_equal(oracle_lib.conv2d(x, w, b, 2, 1, 2, True, res=np.zeros_like(plain)),
                                  oracle_lib.conv2d(x, w, b, 2, 1, 2, True))
    with pytest.raises(ValueError):
        oracle_lib.conv2d(x, w, b, 2, 1, 2, res=res[:, :2])


# ---- channel-last bf16 layers (conv2d_bf16_cl, maxpool2d_bf16_cl) ----

def _bits(t):
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


def test_channel_last_layer_against_torch(oracle_lib):
    """conv2d_bf16_cl against torch: float64 conv2d of the exactly widened
    bf16 values, plus bias and the widened bf16 residual, activation, then
    torch's cast to float32 and to bfloat16, in channel-last order.  Over 120
    random tiny shapes (groups, strides, padding) every output bit agrees."""
    rng = np.random.default_rng(11)
    for case in range(120):
        N = int(rng.integers(1, 3))
        g = int(rng.choice([1, 2]))
        Cg, Kg = int(rng.integers(1, 4)), int(rng.integers(1, 4))
        C, K = Cg * g, Kg * g
        R, S = int(rng.integers(1, 4)), int(rng.integers(1, 4))
        H, W = int(rng.integers(R, 8)), int(rng.integers(S, 8))
        st, pad = int(rng.integers(1, 3)), int(rng.integers(0, 2))
        torch.manual_seed(1100 + case)
        xb = torch.randn(N, H, W, C).to(torch.bfloat16)
        wb = torch.randn(K, Cg, R, S).to(torch.bfloat16)
        b = torch.randn(K) * 0.1
        P, Q = oracle_lib.out_dims(H, W, R, S, st, pad)
        rb = torch.randn(N, P, Q, K).to(torch.bfloat16) if case % 2 else None
        relu = bool(case % 3)
        ref = F.conv2d(xb.permute(0, 3, 1, 2).double(), wb.double(), b.double(), st, pad, 1, g)
        if rb is not None:
            ref = ref + rb.permute(0, 3, 1, 2).double()
        if relu:
            ref = ref.clamp_min(0)
        want = _bits(ref.float().to(torch.bfloat16).permute(0, 2, 3, 1))
        got = oracle_lib.conv2d_bf16_cl(_bits(xb), _bits(wb), b.numpy(), st, pad, g, relu,
                                        None if rb is None else _bits(rb))
        np.testing.assert_array_equal(got, want, err_msg=f"case {case}")


def test_channel_last_layer_rounds_through_fp32(oracle_lib):
    """The reading fixed for a bf16 output: the fp64 sum is rounded to fp32
    first, then to bf16.  x = (1, 2^-8, 2^-30), w = 1 (a 1x1 conv over three
    channels) sums to 1 + 2^-8 + 2^-30; fp32 drops the 2^-30, leaving
    1 + 2^-8, exactly half a bf16 step above 1, which ties to even: 1.0 (bits
    0x3F80).  Rounding the fp64 sum straight to bf16 would give 1.0078125."""
    x = torch.tensor([1.0, 2.0 ** -8, 2.0 ** -30]).to(torch.bfloat16).view(1, 1, 1, 3)
    w = torch.ones(1, 3, 1, 1).to(torch.bfloat16)
    got = oracle_lib.conv2d_bf16_cl(_bits(x), _bits(w))
    assert got.shape == (1, 1, 1, 1) and int(got[0, 0, 0, 0]) == 0x3F80


def test_channel_last_maxpool_against_torch(oracle_lib):
    """maxpool2d_bf16_cl equals torch's max_pool2d of the bf16 values in
    channel-last order, bit for bit (a maximum is one of the inputs)."""
    torch.manual_seed(12)
    for R, st, pad in ((3, 2, 1), (2, 2, 0), (3, 1, 1)):
        xb = torch.randn(2, 9, 11, 16).to(torch.bfloat16)
        want = F.max_pool2d(xb.permute(0, 3, 1, 2).float(), R, st, pad).to(torch.bfloat16)
        got = oracle_lib.maxpool2d_bf16_cl(_bits(xb), R, R, st, pad)
        np.testing.assert_array_equal(got, _bits(want.permute(0, 2, 3, 1)))
