"""GPU: the stack executor (eager and HIP-graph replay) against single calls.

Every layer of a stack must produce, bit for bit, what the same entry point
produces when called on its own; a captured graph replayed several times,
with eager work and synchronisations in between, must give the same bits on
every replay.  The oracle ties the single calls to the definition elsewhere
(test_gpu_parity); here a small-integer stack is also checked against it.
"""
import numpy as np
import pytest
import torch

from paper_1907_02154_amd import miconv
from paper_1907_02154_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    miconv.lib()


def _mobilenet_stack(ints: bool):
    ops, ref_inputs = [], []
    for i, l in enumerate(wl.workload(3).layers[:9]):
        x, w, b = wl.layer_tensors(3, i, l)
        if ints:
            x = wl.small_ints(x.shape, -3, 3, 500 + i)
            w = wl.small_ints(w.shape, -3, 3, 600 + i)
            b = wl.small_ints(b.shape, -8, 8, 700 + i)
        P, Q = miconv.out_dims(l.H, l.W, l.R, l.S, l.stride, l.pad)
        tx, tw, tb = (torch.from_numpy(a).cuda() for a in (x, w, b))
        ty = torch.full((l.N, l.K, P, Q), float("nan"), device="cuda")
        op = miconv.OP_DWCONV_F32 if l.kind == "dw" else miconv.OP_CONV_F32
        ops.append((op, tx, tw, tb, ty, l.stride, l.pad, l.groups, l.relu))
        ref_inputs.append((l, x, w, b))
    return ops, ref_inputs


def _single_calls(ops):
    outs = []
    for op, x, w, b, y, st, pad, g, relu in ops:
        y2 = torch.empty_like(y)
        if op == miconv.OP_DWCONV_F32:
            miconv.dwconv2d_fwd(x, w, b, y2, st, pad, relu)
        else:
            miconv.conv2d_fwd(x, w, b, y2, st, pad, g, relu)
        outs.append(y2)
    torch.cuda.synchronize()
    return outs


def test_stack_eager_and_graph_match_single_calls():
    ops, _ = _mobilenet_stack(ints=False)
    ref = _single_calls(ops)
    s = miconv.Stack(ops)
    s.launch()
    torch.cuda.synchronize()
    for o, r in zip(ops, ref):
        assert torch.equal(o[4], r)
    for o in ops:
        o[4].fill_(float("nan"))
    s.capture(3, timed=True)
    for rep in range(3):
        for o in ops:
            o[4].fill_(float("nan"))          # eager work between replays
        torch.cuda.synchronize()
        s.replay()
        torch.cuda.synchronize()
        for i, (o, r) in enumerate(zip(ops, ref)):
            assert torch.equal(o[4], r), f"replay {rep} layer {i}"
    t = s.times()
    assert t.shape == (3, s.launches) and s.launches >= len(ops) and np.all(t > 0)
    assert [s.launch_info(j)[0] for j in range(s.launches)] == sorted(s.launch_info(j)[0] for j in range(s.launches))
    s.close()


def test_stack_small_ints_against_oracle(oracle_lib):
    ops, refs = _mobilenet_stack(ints=True)
    s = miconv.Stack(ops)
    s.capture(1, timed=False)
    s.replay()
    torch.cuda.synchronize()
    for o, (l, x, w, b) in zip(ops, refs):
        if l.kind == "dw":
            want = oracle_lib.dwconv2d(x, w, b, l.stride, l.pad, l.relu)
        else:
            want = oracle_lib.conv2d(x, w, b, l.stride, l.pad, l.groups, l.relu)
        np.testing.assert_array_equal(o[4].cpu().numpy(), want, err_msg=l.name)
    s.close()


def test_stack_rejects_bad_layer():
    x = torch.zeros((1, 4, 8, 8), device="cuda")
    w = torch.zeros((4, 4, 3, 3), device="cuda")
    y = torch.zeros((1, 4, 8, 8), device="cuda")
    with pytest.raises(miconv.MiconvError):
        miconv.Stack([(miconv.OP_DWCONV_F32, x, w, None, y, 1, 1, 1, False)])


def test_stack_eager_timed_matches():
    ops, _ = _mobilenet_stack(ints=False)
    ref = _single_calls(ops)
    s = miconv.Stack(ops)
    s.launch_timed(2)
    torch.cuda.synchronize()
    for o, r in zip(ops, ref):
        assert torch.equal(o[4], r)
    t = s.times()
    assert t.shape == (2, s.launches) and np.all(t > 0)
    s.close()


def _resnet_stack_ints(config, idxs):
    ops, refs = [], []
    for i in idxs:
        l = wl.workload(config).layers[i]
        x = wl.small_ints((l.N, l.C, l.H, l.W), -3, 3, 800 + i)
        w = wl.small_ints((l.K, l.C // l.groups, l.R, l.S), -3, 3, 900 + i)
        b = wl.small_ints((l.K,), -8, 8, 1000 + i)
        P, Q = miconv.out_dims(l.H, l.W, l.R, l.S, l.stride, l.pad)
        y = torch.full((l.N, l.K, P, Q), float("nan"), device="cuda")
        if wl.workload(config).dtype == "bf16":
            bx, bw = wl.to_bf16_bits(x), wl.to_bf16_bits(w)
            tx = torch.from_numpy(bx.view(np.int16)).cuda().view(torch.bfloat16)
            tw = torch.from_numpy(bw.view(np.int16)).cuda().view(torch.bfloat16)
            ops.append((miconv.OP_CONV_BF16, tx, tw, torch.from_numpy(b).cuda(), y, l.stride, l.pad,
                        l.groups, l.relu))
        else:
            ops.append((miconv.OP_CONV_F32, torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda(),
                        torch.from_numpy(b).cuda(), y, l.stride, l.pad, l.groups, l.relu))
        refs.append((l, x, w, b))
    return ops, refs


@pytest.mark.parametrize("config,idxs", [(2, [0, 2, 12, 25, 44, 48]), (5, [0, 2, 16, 29, 44])])
def test_stack_packed_filters_small_ints(oracle_lib, config, idxs):
    """3x3 layers in a stack read KRSC-packed filters (packed once at create):
    exact against the oracle on small integers, eager and replayed."""
    ops, refs = _resnet_stack_ints(config, idxs)
    s = miconv.Stack(ops)
    names = [s.describe(j) for j in range(len(ops))]
    # 3x3 layers read filters packed once at create (reduction order r, s, c):
    # no per-call packing kernel
    assert any(n.startswith("igemm_wave_f32_kernel<3, 3") and n.split(" + ")[0].endswith(", 1, false>") or "nhwc" in n
               for n in names), names
    assert not any("pack_" in n for n in names), names
    s.launch()
    torch.cuda.synchronize()
    for o, (l, x, w, b) in zip(ops, refs):
        want = oracle_lib.conv2d(x, w, b, l.stride, l.pad, l.groups, l.relu)
        np.testing.assert_array_equal(o[4].cpu().numpy(), want, err_msg=l.name)
        o[4].fill_(float("nan"))
    s.capture(2, timed=False)
    s.replay()
    torch.cuda.synchronize()
    for o, (l, x, w, b) in zip(ops, refs):
        want = oracle_lib.conv2d(x, w, b, l.stride, l.pad, l.groups, l.relu)
        np.testing.assert_array_equal(o[4].cpu().numpy(), want, err_msg=l.name)
    s.close()


def test_stack_resnet_b1_random_within_gate(oracle_lib):
    """The ResNet-50 batch-1 stack (packed 3x3 filters, split reductions) on
    its seeded random layers: e = max|y - y_ref| / max|y_ref| <= 1e-4."""
    ops, refs = [], []
    for i, l in enumerate(wl.workload(2).layers):
        x, w, b = wl.layer_tensors(2, i, l)
        P, Q = miconv.out_dims(l.H, l.W, l.R, l.S, l.stride, l.pad)
        y = torch.empty((l.N, l.K, P, Q), device="cuda")
        ops.append((miconv.OP_CONV_F32, torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda(),
                    torch.from_numpy(b).cuda(), y, l.stride, l.pad, l.groups, l.relu))
        refs.append((l, x, w, b))
    s = miconv.Stack(ops)
    s.capture(1, timed=False)
    s.replay()
    torch.cuda.synchronize()
    for o, (l, x, w, b) in zip(ops, refs):
        want = oracle_lib.conv2d(x, w, b, l.stride, l.pad, l.groups, l.relu)
        got = o[4].cpu().numpy()
        e = np.max(np.abs(got.astype(np.float64) - want)) / np.max(np.abs(want))
        assert e <= 1e-4, (l.name, e)
    s.close()


RAGGED = [  # (N, C, H, W, K, R, S, stride, pad, groups): small layers that take the wave kernel
    (1, 24, 11, 11, 40, 3, 3, 1, 1, 1),    # K % 32 != 0, N*P*Q % 32 != 0
    (1, 5, 9, 7, 7, 1, 1, 1, 0, 1),        # reduction of 5 taps (< one 8-tap block)
    (1, 16, 13, 13, 33, 3, 3, 2, 1, 1),    # stride 2, K = 33
    (1, 32, 10, 10, 48, 3, 3, 1, 1, 2),    # two groups of 16 -> 24
    (2, 12, 8, 8, 20, 5, 5, 1, 2, 1),      # 5x5, two images, reduction 300
    (1, 64, 7, 7, 96, 1, 1, 1, 0, 1),
    (1, 512, 7, 7, 64, 3, 3, 1, 1, 1),     # long reduction: split across work-groups
    (1, 256, 7, 7, 40, 3, 3, 1, 1, 2),     # split, two groups of 20 filters
    (1, 1024, 5, 5, 33, 1, 1, 1, 0, 1),    # split, 25 pixels, K = 33
    (1, 300, 9, 9, 70, 3, 3, 1, 1, 1),     # split, reduction order (c, r, s)
]
SPLIT = RAGGED[-4:]


def test_stack_wave_packed_filters_ragged(oracle_lib):
    """Wave-kernel layers in a stack read filters packed once in the kernel's
    operand order (zero-padded blocks of 32 filters x 8 taps): exact against
    the oracle on small integers for ragged filter counts, reductions, groups
    and strides, eager and replayed; the last four split their reduction
    across work-groups (a reduce launch sums the partials)."""
    ops, refs = [], []
    for i, (N, C, H, W, K, R, S, st, pad, g) in enumerate(RAGGED):
        x = wl.small_ints((N, C, H, W), -3, 3, 900 + i)
        w = wl.small_ints((K, C // g, R, S), -3, 3, 950 + i)
        b = wl.small_ints((K,), -8, 8, 990 + i)
        P, Q = miconv.out_dims(H, W, R, S, st, pad)
        y = torch.full((N, K, P, Q), float("nan"), device="cuda")
        ops.append((miconv.OP_CONV_F32, torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda(),
                    torch.from_numpy(b).cuda(), y, st, pad, g, i % 2 == 0))
        refs.append((x, w, b, st, pad, g, i % 2 == 0))
    s = miconv.Stack(ops)
    names = [s.describe(j) for j in range(len(ops))]
    assert all(n.startswith("igemm_wave_f32_kernel") for n in names), names
    assert not any("pack_wave" in n for n in names), names   # packed once, at stack creation
    for shape, n in zip(RAGGED, names):
        assert ("splitk_reduce" in n) == (shape in SPLIT), (shape, n)
    for replay in (False, True):
        if replay:
            for o in ops:
                o[4].fill_(float("nan"))
            s.capture(2, timed=False)
            s.replay()
        else:
            s.launch()
        torch.cuda.synchronize()
        for o, (x, w, b, st, pad, g, relu), shape in zip(ops, refs, RAGGED):
            want = oracle_lib.conv2d(x, w, b, st, pad, g, relu)
            np.testing.assert_array_equal(o[4].cpu().numpy(), want, err_msg=f"{shape} replay={replay}")
    s.close()


def test_stack_split_replays_bitwise(oracle_lib):
    """ResNet-50 batch-1 layers whose reductions are split across 2-9
    work-groups: the partials are summed in split order, so an eager pass and
    three replays of a graph holding three passes (eager work and
    synchronisation between them) give the same bits; and they meet the
    1e-4 gate."""
    idxs = [12, 25, 28, 43, 44, 46]
    ops, refs = [], []
    for i in idxs:
        l = wl.workload(2).layers[i]
        x, w, b = wl.layer_tensors(2, i, l)
        P, Q = miconv.out_dims(l.H, l.W, l.R, l.S, l.stride, l.pad)
        y = torch.full((l.N, l.K, P, Q), float("nan"), device="cuda")
        ops.append((miconv.OP_CONV_F32, torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda(),
                    torch.from_numpy(b).cuda(), y, l.stride, l.pad, l.groups, l.relu))
        refs.append((l, x, w, b))
    s = miconv.Stack(ops)
    assert s.launches == 2 * len(ops), [s.describe(j) for j in range(len(ops))]   # conv + reduce
    s.launch()
    torch.cuda.synchronize()
    first = [o[4].clone() for o in ops]
    for o, (l, x, w, b) in zip(ops, refs):
        want = oracle_lib.conv2d(x, w, b, l.stride, l.pad, l.groups, l.relu)
        got = o[4].cpu().numpy().astype(np.float64)
        assert np.max(np.abs(got - want)) / np.max(np.abs(want)) <= 1e-4, l.name
    s.capture(3, timed=False)
    for rep in range(3):
        for o in ops:
            o[4].fill_(float("nan"))
        torch.cuda.synchronize()
        s.replay()
        torch.cuda.synchronize()
        for o, f, (l, *_r) in zip(ops, first, refs):
            assert torch.equal(o[4], f), (l.name, rep)
    s.close()
