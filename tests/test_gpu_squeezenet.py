"""GPU: SqueezeNet 1.0 fire modules (the paper's third model, Sec. 4.1).

A fire module is a 1x1 squeeze conv followed by a 1x1 and a 3x3 expand conv
whose outputs are concatenated along channels.  At batch 1 a channel range
of an NCHW tensor is one contiguous run of memory, so each expand conv writes
its half of the concatenation directly (a pointer into the joint output; no
copy kernel).  Small-integer data keep every sum exact: the chained GPU
module, run by single calls and by the stack executor (eager and replayed
graphs), must equal the oracle's chain bit for bit.  Every layer of the
network at full size is checked against the oracle in test_gpu_parity
(config 6).
"""
import numpy as np
import pytest
import torch

from paper_1907_02154_amd import miconv
from paper_1907_02154_amd import workloads as wl

pytestmark = pytest.mark.gpu

# (fire, input channels, squeeze channels, expand channels per branch, extent)
FIRES = [(2, 96, 16, 64, 54), (6, 256, 48, 192, 27), (9, 512, 64, 256, 13)]


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    miconv.lib()


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


@pytest.mark.parametrize("fire", FIRES, ids=lambda f: f"fire{f[0]}")
def test_fire_module_concat_small_ints(oracle_lib, fire):
    f, cin, sq, ex, e = fire
    s0 = 9100 + f * 10
    x = wl.small_ints((1, cin, e, e), 0, 3, s0)
    ws = wl.small_ints((sq, cin, 1, 1), -2, 2, s0 + 1)
    w1 = wl.small_ints((ex, sq, 1, 1), -2, 2, s0 + 2)
    w3 = wl.small_ints((ex, sq, 3, 3), -2, 2, s0 + 3)
    bs, b1, b3 = (wl.small_ints((k,), -8, 8, s0 + 4 + i) for i, k in enumerate((sq, ex, ex)))
    s_ref = oracle_lib.conv2d(x, ws, bs, 1, 0, 1, True)
    ref = np.concatenate([oracle_lib.conv2d(s_ref, w1, b1, 1, 0, 1, True),
                          oracle_lib.conv2d(s_ref, w3, b3, 1, 1, 1, True)], axis=1)

    tx, tws, tw1, tw3, tbs, tb1, tb3 = map(dev, (x, ws, w1, w3, bs, b1, b3))
    ts = torch.empty((1, sq, e, e), device="cuda")
    cat = torch.full((1, 2 * ex, e, e), float("nan"), device="cuda")
    lo, hi = cat[:, :ex], cat[:, ex:]
    assert lo.is_contiguous() and hi.is_contiguous() and hi.data_ptr() == cat.data_ptr() + 4 * ex * e * e

    miconv.conv2d_fwd(tx, tws, tbs, ts, 1, 0, 1, True)
    miconv.conv2d_fwd(ts, tw1, tb1, lo, 1, 0, 1, True)
    miconv.conv2d_fwd(ts, tw3, tb3, hi, 1, 1, 1, True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(cat.cpu().numpy(), ref, err_msg=f"fire{f} single calls")

    op = miconv.OP_CONV_F32
    st = miconv.Stack([(op, tx, tws, tbs, ts, 1, 0, 1, True),
                       (op, ts, tw1, tb1, lo, 1, 0, 1, True),
                       (op, ts, tw3, tb3, hi, 1, 1, 1, True)])
    st.capture(1, timed=False)
    for rep in range(2):
        cat.fill_(float("nan"))
        ts.fill_(float("nan"))
        torch.cuda.synchronize()
        st.replay()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(cat.cpu().numpy(), ref, err_msg=f"fire{f} replay {rep}")
    st.close()


def test_fire_module_concat_batch4_strided(oracle_lib):
    """At batch > 1 a channel range of the joint output is no longer one
    contiguous run: the expand convs write it through the output image
    stride (conv2d_fwd_ex, and stack layers whose y is such a view)."""
    f, cin, sq, ex, e = 6, 256, 48, 192, 27
    N, s0 = 4, 9500
    x = wl.small_ints((N, cin, e, e), 0, 3, s0)
    ws = wl.small_ints((sq, cin, 1, 1), -2, 2, s0 + 1)
    w1 = wl.small_ints((ex, sq, 1, 1), -2, 2, s0 + 2)
    w3 = wl.small_ints((ex, sq, 3, 3), -2, 2, s0 + 3)
    bs, b1, b3 = (wl.small_ints((k,), -8, 8, s0 + 4 + i) for i, k in enumerate((sq, ex, ex)))
    s_ref = oracle_lib.conv2d(x, ws, bs, 1, 0, 1, True)
    ref = np.concatenate([oracle_lib.conv2d(s_ref, w1, b1, 1, 0, 1, True),
                          oracle_lib.conv2d(s_ref, w3, b3, 1, 1, 1, True)], axis=1)
    tx, tws, tw1, tw3, tbs, tb1, tb3 = map(dev, (x, ws, w1, w3, bs, b1, b3))
    ts = torch.empty((N, sq, e, e), device="cuda")
    cat = torch.full((N, 2 * ex, e, e), float("nan"), device="cuda")
    lo, hi = cat[:, :ex], cat[:, ex:]
    assert not lo.is_contiguous()
    miconv.conv2d_fwd(tx, tws, tbs, ts, 1, 0, 1, True)
    miconv.conv2d_fwd_ex(ts, tw1, tb1, lo, 1, 0, 1, True)
    miconv.conv2d_fwd_ex(ts, tw3, tb3, hi, 1, 1, 1, True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(cat.cpu().numpy(), ref)
    op = miconv.OP_CONV_F32
    st = miconv.Stack([(op, tx, tws, tbs, ts, 1, 0, 1, True),
                       (op, ts, tw1, tb1, lo, 1, 0, 1, True),
                       (op, ts, tw3, tb3, hi, 1, 1, 1, True)])
    cat.fill_(float("nan"))
    st.launch()
    torch.cuda.synchronize()
    np.testing.assert_array_equal(cat.cpu().numpy(), ref)
    st.close()
