"""GPU: conv2d_fwd_noalloc, conv2d_fwd_ws on the library's fixed per-GPU
scratch, against conv2d_fwd_ws on a caller workspace.

Both entry points resolve the same plan and run the same kernels, so on the
same inputs their outputs must agree bit for bit; both are also held to the
oracle's gate.  Each case runs twice in a row, the second call on a smaller
input, so the second call reads scratch the first one left behind.
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


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def dev_bf16_bits(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)


# (C, H, W, K, R, S, stride, pad, dtype, batch of the first call, of the second)
CASES = [
    (512, 7, 7, 512, 3, 3, 1, 1, "f32", 1, 1),        # split reduction, partials in scratch
    (1024, 14, 14, 256, 1, 1, 1, 0, "f32", 2, 1),     # split 1x1
    (64, 28, 28, 64, 3, 3, 1, 1, "bf16", 8, 3),       # channel-last copy + KRSC filters in scratch
    (256, 14, 14, 128, 1, 1, 2, 0, "bf16", 16, 5),    # sampled channel-last copy
    (3, 224, 224, 64, 7, 7, 2, 3, "bf16", 4, 1),      # stem: tap-pair filters packed per call
]


def _data(case, N, seed):
    C, H, W, K, R, S, st, pad, dt = case[:9]
    x = wl.uniform01((N, C, H, W), seed)
    w = wl.normal((K, C, R, S), np.sqrt(2.0 / (C * R * S)), seed + 1)
    b = wl.normal((K,), 0.01, seed + 2)
    if dt == "bf16":
        x, w = wl.to_bf16_bits(x), wl.to_bf16_bits(w)
        return x, w, b, dev_bf16_bits(x), dev_bf16_bits(w)
    return x, w, b, dev(x), dev(w)


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c[:8])) + "-" + c[8])
def test_noalloc_matches_workspace_entry_point(oracle_lib, case):
    C, H, W, K, R, S, st, pad, dt, n1, n2 = case
    for j, N in enumerate((n1, n2)):
        need = miconv.conv2d_workspace_bytes(N, C, H, W, K, R, S, st, pad, 1, dt)
        assert 0 < need <= miconv.NOALLOC_SCRATCH_BYTES, need
        x, w, b, tx, tw = _data(case, N, 9100 + 10 * j + sum(case[:8]))
        P, Q = miconv.out_dims(H, W, R, S, st, pad)
        y_ws = torch.full((N, K, P, Q), float("nan"), device="cuda")
        y_na = torch.full((N, K, P, Q), float("nan"), device="cuda")
        miconv.conv2d_fwd_ws(tx, tw, dev(b), y_ws, st, pad, 1, True)
        miconv.conv2d_fwd_noalloc(tx, tw, dev(b), y_na, st, pad, 1, True)
        torch.cuda.synchronize()
        assert torch.equal(y_na, y_ws), f"call {j}: batch {N}"
        f = oracle_lib.conv2d_bf16 if dt == "bf16" else oracle_lib.conv2d
        ref = f(x[:1], w, b, st, pad, 1, True)
        got = y_na[:1].cpu().numpy()
        e = np.max(np.abs(got - ref)) / np.max(np.abs(ref))
        assert e <= (2e-2 if dt == "bf16" else 1e-4), (j, e)


def test_noalloc_residual_and_graph_replay(oracle_lib):
    """A split layer with the residual joined, captured into a HIP graph and
    replayed with eager calls on the same scratch between the replays: every
    replay equals the workspace entry point's output."""
    C, H, W, K = 512, 7, 7, 512
    x = wl.uniform01((1, C, H, W), 9300)
    w = wl.normal((K, C, 3, 3), np.sqrt(2.0 / (C * 9)), 9301)
    b = wl.normal((K,), 0.01, 9302)
    res = wl.normal((1, K, H, W), 1.0, 9303)
    tx, tw, tb, tr = dev(x), dev(w), dev(b), dev(res)
    want = torch.empty((1, K, H, W), device="cuda")
    miconv.conv2d_fwd_ws(tx, tw, tb, want, 1, 1, 1, True, res=tr)
    y = torch.empty_like(want)
    # another split layer that also uses the scratch, eagerly, between replays
    ox = dev(wl.uniform01((2, 1024, 14, 14), 9310))
    ow = dev(wl.normal((256, 1024, 1, 1), np.sqrt(2.0 / 1024), 9311))
    oy = torch.empty((2, 256, 14, 14), device="cuda")
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    with torch.cuda.graph(g, stream=side):
        miconv.conv2d_fwd_noalloc(tx, tw, tb, y, 1, 1, 1, True, res=tr, stream=side)
    for rep in range(3):
        y.fill_(float("nan"))
        miconv.conv2d_fwd_noalloc(ox, ow, None, oy, 1, 0, 1, False)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, want), f"replay {rep}"
    ref = oracle_lib.conv2d(x, w, b, 1, 1, 1, True, res=res)
    assert np.max(np.abs(y.cpu().numpy() - ref)) / np.max(np.abs(ref)) <= 1e-4


def test_noalloc_rejects_plans_beyond_the_scratch():
    """A bf16 3x3 layer at batch 128 on 56 x 56 planes stages a 51 MB
    channel-last copy of x: more than the fixed scratch, so the call fails and
    writes nothing."""
    N, C, H, W, K = 128, 64, 56, 56, 64
    assert miconv.conv2d_workspace_bytes(N, C, H, W, K, 3, 3, 1, 1, 1, "bf16") > miconv.NOALLOC_SCRATCH_BYTES
    x = torch.zeros((N, C, H, W), device="cuda", dtype=torch.bfloat16)
    w = torch.zeros((K, C, 3, 3), device="cuda", dtype=torch.bfloat16)
    y = torch.full((N, K, H, W), float("nan"), device="cuda")
    with pytest.raises(miconv.MiconvError) as e:
        miconv.conv2d_fwd_noalloc(x, w, None, y, 1, 1, 1, True)
    assert e.value.status == miconv.ERR_WORKSPACE
    torch.cuda.synchronize()
    assert torch.isnan(y).all()
