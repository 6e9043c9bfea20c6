"""GPU: whole-network passes (paper_1907_02154_amd.networks) against the oracle.

Each configuration's bench times every layer on its own seeded input; here
the layers are chained as the networks run them (ResNet-50: stem, max-pool,
bottleneck blocks whose last conv joins the shortcut; MobileNet: the 27
layers in sequence), from one seeded input.

* Gate, per layer, on identical inputs: the oracle is fed the exact tensors
  the GPU layer read (its input and, for a join, its shortcut), on sampled
  images, and the layer's output must meet the configuration's tolerance
  (1e-4 fp32, 2e-2 bf16); pools must match bit for bit.
* Report, not gated: an oracle chain from the same input, each oracle layer
  fed the oracle's own previous output; the drift between the two chains,
  layer by layer, is printed as JSON (ResNet-50 keeps it within a few bf16
  steps).  The test asserts only that it stays finite and small.
"""
import json

import numpy as np
import pytest
import torch

from paper_1907_02154_amd import miconv
from paper_1907_02154_amd import networks as nets
from paper_1907_02154_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    miconv.lib()


def bf(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)


def bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def e_inf(y, ref):
    y, ref = np.asarray(y, np.float64), np.asarray(ref, np.float64)
    s = np.max(np.abs(ref))
    return float(np.max(np.abs(y - ref)) / s) if s > 0 else float(np.max(np.abs(y)))


def _params(graph, config, bf16):
    host, dev = {}, {}
    for node in graph:
        if node.kind != "conv":
            continue
        _, w, b = wl.layer_tensors(config, node.index, node.layer)
        if bf16:
            w = wl.to_bf16_bits(w)
            dev[node.name] = (bf(w), torch.from_numpy(b).cuda())
        else:
            dev[node.name] = (torch.from_numpy(w).cuda(), torch.from_numpy(b).cuda())
        host[node.name] = (w, b)
    return host, dev


def _run(graph, config, layout, batch=None):
    bf16 = layout == "bf16_cl"
    x0, _, _ = wl.layer_tensors(config, 0, wl.workload(config, batch).layers[0])
    host, dev = _params(graph, config, bf16)
    tx = bf(wl.to_bf16_bits(x0)) if bf16 else torch.from_numpy(x0).cuda()
    ops, outs = nets.build_stack(graph, tx, dev, layout)
    s = miconv.Stack(ops)
    s.launch()
    torch.cuda.synchronize()
    return s, x0, host, outs


def _host_nchw(t, bf16):
    """A node's GPU output as host NCHW: bf16 bits for a channel-last tensor."""
    if bf16:
        return np.ascontiguousarray(np.transpose(bits(t), (0, 3, 1, 2)))
    return t.cpu().numpy()


def _f32(a, bf16, oracle_lib):
    return oracle_lib.bf16_to_f32(a) if bf16 else a


def _oracle_node(oracle_lib, node, x, res, host, bf16):
    """One node on the oracle, NCHW in and out (bf16 bits for channel-last)."""
    if node.kind == "maxpool":
        R, S, st, pad = node.pool
        if bf16:
            nhwc = np.ascontiguousarray(np.transpose(x, (0, 2, 3, 1)))
            y = oracle_lib.maxpool2d_bf16_cl(nhwc, R, S, st, pad)
            return np.ascontiguousarray(np.transpose(y, (0, 3, 1, 2)))
        return oracle_lib.maxpool2d(x, R, S, st, pad)
    l = node.layer
    w, b = host[node.name]
    if bf16:
        nhwc = np.ascontiguousarray(np.transpose(x, (0, 2, 3, 1)))
        r = None if res is None else np.ascontiguousarray(np.transpose(res, (0, 2, 3, 1)))
        y = oracle_lib.conv2d_bf16_cl(nhwc, w, b, l.stride, l.pad, l.groups, node.relu, r)
        return np.ascontiguousarray(np.transpose(y, (0, 3, 1, 2)))
    if l.kind == "dw":
        return oracle_lib.dwconv2d(x, w, b, l.stride, l.pad, node.relu)
    return oracle_lib.conv2d(x, w, b, l.stride, l.pad, l.groups, node.relu, res=res)


def _check_chain(oracle_lib, graph, config, layout, images, tol, batch=None):
    bf16 = layout == "bf16_cl"
    s, x0, host, outs = _run(graph, config, layout, batch)
    x0h = wl.to_bf16_bits(x0) if bf16 else x0
    sel = sorted(set(images) | {0})                  # images copied back; row j is image sel[j]
    rows = {n: j for j, n in enumerate(sel)}
    gpu = {k: _host_nchw(v[sel], bf16) for k, v in outs.items() if k != "input"}
    gpu["input"] = x0h[sel]
    # gate: each layer on the GPU's own inputs
    for node in graph:
        for n in images:
            j = rows[n]
            res = None if node.res is None else gpu[node.res][j:j + 1]
            ref = _oracle_node(oracle_lib, node, gpu[node.src][j:j + 1], res, host, bf16)
            got = gpu[node.name][j:j + 1]
            if node.kind == "maxpool":
                np.testing.assert_array_equal(got, ref, err_msg=node.name)
            else:
                e = e_inf(_f32(got, bf16, oracle_lib), _f32(ref, bf16, oracle_lib))
                assert e <= tol, f"{node.name} image {n}: e={e:.3e}"
    # report: the oracle's own chain from the same input (image 0)
    j0 = rows[0]
    drift, cur = [], {"input": x0h[:1]}
    for node in graph:
        res = None if node.res is None else cur[node.res]
        cur[node.name] = _oracle_node(oracle_lib, node, cur[node.src], res, host, bf16)
        e = e_inf(_f32(gpu[node.name][j0:j0 + 1], bf16, oracle_lib), _f32(cur[node.name], bf16, oracle_lib))
        drift.append((node.name, e))
    print(json.dumps({"chain": f"config {config} {layout}", "drift": [[n, round(e, 6)] for n, e in drift]}))
    assert all(np.isfinite(e) for _, e in drift)
    return s, outs, drift


def test_resnet50_b64_bf16_channel_last_chain(oracle_lib):
    """ResNet-50 at batch 64 with bf16 channel-last activations: per-layer
    gate 2e-2 on images 0 and 63; the stack's graph replays (projection
    shortcuts overlapped, or not) equal its eager pass bit for bit."""
    graph = nets.resnet50_graph(5)
    s, outs, drift = _check_chain(oracle_lib, graph, 5, "bf16_cl", images=[0, 63], tol=2e-2)
    assert drift[-1][1] < 0.2, drift[-1]
    _replays_match_eager(s, outs, graph)
    s.close()


def _replays_match_eager(s, outs, graph):
    """Graph replays of the pass -- with the four projection shortcuts on the
    second stream, and all in one stream -- reproduce the eager pass bit for
    bit, every node's output."""
    eager = {k: v.clone() for k, v in outs.items()}
    for overlap in (True, False):
        n_side = s.overlap(overlap)
        assert n_side == (4 if overlap else 0), n_side
        s.capture(2, timed=False)
        for rep in range(2):
            for k, v in outs.items():
                if k != "input":
                    v.fill_(float("nan"))
            torch.cuda.synchronize()
            s.replay()
            torch.cuda.synchronize()
            for k, v in outs.items():
                assert torch.equal(v, eager[k]), f"overlap={overlap} replay {rep} node {k}"


def test_resnet50_b1_f32_chain(oracle_lib):
    """ResNet-50 at batch 1, fp32 NCHW: stem, max-pool, bottlenecks with the
    join fused into each block's last conv; per-layer gate 1e-4."""
    graph = nets.resnet50_graph(2)
    s, outs, drift = _check_chain(oracle_lib, graph, 2, "f32", images=[0], tol=1e-4)
    assert drift[-1][1] < 1e-3, drift[-1]
    _replays_match_eager(s, outs, graph)
    s.close()


def test_mobilenet_b1_f32_chain(oracle_lib):
    """MobileNet-v1 at batch 1, fp32: the 27 layers in sequence; gate 1e-4."""
    graph = nets.mobilenet_graph()
    s, _, drift = _check_chain(oracle_lib, graph, 3, "f32", images=[0], tol=1e-4)
    assert drift[-1][1] < 1e-3, drift[-1]
    assert s.overlap(True) == 0          # a chain: nothing can overlap
    s.close()
