"""Whole-network passes of the evaluated models as one stack of layers.

The configurations time every conv layer on its own seeded input.  A network
pass instead feeds each layer the output of the layers before it, with the
glue the models need between convs (ResNet's stem max-pool, the shortcut join
of every bottleneck block, here fused into the last conv of the block).  This
module only wires tensors: ``*_graph`` lists the nodes of a network (which
node feeds which, where the shortcut comes from), and ``build_stack``
allocates the activations and returns the layer tuples of a
``miconv.Stack`` for that graph.  No arithmetic happens here.

Layouts:
  * ``"f32"``: fp32 NCHW activations (the batch-1 configurations);
  * ``"bf16_cl"``: bf16 channel-last activations [N][H][W][C] between layers
    (the graph-level layout choice of Sec. 3.2.3): the stem reads the NCHW
    bf16 image and writes channel-last, every later conv reads and writes
    channel-last bf16, the join included.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List, Optional

import torch

from . import miconv
from . import workloads as wl


@dataclass
class Node:
    name: str
    kind: str                      # "conv" or "maxpool"
    src: str                       # name of the node whose output this node reads ("input": x0)
    layer: Optional[wl.ConvLayer] = None   # conv: shape, stride, padding
    index: int = -1                # conv: index of the layer in its workload (its seeds)
    res: Optional[str] = None      # conv: node whose output is joined before the activation
    relu: bool = True
    pool: tuple = ()               # maxpool: (R, S, stride, pad)


def resnet50_graph(config: int = 5, batch: Optional[int] = None) -> List[Node]:
    """ResNet-50 v1 (the layer table of configs 2 and 5): stem conv, 3x3/2
    max-pool with padding 1, then bottleneck blocks c1 -> c2 -> c3 whose c3
    joins the shortcut (the block input, or its 1x1 projection in the first
    block of a stage) before the ReLU."""
    layers = wl.workload(config, batch).layers
    idx = {l.name: i for i, l in enumerate(layers)}
    g = [Node("stem", "conv", "input", layers[0], 0, relu=True),
         Node("pool", "maxpool", "stem", pool=(3, 3, 2, 1))]
    prev = "pool"
    for stage, blocks in (("s2", 3), ("s3", 4), ("s4", 6), ("s5", 3)):
        for b in range(blocks):
            p = f"{stage}b{b}"
            short = prev
            if b == 0:
                g.append(Node(p + "proj", "conv", prev, layers[idx[p + "proj"]], idx[p + "proj"], relu=False))
                short = p + "proj"
            g.append(Node(p + "c1", "conv", prev, layers[idx[p + "c1"]], idx[p + "c1"], relu=True))
            g.append(Node(p + "c2", "conv", p + "c1", layers[idx[p + "c2"]], idx[p + "c2"], relu=True))
            g.append(Node(p + "c3", "conv", p + "c2", layers[idx[p + "c3"]], idx[p + "c3"], res=short,
                          relu=True))
            prev = p + "c3"
    return g


def mobilenet_graph(batch: Optional[int] = None) -> List[Node]:
    """MobileNet-v1 (config 3): the layers in sequence, bias + ReLU after each."""
    layers = wl.workload(3, batch).layers
    g, prev = [], "input"
    for i, l in enumerate(layers):
        g.append(Node(l.name, "conv", prev, l, i, relu=l.relu))
        prev = l.name
    return g


def _out_shape(node: Node, in_shape, cl: bool):
    """Output extents (N, C_or_K, P, Q) of a node from its input (N, C, H, W)."""
    N, C, H, W = in_shape
    if node.kind == "maxpool":
        R, S, st, pad = node.pool
        P, Q = miconv.out_dims(H, W, R, S, st, pad)
        return (N, C, P, Q)
    l = node.layer
    P, Q = miconv.out_dims(H, W, l.R, l.S, l.stride, l.pad)
    return (N, l.K, P, Q)


def build_stack(graph: List[Node], x0: torch.Tensor, params: Dict[str, tuple], layout: str):
    """Layer tuples of a miconv.Stack running `graph` on x0, and the output
    tensor of every node (name -> tensor; channel-last tensors are
    [N][H][W][C]).  params[name] = (w, bias) device tensors of each conv.
    x0: fp32 NCHW ("f32") or bf16 NCHW ("bf16_cl")."""
    if layout not in ("f32", "bf16_cl"):
        raise ValueError(f"layout must be 'f32' or 'bf16_cl', got {layout!r}")
    cl = layout == "bf16_cl"
    dev = x0.device
    shapes = {"input": tuple(x0.shape)}
    outs = {"input": x0}
    ops = []
    for node in graph:
        shp = _out_shape(node, shapes[node.src], cl)
        shapes[node.name] = shp
        N, K, P, Q = shp
        if cl:
            y = torch.empty((N, P, Q, K), device=dev, dtype=torch.bfloat16)
        else:
            y = torch.empty((N, K, P, Q), device=dev, dtype=torch.float32)
        outs[node.name] = y
        x = outs[node.src]
        if node.kind == "maxpool":
            R, S, st, pad = node.pool
            ops.append(("maxpool", x, y, R, S, st, pad))
            continue
        l = node.layer
        w, b = params[node.name]
        res = outs[node.res] if node.res else None
        if cl:
            lay = miconv.LAYOUT_Y_NHWC_BF16 | (0 if node.src == "input" else miconv.LAYOUT_X_NHWC)
            ops.append((miconv.OP_CONV_BF16, x, w, b, y, l.stride, l.pad, l.groups, node.relu, res, lay))
        else:
            op = miconv.OP_DWCONV_F32 if l.kind == "dw" else miconv.OP_CONV_F32
            ops.append((op, x, w, b, y, l.stride, l.pad, l.groups, node.relu, res))
    return ops, outs
