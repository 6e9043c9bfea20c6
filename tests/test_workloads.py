"""Layer tables of the evaluated networks: counts, chaining and FLOP totals.

ResNet50_v1, MobileNet1.0 and SqueezeNet1.0 are the classification models of
the paper's evaluation (Sec. 4.1); VGG-16 is an extra dense stack.
The FLOP totals are the standard per-network conv counts at 224x224
(2 FLOP per multiply-add).
"""
import pytest

from paper_1907_02154_amd import workloads as wl


def _out(oracle_lib, l):
    return oracle_lib.out_dims(l.H, l.W, l.R, l.S, l.stride, l.pad)


@pytest.mark.parametrize("config,count,gflop", [(1, 1, 0.2312), (2, 53, 7.7123), (3, 27, 1.13543),
                                                (4, 13, 245.546), (5, 53, 493.59)])
def test_counts_and_flops(oracle_lib, config, count, gflop):
    w = wl.workload(config)
    assert len(w.layers) == count
    total = sum(wl.flops(l, *_out(oracle_lib, l)) for l in w.layers)
    assert abs(total / 1e9 - gflop) / gflop < 2e-4, total


def test_resnet_chaining(oracle_lib):
    L = wl.workload(2).layers
    by = {l.name: l for l in L}
    P, Q = _out(oracle_lib, by["stem"])
    assert (P, Q) == (112, 112)
    # 3x3/2 pad-1 max-pool after the stem
    assert oracle_lib.out_dims(112, 112, 3, 3, 2, 1) == (56, 56)
    prev_out = None
    for l in L[1:]:
        if l.name.endswith("c1"):
            if prev_out is not None:
                assert (l.C, l.H) == prev_out, l.name
        if l.name.endswith("c2") or l.name.endswith("c3"):
            assert (l.C, l.H) == prev, l.name
        P, Q = _out(oracle_lib, l)
        if l.name.endswith("c3"):
            prev_out = (l.K, P)
        if l.name.endswith("proj"):
            assert (l.K, P) == prev_out, l.name
        prev = (l.K, P)


def test_mobilenet_chaining(oracle_lib):
    L = wl.workload(3).layers
    c, h = 3, 224
    for l in L:
        assert (l.C, l.H) == (c, h), l.name
        P, Q = _out(oracle_lib, l)
        c, h = l.K, P
        if l.kind == "dw":
            assert l.groups == l.C == l.K
    assert (c, h) == (1024, 7)


def test_vgg_chaining(oracle_lib):
    L = wl.workload(4).layers
    c, h = 3, 224
    for l in L:
        if l.H != h:       # a 2x2/2 pool sits between stages
            assert l.H == oracle_lib.out_dims(h, h, 2, 2, 2, 0)[0], l.name
            h = l.H
        assert l.C == c, l.name
        P, _ = _out(oracle_lib, l)
        c, h = l.K, P
    assert (c, h) == (512, 14)


def test_seeded_inputs_are_deterministic():
    l = wl.workload(1).layers[0]
    x1, w1, b1 = wl.layer_tensors(1, 0, l)
    x2, w2, b2 = wl.layer_tensors(1, 0, l)
    assert (x1 == x2).all() and (w1 == w2).all() and (b1 == b2).all()
    assert x1.min() >= 0 and x1.max() < 1
    assert abs(w1.std() - (2 / 576) ** 0.5) < 0.01 * (2 / 576) ** 0.5 * 10


def test_squeezenet_table(oracle_lib):
    """SqueezeNet 1.0: 26 convs; 0.82 G multiply-adds at 224x224 (the figure
    published for the model); fire modules chain through 3x3/2 ceil-mode
    pools (109 -> 54 -> 27 -> 13); each fire's expand branches read its
    squeeze output and concatenate to the next fire's input channels."""
    L = wl.workload(6).layers
    assert len(L) == 26
    macs = sum(wl.flops(l, *_out(oracle_lib, l)) for l in L) / 2
    assert abs(macs / 0.82e9 - 1) < 0.01, macs
    assert _out(oracle_lib, L[0]) == (109, 109)
    pool = lambda h: -(-(h - 3) // 2) + 1          # 3x3/2, ceil mode
    c, h = L[0].K, _out(oracle_lib, L[0])[0]
    for f in range(8):
        sq, e1, e3 = L[1 + 3 * f: 4 + 3 * f]
        if sq.H != h:
            assert sq.H == pool(h), sq.name
            h = sq.H
        assert (sq.C, sq.R) == (c, 1), sq.name
        assert (e1.C, e3.C, e1.R, e3.R, e3.pad) == (sq.K, sq.K, 1, 3, 1), e1.name
        assert e1.K == e3.K and _out(oracle_lib, e1) == _out(oracle_lib, e3) == (h, h)
        c = e1.K + e3.K
    assert (L[-1].C, L[-1].K, L[-1].H) == (c, 1000, h) == (512, 1000, 13)
