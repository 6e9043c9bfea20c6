"""Pins for the vision-operator oracle (runs without a GPU).

The oracle (oracle/vision.py) writes out segmented argsort, prefix sum and
box_nms (paper Sec. 3.1.1) from their definitions.  These tests tie it to
things other than itself:

* hand-worked examples (tests/golden/vision_examples.json);
* brute force: the rank of every element counted pairwise (argsort), the
  three-stage scan of Fig. 3 carried out step by step over simulated
  processors (prefix sum), and the two properties that single out greedy NMS
  (no two kept boxes of one class overlap above the threshold; every dropped
  candidate overlaps a kept box ranked before it), checked on random inputs;
* closed forms (scan of ones and of 0..n-1) and invariants (argsort returns a
  permutation per segment whose keys are ordered).
"""
import json
import os

import numpy as np
import pytest

GOLD = os.path.join(os.path.dirname(__file__), "golden", "vision_examples.json")


@pytest.fixture(scope="module")
def gold():
    with open(GOLD) as f:
        return json.load(f)


# ---------------------------------------------------------------- argsort

def test_argsort_hand_examples(oracle_lib, gold):
    for c in gold["argsort"]:
        got = oracle_lib.segmented_argsort(np.float32(c["keys"]), c["offsets"], c["descending"])
        assert got.tolist() == c["expect"], c


def _brute_ranks(keys, a, b, descending):
    """Position of each element of keys[a:b] in its segment's sorted order:
    the count of elements that go before it (strictly better key, or an equal
    key at a lower index)."""
    pos = {}
    for i in range(a, b):
        before = 0
        for j in range(a, b):
            better = keys[j] > keys[i] if descending else keys[j] < keys[i]
            if better or (keys[j] == keys[i] and j < i):
                before += 1
        pos[i - a] = before
    return pos


@pytest.mark.parametrize("descending", [True, False])
def test_argsort_brute_force_ranks(oracle_lib, descending):
    rng = np.random.default_rng(17 + descending)
    for trial in range(40):
        n = int(rng.integers(0, 40))
        cuts = np.sort(rng.integers(0, n + 1, size=int(rng.integers(0, 6))))
        off = np.concatenate([[0], cuts, [n]]).astype(np.int64)
        keys = rng.integers(-3, 4, size=n).astype(np.float32)     # many ties
        if trial % 3 == 0:
            keys = rng.standard_normal(n).astype(np.float32)
        got = oracle_lib.segmented_argsort(keys, off, descending)
        for s in range(off.size - 1):
            a, b = int(off[s]), int(off[s + 1])
            for local, p in _brute_ranks(keys, a, b, descending).items():
                assert got[a + p] == local, (trial, s, local)


def test_argsort_invariants(oracle_lib):
    rng = np.random.default_rng(5)
    keys = rng.standard_normal(5000).astype(np.float32)
    off = np.concatenate([[0], np.sort(rng.integers(0, 5000, 30)), [5000]])
    got = oracle_lib.segmented_argsort(keys, off)
    for s in range(off.size - 1):
        a, b = int(off[s]), int(off[s + 1])
        idx = got[a:b]
        assert sorted(idx.tolist()) == list(range(b - a))
        k = keys[a:b][idx]
        assert np.all(k[:-1] >= k[1:])


def test_argsort_rejects_bad_offsets(oracle_lib):
    with pytest.raises(ValueError):
        oracle_lib.segmented_argsort(np.zeros(4, np.float32), [0, 3, 2, 4])
    with pytest.raises(ValueError):
        oracle_lib.segmented_argsort(np.zeros(4, np.float32), [0, 3])


# ---------------------------------------------------------------- scan

def test_scan_hand_example(oracle_lib, gold):
    c = gold["scan"]
    assert oracle_lib.scan_inclusive_i32(c["x"]).tolist() == c["inclusive"]
    assert oracle_lib.scan_exclusive_i32(c["x"]).tolist() == [0] + c["inclusive"][:-1]


def _three_stage(x, procs, per):
    """Fig. 3 carried out literally: each processor scans its block
    sequentially (up-sweep), the block totals are scanned by Hillis-Steele
    passes (in pass d, total i adds total i - 2^d), and every processor adds
    the scanned total of the blocks before it (down-sweep)."""
    x = [int(v) for v in x]
    blocks = [x[p * per:(p + 1) * per] for p in range(procs)]
    local = []
    for blk in blocks:
        run, acc = [], 0
        for v in blk:
            acc += v
            run.append(acc)
        local.append(run)
    tot = [r[-1] if r else 0 for r in local]
    d = 1
    while d < procs:
        tot = [tot[i] + (tot[i - d] if i >= d else 0) for i in range(procs)]
        d *= 2
    out = []
    for p, run in enumerate(local):
        base = tot[p - 1] if p else 0
        out.extend(v + base for v in run)
    return out


def test_scan_three_stage_brute_force(oracle_lib):
    rng = np.random.default_rng(3)
    for n, procs in ((18, 5), (1, 1), (100, 7), (257, 16), (1000, 33)):
        per = -(-n // procs)
        x = rng.integers(-1000, 1000, size=n)
        assert oracle_lib.scan_inclusive_i32(x).tolist() == _three_stage(x, procs, per)


def test_scan_closed_forms(oracle_lib):
    n = 4097
    assert oracle_lib.scan_inclusive_i32(np.ones(n, np.int32)).tolist() == list(range(1, n + 1))
    i = np.arange(n)
    assert np.array_equal(oracle_lib.scan_inclusive_i32(i), i * (i + 1) // 2)
    assert np.array_equal(oracle_lib.scan_exclusive_i32(i), i * (i - 1) // 2)
    assert oracle_lib.scan_inclusive_i32([]).size == 0
    # fp32 scan of small integers is exact: equals the integer scan
    x = np.random.default_rng(9).integers(-50, 50, size=10000)
    assert np.array_equal(oracle_lib.scan_inclusive_f32(x.astype(np.float32)),
                          oracle_lib.scan_inclusive_i32(x).astype(np.float32))
    with pytest.raises(OverflowError):
        oracle_lib.scan_inclusive_i32([2 ** 30, 2 ** 30])


# ---------------------------------------------------------------- box_nms

def test_iou_hand_values(gold):
    from oracle.vision import _iou
    for c in gold["iou"]:
        a, b = np.float32(c["a"]), np.float32(c["b"])
        want = np.float32(np.float32(c["num"]) / np.float32(c["den"]))
        assert _iou(a, b) == want and _iou(b, a) == want, c


def test_nms_hand_examples(oracle_lib, gold):
    for c in gold["nms"]:
        d = np.float32(c["data"])
        out = oracle_lib.box_nms(d[None], c["overlap_thresh"], c["valid_thresh"], c["topk"],
                                 force_suppress=c["force_suppress"])[0]
        k = len(c["kept_rows"])
        np.testing.assert_array_equal(out[:k], d[c["kept_rows"]], err_msg=c["note"])
        assert np.all(out[k:] == -1), c["note"]


def test_nms_without_class_field(oracle_lib):
    # [score, x1, y1, x2, y2]; identical boxes, the lower score goes
    d = np.float32([[0.3, 0, 0, 2, 2], [0.8, 0, 0, 2, 2], [0.5, 5, 5, 6, 6]])
    out = oracle_lib.box_nms(d[None], 0.5, 0.0, -1, id_index=-1, score_index=0, coord_start=1)[0]
    np.testing.assert_array_equal(out, np.float32([d[1], d[2], [-1] * 5]))


def _rand_boxes(rng, B, N, classes):
    xy = rng.uniform(0, 20, size=(B, N, 2))
    wh = rng.uniform(1, 8, size=(B, N, 2))
    d = np.empty((B, N, 6), np.float32)
    d[..., 0] = rng.integers(0, classes, size=(B, N))
    d[..., 1] = np.round(rng.uniform(0, 1, size=(B, N)), 2)              # ties
    d[..., 2:4] = xy
    d[..., 4:6] = xy + wh
    return d


@pytest.mark.parametrize("force", [False, True])
def test_nms_greedy_properties(oracle_lib, force):
    """On random inputs the output is the unique list with the greedy NMS
    properties: kept rows are input rows in rank order, pairwise below the
    threshold within a class, and every dropped candidate (valid, within
    topk) overlaps above the threshold a kept row ranked before it."""
    from oracle.vision import _iou
    rng = np.random.default_rng(11 + force)
    thr, vth, topk = 0.45, 0.2, 25
    d = _rand_boxes(rng, 3, 40, 3)
    out = oracle_lib.box_nms(d, thr, vth, topk, force_suppress=force)
    for b in range(d.shape[0]):
        rows = [tuple(r) for r in d[b]]
        cand = sorted([i for i in range(40) if d[b, i, 1] > np.float32(vth)], key=lambda i: (-d[b, i, 1], i))
        cand = cand[:topk]
        kept = []
        for r in out[b]:
            if np.all(r == -1):
                continue
            kept.append(rows.index(tuple(r)))
        nk = len(kept)
        assert np.all(out[b, nk:] == -1)
        assert kept == [i for i in cand if i in kept]                    # rank order, candidates only
        same = lambda i, j: force or d[b, i, 0] == d[b, j, 0]           # noqa: E731
        for x in range(nk):
            for y in range(x + 1, nk):
                i, j = kept[x], kept[y]
                assert not (same(i, j) and _iou(d[b, i, 2:6], d[b, j, 2:6]) > np.float32(thr))
        for i in cand:
            if i in kept:
                continue
            earlier = [j for j in kept if cand.index(j) < cand.index(i)]
            assert any(same(i, j) and _iou(d[b, j, 2:6], d[b, i, 2:6]) > np.float32(thr) for j in earlier)
