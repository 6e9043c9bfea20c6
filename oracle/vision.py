"""CPU oracle for the paper's vision-specific operators (Sec. 3.1.1).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the bench's CPU
baseline may import this module; the product library never does.  Plain
numpy / Python, written from the operators' definitions:

* segmented argsort (Sec. 3.1.1, "Sorting"; Fig. 2): the rank order of the
  keys inside each segment of a flattened array, numpy.argsort semantics per
  segment (the footnote of that passage names numpy's argsort);
* prefix sum (Sec. 3.1.1, "Prefix sum"; Fig. 3): y[i] = x[0] + ... + x[i];
* box_nms (Sec. 3.1.1 names it; Sec. 4.3 describes the output convention:
  every output entry starts invalid): greedy non-maximum suppression.

Readings where the paper is silent (listed in the design notes):
* argsort order: descending keys for detection scores (ascending offered);
  equal keys keep their original order (stable), so the result is unique;
* box_nms: boxes are corner-encoded (x1, y1, x2, y2); IoU = intersection area
  / union area with widths max(0, .), evaluated in fp32 one operation at a
  time in the order written in ``_iou``, the suppression test is IoU >
  overlap_thresh; candidates are the boxes with score > valid_thresh, ranked
  by score (descending, stable), of which the first topk (all when topk < 0)
  take part; a candidate is suppressed by an earlier kept candidate of the
  same class (any class when force_suppress, or when there is no class
  field); kept boxes are written in rank order, every other output row is
  all -1.
"""
from __future__ import annotations

import numpy as np


# ---------------------------------------------------------------- argsort

def segmented_argsort(keys, seg_offsets, descending=True):
    """keys: fp32 [n]; seg_offsets: int [S + 1], seg_offsets[0] = 0,
    seg_offsets[S] = n, non-decreasing.  Returns int32 [n]: position
    seg_offsets[s] + r holds the index, local to segment s, of the element of
    rank r in that segment (ties: lower index first)."""
    keys = np.asarray(keys, np.float32)
    off = np.asarray(seg_offsets, np.int64)
    if off[0] != 0 or off[-1] != keys.size or np.any(np.diff(off) < 0):
        raise ValueError("bad segment offsets")
    out = np.empty(keys.size, np.int32)
    for s in range(off.size - 1):
        a, b = int(off[s]), int(off[s + 1])
        seg = keys[a:b].astype(np.float64)
        order = np.argsort(-seg if descending else seg, kind="stable")
        out[a:b] = order
    return out


# ---------------------------------------------------------------- scan

def scan_inclusive_i32(x):
    """y[i] = x[0] + ... + x[i], int32 (inputs chosen so no partial sum overflows)."""
    x = np.asarray(x, np.int64)
    y = np.cumsum(x)
    if y.size and (y.max() > 2 ** 31 - 1 or y.min() < -2 ** 31):
        raise OverflowError("partial sum outside int32")
    return y.astype(np.int32)


def scan_exclusive_i32(x):
    """y[i] = x[0] + ... + x[i-1], y[0] = 0."""
    y = scan_inclusive_i32(x)
    return np.concatenate([[0], y[:-1]]).astype(np.int32) if y.size else y


def scan_inclusive_f32(x):
    """y[i] = x[0] + ... + x[i] summed exactly (fp64 running sum of fp32
    values, exact for the test sizes' magnitudes up to its own rounding) and
    rounded once to fp32."""
    return np.cumsum(np.asarray(x, np.float64)).astype(np.float32)


# ---------------------------------------------------------------- box_nms

def _iou(a, b):
    """IoU of two corner-encoded boxes (fp32 arrays x1, y1, x2, y2), each
    operation rounded to fp32 in this order."""
    f = np.float32
    iw = f(max(f(0), f(min(a[2], b[2]) - max(a[0], b[0]))))
    ih = f(max(f(0), f(min(a[3], b[3]) - max(a[1], b[1]))))
    inter = f(iw * ih)
    area_a = f(f(max(f(0), f(a[2] - a[0]))) * f(max(f(0), f(a[3] - a[1]))))
    area_b = f(f(max(f(0), f(b[2] - b[0]))) * f(max(f(0), f(b[3] - b[1]))))
    union = f(f(area_a + area_b) - inter)
    if union <= 0:
        return f(0)
    return f(inter / union)


def box_nms(data, overlap_thresh=0.5, valid_thresh=0.0, topk=-1, id_index=0, score_index=1,
            coord_start=2, force_suppress=False):
    """data: fp32 [B][N][width]; per batch, greedy NMS as in the module
    docstring.  Returns fp32 [B][N][width]."""
    data = np.asarray(data, np.float32)
    B, N, width = data.shape
    out = np.full_like(data, -1.0)
    thr = np.float32(overlap_thresh)
    for b in range(B):
        d = data[b]
        cand = [i for i in range(N) if d[i, score_index] > np.float32(valid_thresh)]
        cand.sort(key=lambda i: -float(d[i, score_index]))      # stable: ties keep index order
        if topk >= 0:
            cand = cand[:topk]
        kept = []
        for i in cand:
            bi = d[i, coord_start:coord_start + 4]
            suppressed = False
            for j in kept:
                same = force_suppress or id_index < 0 or d[i, id_index] == d[j, id_index]
                if same and _iou(d[j, coord_start:coord_start + 4], bi) > thr:
                    suppressed = True
                    break
            if not suppressed:
                kept.append(i)
        for r, i in enumerate(kept):
            out[b, r] = d[i]
    return out
