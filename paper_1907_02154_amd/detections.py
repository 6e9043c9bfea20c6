"""Seeded synthetic inputs for the vision operators (Sec. 3.1.1): decoded
detector output rows, segmented key arrays and scan inputs.

Like ``workloads``, this module is shared by the product side (bench, GPU
tests) and the oracle's tests, and holds none of the operators' arithmetic:
only shapes, seeds and random draws.

Detection rows stand in for the decoded output of an SSD-style detector on a
512x512 image (the paper evaluates SSD_MobileNet1.0 and SSD_ResNet50 in
Sec. 4.3): one row per anchor of a multi-scale anchor grid (feature maps
64, 32, 16, 8, 4, 2, 1 cells per side with 4, 6, 6, 6, 6, 4, 4 anchors per
cell: 24564 rows), each row [class id, score, x1, y1, x2, y2] with
image-normalised corners.  Most rows are background with scores of a few
thousandths; about 2% cluster around a dozen objects per image (jittered
copies of the object's box, its class, scores in (0.05, 0.95) quantised to
1/512 so that equal scores occur), which is what makes suppression happen.
"""
from __future__ import annotations

import numpy as np

SEED_BASE = 1907021540

FEATURE_MAPS = (64, 32, 16, 8, 4, 2, 1)
ANCHORS_PER_CELL = (4, 6, 6, 6, 6, 4, 4)


def anchor_rows() -> int:
    """Rows of the anchor grid above: sum over feature maps of cells x anchors."""
    return sum(f * f * a for f, a in zip(FEATURE_MAPS, ANCHORS_PER_CELL))


def detection_rows(batch: int, num: int = None, classes: int = 20, objects: int = 12, seed: int = 0,
                   object_frac: float = 0.02) -> np.ndarray:
    """fp32 [batch][num][6] rows [class, score, x1, y1, x2, y2]."""
    num = anchor_rows() if num is None else num
    rng = np.random.default_rng(SEED_BASE + seed)
    out = np.empty((batch, num, 6), np.float32)
    for b in range(batch):
        # background: random boxes, low scores
        cxy = rng.uniform(0, 1, size=(num, 2))
        wh = rng.uniform(0.02, 0.4, size=(num, 2))
        cls = rng.integers(0, classes, size=num)
        score = rng.exponential(0.004, size=num)
        # objects: jittered copies of a few boxes
        gc = rng.uniform(0.1, 0.9, size=(objects, 2))
        gwh = rng.uniform(0.05, 0.5, size=(objects, 2))
        gcls = rng.integers(0, classes, size=objects)
        hit = np.nonzero(rng.uniform(0, 1, size=num) < object_frac)[0]
        g = rng.integers(0, objects, size=hit.size)
        cxy[hit] = gc[g] + rng.normal(0, 0.08, size=(hit.size, 2)) * gwh[g]
        wh[hit] = gwh[g] * rng.uniform(0.8, 1.25, size=(hit.size, 2))
        cls[hit] = gcls[g]
        score[hit] = np.round(rng.uniform(0.05, 0.95, size=hit.size) * 512) / 512
        out[b, :, 0] = cls
        out[b, :, 1] = np.minimum(score, 0.999)
        out[b, :, 2:4] = cxy - wh / 2
        out[b, :, 4:6] = cxy + wh / 2
    return out


def segment_offsets(segments: int, n: int, seed: int = 0) -> np.ndarray:
    """int32 [segments + 1] offsets of `segments` consecutive segments
    covering [0, n): the interior cut points are n's positions drawn
    uniformly and sorted, so lengths vary (roughly exponentially, some
    empty)."""
    rng = np.random.default_rng(SEED_BASE + 7 + seed)
    cuts = np.sort(rng.integers(0, n + 1, size=segments - 1))
    return np.concatenate([[0], cuts, [n]]).astype(np.int32)


def keys(n: int, seed: int = 0, ties: bool = False) -> np.ndarray:
    """fp32 sort keys: standard normal, or small integers (many equal keys)."""
    rng = np.random.default_rng(SEED_BASE + 11 + seed)
    if ties:
        return rng.integers(-8, 8, size=n).astype(np.float32)
    return rng.standard_normal(n).astype(np.float32)


def scan_values(shape, lo: int = -1000, hi: int = 1000, seed: int = 0) -> np.ndarray:
    rng = np.random.default_rng(SEED_BASE + 13 + seed)
    return rng.integers(lo, hi, size=shape).astype(np.int32)
