"""Pins for the oracle's non-maximum suppression: facts that do not come from it.

  hand cases       kept lists derived by hand (tests/golden/nms_hand_cases.json): a chain
                   through a removed box, IoU equal to the threshold, categories, score
                   ties, NaN and signed-zero scores, zero-area boxes, max_keep
  IoU closed forms identical 1, disjoint 0, nested small/large, a half overlap, and
                   symmetry, on integer boxes where binary32 is exact
  characterization on random boxes the kept list is exactly the set that greedy NMS is
                   defined by: kept boxes come in rank order, no kept box overlaps a
                   higher-ranked kept box of its category by more than the threshold,
                   and every dropped box does (this determines the set uniquely); the
                   overlaps are computed here with numpy in binary32
"""
from __future__ import annotations

import json
import os

import numpy as np

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def pin_nms_hand_cases(lib):
    cases = json.load(open(os.path.join(GOLDEN, "nms_hand_cases.json")))["cases"]
    for case in cases:
        scores = np.array([float(s) for s in case["scores"]], np.float32)
        keep = oracle.nms(np.array(case["boxes"], np.float32), scores, case["threshold"],
                          case.get("categories"), case.get("max_keep"), lib=lib)
        assert keep.tolist() == case["keep"], "%s: %s != %s" % (case["name"], keep.tolist(),
                                                               case["keep"])


def pin_iou_closed_forms(lib):
    iou = lambda a, b: oracle.box_iou(a, b, lib=lib)
    assert iou([0, 0, 4, 4], [0, 0, 4, 4]) == 1.0
    assert iou([0, 0, 4, 4], [5, 5, 6, 6]) == 0.0
    assert iou([0, 0, 4, 4], [4, 0, 8, 4]) == 0.0            # touching edges
    assert iou([0, 0, 4, 4], [1, 1, 3, 3]) == 0.25           # nested: 4 / 16
    assert iou([0, 0, 4, 2], [2, 0, 6, 2]) == np.float32(4.0) / np.float32(12.0)  # 4 / (8+8-4)
    rng = np.random.default_rng(0)
    for _ in range(200):
        a = np.sort(rng.integers(0, 50, (2, 2)), axis=0).T.reshape(-1)[[0, 2, 1, 3]]
        b = np.sort(rng.integers(0, 50, (2, 2)), axis=0).T.reshape(-1)[[0, 2, 1, 3]]
        assert iou(a, b) == iou(b, a) or (np.isnan(iou(a, b)) and np.isnan(iou(b, a)))


def _iou_np(a, b):
    f = np.float32
    iw = np.maximum(np.minimum(a[2], b[2]) - np.maximum(a[0], b[0]), f(0))
    ih = np.maximum(np.minimum(a[3], b[3]) - np.maximum(a[1], b[1]), f(0))
    inter = f(iw * ih)
    ua = f((a[2] - a[0]) * (a[3] - a[1]))
    ub = f((b[2] - b[0]) * (b[3] - b[1]))
    with np.errstate(invalid="ignore", divide="ignore"):
        return f(inter / f(f(ua + ub) - inter))


def _rank(scores):
    u = scores.view(np.uint32).astype(np.uint64)
    nan = np.isnan(scores)
    asc = np.where(u & 0x80000000, (~u) & 0xFFFFFFFF, u | 0x80000000)
    key = np.where(nan, 0xFFFFFFFF, (~asc) & 0xFFFFFFFF)
    return np.lexsort((np.arange(len(scores)), key))


def pin_nms_characterization(lib):
    rng = np.random.default_rng(1)
    for trial in range(12):
        N = int(rng.integers(1, 160))
        cx, cy = rng.uniform(0, 100, N), rng.uniform(0, 100, N)
        w, h = rng.uniform(1, 40, N), rng.uniform(1, 40, N)
        boxes = np.stack([cx - w / 2, cy - h / 2, cx + w / 2, cy + h / 2], 1).astype(np.float32)
        scores = rng.uniform(0, 1, N).astype(np.float32)
        if trial % 3 == 0:
            scores[rng.integers(0, N, N // 4)] = 0.5        # ties
        cats = rng.integers(0, 3, N).astype(np.int32) if trial % 2 else None
        thr = float(rng.choice([0.3, 0.5, 0.7]))
        keep = oracle.nms(boxes, scores, thr, cats, lib=lib)
        order = _rank(scores)
        pos = {int(i): r for r, i in enumerate(order)}
        assert all(pos[int(a)] < pos[int(b)] for a, b in zip(keep[:-1], keep[1:])), "rank order"
        kept = set(int(i) for i in keep)
        same = (lambda i, j: True) if cats is None else (lambda i, j: cats[i] == cats[j])
        for r, i in enumerate(order):
            i = int(i)
            hit = any(same(i, int(j)) and _iou_np(boxes[int(j)], boxes[i]) > np.float32(thr)
                      for j in order[:r] if int(j) in kept)
            assert (i in kept) == (not hit), "box %d: kept %s, suppressed by a kept box %s" % (
                i, i in kept, hit)


ALL_NMS_PINS = [pin_nms_hand_cases, pin_iou_closed_forms, pin_nms_characterization]


def run_all(lib):
    failures = []
    for pin in ALL_NMS_PINS:
        try:
            pin(lib)
        except AssertionError:
            failures.append(pin.__name__)
    return failures
