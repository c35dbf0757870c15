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
  per-category     hand cases of greedy and Soft-NMS selection (linear and Gaussian
  selection and    decay, strict thresholds, dropping, ties, categories, max_keep);
  Soft-NMS         the Gaussian weight against exp; hard selection equals greedy NMS
                   with categories; coinciding boxes make linear Soft-NMS greedy NMS;
                   sigma to 0 and to infinity; independence of categories; the product
                   form of the decayed scores and the argmax property of each selection
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


# ---------------------------------------------------------------------------
# per-category selection and Soft-NMS
# ---------------------------------------------------------------------------

def _f(v):
    return float(v)   # numbers, or the strings "nan" / "-inf"


def load_soft_cases():
    return json.load(open(os.path.join(GOLDEN, "soft_nms_hand_cases.json")))["cases"]


def run_soft_case(case, lib=None):
    scores = np.array([_f(v) for v in case["scores"]], np.float32)
    return oracle.nms_batched(np.array(case["boxes"], np.float32), scores,
                              case.get("categories"), case["num_categories"], case["method"],
                              case["iou_threshold"], case["sigma"], _f(case["score_threshold"]),
                              case["max_keep"], lib=lib)


def pin_soft_nms_hand_cases(lib):
    for case in load_soft_cases():
        keep, sc, num = run_soft_case(case, lib)
        assert keep.tolist() == case["expected_keep"], (case["name"], keep.tolist())
        assert num.tolist() == case["expected_num"], (case["name"], num.tolist())
        exp = np.array(case["expected_scores"], np.float32)
        assert np.array_equal(sc.view(np.uint32), exp.view(np.uint32)), (case["name"], sc.tolist())


def pin_gauss_weight(lib):
    """The binary32 Gaussian weight is exp(-iou^2 / sigma) correctly rounded except where
    exp lies within 1e-12 (relative) of a rounding boundary; 1 at iou 0 and for a NaN
    IoU; non-increasing in iou; 0 when exp underflows binary32."""
    w = lambda i, s: oracle.soft_gauss_weight(i, s, lib=lib)
    assert w(0.0, 0.5) == 1.0 and w(float("nan"), 0.5) == 1.0
    assert w(1.0, 1e-3) == 0.0
    for sigma in (1e-3, 0.1, 0.5, 2.0, 37.0):
        prev = 1.0
        for iou in np.linspace(0.0, 1.0, 401, dtype=np.float32)[1:]:
            got = w(float(iou), sigma)
            x = -(float(iou) * float(iou)) / float(np.float32(sigma))
            e = np.exp(x)
            f = np.float32(e)
            lo, hi = (f, np.nextafter(f, np.float32(2))) if float(f) <= e else (
                np.nextafter(f, np.float32(0)), f)
            mid = (float(lo) + float(hi)) / 2
            if abs(e - mid) > 1e-12 * e:
                assert got == float(f), (iou, sigma, got, float(f))
            assert got <= prev
            prev = got


def _rand_boxes(rng, N, span=100.0, lo=2.0, hi=30.0, grid=False):
    if grid:
        xy = rng.integers(0, int(span), (N, 2)).astype(np.float32)
        wh = rng.integers(int(lo), int(hi), (N, 2)).astype(np.float32)
    else:
        xy = rng.uniform(0, span, (N, 2)).astype(np.float32)
        wh = rng.uniform(lo, hi, (N, 2)).astype(np.float32)
    return np.concatenate([xy, xy + wh], 1).astype(np.float32)


def pin_batched_hard_is_greedy(lib):
    """Per-category hard selection keeps, in each category, exactly the boxes greedy NMS
    with categories keeps (the separately pinned oracle_nms), in the same order."""
    rng = np.random.default_rng(2)
    for trial in range(6):
        N, C = int(rng.integers(20, 300)), int(rng.integers(1, 6))
        boxes = _rand_boxes(rng, N)
        scores = rng.uniform(0, 1, N).astype(np.float32)
        cats = rng.integers(0, C, N).astype(np.int32)
        thr = float(rng.choice([0.3, 0.5, 0.7]))
        keep, sc, num = oracle.nms_batched(boxes, scores, cats, C, "hard", thr, lib=lib)
        ref = oracle.nms(boxes, scores, thr, cats, lib=lib)
        for c in range(C):
            exp = [int(i) for i in ref if cats[i] == c]
            assert keep[c, :num[c]].tolist() == exp, (trial, c)
            assert np.array_equal(sc[c, :num[c]], scores[exp])


def pin_soft_identical_boxes_is_hard(lib):
    """Boxes that either coincide (IoU exactly 1) or are disjoint: linear decay takes an
    overlapped score to s * (1 - 1) = 0, and with a positive score threshold it is
    dropped, so Soft-NMS keeps exactly greedy NMS's boxes with their input scores."""
    rng = np.random.default_rng(3)
    base = np.array([[10 * i, 0, 10 * i + 5, 5] for i in range(12)], np.float32)
    for trial in range(5):
        pick = rng.integers(0, 12, 60)
        boxes = base[pick]
        scores = rng.uniform(0.01, 1, 60).astype(np.float32)
        cats = rng.integers(0, 3, 60).astype(np.int32)
        keep, sc, num = oracle.nms_batched(boxes, scores, cats, 3, "linear", 0.5,
                                           score_threshold=1e-6, lib=lib)
        ref = oracle.nms(boxes, scores, 0.5, cats, lib=lib)
        for c in range(3):
            exp = [int(i) for i in ref if cats[i] == c]
            assert keep[c, :num[c]].tolist() == exp
            assert np.array_equal(sc[c, :num[c]], scores[exp])


def pin_gaussian_limits(lib):
    """sigma -> 0: every overlapped candidate's weight underflows to 0 and is dropped, so
    Soft-NMS keeps greedy NMS's boxes at IoU threshold 0 (integer boxes: the smallest
    positive IoU is far above the underflow point); sigma -> infinity: no decay, every
    candidate kept in rank order with its input score."""
    rng = np.random.default_rng(4)
    for trial in range(4):
        N = 80
        boxes = _rand_boxes(rng, N, span=60, lo=3, hi=9, grid=True)
        scores = rng.uniform(0.01, 1, N).astype(np.float32)
        keep, sc, num = oracle.nms_batched(boxes, scores, None, 1, "gaussian", sigma=1e-9,
                                           score_threshold=1e-30, lib=lib)
        ref = oracle.nms(boxes, scores, 0.0, None, lib=lib)
        assert keep[0, :num[0]].tolist() == ref.tolist()
        keep, sc, num = oracle.nms_batched(boxes, scores, None, 1, "gaussian", sigma=1e30,
                                           lib=lib)
        order = _rank(scores)
        assert keep[0].tolist() == order.tolist() and np.array_equal(sc[0], scores[order])


def pin_category_independence(lib):
    """A category's result does not depend on the other categories' boxes."""
    rng = np.random.default_rng(5)
    N, C = 150, 4
    boxes = _rand_boxes(rng, N)
    scores = rng.uniform(0, 1, N).astype(np.float32)
    cats = rng.integers(0, C, N).astype(np.int32)
    for method in ("linear", "gaussian"):
        keep, sc, num = oracle.nms_batched(boxes, scores, cats, C, method, 0.4, 0.3, 0.05,
                                           lib=lib)
        for c in range(C):
            sel = np.flatnonzero(cats == c)
            k1, s1, n1 = oracle.nms_batched(boxes[sel], scores[sel], None, 1, method, 0.4, 0.3,
                                            0.05, lib=lib)
            assert n1[0] == num[c]
            assert sel[k1[0, :n1[0]]].tolist() == keep[c, :num[c]].tolist()
            assert np.array_equal(s1[0, :n1[0]], sc[c, :num[c]])


def _soft_weight_f64(method, iou, thr, sigma):
    if np.isnan(iou):
        return 1.0
    if method == "linear":
        return 1.0 - iou if iou > thr else 1.0
    return float(np.exp(-(iou * iou) / sigma))


def pin_soft_product_characterization(lib):
    """On random boxes the selection is the one Soft-NMS is defined by: every output score
    is the input score times the weights of the boxes selected before it (computed here
    in double; binary32 rounding of the sequential products stays within 1e-5); each
    selected box has the largest such score among the remaining candidates; the boxes
    left unselected (when fewer than max_keep were kept) fell below the threshold."""
    rng = np.random.default_rng(6)
    for trial in range(10):
        N = int(rng.integers(5, 90))
        boxes = _rand_boxes(rng, N, span=80)
        scores = rng.uniform(0.05, 1, N).astype(np.float32)
        method = "linear" if trial % 2 else "gaussian"
        thr, sigma, st = 0.3, 0.5, 0.02 * (trial % 3)
        mk = N if trial % 4 else max(1, N // 3)
        keep, sc, num = oracle.nms_batched(boxes, scores, None, 1, method, thr, sigma, st, mk,
                                           lib=lib)
        sel = keep[0, :num[0]].tolist()
        iou = np.array([[oracle.box_iou(boxes[i], boxes[j], lib=lib) for j in range(N)]
                        for i in range(N)], np.float64)
        cur = scores.astype(np.float64).copy()
        alive = scores >= np.float32(st)
        for t, m in enumerate(sel):
            assert alive[m], (trial, t)
            others = np.flatnonzero(alive)
            assert cur[m] >= cur[others].max() * (1 - 1e-5) - 1e-12, (trial, t)
            assert abs(float(sc[0, t]) - cur[m]) <= 1e-5 * cur[m] + 1e-12, (trial, t)
            alive[m] = False
            for j in np.flatnonzero(alive):
                cur[j] *= _soft_weight_f64(method, iou[m, j], thr, sigma)
                if cur[j] < st * (1 - 1e-5):
                    alive[j] = False
        if num[0] < mk:
            assert not np.any(cur[alive] >= st * (1 + 1e-5)), trial


SOFT_NMS_PINS = [pin_soft_nms_hand_cases, pin_gauss_weight, pin_batched_hard_is_greedy,
                 pin_soft_identical_boxes_is_hard, pin_gaussian_limits,
                 pin_category_independence, pin_soft_product_characterization]

ALL_NMS_PINS = [pin_nms_hand_cases, pin_iou_closed_forms, pin_nms_characterization] + \
    SOFT_NMS_PINS


def run_all(lib):
    failures = []
    for pin in ALL_NMS_PINS:
        try:
            pin(lib)
        except AssertionError:
            failures.append(pin.__name__)
    return failures
