"""GPU parity of per-category proposal selection (box_nms_batched: greedy NMS and
Soft-NMS with linear or Gaussian decay, through the C ABI) against the CPU oracle.

Selection is integer work decided by binary32 scores, and both sides take every
decision in binary32 with the same operation order (the Gaussian weight by the same
scaling-and-squaring evaluation in double), so the kept lists must be equal and the
scores at selection equal bit for bit.
"""
import json
import os

import numpy as np
import pytest

import oracle
import paper_1906_07155_amd as rex
from paper_1906_07155_amd import workloads as W
from gpu_helpers import log

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    rex.lib()


def run(name, boxes, scores, cats, C, method, thr=0.5, sigma=0.5, st=float("-inf"),
        max_keep=None):
    N = scores.shape[0]
    mk = N if max_keep is None else max_keep
    log("select case %s: N=%d C=%d %s thr=%g sigma=%g st=%g max_keep=%d" % (
        name, N, C, method, thr, sigma, st, mk))
    b = torch.from_numpy(np.ascontiguousarray(boxes, np.float32)).cuda()
    s = torch.from_numpy(np.ascontiguousarray(scores, np.float32)).cuda()
    c = torch.from_numpy(np.ascontiguousarray(cats, np.int32)).cuda() if cats is not None else None
    keep, ks, num = rex.box_nms_batched(b, s, c, C, method, thr, sigma, st, mk)
    torch.cuda.synchronize()
    rk, rs, rn = oracle.nms_batched(boxes, scores, cats, C, method, thr, sigma, st, mk)
    gk, gs, gn = keep.cpu().numpy(), ks.cpu().numpy(), num.cpu().numpy()
    assert np.array_equal(gn, rn), "%s: counts differ: %s vs %s" % (name, gn[:8], rn[:8])
    bad = np.argwhere(gk != rk)
    assert bad.size == 0, "%s: kept lists differ first at %s (gpu %d, oracle %d)" % (
        name, bad[0], gk[tuple(bad[0])], rk[tuple(bad[0])])
    bad = np.argwhere(gs.view(np.uint32) != rs.view(np.uint32))
    assert bad.size == 0, "%s: scores differ first at %s (gpu %r, oracle %r)" % (
        name, bad[0], gs[tuple(bad[0])], rs[tuple(bad[0])])
    return gk, gs, gn


def test_hand_cases():
    for case in json.load(open(os.path.join(GOLDEN, "soft_nms_hand_cases.json")))["cases"]:
        scores = np.array([float(v) for v in case["scores"]], np.float32)
        gk, gs, gn = run(case["name"], np.array(case["boxes"], np.float32), scores,
                         case.get("categories"), case["num_categories"], case["method"],
                         case["iou_threshold"], case["sigma"], float(case["score_threshold"]),
                         case["max_keep"])
        assert gk.tolist() == case["expected_keep"], case["name"]
        assert np.array_equal(gs, np.array(case["expected_scores"], np.float32)), case["name"]


def proposals(rng, n_images, per_image, lo=8.0, hi=600.0, dup=0.3):
    return W.draw_proposals(rng, n_images, per_image, (800, 1333), (lo, hi), dup)


@pytest.mark.parametrize("method", ["hard", "linear", "gaussian"])
def test_batch_of_images(method):
    rng = np.random.default_rng({"hard": 1, "linear": 2, "gaussian": 3}[method])
    boxes, scores, cats = proposals(rng, 16, 600)
    perm = rng.permutation(boxes.shape[0])          # categories interleaved in the input
    boxes, scores, cats = boxes[perm], scores[perm], cats[perm]
    run("16 x 600 " + method, boxes, scores, cats, 16, method, thr=0.5 if method != "linear" else 0.3,
        sigma=0.5, st=0.05 if method != "hard" else float("-inf"), max_keep=300)


def test_hard_equals_greedy_box_nms():
    """Per-category greedy selection keeps what box_nms with categories keeps."""
    rng = np.random.default_rng(4)
    boxes, scores, cats = proposals(rng, 4, 1500)
    gk, _, gn = run("4 x 1500 hard", boxes, scores, cats, 4, "hard", thr=0.7)
    keep, num = rex.box_nms(torch.from_numpy(boxes).cuda(), torch.from_numpy(scores).cuda(), 0.7,
                            categories=torch.from_numpy(cats).cuda())
    k = keep[:int(num.item())].cpu().numpy()
    for c in range(4):
        assert gk[c, :gn[c]].tolist() == [int(i) for i in k if cats[i] == c]


@pytest.mark.parametrize("method", ["hard", "linear", "gaussian"])
def test_long_category(method):
    """One category longer than the LDS sort (8192 candidates: global-memory bitonic
    sort), the Soft-NMS register slots (4096) and the LDS box cache (3072); a few
    short categories beside it."""
    rng = np.random.default_rng(5)
    b1, s1, _ = proposals(rng, 1, 9000, lo=4.0, hi=80.0, dup=0.2)
    b2, s2, _ = proposals(rng, 1, 300)
    boxes = np.concatenate([b1, b2])
    scores = np.concatenate([s1, s2])
    cats = np.concatenate([np.zeros(9000, np.int32), rng.integers(1, 4, 300).astype(np.int32)])
    mk = {"hard": 9000, "linear": 700, "gaussian": 700}[method]
    run("long category " + method, boxes, scores, cats, 4, method, thr=0.5, sigma=0.3,
        st=0.2 if method != "hard" else float("-inf"), max_keep=mk)


def test_edges():
    rng = np.random.default_rng(6)
    boxes, scores, cats = proposals(rng, 3, 100)
    scores[::7] = np.nan
    scores[::11] = -np.inf
    cats[::13] = 5                                   # outside [0, 3): never a candidate
    cats[::17] = -1
    for method in ("hard", "linear", "gaussian"):
        run("edges " + method, boxes, scores, cats, 3, method, st=0.0 if method != "hard"
            else float("-inf"), max_keep=40)
        run("max_keep 1 " + method, boxes, scores, cats, 3, method, max_keep=1)
        run("max_keep 0 " + method, boxes, scores, cats, 3, method, max_keep=0)
        run("empty categories " + method, boxes, scores, cats, 40, method, max_keep=7)
    run("no boxes", np.zeros((0, 4), np.float32), np.zeros(0, np.float32), None, 1, "hard",
        max_keep=3)
    # degenerate boxes: zero area (NaN IoU between two of them), inverted, identical
    db = np.array([[5, 5, 5, 5], [5, 5, 5, 5], [9, 9, 3, 3], [0, 0, 4, 4], [0, 0, 4, 4],
                   [1, 1, 2, 8]], np.float32)
    ds = np.array([0.9, 0.8, 0.7, 0.6, 0.5, 0.4], np.float32)
    for method in ("hard", "linear", "gaussian"):
        run("degenerate " + method, db, ds, None, 1, method, thr=0.1, sigma=0.2)


def test_many_small_categories():
    rng = np.random.default_rng(7)
    boxes, scores, _ = proposals(rng, 1, 5000)
    cats = rng.integers(0, 1000, 5000).astype(np.int32)
    for method in ("hard", "gaussian"):
        run("1000 categories " + method, boxes, scores, cats, 1000, method, max_keep=5)
