"""GPU parity of the multi-head backward (roi_align_bwd_multi through the C ABI):
the gradient pyramid must equal the oracle's sum of every head's backward, within the
backward tolerance |gpu - ref| <= 1e-4 * S (S = the sum over heads of A^T|g|).

Covers the fused two-head pass (box 7x7 + mask 14x14, two 7x7 heads, both gradient
dtypes, accumulation), an odd number of heads (a pair plus a single head), and the
head-by-head fallback (mixed gradient dtypes, a head without a plan, non
channels-last levels), plus the box and mask heads of the batch-2 workload at full size.
"""
import numpy as np
import pytest

import oracle
import paper_1906_07155_amd as rex
from paper_1906_07155_amd import workloads as W
from gpu_helpers import as_f64, check_bwd, from_device, log, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    rex.lib()


def run(name, shapes, scales, heads, zero_init=True, layout="cl", seed=0):
    """heads: list of dicts with rois (numpy), out_hw, gdt and optional plan (bool)."""
    log("multi-head case %s: shapes=%s heads=%s zero_init=%d layout=%s" % (
        name, shapes, [(h["rois"].shape[0], h["out_hw"], h["gdt"], h.get("plan", True))
                       for h in heads], zero_init, layout))
    rng = np.random.default_rng(seed)
    L = len(shapes)
    C = shapes[0][1]
    dev_heads, ref, aref = [], [np.zeros(s) for s in shapes], [np.zeros(s) for s in shapes]
    feats = [torch.empty(s, dtype=torch.float32, device="cuda") for s in shapes]
    if layout == "cl":
        feats = [f.contiguous(memory_format=torch.channels_last) for f in feats]
    for h in heads:
        rois = h["rois"]
        K = rois.shape[0]
        r_dev = torch.from_numpy(rois).cuda()
        lv_dev, ws = rex.plan(feats, scales, r_dev, 56.0)
        lv = oracle.level_map(rois, L, 56.0)
        g = rng.standard_normal((K, C) + tuple(h["out_hw"]), dtype=np.float32)
        if h["gdt"] == "bf16":
            g = W.f32_to_bf16_bits(g)
        g64 = as_f64(g, h["gdt"])
        for l, (a, b) in enumerate(zip(
                oracle.roi_align_bwd(g64, shapes, scales, rois, lv, *h["out_hw"], 2, True),
                oracle.roi_align_bwd(np.abs(g64), shapes, scales, rois, lv, *h["out_hw"], 2,
                                     True))):
            ref[l] += a
            aref[l] += b
        dev_heads.append({"grad_out": to_device(g, h["gdt"], "nchw"), "rois": r_dev,
                          "roi_levels": lv_dev, "out_size": h["out_hw"],
                          "workspace": ws if h.get("plan", True) else None})
    grads = [torch.full(s, 7.0, dtype=torch.float32, device="cuda") for s in shapes]
    if layout == "cl":
        grads = [x.contiguous(memory_format=torch.channels_last) for x in grads]
    rex.roi_align_bwd_multi(dev_heads, grads, scales, zero_init=zero_init)
    torch.cuda.synchronize()
    base = 0.0 if zero_init else 7.0
    for l in range(L):
        check_bwd(from_device(grads[l]) - base, ref[l], aref[l] + base * 2.0 ** -20 / 1e-4,
                  False, "%s level %d" % (name, l))


PYR = [(2, 100, 24, 40), (2, 100, 12, 20), (2, 100, 6, 10), (2, 100, 3, 5)]
SC = [0.25, 0.125, 0.0625, 0.03125]


def _rois(seed, per_image, lo=4.0, hi=200.0):
    return W.draw_rois(np.random.default_rng(seed), 2, per_image, (96, 160), (lo, hi))


@pytest.mark.parametrize("gdt", ["f32", "bf16"])
def test_box_and_mask_heads_fused(gdt):
    run("box+mask %s" % gdt, PYR, SC, [
        {"rois": _rois(1, 23), "out_hw": (7, 7), "gdt": gdt},
        {"rois": _rois(2, 9, 16.0, 160.0), "out_hw": (14, 14), "gdt": gdt}])


def test_mask_then_box_and_two_box_heads():
    run("mask+box", PYR, SC, [
        {"rois": _rois(3, 9), "out_hw": (14, 14), "gdt": "f32"},
        {"rois": _rois(4, 17), "out_hw": (7, 7), "gdt": "f32"}])
    run("two box heads, accumulate", PYR, SC, [
        {"rois": _rois(5, 15), "out_hw": (7, 7), "gdt": "f32"},
        {"rois": _rois(6, 15), "out_hw": (7, 7), "gdt": "f32"}], zero_init=False)


def test_three_heads_and_fallbacks():
    run("three heads (pair + single)", PYR, SC, [
        {"rois": _rois(7, 11), "out_hw": (7, 7), "gdt": "f32"},
        {"rois": _rois(8, 7), "out_hw": (14, 14), "gdt": "f32"},
        {"rois": _rois(9, 11), "out_hw": (7, 7), "gdt": "f32"}])
    run("mixed gradient dtypes (head by head)", PYR, SC, [
        {"rois": _rois(10, 13), "out_hw": (7, 7), "gdt": "f32"},
        {"rois": _rois(11, 7), "out_hw": (14, 14), "gdt": "bf16"}])
    run("head without a plan (scatter)", PYR, SC, [
        {"rois": _rois(12, 13), "out_hw": (7, 7), "gdt": "f32", "plan": False},
        {"rois": _rois(13, 7), "out_hw": (14, 14), "gdt": "f32"}], zero_init=False)
    run("NCHW levels (scatter)", PYR, SC, [
        {"rois": _rois(14, 13), "out_hw": (7, 7), "gdt": "f32"},
        {"rois": _rois(15, 7), "out_hw": (14, 14), "gdt": "f32"}], layout="nchw")


def test_batch2_box_and_mask_heads_full_size():
    """The box head RoIs of the batch-2 workload and the mask head RoIs of the batch-2
    mask workload, both on the batch-2 FPN pyramid (P2-P5, 256 channels)."""
    box, mask = W.config(2), W.config(3)
    shapes = box.level_shapes()
    run("batch-2 box + mask heads", shapes, list(box.scales), [
        {"rois": box.rois(), "out_hw": (7, 7), "gdt": "f32"},
        {"rois": mask.rois(), "out_hw": (14, 14), "gdt": "f32"}], seed=3)
