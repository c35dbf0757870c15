"""GPU parity of the multi-head forward and backward (roi_align_fwd_multi and
roi_align_bwd_multi through the C ABI).

Forward: every head's output must equal the oracle's within the forward tolerance and
equal the single-head roi_align_fwd bit for bit (the same per-element arithmetic), for
heads that share the launch (7x7 and 14x14, one or both grids), heads that fall back
(adaptive sampling, NCHW levels), empty heads and heads without a plan.

Backward: the gradient pyramid must equal the oracle's sum of every head's backward,
within the backward tolerance |gpu - ref| <= 1e-4 * S (S = the sum over heads of A^T|g|).

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
from gpu_helpers import as_f64, check_bwd, check_fwd, from_device, log, to_device

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


def run_fwd(name, shapes, scales, heads, fdt="f32", odt=None, layout="cl", seed=0):
    """heads: list of dicts with rois (numpy), out_hw, and optional sr (2) and plan (True)."""
    odt = odt or fdt
    log("multi-head forward case %s: shapes=%s fdt=%s odt=%s layout=%s heads=%s" % (
        name, shapes, fdt, odt, layout, [(h["rois"].shape[0], h["out_hw"], h.get("sr", 2),
                                          h.get("plan", True)) for h in heads]))
    rng = np.random.default_rng(seed)
    L = len(shapes)
    host = [rng.standard_normal(s, dtype=np.float32) for s in shapes]
    if fdt == "bf16":
        host = [W.f32_to_bf16_bits(f) for f in host]
    feats = [to_device(f, fdt, layout) for f in host]
    f64 = [as_f64(f, fdt) for f in host]
    tdt = torch.bfloat16 if odt == "bf16" else torch.float32
    dev_heads, refs = [], []
    for h in heads:
        rois = h["rois"]
        r_dev = torch.from_numpy(rois).cuda()
        lv_dev, ws = rex.plan(feats, scales, r_dev, 56.0)
        lv = oracle.level_map(rois, L, 56.0)
        sr = h.get("sr", 2)
        refs.append(oracle.roi_align_fwd(f64, scales, rois, lv, *h["out_hw"], sr, True))
        dev_heads.append({"rois": r_dev, "roi_levels": lv_dev, "out_size": h["out_hw"],
                          "sampling_ratio": sr,
                          "workspace": ws if h.get("plan", True) else None})
    outs = rex.roi_align_fwd_multi(feats, scales, dev_heads, out_dtype=tdt)
    singles = [rex.roi_align_fwd(feats, scales, d["rois"], d["roi_levels"], d["out_size"],
                                 d["sampling_ratio"], True, out_dtype=tdt,
                                 workspace=d["workspace"]) for d in dev_heads]
    torch.cuda.synchronize()
    for i, (o, one, ref) in enumerate(zip(outs, singles, refs)):
        got = from_device(o)
        check_fwd(got, ref, fdt == "bf16" or odt == "bf16", "%s head %d" % (name, i))
        assert torch.equal(o.view(torch.int16) if tdt == torch.bfloat16 else o.view(torch.int32),
                           one.view(torch.int16) if tdt == torch.bfloat16
                           else one.view(torch.int32)), "%s head %d != roi_align_fwd" % (name, i)


@pytest.mark.parametrize("fdt,odt", [("f32", "f32"), ("bf16", "bf16"), ("bf16", "f32"),
                                     ("f32", "bf16")])
def test_fwd_box_and_mask_heads_one_launch(fdt, odt):
    run_fwd("box+mask %s->%s" % (fdt, odt), PYR, SC, [
        {"rois": _rois(21, 23), "out_hw": (7, 7)},
        {"rois": _rois(22, 9, 16.0, 160.0), "out_hw": (14, 14)}], fdt, odt)


@pytest.mark.parametrize("fdt", ["f32", "bf16"])
def test_fwd_cascade_heads(fdt):
    """Three 7x7 heads (the stages of a cascade) in one launch, one without a plan."""
    run_fwd("three 7x7 heads %s" % fdt, PYR, SC, [
        {"rois": _rois(23, 31), "out_hw": (7, 7)},
        {"rois": _rois(24, 17), "out_hw": (7, 7), "plan": False},
        {"rois": _rois(25, 5), "out_hw": (7, 7)}], fdt)
    run_fwd("two 14x14 heads %s" % fdt, PYR, SC, [
        {"rois": _rois(26, 7), "out_hw": (14, 14)},
        {"rois": _rois(27, 12), "out_hw": (14, 14)}], fdt)


def test_fwd_odd_channels_empty_heads_and_fallbacks():
    pyr = [(2, 70, 24, 40), (2, 70, 12, 20), (2, 70, 6, 10), (2, 70, 3, 5)]
    run_fwd("odd channel count bf16", [(2, 35, 24, 40), (2, 35, 12, 20)], SC[:2], [
        {"rois": _rois(28, 9), "out_hw": (7, 7)},
        {"rois": _rois(29, 4), "out_hw": (14, 14)}], "bf16")
    run_fwd("empty heads", pyr, SC, [
        {"rois": np.zeros((0, 5), np.float32), "out_hw": (7, 7)},
        {"rois": _rois(30, 6), "out_hw": (14, 14)},
        {"rois": np.zeros((0, 5), np.float32), "out_hw": (14, 14)}])
    run_fwd("adaptive sampling head (falls back)", pyr, SC, [
        {"rois": _rois(31, 8), "out_hw": (7, 7)},
        {"rois": _rois(32, 8), "out_hw": (7, 7), "sr": 0},
        {"rois": _rois(33, 5), "out_hw": (5, 3)}])
    run_fwd("NCHW levels (every head falls back)", pyr, SC, [
        {"rois": _rois(34, 8), "out_hw": (7, 7)},
        {"rois": _rois(35, 5), "out_hw": (14, 14)}], layout="nchw")


def test_fwd_batch2_box_and_mask_heads_full_size():
    """The box and mask heads of the batch-2 workloads on the batch-2 pyramid (P2-P5,
    256 channels): the fused launch equals the single-head calls bit for bit, and the
    first RoIs of each head (every channel) equal the oracle's."""
    box, mask = W.config(2), W.config(3)
    shapes, scales = box.level_shapes(), list(box.scales)
    host = box.features()
    feats = [to_device(f, "f32") for f in host]
    f64 = [np.asarray(f, np.float64) for f in host]
    del host
    heads, sub = [], []
    for wl, hw in ((box, (7, 7)), (mask, (14, 14))):
        rois = wl.rois()
        r_dev = torch.from_numpy(rois).cuda()
        lv_dev, ws = rex.plan(feats, scales, r_dev, 56.0)
        heads.append({"rois": r_dev, "roi_levels": lv_dev, "out_size": hw, "workspace": ws})
        sub.append((rois[:48], oracle.level_map(rois[:48], len(shapes), 56.0), hw))
    log("multi-head forward batch-2 box %d RoIs + mask %d RoIs" % (
        heads[0]["rois"].shape[0], heads[1]["rois"].shape[0]))
    outs = rex.roi_align_fwd_multi(feats, scales, heads)
    singles = [rex.roi_align_fwd(feats, scales, h["rois"], h["roi_levels"], h["out_size"],
                                 workspace=h["workspace"]) for h in heads]
    torch.cuda.synchronize()
    for i, (o, one, (r, lv, hw)) in enumerate(zip(outs, singles, sub)):
        assert torch.equal(o.view(torch.int32), one.view(torch.int32)), "head %d" % i
        ref = oracle.roi_align_fwd(f64, scales, r, lv, *hw, 2, True)
        check_fwd(from_device(o[:48]), ref, False, "batch-2 head %d" % i)
