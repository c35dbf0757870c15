"""Small inputs first, in a process that has made no large allocation yet.

Kernels that address memory through buffer resources must keep every access inside
the range the hardware checks.  A stray access past a tensor can go unnoticed when a
large allocation happens to map the addresses behind it, so these cases run before
the full-size workloads of the other files (pytest collects this file first): tiny
maps, few RoIs, bins whose pixel count is not a multiple of the RoI max-pooling
kernel's load batch, and channel counts that leave lanes without a channel.
"""
import numpy as np
import pytest

from paper_1906_07155_amd import workloads as W

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.mark.parametrize("C", [16, 64, 70])
@pytest.mark.parametrize("fdt", ["f32", "bf16"])
def test_pool_partial_load_batches(C, fdt):
    from test_gpu_pool import run
    rng = np.random.default_rng(100 + C)
    f = rng.standard_normal((1, C, 9, 11), dtype=np.float32)
    if fdt == "bf16":
        f = W.f32_to_bf16_bits(f)
    # bins of 1x1 up to 9x11 pixels: counts 1, 6, 15, 17, 99 ... (none a multiple of 16
    # except by chance), boxes clipped at every edge
    rois = np.array([[0, 0, 0, 10, 8], [0, 2, 1, 7, 6], [0, -3, -2, 4, 12],
                     [0, 5, 5, 5, 5], [0, 0, 0, 1, 1], [0, 8, 6, 14, 12]], np.float32)
    run("small C=%d %s" % (C, fdt), [f], [1.0], rois, out_hw=(2, 3), fdt=fdt, odt=fdt,
        use_plan=False, roi_levels=[0] * rois.shape[0])


def test_pool_single_bin_whole_map():
    from test_gpu_pool import run
    rng = np.random.default_rng(7)
    f = rng.standard_normal((2, 8, 5, 7), dtype=np.float32)
    rois = np.array([[1, 0, 0, 6, 4], [0, 0, 0, 6, 4]], np.float32)
    run("small whole map", [f], [1.0], rois, out_hw=(1, 1), use_plan=False, roi_levels=[0, 0])


def _golden(name):
    import json
    import os
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", name)
    with open(path) as f:
        return json.load(f)["cases"]


def _ramp_or_fill(lv):
    shape = tuple(lv["shape"])
    if lv.get("ramp_x"):
        return np.broadcast_to(np.arange(shape[3], dtype=np.float32), shape).copy()
    if "fill" in lv:
        return np.full(shape, lv["fill"], np.float32)
    return np.array(lv["values"], np.float32).reshape(shape)


def test_binary32_order_golden_cases():
    """The hand-derived binary32 sample coordinates that pin the oracle's geometry order
    (tests/golden/roi_align_binary32_cases.json), through the library.  With sampling
    ratio 1 (and the capped adaptive grid on a constant map) each output is one sample's
    bilinear value, exact in fp32, so it must equal the hand-derived value bit for bit;
    the 3 x 3 sample mean goes through fp32 sums and is held to the forward tolerance."""
    import paper_1906_07155_amd as rex
    from gpu_helpers import check_fwd, log
    for case in _golden("roi_align_binary32_cases.json"):
        log("binary32 case %s" % case["name"])
        feats = [torch.from_numpy(_ramp_or_fill(lv)).cuda() for lv in case["levels"]]
        scales = [lv["scale"] for lv in case["levels"]]
        rois = torch.tensor(case["rois"], dtype=torch.float32).cuda()
        out = rex.roi_align_fwd(feats, scales, rois, None, tuple(case["out"]),
                                case["sampling_ratio"], case["aligned"])
        got = out.cpu().numpy().astype(np.float64)
        exp = np.array(case["expected_parity"], np.float64)
        if case["sampling_ratio"] == 3:
            check_fwd(got, exp, False, case["name"])
        else:
            assert np.array_equal(got, exp), (case["name"], got.ravel(), exp.ravel())


def test_deform_binary32_shift_order_golden_case():
    import paper_1906_07155_amd as rex
    from gpu_helpers import log
    for case in _golden("deform_binary32_cases.json"):
        log("deform binary32 case %s" % case["name"])
        shape = tuple(case["shape"])
        feat = torch.from_numpy(np.broadcast_to(np.arange(shape[3], dtype=np.float32),
                                                shape).copy()).cuda()
        rois = torch.tensor(case["rois"], dtype=torch.float32).cuda()
        off = torch.tensor(case["offset"], dtype=torch.float32).cuda()
        out = rex.deform_roi_pool_fwd([feat], [case["scale"]], rois, None, tuple(case["out"]),
                                      off, None, case["gamma"], case["sampling_ratio"],
                                      case["aligned"])
        got = out.cpu().numpy().astype(np.float64)
        exp = np.array(case["expected_parity"], np.float64)
        assert np.array_equal(got, exp), (case["name"], got.ravel(), exp.ravel())
