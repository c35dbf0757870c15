"""The allocation-free forward (roi_align_fwd_noalloc, plan kept in the library's fixed
per-GPU array) against roi_align_fwd with a caller workspace, through the C ABI.

Two calls in a row, the second with fewer RoIs and a different pyramid, so the second
call runs on the array the first one left behind; the outputs and levels must equal
the workspace path's, and both are checked against the CPU oracle at the forward
tolerance.  Sizes beyond RE_NOALLOC_MAX_ROIS are refused before anything is enqueued.
"""
import numpy as np
import pytest

import oracle
from paper_1906_07155_amd import binding as B
from paper_1906_07155_amd import workloads as W
from gpu_helpers import as_f64, check_fwd, from_device, log, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()


def _case(seed, n, C, hw, K, fdt):
    rng = np.random.default_rng(seed)
    shapes = [(n, C, h, w) for (h, w) in hw]
    scales = [1.0 / (4 << l) for l in range(len(hw))]
    feats = []
    for s in shapes:
        x = rng.standard_normal(s, dtype=np.float32)
        feats.append(W.f32_to_bf16_bits(x) if fdt == "bf16" else x)
    img = (hw[0][0] * 4, hw[0][1] * 4)
    rois = W.draw_rois(rng, n, K // n, img, (8.0, 0.9 * min(img)))
    return feats, scales, rois


def _run(feats, scales, rois, out_hw, fdt, name):
    log("noalloc case %s: K=%d shapes=%s out=%s %s" % (name, rois.shape[0],
                                                       [f.shape for f in feats], out_hw, fdt))
    dev = [to_device(f, fdt, "cl") for f in feats]
    r = torch.from_numpy(rois).cuda()
    out_a, lv_a = B.roi_align_fwd_noalloc(dev, scales, r, out_hw, 2, True)
    lv_b, ws = B.plan(dev, scales, r, 56.0)
    out_b = B.roi_align_fwd(dev, scales, r, lv_b, out_hw, 2, True, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(lv_a, lv_b), name + ": levels differ"
    assert torch.equal(out_a, out_b), name + ": outputs differ from roi_align_fwd"
    lv = oracle.level_map(rois, len(feats), 56.0)
    assert np.array_equal(lv_a.cpu().numpy(), lv), name + ": levels differ from the oracle"
    ref = oracle.roi_align_fwd([as_f64(f, fdt) for f in feats], scales, rois, lv, *out_hw, 2,
                               True, "parity")
    check_fwd(from_device(out_a), ref, fdt == "bf16", name)


def test_two_calls_second_smaller():
    hw = [(48, 80), (24, 40), (12, 20), (6, 10)]
    f1, s1, r1 = _case(1, 2, 96, hw, 600, "f32")
    _run(f1, s1, r1, (7, 7), "f32", "first, 600 RoIs 7x7")
    f2, s2, r2 = _case(2, 1, 70, hw[:3], 90, "bf16")
    _run(f2, s2, r2, (14, 14), "bf16", "second, 90 RoIs 14x14 bf16")


def test_large_plan_then_small():
    """Above 8192 RoIs the plan takes its five-kernel form (bucket counters cleared by a
    kernel in the array); a small call after it reuses the dirty array."""
    hw = [(50, 84), (25, 42), (13, 21), (7, 11)]
    f1, s1, r1 = _case(3, 4, 64, hw, 9000, "f32")
    _run(f1, s1, r1, (7, 7), "f32", "9000 RoIs")
    f2, s2, r2 = _case(4, 2, 64, hw, 40, "f32")
    _run(f2, s2, r2, (7, 7), "f32", "40 RoIs after 9000")


def test_limit_is_refused():
    rois = torch.zeros((70000, 5), dtype=torch.float32, device="cuda")
    feats = [torch.zeros((1, 8, 16, 16), device="cuda").contiguous(
        memory_format=torch.channels_last)]
    with pytest.raises(B.RoIExtractError) as e:
        B.roi_align_fwd_noalloc(feats, [0.25], rois, (7, 7))
    assert e.value.status == B.RE_ERR_UNSUPPORTED
