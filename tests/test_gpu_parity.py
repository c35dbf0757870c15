"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Full-size workloads run in the launch configuration the benchmark times (the
plan-ordered channels-last kernels).  Workloads 1-4 are compared element by
element in full, the batch-16 workload (both heads, bf16) included.
"""
import numpy as np
import pytest

import oracle
import paper_1906_07155_amd as rex
from paper_1906_07155_amd import workloads as W
from gpu_helpers import Case, as_f64, check_bwd, check_fwd, from_device, log, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    rex.lib()


_CASES = {}


def _case(idx, head=None, fdt=None):
    key = (idx, head, fdt)
    if key not in _CASES:
        wl = W.config(idx, head=head, feat_dtype=fdt)
        feats = None
        if idx == 5:
            other = [c for k, c in _CASES.items() if k[0] == 5]
            if other:
                feats = other[0].feats_np
        _CASES[key] = Case(wl, feats=feats)
    return _CASES[key]


FULL = [(1, None, None), (2, None, None), (3, None, None), (4, None, "f32"), (4, None, "bf16")]
B16 = [(5, "box", None), (5, "mask", None)]


def _run_fwd(c: Case, plan=True):
    levels, ws = rex.plan(c.feats, c.scales, c.rois_dev, c.wl.finest_scale)
    out = rex.roi_align_fwd(c.feats, c.scales, c.rois_dev, levels, c.wl.out_hw,
                            c.wl.sampling_ratio, c.wl.aligned,
                            out_dtype=torch.bfloat16 if c.wl.out_dtype == "bf16" else torch.float32,
                            workspace=ws if plan else None)
    torch.cuda.synchronize()
    return levels, ws, out


def _run_bwd(c: Case, levels, ws, g_np, algorithm, layout="cl"):
    g = to_device(g_np, c.wl.grad_dtype, layout="nchw")
    grads = [torch.full(s, 3.0, dtype=torch.float32, device="cuda") for s in c.shapes]
    if layout == "cl":
        grads = [x.contiguous(memory_format=torch.channels_last) for x in grads]
    rex.roi_align_bwd(g, c.rois_dev, levels, c.wl.out_hw, c.wl.sampling_ratio, c.wl.aligned,
                      grads, c.scales, zero_init=True, workspace=ws, algorithm=algorithm)
    torch.cuda.synchronize()
    return grads


@pytest.mark.parametrize("idx,head,fdt", FULL + B16)
def test_level_map_and_plan(idx, head, fdt):
    c = _case(idx, head, fdt)
    log("level map + plan: workload %d %s %s, K=%d" % (idx, head, fdt, c.K))
    ref = c.oracle_levels()
    L = len(c.shapes)
    lv1 = rex.fpn_level_map(c.rois_dev, L, c.wl.finest_scale)
    levels, ws = rex.plan(c.feats, c.scales, c.rois_dev, c.wl.finest_scale)
    offs = rex.plan_offsets(ws, c.K, L)
    perm = rex.plan_perm(ws, c.K)
    torch.cuda.synchronize()
    assert np.array_equal(lv1.cpu().numpy(), ref)
    assert np.array_equal(levels.cpu().numpy(), ref)
    p = perm.cpu().numpy()
    assert np.array_equal(np.sort(p), np.arange(c.K))
    lv_sorted = ref[p]
    assert np.all(np.diff(lv_sorted) >= 0)
    counts = np.bincount(ref, minlength=L)
    assert np.array_equal(offs.cpu().numpy(), np.concatenate([[0], np.cumsum(counts)]))
    b = np.trunc(c.rois[p, 0]).astype(int)
    for l in range(L):
        seg = b[offs.cpu().numpy()[l]:offs.cpu().numpy()[l + 1]]
        assert np.all(np.diff(seg) >= 0), "images not grouped within level %d" % l


@pytest.mark.parametrize("idx,head,fdt", FULL)
def test_forward_full(idx, head, fdt):
    c = _case(idx, head, fdt)
    log("forward full: workload %d %s, K=%d" % (idx, fdt, c.K))
    levels, ws, out = _run_fwd(c)
    ref_lv = c.oracle_levels()
    ref = oracle.roi_align_fwd([as_f64(f, c.wl.feat_dtype) for f in c.feats_np], c.scales,
                               c.rois, ref_lv, *c.wl.out_hw, c.wl.sampling_ratio,
                               c.wl.aligned, "parity")
    err = check_fwd(from_device(out), ref, c.bf16, "workload %d forward" % idx)
    log("  max abs err %.3e" % err)


def test_forward_full_nchw():
    """Workload 2 forward on contiguous NCHW levels (the general strided kernel), every
    element against the oracle."""
    c = _case(2)
    log("forward full, NCHW levels: workload 2, K=%d" % c.K)
    feats = [to_device(f, c.wl.feat_dtype, "nchw") for f in c.feats_np]
    levels, ws = rex.plan(feats, c.scales, c.rois_dev, c.wl.finest_scale)
    out = rex.roi_align_fwd(feats, c.scales, c.rois_dev, levels, c.wl.out_hw,
                            c.wl.sampling_ratio, c.wl.aligned, workspace=ws)
    torch.cuda.synchronize()
    ref = oracle.roi_align_fwd([as_f64(f, c.wl.feat_dtype) for f in c.feats_np], c.scales,
                               c.rois, c.oracle_levels(), *c.wl.out_hw, c.wl.sampling_ratio,
                               c.wl.aligned, "parity")
    check_fwd(from_device(out), ref, False, "workload 2 NCHW forward")


@pytest.mark.parametrize("algorithm,layout", [("scatter", "cl"), ("gather", "cl"),
                                              ("gather", "nchw")])
@pytest.mark.parametrize("idx,head,fdt", [(2, None, None), (3, None, None)])
def test_backward_full(idx, head, fdt, algorithm, layout):
    """Full-size backward; the gather also into contiguous NCHW gradients (the RoIs are
    planned on the channels-last features, the plan does not depend on the layout)."""
    c = _case(idx, head, fdt)
    log("backward full (%s, %s gradients): workload %d, K=%d" % (algorithm, layout, idx, c.K))
    levels, ws, _ = _run_fwd(c)
    g = c.wl.grad()
    grads = _run_bwd(c, levels, ws, g, algorithm, layout)
    ref_lv = c.oracle_levels()
    g64 = as_f64(g, c.wl.grad_dtype)
    ref = oracle.roi_align_bwd(g64, c.shapes, c.scales, c.rois, ref_lv, *c.wl.out_hw,
                               c.wl.sampling_ratio, c.wl.aligned, "parity")
    absref = oracle.roi_align_bwd(np.abs(g64), c.shapes, c.scales, c.rois, ref_lv,
                                  *c.wl.out_hw, c.wl.sampling_ratio, c.wl.aligned, "parity")
    for l in range(len(c.shapes)):
        r = check_bwd(from_device(grads[l]), ref[l], absref[l], False,
                      "workload %d backward level %d" % (idx, l))
        log("  level %d rel norm err %.3e" % (l, r))


# The batch-16 workload is compared on every RoI and every channel (all four 64-lane
# slices, so the forward's multi-slice workgroups are covered from their first slice to
# their last).
B16_CHANNELS = np.arange(256)
_B16_REF = {}


def _b16_reference(c: Case, head):
    if head not in _B16_REF:
        ref_lv = c.oracle_levels()
        chans = B16_CHANNELS
        feats_sub = [as_f64(f[:, chans], "bf16") for f in c.feats_np]
        fwd = oracle.roi_align_fwd(feats_sub, c.scales, c.rois, ref_lv, *c.wl.out_hw,
                                   c.wl.sampling_ratio, c.wl.aligned, "parity")
        del feats_sub
        g = c.wl.grad()
        g64 = as_f64(g, "bf16")[:, chans]
        shapes = [(s[0], len(chans), s[2], s[3]) for s in c.shapes]
        bwd = oracle.roi_align_bwd(g64, shapes, c.scales, c.rois, ref_lv, *c.wl.out_hw,
                                   c.wl.sampling_ratio, c.wl.aligned, "parity")
        absbwd = oracle.roi_align_bwd(np.abs(g64), shapes, c.scales, c.rois, ref_lv,
                                      *c.wl.out_hw, c.wl.sampling_ratio, c.wl.aligned, "parity")
        _B16_REF[head] = (fwd, g, bwd, absbwd)
    return _B16_REF[head]


@pytest.mark.parametrize("algorithm", ["scatter", "gather"])
@pytest.mark.parametrize("idx,head,fdt", B16)
def test_batch16_full(idx, head, fdt, algorithm):
    c = _case(idx, head, fdt)
    log("batch-16 %s head (%s): fwd+bwd at full size, every element, K=%d" % (
        head, algorithm, c.K))
    levels, ws, out = _run_fwd(c)
    fwd_ref, g, bwd_ref, absref = _b16_reference(c, head)
    grads = _run_bwd(c, levels, ws, g, algorithm)
    ch_dev = torch.from_numpy(B16_CHANNELS).cuda()
    got = from_device(out[:, ch_dev])
    check_fwd(got, fwd_ref, True, "batch-16 %s forward" % head)
    for l in range(len(c.shapes)):
        # the gradient pyramid is fp32 and the oracle reads the same bf16 values, so the
        # fp32 backward tolerance applies
        check_bwd(from_device(grads[l][:, ch_dev]), bwd_ref[l], absref[l], False,
                  "batch-16 %s backward level %d" % (head, l))


def test_forward_is_deterministic_and_plan_independent():
    c = _case(2)
    log("determinism: workload 2 forward x3, with and without plan")
    _, _, a = _run_fwd(c, plan=True)
    _, _, b = _run_fwd(c, plan=True)
    _, _, d = _run_fwd(c, plan=False)
    assert torch.equal(a, b)
    assert torch.equal(a, d)


@pytest.mark.parametrize("algorithm", ["scatter", "gather"])
def test_backward_repeatable_within_tolerance(algorithm):
    c = _case(3)
    log("repeatability: workload 3 backward (%s) x2, and against the other algorithm" % algorithm)
    levels, ws, _ = _run_fwd(c)
    g = c.wl.grad()
    g1 = _run_bwd(c, levels, ws, g, algorithm)
    g2 = _run_bwd(c, levels, ws, g, algorithm)
    g3 = _run_bwd(c, levels, ws, g, "scatter" if algorithm == "gather" else "gather")
    for a, b, d in zip(g1, g2, g3):
        scale = max(a.abs().max().item(), 1e-30)
        assert (a - b).abs().max().item() <= 1e-4 * scale
        assert (a - d).abs().max().item() <= 1e-4 * scale
