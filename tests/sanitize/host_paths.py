"""Valid calls through every entry point of the host-code build (``san_build.py``), at the
workloads' full sizes and at the limits, so that AddressSanitizer and
UndefinedBehaviorSanitizer watch the whole host path: argument checks, workspace
layout, plan sizing (bands, bucket regions), level tables and dispatch.

The launchers of that build do nothing, so device pointers are stand-in addresses
that are never dereferenced.  Collected only when named on the command line, and
skipped unless ``REX_LIBRARY`` names the host-code build.
"""
import ctypes
import os

import pytest

from paper_1906_07155_amd import binding as B
from paper_1906_07155_amd import workloads as W

pytestmark = pytest.mark.skipif(
    not os.environ.get("REX_LIBRARY", "").endswith("_host.so"),
    reason="needs the host-code build of the library")

OK = 0
FAKE = 1 << 20          # a stand-in device address, 256-aligned


@pytest.fixture(scope="module")
def L():
    return B.lib()


def levels_for(wl, layout="cl", dtype=None):
    dt = {"f32": 0, "bf16": 1}[dtype or wl.feat_dtype]
    arr = (B.ReLevel * wl.num_levels)()
    C = wl.channels
    for i, ((h, w), s) in enumerate(zip(wl.level_hw, wl.scales)):
        if layout == "cl":
            st = (h * w * C, 1, w * C, C)
        else:
            st = (C * h * w, h * w, w, 1)
        arr[i] = B.ReLevel(FAKE * (i + 1), dt, 0, wl.n_images, C, h, w, *st, s, 0.0)
    return arr


def workspace(L, lv, nl, K):
    n = ctypes.c_size_t(0)
    assert L.roi_extract_workspace_size(lv, nl, K, ctypes.byref(n)) == OK
    assert n.value % 256 == 0
    return n.value


WLS = [(1, None, None), (2, None, None), (3, None, None), (4, None, "bf16"), (5, "box", None),
       (5, "mask", None)]


@pytest.mark.parametrize("idx,head,fdt", WLS)
@pytest.mark.parametrize("layout", ["cl", "nchw"])
def test_workload_paths(L, idx, head, fdt, layout):
    wl = W.config(idx, head=head, feat_dtype=fdt)
    nl, K = wl.num_levels, wl.num_rois
    lv = levels_for(wl, layout)
    glv = levels_for(wl, layout, "f32")
    oh, ow = wl.out_hw
    odt = {"f32": 0, "bf16": 1}[wl.out_dtype]
    wsb = workspace(L, lv, nl, K)
    for conv in (0, 1):
        assert L.roi_extract_plan_ex(lv, nl, FAKE, K, 56.0, conv, FAKE, FAKE, wsb, None) == OK
    assert L.roi_extract_plan(lv, nl, FAKE, K, 56.0, FAKE, FAKE, wsb, None) == OK
    assert L.roi_extract_plan_offsets(FAKE, wsb, K, nl, FAKE, None) == OK
    for plan, pb in ((FAKE, wsb), (None, 0)):
        assert L.roi_align_fwd(lv, nl, FAKE, K, FAKE, oh, ow, 2, 1, FAKE, odt, plan, pb,
                               None) == OK
        assert L.roi_align_fwd(lv, nl, FAKE, K, FAKE, oh, ow, 0, 0, FAKE, odt, plan, pb,
                               None) == OK
    heads = (B.ReFwdHead * 2)(B.ReFwdHead(FAKE, K, FAKE, oh, ow, 2, 1, FAKE, FAKE, wsb),
                              B.ReFwdHead(FAKE, K // 2, FAKE, 14, 14, 2, 1, FAKE, None, 0))
    assert L.roi_align_fwd_multi(lv, nl, heads, 2, odt, None) == OK
    if K <= 65536:
        assert L.roi_align_fwd_noalloc(lv, nl, FAKE, K, 56.0, FAKE, oh, ow, 2, 1, FAKE, odt,
                                       None) == OK
    gdt = {"f32": 0, "bf16": 1}[wl.grad_dtype]
    for algo in (0, 1, 2):
        for zero in (0, 1):
            assert L.roi_align_bwd(FAKE, gdt, FAKE, K, FAKE, oh, ow, 2, 1, glv, nl, zero, algo,
                                   FAKE, wsb, None) == OK
    assert L.roi_extract_zero_grad(glv, nl, None) == OK
    hd = (B.ReHead * 2)(B.ReHead(FAKE, gdt, oh, ow, 2, 1, 0, FAKE, K, FAKE, FAKE, wsb),
                        B.ReHead(FAKE, gdt, 14, 14, 2, 1, 0, FAKE, K, FAKE, FAKE, wsb))
    for zero in (0, 1):
        assert L.roi_align_bwd_multi(hd, 2, glv, nl, zero, None) == OK
    assert L.roi_pool_fwd(lv, nl, FAKE, K, FAKE, oh, ow, FAKE, odt, FAKE, FAKE, wsb, None) == OK
    assert L.roi_pool_bwd(FAKE, gdt, FAKE, FAKE, K, FAKE, oh, ow, glv, nl, 1, FAKE, wsb,
                          None) == OK
    for mask in (None, FAKE):
        assert L.deform_roi_pool_fwd(lv, nl, FAKE, K, FAKE, oh, ow, 2, 1, FAKE, mask, 0.1,
                                     FAKE, odt, FAKE, wsb, None) == OK
        assert L.deform_roi_pool_bwd(FAKE, gdt, lv, glv, nl, FAKE, K, FAKE, oh, ow, 2, 1, FAKE,
                                     mask, 0.1, 1, FAKE, mask, FAKE, wsb, None) == OK


@pytest.mark.parametrize("K", [0, 1, 255, 8192, 8193, 65536, 1 << 22])
def test_plan_sizes(L, K):
    """Both plan paths (one launch up to 8192 RoIs, five beyond) and the largest K."""
    wl = W.config(5)
    lv = levels_for(wl)
    wsb = workspace(L, lv, wl.num_levels, K)
    assert L.roi_extract_plan(lv, wl.num_levels, FAKE, K, 56.0, FAKE, FAKE, wsb, None) == OK
    glv = levels_for(wl, dtype="f32")
    for algo in (0, 1):
        assert L.roi_align_bwd(FAKE, 1, FAKE, K, FAKE, 7, 7, 2, 1, glv, wl.num_levels, 1, algo,
                               FAKE, wsb, None) == OK
    # 4 Mi RoIs times the 16x16-px tiles of a 200x336 map exceed 2^28 tile-list entries:
    # the plan keeps no tile lists and the gather is refused
    gather = L.roi_align_bwd(FAKE, 1, FAKE, K, FAKE, 7, 7, 2, 1, glv, wl.num_levels, 1, 2,
                             FAKE, wsb, None)
    assert gather == (OK if K < (1 << 22) else 2)


@pytest.mark.parametrize("hw", [(1, 1), (16, 16), (17, 33), (4096, 4096), (1 << 15, 3)])
def test_plan_level_extremes(L, hw):
    """Single-level maps from one pixel to the largest, in the tile plan's arithmetic."""
    arr = (B.ReLevel * 1)(B.ReLevel(FAKE, 0, 0, 3, 64, hw[0], hw[1], hw[0] * hw[1] * 64, 1,
                                    hw[1] * 64, 64, 0.25, 0.0))
    for K in (1, 1000, 9000):
        wsb = workspace(L, arr, 1, K)
        assert L.roi_extract_plan(arr, 1, FAKE, K, 56.0, FAKE, FAKE, wsb, None) == OK
        assert L.roi_align_bwd(FAKE, 0, FAKE, K, FAKE, 7, 7, 2, 1, arr, 1, 0, 0, FAKE, wsb,
                               None) == OK


@pytest.mark.parametrize("N,C", [(1, 1), (1000, 1), (1000, 80), (8192, 1), (1 << 20, 80)])
def test_nms_paths(L, N, C):
    n = ctypes.c_size_t(0)
    if N <= 8192:
        assert L.box_nms_workspace_size(N, ctypes.byref(n)) == OK
        assert L.box_nms(FAKE, FAKE, FAKE if C > 1 else None, N, 0.5, 100, FAKE, FAKE, FAKE,
                         n.value, None) == OK
    assert L.box_nms_batched_workspace_size(N, C, ctypes.byref(n)) == OK
    for method in (0, 1, 2):
        assert L.box_nms_batched(FAKE, FAKE, FAKE, N, C, method, 0.5, 0.5, 0.05, 100, FAKE,
                                 FAKE, FAKE, FAKE, n.value, None) == OK
