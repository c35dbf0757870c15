"""The C ABI on the host: the library loads, exports every declared symbol, and
rejects bad arguments with its documented status codes before enqueuing anything.

No call here reaches a kernel launch, so these run without a GPU.  Device pointers
are stand-in addresses that the library never dereferences on an error path.
"""
import ctypes
import math
import subprocess

import pytest

from paper_1906_07155_amd import binding as B

OK, INVALID, UNSUPPORTED, WORKSPACE, DEVICE = range(5)
FAKE = 0x10000          # a 64 KiB-aligned stand-in device address (never dereferenced)


@pytest.fixture(scope="module")
def L():
    return B.lib()


def test_exports_every_declared_symbol(L):
    names = B.header_functions()
    assert len(names) >= 10
    out = subprocess.check_output(["nm", "-D", "--defined-only", B.LIBRARY]).decode()
    exported = {line.split()[-1] for line in out.splitlines() if line.strip()}
    for n in names:
        assert n in exported, n
        assert hasattr(L, n)


def test_status_strings_and_version(L):
    for s in range(5):
        assert L.roi_extract_status_str(s)
    assert b"unknown" in L.roi_extract_status_str(99)
    assert b"gfx950" in L.roi_extract_version()


def test_workspace_size(L):
    lv = _levels()
    n = ctypes.c_size_t(0)
    assert L.roi_extract_workspace_size(lv, 2, 0, ctypes.byref(n)) == OK
    base = n.value
    assert L.roi_extract_workspace_size(lv, 2, 1024, ctypes.byref(n)) == OK
    # perm + keys (8 B per RoI) + tile lists (4 B per RoI and tile of the largest map:
    # 16x20 px in 16-px tiles = 2 tiles)
    assert n.value >= 8 * 1024 + 4 * 1024 * 2 and n.value > base and n.value % 256 == 0
    assert L.roi_extract_workspace_size(lv, 2, -1, ctypes.byref(n)) == INVALID
    assert L.roi_extract_workspace_size(lv, 0, 10, ctypes.byref(n)) == INVALID
    assert L.roi_extract_workspace_size(lv, 9, 10, ctypes.byref(n)) == INVALID
    assert L.roi_extract_workspace_size(lv, 2, 10, None) == INVALID
    assert L.roi_extract_workspace_size(None, 2, 10, ctypes.byref(n)) == INVALID


def _levels(n=2, c=8, hw=((16, 20), (8, 10)), dtype=0, scales=(0.25, 0.125), data=FAKE):
    arr = (B.ReLevel * len(hw))()
    for i, ((h, w), s) in enumerate(zip(hw, scales)):
        # channels-last strides
        arr[i] = B.ReLevel(data, dtype, 0, n, c, h, w, h * w * c, 1, w * c, c, s, 0.0)
    return arr


def _fwd(L, levels=None, nl=2, rois=FAKE, K=4, roi_levels=FAKE, oh=7, ow=7, sr=2, al=1,
         out=FAKE, odt=0, plan=None, plan_bytes=0):
    levels = levels if levels is not None else _levels()
    return L.roi_align_fwd(levels, nl, rois, K, roi_levels, oh, ow, sr, al, out, odt, plan,
                           plan_bytes, None)


def _bwd(L, levels=None, nl=2, gout=FAKE, gdt=0, K=4, zero=0, sr=2, al=1, oh=7, ow=7,
         plan=None, plan_bytes=0, algo=0):
    levels = levels if levels is not None else _levels()
    return L.roi_align_bwd(gout, gdt, FAKE, K, FAKE, oh, ow, sr, al, levels, nl, zero, algo,
                           plan, plan_bytes, None)


def test_level_map_validation(L):
    assert L.fpn_level_map(FAKE, -1, 4, 56.0, FAKE, None) == INVALID
    assert L.fpn_level_map(FAKE, 3, 0, 56.0, FAKE, None) == INVALID
    assert L.fpn_level_map(FAKE, 3, 9, 56.0, FAKE, None) == INVALID
    for s in (0.0, -1.0, math.inf, math.nan):
        assert L.fpn_level_map(FAKE, 3, 4, s, FAKE, None) == INVALID
    assert L.fpn_level_map(None, 3, 4, 56.0, FAKE, None) == INVALID
    assert L.fpn_level_map(FAKE, 3, 4, 56.0, None, None) == INVALID
    assert L.fpn_level_map(FAKE + 2, 3, 4, 56.0, FAKE, None) == INVALID
    assert L.fpn_level_map(None, 0, 4, 56.0, None, None) == OK      # nothing to do


def test_level_map_box_convention_validation(L):
    # only RE_BOX_CONTINUOUS (0) and RE_BOX_PIXELS (1); checked before anything else
    for conv in (-1, 2, 7):
        assert L.fpn_level_map_ex(FAKE, 3, 4, 56.0, conv, FAKE, None) == INVALID
        assert L.fpn_level_map_ex(None, 0, 4, 56.0, conv, None, None) == INVALID
    assert L.fpn_level_map_ex(None, 0, 4, 56.0, 1, None, None) == OK
    assert L.fpn_level_map_ex(FAKE, 3, 0, 56.0, 1, FAKE, None) == INVALID


def test_forward_validation(L):
    assert _fwd(L, K=0) == OK                                      # nothing to do
    assert _fwd(L, levels=None, nl=0) == INVALID
    assert _fwd(L, nl=9) == INVALID
    assert L.roi_align_fwd(None, 2, FAKE, 4, FAKE, 7, 7, 2, 1, FAKE, 0, None, 0, None) == INVALID
    assert _fwd(L, K=-1) == INVALID
    assert _fwd(L, K=(1 << 22) + 1) == INVALID
    assert _fwd(L, rois=None) == INVALID
    assert _fwd(L, rois=FAKE + 1) == INVALID
    assert _fwd(L, roi_levels=None) == INVALID                     # several levels need them
    assert _fwd(L, oh=0) == INVALID
    assert _fwd(L, ow=257) == INVALID
    assert _fwd(L, sr=-1) == INVALID
    assert _fwd(L, sr=65) == INVALID
    assert _fwd(L, al=2) == INVALID
    assert _fwd(L, out=None) == INVALID
    assert _fwd(L, odt=7) == INVALID
    assert _fwd(L, odt=0, out=FAKE + 2) == INVALID                 # fp32 output misaligned
    assert _fwd(L, plan=FAKE, plan_bytes=16) == WORKSPACE
    assert _fwd(L, plan=FAKE + 64, plan_bytes=1 << 20) == WORKSPACE  # plan not 256-aligned


@pytest.mark.parametrize("field,value", [
    ("dtype", 5), ("reserved", 1), ("n", 0), ("c", 0), ("h", 0), ("w", 0), ("h", 1 << 24),
    ("stride_h", -1), ("spatial_scale", 0.0), ("spatial_scale", -0.5),
    ("spatial_scale", math.inf), ("spatial_scale", math.nan), ("data", None),
    ("reserved2", 1.0)])
def test_forward_rejects_bad_level(L, field, value):
    lv = _levels()
    setattr(lv[1], field, value)
    assert _fwd(L, levels=lv) == INVALID


def test_forward_rejects_mismatched_levels(L):
    lv = _levels()
    lv[1].n = 3
    assert _fwd(L, levels=lv) == INVALID
    lv = _levels()
    lv[1].c = 16
    assert _fwd(L, levels=lv) == INVALID
    lv = _levels()
    lv[1].dtype = 1
    assert _fwd(L, levels=lv) == INVALID
    lv = _levels(data=FAKE + 2)                                    # fp32 data misaligned
    assert _fwd(L, levels=lv) == INVALID


def test_backward_validation(L):
    assert _bwd(L, levels=_levels(dtype=1)) == UNSUPPORTED         # gradient levels must be fp32
    assert _bwd(L, zero=2) == INVALID
    assert _bwd(L, gout=None) == INVALID
    assert _bwd(L, gdt=3) == INVALID
    assert _bwd(L, gdt=0, gout=FAKE + 2) == INVALID
    assert _bwd(L, sr=-2) == INVALID
    assert _bwd(L, plan=FAKE, plan_bytes=8) == WORKSPACE
    assert _bwd(L, K=0, zero=0) == OK                              # nothing to do
    assert _bwd(L, algo=3) == INVALID
    assert _bwd(L, algo=2) == UNSUPPORTED                          # gather needs a plan
    n = ctypes.c_size_t(0)
    assert L.roi_extract_workspace_size(_levels(), 2, 4, ctypes.byref(n)) == OK
    assert _bwd(L, algo=2, plan=FAKE, plan_bytes=n.value, oh=5) == UNSUPPORTED   # 5x7 grid
    assert _bwd(L, algo=2, plan=FAKE, plan_bytes=n.value, sr=0) == UNSUPPORTED   # adaptive
    # the gather stores through 32-bit buffer offsets: levels whose images span 2^30
    # bytes or more (here a channel stride of 2^28 elements) take the scatter only
    wide = _levels()
    for i in range(2):
        wide[i].stride_c, wide[i].stride_h, wide[i].stride_w = 1 << 28, wide[i].w, 1
        wide[i].stride_n = wide[i].c << 28
    assert _bwd(L, levels=wide, algo=2, plan=FAKE, plan_bytes=n.value) == UNSUPPORTED
    assert L.roi_extract_zero_grad(_levels(dtype=1), 2, None) == UNSUPPORTED
    assert L.roi_extract_zero_grad(None, 2, None) == INVALID


def test_plan_validation(L):
    lv = _levels()
    n = ctypes.c_size_t(0)
    assert L.roi_extract_workspace_size(lv, 2, 4, ctypes.byref(n)) == OK
    assert L.roi_extract_plan(lv, 2, FAKE, 4, 56.0, FAKE, None, n.value, None) == WORKSPACE
    assert L.roi_extract_plan(lv, 2, FAKE, 4, 56.0, FAKE, FAKE, n.value - 1, None) == WORKSPACE
    assert L.roi_extract_plan(lv, 2, FAKE, 4, 0.0, FAKE, FAKE, n.value, None) == INVALID
    assert L.roi_extract_plan(lv, 2, None, 4, 56.0, FAKE, FAKE, n.value, None) == INVALID
    assert L.roi_extract_plan(lv, 0, FAKE, 4, 56.0, FAKE, FAKE, n.value, None) == INVALID
    for conv in (-1, 2):
        assert L.roi_extract_plan_ex(lv, 2, FAKE, 4, 56.0, conv, FAKE, FAKE, n.value,
                                     None) == INVALID
    assert L.roi_extract_plan_ex(lv, 2, FAKE, 4, 56.0, 1, FAKE, None, n.value, None) == WORKSPACE
    p = ctypes.c_void_p(0)
    assert L.roi_extract_plan_perm(FAKE, n.value, 4, ctypes.byref(p)) == OK
    assert p.value == FAKE + 256                                   # perm follows the header
    assert L.roi_extract_plan_perm(FAKE, 16, 4, ctypes.byref(p)) == WORKSPACE
    assert L.roi_extract_plan_perm(None, n.value, 4, ctypes.byref(p)) == INVALID
    assert L.roi_extract_plan_offsets(FAKE, n.value, 4, 0, FAKE, None) == INVALID


def test_binding_fails_loudly_without_library(tmp_path):
    with pytest.raises(RuntimeError):
        B.lib(str(tmp_path / "missing.so"))


def _pfwd(L, levels=None, nl=2, K=4, oh=7, ow=7, out=FAKE, odt=0, am=FAKE, plan=None,
          plan_bytes=0):
    levels = levels if levels is not None else _levels()
    return L.roi_pool_fwd(levels, nl, FAKE, K, FAKE, oh, ow, out, odt, am, plan, plan_bytes,
                          None)


def _pbwd(L, levels=None, nl=2, gout=FAKE, gdt=0, am=FAKE, K=4, zero=0, oh=7, ow=7, plan=None,
          plan_bytes=0):
    levels = levels if levels is not None else _levels()
    return L.roi_pool_bwd(gout, gdt, am, FAKE, K, FAKE, oh, ow, levels, nl, zero, plan,
                          plan_bytes, None)


def test_pool_forward_validation(L):
    assert _pfwd(L, K=0) == OK                                     # nothing to do
    assert _pfwd(L, nl=0) == INVALID
    assert _pfwd(L, K=-1) == INVALID
    assert _pfwd(L, oh=0) == INVALID
    assert _pfwd(L, ow=257) == INVALID
    assert _pfwd(L, out=None) == INVALID
    assert _pfwd(L, am=None) == INVALID
    assert _pfwd(L, am=FAKE + 2) == INVALID                        # int32 argmax misaligned
    assert _pfwd(L, odt=9) == INVALID
    assert _pfwd(L, odt=0, out=FAKE + 2) == INVALID
    assert _pfwd(L, plan=FAKE, plan_bytes=16) == WORKSPACE
    big = _levels(hw=((1 << 16, 1 << 15), (8, 10)))                 # H*W = 2^31: argmax overflows
    assert _pfwd(L, levels=big) == INVALID
    assert L.roi_pool_fwd(_levels(), 2, FAKE, 4, None, 7, 7, FAKE, 0, FAKE, None, 0,
                          None) == INVALID                         # several levels need indices


def test_pool_backward_validation(L):
    assert _pbwd(L, levels=_levels(dtype=1)) == UNSUPPORTED        # gradient levels must be fp32
    assert _pbwd(L, zero=2) == INVALID
    assert _pbwd(L, gout=None) == INVALID
    assert _pbwd(L, am=None) == INVALID
    assert _pbwd(L, am=FAKE + 1) == INVALID
    assert _pbwd(L, gdt=4) == INVALID
    assert _pbwd(L, gdt=0, gout=FAKE + 2) == INVALID
    assert _pbwd(L, oh=0) == INVALID
    assert _pbwd(L, plan=FAKE, plan_bytes=8) == WORKSPACE
    assert _pbwd(L, K=0, zero=0) == OK                             # nothing to do


def _head(gout=FAKE, gdt=0, K=4, oh=7, ow=7, sr=2, al=1, reserved=0, plan=None, plan_bytes=0,
          rois=FAKE, roi_levels=FAKE):
    return B.ReHead(gout, gdt, oh, ow, sr, al, reserved, rois, K, roi_levels, plan, plan_bytes)


def _multi(L, heads, nl=2, zero=0, levels=None, n=None):
    levels = levels if levels is not None else _levels()
    arr = (B.ReHead * max(1, len(heads)))(*heads)
    return L.roi_align_bwd_multi(arr, len(heads) if n is None else n, levels, nl, zero, None)


def test_multi_head_backward_validation(L):
    assert _multi(L, [_head(K=0)]) == OK                           # nothing to do
    assert _multi(L, [_head(K=0), _head(K=0, oh=14, ow=14)]) == OK
    assert _multi(L, [_head()], n=0) == INVALID
    assert _multi(L, [_head()] * 9) == INVALID                     # more than RE_MAX_HEADS
    assert L.roi_align_bwd_multi(None, 1, _levels(), 2, 0, None) == INVALID
    assert _multi(L, [_head(), _head(reserved=1)]) == INVALID
    assert _multi(L, [_head(), _head(gout=None)]) == INVALID
    assert _multi(L, [_head(), _head(gdt=5)]) == INVALID
    assert _multi(L, [_head(), _head(oh=0)]) == INVALID
    assert _multi(L, [_head(), _head(sr=-1)]) == INVALID
    assert _multi(L, [_head(), _head(roi_levels=None)]) == INVALID  # several levels
    assert _multi(L, [_head(plan=FAKE, plan_bytes=8)]) == WORKSPACE
    assert _multi(L, [_head()], zero=3) == INVALID
    assert _multi(L, [_head()], levels=_levels(dtype=1)) == UNSUPPORTED   # fp32 gradients only


def _fhead(K=4, oh=7, ow=7, sr=2, al=1, out=FAKE, plan=None, plan_bytes=0, rois=FAKE,
           roi_levels=FAKE):
    return B.ReFwdHead(rois, K, roi_levels, oh, ow, sr, al, out, plan, plan_bytes)


def _fmulti(L, heads, nl=2, odt=0, levels=None, n=None):
    levels = levels if levels is not None else _levels()
    arr = (B.ReFwdHead * max(1, len(heads)))(*heads)
    return L.roi_align_fwd_multi(levels, nl, arr, len(heads) if n is None else n, odt, None)


def test_multi_head_forward_validation(L):
    assert _fmulti(L, [_fhead(K=0)]) == OK                         # nothing to do
    assert _fmulti(L, [_fhead(K=0), _fhead(K=0, oh=14, ow=14, out=None)]) == OK
    assert _fmulti(L, [_fhead()], n=0) == INVALID
    assert _fmulti(L, [_fhead()] * 9) == INVALID                   # more than RE_MAX_HEADS
    assert L.roi_align_fwd_multi(_levels(), 2, None, 1, 0, None) == INVALID
    assert _fmulti(L, [_fhead()], levels=None, nl=0) == INVALID
    assert _fmulti(L, [_fhead()], odt=7) == INVALID
    # a bad head anywhere in the list is refused before any head is launched
    assert _fmulti(L, [_fhead(), _fhead(out=None)]) == INVALID
    assert _fmulti(L, [_fhead(), _fhead(out=FAKE + 2)]) == INVALID   # fp32 output misaligned
    assert _fmulti(L, [_fhead(), _fhead(oh=0)]) == INVALID
    assert _fmulti(L, [_fhead(), _fhead(sr=65)]) == INVALID
    assert _fmulti(L, [_fhead(), _fhead(al=2)]) == INVALID
    assert _fmulti(L, [_fhead(), _fhead(K=-1)]) == INVALID
    assert _fmulti(L, [_fhead(), _fhead(rois=None)]) == INVALID
    assert _fmulti(L, [_fhead(), _fhead(roi_levels=None)]) == INVALID  # several levels
    assert _fmulti(L, [_fhead(), _fhead(plan=FAKE, plan_bytes=8)]) == WORKSPACE


def test_deform_validation(L):
    def fwd(levels=None, K=4, off=FAKE, mask=None, gamma=0.1, out=FAKE, odt=0, sr=2, oh=7):
        lv = levels if levels is not None else _levels()
        return L.deform_roi_pool_fwd(lv, 2, FAKE, K, FAKE, oh, 7, sr, 1, off, mask, gamma, out,
                                     odt, None, 0, None)

    def bwd(levels=None, glevels=None, K=4, off=FAKE, mask=None, goff=FAKE, gmask=None, zero=0,
            gdt=0):
        lv = levels if levels is not None else _levels()
        gl = glevels if glevels is not None else _levels()
        return L.deform_roi_pool_bwd(FAKE, gdt, lv, gl, 2, FAKE, K, FAKE, 7, 7, 2, 1, off, mask,
                                     0.1, zero, goff, gmask, None, 0, None)

    assert fwd(K=0) == OK
    assert fwd(off=None) == INVALID
    assert fwd(off=FAKE + 2) == INVALID
    assert fwd(mask=FAKE + 1) == INVALID
    assert fwd(gamma=math.inf) == INVALID
    assert fwd(gamma=math.nan) == INVALID
    assert fwd(out=None) == INVALID
    assert fwd(odt=3) == INVALID
    assert fwd(sr=-1) == INVALID
    assert fwd(oh=0) == INVALID
    assert bwd(K=0) == OK
    assert bwd(glevels=_levels(dtype=1)) == UNSUPPORTED
    assert bwd(glevels=_levels(hw=((16, 21), (8, 10)))) == INVALID      # shapes differ
    assert bwd(glevels=_levels(scales=(0.5, 0.125))) == INVALID         # scales differ
    assert bwd(goff=None) == INVALID
    assert bwd(gmask=FAKE) == INVALID                                  # mask gradient, no mask
    assert bwd(off=None) == INVALID
    assert bwd(zero=5) == INVALID
    assert bwd(gdt=2) == INVALID


def test_nms_validation(L):
    n = ctypes.c_size_t(0)
    assert L.box_nms_workspace_size(100, ctypes.byref(n)) == OK and n.value >= 100 * (4 + 16 + 4 + 16)
    assert L.box_nms_workspace_size(-1, ctypes.byref(n)) == INVALID
    assert L.box_nms_workspace_size(8193, ctypes.byref(n)) == INVALID
    assert L.box_nms_workspace_size(10, None) == INVALID

    def nms(N=100, boxes=FAKE, scores=FAKE, cats=None, thr=0.5, mk=100, keep=FAKE, nk=FAKE,
            ws=FAKE, wsb=None):
        return L.box_nms(boxes, scores, cats, N, thr, mk, keep, nk, ws,
                         n.value if wsb is None else wsb, None)

    assert L.box_nms_workspace_size(100, ctypes.byref(n)) == OK
    assert nms(N=8193) == UNSUPPORTED
    assert nms(N=-1) == INVALID
    assert nms(thr=math.nan) == INVALID
    assert nms(mk=-1) == INVALID
    assert nms(nk=None) == INVALID
    assert nms(boxes=None) == INVALID
    assert nms(scores=None) == INVALID
    assert nms(keep=None) == INVALID
    assert nms(boxes=FAKE + 2) == INVALID
    assert nms(cats=FAKE + 1) == INVALID
    assert nms(ws=None) == WORKSPACE
    assert nms(ws=FAKE + 64) == WORKSPACE
    assert nms(wsb=16) == WORKSPACE


def test_nms_batched_validation(L):
    n = ctypes.c_size_t(0)
    assert L.box_nms_batched_workspace_size(1000, 16, ctypes.byref(n)) == OK
    assert n.value >= 1000 * 48 and n.value % 256 == 0
    assert L.box_nms_batched_workspace_size(-1, 16, ctypes.byref(n)) == INVALID
    assert L.box_nms_batched_workspace_size(10, 0, ctypes.byref(n)) == INVALID
    assert L.box_nms_batched_workspace_size(10, 8193, ctypes.byref(n)) == INVALID
    assert L.box_nms_batched_workspace_size((1 << 24) + 1, 1, ctypes.byref(n)) == INVALID
    assert L.box_nms_batched_workspace_size(10, 4, None) == INVALID
    assert L.box_nms_batched_workspace_size(1000, 16, ctypes.byref(n)) == OK

    def call(N=1000, C=16, boxes=FAKE, scores=FAKE, cats=FAKE, method=0, thr=0.5, sigma=0.5,
             st=-math.inf, mk=100, keep=FAKE, ks=FAKE, nk=FAKE, ws=FAKE, wsb=None):
        return L.box_nms_batched(boxes, scores, cats, N, C, method, thr, sigma, st, mk, keep, ks,
                                 nk, ws, n.value if wsb is None else wsb, None)

    assert call(C=0) == INVALID
    assert call(cats=None) == INVALID               # several categories need the array
    assert call(method=3) == INVALID
    assert call(thr=math.nan) == INVALID
    assert call(st=math.nan) == INVALID
    assert call(method=2, sigma=0.0) == INVALID
    assert call(method=2, sigma=math.inf) == INVALID
    assert call(mk=-1) == INVALID
    assert call(mk=1 << 28) == INVALID              # max_keep * categories >= 2^31
    assert call(nk=None) == INVALID
    assert call(keep=None) == INVALID
    assert call(ks=None) == INVALID
    assert call(boxes=None) == INVALID
    assert call(scores=FAKE + 2) == INVALID
    assert call(ws=None) == WORKSPACE
    assert call(ws=FAKE + 64) == WORKSPACE
    assert call(wsb=256) == WORKSPACE
