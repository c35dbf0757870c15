"""CPU oracle for multi-level RoIAlign, RoI max pooling, deformable RoI pooling and
non-maximum suppression -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path never does, and this
package imports nothing from the GPU library (they share no code).

The arithmetic lives in ``roi_oracle.c`` (plain C, OpenMP over RoIs for the
forward and over channels for the backward).  This module compiles it with gcc
and marshals numpy arrays through ctypes.  Everything it returns is float64.

Paper anchors (MMDetection, arXiv 1906.07155): §3.1 RoIExtractor /
SingleRoIExtractor (per-level RoI feature extraction with a RoI pooling
operator), §2 (Mask R-CNN, whose RoIAlign that operator is), §3.2 (forward and
backward every training iteration).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(_HERE, "roi_oracle.c")
LIBRARY = os.path.join(_HERE, "liboracle.so")

MODE_MATH = 0
MODE_PARITY = 1
_MODES = {"math": MODE_MATH, "parity": MODE_PARITY}

# -ffp-contract=off: one rounding per written operation in the binary32 geometry.
CFLAGS = ["-O2", "-std=c99", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
          "-fPIC", "-shared"]

_lock = threading.Lock()
_lib = None


def build(source: str = SOURCE, output: str = LIBRARY) -> str:
    """Compile the oracle with gcc (always recompiles)."""
    tmp = output + ".tmp%d" % os.getpid()
    subprocess.check_call(["gcc", *CFLAGS, source, "-o", tmp, "-lm"])
    os.replace(tmp, output)
    return output


def _bind(lib):
    f64pp = ctypes.POINTER(ctypes.c_void_p)
    lib.oracle_num_threads.restype = ctypes.c_int
    lib.oracle_level_map.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
                                     ctypes.c_float, ctypes.c_int32, ctypes.c_void_p]
    lib.oracle_level_map.restype = None
    lib.oracle_level_map_log2.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
                                          ctypes.c_double, ctypes.c_int32, ctypes.c_void_p]
    lib.oracle_level_map_log2.restype = None
    lib.oracle_roi_align_fwd.argtypes = [f64pp, ctypes.c_void_p, ctypes.c_void_p,
                                         ctypes.c_int32, ctypes.c_void_p, ctypes.c_int64,
                                         ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                         ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                         ctypes.c_void_p]
    lib.oracle_roi_align_fwd.restype = None
    lib.oracle_roi_align_bwd.argtypes = [ctypes.c_void_p, f64pp, ctypes.c_void_p,
                                         ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                                         ctypes.c_int64, ctypes.c_void_p, ctypes.c_int32,
                                         ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                         ctypes.c_int32]
    lib.oracle_roi_align_bwd.restype = None
    lib.oracle_roi_pool_fwd.argtypes = [f64pp, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_int32, ctypes.c_void_p, ctypes.c_int64,
                                        ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                        ctypes.c_void_p, ctypes.c_void_p]
    lib.oracle_roi_pool_fwd.restype = None
    lib.oracle_roi_pool_bwd.argtypes = [ctypes.c_void_p, ctypes.c_void_p, f64pp,
                                        ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                                        ctypes.c_int64, ctypes.c_void_p, ctypes.c_int32,
                                        ctypes.c_int32]
    lib.oracle_roi_pool_bwd.restype = None
    lib.oracle_deform_roi_pool_fwd.argtypes = [
        f64pp, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
        ctypes.c_int64, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
        ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_float, ctypes.c_int32,
        ctypes.c_void_p]
    lib.oracle_deform_roi_pool_fwd.restype = None
    lib.oracle_deform_roi_pool_bwd.argtypes = [
        ctypes.c_void_p, f64pp, f64pp, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
        ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
        ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_float,
        ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    lib.oracle_deform_roi_pool_bwd.restype = None
    lib.oracle_box_iou.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    lib.oracle_box_iou.restype = ctypes.c_float
    lib.oracle_nms.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                               ctypes.c_float, ctypes.c_int32, ctypes.c_void_p]
    lib.oracle_nms.restype = ctypes.c_int32
    lib.oracle_soft_gauss_weight.argtypes = [ctypes.c_float, ctypes.c_float]
    lib.oracle_soft_gauss_weight.restype = ctypes.c_float
    lib.oracle_nms_batched.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                       ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                       ctypes.c_float, ctypes.c_float, ctypes.c_float,
                                       ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                       ctypes.c_void_p]
    lib.oracle_nms_batched.restype = None
    return lib


def load(path: str | None = None):
    """Load the compiled oracle, building it first if it is not there."""
    global _lib
    with _lock:
        if path is not None:
            return _bind(ctypes.CDLL(path))
        if _lib is None and os.environ.get("ORACLE_LIBRARY"):
            # a prebuilt copy (the sanitizer build), loaded as it is
            _lib = _bind(ctypes.CDLL(os.environ["ORACLE_LIBRARY"]))
        if _lib is None:
            if not os.path.exists(LIBRARY) or (
                    os.path.getmtime(LIBRARY) < os.path.getmtime(SOURCE)):
                build()
            _lib = _bind(ctypes.CDLL(LIBRARY))
        return _lib


def num_threads(lib=None) -> int:
    return int((lib or load()).oracle_num_threads())


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _rois(rois) -> np.ndarray:
    r = np.ascontiguousarray(rois, dtype=np.float32)
    if r.ndim != 2 or r.shape[1] != 5:
        raise ValueError("rois must be [K, 5]")
    return r


def level_map(rois, num_levels: int, finest_scale: float = 56.0, box_plus1: bool = False,
              lib=None) -> np.ndarray:
    """Threshold form of the FPN level rule (binary32 area and thresholds); with
    box_plus1 the sides are (x2 - x1) + 1 (boxes as inclusive pixel ranges)."""
    lib = lib or load()
    r = _rois(rois)
    out = np.zeros(r.shape[0], dtype=np.int32)
    lib.oracle_level_map(_ptr(r), r.shape[0], int(num_levels), float(finest_scale),
                         int(bool(box_plus1)), _ptr(out))
    return out


def level_map_log2(rois, num_levels: int, finest_scale: float = 56.0, box_plus1: bool = False,
                   lib=None) -> np.ndarray:
    """floor(log2(sqrt(area)/finest_scale)) clamped, in double precision."""
    lib = lib or load()
    r = _rois(rois)
    out = np.zeros(r.shape[0], dtype=np.int32)
    lib.oracle_level_map_log2(_ptr(r), r.shape[0], int(num_levels), float(finest_scale),
                              int(bool(box_plus1)), _ptr(out))
    return out


def _level_args(shapes, scales):
    if len(shapes) != len(scales) or not shapes:
        raise ValueError("one scale per level")
    dims = np.ascontiguousarray(np.array([list(s) for s in shapes], dtype=np.int64).reshape(-1))
    sc = np.ascontiguousarray(np.array(scales, dtype=np.float32))
    return dims, sc


def roi_align_fwd(features, scales, rois, roi_levels, out_h: int, out_w: int,
                  sampling_ratio: int, aligned: bool, mode: str = "parity",
                  lib=None) -> np.ndarray:
    """features: list of [N, C, H, W] arrays (any real dtype; read as float64).

    Returns float64 [K, C, out_h, out_w].
    """
    lib = lib or load()
    feats = [np.ascontiguousarray(f, dtype=np.float64) for f in features]
    dims, sc = _level_args([f.shape for f in feats], scales)
    r = _rois(rois)
    K = r.shape[0]
    C = feats[0].shape[1]
    lv = None if roi_levels is None else np.ascontiguousarray(roi_levels, dtype=np.int32)
    out = np.zeros((K, C, out_h, out_w), dtype=np.float64)
    arr = (ctypes.c_void_p * len(feats))(*[f.ctypes.data for f in feats])
    lib.oracle_roi_align_fwd(arr, _ptr(dims), _ptr(sc), len(feats), _ptr(r), K,
                             None if lv is None else _ptr(lv), int(out_h), int(out_w),
                             int(sampling_ratio), int(bool(aligned)), _MODES[mode], _ptr(out))
    return out


def roi_align_bwd(grad_out, shapes, scales, rois, roi_levels, out_h: int, out_w: int,
                  sampling_ratio: int, aligned: bool, mode: str = "parity",
                  lib=None) -> list:
    """Transpose of roi_align_fwd.  shapes: list of (N, C, H, W) per level.

    Returns a list of float64 gradient arrays, one per level.
    """
    lib = lib or load()
    g = np.ascontiguousarray(grad_out, dtype=np.float64)
    dims, sc = _level_args(shapes, scales)
    r = _rois(rois)
    K = r.shape[0]
    if g.shape != (K, shapes[0][1], out_h, out_w):
        raise ValueError("grad_out must be [K, C, out_h, out_w]")
    lv = None if roi_levels is None else np.ascontiguousarray(roi_levels, dtype=np.int32)
    grads = [np.zeros(tuple(s), dtype=np.float64) for s in shapes]
    arr = (ctypes.c_void_p * len(grads))(*[x.ctypes.data for x in grads])
    lib.oracle_roi_align_bwd(_ptr(g), arr, _ptr(dims), _ptr(sc), len(grads), _ptr(r), K,
                             None if lv is None else _ptr(lv), int(out_h), int(out_w),
                             int(sampling_ratio), int(bool(aligned)), _MODES[mode])
    return grads


def roi_pool_fwd(features, scales, rois, roi_levels, out_h: int, out_w: int, lib=None):
    """RoI max pooling.  Returns (float64 [K, C, out_h, out_w], int32 argmax of the
    same shape: y * W + x within the RoI's (level, image, channel) plane, -1 for none)."""
    lib = lib or load()
    feats = [np.ascontiguousarray(f, dtype=np.float64) for f in features]
    dims, sc = _level_args([f.shape for f in feats], scales)
    r = _rois(rois)
    K = r.shape[0]
    C = feats[0].shape[1]
    lv = None if roi_levels is None else np.ascontiguousarray(roi_levels, dtype=np.int32)
    out = np.zeros((K, C, out_h, out_w), dtype=np.float64)
    am = np.full((K, C, out_h, out_w), -1, dtype=np.int32)
    arr = (ctypes.c_void_p * len(feats))(*[f.ctypes.data for f in feats])
    lib.oracle_roi_pool_fwd(arr, _ptr(dims), _ptr(sc), len(feats), _ptr(r), K,
                            None if lv is None else _ptr(lv), int(out_h), int(out_w),
                            _ptr(out), _ptr(am))
    return out, am


def roi_pool_bwd(grad_out, argmax, shapes, rois, roi_levels, lib=None) -> list:
    """Each output gradient added to its argmax pixel.  Returns float64 gradients."""
    lib = lib or load()
    g = np.ascontiguousarray(grad_out, dtype=np.float64)
    am = np.ascontiguousarray(argmax, dtype=np.int32)
    dims, _ = _level_args(shapes, [1.0] * len(shapes))
    r = _rois(rois)
    K = r.shape[0]
    if g.shape != am.shape or g.shape[:2] != (K, shapes[0][1]):
        raise ValueError("grad_out and argmax must be [K, C, out_h, out_w]")
    lv = None if roi_levels is None else np.ascontiguousarray(roi_levels, dtype=np.int32)
    grads = [np.zeros(tuple(s), dtype=np.float64) for s in shapes]
    arr = (ctypes.c_void_p * len(grads))(*[x.ctypes.data for x in grads])
    lib.oracle_roi_pool_bwd(_ptr(g), _ptr(am), arr, _ptr(dims), len(grads), _ptr(r), K,
                            None if lv is None else _ptr(lv), int(g.shape[2]), int(g.shape[3]))
    return grads


def _deform_args(rois, roi_levels, offset, mask, out_h, out_w):
    r = _rois(rois)
    K = r.shape[0]
    off = np.ascontiguousarray(offset, dtype=np.float32)
    if off.shape != (K, 2, out_h, out_w):
        raise ValueError("offset must be [K, 2, out_h, out_w]")
    m = None if mask is None else np.ascontiguousarray(mask, dtype=np.float32)
    if m is not None and m.shape != (K, out_h, out_w):
        raise ValueError("mask must be [K, out_h, out_w]")
    lv = None if roi_levels is None else np.ascontiguousarray(roi_levels, dtype=np.int32)
    return r, K, off, m, lv


def deform_roi_pool_fwd(features, scales, rois, roi_levels, out_h: int, out_w: int,
                        sampling_ratio: int, aligned: bool, offset, mask=None,
                        gamma: float = 0.1, mode: str = "parity", lib=None) -> np.ndarray:
    """Deformable (modulated when `mask` is given) RoI pooling: RoIAlign bins shifted by
    gamma * offset * box length and scaled by the mask.  offset [K, 2, out_h, out_w]
    (x then y, normalized), mask [K, out_h, out_w] or None.  Returns float64 [K, C, ...]."""
    lib = lib or load()
    feats = [np.ascontiguousarray(f, dtype=np.float64) for f in features]
    dims, sc = _level_args([f.shape for f in feats], scales)
    r, K, off, m, lv = _deform_args(rois, roi_levels, offset, mask, out_h, out_w)
    out = np.zeros((K, feats[0].shape[1], out_h, out_w), dtype=np.float64)
    arr = (ctypes.c_void_p * len(feats))(*[f.ctypes.data for f in feats])
    lib.oracle_deform_roi_pool_fwd(arr, _ptr(dims), _ptr(sc), len(feats), _ptr(r), K,
                                   None if lv is None else _ptr(lv), int(out_h), int(out_w),
                                   int(sampling_ratio), int(bool(aligned)), _ptr(off),
                                   None if m is None else _ptr(m), float(gamma), _MODES[mode],
                                   _ptr(out))
    return out


def deform_roi_pool_bwd(grad_out, features, scales, rois, roi_levels, out_h: int, out_w: int,
                        sampling_ratio: int, aligned: bool, offset, mask=None,
                        gamma: float = 0.1, mode: str = "parity", lib=None):
    """Gradients of deform_roi_pool_fwd.  Returns (feature gradients per level, grad_offset
    [K, 2, out_h, out_w], grad_mask [K, out_h, out_w] or None, and the absolute-value sums
    scale_offset, scale_mask of the same shapes)."""
    lib = lib or load()
    feats = [np.ascontiguousarray(f, dtype=np.float64) for f in features]
    shapes = [f.shape for f in feats]
    dims, sc = _level_args(shapes, scales)
    r, K, off, m, lv = _deform_args(rois, roi_levels, offset, mask, out_h, out_w)
    g = np.ascontiguousarray(grad_out, dtype=np.float64)
    if g.shape != (K, shapes[0][1], out_h, out_w):
        raise ValueError("grad_out must be [K, C, out_h, out_w]")
    grads = [np.zeros(s, dtype=np.float64) for s in shapes]
    goff = np.zeros((K, 2, out_h, out_w), dtype=np.float64)
    soff = np.zeros_like(goff)
    gm = np.zeros((K, out_h, out_w), dtype=np.float64) if m is not None else None
    sm = np.zeros((K, out_h, out_w), dtype=np.float64) if m is not None else None
    farr = (ctypes.c_void_p * len(feats))(*[f.ctypes.data for f in feats])
    garr = (ctypes.c_void_p * len(grads))(*[x.ctypes.data for x in grads])
    lib.oracle_deform_roi_pool_bwd(_ptr(g), farr, garr, _ptr(dims), _ptr(sc), len(feats), _ptr(r),
                                   K, None if lv is None else _ptr(lv), int(out_h), int(out_w),
                                   int(sampling_ratio), int(bool(aligned)), _ptr(off),
                                   None if m is None else _ptr(m), float(gamma), _MODES[mode],
                                   _ptr(goff), None if gm is None else _ptr(gm), _ptr(soff),
                                   None if sm is None else _ptr(sm))
    return grads, goff, gm, soff, sm


def box_iou(a, b, lib=None) -> float:
    """Binary32 IoU of two boxes (x1, y1, x2, y2), one rounding per operation."""
    lib = lib or load()
    a = np.ascontiguousarray(a, dtype=np.float32)
    b = np.ascontiguousarray(b, dtype=np.float32)
    return float(lib.oracle_box_iou(_ptr(a), _ptr(b)))


def nms(boxes, scores, threshold: float, categories=None, max_keep: int | None = None,
        lib=None) -> np.ndarray:
    """Greedy NMS: kept box indices (int32) in rank order."""
    lib = lib or load()
    bx = np.ascontiguousarray(boxes, dtype=np.float32)
    sc = np.ascontiguousarray(scores, dtype=np.float32)
    N = sc.shape[0]
    if bx.shape != (N, 4):
        raise ValueError("boxes must be [N, 4]")
    cats = None if categories is None else np.ascontiguousarray(categories, dtype=np.int32)
    keep = np.zeros(max(N, 1), dtype=np.int32)
    n = lib.oracle_nms(_ptr(bx), _ptr(sc), None if cats is None else _ptr(cats), N,
                       float(threshold), N if max_keep is None else int(max_keep), _ptr(keep))
    return keep[:n].copy()


NMS_METHODS = {"hard": 0, "linear": 1, "gaussian": 2}


def soft_gauss_weight(iou: float, sigma: float, lib=None) -> float:
    """Binary32 Gaussian decay weight exp(-iou^2 / sigma) of Soft-NMS (1 for iou <= 0 or
    NaN)."""
    lib = lib or load()
    return float(lib.oracle_soft_gauss_weight(float(iou), float(sigma)))


def nms_batched(boxes, scores, categories, num_categories: int, method: str = "hard",
                iou_threshold: float = 0.5, sigma: float = 0.5,
                score_threshold: float = float("-inf"), max_keep: int | None = None, lib=None):
    """Per-category proposal selection: greedy NMS ("hard") or Soft-NMS with linear or
    Gaussian decay.  Returns (keep [C, max_keep] int32 padded with -1, scores
    [C, max_keep] float32 padded with 0, num_keep [C] int32)."""
    lib = lib or load()
    bx = np.ascontiguousarray(boxes, dtype=np.float32)
    sc = np.ascontiguousarray(scores, dtype=np.float32)
    N = sc.shape[0]
    if bx.shape != (N, 4):
        raise ValueError("boxes must be [N, 4]")
    cats = None if categories is None else np.ascontiguousarray(categories, dtype=np.int32)
    mk = N if max_keep is None else int(max_keep)
    C = int(num_categories)
    keep = np.zeros((C, max(mk, 1)), dtype=np.int32)
    kept_scores = np.zeros((C, max(mk, 1)), dtype=np.float32)
    num = np.zeros(C, dtype=np.int32)
    lib.oracle_nms_batched(_ptr(bx), _ptr(sc), None if cats is None else _ptr(cats), N, C,
                           NMS_METHODS[method], float(iou_threshold), float(sigma),
                           float(score_threshold), mk, _ptr(keep), _ptr(kept_scores),
                           _ptr(num))
    return keep[:, :mk].copy(), kept_scores[:, :mk].copy(), num
