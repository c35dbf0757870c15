"""Thin ctypes binding of libroi_extract.so (argument marshalling only).

Every operation runs in the library's HIP kernels; this module only turns torch
tensors into the pointers, sizes and strides the C ABI (include/roi_extract.h)
takes, and passes torch's current HIP stream.  PyTorch is used for device memory
and streams.  If the library is not built, loading fails loudly: there is no
fallback path.

Paper anchors (MMDetection, arXiv 1906.07155): §3.1 RoIExtractor /
SingleRoIExtractor (level map + RoI feature extraction), §3.2 (forward and
backward every iteration).
"""
from __future__ import annotations

import ctypes
import os
import re
import threading
from typing import List, Optional, Sequence, Tuple

HERE = os.path.dirname(os.path.abspath(__file__))
# REX_LIBRARY names another build of the same library (the host-code build that the
# sanitizer tests load); unset, the in-tree library is loaded.
LIBRARY = os.environ.get("REX_LIBRARY") or os.path.join(HERE, "libroi_extract.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "roi_extract.h")

RE_OK, RE_ERR_INVALID_ARG, RE_ERR_UNSUPPORTED, RE_ERR_WORKSPACE, RE_ERR_DEVICE = range(5)
RE_DTYPE_F32, RE_DTYPE_BF16 = 0, 1
BWD_AUTO, BWD_SCATTER, BWD_GATHER = 0, 1, 2
NMS_METHODS = {"hard": 0, "linear": 1, "gaussian": 2}   # RE_NMS_HARD / _LINEAR / _GAUSSIAN
_BWD_ALGOS = {"auto": BWD_AUTO, "scatter": BWD_SCATTER, "gather": BWD_GATHER}
MAX_LEVELS = 8
MAX_HEADS = 8


class RoIExtractError(RuntimeError):
    def __init__(self, status: int, where: str, text: str):
        super().__init__("%s failed: %s (status %d)" % (where, text, status))
        self.status = status


class ReLevel(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("dtype", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("n", ctypes.c_int64), ("c", ctypes.c_int64),
                ("h", ctypes.c_int64), ("w", ctypes.c_int64), ("stride_n", ctypes.c_int64),
                ("stride_c", ctypes.c_int64), ("stride_h", ctypes.c_int64),
                ("stride_w", ctypes.c_int64), ("spatial_scale", ctypes.c_float),
                ("reserved2", ctypes.c_float)]


class ReHead(ctypes.Structure):
    _fields_ = [("grad_out", ctypes.c_void_p), ("grad_out_dtype", ctypes.c_int32),
                ("out_h", ctypes.c_int32), ("out_w", ctypes.c_int32),
                ("sampling_ratio", ctypes.c_int32), ("aligned", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("rois", ctypes.c_void_p),
                ("num_rois", ctypes.c_int64), ("roi_levels", ctypes.c_void_p),
                ("plan", ctypes.c_void_p), ("plan_bytes", ctypes.c_size_t)]


class ReFwdHead(ctypes.Structure):
    _fields_ = [("rois", ctypes.c_void_p), ("num_rois", ctypes.c_int64),
                ("roi_levels", ctypes.c_void_p), ("out_h", ctypes.c_int32),
                ("out_w", ctypes.c_int32), ("sampling_ratio", ctypes.c_int32),
                ("aligned", ctypes.c_int32), ("out", ctypes.c_void_p), ("plan", ctypes.c_void_p),
                ("plan_bytes", ctypes.c_size_t)]


_VP, _I32, _I64, _F32, _SZ = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float,
                              ctypes.c_size_t)
_LEVELS = ctypes.POINTER(ReLevel)
_HEADS = ctypes.POINTER(ReHead)

SIGNATURES = {
    "fpn_level_map": [_VP, _I64, _I32, _F32, _VP, _VP],
    "fpn_level_map_ex": [_VP, _I64, _I32, _F32, _I32, _VP, _VP],
    "roi_extract_workspace_size": [_LEVELS, _I32, _I64, ctypes.POINTER(_SZ)],
    "roi_extract_plan": [_LEVELS, _I32, _VP, _I64, _F32, _VP, _VP, _SZ, _VP],
    "roi_extract_plan_ex": [_LEVELS, _I32, _VP, _I64, _F32, _I32, _VP, _VP, _SZ, _VP],
    "roi_extract_plan_offsets": [_VP, _SZ, _I64, _I32, _VP, _VP],
    "roi_extract_plan_perm": [_VP, _SZ, _I64, ctypes.POINTER(_VP)],
    "roi_align_fwd": [_LEVELS, _I32, _VP, _I64, _VP, _I32, _I32, _I32, _I32, _VP, _I32, _VP,
                      _SZ, _VP],
    "roi_extract_zero_grad": [_LEVELS, _I32, _VP],
    "roi_align_fwd_multi": [_LEVELS, _I32, ctypes.POINTER(ReFwdHead), _I32, _I32, _VP],
    "roi_align_fwd_noalloc": [_LEVELS, _I32, _VP, _I64, _F32, _VP, _I32, _I32, _I32, _I32, _VP,
                              _I32, _VP],
    "roi_align_bwd": [_VP, _I32, _VP, _I64, _VP, _I32, _I32, _I32, _I32, _LEVELS, _I32, _I32,
                      _I32, _VP, _SZ, _VP],
    "roi_align_bwd_multi": [_HEADS, _I32, _LEVELS, _I32, _I32, _VP],
    "deform_roi_pool_fwd": [_LEVELS, _I32, _VP, _I64, _VP, _I32, _I32, _I32, _I32, _VP, _VP,
                            _F32, _VP, _I32, _VP, _SZ, _VP],
    "deform_roi_pool_bwd": [_VP, _I32, _LEVELS, _LEVELS, _I32, _VP, _I64, _VP, _I32, _I32, _I32,
                            _I32, _VP, _VP, _F32, _I32, _VP, _VP, _VP, _SZ, _VP],
    "box_nms_workspace_size": [_I64, ctypes.POINTER(_SZ)],
    "box_nms": [_VP, _VP, _VP, _I64, _F32, _I64, _VP, _VP, _VP, _SZ, _VP],
    "box_nms_batched_workspace_size": [_I64, _I32, ctypes.POINTER(_SZ)],
    "box_nms_batched": [_VP, _VP, _VP, _I64, _I32, _I32, _F32, _F32, _F32, _I32, _VP, _VP, _VP,
                        _VP, _SZ, _VP],
    "roi_pool_fwd": [_LEVELS, _I32, _VP, _I64, _VP, _I32, _I32, _VP, _I32, _VP, _VP, _SZ, _VP],
    "roi_pool_bwd": [_VP, _I32, _VP, _VP, _I64, _VP, _I32, _I32, _LEVELS, _I32, _I32, _VP, _SZ,
                     _VP],
}

_lock = threading.Lock()
_lib = None


def header_functions() -> List[str]:
    """Names of the functions include/roi_extract.h declares."""
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return re.findall(r"^\s*(?:re_status_t|const char\s*\*)\s*(\w+)\s*\(", text, flags=re.M)


def lib(path: Optional[str] = None):
    """Load libroi_extract.so (raises if it has not been built)."""
    global _lib
    with _lock:
        if _lib is not None and path is None:
            return _lib
        p = path or LIBRARY
        if not os.path.exists(p):
            raise RuntimeError("%s is not built: run __graft_entry__.build() (hipcc, gfx950)" % p)
        L = ctypes.CDLL(p)
        for name, argtypes in SIGNATURES.items():
            fn = getattr(L, name)
            fn.argtypes = argtypes
            fn.restype = ctypes.c_int
        L.roi_extract_status_str.argtypes = [ctypes.c_int]
        L.roi_extract_status_str.restype = ctypes.c_char_p
        L.roi_extract_version.argtypes = []
        L.roi_extract_version.restype = ctypes.c_char_p
        if path is None:
            _lib = L
        return L


def check(status: int, where: str) -> None:
    if status != RE_OK:
        raise RoIExtractError(status, where, lib().roi_extract_status_str(status).decode())


# ---------------------------------------------------------------------------
# torch marshalling
# ---------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.float32:
        return RE_DTYPE_F32
    if t.dtype == torch.bfloat16:
        return RE_DTYPE_BF16
    raise TypeError("only float32 and bfloat16 tensors are supported, got %s" % t.dtype)


def _need_cuda(t, name: str, like=None):
    if not t.is_cuda:
        raise ValueError("%s must be a GPU tensor" % name)
    if like is not None and t.device != like.device:
        raise ValueError("%s must be on %s (got %s)" % (name, like.device, t.device))


def _on_device(rois, **tensors):
    """After the shape checks: the RoIs and every given tensor (None skipped) are GPU
    tensors on one device."""
    _need_cuda(rois, "rois")
    for name, t in tensors.items():
        if t is not None:
            _need_cuda(t, name, rois)


def _roi_levels(roi_levels, rois, num_levels: int):
    """Device pointer of the per-RoI level array: a contiguous int32 [K] tensor (the
    library reads K int32 values), or None with a single level."""
    torch = _torch()
    if roi_levels is None:
        if num_levels > 1:
            raise ValueError("roi_levels is required with more than one level")
        return None
    K = rois.shape[0]
    if (roi_levels.dtype != torch.int32 or roi_levels.dim() != 1 or roi_levels.numel() != K
            or not roi_levels.is_contiguous()):
        raise ValueError("roi_levels must be a contiguous int32 tensor of shape [%d] (got %s %s)"
                         % (K, roi_levels.dtype, tuple(roi_levels.shape)))
    return roi_levels.data_ptr()


def _block(t, shape, name: str, rois, dtypes=None):
    """A dense [K, C, out_h, out_w] tensor (out, grad_out, argmax) of the expected shape,
    checked before its pointer goes to the library."""
    torch = _torch()
    if tuple(t.shape) != tuple(shape) or not t.is_contiguous():
        raise ValueError("%s must be a contiguous tensor of shape %s (got %s)"
                         % (name, tuple(shape), tuple(t.shape)))
    if dtypes is None:
        _dtype_code(t)
    elif t.dtype not in dtypes:
        raise ValueError("%s must be %s (got %s)" % (name, " or ".join(map(str, dtypes)), t.dtype))
    return t


def _workspace(workspace, rois):
    """(pointer, bytes) of a workspace tensor: contiguous 1-D uint8."""
    torch = _torch()
    if workspace is None:
        return None, 0
    if workspace.dtype != torch.uint8 or workspace.dim() != 1 or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous 1-D uint8 tensor")
    return workspace.data_ptr(), workspace.numel()


def stream_handle(stream=None) -> int:
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


def level_array(tensors: Sequence, scales: Sequence[float], like=None):
    """re_level_t[] describing logically-NCHW tensors (any strides), all on the device of
    `like` when it is given."""
    if len(tensors) != len(scales):
        raise ValueError("one spatial scale per level")
    if not 1 <= len(tensors) <= MAX_LEVELS:
        raise ValueError("between 1 and %d levels" % MAX_LEVELS)
    arr = (ReLevel * max(1, len(tensors)))()
    for i, (t, s) in enumerate(zip(tensors, scales)):
        if t.dim() != 4:
            raise ValueError("feature level %d must be 4-D [N, C, H, W]" % i)
        _dtype_code(t)
        _need_cuda(t, "feature level %d" % i, like if like is not None else tensors[0])
        n, c, h, w = t.shape
        sn, sc, sh, sw = t.stride()
        arr[i] = ReLevel(t.data_ptr(), _dtype_code(t), 0, n, c, h, w, sn, sc, sh, sw, float(s),
                         0.0)
    return arr


def _rois(rois):
    torch = _torch()
    if rois.dim() != 2 or rois.shape[1] != 5 or rois.dtype != torch.float32:
        raise ValueError("rois must be a float32 [K, 5] tensor")
    if not rois.is_contiguous():
        raise ValueError("rois must be contiguous")
    return rois   # its device is checked after the shapes, before the first pointer is taken


def _channels(features: Sequence) -> int:
    if not features or features[0].dim() != 4:
        raise ValueError("features must be a non-empty list of 4-D [N, C, H, W] tensors")
    return int(features[0].shape[1])


# ---------------------------------------------------------------------------
# The C ABI, one function each
# ---------------------------------------------------------------------------

BOX_CONTINUOUS, BOX_PIXELS = 0, 1   # RE_BOX_CONTINUOUS, RE_BOX_PIXELS


def fpn_level_map(rois, num_levels: int, finest_scale: float = 56.0, out=None, stream=None,
                  box_pixels: bool = False):
    """Level of every RoI; box_pixels measures boxes as inclusive pixel ranges
    (fpn_level_map_ex with RE_BOX_PIXELS)."""
    torch = _torch()
    rois = _rois(rois)
    K = rois.shape[0]
    if out is None:
        out = torch.empty(K, dtype=torch.int32, device=rois.device)
    out_ptr = _roi_levels(out, rois, 2)
    _on_device(rois, levels_out=out)
    if box_pixels:
        check(lib().fpn_level_map_ex(rois.data_ptr(), K, num_levels, finest_scale, BOX_PIXELS,
                                     out_ptr, stream_handle(stream)), "fpn_level_map_ex")
    else:
        check(lib().fpn_level_map(rois.data_ptr(), K, num_levels, finest_scale, out_ptr,
                                  stream_handle(stream)), "fpn_level_map")
    return out


def workspace_size(features: Sequence, scales: Sequence[float], num_rois: int) -> int:
    """Workspace bytes of a plan for `num_rois` RoIs over this pyramid."""
    n = ctypes.c_size_t(0)
    arr = level_array(features, scales)
    check(lib().roi_extract_workspace_size(arr, len(features), num_rois, ctypes.byref(n)),
          "roi_extract_workspace_size")
    return int(n.value)


def plan(features: Sequence, scales: Sequence[float], rois, finest_scale: float = 56.0,
         levels_out=None, workspace=None, stream=None,
         box_pixels: bool = False) -> Tuple[object, object]:
    """Level of every RoI plus the launch plan.  Returns (roi_levels, workspace).
    box_pixels: the level rule measures boxes as inclusive pixel ranges
    (roi_extract_plan_ex with RE_BOX_PIXELS)."""
    torch = _torch()
    rois = _rois(rois)
    K, L = rois.shape[0], len(features)
    if levels_out is None:
        levels_out = torch.empty(K, dtype=torch.int32, device=rois.device)
    lv = _roi_levels(levels_out, rois, 2)
    if workspace is not None:
        _workspace(workspace, rois)
    _on_device(rois, levels_out=levels_out, workspace=workspace)
    nbytes = workspace_size(features, scales, K)
    if workspace is None:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=rois.device)
    ws, wsb = _workspace(workspace, rois)
    arr = level_array(features, scales, rois)
    if box_pixels:
        check(lib().roi_extract_plan_ex(arr, L, rois.data_ptr(), K, finest_scale, BOX_PIXELS,
                                        lv, ws, wsb, stream_handle(stream)),
              "roi_extract_plan_ex")
    else:
        check(lib().roi_extract_plan(arr, L, rois.data_ptr(), K, finest_scale, lv, ws, wsb,
                                     stream_handle(stream)), "roi_extract_plan")
    return levels_out, workspace


def plan_offsets(workspace, num_rois: int, num_levels: int, stream=None):
    torch = _torch()
    ws, wsb = _workspace(workspace, workspace)
    out = torch.empty(num_levels + 1, dtype=torch.int32, device=workspace.device)
    check(lib().roi_extract_plan_offsets(ws, wsb, num_rois, num_levels, out.data_ptr(),
                                         stream_handle(stream)), "roi_extract_plan_offsets")
    return out


def plan_perm(workspace, num_rois: int):
    """The plan's permutation (a view into the workspace)."""
    ws, wsb = _workspace(workspace, workspace)
    ptr = ctypes.c_void_p(0)
    check(lib().roi_extract_plan_perm(ws, wsb, num_rois, ctypes.byref(ptr)),
          "roi_extract_plan_perm")
    off = (ptr.value or 0) - workspace.data_ptr()
    return workspace[off:off + 4 * num_rois].view(_torch().int32)


def roi_align_fwd(features: Sequence, scales: Sequence[float], rois, roi_levels,
                  out_size: Tuple[int, int], sampling_ratio: int = 2, aligned: bool = True,
                  out_dtype=None, workspace=None, out=None, stream=None):
    torch = _torch()
    rois = _rois(rois)
    K, L = rois.shape[0], len(features)
    C = _channels(features)
    ph, pw = out_size
    lv = _roi_levels(roi_levels, rois, L)
    if out is None:
        out = torch.empty((K, C, ph, pw), dtype=out_dtype or features[0].dtype,
                          device=rois.device)
    _block(out, (K, C, ph, pw), "out", rois)
    ws, wsb = _workspace(workspace, rois)
    _on_device(rois, roi_levels=roi_levels, out=out, workspace=workspace)
    arr = level_array(features, scales, rois)
    check(lib().roi_align_fwd(arr, L, rois.data_ptr(), K, lv, ph, pw, sampling_ratio,
                              int(bool(aligned)), out.data_ptr(), _dtype_code(out), ws, wsb,
                              stream_handle(stream)), "roi_align_fwd")
    return out


def roi_align_fwd_noalloc(features: Sequence, scales: Sequence[float], rois,
                          out_size: Tuple[int, int], sampling_ratio: int = 2,
                          aligned: bool = True, finest_scale: float = 56.0, levels_out=None,
                          out=None, out_dtype=None, stream=None):
    """Level map, launch plan and forward in one call that allocates no device memory in
    the library (the plan lives in the library's fixed per-GPU array; calls overlapping
    on one GPU race).  Returns (out, levels_out); pass preallocated `out` and
    `levels_out` for a call that allocates nothing at all."""
    torch = _torch()
    rois = _rois(rois)
    K, L = rois.shape[0], len(features)
    C = _channels(features)
    ph, pw = out_size
    if levels_out is None:
        levels_out = torch.empty(K, dtype=torch.int32, device=rois.device)
    lv = _roi_levels(levels_out, rois, 2)
    if out is None:
        out = torch.empty((K, C, ph, pw), dtype=out_dtype or features[0].dtype,
                          device=rois.device)
    _block(out, (K, C, ph, pw), "out", rois)
    _on_device(rois, levels_out=levels_out, out=out)
    arr = level_array(features, scales, rois)
    check(lib().roi_align_fwd_noalloc(arr, L, rois.data_ptr(), K, finest_scale, lv, ph, pw,
                                      sampling_ratio, int(bool(aligned)), out.data_ptr(),
                                      _dtype_code(out), stream_handle(stream)),
          "roi_align_fwd_noalloc")
    return out, levels_out


def roi_align_fwd_multi(features: Sequence, scales: Sequence[float], heads: Sequence[dict],
                        out_dtype=None, stream=None):
    """Forward of several heads in one launch.  Each head is a dict with rois, roi_levels,
    out_size and optionally sampling_ratio (2), aligned (True), workspace (its plan) and
    out.  Returns the list of outputs ([K_h, C, out_h, out_w] of out_dtype, default the
    features' dtype)."""
    torch = _torch()
    C, L = _channels(features), len(features)
    odt = out_dtype or features[0].dtype
    if odt not in (torch.float32, torch.bfloat16):
        raise TypeError("out_dtype must be float32 or bfloat16 (got %s)" % odt)
    if not 1 <= len(heads) <= MAX_HEADS:
        raise ValueError("between 1 and %d heads" % MAX_HEADS)
    arr = (ReFwdHead * len(heads))()
    outs, fields = [], []
    for i, h in enumerate(heads):          # every head's shapes first, then the devices
        rois = _rois(h["rois"])
        K = rois.shape[0]
        ph, pw = h["out_size"]
        lv = _roi_levels(h.get("roi_levels"), rois, L)
        out = h.get("out")
        if out is not None:
            _block(out, (K, C, ph, pw), "out of head %d" % i, rois, (odt,))
        ws, wsb = _workspace(h.get("workspace"), rois)
        fields.append((rois, K, lv, ph, pw, ws, wsb))
    for i, h in enumerate(heads):
        rois, K, lv, ph, pw, ws, wsb = fields[i]
        _on_device(rois, roi_levels=h.get("roi_levels"), out=h.get("out"),
                   workspace=h.get("workspace"))
        out = h.get("out")
        if out is None:
            out = torch.empty((K, C, ph, pw), dtype=odt, device=rois.device)
        arr[i] = ReFwdHead(rois.data_ptr(), K, lv, ph, pw, int(h.get("sampling_ratio", 2)),
                           int(bool(h.get("aligned", True))), out.data_ptr(), ws, wsb)
        outs.append(out)
    levels = level_array(features, scales, heads[0]["rois"] if heads else None)
    check(lib().roi_align_fwd_multi(levels, L, arr, len(heads),
                                    RE_DTYPE_BF16 if odt == torch.bfloat16 else RE_DTYPE_F32,
                                    stream_handle(stream)), "roi_align_fwd_multi")
    return outs


def zero_grad(grads: Sequence, scales: Sequence[float], stream=None):
    arr = level_array(grads, scales)
    check(lib().roi_extract_zero_grad(arr, len(grads), stream_handle(stream)),
          "roi_extract_zero_grad")


def roi_align_bwd(grad_out, rois, roi_levels, out_size: Tuple[int, int], sampling_ratio: int,
                  aligned: bool, grads: Sequence, scales: Sequence[float], zero_init: bool = True,
                  workspace=None, stream=None, algorithm: str = "auto"):
    """Accumulate the backward into `grads` (float32 levels, cleared first if zero_init).

    algorithm: 'scatter' (fp32 atomics), 'gather' (per-tile, needs the plan workspace) or
    'auto' (gather when eligible)."""
    rois = _rois(rois)
    K, L = rois.shape[0], len(grads)
    C = _channels(grads)
    ph, pw = out_size
    if algorithm not in _BWD_ALGOS:
        raise ValueError("algorithm must be one of %s" % sorted(_BWD_ALGOS))
    lv = _roi_levels(roi_levels, rois, L)
    _block(grad_out, (K, C, ph, pw), "grad_out", rois)
    ws, wsb = _workspace(workspace, rois)
    _on_device(rois, roi_levels=roi_levels, grad_out=grad_out, workspace=workspace)
    arr = level_array(grads, scales, rois)
    check(lib().roi_align_bwd(grad_out.data_ptr(), _dtype_code(grad_out), rois.data_ptr(), K, lv,
                              ph, pw, sampling_ratio, int(bool(aligned)), arr, L,
                              int(bool(zero_init)), _BWD_ALGOS[algorithm], ws, wsb,
                              stream_handle(stream)),
          "roi_align_bwd")
    return grads


def roi_pool_fwd(features: Sequence, scales: Sequence[float], rois, roi_levels,
                 out_size: Tuple[int, int], out_dtype=None, workspace=None, out=None,
                 argmax=None, stream=None):
    """RoI max pooling.  Returns (out [K, C, out_h, out_w], argmax int32 of the same shape:
    y * W + x of the chosen pixel in its level plane, -1 for none)."""
    torch = _torch()
    rois = _rois(rois)
    K, L = rois.shape[0], len(features)
    C = _channels(features)
    ph, pw = out_size
    lv = _roi_levels(roi_levels, rois, L)
    if out is None:
        out = torch.empty((K, C, ph, pw), dtype=out_dtype or features[0].dtype,
                          device=rois.device)
    if argmax is None:
        argmax = torch.empty((K, C, ph, pw), dtype=torch.int32, device=rois.device)
    _block(out, (K, C, ph, pw), "out", rois)
    _block(argmax, (K, C, ph, pw), "argmax", rois, (torch.int32,))
    ws, wsb = _workspace(workspace, rois)
    _on_device(rois, roi_levels=roi_levels, out=out, argmax=argmax, workspace=workspace)
    arr = level_array(features, scales, rois)
    check(lib().roi_pool_fwd(arr, L, rois.data_ptr(), K, lv, ph, pw, out.data_ptr(),
                             _dtype_code(out), argmax.data_ptr(), ws, wsb, stream_handle(stream)),
          "roi_pool_fwd")
    return out, argmax


def roi_pool_bwd(grad_out, argmax, rois, roi_levels, grads: Sequence, scales: Sequence[float],
                 zero_init: bool = True, workspace=None, stream=None):
    """Add every upstream gradient to its argmax pixel of `grads` (float32 levels, cleared
    first if zero_init)."""
    torch = _torch()
    rois = _rois(rois)
    K, L = rois.shape[0], len(grads)
    C = _channels(grads)
    if grad_out.dim() != 4:
        raise ValueError("grad_out must be 4-D [K, C, out_h, out_w]")
    ph, pw = grad_out.shape[2], grad_out.shape[3]
    lv = _roi_levels(roi_levels, rois, L)
    _block(grad_out, (K, C, ph, pw), "grad_out", rois)
    _block(argmax, (K, C, ph, pw), "argmax", rois, (torch.int32,))
    ws, wsb = _workspace(workspace, rois)
    _on_device(rois, roi_levels=roi_levels, grad_out=grad_out, argmax=argmax,
               workspace=workspace)
    arr = level_array(grads, scales, rois)
    check(lib().roi_pool_bwd(grad_out.data_ptr(), _dtype_code(grad_out), argmax.data_ptr(),
                             rois.data_ptr(), K, lv, ph, pw, arr, L, int(bool(zero_init)), ws,
                             wsb, stream_handle(stream)), "roi_pool_bwd")
    return grads


def roi_align_bwd_multi(heads: Sequence[dict], grads: Sequence, scales: Sequence[float],
                        zero_init: bool = True, stream=None):
    """Backward of several heads into one gradient pyramid (float32 levels, cleared first if
    zero_init).  Each head is a dict with grad_out, rois, roi_levels, out_size and optionally
    sampling_ratio (2), aligned (True) and workspace (its plan)."""
    C, L = _channels(grads), len(grads)
    arr = (ReHead * max(1, len(heads)))()
    for i, h in enumerate(heads):
        rois = _rois(h["rois"])
        K = rois.shape[0]
        ph, pw = h["out_size"]
        g = _block(h["grad_out"], (K, C, ph, pw), "grad_out of head %d" % i, rois)
        lv = _roi_levels(h.get("roi_levels"), rois, L)
        ws, wsb = _workspace(h.get("workspace"), rois)
        _on_device(rois, roi_levels=h.get("roi_levels"), grad_out=g,
                   workspace=h.get("workspace"))
        arr[i] = ReHead(g.data_ptr(), _dtype_code(g), ph, pw, int(h.get("sampling_ratio", 2)),
                        int(bool(h.get("aligned", True))), 0, rois.data_ptr(), K, lv, ws, wsb)
    levels = level_array(grads, scales)
    check(lib().roi_align_bwd_multi(arr, len(heads), levels, len(grads), int(bool(zero_init)),
                                    stream_handle(stream)), "roi_align_bwd_multi")
    return grads


def _f32_contig(t, name, shape=None, like=None):
    torch = _torch()
    if t.dtype != torch.float32 or not t.is_contiguous():
        raise ValueError("%s must be a contiguous float32 tensor" % name)
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError("%s must have shape %s (got %s)" % (name, tuple(shape), tuple(t.shape)))
    return t


def deform_roi_pool_fwd(features: Sequence, scales: Sequence[float], rois, roi_levels,
                        out_size: Tuple[int, int], offset, mask=None, gamma: float = 0.1,
                        sampling_ratio: int = 2, aligned: bool = True, out_dtype=None,
                        workspace=None, out=None, stream=None):
    """Deformable (modulated when `mask` is given) RoI pooling.  offset: float32
    [K, 2, out_h, out_w] (x then y, normalized to the box size); mask: float32
    [K, out_h, out_w] or None."""
    torch = _torch()
    rois = _rois(rois)
    K, L = rois.shape[0], len(features)
    C = _channels(features)
    ph, pw = out_size
    lv = _roi_levels(roi_levels, rois, L)
    _f32_contig(offset, "offset", (K, 2, ph, pw), rois)
    if mask is not None:
        _f32_contig(mask, "mask", (K, ph, pw), rois)
    if out is None:
        out = torch.empty((K, C, ph, pw), dtype=out_dtype or features[0].dtype,
                          device=rois.device)
    _block(out, (K, C, ph, pw), "out", rois)
    ws, wsb = _workspace(workspace, rois)
    _on_device(rois, roi_levels=roi_levels, offset=offset, mask=mask, out=out,
               workspace=workspace)
    arr = level_array(features, scales, rois)
    check(lib().deform_roi_pool_fwd(arr, L, rois.data_ptr(), K, lv, ph, pw, sampling_ratio,
                                    int(bool(aligned)), offset.data_ptr(),
                                    mask.data_ptr() if mask is not None else None, float(gamma),
                                    out.data_ptr(), _dtype_code(out), ws, wsb,
                                    stream_handle(stream)), "deform_roi_pool_fwd")
    return out


def deform_roi_pool_bwd(grad_out, features: Sequence, rois, roi_levels, offset, mask,
                        grads: Sequence, scales: Sequence[float], gamma: float = 0.1,
                        sampling_ratio: int = 2, aligned: bool = True, zero_init: bool = True,
                        grad_offset=None, grad_mask=None, workspace=None, stream=None):
    """Gradients of deform_roi_pool_fwd: feature gradients added into `grads` (float32
    levels, cleared first if zero_init); returns (grads, grad_offset, grad_mask)."""
    torch = _torch()
    rois = _rois(rois)
    K, L = rois.shape[0], len(grads)
    C = _channels(grads)
    if grad_out.dim() != 4:
        raise ValueError("grad_out must be 4-D [K, C, out_h, out_w]")
    ph, pw = grad_out.shape[2], grad_out.shape[3]
    lv = _roi_levels(roi_levels, rois, L)
    _block(grad_out, (K, C, ph, pw), "grad_out", rois)
    _f32_contig(offset, "offset", (K, 2, ph, pw), rois)
    if mask is not None:
        _f32_contig(mask, "mask", (K, ph, pw), rois)
    if grad_offset is None:
        grad_offset = torch.empty((K, 2, ph, pw), dtype=torch.float32, device=rois.device)
    _f32_contig(grad_offset, "grad_offset", (K, 2, ph, pw), rois)
    if grad_mask is None and mask is not None:
        grad_mask = torch.empty((K, ph, pw), dtype=torch.float32, device=rois.device)
    if grad_mask is not None:
        _f32_contig(grad_mask, "grad_mask", (K, ph, pw), rois)
    ws, wsb = _workspace(workspace, rois)
    _on_device(rois, roi_levels=roi_levels, grad_out=grad_out, offset=offset, mask=mask,
               grad_offset=grad_offset, grad_mask=grad_mask, workspace=workspace)
    farr = level_array(features, scales, rois)
    garr = level_array(grads, scales, rois)
    check(lib().deform_roi_pool_bwd(grad_out.data_ptr(), _dtype_code(grad_out), farr, garr, L,
                                    rois.data_ptr(), K, lv, ph, pw, sampling_ratio,
                                    int(bool(aligned)), offset.data_ptr(),
                                    mask.data_ptr() if mask is not None else None, float(gamma),
                                    int(bool(zero_init)), grad_offset.data_ptr(),
                                    grad_mask.data_ptr() if grad_mask is not None else None,
                                    ws, wsb, stream_handle(stream)), "deform_roi_pool_bwd")
    return grads, grad_offset, grad_mask


def box_nms(boxes, scores, iou_threshold: float, categories=None, max_keep: int | None = None,
            workspace=None, keep=None, num_keep=None, stream=None):
    """Greedy NMS on the GPU.  Returns (keep int32 [min(N, max_keep)]: kept indices in rank
    order then -1, num_keep int32 [1]); both stay on the device."""
    torch = _torch()
    if scores.dtype != torch.float32 or scores.dim() != 1 or not scores.is_contiguous():
        raise ValueError("scores must be a contiguous float32 [N] tensor")
    N = scores.shape[0]
    if boxes.dtype != torch.float32 or tuple(boxes.shape) != (N, 4) or not boxes.is_contiguous():
        raise ValueError("boxes must be a contiguous float32 [N, 4] tensor")
    if categories is not None and (categories.dtype != torch.int32 or
                                   tuple(categories.shape) != (N,) or
                                   not categories.is_contiguous()):
        raise ValueError("categories must be a contiguous int32 [N] tensor")
    mk = N if max_keep is None else int(max_keep)
    if mk < 0:
        raise ValueError("max_keep must be >= 0")
    if keep is not None and (keep.dtype != torch.int32 or not keep.is_contiguous() or
                             keep.numel() < min(N, mk)):
        raise ValueError("keep must be a contiguous int32 tensor of at least %d elements"
                         % min(N, mk))
    if num_keep is not None and (num_keep.dtype != torch.int32 or num_keep.numel() < 1):
        raise ValueError("num_keep must be an int32 tensor of at least 1 element")
    _need_cuda(boxes, "boxes")
    _need_cuda(scores, "scores", boxes)
    if categories is not None:
        _need_cuda(categories, "categories", boxes)
    n = ctypes.c_size_t(0)
    check(lib().box_nms_workspace_size(N, ctypes.byref(n)), "box_nms_workspace_size")
    if workspace is None:
        workspace = torch.empty(n.value, dtype=torch.uint8, device=boxes.device)
    if keep is None:
        keep = torch.empty(max(min(N, mk), 1), dtype=torch.int32, device=boxes.device)
    if num_keep is None:
        num_keep = torch.empty(1, dtype=torch.int32, device=boxes.device)
    _need_cuda(keep, "keep", boxes)
    _need_cuda(num_keep, "num_keep", boxes)
    ws, wsb = _workspace(workspace, boxes)
    check(lib().box_nms(boxes.data_ptr(), scores.data_ptr(),
                        categories.data_ptr() if categories is not None else None, N,
                        float(iou_threshold), mk, keep.data_ptr(), num_keep.data_ptr(),
                        ws, wsb, stream_handle(stream)), "box_nms")
    return keep[:min(N, mk)], num_keep


def box_nms_batched(boxes, scores, categories=None, num_categories: int = 1,
                    method: str = "hard", iou_threshold: float = 0.5, sigma: float = 0.5,
                    score_threshold: float = float("-inf"), max_keep: int | None = None,
                    workspace=None, keep=None, kept_scores=None, num_keep=None, stream=None):
    """Per-category proposal selection on the GPU: greedy NMS ("hard") or Soft-NMS
    ("linear", "gaussian").  Returns (keep int32 [C, max_keep]: kept indices of each
    category in selection order then -1, kept_scores float32 [C, max_keep]: score at
    selection then 0, num_keep int32 [C]); all stay on the device."""
    torch = _torch()
    if method not in NMS_METHODS:
        raise ValueError("method must be one of %s" % sorted(NMS_METHODS))
    if scores.dtype != torch.float32 or scores.dim() != 1 or not scores.is_contiguous():
        raise ValueError("scores must be a contiguous float32 [N] tensor")
    N = scores.shape[0]
    if boxes.dtype != torch.float32 or tuple(boxes.shape) != (N, 4) or not boxes.is_contiguous():
        raise ValueError("boxes must be a contiguous float32 [N, 4] tensor")
    if categories is not None and (categories.dtype != torch.int32 or
                                   tuple(categories.shape) != (N,) or
                                   not categories.is_contiguous()):
        raise ValueError("categories must be a contiguous int32 [N] tensor")
    C = int(num_categories)
    mk = N if max_keep is None else int(max_keep)
    if mk < 0:
        raise ValueError("max_keep must be >= 0")
    for t, name, dt, shape in ((keep, "keep", torch.int32, (C, mk)),
                               (kept_scores, "kept_scores", torch.float32, (C, mk)),
                               (num_keep, "num_keep", torch.int32, (C,))):
        if t is not None and (t.dtype != dt or tuple(t.shape) != shape or not t.is_contiguous()):
            raise ValueError("%s must be a contiguous %s tensor of shape %s" % (name, dt, shape))
    if workspace is not None:
        _workspace(workspace, boxes)
    _need_cuda(boxes, "boxes")
    for t, name in ((scores, "scores"), (categories, "categories"), (keep, "keep"),
                    (kept_scores, "kept_scores"), (num_keep, "num_keep"),
                    (workspace, "workspace")):
        if t is not None:
            _need_cuda(t, name, boxes)
    n = ctypes.c_size_t(0)
    check(lib().box_nms_batched_workspace_size(N, C, ctypes.byref(n)),
          "box_nms_batched_workspace_size")
    dev = boxes.device
    if workspace is None:
        workspace = torch.empty(n.value, dtype=torch.uint8, device=dev)
    if keep is None:
        keep = torch.empty((C, mk), dtype=torch.int32, device=dev)
    if kept_scores is None:
        kept_scores = torch.empty((C, mk), dtype=torch.float32, device=dev)
    if num_keep is None:
        num_keep = torch.empty(C, dtype=torch.int32, device=dev)
    ws, wsb = _workspace(workspace, boxes)
    check(lib().box_nms_batched(boxes.data_ptr(), scores.data_ptr(),
                                categories.data_ptr() if categories is not None else None, N, C,
                                NMS_METHODS[method], float(iou_threshold), float(sigma),
                                float(score_threshold), mk,
                                keep.data_ptr() if mk * C > 0 else None,
                                kept_scores.data_ptr() if mk * C > 0 else None,
                                num_keep.data_ptr(), ws, wsb, stream_handle(stream)),
          "box_nms_batched")
    return keep, kept_scores, num_keep
