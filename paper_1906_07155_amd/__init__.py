"""MI355X-native multi-level RoIAlign (the RoIExtractor of MMDetection, arXiv 1906.07155).

The work runs in hand-written HIP kernels for gfx950 behind the C ABI in
include/roi_extract.h (libroi_extract.so, built in-tree by `build.py`).  This
package only marshals torch tensors into that ABI.
"""
from .binding import (RoIExtractError, box_nms, box_nms_batched, deform_roi_pool_bwd, deform_roi_pool_fwd,
                      fpn_level_map, lib, plan, plan_offsets, plan_perm,
                      roi_align_bwd, roi_align_bwd_multi, roi_align_fwd,
                      roi_align_fwd_multi, roi_align_fwd_noalloc, roi_pool_bwd,
                      roi_pool_fwd, workspace_size, zero_grad)

__all__ = ["RoIExtractError", "box_nms", "box_nms_batched", "deform_roi_pool_bwd", "deform_roi_pool_fwd", "fpn_level_map", "lib", "plan", "plan_offsets", "plan_perm",
           "roi_align_bwd", "roi_align_bwd_multi", "roi_align_fwd", "roi_align_fwd_multi", "roi_align_fwd_noalloc", "roi_pool_bwd", "roi_pool_fwd", "workspace_size",
           "zero_grad", "roi_extract",
           "RoIAlignFunction"]


def __getattr__(name):
    if name in ("roi_extract", "RoIAlignFunction"):
        from . import extractor
        return getattr(extractor, name)
    raise AttributeError(name)
