"""SingleRoIExtractor-style entry point with autograd (MMDetection §3.1, §3.2).

`roi_extract` assigns every RoI to its FPN level, builds the launch plan and runs
the RoIAlign forward; the backward (the transpose) reuses the same levels and plan:
by default every tile of the gradient pyramid gathers the RoIs the plan binned to it
and is written once with plain stores (the fp32-atomic scatter serves the cases the
gather does not cover).  All arithmetic runs in the HIP library; this module only
wires it into torch.autograd.
"""
from __future__ import annotations

from typing import Sequence, Tuple

import torch

from . import binding


class RoIAlignFunction(torch.autograd.Function):
    @staticmethod
    def forward(ctx, rois, roi_levels, workspace, out_size, sampling_ratio, aligned, scales,
                *features):
        out = binding.roi_align_fwd(features, scales, rois, roi_levels, out_size,
                                    sampling_ratio, aligned, workspace=workspace)
        ctx.save_for_backward(rois, roi_levels, workspace)
        ctx.cfg = (tuple(out_size), int(sampling_ratio), bool(aligned), tuple(scales),
                   [(f.shape, f.dtype) for f in features])
        return out

    @staticmethod
    def backward(ctx, grad_out):
        rois, roi_levels, workspace = ctx.saved_tensors
        out_size, sr, aligned, scales, metas = ctx.cfg
        grads = [torch.empty(shape, dtype=torch.float32, device=grad_out.device,
                             memory_format=torch.channels_last) for shape, _ in metas]
        binding.roi_align_bwd(grad_out.contiguous(), rois, roi_levels, out_size, sr, aligned,
                              grads, scales, zero_init=True, workspace=workspace)
        grads = [g if dt == torch.float32 else g.to(dt) for g, (_, dt) in zip(grads, metas)]
        return (None, None, None, None, None, None, None, *grads)


def roi_extract(features: Sequence[torch.Tensor], scales: Sequence[float], rois: torch.Tensor,
                out_size: Tuple[int, int] = (7, 7), sampling_ratio: int = 2,
                aligned: bool = True, finest_scale: float = 56.0) -> torch.Tensor:
    """Multi-level RoIAlign of `rois` ([K, 5] float32: batch index, x1, y1, x2, y2) over the
    pyramid `features` (list of [N, C, H_l, W_l] tensors, channels-last for the fast path)
    with `scales` (e.g. 1/4 .. 1/32).  Returns [K, C, out_h, out_w]."""
    roi_levels, workspace = binding.plan(features, scales, rois, finest_scale)
    return RoIAlignFunction.apply(rois, roi_levels, workspace, tuple(out_size), sampling_ratio,
                                  aligned, tuple(scales), *features)
