"""The Python binding rejects mis-shaped or mistyped tensors before any pointer reaches
the library.

A wrong-dtype level array (torch's default int64) would be read by the library as
pairs of int32 values, and a short level array or an output smaller than
[K, C, out_h, out_w] would let the kernels read or write past the tensor, so the
binding checks shape, dtype and contiguity of every tensor it passes.  These checks
come before the device checks, so they run on CPU tensors here; a tensor that passes
them and is not on the GPU is then refused as such.  No library call is made.
"""
import pytest
import torch

from paper_1906_07155_amd import binding as B

K, C, N = 6, 8, 2
SCALES = [0.25, 0.125]


def _feats():
    return [torch.zeros(N, C, 16, 20), torch.zeros(N, C, 8, 10)]


def _rois():
    return torch.zeros(K, 5, dtype=torch.float32)


def _levels(dtype=torch.int32, n=K):
    return torch.zeros(n, dtype=dtype)


def test_fwd_roi_levels_dtype_and_length():
    with pytest.raises(ValueError, match="roi_levels"):
        B.roi_align_fwd(_feats(), SCALES, _rois(), _levels(torch.int64), (7, 7))
    with pytest.raises(ValueError, match="roi_levels"):
        B.roi_align_fwd(_feats(), SCALES, _rois(), _levels(n=K - 1), (7, 7))
    with pytest.raises(ValueError, match="roi_levels is required"):
        B.roi_align_fwd(_feats(), SCALES, _rois(), None, (7, 7))


def test_fwd_out_shape_and_dtype():
    with pytest.raises(ValueError, match="out must be"):
        B.roi_align_fwd(_feats(), SCALES, _rois(), _levels(), (7, 7),
                        out=torch.zeros(K, C, 7, 6))
    with pytest.raises(ValueError, match="out must be"):
        B.roi_align_fwd(_feats(), SCALES, _rois(), _levels(), (7, 7),
                        out=torch.zeros(K - 1, C, 7, 7))
    with pytest.raises(ValueError, match="out must be"):
        B.roi_align_fwd(_feats(), SCALES, _rois(), _levels(), (7, 7),
                        out=torch.zeros(K, C, 7, 7).transpose(2, 3))
    with pytest.raises(TypeError):
        B.roi_align_fwd(_feats(), SCALES, _rois(), _levels(), (7, 7),
                        out=torch.zeros(K, C, 7, 7, dtype=torch.float16))


def test_bwd_grad_out_and_levels():
    grads = _feats()
    with pytest.raises(ValueError, match="grad_out must be"):
        B.roi_align_bwd(torch.zeros(K, C, 7, 7), _rois(), _levels(), (14, 14), 2, True, grads,
                        SCALES)
    with pytest.raises(ValueError, match="grad_out must be"):
        B.roi_align_bwd(torch.zeros(K, C + 1, 7, 7), _rois(), _levels(), (7, 7), 2, True,
                        grads, SCALES)
    with pytest.raises(ValueError, match="roi_levels"):
        B.roi_align_bwd(torch.zeros(K, C, 7, 7), _rois(), _levels(torch.int64), (7, 7), 2, True,
                        grads, SCALES)
    with pytest.raises(ValueError, match="algorithm"):
        B.roi_align_bwd(torch.zeros(K, C, 7, 7), _rois(), _levels(), (7, 7), 2, True, grads,
                        SCALES, algorithm="fast")


def test_pool_and_deform_blocks():
    with pytest.raises(ValueError, match="argmax"):
        B.roi_pool_fwd(_feats(), SCALES, _rois(), _levels(), (7, 7),
                       argmax=torch.zeros(K, C, 7, 7, dtype=torch.int64))
    with pytest.raises(ValueError, match="argmax"):
        B.roi_pool_bwd(torch.zeros(K, C, 7, 7), torch.zeros(K, C, 7, 6, dtype=torch.int32),
                       _rois(), _levels(), _feats(), SCALES)
    with pytest.raises(ValueError, match="offset"):
        B.deform_roi_pool_fwd(_feats(), SCALES, _rois(), _levels(), (7, 7),
                              torch.zeros(K, 2, 7, 6))
    with pytest.raises(ValueError, match="mask"):
        B.deform_roi_pool_fwd(_feats(), SCALES, _rois(), _levels(), (7, 7),
                              torch.zeros(K, 2, 7, 7), mask=torch.zeros(K, 7))


def test_workspace_and_rois():
    with pytest.raises(ValueError, match="workspace"):
        B.roi_align_fwd(_feats(), SCALES, _rois(), _levels(), (7, 7),
                        out=torch.zeros(K, C, 7, 7), workspace=torch.zeros(64, dtype=torch.int32))
    with pytest.raises(ValueError, match="rois"):
        B.roi_align_fwd(_feats(), SCALES, torch.zeros(K, 4), _levels(), (7, 7))
    with pytest.raises(ValueError, match="rois"):
        B.roi_align_fwd(_feats(), SCALES, torch.zeros(K, 5, dtype=torch.float64), _levels(),
                        (7, 7))


def test_well_formed_cpu_tensors_are_refused_as_not_on_the_gpu():
    with pytest.raises(ValueError, match="GPU tensor"):
        B.roi_align_fwd(_feats(), SCALES, _rois(), _levels(), (7, 7),
                        out=torch.zeros(K, C, 7, 7))
    with pytest.raises(ValueError, match="GPU tensor"):
        B.roi_align_bwd(torch.zeros(K, C, 7, 7), _rois(), _levels(), (7, 7), 2, True, _feats(),
                        SCALES)


def test_nms_shapes():
    boxes = torch.zeros(10, 4)
    scores = torch.zeros(10)
    with pytest.raises(ValueError, match="categories"):
        B.box_nms(boxes, scores, 0.5, categories=torch.zeros(9, dtype=torch.int32))
    with pytest.raises(ValueError, match="boxes"):
        B.box_nms(torch.zeros(10, 5), scores, 0.5)
    with pytest.raises(ValueError, match="keep"):
        B.box_nms(boxes, scores, 0.5, keep=torch.zeros(5, dtype=torch.int32))
    with pytest.raises(ValueError, match="GPU tensor"):
        B.box_nms(boxes, scores, 0.5)


def test_multi_head_forward_blocks():
    heads = [dict(rois=_rois(), roi_levels=_levels(), out_size=(7, 7)),
             dict(rois=_rois(), roi_levels=_levels(n=K - 1), out_size=(14, 14))]
    with pytest.raises(ValueError, match="roi_levels"):
        B.roi_align_fwd_multi(_feats(), SCALES, heads)
    heads[1]["roi_levels"] = _levels()
    heads[1]["out"] = torch.zeros(K, C, 7, 7)
    with pytest.raises(ValueError, match="out of head 1"):
        B.roi_align_fwd_multi(_feats(), SCALES, heads)
    del heads[1]["out"]
    with pytest.raises(ValueError, match="GPU tensor"):
        B.roi_align_fwd_multi(_feats(), SCALES, heads)
