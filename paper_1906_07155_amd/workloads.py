"""Seeded synthetic inputs shaped like FPN Faster/Mask R-CNN RoI extraction.

This module only draws random numbers and lays them out.  It holds none of the
RoIAlign arithmetic, so both the GPU path (tests, bench) and the CPU oracle can
be fed from it without sharing any of the method's code.

Shapes follow the paper's setting: images resized to 1333x800 (§4.1
"Implementation details"), padded here to a multiple of 32 (800x1344), an FPN
neck (§3.1) giving P2..P5 at strides 4..32 with 256 channels, and two-stage
heads consuming 7x7 (box) or 14x14 (mask) RoI features (§3.1 RoIHead).  COCO
proposals are not available, so RoIs are drawn: centres uniform in the image,
width and height log-uniform in a size range, clipped to the image, batch index
in column 0.  Features and upstream gradients are standard normal.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Tuple

import numpy as np

BASE_SEED = 19060715500
STREAM_FEATURES, STREAM_ROIS, STREAM_GRADS, STREAM_DUPS = 0, 1, 2, 3
# a second RoI set drawn on the same pyramid (the mask head of the batch-16 workload)
HEAD_STREAM_OFFSET = 10

FPN_STRIDES = (4, 8, 16, 32)


def rng_for(seed: int, stream: int) -> np.random.Generator:
    return np.random.default_rng([int(seed), int(stream)])


# --------------------------------------------------------------------------
# bfloat16 storage (numpy has no bf16 type: values are kept as uint16 bits)
# --------------------------------------------------------------------------

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    nan = np.isnan(np.ascontiguousarray(x, dtype=np.float32))
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)
    if nan.any():
        r = np.where(nan, ((u >> 16) | 0x40).astype(np.uint16), r)
    return r


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# --------------------------------------------------------------------------
# Drawing RoIs, features and gradients
# --------------------------------------------------------------------------

def draw_rois(rng: np.random.Generator, n_images: int, per_image: int,
              img_hw: Tuple[int, int], size_range: Tuple[float, float]) -> np.ndarray:
    """[n_images*per_image, 5] float32, image-major, random order inside an image."""
    H, W = img_hw
    lo, hi = size_range
    out = np.empty((n_images * per_image, 5), dtype=np.float32)
    for i in range(n_images):
        cx = rng.uniform(0.0, W, per_image)
        cy = rng.uniform(0.0, H, per_image)
        w = np.exp(rng.uniform(np.log(lo), np.log(hi), per_image))
        h = np.exp(rng.uniform(np.log(lo), np.log(hi), per_image))
        blk = out[i * per_image:(i + 1) * per_image]
        blk[:, 0] = i
        blk[:, 1] = np.clip(cx - w / 2, 0, W)
        blk[:, 2] = np.clip(cy - h / 2, 0, H)
        blk[:, 3] = np.clip(cx + w / 2, 0, W)
        blk[:, 4] = np.clip(cy + h / 2, 0, H)
    return out


def add_duplicates(rng: np.random.Generator, rois: np.ndarray, frac: float,
                   jitter: float, img_hw: Tuple[int, int]) -> np.ndarray:
    """Overwrite floor(frac*K) slots with jittered copies of other RoIs of the same image.

    Destination slots are drawn without replacement; each copies a non-destination
    RoI of the same image and adds U(-jitter, jitter) pixels to every coordinate,
    then re-clips and re-orders the corners.
    """
    H, W = img_hw
    r = rois.copy()
    K = r.shape[0]
    n = int(np.floor(frac * K))
    if n == 0:
        return r
    dst = rng.choice(K, size=n, replace=False)
    is_dst = np.zeros(K, dtype=bool)
    is_dst[dst] = True
    for d in dst:
        img = r[d, 0]
        pool = np.flatnonzero((rois[:, 0] == img) & ~is_dst)
        src = pool[rng.integers(0, pool.size)]
        box = rois[src, 1:].astype(np.float64) + rng.uniform(-jitter, jitter, 4)
        x1, y1, x2, y2 = box
        x1, x2 = np.clip([x1, x2], 0, W)
        y1, y2 = np.clip([y1, y2], 0, H)
        if x1 > x2:
            x1, x2 = x2, x1
        if y1 > y2:
            y1, y2 = y2, y1
        r[d, 1:] = (x1, y1, x2, y2)
    return r


def draw_proposals(rng: np.random.Generator, n_images: int, per_image: int,
                   img_hw: Tuple[int, int] = (800, 1333), size_range=(8.0, 600.0),
                   dup: float = 0.3):
    """Scored proposals of a batch, the input of NMS (a synthetic stand-in for a dense
    head's output): centres uniform in the image, log-uniform sides, a share `dup` of
    slots overwritten with copies of other boxes jittered by up to 10% of their size
    (the heavy overlaps NMS exists for), clipped to the image; scores uniform in [0, 1).
    Returns (boxes float32 [N, 4], scores float32 [N], image index int32 [N]), the
    images' boxes contiguous."""
    H, W = img_hw
    lo, hi = size_range
    N = n_images * per_image
    cx, cy = rng.uniform(0, W, N), rng.uniform(0, H, N)
    w = np.exp(rng.uniform(np.log(lo), np.log(hi), N))
    h = np.exp(rng.uniform(np.log(lo), np.log(hi), N))
    boxes = np.stack([cx - w / 2, cy - h / 2, cx + w / 2, cy + h / 2], 1)
    nd = int(dup * N)
    src = rng.integers(0, N, nd)
    dst = rng.choice(N, nd, replace=False)
    boxes[dst] = boxes[src] + rng.uniform(-0.1, 0.1, (nd, 4)) * np.stack([w[src], h[src]] * 2, 1)
    boxes = np.clip(boxes, 0, [W, H, W, H]).astype(np.float32)
    scores = rng.uniform(0, 1, N).astype(np.float32)
    images = np.repeat(np.arange(n_images, dtype=np.int32), per_image)
    return boxes, scores, images


def draw_features(rng: np.random.Generator, n: int, c: int,
                  level_hw: List[Tuple[int, int]], dtype: str) -> List[np.ndarray]:
    """Standard-normal NCHW maps.  dtype 'f32' -> float32, 'bf16' -> uint16 bf16 bits."""
    feats = []
    for (h, w) in level_hw:
        x = rng.standard_normal((n, c, h, w), dtype=np.float32)
        feats.append(f32_to_bf16_bits(x) if dtype == "bf16" else x)
    return feats


def draw_grad(rng: np.random.Generator, shape, dtype: str) -> np.ndarray:
    g = rng.standard_normal(shape, dtype=np.float32)
    return f32_to_bf16_bits(g) if dtype == "bf16" else g


# --------------------------------------------------------------------------
# The five workloads
# --------------------------------------------------------------------------

@dataclasses.dataclass
class Workload:
    name: str
    n_images: int
    channels: int
    level_hw: List[Tuple[int, int]]
    scales: List[float]
    img_hw: Tuple[int, int]
    out_hw: Tuple[int, int]
    sampling_ratio: int
    aligned: bool
    feat_dtype: str          # 'f32' | 'bf16'
    out_dtype: str           # 'f32' | 'bf16'
    grad_dtype: str          # 'f32' | 'bf16' (upstream gradient)
    backward: bool
    seed: int
    per_image: int
    size_range: Tuple[float, float]
    dup_frac: float = 0.0
    dup_jitter: float = 0.0
    fpn: bool = True         # levels assigned by the FPN rule (else single level)
    finest_scale: float = 56.0
    stream_offset: int = 0   # RoI / gradient substreams of a second head on the same pyramid

    @property
    def num_levels(self) -> int:
        return len(self.level_hw)

    @property
    def tag(self) -> str:
        """Short file-name tag: head, batch and dtype (e.g. box_batch2_fp32)."""
        if not self.fpn:
            return "single_level_batch%d" % self.n_images
        head = "box" if self.out_hw == (7, 7) else "mask"
        if not self.backward:
            head = "infer"
        dt = {"f32": "fp32", "bf16": "bf16"}[self.feat_dtype]
        return "%s_batch%d_%s" % (head, self.n_images, dt)

    @property
    def num_rois(self) -> int:
        return self.n_images * self.per_image

    def level_shapes(self):
        return [(self.n_images, self.channels, h, w) for (h, w) in self.level_hw]

    def rois(self) -> np.ndarray:
        r = draw_rois(rng_for(self.seed, STREAM_ROIS + self.stream_offset), self.n_images,
                      self.per_image, self.img_hw, self.size_range)
        if self.dup_frac > 0:
            r = add_duplicates(rng_for(self.seed, STREAM_DUPS + self.stream_offset), r,
                               self.dup_frac, self.dup_jitter, self.img_hw)
        return r

    def features(self) -> List[np.ndarray]:
        return draw_features(rng_for(self.seed, STREAM_FEATURES), self.n_images,
                             self.channels, self.level_hw, self.feat_dtype)

    def grad(self) -> np.ndarray:
        K = self.num_rois
        return draw_grad(rng_for(self.seed, STREAM_GRADS + self.stream_offset),
                         (K, self.channels, self.out_hw[0], self.out_hw[1]), self.grad_dtype)


def _pyramid(img_hw):
    H, W = img_hw
    return [(H // s, W // s) for s in FPN_STRIDES], [1.0 / s for s in FPN_STRIDES]


def config(index: int, head: Optional[str] = None, feat_dtype: Optional[str] = None) -> Workload:
    """Workload `index` (1..5).  The batch-1 inference workload (4) takes feat_dtype 'f32'
    or 'bf16'; the batch-16 workload (5) takes head 'box' or 'mask'."""
    seed = BASE_SEED + index
    if index == 1:
        return Workload("single-level 1x256x50x68 fwd, 128 RoIs, 7x7", 1, 256, [(50, 68)],
                        [1.0 / 16], (800, 1088), (7, 7), 2, True, "f32", "f32", "f32",
                        False, seed, 128, (16.0, 512.0), fpn=False)
    lv, sc = _pyramid((800, 1344))
    if index == 2:
        return Workload("FPN box head fwd+bwd, batch 2, 1024 RoIs, 7x7, fp32", 2, 256, lv, sc,
                        (800, 1344), (7, 7), 2, True, "f32", "f32", "f32", True, seed, 512,
                        (8.0, 800.0))
    if index == 3:
        return Workload("FPN mask head fwd+bwd, batch 2, 256 RoIs, 14x14, fp32", 2, 256, lv,
                        sc, (800, 1344), (14, 14), 2, True, "f32", "f32", "f32", True, seed,
                        128, (32.0, 512.0))
    if index == 4:
        fd = feat_dtype or "f32"
        return Workload("FPN inference fwd, batch 1, 1000 RoIs, 7x7, %s features" % fd, 1, 256,
                        lv, sc, (800, 1344), (7, 7), 2, True, fd, fd, fd, False, seed, 1000,
                        (8.0, 800.0))
    if index == 5:
        h = head or "box"
        if h == "box":
            return Workload("FPN batch 16 box head fwd+bwd, 8192 RoIs, 7x7, bf16", 16, 256, lv,
                            sc, (800, 1344), (7, 7), 2, True, "bf16", "bf16", "bf16", True,
                            seed, 512, (8.0, 800.0), dup_frac=0.2, dup_jitter=2.0)
        return Workload("FPN batch 16 mask head fwd+bwd, 2048 RoIs, 14x14, bf16", 16, 256, lv,
                        sc, (800, 1344), (14, 14), 2, True, "bf16", "bf16", "bf16", True,
                        seed, 128, (8.0, 800.0), dup_frac=0.2, dup_jitter=2.0,
                        stream_offset=HEAD_STREAM_OFFSET)
    raise ValueError("config index must be 1..5")
