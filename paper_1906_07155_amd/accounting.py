"""Algorithmic byte counts for the roofline figures of the benchmark.

For every RoI the forward reads a separable footprint of feature pixels: the
distinct tap rows of its valid sample rows times the distinct tap columns of its
valid sample columns (validity and taps are separable, so the product is exact).
With C channels of s bytes:

  E_fwd  = sum_r F_r*C*s_feat + K*C*PH*PW*s_out + 24*K        (effective bytes)
  E_bwd  = K*C*PH*PW*s_gout + 2*sum_r F_r*C*4 + 24*K          (RMW of fp32 atomics)
  zero   = sum_l N*C*H_l*W_l*4                                 (clearing the gradients)
  U_*    = the same with sum_r F_r replaced by the size of the union of footprints
  T_fwd  = K*PH*PW*gh*gw*4*C*s_feat                            (every tap, no reuse)

24*K is the RoI (20 bytes) and level (4 bytes) read.  The footprints use the
binary32 sample geometry of the operator (numpy float32 arithmetic, one rounding
per operation); this module is measurement code and shares nothing with the
kernels or the oracle.
"""
from __future__ import annotations

import dataclasses
from typing import Sequence, Tuple

import numpy as np

F32 = np.float32


def _axis_taps(c1: np.ndarray, c2: np.ndarray, scale: float, aligned: bool, P: int, S: int,
               size: int):
    """Tap indices of every sample along one axis: lo, hi [K, P*S] (-1 where invalid)."""
    off = F32(0.5 if aligned else 0.0)
    s = c1.astype(F32) * F32(scale)
    s = s - off
    e = c2.astype(F32) * F32(scale)
    e = e - off
    ln = e - s
    if not aligned:
        ln = np.maximum(ln, F32(1.0))
    b = ln / F32(P)
    if S > 0:
        grid = np.full(c1.shape, S, dtype=np.int64)
    else:
        grid = np.where(b > 0, np.minimum(np.ceil(b), 64), 0).astype(np.int64)
    gmax = int(grid.max()) if grid.size else 0
    K = c1.shape[0]
    lo = np.full((K, P, max(gmax, 1)), -1, dtype=np.int64)
    hi = np.full((K, P, max(gmax, 1)), -1, dtype=np.int64)
    if gmax == 0:
        return lo.reshape(K, -1), hi.reshape(K, -1), grid
    p = np.arange(P, dtype=F32)[None, :, None]
    i = np.arange(gmax, dtype=F32)[None, None, :]
    t1 = p * b[:, None, None]
    t2 = s[:, None, None] + t1
    t3 = i + F32(0.5)
    t4 = t3 * b[:, None, None]
    t5 = t4 / np.maximum(grid, 1).astype(F32)[:, None, None]
    v = t2 + t5
    exists = np.arange(gmax)[None, None, :] < grid[:, None, None]
    valid = exists & ~((v < F32(-1.0)) | (v > F32(size)))
    v = np.maximum(v, F32(0.0))
    l = np.floor(v).astype(np.int64)
    h = l + 1
    edge = l >= size - 1
    l = np.where(edge, size - 1, l)
    h = np.where(edge, size - 1, h)
    lo[valid] = l[valid]
    hi[valid] = h[valid]
    return lo.reshape(K, -1), hi.reshape(K, -1), grid


def _distinct(lo: np.ndarray, hi: np.ndarray):
    """Per row: sorted distinct non-negative values of lo and hi."""
    both = np.sort(np.concatenate([lo, hi], axis=1), axis=1)
    keep = both >= 0
    keep[:, 1:] &= both[:, 1:] != both[:, :-1]
    return both, keep


@dataclasses.dataclass
class Bytes:
    K: int
    footprint_px: int        # sum over RoIs of F_r
    union_px: int            # pixels in the union of footprints
    taps_px: int             # sum over RoIs of PH*PW*gh*gw*4
    e_fwd: int
    e_bwd: int
    u_fwd: int
    u_bwd: int
    t_fwd: int
    zero: int
    out_bytes: int


def count(rois: np.ndarray, levels: np.ndarray, level_hw: Sequence[Tuple[int, int]],
          scales: Sequence[float], n_images: int, C: int, out_hw: Tuple[int, int], S: int,
          aligned: bool, s_feat: int, s_out: int, s_gout: int) -> Bytes:
    K = rois.shape[0]
    PH, PW = out_hw
    fp_total = 0
    union_total = 0
    taps_total = 0
    for l, ((H, W), sc) in enumerate(zip(level_hw, scales)):
        idx = np.flatnonzero(levels == l)
        if idx.size == 0:
            continue
        r = rois[idx]
        b = np.trunc(r[:, 0]).astype(np.int64)
        ok = (b >= 0) & (b < n_images)
        ylo, yhi, gy = _axis_taps(r[:, 2], r[:, 4], sc, aligned, PH, S, H)
        xlo, xhi, gx = _axis_taps(r[:, 1], r[:, 3], sc, aligned, PW, S, W)
        ys, ykeep = _distinct(ylo, yhi)
        xs, xkeep = _distinct(xlo, xhi)
        nrow = ykeep.sum(1)
        ncol = xkeep.sum(1)
        fp_total += int((nrow * ncol)[ok].sum())
        taps_total += int((PH * PW * gy * gx * 4)[ok].sum())
        masks = np.zeros((n_images, H, W), dtype=bool)
        for j in np.flatnonzero(ok):
            rows = ys[j][ykeep[j]]
            cols = xs[j][xkeep[j]]
            if rows.size and cols.size:
                masks[b[j]][np.ix_(rows, cols)] = True
        union_total += int(masks.sum())
    out_elems = K * C * PH * PW
    zero = sum(n_images * C * H * W * 4 for (H, W) in level_hw)
    return Bytes(
        K=K, footprint_px=fp_total, union_px=union_total, taps_px=taps_total,
        e_fwd=fp_total * C * s_feat + out_elems * s_out + 24 * K,
        e_bwd=out_elems * s_gout + 2 * fp_total * C * 4 + 24 * K,
        u_fwd=union_total * C * s_feat + out_elems * s_out + 24 * K,
        u_bwd=out_elems * s_gout + 2 * union_total * C * 4 + 24 * K,
        t_fwd=taps_total * C * s_feat, zero=zero, out_bytes=out_elems * s_out)


def _round_half_away(x32: np.ndarray) -> np.ndarray:
    """roundf of binary32 values (halves away from zero), exact in float64."""
    x = x32.astype(np.float64)
    return np.sign(x) * np.floor(np.abs(x) + 0.5)


@dataclasses.dataclass
class PoolBytes:
    K: int
    box_px: int              # sum over RoIs of the quantized box clipped to the map
    e_fwd: int               # box pixels x C read, values and argmax written
    e_bwd: int               # gradient and argmax read, one fp32 read-modify-write each
    zero: int
    g_bwd: int               # tile-gather form: gradient and argmax read, every element written once


def count_pool(rois: np.ndarray, levels: np.ndarray, level_hw: Sequence[Tuple[int, int]],
               scales: Sequence[float], n_images: int, C: int, out_hw: Tuple[int, int],
               s_feat: int, s_out: int, s_gout: int) -> PoolBytes:
    """Effective bytes of RoI max pooling.  The bins of a RoI tile its quantized box
    [round(x1 s), round(x2 s)] (both ends included) clipped to the map, so the forward
    reads that box once per channel:

      E_fwd = sum_r box_r*C*s_feat + K*C*PH*PW*(s_out + 4) + 24*K
      E_bwd = K*C*PH*PW*(s_gout + 4) + K*C*PH*PW*8 + 24*K     (+ clearing, reported apart)

    The tile-gather backward reads the upstream gradient and the argmax once and writes
    every element of the binary32 gradient pyramid once (no clearing, no atomics):

      G_bwd = K*C*PH*PW*(s_gout + 4) + 24*K + N*C*sum_l H_l*W_l*4
    """
    K = rois.shape[0]
    PH, PW = out_hw
    box = 0
    for l, ((H, W), sc) in enumerate(zip(level_hw, scales)):
        idx = np.flatnonzero(levels == l)
        if idx.size == 0:
            continue
        r = rois[idx]
        b = np.trunc(r[:, 0]).astype(np.int64)
        ok = (b >= 0) & (b < n_images)
        s = F32(sc)
        xs = _round_half_away(r[:, 1].astype(F32) * s)
        xe = _round_half_away(r[:, 3].astype(F32) * s)
        ys = _round_half_away(r[:, 2].astype(F32) * s)
        ye = _round_half_away(r[:, 4].astype(F32) * s)
        w = np.maximum(xe - xs + 1, 1)
        h = np.maximum(ye - ys + 1, 1)
        cols = np.clip(xs + w, 0, W) - np.clip(xs, 0, W)
        rows = np.clip(ys + h, 0, H) - np.clip(ys, 0, H)
        box += int((cols * rows)[ok].sum())
    elems = K * C * PH * PW
    zero = sum(n_images * C * H * W * 4 for (H, W) in level_hw)
    return PoolBytes(K=K, box_px=box, e_fwd=box * C * s_feat + elems * (s_out + 4) + 24 * K,
                     e_bwd=elems * (s_gout + 4) + elems * 8 + 24 * K, zero=zero,
                     g_bwd=elems * (s_gout + 4) + 24 * K + zero)


def deform_footprint(rois: np.ndarray, levels: np.ndarray, level_hw: Sequence[Tuple[int, int]],
                     scales: Sequence[float], n_images: int, out_hw: Tuple[int, int], S: int,
                     aligned: bool, offset: np.ndarray, gamma: float) -> int:
    """Sum over RoIs of the distinct pixels the bilinear corners of its shifted samples
    touch (float64 geometry; used only for byte counts)."""
    PH, PW = out_hw
    total = 0
    off_half = 0.5 if aligned else 0.0
    for k in range(rois.shape[0]):
        l = int(levels[k])
        if l < 0 or l >= len(level_hw) or not (0 <= int(rois[k, 0]) < n_images):
            continue
        H, W = level_hw[l]
        s = float(scales[l])
        x0 = float(rois[k, 1]) * s - off_half
        y0 = float(rois[k, 2]) * s - off_half
        w = float(rois[k, 3]) * s - off_half - x0
        h = float(rois[k, 4]) * s - off_half - y0
        if not aligned:
            w, h = max(w, 1.0), max(h, 1.0)
        bw, bh = w / PW, h / PH
        gx = S if S > 0 else max(1, min(64, int(np.ceil(bw))))
        gy = S if S > 0 else max(1, min(64, int(np.ceil(bh))))
        dx = gamma * offset[k, 0].astype(np.float64) * w
        dy = gamma * offset[k, 1].astype(np.float64) * h
        pw = np.arange(PW)[None, :, None, None]
        ph = np.arange(PH)[:, None, None, None]
        ix = np.arange(gx)[None, None, None, :]
        iy = np.arange(gy)[None, None, :, None]
        x = x0 + pw * bw + dx[:, :, None, None] + (ix + 0.5) * bw / gx
        y = y0 + ph * bh + dy[:, :, None, None] + (iy + 0.5) * bh / gy
        x, y = np.broadcast_arrays(x, y)
        ok = (x >= -1) & (x <= W) & (y >= -1) & (y <= H)
        xc = np.clip(x[ok], 0, W - 1)
        yc = np.clip(y[ok], 0, H - 1)
        xl = np.floor(xc).astype(np.int64)
        yl = np.floor(yc).astype(np.int64)
        xh = np.minimum(xl + 1, W - 1)
        yh = np.minimum(yl + 1, H - 1)
        px = np.concatenate([yl * W + xl, yl * W + xh, yh * W + xl, yh * W + xh])
        total += int(np.unique(px).size)
    return total
