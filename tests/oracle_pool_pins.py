"""Pins for the oracle's RoI max pooling: facts that do not come from the oracle.

  hand cases     values and argmax derived by hand (tests/golden/roi_pool_hand_cases.json):
                 quantization with halves rounded away from zero, the +1 box size,
                 clipping, an empty bin, ties, an invalid batch index
  global max     a box covering the whole map with one bin gives np.max, and the
                 argmax is np.argmax (first maximum in row-major order)
  crop           a box of exactly PH x PW pixels gives the crop itself
  block max      a 2m x 2m box pooled to m x m gives 2x2 max pooling (reshape + max)
  ramp bounds    on an increasing ramp the maximum of every bin is its last pixel, on
                 a decreasing ramp its first: the bins of a box tile it, in order,
                 each non-empty, consecutive bins overlapping by at most one pixel
  backward       the gradient is g placed at the argmax pixels (np.add.at), and for
                 the whole-map bin it is g at np.argmax
"""
from __future__ import annotations

import json
import os

import numpy as np

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _ramp(shape):
    n, c, h, w = shape
    f = 10.0 * np.arange(h)[:, None] + np.arange(w)[None, :]
    return np.broadcast_to(f, shape).astype(np.float64).copy()


def pin_pool_hand_cases(lib):
    cases = json.load(open(os.path.join(GOLDEN, "roi_pool_hand_cases.json")))["cases"]
    for case in cases:
        shape = tuple(case["shape"])
        f = _ramp(shape) if case["map"] == "ramp" else np.full(shape, case["fill"], np.float64)
        ph, pw = case["out"]
        out, am = oracle.roi_pool_fwd([f], [case["scale"]], np.array([case["roi"]], np.float32),
                                      None, ph, pw, lib=lib)
        assert np.array_equal(out[0, 0], np.array(case["expected"], np.float64)), (case["name"], out)
        assert np.array_equal(am[0, 0], np.array(case["argmax"], np.int32)), (case["name"], am)
        if "grad_out" in case:
            g = np.array(case["grad_out"], np.float64)[None, None]
            gr = oracle.roi_pool_bwd(g, am, [shape], np.array([case["roi"]], np.float32), None,
                                     lib=lib)[0]
            exp = np.zeros(shape)
            for idx, v in case["grad_at"].items():
                exp.reshape(-1)[int(idx)] = v
            assert np.array_equal(gr, exp), (case["name"], gr)


def pin_pool_global_max(lib):
    rng = np.random.default_rng(1)
    for (h, w) in [(5, 7), (1, 1), (6, 3)]:
        f = rng.integers(-20, 20, (1, 2, h, w)).astype(np.float64)   # many ties
        roi = np.array([[0, 0, 0, w - 1, h - 1]], np.float32)
        out, am = oracle.roi_pool_fwd([f], [1.0], roi, None, 1, 1, lib=lib)
        for c in range(2):
            assert out[0, c, 0, 0] == f[0, c].max()
            assert am[0, c, 0, 0] == int(np.argmax(f[0, c]))
        g = rng.standard_normal((1, 2, 1, 1))
        gr = oracle.roi_pool_bwd(g, am, [f.shape], roi, None, lib=lib)[0]
        exp = np.zeros(f.shape)
        for c in range(2):
            exp[0, c].reshape(-1)[np.argmax(f[0, c])] = g[0, c, 0, 0]
        assert np.array_equal(gr, exp)


def pin_pool_crop(lib):
    rng = np.random.default_rng(2)
    f = rng.standard_normal((2, 3, 9, 11))
    for (b, x0, y0, ph, pw) in [(0, 2, 1, 4, 5), (1, 0, 0, 9, 11), (1, 6, 4, 3, 2)]:
        roi = np.array([[b, x0, y0, x0 + pw - 1, y0 + ph - 1]], np.float32)
        out, am = oracle.roi_pool_fwd([f], [1.0], roi, None, ph, pw, lib=lib)
        assert np.array_equal(out[0], f[b, :, y0:y0 + ph, x0:x0 + pw])
        ys, xs = np.meshgrid(np.arange(y0, y0 + ph), np.arange(x0, x0 + pw), indexing="ij")
        assert np.array_equal(am[0], np.broadcast_to(ys * 11 + xs, am[0].shape))


def pin_pool_block_max(lib):
    rng = np.random.default_rng(3)
    f = rng.standard_normal((1, 4, 12, 10))
    for (m, x0, y0) in [(3, 0, 0), (2, 4, 6), (5, 0, 2)]:
        roi = np.array([[0, x0, y0, x0 + 2 * m - 1, y0 + 2 * m - 1]], np.float32)
        out, am = oracle.roi_pool_fwd([f], [1.0], roi, None, m, m, lib=lib)
        blk = f[0, :, y0:y0 + 2 * m, x0:x0 + 2 * m].reshape(4, m, 2, m, 2)
        assert np.array_equal(out[0], blk.max(axis=(2, 4)))
        g = rng.standard_normal(out.shape)
        gr = oracle.roi_pool_bwd(g, am, [f.shape], roi, None, lib=lib)[0]
        exp = np.zeros(f.shape)
        sub = blk.transpose(0, 1, 3, 2, 4).reshape(4, m, m, 4)
        first = sub.argmax(axis=3)   # first maximum within each 2x2 block, row-major
        for c in range(4):
            for i in range(m):
                for j in range(m):
                    dy, dx = divmod(int(first[c, i, j]), 2)
                    exp[0, c, y0 + 2 * i + dy, x0 + 2 * j + dx] += g[0, c, i, j]
        assert np.allclose(gr, exp, rtol=0, atol=1e-15)


def pin_pool_ramp_bounds(lib):
    rng = np.random.default_rng(4)
    H, W = 40, 50
    inc = np.broadcast_to(1000.0 * np.arange(H)[:, None] + np.arange(W), (1, 1, H, W)).copy()
    rois = []
    for _ in range(40):
        x1, x2 = np.sort(rng.uniform(0, W - 1, 2))
        y1, y2 = np.sort(rng.uniform(0, H - 1, 2))
        rois.append([0, x1, y1, x2, y2])
    rois = np.array(rois, np.float32)
    for (ph, pw) in [(7, 7), (3, 5), (1, 4)]:
        oi, ai = oracle.roi_pool_fwd([inc], [1.0], rois, None, ph, pw, lib=lib)
        od, ad = oracle.roi_pool_fwd([-inc], [1.0], rois, None, ph, pw, lib=lib)
        for k in range(len(rois)):
            # halves away from zero (coordinates here are positive)
            sx, ex = np.floor(rois[k, 1] + 0.5), np.floor(rois[k, 3] + 0.5)
            sy, ey = np.floor(rois[k, 2] + 0.5), np.floor(rois[k, 4] + 0.5)
            last = ai[k, 0]            # bottom-right pixel of each bin
            first = ad[k, 0]           # top-left pixel of each bin
            assert (last >= 0).all() and (first >= 0).all()   # no empty bins inside the map
            ly, lx = last // W, last % W
            fy, fx = first // W, first % W
            # the bins tile the box: first bin starts at the box start, last ends at its end
            assert (fy[0] == sy).all() and (fx[:, 0] == sx).all()
            assert (ly[-1] == ey).all() and (lx[:, -1] == ex).all()
            # in order, each bin starting at or before the previous end + 1, overlap <= 1 px
            assert (fy[1:] <= ly[:-1] + 1).all() and (fy[1:] >= ly[:-1]).all()
            assert (fx[:, 1:] <= lx[:, :-1] + 1).all() and (fx[:, 1:] >= lx[:, :-1]).all()


ALL_POOL_PINS = [pin_pool_hand_cases, pin_pool_global_max, pin_pool_crop, pin_pool_block_max,
                 pin_pool_ramp_bounds]


def run_all(lib):
    failures = []
    for pin in ALL_POOL_PINS:
        try:
            pin(lib)
        except AssertionError as e:
            failures.append((pin.__name__, str(e)[:200]))
    return failures
