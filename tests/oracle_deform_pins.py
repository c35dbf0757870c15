"""Pins for the oracle's deformable (modulated) RoI pooling: facts that do not come from
the oracle's deformable code.

  zero offsets     with every offset 0 and no mask the operator is RoIAlign: the
                   forward and the feature gradient equal the (separately pinned)
                   RoIAlign oracle's bit for bit, and with a mask of ones the mask
                   gradient is sum_c g * out
  constant map     F = c gives c * mask wherever all samples are valid
  affine map       F = a + b x + e y: bilinear sampling is exact, so a bin's average is
                   a + b (x0 + (pw + 1/2) bw + dx) + e (y0 + (ph + 1/2) bh + dy), the
                   offset gradients are sum_c g m b gamma w and sum_c g m e gamma h,
                   and the mask gradient is sum_c g * (unmodulated average)
  mask linearity   out(mask) = mask * out(no mask)
  finite diffs     central differences of the forward in the offsets and the mask
                   match the gradients (the forward is piecewise bilinear in the
                   shift, so a tiny step is exact away from pixel boundaries); boxes
                   that stick out of the map check the zero slope of clamped samples
  adjoint          <fwd(x), g> = <x, bwd(g)> for the feature gradient
  brute force      every sample as a tent-kernel sum over all pixels, written here
  integer shift    a shift of exactly 2 pixels equals RoIAlign of the box moved by
                   2 pixels (math mode)
  parity vs math   the binary32-geometry gradients follow the finite-difference pinned
                   math-mode ones within the rounding scale, clamped samples included
  binary32 order   hand-derived binary32 sample coordinates on a ramp map fix where the
                   shift enters the rounded sum (tests/golden/deform_binary32_cases.json)
"""
from __future__ import annotations

import numpy as np

import oracle

# gamma reaches the operator as a binary32 value
G01 = float(np.float32(0.1))


def _map(rng, shapes):
    return [rng.standard_normal(s) for s in shapes]


def _interior_rois(rng, K, H, W, scale, margin=3.0, n_images=1):
    """Boxes (in image pixels) whose bins, shifted by at most `margin` feature pixels,
    keep every sample inside [0, W-1) x [0, H-1)."""
    r = np.zeros((K, 5), np.float32)
    for k in range(K):
        w = rng.uniform(2.0, (W - 2 * margin - 2) * 0.6)
        h = rng.uniform(2.0, (H - 2 * margin - 2) * 0.6)
        x0 = rng.uniform(margin + 0.5, W - 1 - margin - w)
        y0 = rng.uniform(margin + 0.5, H - 1 - margin - h)
        r[k] = [rng.integers(0, n_images), (x0 + 0.5) / scale, (y0 + 0.5) / scale,
                (x0 + w + 0.5) / scale, (y0 + h + 0.5) / scale]
    return r


def _offsets(rng, K, PH, PW, amp):
    return rng.uniform(-amp, amp, (K, 2, PH, PW)).astype(np.float32)


def pin_zero_offsets_are_roialign(lib, mode):
    rng = np.random.default_rng(1)
    shapes = [(2, 3, 14, 18), (2, 3, 7, 9)]
    scales = [0.25, 0.125]
    f = _map(rng, shapes)
    rois = np.zeros((9, 5), np.float32)
    a = rng.uniform(-10, 80, (9, 2))
    b = rng.uniform(-10, 60, (9, 2))
    rois[:, 0] = rng.integers(0, 2, 9)
    rois[:, 1], rois[:, 3] = a.min(1), a.max(1)
    rois[:, 2], rois[:, 4] = b.min(1), b.max(1)
    lv = np.arange(9, dtype=np.int32) % 2
    for S, aligned in [(2, True), (0, False), (3, True)]:
        off = np.zeros((9, 2, 3, 4), np.float32)
        got = oracle.deform_roi_pool_fwd(f, scales, rois, lv, 3, 4, S, aligned, off, None,
                                         0.1, mode, lib=lib)
        ref = oracle.roi_align_fwd(f, scales, rois, lv, 3, 4, S, aligned, mode, lib=lib)
        assert np.array_equal(got, ref), "zero offsets: forward differs from RoIAlign"
        g = rng.standard_normal(got.shape)
        gf, _, _, _, _ = oracle.deform_roi_pool_bwd(g, f, scales, rois, lv, 3, 4, S, aligned,
                                                    off, None, 0.1, mode, lib=lib)
        gr = oracle.roi_align_bwd(g, shapes, scales, rois, lv, 3, 4, S, aligned, mode, lib=lib)
        for x, y in zip(gf, gr):
            assert np.array_equal(x, y), "zero offsets: feature gradient differs from RoIAlign"
        ones = np.ones((9, 3, 4), np.float32)
        _, _, gm, _, _ = oracle.deform_roi_pool_bwd(g, f, scales, rois, lv, 3, 4, S, aligned,
                                                    off, ones, 0.1, mode, lib=lib)
        assert np.allclose(gm, (g * ref).sum(1), rtol=1e-12, atol=1e-12), "mask gradient"


def pin_constant_map(lib, mode):
    rng = np.random.default_rng(2)
    H, W, s = 20, 24, 0.5
    f = [np.full((1, 2, H, W), 3.25)]
    rois = _interior_rois(rng, 6, H, W, s)
    off = _offsets(rng, 6, 3, 3, 0.3)
    m = rng.uniform(0.1, 1.0, (6, 3, 3)).astype(np.float32)
    out = oracle.deform_roi_pool_fwd(f, [s], rois, None, 3, 3, 2, True, off, m, 0.1, mode,
                                     lib=lib)
    assert np.allclose(out, 3.25 * m[:, None].astype(np.float64), rtol=1e-6, atol=1e-12), \
        "constant map"


def pin_affine_closed_form(lib, mode):
    rng = np.random.default_rng(3)
    H, W, s, gamma = 30, 40, 0.5, G01
    C = 3
    al, be, ep = rng.standard_normal(C), rng.standard_normal(C), rng.standard_normal(C)
    yy, xx = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    f = [(al[:, None, None] + be[:, None, None] * xx + ep[:, None, None] * yy)[None]]
    K, PH, PW = 7, 3, 4
    rois = _interior_rois(rng, K, H, W, s, margin=3.0)
    off = _offsets(rng, K, PH, PW, 0.4)
    m = rng.uniform(0.2, 1.0, (K, PH, PW)).astype(np.float32)
    out = oracle.deform_roi_pool_fwd(f, [s], rois, None, PH, PW, 2, True, off, m, gamma, mode,
                                     lib=lib)
    g = rng.standard_normal(out.shape)
    _, goff, gm, _, _ = oracle.deform_roi_pool_bwd(g, f, [s], rois, None, PH, PW, 2, True, off,
                                                   m, gamma, mode, lib=lib)
    tol = 1e-9 if mode == "math" else 1e-4
    for k in range(K):
        x0 = float(rois[k, 1]) * s - 0.5
        y0 = float(rois[k, 2]) * s - 0.5
        w = float(rois[k, 3]) * s - float(rois[k, 1]) * s
        h = float(rois[k, 4]) * s - float(rois[k, 2]) * s
        for ph in range(PH):
            for pw in range(PW):
                dx = gamma * float(off[k, 0, ph, pw]) * w
                dy = gamma * float(off[k, 1, ph, pw]) * h
                xc = x0 + (pw + 0.5) * w / PW + dx
                yc = y0 + (ph + 0.5) * h / PH + dy
                avg = al + be * xc + ep * yc
                mm = float(m[k, ph, pw])
                assert np.allclose(out[k, :, ph, pw], mm * avg, rtol=tol, atol=tol), "affine fwd"
                gx = float((g[k, :, ph, pw] * mm * be).sum() * gamma * w)
                gy = float((g[k, :, ph, pw] * mm * ep).sum() * gamma * h)
                gmm = float((g[k, :, ph, pw] * avg).sum())
                assert abs(goff[k, 0, ph, pw] - gx) <= tol * (1 + abs(gx)), "affine offset x"
                assert abs(goff[k, 1, ph, pw] - gy) <= tol * (1 + abs(gy)), "affine offset y"
                assert abs(gm[k, ph, pw] - gmm) <= tol * (1 + abs(gmm)), "affine mask gradient"


def pin_mask_linearity(lib, mode):
    rng = np.random.default_rng(4)
    f = _map(rng, [(1, 4, 16, 20)])
    rois = np.array([[0, 3, 2, 50, 40], [0, -8, -6, 30, 70], [0, 10, 10, 11, 12]], np.float32)
    off = _offsets(rng, 3, 5, 5, 0.5)
    m = rng.uniform(-1.0, 2.0, (3, 5, 5)).astype(np.float32)
    a = oracle.deform_roi_pool_fwd(f, [0.25], rois, None, 5, 5, 2, True, off, m, 0.1, mode,
                                   lib=lib)
    b = oracle.deform_roi_pool_fwd(f, [0.25], rois, None, 5, 5, 2, True, off, None, 0.1, mode,
                                   lib=lib)
    assert np.array_equal(a, m[:, None].astype(np.float64) * b), "mask linearity"


def pin_finite_differences(lib, mode):
    """Central differences of sum(g * out) in every offset and mask entry (math mode)."""
    rng = np.random.default_rng(5)
    shapes = [(1, 3, 12, 15)]
    f = _map(rng, shapes)
    s, gamma, PH, PW = 0.25, G01, 3, 3
    # an interior box and two that stick out of the map on the low and the high side
    rois = np.array([[0, 9.0, 7.0, 41.0, 33.0], [0, -5.0, -3.0, 20.0, 18.0],
                     [0, 35.0, 30.0, 63.0, 52.0]], np.float32)
    K = rois.shape[0]
    off = _offsets(rng, K, PH, PW, 0.6)
    m = rng.uniform(0.2, 1.0, (K, PH, PW)).astype(np.float32)
    g = rng.standard_normal((K, 3, PH, PW))
    _, goff, gm, _, _ = oracle.deform_roi_pool_bwd(g, f, [s], rois, None, PH, PW, 2, True, off, m,
                                                   gamma, mode, lib=lib)

    def loss(o, mm):
        out = oracle.deform_roi_pool_fwd(f, [s], rois, None, PH, PW, 2, True, o, mm, gamma, mode,
                                         lib=lib)
        return float((g * out).sum())

    hstep = 1e-3
    for k in range(K):
        for a in range(2):
            for ph in range(PH):
                for pw in range(PW):
                    # offsets are binary32: steps of 2^-10 are exact around values of
                    # magnitude < 1, and the shift stays far from any pixel boundary
                    # crossing for all but a measure-zero set of draws
                    op = off.copy()
                    om = off.copy()
                    op[k, a, ph, pw] += hstep
                    om[k, a, ph, pw] -= hstep
                    fd = (loss(op, m) - loss(om, m)) / (float(op[k, a, ph, pw]) -
                                                        float(om[k, a, ph, pw]))
                    assert abs(fd - goff[k, a, ph, pw]) <= 1e-6 * (1 + abs(fd)), \
                        "offset gradient vs finite difference at %s" % ((k, a, ph, pw),)
        for ph in range(PH):
            for pw in range(PW):
                mp = m.copy()
                mn = m.copy()
                mp[k, ph, pw] += 0.25
                mn[k, ph, pw] -= 0.25
                fd = (loss(off, mp) - loss(off, mn)) / (float(mp[k, ph, pw]) -
                                                         float(mn[k, ph, pw]))
                assert abs(fd - gm[k, ph, pw]) <= 1e-9 * (1 + abs(fd)), "mask gradient vs FD"


def pin_adjoint(lib, mode):
    rng = np.random.default_rng(6)
    shapes = [(2, 3, 10, 13), (2, 3, 5, 7)]
    scales = [0.5, 0.25]
    f = _map(rng, shapes)
    rois = np.array([[0, 1, 2, 15, 17], [1, -4, 3, 30, 14], [1, 5, 5, 6, 6], [0, 2, 0, 25, 19]],
                    np.float32)
    lv = np.array([0, 1, 0, 1], np.int32)
    off = _offsets(rng, 4, 4, 3, 1.5)
    m = rng.uniform(-1, 1, (4, 4, 3)).astype(np.float32)
    out = oracle.deform_roi_pool_fwd(f, scales, rois, lv, 4, 3, 2, True, off, m, 0.1, mode,
                                     lib=lib)
    g = rng.standard_normal(out.shape)
    gf, _, _, _, _ = oracle.deform_roi_pool_bwd(g, f, scales, rois, lv, 4, 3, 2, True, off, m, 0.1,
                                                mode, lib=lib)
    lhs = float((out * g).sum())
    rhs = float(sum((a * b).sum() for a, b in zip(f, gf)))
    assert abs(lhs - rhs) <= 1e-10 * max(1.0, abs(lhs)), "adjoint identity"


def pin_brute_force_tent(lib, mode):
    """Every sample written out here (math geometry) as a sum over all pixels of the
    tent kernel max(0, 1 - |t - i|) at the clamped coordinates."""
    rng = np.random.default_rng(7)
    H, W, C = 5, 6, 2
    f = [rng.standard_normal((1, C, H, W))]
    s, gamma, PH, PW, S = 1.0, G01, 2, 3, 2
    rois = np.array([[0, -0.8, 0.3, 4.9, 4.2], [0, 1.2, -0.4, 3.3, 2.6]], np.float32)
    off = _offsets(rng, 2, PH, PW, 2.0)
    m = rng.uniform(0.5, 1.5, (2, PH, PW)).astype(np.float32)
    out = oracle.deform_roi_pool_fwd(f, [s], rois, None, PH, PW, S, True, off, m, gamma, "math",
                                     lib=lib)
    for k in range(2):
        x0 = float(rois[k, 1]) * s - 0.5
        y0 = float(rois[k, 2]) * s - 0.5
        w = float(rois[k, 3]) * s - 0.5 - x0
        h = float(rois[k, 4]) * s - 0.5 - y0
        for ph in range(PH):
            for pw in range(PW):
                dx = gamma * float(off[k, 0, ph, pw]) * w
                dy = gamma * float(off[k, 1, ph, pw]) * h
                acc = np.zeros(C)
                for iy in range(S):
                    y = y0 + ph * h / PH + dy + (iy + 0.5) * (h / PH) / S
                    for ix in range(S):
                        x = x0 + pw * w / PW + dx + (ix + 0.5) * (w / PW) / S
                        if y < -1 or y > H or x < -1 or x > W:
                            continue
                        yc = min(max(y, 0.0), H - 1.0)
                        xc = min(max(x, 0.0), W - 1.0)
                        ty = np.maximum(0.0, 1 - np.abs(yc - np.arange(H)))
                        tx = np.maximum(0.0, 1 - np.abs(xc - np.arange(W)))
                        acc += np.einsum("i,j,cij->c", ty, tx, f[0][0])
                ref = float(m[k, ph, pw]) * acc / (S * S)
                assert np.allclose(out[k, :, ph, pw], ref, rtol=1e-12, atol=1e-12), "brute force"


def pin_integer_shift(lib, mode):
    rng = np.random.default_rng(8)
    H, W, s, gamma = 20, 26, 0.5, G01
    f = _map(rng, [(1, 3, H, W)])
    rois = _interior_rois(rng, 5, H, W, s, margin=3.0)
    off = np.zeros((5, 2, 2, 3), np.float32)
    w = rois[:, 3].astype(np.float64) * s - rois[:, 1].astype(np.float64) * s
    h = rois[:, 4].astype(np.float64) * s - rois[:, 2].astype(np.float64) * s
    off[:, 0] = (2.0 / (gamma * w))[:, None, None]
    off[:, 1] = (-1.0 / (gamma * h))[:, None, None]
    got = oracle.deform_roi_pool_fwd(f, [s], rois, None, 2, 3, 2, True, off, None, gamma, "math",
                                     lib=lib)
    moved = rois.copy()
    moved[:, 1] += 2.0 / s
    moved[:, 3] += 2.0 / s
    moved[:, 2] -= 1.0 / s
    moved[:, 4] -= 1.0 / s
    ref = oracle.roi_align_fwd(f, [s], moved, None, 2, 3, 2, True, "math", lib=lib)
    # the shift is 2 (and -1) pixels up to the binary32 offsets: compare to 1e-5
    assert np.allclose(got, ref, rtol=1e-5, atol=1e-5), "integer shift"


def pin_parity_gradients_follow_math(lib, mode):
    """The binary32 geometry only moves samples by rounding, so on random inputs the
    parity-mode gradients equal the (finite-difference pinned) math-mode gradients to
    within the rounding scale; boxes that stick out of the map on both sides make
    clamped samples (zero slope) part of the comparison."""
    rng = np.random.default_rng(9)
    shapes = [(2, 4, 14, 17), (2, 4, 7, 9)]
    scales = [0.25, 0.125]
    f = _map(rng, shapes)
    rois = np.array([[0, -6.0, -5.0, 30.0, 26.0], [1, 20.0, 14.0, 75.0, 60.0],
                     [0, 9.0, 7.0, 41.0, 33.0], [1, -3.0, 30.0, 40.0, 90.0]], np.float32)
    lv = np.array([0, 0, 1, 1], np.int32)
    off = _offsets(rng, 4, 3, 3, 0.8)
    m = rng.uniform(0.2, 1.0, (4, 3, 3)).astype(np.float32)
    g = rng.standard_normal((4, 4, 3, 3))
    res = {md: oracle.deform_roi_pool_bwd(g, f, scales, rois, lv, 3, 3, 2, True, off, m, G01, md,
                                          lib=lib) for md in ("math", "parity")}
    _, om, mm, so, sm = res["math"]
    _, op, mp, _, _ = res["parity"]
    assert np.all(np.abs(op - om) <= 1e-4 * (so + 1e-12)), "parity offset gradient"
    assert np.all(np.abs(mp - mm) <= 1e-4 * (sm + 1e-12)), "parity mask gradient"


def pin_binary32_shift_order(lib, mode):
    """Hand-derived binary32 sample coordinates (tests/golden/deform_binary32_cases.json)
    that fix where the bin shift enters the rounded sum: after the bin start is rounded
    and before the within-bin offset.  A ramp map returns the sample coordinate, so one
    ulp of difference shows; the comparison is exact."""
    import json
    import os
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                        "deform_binary32_cases.json")
    with open(path) as f:
        cases = json.load(f)["cases"]
    for case in cases:
        shape = tuple(case["shape"])
        feat = np.broadcast_to(np.arange(shape[3], dtype=np.float64), shape).copy()
        ph, pw = case["out"]
        out = oracle.deform_roi_pool_fwd([feat], [case["scale"]],
                                         np.array(case["rois"], np.float32), None, ph, pw,
                                         case["sampling_ratio"], case["aligned"],
                                         np.array(case["offset"], np.float32),
                                         gamma=case["gamma"], mode=mode, lib=lib)
        exp = np.array(case["expected_parity" if mode == "parity" else "expected_math"])
        rtol = 0.0 if mode == "parity" else 1e-12
        assert np.allclose(out, exp, rtol=rtol, atol=0.0), (case["name"], mode, out.ravel())


ALL_DEFORM_PINS = [pin_zero_offsets_are_roialign, pin_constant_map, pin_mask_linearity,
                   pin_adjoint, pin_binary32_shift_order]
AFFINE_PINS = [pin_affine_closed_form]
MATH_ONLY_DEFORM_PINS = [pin_finite_differences, pin_brute_force_tent, pin_integer_shift,
                         pin_parity_gradients_follow_math]


def run_all(lib):
    """Names of the pins that fail on `lib` (every mode each pin takes)."""
    failures = []
    for pin in ALL_DEFORM_PINS + AFFINE_PINS:
        for mode in ("math", "parity"):
            try:
                pin(lib, mode)
            except AssertionError:
                failures.append("%s/%s" % (pin.__name__, mode))
    for pin in MATH_ONLY_DEFORM_PINS:
        try:
            pin(lib, "math")
        except AssertionError:
            failures.append(pin.__name__)
    return failures
