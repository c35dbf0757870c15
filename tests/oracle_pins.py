"""Pins for the CPU oracle: checks against facts that do not come from the oracle.

Every function takes a loaded oracle library (``lib``) and a geometry mode and
raises AssertionError when the oracle disagrees with a fact fixed by the paper's
operator and by mathematics:

  hand cases      values derived by hand (tests/golden/), incl. the -1/size cut,
                  the divisor that counts invalid samples, clamping, adaptive grid
  binary32 order  hand-derived binary32 sample coordinates on ramp maps: the order
                  and association of every rounding step of the geometry, the grid cap
  level cases     hand-derived FPN level thresholds, bit-exact (golden)
  constant        a constant map returns the constant (weights sum to one)
  affine          on an affine map a bin average is the affine value at the bin centre
  adjoint         <fwd(x), g> = <x, bwd(g)>
  tent            brute force: bilinear value written as a sum of tent kernels over
                  every pixel (independent of the corner/index code)
  dense matrix    bwd(g) equals A^T g with A assembled column by column from fwd
  textbook        aligned box on integer grid = 2x2 average pooling / exact crop
  mirror          flipping the map and the box flips the output
  mass            with every sample valid, sum of grad_features equals sum of grad_out

They are plain functions so the same checks can be aimed at deliberately broken
copies of the oracle (the planted-mistake tests) as well as at the real one.
"""
from __future__ import annotations

import json
import os

import numpy as np

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _tol(mode, math_tol, parity_tol):
    return math_tol if mode == "math" else parity_tol


# ---------------------------------------------------------------------------
# golden fixtures
# ---------------------------------------------------------------------------

def load_hand_cases():
    with open(os.path.join(GOLDEN, "roi_align_hand_cases.json")) as f:
        return json.load(f)["cases"]


def _case_levels(case):
    feats, scales = [], []
    for lv in case["levels"]:
        shape = tuple(lv["shape"])
        if "fill" in lv:
            f = np.full(shape, lv["fill"], dtype=np.float64)
        elif lv.get("ramp_x"):
            f = np.broadcast_to(np.arange(shape[3], dtype=np.float64), shape).copy()
        else:
            f = np.array(lv["values"], dtype=np.float64).reshape(shape)
        feats.append(f)
        scales.append(lv["scale"])
    return feats, scales


def pin_hand_cases(lib, mode):
    for case in load_hand_cases():
        feats, scales = _case_levels(case)
        ph, pw = case["out"]
        out = oracle.roi_align_fwd(feats, scales, np.array(case["rois"], np.float32),
                                   np.array(case["roi_levels"], np.int32), ph, pw,
                                   case["sampling_ratio"], case["aligned"], mode, lib=lib)
        exp = np.array(case["expected"], dtype=np.float64)
        assert out.shape == exp.shape, case["name"]
        tol = _tol(mode, 1e-12, 2e-6)
        assert np.allclose(out, exp, rtol=tol, atol=tol), (case["name"], out, exp)


def load_binary32_cases():
    with open(os.path.join(GOLDEN, "roi_align_binary32_cases.json")) as f:
        return json.load(f)["cases"]


def pin_binary32_order(lib, mode):
    """Hand-derived sample coordinates that fix the binary32 order of the geometry (which
    association of the bin start and the within-bin offset, where the division by the
    grid comes, IEEE division for the bin size) and the adaptive-grid cap.  A ramp map
    returns the sample coordinate itself, so one ulp of difference in any rounding step
    shows; the comparison is therefore exact up to double rounding of the final mean."""
    for case in load_binary32_cases():
        feats, scales = _case_levels(case)
        ph, pw = case["out"]
        out = oracle.roi_align_fwd(feats, scales, np.array(case["rois"], np.float32),
                                   np.array(case["roi_levels"], np.int32), ph, pw,
                                   case["sampling_ratio"], case["aligned"], mode, lib=lib)
        exp = np.array(case["expected_parity" if mode == "parity" else "expected_math"],
                       dtype=np.float64)
        assert out.shape == exp.shape, case["name"]
        rtol = 1e-14 if mode == "parity" else 1e-12
        assert np.allclose(out, exp, rtol=rtol, atol=0.0), (case["name"], mode, out.ravel(),
                                                            exp.ravel())


def load_level_cases():
    rows = []
    with open(os.path.join(GOLDEN, "level_map_cases.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            v = line.split()
            plus1 = bool(int(v[7])) if len(v) > 7 else False
            rows.append(([0.0] + [float(x) for x in v[:4]], int(v[4]), float(v[5]), int(v[6]),
                         plus1))
    return rows


def pin_level_cases(lib, mode=None):
    for roi, L, fs, exp, plus1 in load_level_cases():
        got = oracle.level_map(np.array([roi], np.float32), L, fs, box_plus1=plus1, lib=lib)[0]
        assert got == exp, (roi, L, fs, plus1, got, exp)


def pin_level_plus1_is_shifted_box(lib, mode=None):
    """Inclusive pixel boxes: on integer coordinates (where every difference is
    exact) the level of (x1, y1, x2, y2) with box_plus1 is the level of the continuous
    box (x1, y1, x2 + 1, y2 + 1)."""
    rng = np.random.default_rng(11)
    K = 3000
    xy = rng.integers(0, 1000, (K, 2))
    wh = rng.integers(0, 700, (K, 2))
    rois = np.zeros((K, 5), np.float32)
    rois[:, 1:3] = xy
    rois[:, 3:5] = xy + wh
    shifted = rois.copy()
    shifted[:, 3:5] += 1
    a = oracle.level_map(rois, 4, 56.0, box_plus1=True, lib=lib)
    b = oracle.level_map(shifted, 4, 56.0, lib=lib)
    assert np.array_equal(a, b)
    assert set(np.unique(a)) == {0, 1, 2, 3}


def pin_level_log2_agrees(lib, mode=None):
    """Threshold form == logarithmic form away from the thresholds (random boxes)."""
    rng = np.random.default_rng(7)
    K = 4000
    xy = rng.uniform(0, 1000, (K, 2))
    wh = np.exp(rng.uniform(np.log(2), np.log(1500), (K, 2)))
    rois = np.zeros((K, 5), np.float32)
    rois[:, 1:3] = xy
    rois[:, 3:5] = xy + wh
    for plus1 in (False, True):
        a = oracle.level_map(rois, 4, 56.0, box_plus1=plus1, lib=lib)
        b = oracle.level_map_log2(rois, 4, 56.0, box_plus1=plus1, lib=lib)
        w = rois[:, 3].astype(np.float64) - rois[:, 1] + plus1
        h = rois[:, 4].astype(np.float64) - rois[:, 2] + plus1
        s = np.sqrt(w * h)
        near = np.zeros(K, bool)
        for t in (112.0, 224.0, 448.0):
            near |= np.abs(s / t - 1.0) < 1e-5
        assert np.array_equal(a[~near], b[~near])
        assert set(np.unique(a)) == {0, 1, 2, 3}


# ---------------------------------------------------------------------------
# random helpers
# ---------------------------------------------------------------------------

def _rand_rois_inside(rng, K, n_images, img_w, img_h, lo=2.0, hi=None):
    hi = hi or min(img_w, img_h)
    r = np.zeros((K, 5), np.float32)
    w = rng.uniform(lo, hi, K)
    h = rng.uniform(lo, hi, K)
    x1 = rng.uniform(0, img_w - w)
    y1 = rng.uniform(0, img_h - h)
    r[:, 0] = rng.integers(0, n_images, K)
    r[:, 1], r[:, 2], r[:, 3], r[:, 4] = x1, y1, x1 + w, y1 + h
    return r


def _rand_rois_anywhere(rng, K, n_images, img_w, img_h):
    r = np.zeros((K, 5), np.float32)
    a = rng.uniform(-0.3 * img_w, 1.3 * img_w, (K, 2))
    b = rng.uniform(-0.3 * img_h, 1.3 * img_h, (K, 2))
    r[:, 0] = rng.integers(0, n_images, K)
    r[:, 1], r[:, 3] = a.min(1), a.max(1)
    r[:, 2], r[:, 4] = b.min(1), b.max(1)
    return r


# ---------------------------------------------------------------------------
# invariants and closed forms
# ---------------------------------------------------------------------------

def pin_constant(lib, mode):
    """Constant maps (a different constant per level and image) return the constant."""
    rng = np.random.default_rng(11)
    shapes = [(2, 3, 24, 32), (2, 3, 12, 16)]
    scales = [0.25, 0.125]
    feats = []
    for l, s in enumerate(shapes):
        f = np.empty(s)
        for b in range(s[0]):
            f[b] = 1.5 + l + 10 * b
        feats.append(f)
    rois = _rand_rois_inside(rng, 24, 2, 128, 96, 4.0, 90.0)
    lv = rng.integers(0, 2, 24).astype(np.int32)
    for S in (1, 2, 0):
        for aligned in (True, False):
            out = oracle.roi_align_fwd(feats, scales, rois, lv, 3, 4, S, aligned, mode, lib=lib)
            exp = (1.5 + lv + 10 * rois[:, 0].astype(int))[:, None, None, None]
            tol = _tol(mode, 1e-12, 1e-6)
            assert np.allclose(out, np.broadcast_to(exp, out.shape), rtol=tol, atol=tol), \
                (S, aligned)


def pin_affine(lib, mode):
    """Affine map a + b*x + c*y: a bin average equals the affine value at the bin centre
    (bilinear interpolation reproduces affine functions; the mean of (i + 1/2)/g over a
    grid of g samples is 1/2)."""
    rng = np.random.default_rng(12)
    H, W, C = 20, 28, 3
    scale = 0.5
    alpha, beta, gamma = rng.normal(size=C), rng.normal(size=C), rng.normal(size=C)
    yy, xx = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    f = alpha[:, None, None] + beta[:, None, None] * xx + gamma[:, None, None] * yy
    feats = [f[None]]
    # keep every sample inside [1, size - 2] so no clamping happens
    K = 16
    rois = np.zeros((K, 5), np.float32)
    w = rng.uniform(1.0, 2 * (W - 4) - 10, K)
    h = rng.uniform(1.0, 2 * (H - 4) - 10, K)
    x1 = rng.uniform(3.0 + 1.0, 2 * (W - 2) - w - 1.0)
    y1 = rng.uniform(3.0 + 1.0, 2 * (H - 2) - h - 1.0)
    rois[:, 1], rois[:, 2], rois[:, 3], rois[:, 4] = x1, y1, x1 + w, y1 + h
    lv = np.zeros(K, np.int32)
    PH, PW = 3, 5
    for S in (1, 2, 3, 0):
        for aligned in (True, False):
            out = oracle.roi_align_fwd(feats, [scale], rois, lv, PH, PW, S, aligned, mode,
                                       lib=lib)
            off = 0.5 if aligned else 0.0
            r = rois.astype(np.float64)
            x0 = r[:, 1] * scale - off
            y0 = r[:, 2] * scale - off
            rw = r[:, 3] * scale - off - x0
            rh = r[:, 4] * scale - off - y0
            if not aligned:
                rw, rh = np.maximum(rw, 1.0), np.maximum(rh, 1.0)
            bw, bh = rw / PW, rh / PH
            cx = x0[:, None] + (np.arange(PW)[None, :] + 0.5) * bw[:, None]      # [K, PW]
            cy = y0[:, None] + (np.arange(PH)[None, :] + 0.5) * bh[:, None]      # [K, PH]
            exp = (alpha[None, :, None, None] + beta[None, :, None, None] * cx[:, None, None, :]
                   + gamma[None, :, None, None] * cy[:, None, :, None])
            tol = _tol(mode, 1e-11, 2e-5)
            assert np.allclose(out, exp, rtol=tol, atol=tol), (S, aligned,
                                                                np.abs(out - exp).max())


def _adjoint_setup(rng):
    shapes = [(2, 3, 9, 11), (2, 3, 5, 6), (2, 3, 3, 3)]
    scales = [0.5, 0.25, 0.125]
    feats = [rng.normal(size=s) for s in shapes]
    K = 20
    rois = _rand_rois_anywhere(rng, K, 2, 22, 18)
    lv = rng.integers(0, 3, K).astype(np.int32)
    return shapes, scales, feats, rois, lv


def pin_adjoint(lib, mode):
    """<fwd(x), g> = sum_l <x_l, bwd(g)_l> (backward is the transpose of forward)."""
    rng = np.random.default_rng(13)
    shapes, scales, feats, rois, lv = _adjoint_setup(rng)
    for S, aligned, (PH, PW) in ((2, True, (3, 4)), (0, True, (2, 2)), (1, False, (4, 3)),
                                 (3, False, (2, 5))):
        g = rng.normal(size=(rois.shape[0], 3, PH, PW))
        out = oracle.roi_align_fwd(feats, scales, rois, lv, PH, PW, S, aligned, mode, lib=lib)
        grads = oracle.roi_align_bwd(g, shapes, scales, rois, lv, PH, PW, S, aligned, mode,
                                     lib=lib)
        lhs = float(np.sum(out * g))
        rhs = float(sum(np.sum(f * gr) for f, gr in zip(feats, grads)))
        assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs)), (S, aligned, lhs, rhs)
        assert abs(lhs) > 1e-3


def _tent_reference(feats, scales, rois, lv, PH, PW, S, aligned):
    """Bilinear sampling written as a tent-kernel sum over all pixels (float64)."""
    K = rois.shape[0]
    C = feats[0].shape[1]
    out = np.zeros((K, C, PH, PW))
    for k in range(K):
        l = int(lv[k])
        F = feats[l]
        N, _, H, W = F.shape
        t = float(np.trunc(rois[k, 0]))
        if not (0 <= t < N):
            continue
        b = int(t)
        s = scales[l]
        off = 0.5 if aligned else 0.0
        x0 = float(rois[k, 1]) * s - off
        y0 = float(rois[k, 2]) * s - off
        rw = float(rois[k, 3]) * s - off - x0
        rh = float(rois[k, 4]) * s - off - y0
        if not aligned:
            rw, rh = max(rw, 1.0), max(rh, 1.0)
        bw, bh = rw / PW, rh / PH
        gw = S if S > 0 else max(int(np.ceil(bw)), 0)
        gh = S if S > 0 else max(int(np.ceil(bh)), 0)
        count = max(gh * gw, 1)
        iy_pix = np.arange(H)[:, None]
        ix_pix = np.arange(W)[None, :]
        for ph in range(PH):
            for pw in range(PW):
                acc = np.zeros(C)
                for iy in range(gh):
                    y = y0 + ph * bh + (iy + 0.5) * bh / gh
                    for ix in range(gw):
                        x = x0 + pw * bw + (ix + 0.5) * bw / gw
                        if y < -1 or y > H or x < -1 or x > W:
                            continue
                        yc = min(max(y, 0.0), H - 1.0)
                        xc = min(max(x, 0.0), W - 1.0)
                        tent = (np.maximum(0.0, 1 - np.abs(yc - iy_pix))
                                * np.maximum(0.0, 1 - np.abs(xc - ix_pix)))
                        acc += np.tensordot(F[b], tent, axes=([1, 2], [0, 1]))
                out[k, :, ph, pw] = acc / count
    return out


def pin_tent(lib, mode):
    rng = np.random.default_rng(14)
    shapes = [(2, 2, 5, 6), (2, 2, 3, 4)]
    scales = [0.5, 0.25]
    feats = [rng.normal(size=s) for s in shapes]
    rois = _rand_rois_anywhere(rng, 6, 2, 12, 10)
    rois[0, 1:] = (-3.0, -3.0, 1.0, 1.0)      # mostly outside, low side
    rois[1, 1:] = (9.0, 7.0, 14.0, 13.0)      # past the high edges
    lv = rng.integers(0, 2, 6).astype(np.int32)
    for S, aligned, (PH, PW) in ((2, True, (2, 3)), (0, True, (2, 2)), (1, False, (3, 2)),
                                 (3, True, (1, 1))):
        out = oracle.roi_align_fwd(feats, scales, rois, lv, PH, PW, S, aligned, mode, lib=lib)
        ref = _tent_reference(feats, scales, rois, lv, PH, PW, S, aligned)
        tol = _tol(mode, 1e-12, 1e-4)
        assert np.allclose(out, ref, rtol=tol, atol=tol), (S, aligned, np.abs(out - ref).max())


def pin_dense_matrix(lib, mode):
    """Assemble A from fwd(e_j) and check bwd(g) == A^T g."""
    rng = np.random.default_rng(15)
    shapes = [(1, 1, 3, 4), (1, 1, 2, 2)]
    scales = [0.5, 0.25]
    rois = _rand_rois_anywhere(rng, 3, 1, 8, 6)
    lv = np.array([0, 1, 0], np.int32)
    PH, PW, S, aligned = 2, 2, 2, True
    cols = []
    for l, s in enumerate(shapes):
        for j in range(int(np.prod(s))):
            feats = [np.zeros(t) for t in shapes]
            feats[l].reshape(-1)[j] = 1.0
            cols.append(oracle.roi_align_fwd(feats, scales, rois, lv, PH, PW, S, aligned, mode,
                                             lib=lib).reshape(-1))
    A = np.stack(cols, axis=1)
    assert np.count_nonzero(A) > 10
    g = rng.normal(size=(3, 1, PH, PW))
    grads = oracle.roi_align_bwd(g, shapes, scales, rois, lv, PH, PW, S, aligned, mode, lib=lib)
    got = np.concatenate([x.reshape(-1) for x in grads])
    assert np.allclose(got, A.T @ g.reshape(-1), rtol=1e-13, atol=1e-13)


def pin_textbook(lib, mode):
    """Aligned box on the integer grid: 2x2 average pooling of the crop (sampling 2,
    box side 2P) and the exact crop (sampling 1, box side P)."""
    rng = np.random.default_rng(16)
    F = rng.normal(size=(1, 2, 12, 14))
    P = 4
    for oy, ox in ((0, 0), (2, 3), (4, 6)):
        rois = np.array([[0, ox, oy, ox + 2 * P, oy + 2 * P]], np.float32)
        out = oracle.roi_align_fwd([F], [1.0], rois, None, P, P, 2, True, mode, lib=lib)
        crop = F[0, :, oy:oy + 2 * P, ox:ox + 2 * P]
        pool = crop.reshape(2, P, 2, P, 2).mean(axis=(2, 4))
        assert np.allclose(out[0], pool, rtol=1e-13, atol=1e-13), (oy, ox)
        rois = np.array([[0, ox, oy, ox + P, oy + P]], np.float32)
        out = oracle.roi_align_fwd([F], [1.0], rois, None, P, P, 1, True, mode, lib=lib)
        assert np.array_equal(out[0], F[0, :, oy:oy + P, ox:ox + P]), (oy, ox)


def pin_mirror(lib, mode="math"):
    """Flip the map left-right and map the box x -> W_img - x: the output flips in pw."""
    rng = np.random.default_rng(17)
    F = rng.normal(size=(1, 2, 5, 7))
    scale = 0.5
    W_img = 7 / scale
    # coordinates on a 1/16 grid so that W_img - x is exact in binary32
    rois = np.round(_rand_rois_anywhere(rng, 8, 1, W_img, 10) * 16) / 16
    mir = rois.copy()
    mir[:, 1] = W_img - rois[:, 3]
    mir[:, 3] = W_img - rois[:, 1]
    for S in (2, 0):
        a = oracle.roi_align_fwd([F], [scale], rois, None, 3, 4, S, True, mode, lib=lib)
        b = oracle.roi_align_fwd([F[..., ::-1]], [scale], mir, None, 3, 4, S, True, mode,
                                 lib=lib)
        assert np.allclose(b, a[..., ::-1], rtol=1e-12, atol=1e-12), S


def pin_mass(lib, mode):
    """All samples valid: the backward conserves the total gradient."""
    rng = np.random.default_rng(18)
    shapes = [(2, 2, 16, 20), (2, 2, 8, 10)]
    scales = [0.25, 0.125]
    rois = _rand_rois_inside(rng, 12, 2, 80, 64, 2.0, 60.0)
    lv = rng.integers(0, 2, 12).astype(np.int32)
    g = rng.normal(size=(12, 2, 3, 3))
    grads = oracle.roi_align_bwd(g, shapes, scales, rois, lv, 3, 3, 2, True, mode, lib=lib)
    tot = sum(x.sum(axis=(0, 2, 3)) for x in grads)
    tol = _tol(mode, 1e-12, 1e-6)
    assert np.allclose(tot, g.sum(axis=(0, 2, 3)), rtol=tol, atol=tol)


def pin_guards(lib, mode):
    """A level index outside [0, L) or a batch index outside [0, N) gives zeros and no
    gradient."""
    rng = np.random.default_rng(19)
    shapes = [(1, 2, 6, 6)]
    feats = [rng.normal(size=shapes[0])]
    rois = np.array([[0, 1, 1, 9, 9], [0, 1, 1, 9, 9], [3, 1, 1, 9, 9]], np.float32)
    lv = np.array([0, 5, 0], np.int32)
    out = oracle.roi_align_fwd(feats, [0.5], rois, lv, 2, 2, 2, True, mode, lib=lib)
    assert np.abs(out[0]).sum() > 0
    assert not out[1].any() and not out[2].any()
    g = np.zeros((3, 2, 2, 2))
    g[1:] = 1.0
    grads = oracle.roi_align_bwd(g, shapes, [0.5], rois, lv, 2, 2, 2, True, mode, lib=lib)
    assert not grads[0].any()


ALL_PINS = [pin_hand_cases, pin_binary32_order, pin_level_cases, pin_level_log2_agrees, pin_level_plus1_is_shifted_box,
            pin_constant, pin_affine,
            pin_adjoint, pin_tent, pin_dense_matrix, pin_textbook, pin_mass, pin_guards]
MATH_ONLY_PINS = [pin_mirror]


def run_all(lib, modes=("math", "parity")):
    """Run every pin; returns the list of (pin name, mode, message) that failed."""
    failures = []
    for mode in modes:
        for pin in ALL_PINS + (MATH_ONLY_PINS if mode == "math" else []):
            try:
                pin(lib, mode)
            except AssertionError as e:
                failures.append((pin.__name__, mode, str(e)[:200]))
    return failures
