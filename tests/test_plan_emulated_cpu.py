"""The plan kernels run on the CPU (``emulate/emu_main.cpp``: their own source, one
fiber per work-item, AddressSanitizer and UndefinedBehaviorSanitizer, LDS filled with
garbage at every workgroup's start), on the edge cases of the plan and on four
full-size workloads, through both launch paths (one launch, and the five-kernel
path).

Every output is checked against what it must be, computed here without the library:
levels against the oracle's level map; the permutation is one, ordered by (level,
image); offsets are the level counts' prefix sums; tile lists are disjoint ranges of
distinct RoIs of the tile's own level and image; every RoI is listed at every tile
that one of its bilinear taps (7x7 and 14x14 grids, sampling ratio 2, either
alignment) falls in; tiles are ordered longest list first.
"""
import os
import shutil
import struct
import subprocess
import sys

import numpy as np
import pytest

import oracle
from paper_1906_07155_amd import workloads as W

HERE = os.path.dirname(os.path.abspath(__file__))


def _builder():
    if shutil.which("g++") is None:
        pytest.skip("g++ not available")
    sys.path.insert(0, os.path.join(HERE, "emulate"))
    import emu_build
    return emu_build


@pytest.fixture(scope="module")
def emu(tmp_path_factory):
    return _builder().build(str(tmp_path_factory.mktemp("emu")))


def run(emu, tmp, level_hw, scales, N, rois, fs=56.0, conv=0, multi=False):
    K, L = len(rois), len(level_hw)
    inp, out = str(tmp / "in.bin"), str(tmp / "out.bin")
    with open(inp, "wb") as f:
        f.write(struct.pack("iii", L, N, 8))
        for (h, w), s in zip(level_hw, scales):
            f.write(struct.pack("iif", h, w, s))
        f.write(struct.pack("fii", fs, K, conv))
        f.write(np.ascontiguousarray(rois, np.float32).tobytes())
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    env.pop("LD_PRELOAD", None)
    r = subprocess.run([emu, inp, out] + (["multi"] if multi else []), capture_output=True,
                       text=True, timeout=600, env=env)
    assert r.returncode == 0 and "done" in r.stdout, (r.stdout + r.stderr)[-4000:]
    d = np.fromfile(out, np.int32)
    ntiles, cap, K2, L2, shift = d[:5]
    o = 5
    ntx, nty, tbase = d[o:o + 8], d[o + 8:o + 16], d[o + 16:o + 25]
    o += 25
    take = {}
    for name, n in (("lv", K), ("offs", L + 1), ("keys", K), ("perm", K), ("ts", ntiles),
                    ("te", ntiles), ("order", ntiles), ("tr", cap)):
        take[name] = d[o:o + n]
        o += n
    assert (K2, L2) == (K, L) and o == len(d)
    check(take, rois, level_hw, scales, N, fs, conv, ntiles, cap, shift, ntx, nty, tbase)
    return take


def taps(lo, size, n, extent, aligned):
    """Feature pixels read by the bilinear taps of n x 2 samples along one axis (binary32
    geometry as in RoIAlign: start, bin size, sample centres; taps outside [-1, extent]
    read nothing)."""
    f32 = np.float32
    off = f32(0.5) if aligned else f32(0.0)
    start = f32(lo) - off
    if not aligned:
        size = max(f32(size), f32(1.0))
    b = f32(size) / f32(n)
    i = np.arange(2 * n, dtype=f32)
    x = start + (np.floor(i / 2) * b + (i % 2 + f32(0.5)) * b / f32(2)).astype(f32)
    x = x[(x >= -1) & (x <= extent)]
    x = np.maximum(x, 0)
    x0 = np.floor(x).astype(np.int64)
    hi = x0 >= extent - 1
    x0 = np.minimum(x0, extent - 1)
    x1 = np.where(hi, x0, x0 + 1)
    return np.unique(np.concatenate([x0, x1]))


def check(t, rois, level_hw, scales, N, fs, conv, ntiles, cap, shift, ntx, nty, tbase):
    K, L = len(rois), len(level_hw)
    ref = oracle.level_map(rois, L, fs, box_plus1=bool(conv)) if L > 1 else np.zeros(K, np.int32)
    assert np.array_equal(t["lv"], ref), "levels"
    perm = t["perm"]
    assert np.array_equal(np.sort(perm), np.arange(K)), "permutation"
    assert np.array_equal(t["offs"], np.concatenate([[0], np.cumsum(np.bincount(ref, minlength=L))]))
    assert np.all(np.diff(t["keys"][perm]) >= 0), "keys out of order"
    assert np.all(np.diff(ref[perm]) >= 0), "levels out of order"
    img = np.trunc(rois[:, 0]).astype(np.int64)
    for l in range(L):
        seg = img[perm[t["offs"][l]:t["offs"][l + 1]]]
        seg = seg[(seg >= 0) & (seg < N)]          # RoIs of no image are keyed as image 0
        assert np.all(np.diff(seg) >= 0), "images not grouped on level %d" % l
    if ntiles == 0:
        return
    ts, te, tr, order = t["ts"], t["te"], t["tr"], t["order"]
    lens = te - ts
    assert (lens >= 0).all() and (ts >= 0).all() and (te <= cap).all(), "tile ranges"
    o = np.argsort(ts, kind="stable")
    assert (ts[o][1:] >= te[o][:-1]).all(), "tile lists overlap"
    assert np.array_equal(np.sort(order), np.arange(ntiles)), "order is not a permutation"
    assert (np.diff(lens[order]) <= 0).all() or (np.diff(np.minimum(lens[order], 255)) <= 0).all()
    members = [set(tr[ts[i]:te[i]].tolist()) for i in range(ntiles)]
    for i in range(ntiles):
        assert len(members[i]) == lens[i], "tile %d lists a RoI twice" % i
    for k in range(K):
        b, l = img[k], ref[k]
        if not (0 <= b < N) or not np.all(np.isfinite(rois[k, 1:])):
            continue
        H, Wd = level_hw[l]
        s = np.float32(scales[l])
        x1, y1, x2, y2 = (np.float32(v) for v in rois[k, 1:])
        for n in (7, 14):
            for aligned in (0, 1):
                xs = taps(x1 * s, x2 * s - x1 * s, n, Wd, aligned)
                ys = taps(y1 * s, y2 * s - y1 * s, n, H, aligned)
                for ty in np.unique(ys >> shift):
                    for tx in np.unique(xs >> shift):
                        tile = tbase[l] + (b * nty[l] + ty) * ntx[l] + tx
                        assert k in members[tile], (
                            "RoI %d missing from tile %d (level %d image %d)" % (k, tile, l, b))
    # entries belong to the tile's own level and image
    for l in range(L):
        for b in range(N):
            first = tbase[l] + b * nty[l] * ntx[l]
            for i in range(first, first + nty[l] * ntx[l]):
                for k in members[i]:
                    assert ref[k] == l and img[k] == b, "RoI %d in a tile of level %d image %d" % (k, l, b)


PYR = [(24, 40), (12, 20), (6, 10), (3, 5)]
SC = [0.25, 0.125, 0.0625, 0.03125]


def edge_rois():
    rng = np.random.default_rng(0)
    r = W.draw_rois(rng, 3, 40, (96, 160), (4.0, 200.0))
    r[::7, 0] = -1                        # no image
    r[::11, 0] = 7                        # image beyond the batch
    r[5, 1:] = np.nan
    r[9, 1:] = [1e30, -1e30, 5, 5]
    r[13, 1:] = [50, 40, 20, 10]          # x2 < x1, y2 < y1
    r[17, 1:] = [-30, -30, -10, -10]      # off the map
    r[19, 1:] = [159, 95, 159, 95]        # a point at the far corner
    return r


@pytest.mark.parametrize("multi", [False, True])
@pytest.mark.parametrize("case", ["edges", "one", "65", "dense", "identical"])
def test_plan_edges(emu, tmp_path, case, multi):
    rng = np.random.default_rng(1)
    if case == "edges":
        rois, N = edge_rois(), 3
    elif case == "one":
        rois, N = edge_rois()[:1], 3
    elif case == "65":
        rois, N = edge_rois()[:65], 3
    elif case == "dense":
        rois, N = W.draw_rois(rng, 2, 1100, (96, 160), (4.0, 200.0)), 2
    else:
        rois, N = np.tile(np.array([[0, 10, 10, 60, 50]], np.float32), (3000, 1)), 1
    run(emu, tmp_path, PYR, SC, N, rois, multi=multi)
    if case == "edges":
        run(emu, tmp_path, PYR, SC, N, rois, conv=1, multi=multi)


def test_plan_single_level_and_many_rois(emu, tmp_path):
    rng = np.random.default_rng(2)
    run(emu, tmp_path, [(50, 68)], [1.0 / 16], 1, W.draw_rois(rng, 1, 128, (800, 1088), (16.0, 512.0)))
    run(emu, tmp_path, PYR, SC, 2, W.draw_rois(rng, 2, 4600, (96, 160), (4.0, 200.0)))


@pytest.mark.parametrize("idx,head", [(2, None), (3, None), (5, "box"), (5, "mask")])
def test_plan_full_workload(emu, tmp_path, idx, head):
    wl = W.config(idx, head=head)
    run(emu, tmp_path, wl.level_hw, wl.scales, wl.n_images, wl.rois(), wl.finest_scale)


def test_emulator_catches_a_missing_barrier(tmp_path):
    """The fault class the emulator exists for: with the barrier between filling the
    level table in LDS and reading it taken out of the band role, the garbage that LDS
    starts with must end the run (an access outside an array) or fail a check."""
    mark = "__syncthreads();   // the level table is read only after this barrier"
    emu = _builder().build(str(tmp_path), edit=lambda s: s.replace(mark, "", 1))
    rois = W.draw_rois(np.random.default_rng(1), 2, 1100, (96, 160), (4.0, 200.0))
    with pytest.raises(AssertionError):
        run(emu, tmp_path, PYR, SC, 2, rois)
