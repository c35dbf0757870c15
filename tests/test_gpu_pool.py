"""GPU parity of RoI max pooling (roi_pool_fwd / roi_pool_bwd through the C ABI)
against the CPU oracle.

The forward value is one of the input values, so it is compared bit for bit (after
rounding the oracle's value to the output dtype), and the argmax is compared exactly.
The backward sums in an order of its own (LDS atomics in the tile gather, which runs
whenever the plan holds tile lists and the grid is 7x7; device atomics otherwise), so it
is compared with the backward tolerance: |gpu - ref| <= 1e-4 * S elementwise, S = the
oracle's backward of |g|.
"""
import numpy as np
import pytest

import oracle
import paper_1906_07155_amd as rex
from paper_1906_07155_amd import workloads as W
from gpu_helpers import as_f64, check_bwd, from_device, log, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    rex.lib()


def _expected_bits(ref: np.ndarray, odt: str) -> np.ndarray:
    """Oracle values in the output dtype: binary32 as is, bf16 rounded to nearest even
    (the -FLT_MAX sentinel of an all-NaN bin is not produced by these cases)."""
    f = ref.astype(np.float32)
    return W.f32_to_bf16_bits(f) if odt == "bf16" else f.view(np.uint32)


def _got_bits(t, odt: str) -> np.ndarray:
    if odt == "bf16":
        return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    return t.contiguous().cpu().numpy().view(np.uint32)


def run(name, feats_np, scales, rois, out_hw=(7, 7), fdt="f32", odt="f32", gdt="f32",
        layout="cl", use_plan=True, zero_init=True, roi_levels=None, seed=0, backward=True):
    shapes = [f.shape for f in feats_np]
    log("pool case %s: shapes=%s K=%d out=%s %s->%s grad %s layout=%s plan=%d" % (
        name, shapes, rois.shape[0], out_hw, fdt, odt, gdt, layout, use_plan))
    rng = np.random.default_rng(seed)
    feats = [to_device(f, fdt, layout) for f in feats_np]
    if layout == "nchw_view":
        feats = [to_device(np.pad(f, ((0, 0), (1, 2), (0, 1), (2, 0))), fdt, "nchw")[
            :, 1:1 + f.shape[1], :f.shape[2], 2:] for f in feats_np]
    K, L = rois.shape[0], len(shapes)
    C = shapes[0][1]
    r_dev = torch.from_numpy(rois).cuda()
    if roi_levels is None:
        lv_dev, ws = rex.plan(feats, scales, r_dev, 56.0)
        lv = oracle.level_map(rois, L, 56.0)
        if not use_plan:
            ws = None
    else:
        lv = np.asarray(roi_levels, np.int32)
        lv_dev, ws = torch.from_numpy(lv).cuda(), None
    out, am = rex.roi_pool_fwd(feats, scales, r_dev, lv_dev, out_hw,
                               out_dtype=torch.bfloat16 if odt == "bf16" else torch.float32,
                               workspace=ws)
    torch.cuda.synchronize()
    f64 = [as_f64(f, fdt) for f in feats_np]
    ref, am_ref = oracle.roi_pool_fwd(f64, scales, rois, lv, out_hw[0], out_hw[1])
    got_am = am.cpu().numpy()
    bad = got_am != am_ref
    assert not bad.any(), "%s argmax: %d differ, first at %s (gpu %d, oracle %d)" % (
        name, int(bad.sum()), np.argwhere(bad)[0], got_am[bad][0], am_ref[bad][0])
    gb, eb = _got_bits(out, odt), _expected_bits(ref, odt)
    bad = gb != eb
    assert not bad.any(), "%s values: %d differ, first at %s" % (name, int(bad.sum()),
                                                                 np.argwhere(bad)[0])
    if not backward:
        return out, am
    g = rng.standard_normal((K, C) + tuple(out_hw), dtype=np.float32)
    if gdt == "bf16":
        g = W.f32_to_bf16_bits(g)
    g64 = as_f64(g, gdt)
    gref = oracle.roi_pool_bwd(g64, am_ref, shapes, rois, lv)
    aref = oracle.roi_pool_bwd(np.abs(g64), am_ref, shapes, rois, lv)
    grads = [torch.full(s, 5.0, dtype=torch.float32, device="cuda") for s in shapes]
    if layout == "cl":
        grads = [x.contiguous(memory_format=torch.channels_last) for x in grads]
    rex.roi_pool_bwd(to_device(g, gdt, "nchw"), am, r_dev, lv_dev, grads, scales,
                     zero_init=zero_init, workspace=ws)
    torch.cuda.synchronize()
    base = 0.0 if zero_init else 5.0
    for l in range(L):
        scale = aref[l] + base * 2.0 ** -20 / 1e-4
        check_bwd(from_device(grads[l]) - base, gref[l], scale, False,
                  "%s backward level %d" % (name, l))
    return out, am


PYR = [(2, 24, 40), (2, 12, 20), (2, 6, 10), (2, 3, 5)]
SC = [0.25, 0.125, 0.0625, 0.03125]


def _pyr(rng, C, fdt="f32"):
    out = []
    for (n, h, w) in PYR:
        x = rng.standard_normal((n, C, h, w), dtype=np.float32)
        out.append(W.f32_to_bf16_bits(x) if fdt == "bf16" else x)
    return out


def _rois(rng, K, outside=0.2, img=(96, 160)):
    H, Wd = img
    a = rng.uniform(-outside * Wd, (1 + outside) * Wd, (K, 2))
    b = rng.uniform(-outside * H, (1 + outside) * H, (K, 2))
    r = np.zeros((K, 5), np.float32)
    r[:, 0] = rng.integers(0, 2, K)
    r[:, 1], r[:, 3] = a.min(1), a.max(1)
    r[:, 2], r[:, 4] = b.min(1), b.max(1)
    return r


@pytest.mark.parametrize("C", [1, 3, 100, 256, 320])
def test_pool_channels_ragged(C):
    rng = np.random.default_rng(100 + C)
    run("C=%d" % C, _pyr(rng, C), SC, W.draw_rois(rng, 2, 23, (96, 160), (4.0, 200.0)))


@pytest.mark.parametrize("layout", ["nchw", "nchw_view"])
def test_pool_layouts(layout):
    rng = np.random.default_rng(110)
    run("layout %s" % layout, _pyr(rng, 70), SC, _rois(rng, 31), layout=layout)


@pytest.mark.parametrize("fdt,odt,gdt", [("bf16", "bf16", "bf16"), ("bf16", "f32", "f32"),
                                         ("f32", "bf16", "bf16")])
def test_pool_dtypes(fdt, odt, gdt):
    rng = np.random.default_rng(120)
    run("dtypes %s/%s/%s" % (fdt, odt, gdt), _pyr(rng, 130, fdt), SC,
        W.draw_rois(rng, 2, 21, (96, 160), (4.0, 200.0)), fdt=fdt, odt=odt, gdt=gdt)


def test_pool_output_sizes_and_generic_path():
    rng = np.random.default_rng(130)
    f = _pyr(rng, 40)
    r = _rois(rng, 19)
    run("out 14x14 (general kernel)", f, SC, r, out_hw=(14, 14))
    run("out 5x3", f, SC, r, out_hw=(5, 3))
    run("out 8x12 (96 bins, the largest channels-last grid)", f, SC, r, out_hw=(8, 12))
    run("out 4x24", f, SC, r, out_hw=(4, 24))
    run("out 1x1", f, SC, r, out_hw=(1, 1))
    run("out 7x7 without plan", f, SC, r, use_plan=False)


def test_pool_accumulates_and_duplicates():
    rng = np.random.default_rng(140)
    base = np.array([0, 20.0, 12.0, 60.0, 44.0], np.float32)
    rois = np.tile(base, (60, 1))
    rois[:, 1:] += rng.uniform(-2, 2, (60, 4)).astype(np.float32)
    rois[:, 0] = rng.integers(0, 2, 60)
    run("60 stacked RoIs", _pyr(rng, 64), SC, rois, zero_init=False)


def test_pool_ties_and_degenerate_boxes():
    """Constant maps (every bin ties: the first pixel of the bin wins), boxes smaller
    than the grid, inverted and out-of-map boxes, invalid batch and level indices."""
    rng = np.random.default_rng(150)
    feats = [np.full((2, 33, h, w), 1.5, np.float32) for (_, h, w) in PYR]
    rois = np.array([[0, 10.0, 10.0, 10.0, 10.0],      # one pixel, every bin the same
                     [1, 30.0, 20.0, 33.0, 22.0],      # smaller than 7x7 bins
                     [0, 50.0, 40.0, 20.0, 10.0],      # inverted
                     [1, -90.0, -90.0, -40.0, -40.0],  # outside the map
                     [0, 150.0, 80.0, 400.0, 300.0],   # past the far edges
                     [2, 10.0, 10.0, 60.0, 60.0],      # batch index outside
                     [-1, 10.0, 10.0, 60.0, 60.0]], np.float32)
    run("ties/degenerate", feats, SC, rois, roi_levels=[0, 1, 0, 2, 3, 0, 1])
    run("invalid level", _pyr(rng, 33), SC, rois[:2], roi_levels=[4, -1])


def test_pool_non_finite_features():
    rng = np.random.default_rng(160)
    feats = _pyr(rng, 64)
    feats[0][0, :, 3:9, 5:15] = np.nan
    feats[0][1, 3, :, :] = -np.inf
    feats[1][0, 7, 2, 2] = np.inf
    rois = W.draw_rois(rng, 2, 25, (96, 160), (4.0, 120.0))
    run("non-finite", feats, SC, rois)


def test_pool_full_box_head_workload():
    """The FPN box head workload (batch 2, P2-P5 with 256 channels, 1024 RoIs, 7x7)
    in the launch configuration a caller uses: plan, channels-last, forward + backward."""
    wl = W.config(2)
    feats = wl.features()
    rois = wl.rois()
    run("box head workload", feats, list(wl.scales), rois, seed=2)


def test_pool_gather_long_lists_and_five_kernel_plan():
    """The tile gather on many long tile lists (40 hot spots of 40 RoIs, accumulating too)
    and on a plan of more than 8192 RoIs (five kernels)."""
    rng = np.random.default_rng(170)
    shapes = [(1, 64, 128, 128), (1, 64, 64, 64), (1, 64, 32, 32), (1, 64, 16, 16)]
    feats = [rng.standard_normal(s, dtype=np.float32) for s in shapes]
    centres = rng.uniform(40, 472, (40, 2))
    rows = []
    for cx, cy in centres:
        half = rng.uniform(8, 24, (40, 2))
        jit = rng.uniform(-6, 6, (40, 2))
        x1 = np.clip(cx + jit[:, 0] - half[:, 0], 0, 512)
        x2 = np.clip(cx + jit[:, 0] + half[:, 0], 0, 512)
        y1 = np.clip(cy + jit[:, 1] - half[:, 1], 0, 512)
        y2 = np.clip(cy + jit[:, 1] + half[:, 1], 0, 512)
        rows.append(np.stack([np.zeros(40), x1, y1, x2, y2], 1))
    rois = np.concatenate(rows).astype(np.float32)
    run("40 hot spots", feats, SC, rois)
    run("40 hot spots accumulate", feats, SC, rois, zero_init=False)
    run("9400 RoIs (five-kernel plan)", _pyr(rng, 16), SC,
        W.draw_rois(rng, 2, 4700, (96, 160), (4.0, 200.0)))


def test_pool_gather_wide_tiles():
    """One 2048 x 2048 map: the tile layout takes 32-pixel tiles and a gather workgroup
    owns an 8 x 32 band of a tile."""
    rng = np.random.default_rng(171)
    feats = [rng.standard_normal((1, 8, 2048, 2048), dtype=np.float32)]
    rois = _rois(rng, 48, outside=0.05, img=(8192, 8192))
    rois[:, 0] = 0
    run("2048 x 2048 map", feats, [0.25], rois)


def test_pool_map_of_2_24_pixels():
    """A 4096 x 4096 map: pixel indices no longer fit the 24 bits of the channels-last
    forward's pixel sequence, so the forward takes the general kernel; the backward's
    tile layout widens the tiles to 64 pixels (a gather workgroup owns an 8 x 32 band of
    a tile, 16 workgroups per tile)."""
    rng = np.random.default_rng(172)
    feats = [rng.standard_normal((1, 4, 4096, 4096), dtype=np.float32)]
    rois = _rois(rng, 24, outside=0.05, img=(4096, 4096))
    rois[:, 0] = 0
    run("4096 x 4096 map", feats, [1.0], rois)
