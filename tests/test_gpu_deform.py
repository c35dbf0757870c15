"""GPU parity of deformable (modulated) RoI pooling (deform_roi_pool_fwd / _bwd through
the C ABI) against the CPU oracle.

  forward            fp32: |gpu - ref| <= 1e-6 + 1e-5 |ref|;  bf16: 1e-4 + 1e-2 |ref|
  feature gradient   |gpu - ref| <= 1e-4 * S, S = the oracle's backward of |g| with |mask|
  offset, mask grads |gpu - ref| <= 1e-4 * (sum of the absolute values of the terms, from
                     the oracle) + 1e-7: fp32 sums over channels and samples
"""
import numpy as np
import pytest

import oracle
import paper_1906_07155_amd as rex
from paper_1906_07155_amd import workloads as W
from gpu_helpers import as_f64, check_bwd, check_fwd, from_device, log, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    rex.lib()


def run(name, feats_np, scales, rois, out_hw=(7, 7), S=2, aligned=True, fdt="f32", odt="f32",
        gdt="f32", layout="cl", offset_std=0.3, with_mask=True, gamma=0.1, roi_levels=None,
        zero_init=True, seed=0, nan_bin=False, use_plan=True):
    shapes = [f.shape for f in feats_np]
    log("deform case %s: shapes=%s K=%d out=%s S=%d aligned=%d %s->%s grad %s layout=%s "
        "mask=%d" % (name, shapes, rois.shape[0], out_hw, S, aligned, fdt, odt, gdt, layout,
                     with_mask))
    rng = np.random.default_rng(seed)
    K, L = rois.shape[0], len(shapes)
    C = shapes[0][1]
    PH, PW = out_hw
    off = (rng.standard_normal((K, 2, PH, PW)) * offset_std).astype(np.float32)
    if nan_bin:
        off[0, 0, 0, 0] = np.nan
    m = rng.uniform(0.0, 1.0, (K, PH, PW)).astype(np.float32) if with_mask else None
    feats = [to_device(f, fdt, "cl" if layout == "cl" else "nchw") for f in feats_np]
    r_dev = torch.from_numpy(rois).cuda()
    if roi_levels is None:
        lv_dev, ws = rex.plan(feats, scales, r_dev, 56.0)
        lv = oracle.level_map(rois, L, 56.0)
        if not use_plan:
            ws = None
    else:
        lv = np.asarray(roi_levels, np.int32)
        lv_dev, ws = torch.from_numpy(lv).cuda(), None
    off_dev = torch.from_numpy(off).cuda()
    m_dev = torch.from_numpy(m).cuda() if m is not None else None
    out = rex.deform_roi_pool_fwd(feats, scales, r_dev, lv_dev, out_hw, off_dev, m_dev, gamma, S,
                                  aligned, out_dtype=torch.bfloat16 if odt == "bf16" else
                                  torch.float32, workspace=ws)
    torch.cuda.synchronize()
    f64 = [as_f64(f, fdt) for f in feats_np]
    ref = oracle.deform_roi_pool_fwd(f64, scales, rois, lv, PH, PW, S, aligned, off, m, gamma)
    check_fwd(from_device(out), ref, fdt == "bf16" or odt == "bf16", name + " forward")

    g = rng.standard_normal((K, C, PH, PW), dtype=np.float32)
    if gdt == "bf16":
        g = W.f32_to_bf16_bits(g)
    g64 = as_f64(g, gdt)
    gf, goff, gm, soff, sm = oracle.deform_roi_pool_bwd(g64, f64, scales, rois, lv, PH, PW, S,
                                                        aligned, off, m, gamma)
    af, _, _, _, _ = oracle.deform_roi_pool_bwd(np.abs(g64), f64, scales, rois, lv, PH, PW, S,
                                                aligned, off, None if m is None else np.abs(m),
                                                gamma)
    grads = [torch.full(s, 7.0, dtype=torch.float32, device="cuda") for s in shapes]
    if layout == "cl":
        grads = [x.contiguous(memory_format=torch.channels_last) for x in grads]
    _, goff_dev, gm_dev = rex.deform_roi_pool_bwd(to_device(g, gdt, "nchw"), feats, r_dev, lv_dev,
                                                  off_dev, m_dev, grads, scales, gamma, S,
                                                  aligned, zero_init=zero_init, workspace=ws)
    torch.cuda.synchronize()
    base = 0.0 if zero_init else 7.0
    for l in range(L):
        check_bwd(from_device(grads[l]) - base, gf[l], af[l] + base * 2.0 ** -20 / 1e-4, False,
                  "%s feature gradient level %d" % (name, l))
    tol = 1e-2 if fdt == "bf16" else 1e-4
    got = goff_dev.cpu().numpy().astype(np.float64)
    bad = np.abs(got - goff) > tol * soff + 1e-7
    assert not bad.any(), "%s offset gradient: %d of %d out of tolerance, first at %s" % (
        name, int(bad.sum()), bad.size, np.argwhere(bad)[0])
    if m is not None:
        got = gm_dev.cpu().numpy().astype(np.float64)
        bad = np.abs(got - gm) > tol * sm + 1e-7
        assert not bad.any(), "%s mask gradient: %d out of tolerance" % (name, int(bad.sum()))
    return out


PYR = [(2, 24, 40), (2, 12, 20), (2, 6, 10), (2, 3, 5)]
SC = [0.25, 0.125, 0.0625, 0.03125]


def _pyr(rng, C, fdt="f32"):
    out = []
    for (n, h, w) in PYR:
        x = rng.standard_normal((n, C, h, w), dtype=np.float32)
        out.append(W.f32_to_bf16_bits(x) if fdt == "bf16" else x)
    return out


@pytest.mark.parametrize("C", [1, 3, 100, 256])
def test_deform_channels_ragged(C):
    rng = np.random.default_rng(200 + C)
    run("C=%d" % C, _pyr(rng, C), SC, W.draw_rois(rng, 2, 17, (96, 160), (4.0, 200.0)))


@pytest.mark.parametrize("S,aligned", [(0, True), (1, False), (3, True), (4, False)])
def test_deform_sampling_and_alignment(S, aligned):
    rng = np.random.default_rng(210 + S)
    run("S=%d aligned=%d" % (S, aligned), _pyr(rng, 40), SC,
        W.draw_rois(rng, 2, 13, (96, 160), (4.0, 200.0)), S=S, aligned=aligned)


@pytest.mark.parametrize("fdt,odt,gdt", [("bf16", "bf16", "bf16"), ("f32", "bf16", "bf16")])
def test_deform_dtypes(fdt, odt, gdt):
    rng = np.random.default_rng(220)
    run("dtypes %s/%s/%s" % (fdt, odt, gdt), _pyr(rng, 70, fdt), SC,
        W.draw_rois(rng, 2, 15, (96, 160), (4.0, 200.0)), fdt=fdt, odt=odt, gdt=gdt)


def test_deform_layouts_grids_and_no_mask():
    rng = np.random.default_rng(230)
    f = _pyr(rng, 33)
    r = W.draw_rois(rng, 2, 11, (96, 160), (4.0, 200.0))
    run("NCHW levels (general kernels)", f, SC, r, layout="nchw")
    run("14x14", f, SC, r, out_hw=(14, 14))
    run("14x14 S=4 (784 samples per wave: 13 located chunks)", f, SC, r, out_hw=(14, 14), S=4)
    run("16x16 (general kernels)", f, SC, r, out_hw=(16, 16))
    run("5x3 without mask", f, SC, r, out_hw=(5, 3), with_mask=False)
    run("without plan, accumulate", f, SC, r, use_plan=False, zero_init=False)
    run("with plan (tile gather), accumulate", f, SC, r, zero_init=False)
    run("with plan (tile gather), S=1, large offsets", f, SC, r, S=1, offset_std=3.0)


def test_deform_large_offsets_and_degenerate_inputs():
    """Offsets that push samples past the map edges (cut and clamp, zero slopes), a bin
    with a NaN offset (its samples are invalid), invalid batch and level indices."""
    rng = np.random.default_rng(240)
    f = _pyr(rng, 24)
    r = W.draw_rois(rng, 2, 13, (96, 160), (4.0, 200.0))
    run("large offsets", f, SC, r, offset_std=3.0, nan_bin=True)
    rois = np.array([[0, 10, 10, 60, 50], [2, 10, 10, 60, 50], [-1, 5, 5, 30, 30],
                     [1, 40, 30, 41, 31]], np.float32)
    run("invalid indices", f, SC, rois, roi_levels=[0, 0, 1, 5])


def test_deform_wide_bins():
    """RoIs spanning most of the finest map: bins wider than 4 pixels put a bin's two
    samples more than 2 pixels apart along x, so their taps do not fit one 4-pixel
    window (per-sample atomics); along y they do."""
    rng = np.random.default_rng(250)
    f = _pyr(rng, 24)
    rois = np.array([[0, 0, 0, 150, 90], [1, 10, 5, 140, 95], [0, 30, 20, 100, 80],
                     [1, 0, 0, 20, 20]], np.float32)
    run("wide bins", f, SC, rois, roi_levels=[0, 0, 0, 0])
    run("wide bins S=1", f, SC, rois, roi_levels=[0, 0, 0, 0], S=1)
    run("wide bins 14x14", f, SC, rois, roi_levels=[0, 0, 0, 0], out_hw=(14, 14))


def test_deform_full_box_head_workload():
    """The FPN box head workload (batch 2, P2-P5 with 256 channels, 1024 RoIs, 7x7) with
    offsets ~ N(0, 0.3^2) and modulation ~ U(0, 1)."""
    wl = W.config(2)
    run("box head workload", wl.features(), list(wl.scales), wl.rois(), seed=5)


def test_deform_gather_wide_tiles_and_five_kernel_plan():
    """The feature-gradient gather on a map with 32-pixel tiles (one 2048 x 2048 image:
    a workgroup owns an 8 x 32 band of a tile) and on a plan of more than 8192 RoIs
    (five kernels)."""
    rng = np.random.default_rng(260)
    feats = [rng.standard_normal((1, 8, 2048, 2048), dtype=np.float32)]
    a = rng.uniform(0, 8192, (40, 2))
    b = rng.uniform(0, 8192, (40, 2))
    rois = np.zeros((40, 5), np.float32)
    rois[:, 1], rois[:, 3] = a.min(1), a.max(1)
    rois[:, 2], rois[:, 4] = b.min(1), b.max(1)
    run("2048 x 2048 map, 32-pixel tiles", feats, [0.25], rois)
    run("9400 RoIs (five-kernel plan)", _pyr(rng, 16), SC,
        W.draw_rois(rng, 2, 4700, (96, 160), (4.0, 200.0)))
