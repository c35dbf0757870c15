"""Planted mistakes: the pins must catch a plausible error anywhere in the oracle.

Each case copies the oracle source to a temporary directory, plants one mistake
(a dropped term, a wrong sign, a wrong index, a transposed operand, an
off-by-one), compiles the copy with the oracle's own flags, and requires at least
one pin in tests/oracle_pins.py to fail.  All planted mistakes keep every memory
access in bounds (indices stay clamped), so the broken copies are safe to run
in-process.  CPU only.
"""

import pytest

import oracle
import oracle_pins as P

MUTANTS = [
    ("sample offset (i+1 instead of i+1/2), binary32",
     "float c = (float)i + 0.5f;", "float c = (float)i + 1.0f;"),
    ("sample offset, double",
     "((double)i + 0.5) * g->bin_d", "((double)i + 1.0) * g->bin_d"),
    ("aligned shift sign",
     "const float off = aligned ? 0.5f : 0.0f;", "const float off = aligned ? -0.5f : 0.0f;"),
    ("aligned shift dropped, double",
     "const double off = aligned ? 0.5 : 0.0;", "const double off = 0.0;"),
    ("validity cut at 0 instead of -1",
     "if (v < -1.0f || v > (float)size)", "if (v < 0.0f || v > (float)size)"),
    ("validity cut, double, upper bound size-1",
     "if (v < -1.0 || v > (double)size)", "if (v < -1.0 || v > (double)(size - 1))"),
    ("divisor off by one",
     "o[(c * PH + ph) * PW + pw] = sum / (double)count;",
     "o[(c * PH + ph) * PW + pw] = sum / (double)(count + 1);"),
    ("bilinear weights swapped",
     "t.w_lo = (double)rest;\n        t.w_hi = (double)frac;",
     "t.w_lo = (double)frac;\n        t.w_hi = (double)rest;"),
    ("transposed corner in the forward",
     "sum += ty.w_lo * tx.w_hi * F[ty.lo * W + tx.hi];",
     "sum += ty.w_lo * tx.w_hi * F[ty.hi * W + tx.lo];"),
    ("corner term dropped in the forward",
     "sum += ty.w_hi * tx.w_hi * F[ty.hi * W + tx.hi];", ""),
    ("level threshold compared with >",
     "if (area >= thr)", "if (area > thr)"),
    ("inclusive pixel boxes: +1 dropped on one side",
     "            h = h + 1.0f;\n", ""),
    ("inclusive pixel boxes: +1 applied to the continuous rule too",
     "        if (box_plus1) {\n            w = w + 1.0f;", "        if (1) {\n            w = w + 1.0f;"),
    ("level thresholds from finest_scale*2^(j-1)",
     "float side = finest_scale * (float)(1 << j);",
     "float side = finest_scale * (float)(1 << (j - 1));"),
    ("backward weight uses the wrong corner",
     "G[ty.lo * W + tx.hi] += gv * ty.w_lo * tx.w_hi;",
     "G[ty.lo * W + tx.hi] += gv * ty.w_lo * tx.w_lo;"),
    ("backward divisor dropped",
     "double gv = g[ph * PW + pw] / (double)count;", "double gv = g[ph * PW + pw];"),
    ("bin position off by one",
     "float a = (float)p * g->bin_f;", "float a = (float)(p + 1) * g->bin_f;"),
    ("minimum box size dropped when not aligned",
     "len = fmaxf(len, 1.0f);", "len = fmaxf(len, 0.0f);"),
    ("x axis built from y coordinates",
     "axis_geom gx = axis_setup(mode, r[1], r[3], scales[lvl], aligned, PW, sampling_ratio);\n"
     "        axis_geom gy = axis_setup(mode, r[2], r[4], scales[lvl], aligned, PH, sampling_ratio);\n"
     "        int count = gy.grid * gx.grid;\n        if (count < 1)\n            count = 1;\n"
     "        for (int64_t c = 0; c < C; ++c) {",
     "axis_geom gx = axis_setup(mode, r[2], r[4], scales[lvl], aligned, PW, sampling_ratio);\n"
     "        axis_geom gy = axis_setup(mode, r[2], r[4], scales[lvl], aligned, PH, sampling_ratio);\n"
     "        int count = gy.grid * gx.grid;\n        if (count < 1)\n            count = 1;\n"
     "        for (int64_t c = 0; c < C; ++c) {"),
    ("batch index rounded instead of truncated",
     "float t = truncf(v);", "float t = roundf(v);"),
    ("adaptive grid uses floor",
     "double g = ceil(bin);", "double g = floor(bin);"),
    ("scale applied after the shift",
     "float s = c1 * scale;\n        s = s - off;", "float s = c1 - off;\n        s = s * scale;"),
    ("bin start and within-bin offset summed first, binary32",
     "float b = g->start_f + a;\n        float c = (float)i + 0.5f;\n"
     "        float d = c * g->bin_f;\n        float e = d / (float)g->grid;\n"
     "        float v = b + e;",
     "float b = a;\n        float c = (float)i + 0.5f;\n"
     "        float d = c * g->bin_f;\n        float e = d / (float)g->grid;\n"
     "        float v = g->start_f + (b + e);"),
    ("within-bin offset as (i + 1/2) * (bin / grid), binary32",
     "float d = c * g->bin_f;\n        float e = d / (float)g->grid;",
     "float d = g->bin_f / (float)g->grid;\n        float e = c * d;"),
    ("bin size by the reciprocal of the bin count, binary32",
     "float bin = len / (float)P;\n        g.len_f = len;",
     "float bin = len * (1.0f / (float)P);\n        g.len_f = len;"),
    ("adaptive grid cap raised", "#define ADAPTIVE_GRID_CAP 64", "#define ADAPTIVE_GRID_CAP 128"),
    ("adaptive grid uncapped",
     "    if (g > (double)ADAPTIVE_GRID_CAP)\n        g = (double)ADAPTIVE_GRID_CAP;\n", ""),
]


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_is_caught(tmp_path, name, old, new):
    src = open(oracle.SOURCE).read()
    assert src.count(old) == 1, "planted-mistake pattern no longer matches the oracle: " + name
    path = tmp_path / "mutant.c"
    path.write_text(src.replace(old, new))
    lib_path = str(tmp_path / "libmutant.so")
    oracle.build(str(path), lib_path)
    lib = oracle.load(lib_path)
    failures = P.run_all(lib)
    assert failures, "no pin caught: " + name


def test_unmodified_copy_passes_every_pin(tmp_path):
    """The same harness on an unmodified copy finds nothing (so a failure above is the
    planted mistake's doing)."""
    lib_path = str(tmp_path / "libcopy.so")
    oracle.build(oracle.SOURCE, lib_path)
    assert P.run_all(oracle.load(lib_path)) == []
