"""The oracle's deformable (modulated) RoI pooling against its pins, and planted
mistakes the pins must catch (CPU only; every planted mistake keeps memory accesses in
bounds: indices stay clamped)."""
import pytest

import oracle
import oracle_deform_pins as P


@pytest.fixture(scope="module")
def lib():
    return oracle.load()


@pytest.mark.parametrize("mode", ["math", "parity"])
@pytest.mark.parametrize("pin", P.ALL_DEFORM_PINS + P.AFFINE_PINS, ids=lambda f: f.__name__)
def test_deform_pin(lib, pin, mode):
    pin(lib, mode)


@pytest.mark.parametrize("pin", P.MATH_ONLY_DEFORM_PINS, ids=lambda f: f.__name__)
def test_deform_pin_math_only(lib, pin):
    pin(lib, "math")


MUTANTS = [
    ("shift subtracted, binary32", "float b2 = b + shift_f;", "float b2 = b - shift_f;"),
    ("shift subtracted, double", "g->bin_d + shift_d + within;", "g->bin_d - shift_d + within;"),
    ("shift scaled by the bin instead of the box, binary32",
     "float b = a * g->len_f;", "float b = a * g->bin_f;"),
    ("shift scaled by the bin instead of the box, double",
     "*sd = (double)gamma * (double)off * g->len_d;",
     "*sd = (double)gamma * (double)off * g->bin_d;"),
    ("offset channels swapped in the forward",
     "deform_shift(mode, &d.gx, gamma, offset[(k * 2 + 0) * PH * PW + bin], &sxf, &sxd);\n"
     "                deform_shift(mode, &d.gy, gamma, offset[(k * 2 + 1) * PH * PW + bin], &syf, &syd);\n"
     "                const double m = mask ? (double)mask[k * PH * PW + bin] : 1.0;\n"
     "                for (int64_t c = 0; c < C; ++c) {\n"
     "                    const double *F",
     "deform_shift(mode, &d.gx, gamma, offset[(k * 2 + 1) * PH * PW + bin], &sxf, &sxd);\n"
     "                deform_shift(mode, &d.gy, gamma, offset[(k * 2 + 0) * PH * PW + bin], &syf, &syd);\n"
     "                const double m = mask ? (double)mask[k * PH * PW + bin] : 1.0;\n"
     "                for (int64_t c = 0; c < C; ++c) {\n"
     "                    const double *F"),
    ("modulation dropped in the forward",
     "o[c * PH * PW + bin] = m * (sum / (double)d.count);",
     "o[c * PH * PW + bin] = sum / (double)d.count;"),
    ("modulation dropped in the feature gradient",
     "const double gv = g[bin] * m / (double)d.count;",
     "const double gv = g[bin] / (double)d.count;"),
    ("mask gradient modulated", "om += gc * sum / (double)d.count;",
     "om += gc * m * sum / (double)d.count;"),
    ("gamma dropped from the offset gradient",
     "const double jx = (double)gamma * (mode == MODE_PARITY ? (double)d.gx.len_f : d.gx.len_d);",
     "const double jx = (mode == MODE_PARITY ? (double)d.gx.len_f : d.gx.len_d);"),
    ("x slope with swapped row weights",
     "dvx += ty.t.w_lo * (v12 - v11) + ty.t.w_hi * (v22 - v21);",
     "dvx += ty.t.w_hi * (v12 - v11) + ty.t.w_lo * (v22 - v21);"),
    ("y slope from the wrong corners",
     "dvy += tx.t.w_lo * (v21 - v11) + tx.t.w_hi * (v22 - v12);",
     "dvy += tx.t.w_lo * (v12 - v11) + tx.t.w_hi * (v22 - v21);"),
    ("slope kept for samples clamped at 0, double",
     "        d.slope = v >= 0.0;\n        v = fmax(v, 0.0);",
     "        d.slope = 1;\n        v = fmax(v, 0.0);"),
    ("slope kept for samples clamped at 0, binary32",
     "        d.slope = v >= 0.0f;\n        v = fmaxf(v, 0.0f);",
     "        d.slope = 1;\n        v = fmaxf(v, 0.0f);"),
    ("shift added after the within-bin term is rounded away, binary32",
     "float v = b2 + e;", "float v = b + e;"),
    ("shift added to the within-bin offset first, binary32",
     "float b2 = b + shift_f;\n        float half = (float)i + 0.5f;\n"
     "        float e0 = half * g->bin_f;\n        float e = e0 / (float)g->grid;\n"
     "        float v = b2 + e;",
     "float b2 = b;\n        float half = (float)i + 0.5f;\n"
     "        float e0 = half * g->bin_f;\n        float e = e0 / (float)g->grid;\n"
     "        float v = b2 + (shift_f + e);"),
    ("shift added to the bin position first, binary32",
     "float b = g->start_f + pos;\n        float b2 = b + shift_f;",
     "float b = g->start_f + (pos + shift_f);\n        float b2 = b;"),
]


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_is_caught(tmp_path, name, old, new):
    src = open(oracle.SOURCE).read()
    assert src.count(old) == 1, "planted-mistake pattern no longer matches the oracle: " + name
    path = tmp_path / "mutant.c"
    path.write_text(src.replace(old, new))
    lib_path = str(tmp_path / "libmutant.so")
    oracle.build(str(path), lib_path)
    failures = P.run_all(oracle.load(lib_path))
    assert failures, "no pin caught: " + name


def test_unmodified_copy_passes_every_pin(tmp_path):
    lib_path = str(tmp_path / "libcopy.so")
    oracle.build(oracle.SOURCE, lib_path)
    assert P.run_all(oracle.load(lib_path)) == []
