"""The oracle's non-maximum suppression against its pins, and planted mistakes the pins
must catch (CPU only)."""
import pytest

import oracle
import oracle_nms_pins as P


@pytest.fixture(scope="module")
def lib():
    return oracle.load()


@pytest.mark.parametrize("pin", P.ALL_NMS_PINS, ids=lambda f: f.__name__)
def test_nms_pin(lib, pin):
    pin(lib)


MUTANTS = [
    ("suppression at IoU equal to the threshold", "> threshold)\n                removed[q] = 1;",
     ">= threshold)\n                removed[q] = 1;"),
    ("removed boxes also suppress", "        if (removed[r])\n            continue;\n        const int32_t i = it[r].idx;\n        keep_out[n++] = i;",
     "        const int32_t i = it[r].idx;\n        if (!removed[r])\n            keep_out[n++] = i;"),
    ("categories ignored", "if (removed[q] || (cats && cats[j] != cats[i]))", "if (removed[q])"),
    ("lowest score first", "    return ~asc;                               /* larger score, smaller key */",
     "    return asc;"),
    ("equal scores by decreasing index", "    return a->idx < b->idx ? -1 : (a->idx > b->idx ? 1 : 0);",
     "    return a->idx > b->idx ? -1 : (a->idx < b->idx ? 1 : 0);"),
    ("union without the intersection removed", "    float uni = sum - inter;", "    float uni = sum;"),
    ("negative overlaps kept (both clamps dropped)",
     "    iw = fmaxf(iw, 0.0f);\n    ih = fmaxf(ih, 0.0f);", ""),
    ("NaN scores first", "        return 0xffffffffu;                    /* NaN: after every number */",
     "        return 0u;"),
    ("one box too many", "for (int32_t r = 0; r < N && n < max_keep; ++r) {",
     "for (int32_t r = 0; r < N && n <= max_keep; ++r) {"),
]


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_is_caught(tmp_path, name, old, new):
    src = open(oracle.SOURCE).read()
    assert src.count(old) == 1, "planted-mistake pattern no longer matches the oracle: " + name
    path = tmp_path / "mutant.c"
    path.write_text(src.replace(old, new))
    lib_path = str(tmp_path / "libmutant.so")
    oracle.build(str(path), lib_path)
    assert P.run_all(oracle.load(lib_path)), "no pin caught: " + name


def test_unmodified_copy_passes_every_pin(tmp_path):
    lib_path = str(tmp_path / "libcopy.so")
    oracle.build(oracle.SOURCE, lib_path)
    assert P.run_all(oracle.load(lib_path)) == []
