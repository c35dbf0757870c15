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
    ("soft: linear decay at IoU equal to the threshold",
     "                        if (iou > iou_threshold) {\n                            const float w",
     "                        if (iou >= iou_threshold) {\n                            const float w"),
    ("soft: linear weight iou instead of 1 - iou",
     "const float w = 1.0f - iou;", "const float w = iou;"),
    ("soft: gaussian without the square",
     "double x = -((double)iou * (double)iou) / (double)sigma;",
     "double x = -((double)iou) / (double)sigma;"),
    ("soft: gaussian multiplied by sigma",
     "double x = -((double)iou * (double)iou) / (double)sigma;",
     "double x = -((double)iou * (double)iou) * (double)sigma;"),
    ("soft: exp series cut to three terms",
     "for (int n = 16; n >= 1; --n)", "for (int n = 3; n >= 1; --n)"),
    ("soft: exp without squaring back",
     "    for (int i = 0; i < k; ++i)\n        e = e * e;\n", ""),
    ("soft: equal current scores go to the later rank",
     "nms_rank_key(cur[r]) < nms_rank_key(cur[best])",
     "nms_rank_key(cur[r]) <= nms_rank_key(cur[best])"),
    ("soft: output score is the input score",
     "so[kept] = cur[best];", "so[kept] = scores[m];"),
    ("soft: a score equal to the threshold is dropped",
     "if (cur[r] < score_threshold)", "if (cur[r] <= score_threshold)"),
    ("batched: categories ignored",
     "if (ci != c || !(scores[i] >= score_threshold))", "if (!(scores[i] >= score_threshold))"),
    ("batched: no score threshold",
     "if (ci != c || !(scores[i] >= score_threshold))", "if (ci != c)"),
    ("batched hard: suppression at IoU equal to the threshold",
     "boxes + 4 * (int64_t)it[q].idx) > iou_threshold)",
     "boxes + 4 * (int64_t)it[q].idx) >= iou_threshold)"),
    ("batched hard: removed boxes still suppress",
     "            for (int32_t r = 0; r < n && kept < max_keep; ++r) {\n                if (!alive[r])\n                    continue;\n",
     "            for (int32_t r = 0; r < n && kept < max_keep; ++r) {\n                if (!alive[r] && r < 0)\n                    continue;\n"),
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
