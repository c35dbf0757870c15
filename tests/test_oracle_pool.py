"""The oracle's RoI max pooling against its pins, and planted mistakes the pins must
catch (CPU only; every planted mistake keeps memory accesses in bounds)."""
import pytest

import oracle
import oracle_pool_pins as P


@pytest.fixture(scope="module")
def lib():
    return oracle.load()


@pytest.mark.parametrize("pin", P.ALL_POOL_PINS, ids=lambda f: f.__name__)
def test_pool_pin(lib, pin):
    pin(lib)


MUTANTS = [
    ("box start truncated instead of rounded",
     "float s = roundf(c1 * scale);", "float s = truncf(c1 * scale);"),
    ("box end truncated instead of rounded",
     "float e = roundf(c2 * scale);", "float e = truncf(c2 * scale);"),
    ("inclusive +1 dropped from the box size",
     "    len = len + 1.0f;\n", ""),
    ("bin end floored instead of ceiled",
     "int hi = (int)ceilf(b) + (int)s;", "int hi = (int)floorf(b) + (int)s;"),
    ("bin start not shifted by the box start",
     "int lo = (int)floorf(a) + (int)s;", "int lo = (int)floorf(a);"),
    ("clip to size - 1",
     "r.hi = hi < 0 ? 0 : (hi > size ? size : hi);",
     "r.hi = hi < 0 ? 0 : (hi > size - 1 ? size - 1 : hi);"),
    ("ties: last maximum wins",
     "if (F[y * W + x] > best) {", "if (F[y * W + x] >= best) {"),
    ("columns binned with the row count",
     "pool_range rx = pool_bin(r[1], r[3], scales[lvl], PW, pw, (int)W);",
     "pool_range rx = pool_bin(r[1], r[3], scales[lvl], PH, pw, (int)W);"),
    ("x range from the y coordinates",
     "pool_range rx = pool_bin(r[1], r[3], scales[lvl], PW, pw, (int)W);",
     "pool_range rx = pool_bin(r[2], r[4], scales[lvl], PW, pw, (int)W);"),
    ("argmax index transposed",
     "where = (int32_t)(y * W + x);", "where = (int32_t)(x * H + y);"),
    ("backward skips pixel 0",
     "if (argmax[i] >= 0 && argmax[i] < H * W)", "if (argmax[i] > 0 && argmax[i] < H * W)"),
]


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_pool_mistake_is_caught(tmp_path, name, old, new):
    src = open(oracle.SOURCE).read()
    assert src.count(old) == 1, "planted-mistake pattern no longer matches the oracle: " + name
    path = tmp_path / "mutant.c"
    path.write_text(src.replace(old, new))
    lib_path = str(tmp_path / "libmutant.so")
    oracle.build(str(path), lib_path)
    failures = P.run_all(oracle.load(lib_path))
    assert failures, "no pin caught: " + name


def test_unmodified_copy_passes_every_pool_pin(tmp_path):
    path = tmp_path / "copy.c"
    path.write_text(open(oracle.SOURCE).read())
    lib_path = str(tmp_path / "libcopy.so")
    oracle.build(str(path), lib_path)
    assert P.run_all(oracle.load(lib_path)) == []
