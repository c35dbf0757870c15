"""The C ABI's host code and the oracle under AddressSanitizer and
UndefinedBehaviorSanitizer (gcc, CPU only).

``sanitize/san_build.py`` compiles ``api.hip`` for the host with kernel launchers that do
nothing, and the oracle's C source, both with ``-fsanitize=address,undefined``.  A
child Python with the ASan runtime preloaded then runs the ABI tests, the binding
tests, valid calls through every entry point at the workloads' sizes
(``sanitize/host_paths.py``) and the oracle's pins against those builds.  Any report
ends the child with a failure.
"""
import os
import shutil
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))

SUITES = ["test_abi_cpu.py", "test_binding_cpu.py", "sanitize/host_paths.py",
          "test_oracle_pins.py", "test_oracle_pool.py", "test_oracle_nms.py",
          "test_oracle_deform.py"]


def _san():
    sys.path.insert(0, os.path.join(HERE, "sanitize"))
    import san_build
    return san_build


@pytest.fixture(scope="module")
def builds(tmp_path_factory):
    if shutil.which("g++") is None or shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    d = str(tmp_path_factory.mktemp("sanitize"))
    return _san().build_library(d), _san().build_oracle(d)


def test_host_code_and_oracle_under_sanitizers(builds, tmp_path):
    lib, orc = builds
    san = _san()
    env = dict(os.environ)
    env.update(LD_PRELOAD=san.preload(), REX_LIBRARY=lib, ORACLE_LIBRARY=orc,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    # the planted-mistake tests compile unsanitized copies of the oracle: not needed here
    cmd = [sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
           "-m", "not gpu", "-k", "not planted", *[os.path.join(HERE, s) for s in SUITES]]
    r = subprocess.run(cmd, env=env, cwd=str(tmp_path), capture_output=True, text=True,
                       timeout=900)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "passed" in r.stdout and "ERROR: AddressSanitizer" not in r.stderr, tail
    assert "runtime error" not in r.stderr, tail
