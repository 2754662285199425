"""The C ABI's host code under AddressSanitizer (no GPU needed): the library is
rebuilt with ASan on its host side and every argument-error and workspace
check of tests/test_abi_cpu.py runs against it in a child Python with the
ASan runtime preloaded.  Any invalid host memory access in the validation,
workspace carving or dispatch code would abort the child with an ASan
report."""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_abi_error_paths_under_asan(tmp_path):
    sys.path.insert(0, ROOT)
    from tests import asan_build

    try:
        rt = asan_build.asan_runtime()
    except FileNotFoundError as e:  # pragma: no cover
        pytest.skip(str(e))
    lib = asan_build.build_asan(str(tmp_path / "asan"))
    # the host code really is instrumented
    syms = subprocess.run(["nm", "-D", lib], capture_output=True, text=True).stdout
    assert "__asan_report" in syms
    env = dict(os.environ)
    env.update(LD_PRELOAD=rt, DUO_TEST_LIB=lib, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1:halt_on_error=1",
               PYTHONDONTWRITEBYTECODE="1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi_cpu.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert " passed" in r.stdout
