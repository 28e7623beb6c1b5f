"""include/odb.h as plain C (no GPU): the C drivers of the window pipeline and of the
streaming iteration compile as strict C11 with warnings as errors, link against libodb.so
and the HIP runtime, and start (their shared libraries resolve) with a usage error when
given no arguments."""
import importlib.util
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))


def _builder():
    spec = importlib.util.spec_from_file_location("odb_c_abi_build", os.path.join(HERE, "c_abi", "build_program.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_c_drivers_compile_link_and_start(tmp_path):
    exes = _builder().build(str(tmp_path))
    assert len(exes) == 2
    for exe in exes:
        r = subprocess.run([exe], capture_output=True, text=True, timeout=60)
        assert r.returncode == 2, (exe, r.returncode, r.stderr)
        assert "usage:" in r.stderr, exe
