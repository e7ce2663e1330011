"""The C-ABI tests again, against a build of the library whose host code runs
under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only: argument
validation, workspace layouts and the binding's checks; no kernel runs)."""
import importlib.util
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _build_module():
    spec = importlib.util.spec_from_file_location("_gm_build", os.path.join(ROOT, "paper_2609_33977_amd", "build.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_abi_layer_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    b = _build_module()
    try:
        lib = b.build_host_sanitized(str(tmp_path))
        rt = b.asan_runtime()
    except FileNotFoundError as e:
        pytest.skip(str(e))
    env = dict(os.environ, GM_LIBRARY_PATH=lib, LD_PRELOAD=rt,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_abi_cpu.py"), "-q", "-x",
                        "-p", "no:cacheprovider"], env=env, capture_output=True, text=True, timeout=600, cwd=ROOT)
    out = r.stdout[-4000:] + r.stderr[-4000:]
    assert r.returncode == 0, out
    assert "Sanitizer" not in out, out
    assert " passed" in r.stdout
