import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def _has_gpu() -> bool:
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


def pytest_collection_modifyitems(config, items):
    if _has_gpu():
        return
    skip = pytest.mark.skip(reason="no GPU in this environment")
    for item in items:
        if "gpu" in item.keywords:
            item.add_marker(skip)


@pytest.hookimpl(hookwrapper=True)
def pytest_runtest_makereport(item, call):
    # On a failing GPU test, report the HIP runtime's pending error (if any) by name.
    outcome = yield
    rep = outcome.get_result()
    if rep.when == "call" and rep.failed and "gpu" in item.keywords:
        try:
            import ctypes
            hip = ctypes.CDLL("libamdhip64.so")
            hip.hipGetLastError.restype = ctypes.c_int
            hip.hipGetErrorName.restype = ctypes.c_char_p
            code = hip.hipGetLastError()
            rep.sections.append(("hip", f"pending HIP error after the failure: {code} {hip.hipGetErrorName(code).decode()}"))
        except OSError:
            pass

