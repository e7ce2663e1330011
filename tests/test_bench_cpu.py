"""Host-side checks of bench.py's contract: one GPU only, a clean exit without a GPU, every leg switchable, and
the HBM traffic figure reported only for the GEMM sources its counters were taken on."""
import importlib.util
import os
import re
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")


def _bench_module():
    spec = importlib.util.spec_from_file_location("_bench_under_test", BENCH)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _run(*args, timeout=300):
    return subprocess.run([sys.executable, BENCH, *args], cwd=ROOT, capture_output=True, text=True, timeout=timeout)


def test_more_than_one_gpu_exits_with_a_message():
    r = _run("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_help_lists_every_leg_switch():
    r = _run("--help")
    assert r.returncode == 0
    for flag in ("--no-cpu-baseline", "--no-gemv", "--no-square", "--no-distill", "--no-hyper", "--no-model",
                 "--no-sweep", "--no-prefill", "--steps", "--warmup"):
        assert flag in r.stdout, flag


@pytest.mark.skipif(os.path.exists("/dev/kfd"), reason="a GPU driver is present")
def test_without_a_gpu_exits_cleanly():
    r = _run("--steps", "1", "--warmup", "1")
    assert r.returncode == 2
    assert "needs a GPU" in r.stderr
    assert r.stdout == ""


def test_traffic_follows_the_counted_sources():
    b = _bench_module()
    t = b.DGATE_TRAFFIC
    expected = (t["fetch_kib"] * t["fetch_scale"] + t["write_kib"] * t["write_scale"]) * 1024.0
    if t["sources_sha256"] == b._sources_digest():
        assert b._dgate_traffic_bytes() == expected
        # the committed counter summary is of these sources and these readings
        with open(os.path.join(ROOT, "profiles", "dgate_kernel_attn4096_traffic.md")) as f:
            text = f.read()
        assert t["sources_sha256"] in text
        assert re.search(r"\b%.1f\b" % t["fetch_kib"], text)
    else:
        assert b._dgate_traffic_bytes() is None


def test_traffic_is_null_for_other_sources():
    b = _bench_module()
    b.DGATE_TRAFFIC = dict(b.DGATE_TRAFFIC, sources_sha256="0" * 64)
    assert b._dgate_traffic_bytes() is None
