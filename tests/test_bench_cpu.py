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
    if t["sources_sha256"] is not None and t["sources_sha256"] == b._sources_digest():
        expected = (t["fetch_kib"] * t["fetch_scale"] + t["write_kib"] * t["write_scale"]) * 1024.0
        assert b._dgate_traffic_bytes() == expected
        assert b._dgate_traffic_bytes(t["launch_mix"]) == expected
        assert b._dgate_traffic_bytes("another launch mix") is None
        # the committed counter summary is of these sources and these readings
        with open(os.path.join(ROOT, "profiles", "dgate_kernel_llama2_7b_step_traffic.md")) as f:
            text = f.read()
        assert t["sources_sha256"] in text
        assert f'launch mix: {t["launch_mix"]}' in text
        assert re.search(r"\b%.1f\b" % t["fetch_kib"], text)
    else:
        assert b._dgate_traffic_bytes() is None


def test_trace_summary_finds_the_roofline_batch(tmp_path):
    b = _bench_module()
    hdr = ('"Kind","Dispatch_Id","Kernel_Name","Start_Timestamp","End_Timestamp","Workgroup_Size_X",'
           '"Grid_Size_X"\n')
    rows, t = [], 0
    dg = "void gm::dgate_kernel<256, 1>(int)"
    seq = ([("void gm::fwd_kernel<256, 1>(int)", 256, 100), (dg, 256, 110), ("void gm::dx_kernel<256, 1>(int)", 256, 60)]
           + [(dg, w, d) for w, d in [(256, 120), (688, 330)] * 3])
    for name, wg, dur in seq:
        rows.append(f'"KERNEL_DISPATCH",{len(rows) + 1},"{name}",{t},{t + dur * 1000},512,{wg * 512}\n')
        t += dur * 1000 + 500
    p = tmp_path / "k.csv"
    p.write_text(hdr + "".join(rows))
    out = b._trace_summary(str(p))
    assert "| `gm::dgate_kernel<256, 1>` | 688 | 3 | 330.0 |" in out
    assert ("Longest back-to-back run of `gm::dgate_kernel<256, 1>`: 6 dispatches (workgroups: 256 x 3, 688 x 3)"
            in out)
    assert "mean 225.00 µs" in out


def test_traffic_is_null_for_other_sources():
    b = _bench_module()
    b.DGATE_TRAFFIC = dict(b.DGATE_TRAFFIC, sources_sha256="0" * 64)
    assert b._dgate_traffic_bytes() is None
