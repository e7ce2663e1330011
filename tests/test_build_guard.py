"""The build's kernel resource check (CPU): clang's resource remarks of a
kernel that spills, uses scratch, or crowds the register file with tied MFMA
accumulators fail the build; the figures of the kernels as built pass."""
import importlib.util
import os

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _build_module():
    spec = importlib.util.spec_from_file_location("_gm_build", os.path.join(ROOT, "paper_2609_33977_amd", "build.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _remarks(name, vgprs, agprs, scratch=0, spill=0):
    r = f"x.hip:1:1: remark: {{}} [-Rpass-analysis=kernel-resource-usage]\n"
    return "".join(r.format(t) for t in (
        f"Function Name: {name}", f"    VGPRs: {vgprs}", f"    AGPRs: {agprs}",
        f"    ScratchSize [bytes/lane]: {scratch}", f"    SGPRs Spill: 6", f"    VGPRs Spill: {spill}"))


def test_resource_check():
    b = _build_module()
    ok = _remarks("_ZN2gm10fwd_kernelILi256ELi1EEEv", 128, 107)  # the forward GEMM as built: 235 registers
    kernels, problems = b._resource_report("gemm.hip", ok)
    assert problems == [] and kernels["_ZN2gm10fwd_kernelILi256ELi1EEEv"]["AGPRs"] == 107
    assert b._resource_report("gemm.hip", _remarks("k", 128, 126))[1]          # 254 registers, tied accumulators
    assert b._resource_report("gemv.hip", _remarks("k", 128, 126))[1] == []     # no tied accumulators there
    assert b._resource_report("gate.hip", _remarks("k", 40, 0, scratch=16))[1]  # scratch anywhere
    assert b._resource_report("hyper.hip", _remarks("k", 40, 0, spill=2))[1]    # vector spills anywhere
