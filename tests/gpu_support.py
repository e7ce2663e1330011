"""Helpers for the GPU parity tests: move seeded host inputs to the device, run
the library through its C ABI, and compare with the fp64 oracle."""
from __future__ import annotations

import sys

import numpy as np

import oracle

TOL = 1e-2  # relative Frobenius error bound for Y, dX and dgate with bf16 inputs


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def torch_mod():
    import torch
    return torch


def dev_bf16(bits: np.ndarray):
    torch = torch_mod()
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16)
    return t.cuda()


def dev_f32(a):
    torch = torch_mod()
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def host_bits(t) -> np.ndarray:
    torch = torch_mod()
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def host_f64_from_bf16(t) -> np.ndarray:
    return oracle.from_bf16(host_bits(t))


def empty_bf16(*shape):
    torch = torch_mod()
    return torch.empty(shape, dtype=torch.bfloat16, device="cuda")


def empty_f32(*shape):
    torch = torch_mod()
    return torch.empty(shape, dtype=torch.float32, device="cuda")


def workspace(nbytes: int):
    torch = torch_mod()
    return torch.empty(max(nbytes, 16), dtype=torch.uint8, device="cuda")


def rel_fro(got: np.ndarray, ref: np.ndarray) -> float:
    den = float(np.linalg.norm(ref))
    num = float(np.linalg.norm(np.asarray(got, dtype=np.float64) - ref))
    return num / den if den > 0 else num


def assert_close(name: str, got, ref, tol: float = TOL) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, f"{name}: shape {got.shape} vs {ref.shape}"
    assert np.all(np.isfinite(got)), f"{name}: non-finite values"
    if not np.any(ref):
        assert not np.any(got), f"{name}: oracle is exactly zero, GPU is not"
        return 0.0
    err = rel_fro(got, ref)
    say(f"  {name}: rel-Frobenius {err:.3e}")
    assert err <= tol, f"{name}: rel-Frobenius {err:.3e} > {tol}"
    return err


def sync():
    torch_mod().cuda.synchronize()
