"""Helpers for the GPU parity tests: move seeded host inputs to the device, run
the library through its C ABI, and compare with the fp64 oracle."""
from __future__ import annotations

import dataclasses
import sys

import numpy as np

import oracle
import workloads

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


# ------------------------------------------------------------ elementwise error bounds
#
# The products of two bf16 values are exact in fp32 (8 + 8 significant bits fit
# in 24), so an output of the masked GEMMs differs from the exact fp64 value
# only by fp32 summation error and, for Y and dX, by the final rounding to bf16.
#   * A sum of K terms in fp32 is within K u32 sum|terms| of the exact sum
#     (round to nearest, any order); the bound below doubles it, which also
#     covers a matrix core that rounds once per product pair instead of once per
#     addition.  Soft selectors scale a weight in bf16 first, which adds u16 of
#     every term.
#   * The bf16 store (round to nearest even) adds at most u16 of the stored value.
# sum|terms| is the same product taken on absolute values: |X| |W_hat|^T for Y,
# |dY| |W_hat| for dX, and for dgate the group sums of |W| (|dY|^T |X|).
# For dgate the worst-case form (about 2 T u32 of that sum) is loose, so its
# elementwise check uses the probabilistic bound of rounding-error analysis:
# with independent round-to-nearest errors a sum of n terms is within
# lam sqrt(n) u32 sum|terms| except with probability below 2 exp(-lam^2 / 2)
# (lam = 8: about 3e-14 per element), with n = T (the token sum) + g (the group sum).

U32 = 2.0 ** -24  # unit roundoff of fp32
U16 = 2.0 ** -8   # unit roundoff of bf16 (8 significant bits)
LAM = 8.0


def _soft(m) -> bool:
    m = np.asarray(m)
    return bool(np.any((m != 0) & (m != 1)))


def bound_fwd(X, W, m, g, g_out=1, ref=None):
    """Elementwise bound on |Y_gpu - Y| for Y = X W_hat^T in bf16 (X, W, ref in fp64)."""
    S = oracle.linear_fwd(np.abs(X), np.abs(W), np.abs(np.asarray(m, dtype=np.float64)), g, g_out)
    acc = (2.0 * X.shape[1] * U32 + (U16 if _soft(m) else 0.0)) * S
    ref = oracle.linear_fwd(X, W, m, g, g_out) if ref is None else ref
    return U16 * (np.abs(ref) + acc) + acc


def bound_dx(dY, W, m, g, g_out=1, ref=None):
    """Elementwise bound on |dX_gpu - dX| for dX = dY W_hat in bf16."""
    S = oracle.linear_bwd_dx(np.abs(dY), np.abs(W), np.abs(np.asarray(m, dtype=np.float64)), g, g_out)
    acc = (2.0 * dY.shape[1] * U32 + (U16 if _soft(m) else 0.0)) * S
    ref = oracle.linear_bwd_dx(dY, W, m, g, g_out) if ref is None else ref
    return U16 * (np.abs(ref) + acc) + acc


def bound_dgate(dY, X, W, g, g_out=1):
    """Probabilistic elementwise bound on |dgate_gpu - dgate| (fp32 throughout)."""
    S = oracle.linear_bwd_dgate(np.abs(dY), np.abs(X), np.abs(W), g, g_out)
    return LAM * np.sqrt(dY.shape[0] + g * g_out) * U32 * S


def ref_fwd(X, W, m, g, g_out=1):
    ref = oracle.linear_fwd(X, W, m, g, g_out)
    return ref, bound_fwd(X, W, m, g, g_out, ref)


def ref_dx(dY, W, m, g, g_out=1):
    ref = oracle.linear_bwd_dx(dY, W, m, g, g_out)
    return ref, bound_dx(dY, W, m, g, g_out, ref)


def ref_dgate(dY, X, W, g, g_out=1):
    return oracle.linear_bwd_dgate(dY, X, W, g, g_out), bound_dgate(dY, X, W, g, g_out)


MIN_ROW = 64  # per-row relative errors are checked on rows of at least this many elements


def check_close(name: str, got, ref, tol: float = TOL, bound=None, rows=None) -> str:
    """The parity checks as one verdict: '' when every check passes, else what failed.

    * relative Frobenius error of the whole tensor <= tol (the headline bar);
    * with ``rows`` (by default: whenever a bound is given, i.e. for the masked
      linear's Y, dX and dgate), for 2-D tensors the same relative error <= tol
      for every row and every column of at least MIN_ROW elements, and an
      exactly zero GPU slice where the oracle's slice is exactly zero;
    * with ``bound``, |got - ref| <= bound for every element.
    """
    rows = bound is not None if rows is None else rows
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if got.shape != ref.shape:
        return f"{name}: shape {got.shape} vs {ref.shape}"
    if not np.all(np.isfinite(got)):
        return f"{name}: non-finite values"
    if not np.any(ref):
        return "" if not np.any(got) else f"{name}: oracle is exactly zero, GPU is not"
    err = rel_fro(got, ref)
    if err > tol:
        return f"{name}: rel-Frobenius {err:.3e} > {tol}"
    if rows and got.ndim == 2:
        diff = got - ref
        for axis, what in ((1, "row"), (0, "column")):
            if ref.shape[axis] < MIN_ROW:
                continue
            den = np.linalg.norm(ref, axis=axis)
            num = np.linalg.norm(diff, axis=axis)
            zero = den == 0
            if np.any(num[zero] != 0):
                return f"{name}: {what} {int(np.flatnonzero(zero & (num != 0))[0])} is exactly zero in the oracle, not on the GPU"
            rel = num[~zero] / den[~zero]
            if rel.size and rel.max() > tol:
                return f"{name}: {what} {int(np.flatnonzero(~zero)[np.argmax(rel)])} rel-Frobenius {rel.max():.3e} > {tol}"
    if bound is not None:
        over = np.abs(got - ref) > np.asarray(bound, dtype=np.float64)
        if np.any(over):
            idx = np.unravel_index(int(np.flatnonzero(over)[0]), got.shape)
            return (f"{name}: {int(over.sum())} element(s) outside the error bound, first at {idx}: "
                    f"|{got[idx]:.6g} - {ref[idx]:.6g}| > {np.asarray(bound)[idx]:.3g}")
    return ""


def assert_close(name: str, got, ref, tol: float = TOL, bound=None, rows=None) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    msg = check_close(name, got, ref, tol, bound, rows)
    assert not msg, msg
    if not np.any(ref):
        return 0.0
    err = rel_fro(got, ref)
    extra = ""
    if bound is not None:
        ratio = np.abs(got - ref) / np.maximum(np.asarray(bound, dtype=np.float64), 1e-300)
        extra = f", max |err| / bound {float(ratio.max()):.2f}"
    say(f"  {name}: rel-Frobenius {err:.3e}{extra}")
    return err


def assert_fwd(name, got, X, W, m, g, g_out=1, rows=None):
    """Y parity: oracle reference (optionally on the token rows ``rows``), norm, per-row and elementwise checks."""
    Xs = X if rows is None else X[rows]
    ref, b = ref_fwd(Xs, W, m, g, g_out)
    return assert_close(name, got, ref, bound=b)


def assert_dx(name, got, dY, W, m, g, g_out=1, rows=None):
    dYs = dY if rows is None else dY[rows]
    ref, b = ref_dx(dYs, W, m, g, g_out)
    return assert_close(name, got, ref, bound=b)


def assert_dgate(name, got, dY, X, W, g, g_out=1):
    ref, b = ref_dgate(dY, X, W, g, g_out)
    return assert_close(name, got, ref, bound=b)


# ------------------------------------------------------------ gate inputs of the workloads

def budget_shift(logits, noise, kept: int) -> float:
    """The logit offset that makes exactly ``kept`` gates pass, decided by the oracle's fp64 gate:
    the midpoint between the kept-th and (kept+1)-th largest z = logit + ln u - ln(1 - u)."""
    z = np.sort(np.asarray(logits, dtype=np.float64) + oracle.logistic_noise(noise))[::-1]
    if kept <= 0:
        return -float(z[0]) - 1.0
    if kept >= z.size:
        return -float(z[-1]) + 1.0
    return -0.5 * float(z[kept - 1] + z[kept])


def budgeted_independent_inputs(rng, n: int, kept: int, tau: float):
    """Independent draws (logits ~ N(0, 1), u ~ U(0, 1)) shifted by one offset so that the oracle's
    hard gate keeps exactly ``kept`` of the n groups; returns (logits f32, noise f32, oracle mask)."""
    logits, noise = workloads.independent_gate_inputs(rng, n)
    shifted = (logits.astype(np.float64) + budget_shift(logits, noise, kept)).astype(np.float32)
    m, _ = oracle.gate(shifted, noise, tau, True)
    assert int(m.sum()) == kept, "the fp32 shift moved a gate across the threshold"
    return shifted, noise, m.astype(np.float32)


def independent_case(key, T, d_in, d_out, g, kept=None, tau=0.5, g_out=1):
    """A linear case whose gate inputs are independent draws with an exact kept budget (the mask is
    the oracle's decision on them); X, W and dY as in workloads.make_linear_case."""
    case = workloads.make_linear_case(key, T, d_in, d_out, g, kept, tau=tau, g_out=g_out)
    shape = case.mask.shape
    r = workloads.gen.rng_for(310, *key)
    logits, noise, m = budgeted_independent_inputs(r, case.mask.size, case.kept, tau)
    return dataclasses.replace(case, logits=logits.reshape(shape), noise=noise.reshape(shape), mask=m.reshape(shape))


def check_gate(mask_gpu, logits, noise, tau, band: float = 1e-6):
    """Hard mask against the oracle: bit-exact outside the near-threshold band, those inside counted.
    Returns (oracle mask, oracle y, near-threshold flags)."""
    m_ref, y_ref = oracle.gate(np.asarray(logits, np.float64).ravel(), np.asarray(noise).ravel(), tau, True)
    near = oracle.near_threshold(y_ref, band)
    m = np.asarray(mask_gpu, dtype=np.float64).ravel()
    mism = (m != m_ref) & ~near
    say(f"  hard gate: {int(near.sum())} of {near.size} within {band} of the threshold; "
        f"{int(mism.sum())} mismatches outside")
    assert not mism.any(), "hard mask differs from the oracle outside the near-threshold band"
    assert set(np.unique(m)) <= {0.0, 1.0}
    return m_ref, y_ref, near


def sync():
    torch_mod().cuda.synchronize()
