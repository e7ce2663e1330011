"""The parity checker of the GPU tests, exercised on the CPU.

A result computed the way the GPU computes it (fp32 sums of exact bf16
products, stored in bf16) passes every check.  Results with one planted
mistake pass the relative Frobenius bar of 1e-2 alone but fail the per-row or
elementwise checks: a group dropped from one 16 x 16 output fragment, one
element missing a 32-deep K slice, one dgate entry summed over 7/8 of its
group, 16 dX entries of one token computed from the wrong group column."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_support import TOL, bound_dgate, bound_dx, bound_fwd, check_close, rel_fro

T, D_IN, D_OUT, G = 2048, 1024, 2048, 256


@pytest.fixture(scope="module")
def case():
    c = workloads.make_linear_case((950,), T, D_IN, D_OUT, G, None)
    X, W, dY = oracle.from_bf16(c.X), oracle.from_bf16(c.W), oracle.from_bf16(c.dY)
    m = c.mask.astype(np.float64)
    return X, W, dY, m


def _bf16(a):
    return oracle.from_bf16(workloads.bf16_bits_from_f32(np.asarray(a, dtype=np.float32)))


def _fp32_like_gpu(case):
    """Y, dX in fp32 products/sums rounded to bf16 and dgate in fp32, as the kernels produce them."""
    X, W, dY, m = case
    Wm = (W * oracle.expand_mask(m, G)).astype(np.float32)
    Y = _bf16(X.astype(np.float32) @ Wm.T)
    dX = _bf16(dY.astype(np.float32) @ Wm)
    C = dY.astype(np.float32).T @ X.astype(np.float32)
    dgate = (W.astype(np.float32) * C).reshape(D_OUT, D_IN // G, G).sum(axis=2, dtype=np.float32)
    return Y, dX, dgate.astype(np.float64)


def test_gpu_like_results_pass(case):
    X, W, dY, m = case
    Y, dX, dgate = _fp32_like_gpu(case)
    assert check_close("Y", Y, oracle.linear_fwd(X, W, m, G), bound=bound_fwd(X, W, m, G)) == ""
    assert check_close("dX", dX, oracle.linear_bwd_dx(dY, W, m, G), bound=bound_dx(dY, W, m, G)) == ""
    assert check_close("dgate", dgate, oracle.linear_bwd_dgate(dY, X, W, G), bound=bound_dgate(dY, X, W, G)) == ""


def _kept_group(m, o):
    """First kept group of row o (None when the row keeps none)."""
    k = np.flatnonzero(m[o])
    return int(k[0]) if k.size else None


def test_dropped_group_in_one_fragment_is_caught(case):
    X, W, dY, m = case
    ref = oracle.linear_fwd(X, W, m, G)
    Y, _, _ = _fp32_like_gpu(case)
    t0, o0 = 512, 768
    bad = Y.copy()
    for o in range(o0, o0 + 16):  # each row of the fragment that keeps a group loses one
        v = _kept_group(m, o)
        if v is None:
            continue
        sl = slice(v * G, (v + 1) * G)
        bad[t0:t0 + 16, o] -= X[t0:t0 + 16, sl] @ W[o, sl]
    assert rel_fro(bad, ref) <= TOL  # the norm alone passes
    assert check_close("Y", bad, ref, bound=bound_fwd(X, W, m, G)) != ""


def test_single_wrong_element_is_caught(case):
    X, W, dY, m = case
    ref = oracle.linear_fwd(X, W, m, G)
    Y, _, _ = _fp32_like_gpu(case)
    bad = Y.copy()
    t = 3
    o = next(o for o in range(77, D_OUT) if _kept_group(m, o) is not None)
    v = _kept_group(m, o)
    bad[t, o] -= X[t, v * G:v * G + 32] @ W[o, v * G:v * G + 32]  # one 32-deep K slice of a kept group missing
    assert rel_fro(bad, ref) <= TOL
    assert check_close("Y", bad, ref, rows=True) == ""  # it hides in every row and column norm
    assert "outside the error bound" in check_close("Y", bad, ref, bound=bound_fwd(X, W, m, G))


def test_dgate_entry_summed_over_part_of_its_group_is_caught(case):
    X, W, dY, m = case
    ref = oracle.linear_bwd_dgate(dY, X, W, G)
    _, _, dgate = _fp32_like_gpu(case)
    bad = dgate.copy()
    o, v = 100, 1
    cols = slice(v * G, v * G + 32)  # the epilogue's sum misses 32 of the group's 256 columns
    bad[o, v] -= float(W[o, cols] @ (dY[:, o] @ X[:, cols]))
    assert rel_fro(bad, ref) <= TOL
    assert check_close("dgate", bad, ref, rows=True) == ""
    assert "outside the error bound" in check_close("dgate", bad, ref, bound=bound_dgate(dY, X, W, G))


def test_dx_row_with_a_misindexed_group_column_is_caught(case):
    X, W, dY, m = case
    ref = oracle.linear_bwd_dx(dY, W, m, G)
    _, dX, _ = _fp32_like_gpu(case)
    bad = dX.copy()
    t = 900
    Wm = W * oracle.expand_mask(m, G)
    bad[t, 0:16] = dY[t] @ Wm[:, G:G + 16]  # 16 columns of group 0 computed from group 1
    assert rel_fro(bad, ref) <= TOL
    assert check_close("dX", bad, ref, bound=bound_dx(dY, W, m, G)) != ""


def test_zero_row_must_stay_zero(case):
    X, W, dY, m = case
    m0 = m.copy()
    m0[5] = 0.0  # output row 5 fully pruned: column 5 of Y is exactly zero
    ref = oracle.linear_fwd(X, W, m0, G)
    bad = _bf16(ref)
    bad[17, 5] = 2.0 ** -40
    assert "exactly zero" in check_close("Y", bad, ref, rows=True)
