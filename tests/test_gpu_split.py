"""GPU parity of the forward GEMM with split K (launches of at most 128 output
tiles spread each tile's visited column units over several blocks and add
their fp32 partial tiles in a fixed order) against the fp64 oracle (Eq. 1).

Each case also runs the same call without a workspace (the unsplit kernel):
both must meet the oracle's tolerance, and the split result must be the same
bits on a second call (fixed summation order)."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_support import (assert_close, assert_fwd, dev_bf16, dev_f32, empty_bf16, host_bits, host_f64_from_bf16, ref_fwd,
                         say, sync, workspace)

pytestmark = pytest.mark.gpu


def _split_bytes(T, d_in, d_out, g, g_out=1):
    import paper_2609_33977_amd as gm
    return gm.gm_workspace_size(gm.GM_OP_FWD, T, d_in, d_out, g, g_out)


def _run(X, W, m, g, g_out, T, d_out, ws):
    import paper_2609_33977_amd as gm
    Y = empty_bf16(T, d_out)
    gm.gm_masked_linear_fwd(X, W, m, g, Y, ws, g_out=g_out)
    sync()
    return Y


def _check(case, mask, g_out=1):
    T, d_in, d_out, g = case.T, case.d_in, case.d_out, case.g
    need = _split_bytes(T, d_in, d_out, g, g_out)
    assert need > 0, "the shape is meant to take the split path"
    X, W, m = dev_bf16(case.X), dev_bf16(case.W), dev_f32(mask)
    ws = workspace(need)
    Ys = _run(X, W, m, g, g_out, T, d_out, ws)
    Ys2 = _run(X, W, m, g, g_out, T, d_out, ws)
    Yu = _run(X, W, m, g, g_out, T, d_out, None)
    ref, b = ref_fwd(oracle.from_bf16(case.X), oracle.from_bf16(case.W), mask, g, g_out)
    assert_close("Y (split K)", host_f64_from_bf16(Ys), ref, bound=b)
    assert_close("Y (unsplit)", host_f64_from_bf16(Yu), ref, bound=b)
    assert np.array_equal(host_bits(Ys), host_bits(Ys2)), "split-K forward is not deterministic"
    return Ys


@pytest.mark.parametrize("T,d_in,d_out,g", [
    (512, 2048, 1024, 256),    # 8 tiles, 2 shares of 4 units
    (300, 4096, 520, 256),     # ragged T and d_out, 4 shares
    (17, 4096, 4096, 256),     # smallest GEMM token count, 16 tiles
    (257, 4096, 1024, 512),    # 4-unit shares of 512-wide groups
    (700, 3072, 768, 64),      # 64-wide groups, 48 units
    (2048, 1024, 4096, 128),   # 128 tiles: 2 shares
])
def test_split_forward_parity(T, d_in, d_out, g):
    say(f"split-K forward: T={T} d_in={d_in} d_out={d_out} g={g}")
    case = workloads.make_linear_case((270, T, d_in, d_out, g), T, d_in, d_out, g, None)
    _check(case, case.mask)


@pytest.mark.parametrize("g", [16, 32, 64, 128])
def test_split_forward_square_groups(g):
    T, d_in, d_out = 260, 2048, 512
    say(f"split-K forward, {g}x{g} groups: T={T} d_in={d_in} d_out={d_out}")
    case = workloads.make_linear_case((271, g), T, d_in, d_out, g, None, g_out=g)
    _check(case, case.mask, g_out=g)


def test_split_forward_soft_selectors():
    T, d_in, d_out, g = 400, 2048, 768, 256
    say("split-K forward, fractional selectors")
    case = workloads.make_linear_case((272,), T, d_in, d_out, g, None)
    r = workloads.gen.rng_for(273)
    soft = r.uniform(0.05, 1.5, size=case.mask.shape).astype(np.float32)
    soft[r.uniform(size=soft.shape) < 0.4] = 0.0
    _check(case, soft)


def test_split_forward_empty_shares_and_all_pruned():
    # one kept group column per tile: most shares see no unit and add zeros;
    # an all-zero mask gives exactly zero
    T, d_in, d_out, g = 300, 4096, 512, 256
    say("split-K forward, sparse and empty tiles")
    case = workloads.make_linear_case((274,), T, d_in, d_out, g, None)
    sparse = np.zeros_like(case.mask)
    sparse[:, 5] = 1.0
    sparse[::7, 11] = 1.0
    _check(case, sparse)
    X, W = dev_bf16(case.X), dev_bf16(case.W)
    zero = np.zeros_like(case.mask)
    Y = _run(X, W, dev_f32(zero), g, 1, T, d_out, workspace(_split_bytes(T, d_in, d_out, g)))
    assert not np.any(host_bits(Y) & 0x7FFF), "all groups pruned: Y must be exactly zero"


@pytest.mark.parametrize("name,d_out,d_in", [("q", 5120, 5120), ("gate", 13824, 5120), ("down", 5120, 13824)])
def test_split_forward_llama2_13b_t512(name, d_out, d_in):
    # the T = 512 forward at LLaMA-2-13B shapes, in the launch the bench times;
    # the oracle checks 96 sampled output rows (all 512 tokens)
    import torch
    import paper_2609_33977_amd as gm
    T, g = 512, 256
    say(f"split-K forward, LLaMA-2-13B {name} [{d_out}x{d_in}] at T={T}")
    r = workloads.gen.rng_for(275, d_out, d_in)
    X = workloads.bf16_bits_from_f32(r.standard_normal((T, d_in), dtype=np.float32))
    W = workloads.bf16_bits_from_f32(r.standard_normal((d_out, d_in), dtype=np.float32) * np.float32(0.02))
    G_in = d_in // g
    mask = workloads.random_kept_mask(r, d_out * G_in, d_out * G_in // 2).reshape(d_out, G_in)
    Y = _run(dev_bf16(X), dev_bf16(W), dev_f32(mask), g, 1, T, d_out, workspace(_split_bytes(T, d_in, d_out, g)))
    rows = np.sort(r.choice(d_out, size=96, replace=False))
    Wr = oracle.from_bf16(W[rows])
    assert_fwd("Y (sampled rows)", host_f64_from_bf16(Y)[:, rows], oracle.from_bf16(X), Wr, mask[rows], g)
    del torch, gm
