"""GPU parity of the masked linear with square g x g groups (Sec. 2.1 group
shapes; the 16 x 16 .. 128 x 128 variants of App. C) against the fp64 oracle:
forward, dX, dgate, the decode GEMV and the row-wise export, on shapes that
span several tiles with ragged tails, plus one LLaMA-2-7B-sized layer checked
on sampled tokens and group rows."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_support import (assert_close, assert_dgate, assert_dx, assert_fwd, dev_bf16, dev_f32, empty_bf16, empty_f32,
                         host_bits, host_f64_from_bf16, ref_dgate, ref_dx, ref_fwd, say, sync, workspace)

pytestmark = pytest.mark.gpu


def _dev(case, mask=None):
    m = case.mask if mask is None else mask
    return dict(X=dev_bf16(case.X), W=dev_bf16(case.W), dY=dev_bf16(case.dY), mask=dev_f32(m))


def _fwd(d, g):
    import paper_2609_33977_amd as gm
    T = d["X"].shape[0]
    Y = empty_bf16(T, d["W"].shape[0])
    gm.gm_masked_linear_fwd(d["X"], d["W"], d["mask"], g, Y, g_out=g)
    sync()
    return Y


def _bwd(d, g, want_dx=True, want_dgate=True):
    import paper_2609_33977_amd as gm
    T, d_in = d["X"].shape
    d_out = d["W"].shape[0]
    dX = empty_bf16(T, d_in) if want_dx else None
    dgate = empty_f32(d_out // g, d_in // g) if want_dgate else None
    ws = workspace(gm.gm_workspace_size(gm.GM_OP_BWD, T, d_in, d_out, g, g))
    gm.gm_masked_linear_bwd(d["dY"], d["X"], d["W"], d["mask"], g, dX, dgate, ws, g_out=g)
    sync()
    return dX, dgate


def _oracle(case, mask=None):
    """Oracle Y, dX, dgate and their elementwise error bounds."""
    m = case.mask if mask is None else mask
    X, W, dY = oracle.from_bf16(case.X), oracle.from_bf16(case.W), oracle.from_bf16(case.dY)
    Y, bY = ref_fwd(X, W, m, case.g, case.g_out)
    dX, bdX = ref_dx(dY, W, m, case.g, case.g_out)
    dgate, bdg = ref_dgate(dY, X, W, case.g, case.g_out)
    return Y, dX, dgate, bY, bdX, bdg


def _case(key, T, d_in, d_out, g, kept=None):
    return workloads.make_linear_case(key, T, d_in, d_out, g, kept, g_out=g)


SHAPES = [  # (T, d_in, d_out, g): d_in a multiple of max(g, 64), d_out of g; tails in every tile dimension
    (300, 1024, 528, 16),
    (77, 640, 416, 32),
    (260, 1344, 320, 64),
    (130, 1152, 384, 128),
    (513, 2048, 1024, 16),
    (256, 768, 256, 128),
]


@pytest.mark.parametrize("T,d_in,d_out,g", SHAPES)
def test_square_fwd_bwd_parity(T, d_in, d_out, g):
    say(f"square {g}x{g}: T={T} d_in={d_in} d_out={d_out}")
    case = _case((220, T, d_in, d_out, g), T, d_in, d_out, g)
    d = _dev(case)
    Y = _fwd(d, g)
    dX, dgate = _bwd(d, g)
    Yr, dXr, dgr, bY, bdX, bdg = _oracle(case)
    assert_close("Y", host_f64_from_bf16(Y), Yr, bound=bY)
    assert_close("dX", host_f64_from_bf16(dX), dXr, bound=bdX)
    assert_close("dgate", dgate.cpu().numpy(), dgr, bound=bdg)


@pytest.mark.parametrize("g", [16, 32, 64, 128])
def test_square_soft_mask(g):
    T, d_in, d_out = 200, 1024, 512
    say(f"square {g}x{g} soft mask")
    case = _case((221, g), T, d_in, d_out, g)
    r = workloads.gen.rng_for(222, g)
    soft = r.uniform(0.05, 1.5, size=case.mask.shape).astype(np.float32)
    soft[r.uniform(size=soft.shape) < 0.4] = 0.0
    d = _dev(case, soft)
    Y = _fwd(d, g)
    dX, dgate = _bwd(d, g)
    Yr, dXr, dgr, bY, bdX, bdg = _oracle(case, soft)
    assert_close("Y", host_f64_from_bf16(Y), Yr, bound=bY)
    assert_close("dX", host_f64_from_bf16(dX), dXr, bound=bdX)
    assert_close("dgate", dgate.cpu().numpy(), dgr, bound=bdg)


@pytest.mark.parametrize("g", [16, 32])
def test_square_soft_selectors_in_the_first_chunk_only(g):
    """List columns of 64 input columns hold 64/g group columns and are built per
    1024-row chunk: fractional selectors only in the rows of the first chunk
    (of three, the last one ragged) must still mark the list column soft."""
    T, d_in, d_out = 64, 512, 3008
    say(f"square {g}x{g}: soft selectors only in the first 1024-row chunk, d_out={d_out}")
    case = _case((232, g), T, d_in, d_out, g)
    m = case.mask.astype(np.float32).copy()
    u = np.arange(1, 1024 // g, 5)           # mask rows inside output rows 0 .. 1023
    m[u, 1] = np.where(np.arange(u.size) % 2, 0.5, 1.25).astype(np.float32)  # group column 1 (list column 0)
    d = _dev(case, m)
    dX, dgate = _bwd(d, g)
    Yr, dXr, dgr, bY, bdX, bdg = _oracle(case, m)
    assert_close("dX", host_f64_from_bf16(dX), dXr, bound=bdX)
    assert_close("dgate", dgate.cpu().numpy(), dgr, bound=bdg)


@pytest.mark.parametrize("g", [16, 128])
def test_square_dense_and_empty_masks(g):
    T, d_in, d_out = 256, 1024, 768
    case = _case((223, g), T, d_in, d_out, g)
    ones, zeros = np.ones_like(case.mask), np.zeros_like(case.mask)
    say(f"square {g}x{g}: all-ones mask")
    d = _dev(case, ones)
    Y = _fwd(d, g)
    dX, _ = _bwd(d, g, want_dgate=False)
    Yr, dXr, _, bY, bdX, _ = _oracle(case, ones)
    assert_close("Y (dense)", host_f64_from_bf16(Y), Yr, bound=bY)
    assert_close("dX (dense)", host_f64_from_bf16(dX), dXr, bound=bdX)
    say(f"square {g}x{g}: all-zeros mask")
    d = _dev(case, zeros)
    Y = _fwd(d, g)
    dX, dgate = _bwd(d, g)
    assert not np.any(host_bits(Y) & 0x7FFF)
    assert not np.any(host_bits(dX) & 0x7FFF)
    _, _, dgr, _, _, bdg = _oracle(case, zeros)
    assert_close("dgate (all pruned)", dgate.cpu().numpy(), dgr, bound=bdg)


def test_square_one_group_per_unit_kept():
    # 16 x 16: every 32-column unit keeps exactly one of its two groups, in a
    # checkerboard over the mask rows, so each K slice mixes read and
    # zero-filled chunks and each dX list column mixes kept bits
    T, d_in, d_out, g = 160, 512, 256, 16
    case = _case((224,), T, d_in, d_out, g)
    u, v = np.meshgrid(np.arange(d_out // g), np.arange(d_in // g), indexing="ij")
    checker = ((u + v) % 2).astype(np.float32)
    say("square 16x16 checkerboard mask")
    d = _dev(case, checker)
    Y = _fwd(d, g)
    dX, dgate = _bwd(d, g)
    Yr, dXr, dgr, bY, bdX, bdg = _oracle(case, checker)
    assert_close("Y", host_f64_from_bf16(Y), Yr, bound=bY)
    assert_close("dX", host_f64_from_bf16(dX), dXr, bound=bdX)
    assert_close("dgate", dgate.cpu().numpy(), dgr, bound=bdg)


@pytest.mark.parametrize("g", [16, 64])
def test_square_dgate_mask_independence_and_single_outputs(g):
    T, d_in, d_out = 192, 1024, 512
    case = _case((225, g), T, d_in, d_out, g)
    say(f"square {g}x{g}: dgate mask independence, dgate-only and dX-only calls")
    d1 = _dev(case)
    d2 = _dev(case, np.ones_like(case.mask))
    _, g1 = _bwd(d1, g)
    _, g2 = _bwd(d2, g, want_dx=False)
    assert np.array_equal(g1.cpu().numpy(), g2.cpu().numpy())
    dX_only, _ = _bwd(d1, g, want_dgate=False)
    dX_both, _ = _bwd(d1, g)
    assert np.array_equal(host_bits(dX_only), host_bits(dX_both))


@pytest.mark.parametrize("T", [1, 5, 16])
@pytest.mark.parametrize("g,d_in", [(16, 11008), (32, 4096), (128, 2048)])
def test_square_decode_forward(T, g, d_in):
    # 16 x 16 over 11008 inputs: 688 groups per row, the larger per-wave list
    d_out = 384
    say(f"square {g}x{g} decode: T={T} d_in={d_in}")
    case = _case((226, T, g), T, d_in, d_out, g)
    d = _dev(case)
    Y = _fwd(d, g)
    Yr, _, _, bY, _, _ = _oracle(case)
    assert_close("Y", host_f64_from_bf16(Y), Yr, bound=bY)


@pytest.mark.parametrize("g", [16, 32, 128])
def test_square_export_and_packed_forward(g):
    import torch
    import paper_2609_33977_amd as gm
    d_in, d_out = 2048, 256
    say(f"square {g}x{g}: export and packed forward")
    case = _case((227, g), 16, d_in, d_out, g)
    soft = case.mask * workloads.gen.rng_for(228, g).uniform(0.5, 1.5, size=case.mask.shape).astype(np.float32)
    d = _dev(case, soft)
    cap = d_out * (d_in // g)
    Wp = torch.zeros(cap, g, dtype=torch.bfloat16, device="cuda")
    chunk = torch.full((cap,), -1, dtype=torch.int32, device="cuda")
    scale = torch.zeros(cap, dtype=torch.float32, device="cuda")
    rowptr = torch.zeros(d_out + 1, dtype=torch.int32, device="cuda")
    gm.gm_pack_rows(d["W"], d["mask"], g, cap, Wp, chunk, scale, rowptr, g_out=g)
    sync()
    # expected: every output row carries the kept groups of its mask row, in column order
    rows = np.repeat(soft, g, axis=0)
    keep = rows != 0
    rp = np.concatenate([[0], np.cumsum(keep.sum(axis=1))]).astype(np.int32)
    o_idx, v_idx = np.nonzero(keep)
    k = rp[-1]
    assert np.array_equal(rowptr.cpu().numpy(), rp)
    assert np.array_equal(chunk.cpu().numpy()[:k], v_idx.astype(np.int32))
    assert np.array_equal(scale.cpu().numpy()[:k], rows[o_idx, v_idx])
    assert np.array_equal(host_bits(Wp)[:k], case.W.reshape(d_out, d_in // g, g)[o_idx, v_idx])
    Y = empty_bf16(16, d_out)
    gm.gm_packed_linear_fwd(d["X"], Wp, chunk, scale, rowptr, d_out, g, Y)
    sync()
    Yr, _, _, bY, _, _ = _oracle(case, soft)
    assert_close("Y (packed)", host_f64_from_bf16(Y), Yr, bound=bY)
    Yi = _fwd(d, g)
    assert_close("Y (in place, 16-token MFMA path)", host_f64_from_bf16(Yi), Yr, bound=bY)
    # both layouts run the 16-token MFMA kernel with the same products in the same order
    assert np.array_equal(host_bits(Y), host_bits(Yi))


@pytest.mark.parametrize("g", [16, 64])
def test_square_llama2_7b_down_projection(g):
    # the 4096 x 11008 down projection of LLaMA-2-7B at the mask-learning
    # step's token count, half of its groups kept; sampled tokens and group rows
    cfg = workloads.config("llama2_7b_step")
    T = cfg["T"]
    d_out, d_in = 4096, 11008
    say(f"square {g}x{g}: llama2-7b down projection T={T}")
    case = _case((229, g), T, d_in, d_out, g)
    d = _dev(case)
    Y = _fwd(d, g)
    dX, dgate = _bwd(d, g)
    r = workloads.gen.rng_for(230, g)
    X, W, dY = oracle.from_bf16(case.X), oracle.from_bf16(case.W), oracle.from_bf16(case.dY)
    m = case.mask.astype(np.float64)
    t_s = np.sort(r.choice(T, size=32, replace=False))
    u_s = np.sort(r.choice(d_out // g, size=4, replace=False))
    rows = (u_s[:, None] * g + np.arange(g)[None, :]).reshape(-1)
    assert_fwd("Y (sampled tokens)", host_f64_from_bf16(Y)[t_s], X, W, m, g, g, rows=t_s)
    assert_dx("dX (sampled tokens)", host_f64_from_bf16(dX)[t_s], dY, W, m, g, g, rows=t_s)
    assert_dgate("dgate (sampled group rows)", dgate.cpu().numpy()[u_s], dY[:, rows], X, W[rows], g, g)


def test_square_16_widest_rows():
    # 16 x 16 groups over 16384 inputs: 1024 selectors per mask row, the
    # forward's and the decode GEMV's largest per-row lists
    T, d_in, d_out, g = 130, 16384, 128, 16
    say(f"square 16x16 widest rows: T={T} d_in={d_in}")
    case = _case((231,), T, d_in, d_out, g)
    d = _dev(case)
    Y = _fwd(d, g)
    dX, dgate = _bwd(d, g)
    Yr, dXr, dgr, bY, bdX, bdg = _oracle(case)
    assert_close("Y", host_f64_from_bf16(Y), Yr, bound=bY)
    assert_close("dX", host_f64_from_bf16(dX), dXr, bound=bdX)
    assert_close("dgate", dgate.cpu().numpy(), dgr, bound=bdg)
    case1 = _case((232,), 3, d_in, d_out, g)
    Y1 = _fwd(_dev(case1), g)
    o1 = _oracle(case1)
    assert_close("Y (decode)", host_f64_from_bf16(Y1), o1[0], bound=o1[3])
