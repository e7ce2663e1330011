"""GPU parity of the masked linear (forward, dX, dgate, decode and packed paths)
against the fp64 oracle, on shapes that span several tiles and ragged tails."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_support import (assert_close, dev_bf16, dev_f32, empty_bf16, empty_f32, host_bits, host_f64_from_bf16,
                         ref_dgate, ref_dx, ref_fwd, say, sync, workspace)

pytestmark = pytest.mark.gpu


def _dev_case(case, mask=None):
    m = case.mask if mask is None else mask
    return dict(X=dev_bf16(case.X), W=dev_bf16(case.W), dY=dev_bf16(case.dY), mask=dev_f32(m))


def _fwd(d, g):
    import paper_2609_33977_amd as gm
    T = d["X"].shape[0]
    d_out = d["W"].shape[0]
    Y = empty_bf16(T, d_out)
    ws = workspace(gm.gm_workspace_size(gm.GM_OP_FWD, T, d["X"].shape[1], d_out, g))
    gm.gm_masked_linear_fwd(d["X"], d["W"], d["mask"], g, Y, ws)
    sync()
    return Y


def _bwd(d, g, want_dx=True, want_dgate=True):
    import paper_2609_33977_amd as gm
    T, d_in = d["X"].shape
    d_out = d["W"].shape[0]
    dX = empty_bf16(T, d_in) if want_dx else None
    dgate = empty_f32(d_out, d_in // g) if want_dgate else None
    ws = workspace(gm.gm_workspace_size(gm.GM_OP_BWD, T, d_in, d_out, g))
    gm.gm_masked_linear_bwd(d["dY"], d["X"], d["W"], d["mask"], g, dX, dgate, ws)
    sync()
    return dX, dgate


def _oracle_all(case, mask=None):
    """Oracle Y, dX, dgate and their elementwise error bounds."""
    m = case.mask if mask is None else mask
    X, W, dY = oracle.from_bf16(case.X), oracle.from_bf16(case.W), oracle.from_bf16(case.dY)
    Y, bY = ref_fwd(X, W, m, case.g)
    dX, bdX = ref_dx(dY, W, m, case.g)
    dgate, bdg = ref_dgate(dY, X, W, case.g)
    return Y, dX, dgate, bY, bdX, bdg


SHAPES = [  # (T, d_in, d_out, g): several tiles in every dimension plus ragged tails
    (128, 1024, 1024, 256),   # single masked linear of the smallest workload
    (77, 320, 200, 64),       # T, d_in and d_out all ragged
    (300, 1024, 264, 128),
    (257, 1024, 512, 512),    # a group spans two dgate tiles
    (33, 2048, 136, 256),
    (520, 768, 1000, 256),
]


@pytest.mark.parametrize("T,d_in,d_out,g", SHAPES)
def test_fwd_bwd_parity(T, d_in, d_out, g):
    say(f"linear fwd+bwd: T={T} d_in={d_in} d_out={d_out} g={g}")
    case = workloads.make_linear_case((200, T, d_in, d_out, g), T, d_in, d_out, g, None)
    d = _dev_case(case)
    Y = _fwd(d, g)
    dX, dgate = _bwd(d, g)
    Yr, dXr, dgr, bY, bdX, bdg = _oracle_all(case)
    assert_close("Y", host_f64_from_bf16(Y), Yr, bound=bY)
    assert_close("dX", host_f64_from_bf16(dX), dXr, bound=bdX)
    assert_close("dgate", dgate.cpu().numpy(), dgr, bound=bdg)


@pytest.mark.parametrize("T,d_in,d_out,g", [(200, 1024, 512, 256), (96, 512, 128, 64)])
def test_soft_mask_scales_groups(T, d_in, d_out, g):
    say(f"soft mask: T={T} d_in={d_in} d_out={d_out} g={g}")
    case = workloads.make_linear_case((201, T), T, d_in, d_out, g, None)
    r = workloads.gen.rng_for(202, T)
    soft = r.uniform(0.05, 1.5, size=case.mask.shape).astype(np.float32)
    soft[r.uniform(size=soft.shape) < 0.4] = 0.0
    d = _dev_case(case, soft)
    Y = _fwd(d, g)
    dX, dgate = _bwd(d, g)
    Yr, dXr, dgr, bY, bdX, bdg = _oracle_all(case, soft)
    assert_close("Y", host_f64_from_bf16(Y), Yr, bound=bY)
    assert_close("dX", host_f64_from_bf16(dX), dXr, bound=bdX)
    assert_close("dgate", dgate.cpu().numpy(), dgr, bound=bdg)


@pytest.mark.parametrize("where", ["first", "middle", "last"])
def test_soft_selectors_in_one_chunk_of_a_long_column(where):
    """Column lists are built per 1024-row chunk: a column whose only fractional
    selectors lie in one chunk (first, middle or last of three, the last one
    ragged) must still be marked soft, so that dX scales those rows."""
    T, d_in, d_out, g = 64, 512, 3000, 256
    say(f"soft selectors only in the {where} 1024-row chunk: T={T} d_in={d_in} d_out={d_out} g={g}")
    case = workloads.make_linear_case((231, T), T, d_in, d_out, g, None)
    m = case.mask.astype(np.float32).copy()
    lo = {"first": 0, "middle": 1024, "last": 2048}[where]
    rows = np.arange(lo + 5, min(lo + 1024, d_out), 97)
    m[rows, 0] = np.where(np.arange(rows.size) % 2, 0.5, 1.25).astype(np.float32)  # column 0 only
    d = _dev_case(case, m)
    dX, dgate = _bwd(d, g)
    Yr, dXr, dgr, bY, bdX, bdg = _oracle_all(case, m)
    assert_close("dX", host_f64_from_bf16(dX), dXr, bound=bdX)
    assert_close("dgate", dgate.cpu().numpy(), dgr, bound=bdg)


def test_all_ones_is_dense_and_all_zeros_is_exact_zero():
    import torch
    T, d_in, d_out, g = 256, 1024, 768, 256
    case = workloads.make_linear_case((203,), T, d_in, d_out, g, None)
    ones = np.ones_like(case.mask)
    zeros = np.zeros_like(case.mask)
    say("all-ones mask")
    d = _dev_case(case, ones)
    Y = _fwd(d, g)
    dX, _ = _bwd(d, g, want_dgate=False)
    Yr, dXr, _, bY, bdX, _ = _oracle_all(case, ones)
    assert_close("Y (dense)", host_f64_from_bf16(Y), Yr, bound=bY)
    assert_close("dX (dense)", host_f64_from_bf16(dX), dXr, bound=bdX)
    # the dense product of the same bf16 values in fp32
    ref32 = (d["X"].float() @ d["W"].float().t()).cpu().numpy()
    assert_close("Y vs fp32 dense product", host_f64_from_bf16(Y), ref32)
    say("all-zeros mask")
    d = _dev_case(case, zeros)
    Y = _fwd(d, g)
    dX, dgate = _bwd(d, g)
    assert not np.any(host_bits(Y) & 0x7FFF)
    assert not np.any(host_bits(dX) & 0x7FFF)
    _, _, dgr, _, _, bdg = _oracle_all(case, zeros)
    assert_close("dgate (all pruned)", dgate.cpu().numpy(), dgr, bound=bdg)
    del torch


@pytest.mark.parametrize("T,d_in,d_out,g", [(192, 1024, 512, 128), (64, 512, 3000, 256), (33, 1024, 2056, 64)])
def test_dgate_does_not_depend_on_mask_and_single_outputs(T, d_in, d_out, g):
    """dgate with or without dX and whatever the mask; dX alone (column lists
    from their own launch, dY^T from the transpose) equal to dX beside dgate
    (lists built by the dgate launch's spare blocks, dY^T its side output),
    also with several 1024-row list chunks and a ragged last one."""
    case = workloads.make_linear_case((204, d_out), T, d_in, d_out, g, None)
    say(f"dgate mask independence, dgate-only and dX-only calls: T={T} d_in={d_in} d_out={d_out} g={g}")
    d1 = _dev_case(case)
    d2 = _dev_case(case, np.ones_like(case.mask))
    _, g1 = _bwd(d1, g)
    _, g2 = _bwd(d2, g, want_dx=False)
    assert np.array_equal(g1.cpu().numpy(), g2.cpu().numpy())
    dX_only, _ = _bwd(d1, g, want_dgate=False)   # dY^T from the standalone transpose
    dX_both, _ = _bwd(d1, g)                     # dY^T from the dgate side output
    assert np.array_equal(host_bits(dX_only), host_bits(dX_both))


@pytest.mark.parametrize("T", [1, 3, 8, 16])
@pytest.mark.parametrize("g", [64, 256, 512])
def test_decode_forward(T, g):
    d_in, d_out = 2048, 328
    say(f"decode forward: T={T} g={g}")
    case = workloads.make_linear_case((205, T, g), T, d_in, d_out, g, None)
    d = _dev_case(case)
    Y = _fwd(d, g)
    Yr, _, _, bY, _, _ = _oracle_all(case)
    assert_close("Y", host_f64_from_bf16(Y), Yr, bound=bY)


@pytest.mark.parametrize("T,d_out,g_out", [(8, 12296, 1), (16, 12296, 1), (5, 12304, 16), (12, 12416, 64)])
def test_decode_four_row_tiles(T, d_out, g_out):
    # d_out / 64 >= 192 blocks: the MFMA decode path takes four 16-row tiles per
    # block; the last block holds 8, 16 or all 64 of its rows
    d_in = 1024
    g = 256 if g_out == 1 else g_out
    say(f"decode, four row tiles: T={T} d_out={d_out} groups {g_out}x{g}")
    case = workloads.make_linear_case((212, T, d_out, g_out), T, d_in, d_out, g, None, g_out=g_out)
    d = _dev_case(case)
    import paper_2609_33977_amd as gm
    Y = empty_bf16(T, d_out)
    gm.gm_masked_linear_fwd(d["X"], d["W"], d["mask"], g, Y, g_out=g_out)
    sync()
    Yr, bY = ref_fwd(oracle.from_bf16(case.X), oracle.from_bf16(case.W), case.mask, g, g_out)
    assert_close("Y", host_f64_from_bf16(Y), Yr, bound=bY)


def _pack(d, g):
    import torch
    import paper_2609_33977_amd as gm
    d_out, d_in = d["W"].shape
    cap = d_out * (d_in // g)
    Wp = torch.zeros(cap, g, dtype=torch.bfloat16, device="cuda")
    chunk = torch.full((cap,), -1, dtype=torch.int32, device="cuda")
    scale = torch.zeros(cap, dtype=torch.float32, device="cuda")
    rowptr = torch.zeros(d_out + 1, dtype=torch.int32, device="cuda")
    gm.gm_pack_rows(d["W"], d["mask"], g, cap, Wp, chunk, scale, rowptr)
    sync()
    return Wp, chunk, scale, rowptr


@pytest.mark.parametrize("g", [64, 128, 256, 512])
def test_pack_rows_is_exact(g):
    d_in, d_out = 2048, 200
    say(f"pack rows: g={g}")
    case = workloads.make_linear_case((206, g), 1, d_in, d_out, g, None)
    soft = case.mask * workloads.gen.rng_for(207, g).uniform(0.5, 1.5, size=case.mask.shape).astype(np.float32)
    d = _dev_case(case, soft)
    Wp, chunk, scale, rowptr = _pack(d, g)
    # expected export, built from the definition (row-major order of the kept groups)
    keep = soft != 0
    rp = np.concatenate([[0], np.cumsum(keep.sum(axis=1))]).astype(np.int32)
    o_idx, v_idx = np.nonzero(keep)
    k = rp[-1]
    assert np.array_equal(rowptr.cpu().numpy(), rp)
    assert np.array_equal(chunk.cpu().numpy()[:k], v_idx.astype(np.int32))
    assert np.array_equal(scale.cpu().numpy()[:k], soft[o_idx, v_idx])
    Wg = case.W.reshape(d_out, d_in // g, g)
    assert np.array_equal(host_bits(Wp)[:k], Wg[o_idx, v_idx])


@pytest.mark.parametrize("T", [1, 2, 8, 16, 40])
def test_packed_forward(T):
    d_in, d_out, g = 3072, 264, 256
    import paper_2609_33977_amd as gm
    say(f"packed forward: T={T}")
    case = workloads.make_linear_case((208, T), T, d_in, d_out, g, None)
    d = _dev_case(case)
    Wp, chunk, scale, rowptr = _pack(d, g)
    Y = empty_bf16(T, d_out)
    gm.gm_packed_linear_fwd(d["X"], Wp, chunk, scale, rowptr, d_out, g, Y)
    sync()
    Yr, _, _, bY, _, _ = _oracle_all(case)
    assert_close("Y", host_f64_from_bf16(Y), Yr, bound=bY)
    Y2 = _fwd(d, g)
    if T <= 16:  # one kernel reads both layouts (one token; 2-16 tokens on MFMA): identical results
        assert np.array_equal(host_bits(Y), host_bits(Y2))


@pytest.mark.parametrize("T,d_in,d_out,g", [
    (2, 2048, 200, 64),      # 32 groups per row, ragged last block (200 = 6 x 32 + 8 rows)
    (16, 4096, 72, 512),     # pieces of 512 weights, rows of 8 groups
    (7, 32768, 40, 64),      # 512 groups per row (the most a row may have): 16-row blocks, a 16 x 512 table
])
def test_packed_matches_in_place_at_2_to_16_tokens(T, d_in, d_out, g):
    import paper_2609_33977_amd as gm
    say(f"packed vs in place: T={T} d_in={d_in} d_out={d_out} g={g}")
    case = workloads.make_linear_case((217, T, d_in, g), T, d_in, d_out, g, None)
    d = _dev_case(case)
    Wp, chunk, scale, rowptr = _pack(d, g)
    Yp = empty_bf16(T, d_out)
    gm.gm_packed_linear_fwd(d["X"], Wp, chunk, scale, rowptr, d_out, g, Yp)
    sync()
    Yr, _, _, bY, _, _ = _oracle_all(case)
    assert_close("Y packed", host_f64_from_bf16(Yp), Yr, bound=bY)
    Yi = _fwd(d, g)
    assert_close("Y in place", host_f64_from_bf16(Yi), Yr, bound=bY)
    # both layouts on the MFMA kernel: the same products in the same order
    assert np.array_equal(host_bits(Yp), host_bits(Yi))


def test_workspace_too_small_is_rejected_without_launch():
    import paper_2609_33977_amd as gm
    T, d_in, d_out, g = 64, 512, 256, 256
    case = workloads.make_linear_case((209,), T, d_in, d_out, g, None)
    d = _dev_case(case)
    need = gm.gm_workspace_size(gm.GM_OP_BWD, T, d_in, d_out, g)
    small = workspace(need - 256)
    dX = empty_bf16(T, d_in)
    with pytest.raises(gm.GroupMaskError) as ei:
        gm.gm_masked_linear_bwd(d["dY"], d["X"], d["W"], d["mask"], g, dX, None, small)
    assert ei.value.status == gm.GM_ERR_WORKSPACE


@pytest.mark.parametrize("T,d_in,d_out,g", [
    (17, 64, 8, 64),          # smallest GEMM-path token count, one group column, eight output rows
    (300, 32768, 256, 64),    # 512 group columns per row: the forward's per-tile limit
    (16, 32768, 264, 64),     # the same row width on the decode path
    (40, 2048, 8, 512),       # a single 8-row tile row, groups spanning two dgate tiles
])
def test_edge_shapes(T, d_in, d_out, g):
    say(f"edge shape: T={T} d_in={d_in} d_out={d_out} g={g}")
    case = workloads.make_linear_case((210, T, d_in, d_out, g), T, d_in, d_out, g, None)
    d = _dev_case(case)
    Y = _fwd(d, g)
    Yr, dXr, dgr, bY, bdX, bdg = _oracle_all(case)
    assert_close("Y", host_f64_from_bf16(Y), Yr, bound=bY)
    if T > 16:
        dX, dgate = _bwd(d, g)
        assert_close("dX", host_f64_from_bf16(dX), dXr, bound=bdX)
        assert_close("dgate", dgate.cpu().numpy(), dgr, bound=bdg)


def test_decode_and_gemm_paths_agree_at_the_boundary():
    # T = 16 runs the GEMV, T = 17 the GEMM: the first 16 rows of the larger
    # batch must match the smaller batch's rows to rounding
    d_in, d_out, g = 1024, 256, 256
    case = workloads.make_linear_case((211,), 17, d_in, d_out, g, None)
    d17 = _dev_case(case)
    d16 = dict(d17, X=d17["X"][:16].contiguous())
    Y17 = host_f64_from_bf16(_fwd(d17, g))[:16]
    Y16 = host_f64_from_bf16(_fwd(d16, g))
    assert_close("Y (GEMV vs GEMM)", Y16, Y17, 1e-2)


@pytest.mark.parametrize("T", [1, 5, 16])
@pytest.mark.parametrize("g", [64, 256])
def test_decode_soft_selectors_in_place_and_packed(T, g):
    # fractional selectors (a group scaled by its mask value, skipped at 0) on
    # the decode paths: the one-token kernel (in place and packed) and the
    # 2-16 token MFMA kernel (in place), against the oracle
    d_in, d_out = 4096, 136
    say(f"decode soft selectors: T={T} g={g}")
    case = workloads.make_linear_case((213, T, g), T, d_in, d_out, g, None)
    r = workloads.gen.rng_for(214, T, g)
    soft = r.uniform(0.05, 1.5, size=case.mask.shape).astype(np.float32)
    soft[r.uniform(size=soft.shape) < 0.4] = 0.0
    d = _dev_case(case, soft)
    Yr, _, _, bY, _, _ = _oracle_all(case, soft)
    assert_close("Y in place", host_f64_from_bf16(_fwd(d, g)), Yr, bound=bY)
    import paper_2609_33977_amd as gm
    Wp, chunk, scale, rowptr = _pack(d, g)
    Yp = empty_bf16(T, d_out)
    gm.gm_packed_linear_fwd(d["X"], Wp, chunk, scale, rowptr, d_out, g, Yp)
    sync()
    assert_close("Y packed", host_f64_from_bf16(Yp), Yr, bound=bY)
    assert np.array_equal(host_bits(Yp), host_bits(_fwd(d, g))), "packed and in place differ"


@pytest.mark.parametrize("T", [2, 8, 16])
def test_decode_one_soft_selector_among_binary(T):
    # the 2-16 token kernel scales weights only in blocks whose staged
    # selectors include a fractional one: a binary mask with a single
    # fractional selector (row 333) mixes both kinds of block in one launch
    d_in, d_out, g = 4096, 640, 256
    say(f"decode one soft selector: T={T}")
    case = workloads.make_linear_case((216, T), T, d_in, d_out, g, None)
    m = case.mask.astype(np.float32).copy()
    m[333, 5] = 0.37
    d = _dev_case(case, m)
    Yr, _, _, bY, _, _ = _oracle_all(case, m)
    Y = host_f64_from_bf16(_fwd(d, g))
    assert_close("Y", Y, Yr, bound=bY)
    assert_close("Y row 333", Y[:, 333:334], Yr[:, 333:334], bound=bY[:, 333:334])


@pytest.mark.parametrize("T", [1, 8])
def test_decode_degenerate_rows(T):
    # rows with every group kept (64 groups: the one-token kernel's longest
    # in-place list), rows with none (exact zero outputs), rows with a single
    # kept group (first, last), and an all-zero mask
    d_in, d_out, g = 4096, 64, 64
    say(f"decode degenerate rows: T={T}")
    case = workloads.make_linear_case((215, T), T, d_in, d_out, g, None)
    m = case.mask.copy()
    m[0:8] = 1.0
    m[8:16] = 0.0
    m[16:24] = 0.0
    m[16:20, 0] = 1.0
    m[20:24, d_in // g - 1] = 1.0
    d = _dev_case(case, m)
    Y = _fwd(d, g)
    Yr, _, _, bY, _, _ = _oracle_all(case, m)
    assert_close("Y", host_f64_from_bf16(Y), Yr, bound=bY)
    assert not np.any(host_bits(Y)[:, 8:16] & 0x7FFF), "pruned rows must be exactly zero"
    zeros = np.zeros_like(m)
    Yz = _fwd(_dev_case(case, zeros), g)
    assert not np.any(host_bits(Yz) & 0x7FFF)


def test_stacked_linears_match_their_members():
    # linears that read one input (a layer's q, k and v) launched as one stacked linear: its Y is the members'
    # Y side by side and its dgate their dgate (bit for bit), and its dX the sum the shared input receives
    import torch
    T, d_in, g = 300, 1024, 256
    rows = (512, 384, 128)  # member boundaries on and off the 256-row tiles
    say(f"stacked linears: T={T} rows={rows}")
    cases = [workloads.make_linear_case((218, j), T, d_in, r, g, None) for j, r in enumerate(rows)]
    X = cases[0].X
    members = []
    for c in cases:
        d = _dev_case(c)
        d["X"] = dev_bf16(X)
        members.append(d)
    import paper_2609_33977_amd as gm

    def fwd_unsplit(d):  # no workspace: K is not split, so the two tilings sum each element in one order
        Y = empty_bf16(T, d["W"].shape[0])
        gm.gm_masked_linear_fwd(d["X"], d["W"], d["mask"], g, Y)
        sync()
        return Y
    Ys = [fwd_unsplit(d) for d in members]
    bw = [_bwd(d, g) for d in members]
    stack = dict(X=dev_bf16(X), W=torch.cat([d["W"] for d in members]), mask=torch.cat([d["mask"] for d in members]),
                 dY=torch.cat([d["dY"] for d in members], dim=1).contiguous())
    Y = fwd_unsplit(stack)
    dX, dgate = _bwd(stack, g)
    assert torch.equal(Y, torch.cat(Ys, dim=1))
    assert torch.equal(dgate, torch.cat([b[1] for b in bw]))
    m = np.concatenate([c.mask for c in cases])
    W = np.concatenate([oracle.from_bf16(c.W) for c in cases])
    dY = np.concatenate([oracle.from_bf16(c.dY) for c in cases], axis=1)
    ref, bnd = ref_dx(dY, W, m, g)
    assert_close("dX (stack)", host_f64_from_bf16(dX), ref, bound=bnd)
    # the members' dX summed in fp32 agree with it to their bf16 rounding
    summed = sum(host_f64_from_bf16(b[0]) for b in bw)
    assert_close("dX (sum of members)", summed, ref, tol=1e-2)


def test_debug_sync_mode_gives_the_same_results(tmp_path):
    # GM_DEBUG is read once per process: a child process runs the same forward and
    # backward with a device synchronisation and error check after every launch
    import os
    import subprocess
    import sys
    T, d_in, d_out, g = 200, 1024, 512, 256
    say("GM_DEBUG=sync in a child process")
    case = workloads.make_linear_case((219,), T, d_in, d_out, g, None)
    d = _dev_case(case)
    Y = host_bits(_fwd(d, g))
    dX, dgate = _bwd(d, g)
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    out = tmp_path / "child.npz"
    code = f"""
import sys
sys.path[:0] = [{root!r}, {os.path.join(root, 'tests')!r}]
import numpy as np, workloads, test_gpu_linear as t
case = workloads.make_linear_case((219,), {T}, {d_in}, {d_out}, {g}, None)
d = t._dev_case(case)
Y = t.host_bits(t._fwd(d, {g}))
dX, dgate = t._bwd(d, {g})
np.savez({str(out)!r}, Y=Y, dX=t.host_bits(dX), dgate=dgate.cpu().numpy())
"""
    env = dict(os.environ, GM_DEBUG="sync")
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, r.stderr[-2000:]
    got = np.load(out)
    assert np.array_equal(got["Y"], Y)
    assert np.array_equal(got["dX"], host_bits(dX))
    assert np.array_equal(got["dgate"], dgate.cpu().numpy())
