"""GPU parity at the largest sizes the library accepts: every GEMM addresses
a matrix with 32-bit byte offsets, so W may hold at most 2^30 - 2^22 bf16
elements (just under 2 GiB); W [32640, 32768] is exactly that.  The forward
(GEMM and decode paths, in place and packed), dX and dgate are checked against
the fp64 oracle on sampled output rows (forward, dgate) and sampled group
columns (dX); one row more is rejected before any launch."""
import numpy as np
import pytest

import oracle
import workloads
from workloads.gen import rng_for
from gpu_support import (assert_close, assert_dgate, assert_dx, assert_fwd, empty_bf16, empty_f32, host_bits, ref_fwd,
                         say, sync, workspace)

pytestmark = pytest.mark.gpu

D_OUT, D_IN, G = 32640, 32768, 256   # D_OUT * D_IN == 2^30 - 2^22


@pytest.fixture(scope="module")
def big():
    import torch
    assert D_OUT * D_IN == (1 << 30) - (1 << 22)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(workloads.SEED + 500)
    W = torch.empty(D_OUT, D_IN, dtype=torch.bfloat16, device="cuda")
    for r0 in range(0, D_OUT, 4096):  # fp32 draws in slices: a few hundred MB at a time
        r1 = min(D_OUT, r0 + 4096)
        W[r0:r1] = (torch.randn(r1 - r0, D_IN, device="cuda", generator=gen) * 0.02).to(torch.bfloat16)
    Gn = D_OUT * (D_IN // G)
    m = torch.zeros(Gn, device="cuda")
    m[torch.randperm(Gn, device="cuda", generator=gen)[: Gn // 2]] = 1.0
    m = m.view(D_OUT, D_IN // G)
    sync()
    yield dict(W=W, mask=m, gen=gen)
    del W, m
    torch.cuda.empty_cache()


def _rows_host(d, rows):
    import torch
    idx = torch.as_tensor(rows, device="cuda")
    return oracle.from_bf16(host_bits(d["W"][idx])), d["mask"][idx].cpu().numpy()


def _x(d, T):
    import torch
    return torch.randn(T, D_IN, device="cuda", generator=d["gen"]).to(torch.bfloat16)


def test_largest_matrix_forward_and_backward(big):
    import torch
    import paper_2609_33977_amd as gm
    T = 40
    say(f"largest W [{D_OUT}, {D_IN}]: fwd, dX, dgate at T={T}")
    X = _x(big, T)
    dY = torch.randn(T, D_OUT, device="cuda", generator=big["gen"]).to(torch.bfloat16)
    Y = empty_bf16(T, D_OUT)
    wsf = workspace(gm.gm_workspace_size(gm.GM_OP_FWD, T, D_IN, D_OUT, G))
    gm.gm_masked_linear_fwd(X, big["W"], big["mask"], G, Y, wsf)
    dX = empty_bf16(T, D_IN)
    dgate = empty_f32(D_OUT, D_IN // G)
    wsb = workspace(gm.gm_workspace_size(gm.GM_OP_BWD, T, D_IN, D_OUT, G))
    gm.gm_masked_linear_bwd(dY, X, big["W"], big["mask"], G, dX, dgate, wsb)
    sync()
    rows = np.sort(rng_for(500, 1).choice(D_OUT, 96, replace=False))
    rows[-1] = D_OUT - 1  # the last row touches the end of the addressable range
    Wr, mr = _rows_host(big, rows)
    Xo, dYo = oracle.from_bf16(host_bits(X)), oracle.from_bf16(host_bits(dY))
    assert_fwd("Y (sampled rows)", oracle.from_bf16(host_bits(Y))[:, rows], Xo, Wr, mr, G)
    assert_dgate("dgate (sampled rows)", dgate.cpu().numpy()[rows], dYo[:, rows], Xo, Wr, G)
    # dX on two group columns (the first and the last): all rows of W over those columns
    for v in (0, D_IN // G - 1):
        cols = slice(v * G, (v + 1) * G)
        Wc = oracle.from_bf16(host_bits(big["W"][:, cols].contiguous()))
        mc = big["mask"][:, v: v + 1].cpu().numpy()
        assert_dx(f"dX (group column {v})", oracle.from_bf16(host_bits(dX))[:, cols], dYo, Wc, mc, G)


def test_largest_matrix_decode_in_place_and_packed(big):
    import torch
    import paper_2609_33977_amd as gm
    say(f"largest W [{D_OUT}, {D_IN}]: one-token decode, in place and packed")
    x = _x(big, 1)
    Y = empty_bf16(1, D_OUT)
    gm.gm_masked_linear_fwd(x, big["W"], big["mask"], G, Y)
    cap = D_OUT * (D_IN // G) // 2  # exactly the kept groups: rowptr[-1] must equal it
    Wp = torch.empty(cap, G, dtype=torch.bfloat16, device="cuda")
    chunk = torch.empty(cap, dtype=torch.int32, device="cuda")
    scale = torch.empty(cap, dtype=torch.float32, device="cuda")
    rowptr = torch.empty(D_OUT + 1, dtype=torch.int32, device="cuda")
    gm.gm_pack_rows(big["W"], big["mask"], G, cap, Wp, chunk, scale, rowptr)
    Yp = empty_bf16(1, D_OUT)
    gm.gm_packed_linear_fwd(x, Wp, chunk, scale, rowptr, D_OUT, G, Yp)
    sync()
    assert int(rowptr[-1].item()) == cap
    rows = np.sort(rng_for(500, 2).choice(D_OUT, 128, replace=False))
    rows[-1] = D_OUT - 1
    Wr, mr = _rows_host(big, rows)
    ref, b = ref_fwd(oracle.from_bf16(host_bits(x)), Wr, mr, G)
    assert_close("Y in place (sampled rows)", oracle.from_bf16(host_bits(Y))[:, rows], ref, bound=b)
    assert_close("Y packed (sampled rows)", oracle.from_bf16(host_bits(Yp))[:, rows], ref, bound=b)
    del Wp


def test_one_row_past_the_limit_is_rejected():
    import torch
    import paper_2609_33977_amd as gm
    assert gm.LIB.gm_workspace_size(gm.GM_OP_FWD, 40, D_IN, D_OUT + 8, G, 1,
                                    __import__("ctypes").byref(__import__("ctypes").c_size_t())) == gm.GM_ERR_SHAPE
    X = torch.zeros(1, D_IN, dtype=torch.bfloat16, device="cuda")
    W = torch.zeros(8, D_IN, dtype=torch.bfloat16, device="cuda")  # never read: rejected on its declared shape
    m = torch.zeros(8, D_IN // G, device="cuda")
    Y = empty_bf16(1, D_OUT + 8)
    st = gm.LIB.gm_masked_linear_fwd(X.data_ptr(), W.data_ptr(), m.data_ptr(), 1, D_IN, D_OUT + 8, G, 1,
                                     Y.data_ptr(), None, 0, None)
    assert st == gm.GM_ERR_SHAPE


def test_longest_token_batch_forward_and_backward():
    # the token dimension at the same limit: X and dX [32640, 32768] hold
    # 2^30 - 2^22 elements each (T a multiple of 8, so the padded dY^T rows
    # of the backward stay inside the limit too); a narrow W keeps the
    # products small.  Sampled tokens for Y and dX, sampled groups for dgate.
    import torch
    import paper_2609_33977_amd as gm
    T, d_in, d_out, g = 32640, 32768, 256, 256
    say(f"longest token batch: X [{T}, {d_in}], W [{d_out}, {d_in}]")
    gen = torch.Generator(device="cuda")
    gen.manual_seed(workloads.SEED + 501)
    X = torch.empty(T, d_in, dtype=torch.bfloat16, device="cuda")
    for r0 in range(0, T, 4096):
        r1 = min(T, r0 + 4096)
        X[r0:r1] = torch.randn(r1 - r0, d_in, device="cuda", generator=gen).to(torch.bfloat16)
    W = (torch.randn(d_out, d_in, device="cuda", generator=gen) * 0.02).to(torch.bfloat16)
    dY = torch.randn(T, d_out, device="cuda", generator=gen).to(torch.bfloat16)
    Gn = d_out * (d_in // g)
    m = torch.zeros(Gn, device="cuda")
    m[torch.randperm(Gn, device="cuda", generator=gen)[: Gn // 2]] = 1.0
    m = m.view(d_out, d_in // g)
    Y = empty_bf16(T, d_out)
    gm.gm_masked_linear_fwd(X, W, m, g, Y, workspace(gm.gm_workspace_size(gm.GM_OP_FWD, T, d_in, d_out, g)))
    dX = empty_bf16(T, d_in)
    dgate = empty_f32(d_out, d_in // g)
    gm.gm_masked_linear_bwd(dY, X, W, m, g, dX, dgate, workspace(gm.gm_workspace_size(gm.GM_OP_BWD, T, d_in, d_out, g)))
    sync()
    Wo, mo = oracle.from_bf16(host_bits(W)), m.cpu().numpy()
    toks = np.sort(rng_for(501, 1).choice(T, 48, replace=False))
    toks[-1] = T - 1  # the last token touches the end of X's and dX's addressable range
    idx = torch.as_tensor(toks, device="cuda")
    Xs, dYs = oracle.from_bf16(host_bits(X[idx])), oracle.from_bf16(host_bits(dY[idx]))
    assert_fwd("Y (sampled tokens)", oracle.from_bf16(host_bits(Y[idx])), Xs, Wo, mo, g)
    assert_dx("dX (sampled tokens)", oracle.from_bf16(host_bits(dX[idx])), dYs, Wo, mo, g)
    dYo = oracle.from_bf16(host_bits(dY))
    for v in (0, d_in // g - 1):  # every token, two group columns (all rows of W)
        cols = slice(v * g, (v + 1) * g)
        Xc = oracle.from_bf16(host_bits(X[:, cols].contiguous()))
        assert_dgate(f"dgate (group column {v})", dgate.cpu().numpy()[:, v: v + 1], dYo, Xc, Wo[:, cols], g)
    del X, dX
    torch.cuda.empty_cache()
