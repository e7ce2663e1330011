"""The C-ABI library loads, exports every declared entry point, and rejects bad
arguments before touching any device (no compute call here: no GPU needed)."""
import ctypes
import os
import re

import pytest

import paper_2609_33977_amd as gm

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "groupmask.h")

FAKE = ctypes.c_void_p(1 << 20)      # non-NULL, 16-byte aligned; never dereferenced on the error paths used
MISALIGNED = ctypes.c_void_p((1 << 20) + 4)


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gm_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    declared = _declared_functions()
    assert declared, "no declarations parsed"
    assert sorted(gm.EXPORTS) == declared
    for name in declared:
        assert hasattr(gm.LIB, name), name


def test_abi_version_and_status_strings():
    assert gm.gm_abi_version() == 3
    for s in range(7):
        assert gm.status_string(s)
    assert gm.status_string(99) == "unknown status"


def test_workspace_size_host_only():
    ws = gm.gm_workspace_size(gm.GM_OP_BWD, 4096, 4096, 4096, 256)
    # per-column counts and soft flags, then row lists and scales (each with
    # 128 entries of look-ahead padding), then dY^T; every part rounded up to
    # 256 bytes
    G_in = 4096 // 256
    r256 = lambda x: (x + 255) // 256 * 256
    expect = 2 * r256(G_in * 4) + 2 * r256((G_in * 4096 + 128) * 4) + r256(4096 * 4096 * 2)
    assert ws == expect
    assert gm.gm_workspace_size(gm.GM_OP_FWD, 4096, 4096, 4096, 256) == 0
    # ragged T: dY^T rows padded to a multiple of 8 tokens
    assert gm.gm_workspace_size(gm.GM_OP_BWD, 77, 320, 200, 64) > 200 * 80 * 2


@pytest.mark.parametrize("g,nsub", [(16, 4), (32, 2), (64, 1), (128, 1)])
def test_workspace_size_square_groups(g, nsub):
    # list columns of max(g, 64) input columns with nsub groups each: one
    # scale per group and entry, and kept bits per entry when nsub > 1
    T, d_in, d_out = 1000, 4096, 2048
    NL = d_in // max(g, 64)
    r256 = lambda x: (x + 255) // 256 * 256
    lst = NL * d_out + 128
    expect = (2 * r256(NL * 4) + r256(lst * 4) + r256(lst * nsub * 4) + (r256(lst * 4) if nsub > 1 else 0)
              + r256(d_out * 1000 * 2))
    assert gm.gm_workspace_size(gm.GM_OP_BWD, T, d_in, d_out, g, g) == expect
    # 4 x 8 output tiles: the forward splits K over 8 shares
    assert gm.gm_workspace_size(gm.GM_OP_FWD, T, d_in, d_out, g, g) == _fwd_split_bytes(T, d_in, d_out, g)
    assert gm.gm_workspace_size(gm.GM_OP_FWD, T, d_in, d_out, g, g) == r256(8 * T * d_out * 4)


def _fwd_split_bytes(T, d_in, d_out, g):
    """The documented rule: at most 128 output tiles of 256 x 256 (and T > 16) split K into
    min(256 // tiles, 8, units // 4) shares of fp32 partial tiles (units // 1 with at most 16 tiles);
    units of max(g, 32) columns."""
    if T <= 16:
        return 0
    tiles = -(-T // 256) * -(-d_out // 256)
    if tiles > 128:
        return 0
    ks = min(256 // tiles, 8, d_in // max(g, 32) // (1 if tiles <= 16 else 4))
    return 0 if ks <= 1 else (ks * T * d_out * 4 + 255) // 256 * 256


@pytest.mark.parametrize("T,d_in,d_out,g,expect", [
    (4096, 4096, 4096, 256, 0),                       # 256 tiles: unsplit
    (16, 5120, 5120, 256, 0),                         # decode path
    (512, 5120, 5120, 256, 5 * 512 * 5120 * 4),       # 40 tiles, 20 units: 5 shares
    (512, 5120, 13824, 256, 2 * 512 * 13824 * 4),     # 108 tiles: 2 shares
    (512, 13824, 5120, 256, 6 * 512 * 5120 * 4),
    (2048, 4096, 4096, 256, 2 * 2048 * 4096 * 4),     # 128 tiles: 2 shares
    (2048, 4096, 4352, 256, 0),                       # 136 tiles: unsplit
    (17, 4096, 4096, 256, 8 * 17 * 4096 * 4),         # 16 tiles, 16 units: 8 shares of two
    (128, 1024, 1024, 256, 4 * 128 * 1024 * 4),       # 4 tiles, 4 units: one unit per share
    (300, 2048, 1024, 512, 4 * 300 * 1024 * 4),       # 8 tiles, 4 units
    (520, 2048, 4608, 512, 0),                        # 54 tiles, 4 units: a share would hold fewer than four
    (520, 8192, 4608, 512, 4 * 520 * 4608 * 4),
])
def test_forward_split_workspace(T, d_in, d_out, g, expect):
    assert gm.gm_workspace_size(gm.GM_OP_FWD, T, d_in, d_out, g) == expect == _fwd_split_bytes(T, d_in, d_out, g)


@pytest.mark.parametrize("args,code", [
    ((4096, 4096, 4096, 100, 1), gm.GM_ERR_SHAPE),     # group size not supported
    ((4096, 4000, 4096, 256, 1), gm.GM_ERR_SHAPE),     # d_in not a multiple of g
    ((0, 4096, 4096, 256, 1), gm.GM_ERR_SHAPE),        # empty T
    ((16, 4096, 4092, 256, 1), gm.GM_ERR_SHAPE),       # d_out not a multiple of 8
    ((16, 64 * 1024, 64, 64, 1), gm.GM_ERR_SHAPE),     # more than 512 group columns
    ((16, 4096, 4096, 16, 1), gm.GM_ERR_SHAPE),        # 1 x 16 is not a built shape
    ((16, 4096, 4096, 32, 16), gm.GM_ERR_SHAPE),       # not square
    ((16, 4096, 4096, 256, 256), gm.GM_ERR_SHAPE),     # square groups stop at 128
    ((16, 4096 + 32, 4096, 16, 16), gm.GM_ERR_SHAPE),  # 16 x 16 needs d_in a multiple of 64
    ((16, 4096, 4096 + 8, 16, 16), gm.GM_ERR_SHAPE),   # d_out not a multiple of g_out
    ((16, 16384 + 64, 64, 16, 16), gm.GM_ERR_SHAPE),   # more than 512 units of 32 columns
    ((16, 4096, 4096, 64, 0), gm.GM_ERR_SHAPE),
])
def test_workspace_size_rejects_bad_shapes(args, code):
    out = ctypes.c_size_t(0)
    assert gm.LIB.gm_workspace_size(gm.GM_OP_BWD, *args, ctypes.byref(out)) == code


@pytest.mark.parametrize("args", [(16, 16384, 64, 16, 16), (16, 11008, 4096, 16, 16), (16, 11008, 4096, 32, 32),
                                  (16, 4096, 4096, 128, 128), (1, 64, 128, 64, 64)])
def test_workspace_size_accepts_square_groups(args):
    out = ctypes.c_size_t(0)
    assert gm.LIB.gm_workspace_size(gm.GM_OP_BWD, *args, ctypes.byref(out)) == gm.GM_OK


def test_workspace_size_rejects_bad_op_and_null():
    out = ctypes.c_size_t(0)
    assert gm.LIB.gm_workspace_size(7, 16, 256, 256, 256, 1, ctypes.byref(out)) == gm.GM_ERR_VALUE
    assert gm.LIB.gm_workspace_size(gm.GM_OP_FWD, 16, 256, 256, 256, 1, None) == gm.GM_ERR_NULL


def test_gate_argument_errors():
    L = gm.LIB
    assert L.gm_gate(None, None, 16, 0.5, 1, FAKE, None, None) == gm.GM_ERR_NULL
    assert L.gm_gate(FAKE, None, 16, 0.5, 1, None, None, None) == gm.GM_ERR_NULL
    assert L.gm_gate(FAKE, None, -1, 0.5, 1, FAKE, None, None) == gm.GM_ERR_SHAPE
    assert L.gm_gate(FAKE, None, 16, 0.0, 1, FAKE, None, None) == gm.GM_ERR_VALUE
    assert L.gm_gate(FAKE, None, 16, -1.0, 1, FAKE, None, None) == gm.GM_ERR_VALUE
    assert L.gm_gate(FAKE, None, 16, float("nan"), 1, FAKE, None, None) == gm.GM_ERR_VALUE
    assert L.gm_gate(FAKE, None, 16, float("inf"), 1, FAKE, None, None) == gm.GM_ERR_VALUE
    assert L.gm_gate(FAKE, None, 16, 0.5, 2, FAKE, None, None) == gm.GM_ERR_VALUE
    assert L.gm_gate(MISALIGNED, None, 16, 0.5, 1, FAKE, None, None) == gm.GM_ERR_ALIGN
    assert L.gm_gate(FAKE, MISALIGNED, 16, 0.5, 1, FAKE, None, None) == gm.GM_ERR_ALIGN
    assert L.gm_gate(FAKE, None, 16, 0.5, 1, FAKE, MISALIGNED, None) == gm.GM_ERR_ALIGN
    # n == 0 is a no-op that succeeds without a device
    assert L.gm_gate(FAKE, None, 0, 0.5, 1, FAKE, None, None) == gm.GM_OK


def test_gate_bwd_argument_errors():
    L = gm.LIB
    assert L.gm_gate_bwd(None, FAKE, 8, 0.4, FAKE, None) == gm.GM_ERR_NULL
    assert L.gm_gate_bwd(FAKE, None, 8, 0.4, FAKE, None) == gm.GM_ERR_NULL
    assert L.gm_gate_bwd(FAKE, FAKE, 8, 0.4, None, None) == gm.GM_ERR_NULL
    assert L.gm_gate_bwd(FAKE, FAKE, -3, 0.4, FAKE, None) == gm.GM_ERR_SHAPE
    assert L.gm_gate_bwd(FAKE, FAKE, 8, 0.0, FAKE, None) == gm.GM_ERR_VALUE
    assert L.gm_gate_bwd(FAKE, FAKE, 8, 0.4, MISALIGNED, None) == gm.GM_ERR_ALIGN
    assert L.gm_gate_bwd(FAKE, FAKE, 0, 0.4, FAKE, None) == gm.GM_OK


def test_budget_argument_errors():
    L = gm.LIB
    ODD8 = ctypes.c_void_p(FAKE.value + 4)  # 4-byte but not 8-byte aligned
    ok = (FAKE, 64, FAKE, FAKE, 3, 0.5, 16.0, 0, FAKE, FAKE, FAKE, None)

    def call(**kw):
        names = ("mask", "n", "offsets", "params", "L", "s_t", "lam", "uniform", "kept", "loss", "coeff", "stream")
        args = dict(zip(names, ok))
        args.update(kw)
        return L.gm_budget_loss(*[args[k] for k in names])

    for k in ("mask", "offsets", "params", "kept", "loss", "coeff"):
        assert call(**{k: None}) == gm.GM_ERR_NULL, k
    assert call(n=0) == gm.GM_ERR_SHAPE
    assert call(L=0) == gm.GM_ERR_SHAPE
    for st in (0.0, 1.0, -0.2, float("nan")):
        assert call(s_t=st) == gm.GM_ERR_VALUE, st
    for lam in (-1.0, float("inf"), float("nan")):
        assert call(lam=lam) == gm.GM_ERR_VALUE, lam
    assert call(uniform=2) == gm.GM_ERR_VALUE
    assert call(mask=MISALIGNED) == gm.GM_ERR_ALIGN
    for k in ("offsets", "params", "kept", "loss"):
        assert call(**{k: ODD8}) == gm.GM_ERR_ALIGN, k

    bwd = L.gm_gate_bwd_budget
    assert bwd(None, FAKE, 8, 0.4, FAKE, 2, FAKE, FAKE, None) == gm.GM_ERR_NULL
    assert bwd(FAKE, FAKE, 8, 0.4, None, 2, FAKE, FAKE, None) == gm.GM_ERR_NULL
    assert bwd(FAKE, FAKE, 8, 0.4, FAKE, 2, None, FAKE, None) == gm.GM_ERR_NULL
    assert bwd(FAKE, FAKE, 0, 0.4, FAKE, 2, FAKE, FAKE, None) == gm.GM_ERR_SHAPE
    assert bwd(FAKE, FAKE, 8, 0.4, FAKE, 0, FAKE, FAKE, None) == gm.GM_ERR_SHAPE
    assert bwd(FAKE, FAKE, 8, 0.0, FAKE, 2, FAKE, FAKE, None) == gm.GM_ERR_VALUE
    assert bwd(FAKE, FAKE, 8, 0.4, FAKE, 2, FAKE, MISALIGNED, None) == gm.GM_ERR_ALIGN
    assert bwd(FAKE, FAKE, 8, 0.4, ODD8, 2, FAKE, FAKE, None) == gm.GM_ERR_ALIGN


def test_linear_argument_errors():
    L = gm.LIB
    fwd = L.gm_masked_linear_fwd
    assert fwd(None, FAKE, FAKE, 16, 256, 256, 256, 1, FAKE, None, 0, None) == gm.GM_ERR_NULL
    assert fwd(FAKE, FAKE, None, 16, 256, 256, 256, 1, FAKE, None, 0, None) == gm.GM_ERR_NULL
    assert fwd(FAKE, FAKE, FAKE, 16, 256, 256, 96, 1, FAKE, None, 0, None) == gm.GM_ERR_SHAPE
    assert fwd(FAKE, FAKE, FAKE, 0, 256, 256, 256, 1, FAKE, None, 0, None) == gm.GM_ERR_SHAPE
    assert fwd(FAKE, FAKE, FAKE, 16, 256, 250, 256, 1, FAKE, None, 0, None) == gm.GM_ERR_SHAPE
    assert fwd(FAKE, FAKE, FAKE, 16, 256, 256, 256, 2, FAKE, None, 0, None) == gm.GM_ERR_SHAPE
    assert fwd(FAKE, FAKE, FAKE, 16, 256, 264, 16, 16, FAKE, None, 0, None) == gm.GM_ERR_SHAPE
    assert fwd(FAKE, MISALIGNED, FAKE, 16, 256, 256, 256, 1, FAKE, None, 0, None) == gm.GM_ERR_ALIGN
    assert fwd(FAKE, FAKE, MISALIGNED, 16, 256, 256, 32, 32, FAKE, None, 0, None) == gm.GM_ERR_ALIGN
    # a workspace, when given, must be aligned and at least the split size
    need = gm.gm_workspace_size(gm.GM_OP_FWD, 512, 2048, 1024, 256)
    assert need > 0
    assert fwd(FAKE, FAKE, FAKE, 512, 2048, 1024, 256, 1, FAKE, FAKE, need - 1, None) == gm.GM_ERR_WORKSPACE
    assert fwd(FAKE, FAKE, FAKE, 512, 2048, 1024, 256, 1, FAKE, MISALIGNED, need, None) == gm.GM_ERR_ALIGN

    bwd = L.gm_masked_linear_bwd
    # dX requested without a mask
    assert bwd(FAKE, FAKE, FAKE, None, 16, 256, 256, 256, 1, FAKE, None, FAKE, 1 << 30, None) == gm.GM_ERR_NULL
    assert bwd(None, FAKE, FAKE, FAKE, 16, 256, 256, 256, 1, FAKE, FAKE, FAKE, 1 << 30, None) == gm.GM_ERR_NULL
    # both outputs NULL: nothing to do
    assert bwd(FAKE, FAKE, FAKE, FAKE, 16, 256, 256, 256, 1, None, None, None, 0, None) == gm.GM_OK
    assert bwd(FAKE, FAKE, FAKE, FAKE, 16, 256, 256, 16, 32, None, None, None, 0, None) == gm.GM_ERR_SHAPE
    # dX needs the workspace
    need = gm.gm_workspace_size(gm.GM_OP_BWD, 16, 256, 256, 256)
    assert bwd(FAKE, FAKE, FAKE, FAKE, 16, 256, 256, 256, 1, FAKE, None, None, 0, None) == gm.GM_ERR_WORKSPACE
    assert bwd(FAKE, FAKE, FAKE, FAKE, 16, 256, 256, 256, 1, FAKE, None, FAKE, need - 1, None) == gm.GM_ERR_WORKSPACE
    assert bwd(FAKE, FAKE, FAKE, FAKE, 16, 256, 256, 256, 1, FAKE, None, MISALIGNED, need, None) == gm.GM_ERR_ALIGN
    assert bwd(FAKE, FAKE, FAKE, FAKE, 16, 256, 512, 256, 1, FAKE, MISALIGNED, FAKE, need, None) == gm.GM_ERR_ALIGN
    need16 = gm.gm_workspace_size(gm.GM_OP_BWD, 16, 256, 256, 16, 16)
    assert need16 > need
    assert bwd(FAKE, FAKE, FAKE, FAKE, 16, 256, 256, 16, 16, FAKE, None, FAKE, need16 - 1, None) == gm.GM_ERR_WORKSPACE


def test_pack_argument_errors():
    L = gm.LIB
    assert L.gm_pack_rows(FAKE, FAKE, 256, 16, 256, 1, 16, FAKE, FAKE, None, FAKE, None) == gm.GM_ERR_NULL
    assert L.gm_pack_rows(FAKE, FAKE, 256, 16, 256, 1, 17, FAKE, FAKE, FAKE, FAKE, None) == gm.GM_ERR_SHAPE
    assert L.gm_pack_rows(FAKE, FAKE, 256, 16, 256, 1, -1, FAKE, FAKE, FAKE, FAKE, None) == gm.GM_ERR_SHAPE
    assert L.gm_pack_rows(FAKE, FAKE, 256, 16, 32, 32, 1, FAKE, FAKE, FAKE, FAKE, None) == gm.GM_ERR_SHAPE
    assert L.gm_pack_rows(FAKE, FAKE, 256, 16, 32, 16, 1, FAKE, FAKE, FAKE, FAKE, None) == gm.GM_ERR_SHAPE
    assert L.gm_packed_linear_fwd(FAKE, FAKE, FAKE, FAKE, None, 1, 256, 16, 256, FAKE, None) == gm.GM_ERR_NULL
    assert L.gm_packed_linear_fwd(FAKE, FAKE, FAKE, FAKE, FAKE, 1, 200, 16, 256, FAKE, None) == gm.GM_ERR_SHAPE


def test_distill_workspace_size():
    N, d, V = 4096, 4096, 32000
    r256 = lambda x: (x + 255) // 256 * 256
    tiles = (V + 255) // 256
    ldv = (V + 31) // 32 * 32
    expect = 2 * r256(N * V * 4) + r256(5 * tiles * N * 4) + 4 * r256(N * 4) + r256(N * ldv * 2)
    assert gm.gm_distill_workspace_size(N, d, V) == expect
    assert gm.gm_distill_workspace_size(77, 96, 1000) > 77 * 1000 * 8


@pytest.mark.parametrize("N,d,V", [(0, 256, 1000), (16, 48, 1000), (16, 16, 1000), (16, 256, 1004), (16, 256, 0),
                                   (16, 65536 + 32, 64), (16, 64, (1 << 20) + 8), (1 << 20, 2048, 64)])
def test_distill_rejects_bad_shapes(N, d, V):
    out = ctypes.c_size_t(0)
    assert gm.LIB.gm_distill_workspace_size(N, d, V, ctypes.byref(out)) == gm.GM_ERR_SHAPE


def test_distill_argument_errors():
    L = gm.LIB
    need = gm.gm_distill_workspace_size(16, 256, 1000)
    fwd = L.gm_distill_fwd
    assert fwd(None, FAKE, FAKE, None, 16, 256, 1000, FAKE, None, FAKE, need, None) == gm.GM_ERR_NULL
    assert fwd(FAKE, FAKE, FAKE, None, 16, 256, 1000, None, None, FAKE, need, None) == gm.GM_ERR_NULL
    assert fwd(FAKE, FAKE, FAKE, None, 16, 256, 1000, FAKE, None, None, need, None) == gm.GM_ERR_NULL
    assert fwd(FAKE, FAKE, FAKE, None, 16, 250, 1000, FAKE, None, FAKE, need, None) == gm.GM_ERR_SHAPE
    assert fwd(FAKE, MISALIGNED, FAKE, None, 16, 256, 1000, FAKE, None, FAKE, need, None) == gm.GM_ERR_ALIGN
    odd = ctypes.c_void_p(FAKE.value + 2)
    assert fwd(FAKE, FAKE, FAKE, None, 16, 256, 1000, odd, None, FAKE, need, None) == gm.GM_ERR_ALIGN
    assert fwd(FAKE, FAKE, FAKE, None, 16, 256, 1000, FAKE, None, FAKE, need - 1, None) == gm.GM_ERR_WORKSPACE
    bwd = L.gm_distill_bwd
    assert bwd(None, 16, 256, 1000, FAKE, FAKE, need, None) == gm.GM_ERR_NULL
    assert bwd(FAKE, 16, 256, 1000, None, FAKE, need, None) == gm.GM_ERR_NULL
    assert bwd(FAKE, 16, 256, 1001, FAKE, FAKE, need, None) == gm.GM_ERR_SHAPE
    assert bwd(FAKE, 16, 256, 1000, MISALIGNED, FAKE, need, None) == gm.GM_ERR_ALIGN
    assert bwd(FAKE, 16, 256, 1000, FAKE, FAKE, need - 256, None) == gm.GM_ERR_WORKSPACE


def test_hyper_workspace_and_argument_errors():
    L = gm.LIB
    need = gm.gm_hyper_workspace_size(224, 64, 64, 25296896)
    chunks = -(-25296896 // 2048) + 224
    assert need > chunks * 128 * 4  # the chunk partials of do dominate
    out = ctypes.c_size_t(0)
    for args in ((0, 64, 64, 100), (4, 0, 64, 100), (4, 64, 48, 100), (4, 64, 64, 0), (70000, 64, 64, 100)):
        assert L.gm_hyper_workspace_size(*args, ctypes.byref(out)) == gm.GM_ERR_SHAPE, args
    ws = gm.gm_hyper_workspace_size(4, 8, 32, 100)
    fwd = L.gm_hyper_fwd
    assert fwd(FAKE, FAKE, FAKE, FAKE, None, 4, 8, 32, 100, FAKE, FAKE, ws, None) == gm.GM_ERR_NULL
    assert fwd(FAKE, FAKE, MISALIGNED, FAKE, FAKE, 4, 8, 32, 100, FAKE, FAKE, ws, None) == gm.GM_ERR_ALIGN
    assert fwd(FAKE, FAKE, FAKE, FAKE, FAKE, 4, 8, 32, 100, FAKE, FAKE, ws - 1, None) == gm.GM_ERR_WORKSPACE
    bwd = L.gm_hyper_bwd
    ok = [FAKE] * 9 + [4, 8, 32, 100, 1e-3, 0.9, 0.999, 1e-8, 0.05, 1, FAKE, FAKE, ws, None]

    def call(i, val):
        a = list(ok)
        a[i] = val
        return bwd(*a)

    for i in range(9):
        assert call(i, None) == gm.GM_ERR_NULL, i
    assert call(19, None) == gm.GM_ERR_NULL
    for i, bad in ((13, -1.0), (14, 1.0), (15, -0.5), (16, 0.0), (17, -0.1), (18, 0)):
        assert call(i, bad) == gm.GM_ERR_VALUE, (i, bad)
    assert call(5, MISALIGNED) == gm.GM_ERR_ALIGN
    assert call(21, ws - 1) == gm.GM_ERR_WORKSPACE
    assert L.gm_adamw(FAKE, FAKE, FAKE, None, 10, 1e-3, 0.9, 0.999, 1e-8, 0.05, 1, None) == gm.GM_ERR_NULL
    assert L.gm_adamw(FAKE, FAKE, FAKE, FAKE, -1, 1e-3, 0.9, 0.999, 1e-8, 0.05, 1, None) == gm.GM_ERR_SHAPE
    assert L.gm_adamw(FAKE, FAKE, FAKE, FAKE, 10, 1e-3, 0.9, 0.999, 1e-8, 0.05, 0, None) == gm.GM_ERR_VALUE
    assert L.gm_adamw(FAKE, FAKE, FAKE, FAKE, 0, 1e-3, 0.9, 0.999, 1e-8, 0.05, 1, None) == gm.GM_OK


# ------------------------------------------------- the binding checks its tensors

def _t(shape, dtype):
    import torch
    return torch.zeros(shape, dtype=dtype)


def test_binding_rejects_wrong_dtypes_and_short_outputs_before_the_call():
    import torch
    T, d_in, d_out, g = 32, 512, 256, 256
    X, W = _t((T, d_in), torch.bfloat16), _t((d_out, d_in), torch.bfloat16)
    mask, Y = _t((d_out, d_in // g), torch.float32), _t((T, d_out), torch.bfloat16)
    cases = [
        (lambda: gm.gm_masked_linear_fwd(X.float(), W, mask, g, Y), "X must be torch.bfloat16"),
        (lambda: gm.gm_masked_linear_fwd(X, W[:, :256], mask, g, Y), "W must have shape"),
        (lambda: gm.gm_masked_linear_fwd(X, W, mask[:-1], g, Y), "mask must hold 512 elements"),
        (lambda: gm.gm_masked_linear_fwd(X, W, mask.double(), g, Y), "mask must be torch.float32"),
        (lambda: gm.gm_masked_linear_fwd(X, W, mask, g, Y[:-1]), "Y must have shape"),
        (lambda: gm.gm_masked_linear_fwd(X, W, mask, 100, Y), "not tiled by"),
        (lambda: gm.gm_masked_linear_bwd(Y, X, W, mask, g, X[:-1], None), "dX must have shape"),
        (lambda: gm.gm_masked_linear_bwd(Y, X, W, mask, g, None, mask[:, :1]), "dgate must hold"),
        (lambda: gm.gm_masked_linear_bwd(Y[:, :8], X, W, mask, g, X, None), "dY must have shape"),
        (lambda: gm.gm_masked_linear_bwd(Y, X, W, None, g, X, None), "mask is required"),
        (lambda: gm.gm_gate(mask, mask[:1], 0.5, True, mask), "noise must hold"),
        (lambda: gm.gm_gate(mask, None, 0.5, True, Y), "mask_out must be torch.float32"),
        (lambda: gm.gm_gate_bwd(mask, mask, 0.5, mask[1:]), "dlogits must hold"),
        (lambda: gm.gm_adamw(mask, mask, mask, mask[1:], 1e-3, 0.9, 0.999, 1e-8, 0.0, 1), "v must hold"),
        (lambda: gm.gm_pack_rows(W, mask, g, 10, Y, _t(10, torch.int32), _t(10, torch.float32),
                                 _t(d_out, torch.int32)), "rowptr must hold"),
    ]
    for call, msg in cases:
        with pytest.raises(ValueError, match=msg):
            call()
    # well-formed host tensors get as far as the device check
    with pytest.raises(ValueError, match="must live on the GPU"):
        gm.gm_masked_linear_fwd(X, W, mask, g, Y)
    with pytest.raises(ValueError, match="must be contiguous"):
        gm.gm_gate_bwd(mask.t(), mask.t(), 0.5, mask.t())
