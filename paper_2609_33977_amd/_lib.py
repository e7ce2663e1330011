"""ctypes binding of libgroupmask (argument marshalling only).

Each function has the name of the C entry point it calls, takes torch tensors
that already live on the GPU, passes their device pointers and the current
HIP stream, and raises GroupMaskError on any status other than GM_OK.  All
computation happens in the library's HIP kernels.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libgroupmask.so")

GM_OK, GM_ERR_NULL, GM_ERR_SHAPE, GM_ERR_VALUE, GM_ERR_ALIGN, GM_ERR_WORKSPACE, GM_ERR_DEVICE = range(7)
GM_OP_FWD, GM_OP_BWD = 0, 1

EXPORTS = (
    "gm_abi_version", "gm_status_string", "gm_gate", "gm_gate_bwd", "gm_budget_loss", "gm_gate_bwd_budget",
    "gm_workspace_size",
    "gm_masked_linear_fwd", "gm_masked_linear_bwd", "gm_pack_rows", "gm_packed_linear_fwd",
    "gm_distill_workspace_size", "gm_distill_fwd", "gm_distill_bwd",
    "gm_hyper_workspace_size", "gm_hyper_fwd", "gm_hyper_bwd", "gm_adamw",
)


class GroupMaskError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: status {status} ({status_string(status)})")


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it first (python paper_2609_33977_amd/build.py)")
    # torch carries its own copy of the HIP runtime and names it without the
    # version suffix, so the dynamic linker would load the system copy for
    # this library if it came first; a second runtime in the process sees no
    # device.  Loading torch first makes this library bind to torch's runtime.
    import torch  # noqa: F401
    lib = ctypes.CDLL(LIB_PATH)
    P, I64, I32, F32, SZ = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_float, ctypes.c_size_t
    F64 = ctypes.c_double
    sigs = {
        "gm_abi_version": ([], ctypes.c_int),
        "gm_status_string": ([ctypes.c_int], ctypes.c_char_p),
        "gm_gate": ([P, P, I64, F32, ctypes.c_int, P, P, P], ctypes.c_int),
        "gm_gate_bwd": ([P, P, I64, F32, P, P], ctypes.c_int),
        "gm_budget_loss": ([P, I64, P, P, I32, F32, F32, ctypes.c_int, P, P, P, P], ctypes.c_int),
        "gm_gate_bwd_budget": ([P, P, I64, F32, P, I32, P, P, P], ctypes.c_int),
        "gm_workspace_size": ([ctypes.c_int, I64, I64, I64, I32, I32, ctypes.POINTER(SZ)], ctypes.c_int),
        "gm_masked_linear_fwd": ([P, P, P, I64, I64, I64, I32, I32, P, P, SZ, P], ctypes.c_int),
        "gm_masked_linear_bwd": ([P, P, P, P, I64, I64, I64, I32, I32, P, P, P, SZ, P], ctypes.c_int),
        "gm_pack_rows": ([P, P, I64, I64, I32, I32, I64, P, P, P, P, P], ctypes.c_int),
        "gm_packed_linear_fwd": ([P, P, P, P, P, I64, I64, I64, I32, P, P], ctypes.c_int),
        "gm_distill_workspace_size": ([I64, I64, I64, ctypes.POINTER(SZ)], ctypes.c_int),
        "gm_distill_fwd": ([P, P, P, P, I64, I64, I64, P, P, P, SZ, P], ctypes.c_int),
        "gm_distill_bwd": ([P, I64, I64, I64, P, P, SZ, P], ctypes.c_int),
        "gm_hyper_workspace_size": ([I64, I64, I64, I64, ctypes.POINTER(SZ)], ctypes.c_int),
        "gm_hyper_fwd": ([P, P, P, P, P, I64, I64, I64, I64, P, P, SZ, P], ctypes.c_int),
        "gm_hyper_bwd": ([P, P, P, P, P, P, P, P, P, I64, I64, I64, I64, F64, F64, F64, F64, F64, I32, P, P, SZ, P],
                         ctypes.c_int),
        "gm_adamw": ([P, P, P, P, I64, F64, F64, F64, F64, F64, I32, P], ctypes.c_int),
    }
    for name, (args, res) in sigs.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    return lib


LIB = _load()


def status_string(status: int) -> str:
    return LIB.gm_status_string(int(status)).decode()


def gm_abi_version() -> int:
    return LIB.gm_abi_version()


def _check(status: int, where: str) -> None:
    if status != GM_OK:
        raise GroupMaskError(status, where)


def _ptr(t):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensor must live on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def gm_gate(logits, noise, tau: float, hard: bool, mask_out, soft_out=None, stream=None) -> None:
    _check(LIB.gm_gate(_ptr(logits), _ptr(noise), logits.numel(), float(tau), int(bool(hard)), _ptr(mask_out),
                       _ptr(soft_out), _stream(stream)), "gm_gate")


def gm_gate_bwd(dmask, soft, tau: float, dlogits, stream=None) -> None:
    _check(LIB.gm_gate_bwd(_ptr(dmask), _ptr(soft), dmask.numel(), float(tau), _ptr(dlogits), _stream(stream)),
           "gm_gate_bwd")


def gm_budget_loss(mask, offsets, params, s_target: float, lam: float, uniform: bool, kept, loss, coeff,
                   stream=None) -> None:
    """Sparsity-budget regulariser over the layers of a flat selector array (see gm_budget_loss in the header)."""
    _check(LIB.gm_budget_loss(_ptr(mask), mask.numel(), _ptr(offsets), _ptr(params), params.numel(), float(s_target),
                              float(lam), int(bool(uniform)), _ptr(kept), _ptr(loss), _ptr(coeff), _stream(stream)),
           "gm_budget_loss")


def gm_gate_bwd_budget(dgate, soft, tau: float, offsets, coeff, dlogits, stream=None) -> None:
    _check(LIB.gm_gate_bwd_budget(_ptr(dgate), _ptr(soft), dgate.numel(), float(tau), _ptr(offsets), coeff.numel(),
                                  _ptr(coeff), _ptr(dlogits), _stream(stream)), "gm_gate_bwd_budget")


def gm_workspace_size(op: int, T: int, d_in: int, d_out: int, g: int, g_out: int = 1) -> int:
    out = ctypes.c_size_t(0)
    _check(LIB.gm_workspace_size(int(op), int(T), int(d_in), int(d_out), int(g), int(g_out), ctypes.byref(out)),
           "gm_workspace_size")
    return out.value


def gm_masked_linear_fwd(X, W, mask, g: int, Y, ws=None, stream=None, g_out: int = 1) -> None:
    T, d_in = X.shape
    d_out = W.shape[0]
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(LIB.gm_masked_linear_fwd(_ptr(X), _ptr(W), _ptr(mask), T, d_in, d_out, int(g), int(g_out), _ptr(Y),
                                    _ptr(ws), nbytes, _stream(stream)), "gm_masked_linear_fwd")


def gm_masked_linear_bwd(dY, X, W, mask, g: int, dX=None, dgate=None, ws=None, stream=None, g_out: int = 1) -> None:
    T, d_in = X.shape
    d_out = W.shape[0]
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(LIB.gm_masked_linear_bwd(_ptr(dY), _ptr(X), _ptr(W), _ptr(mask), T, d_in, d_out, int(g), int(g_out),
                                    _ptr(dX), _ptr(dgate), _ptr(ws), nbytes, _stream(stream)), "gm_masked_linear_bwd")


def gm_pack_rows(W, mask, g: int, capacity: int, Wp, chunk, scale, rowptr, stream=None, g_out: int = 1) -> None:
    d_out, d_in = W.shape
    _check(LIB.gm_pack_rows(_ptr(W), _ptr(mask), d_in, d_out, int(g), int(g_out), int(capacity), _ptr(Wp),
                            _ptr(chunk), _ptr(scale), _ptr(rowptr), _stream(stream)), "gm_pack_rows")


def gm_packed_linear_fwd(X, Wp, chunk, scale, rowptr, d_out: int, g: int, Y, stream=None) -> None:
    T, d_in = X.shape
    _check(LIB.gm_packed_linear_fwd(_ptr(X), _ptr(Wp), _ptr(chunk), _ptr(scale), _ptr(rowptr), T, d_in, int(d_out),
                                    int(g), _ptr(Y), _stream(stream)), "gm_packed_linear_fwd")


def gm_distill_workspace_size(N: int, d: int, V: int) -> int:
    out = ctypes.c_size_t(0)
    _check(LIB.gm_distill_workspace_size(int(N), int(d), int(V), ctypes.byref(out)), "gm_distill_workspace_size")
    return out.value


def gm_distill_fwd(Ht, Hs, W, valid, loss, ce, ws, stream=None) -> None:
    """Distillation loss of Eq. 4 (see gm_distill_fwd in the header); valid and ce may be None."""
    N, d = Ht.shape
    V = W.shape[0]
    _check(LIB.gm_distill_fwd(_ptr(Ht), _ptr(Hs), _ptr(W), _ptr(valid), N, d, V, _ptr(loss), _ptr(ce), _ptr(ws),
                              ws.numel() * ws.element_size(), _stream(stream)), "gm_distill_fwd")


def gm_distill_bwd(W, dHs, ws, stream=None) -> None:
    """Gradient of the distillation loss to the student hidden states, from the forward's workspace."""
    N, d = dHs.shape
    V = W.shape[0]
    _check(LIB.gm_distill_bwd(_ptr(W), N, d, V, _ptr(dHs), _ptr(ws), ws.numel() * ws.element_size(),
                              _stream(stream)), "gm_distill_bwd")


def gm_hyper_workspace_size(L: int, D: int, H: int, G_total: int) -> int:
    out = ctypes.c_size_t(0)
    _check(LIB.gm_hyper_workspace_size(int(L), int(D), int(H), int(G_total), ctypes.byref(out)),
           "gm_hyper_workspace_size")
    return out.value


def gm_hyper_fwd(z, gru, A, c, offsets, H: int, logits, ws, stream=None) -> None:
    """Selector logits from the hypernetwork (see gm_hyper_fwd in the header)."""
    L, D = z.shape
    _check(LIB.gm_hyper_fwd(_ptr(z), _ptr(gru), _ptr(A), _ptr(c), _ptr(offsets), L, D, int(H), A.shape[0],
                            _ptr(logits), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)), "gm_hyper_fwd")


def gm_hyper_bwd(dlogits, z, gru, A, c, mA, vA, mc, vc, H: int, lr: float, beta1: float, beta2: float, eps: float,
                 weight_decay: float, step: int, dgru, ws, stream=None) -> None:
    """Backward of the hypernetwork with one AdamW step on its heads; the GRU gradient goes to dgru."""
    L, D = z.shape
    _check(LIB.gm_hyper_bwd(_ptr(dlogits), _ptr(z), _ptr(gru), _ptr(A), _ptr(c), _ptr(mA), _ptr(vA), _ptr(mc),
                            _ptr(vc), L, D, int(H), A.shape[0], float(lr), float(beta1), float(beta2), float(eps),
                            float(weight_decay), int(step), _ptr(dgru), _ptr(ws), ws.numel() * ws.element_size(),
                            _stream(stream)), "gm_hyper_bwd")


def gm_adamw(p, g, m, v, lr: float, beta1: float, beta2: float, eps: float, weight_decay: float, step: int,
             stream=None) -> None:
    _check(LIB.gm_adamw(_ptr(p), _ptr(g), _ptr(m), _ptr(v), p.numel(), float(lr), float(beta1), float(beta2),
                        float(eps), float(weight_decay), int(step), _stream(stream)), "gm_adamw")
