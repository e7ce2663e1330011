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
# GM_LIBRARY_PATH selects another build of the same library (the host-sanitizer
# build of the CPU tests); by default the in-tree build is loaded.
LIB_PATH = os.environ.get("GM_LIBRARY_PATH") or os.path.join(HERE, "libgroupmask.so")

GM_OK, GM_ERR_NULL, GM_ERR_SHAPE, GM_ERR_VALUE, GM_ERR_ALIGN, GM_ERR_WORKSPACE, GM_ERR_DEVICE = range(7)
GM_OP_FWD, GM_OP_BWD = 0, 1

EXPORTS = (
    "gm_abi_version", "gm_status_string", "gm_gate", "gm_gate_bwd", "gm_budget_loss", "gm_gate_bwd_budget",
    "gm_workspace_size",
    "gm_masked_linear_fwd", "gm_masked_linear_bwd", "gm_masked_linear_bwd_noalloc", "gm_pack_rows", "gm_packed_linear_fwd",
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
        "gm_masked_linear_bwd_noalloc": ([P, P, P, P, I64, I64, I64, I32, I32, P, P, P], ctypes.c_int),
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
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    if not t.is_cuda:
        raise ValueError("tensor must live on the GPU")
    return ctypes.c_void_p(t.data_ptr())


# Argument checks run before any call into the library: the C entry points see
# only pointers, so a tensor of the wrong dtype or too few elements would
# otherwise be read or written out of bounds by the kernels.  Every tensor's
# dtype and size are checked first; _ptr then checks layout and device as it
# takes each pointer.

def _dt(name):
    import torch
    return {"bf16": torch.bfloat16, "f32": torch.float32, "f64": torch.float64, "i32": torch.int32,
            "i64": torch.int64, "u8": torch.uint8}[name]


def _arg(where, what, t, dtype, shape=None, numel=None, at_least=None, optional=False):
    """Check one tensor argument: dtype, exact shape (None entries are free), element count."""
    if t is None:
        if optional:
            return
        raise ValueError(f"{where}: {what} is required")
    want = _dt(dtype)
    if dtype == "i64" and str(t.dtype) == "torch.uint64":
        want = t.dtype  # counters may be handed over as unsigned 64-bit
    if t.dtype != want:
        raise ValueError(f"{where}: {what} must be {want}, got {t.dtype}")
    if shape is not None:
        if t.dim() != len(shape) or any(w is not None and int(d) != int(w) for d, w in zip(t.shape, shape)):
            raise ValueError(f"{where}: {what} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{where}: {what} must hold {numel} elements, got {t.numel()}")
    if at_least is not None and t.numel() < at_least:
        raise ValueError(f"{where}: {what} must hold at least {at_least} elements, got {t.numel()}")


def _groups(d_out, d_in, g, g_out, where):
    if g <= 0 or g_out <= 0 or d_in % g or d_out % g_out:
        raise ValueError(f"{where}: [{d_out}, {d_in}] is not tiled by {g_out} x {g} groups")
    return (d_out // g_out) * (d_in // g)


def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def gm_gate(logits, noise, tau: float, hard: bool, mask_out, soft_out=None, stream=None) -> None:
    n = logits.numel()
    _arg("gm_gate", "logits", logits, "f32")
    _arg("gm_gate", "noise", noise, "f32", numel=n, optional=True)
    _arg("gm_gate", "mask_out", mask_out, "f32", numel=n)
    _arg("gm_gate", "soft_out", soft_out, "f32", numel=n, optional=True)
    _check(LIB.gm_gate(_ptr(logits), _ptr(noise), logits.numel(), float(tau), int(bool(hard)), _ptr(mask_out),
                       _ptr(soft_out), _stream(stream)), "gm_gate")


def gm_gate_bwd(dmask, soft, tau: float, dlogits, stream=None) -> None:
    n = dmask.numel()
    _arg("gm_gate_bwd", "dmask", dmask, "f32")
    _arg("gm_gate_bwd", "soft", soft, "f32", numel=n)
    _arg("gm_gate_bwd", "dlogits", dlogits, "f32", numel=n)
    _check(LIB.gm_gate_bwd(_ptr(dmask), _ptr(soft), dmask.numel(), float(tau), _ptr(dlogits), _stream(stream)),
           "gm_gate_bwd")


def gm_budget_loss(mask, offsets, params, s_target: float, lam: float, uniform: bool, kept, loss, coeff,
                   stream=None) -> None:
    """Sparsity-budget regulariser over the layers of a flat selector array (see gm_budget_loss in the header)."""
    L = params.numel()
    _arg("gm_budget_loss", "mask", mask, "f32")
    _arg("gm_budget_loss", "offsets", offsets, "i64", numel=L + 1)
    _arg("gm_budget_loss", "params", params, "i64")
    _arg("gm_budget_loss", "kept", kept, "i64", numel=L)
    _arg("gm_budget_loss", "loss", loss, "f64", numel=1)
    _arg("gm_budget_loss", "coeff", coeff, "f32", numel=L)
    _check(LIB.gm_budget_loss(_ptr(mask), mask.numel(), _ptr(offsets), _ptr(params), params.numel(), float(s_target),
                              float(lam), int(bool(uniform)), _ptr(kept), _ptr(loss), _ptr(coeff), _stream(stream)),
           "gm_budget_loss")


def gm_gate_bwd_budget(dgate, soft, tau: float, offsets, coeff, dlogits, stream=None) -> None:
    n, L = dgate.numel(), coeff.numel()
    _arg("gm_gate_bwd_budget", "dgate", dgate, "f32")
    _arg("gm_gate_bwd_budget", "soft", soft, "f32", numel=n)
    _arg("gm_gate_bwd_budget", "offsets", offsets, "i64", numel=L + 1)
    _arg("gm_gate_bwd_budget", "coeff", coeff, "f32")
    _arg("gm_gate_bwd_budget", "dlogits", dlogits, "f32", numel=n)
    _check(LIB.gm_gate_bwd_budget(_ptr(dgate), _ptr(soft), dgate.numel(), float(tau), _ptr(offsets), coeff.numel(),
                                  _ptr(coeff), _ptr(dlogits), _stream(stream)), "gm_gate_bwd_budget")


def gm_workspace_size(op: int, T: int, d_in: int, d_out: int, g: int, g_out: int = 1) -> int:
    out = ctypes.c_size_t(0)
    _check(LIB.gm_workspace_size(int(op), int(T), int(d_in), int(d_out), int(g), int(g_out), ctypes.byref(out)),
           "gm_workspace_size")
    return out.value


def gm_masked_linear_fwd(X, W, mask, g: int, Y, ws=None, stream=None, g_out: int = 1) -> None:
    w = "gm_masked_linear_fwd"
    _arg(w, "X", X, "bf16", shape=(None, None))
    T, d_in = X.shape
    _arg(w, "W", W, "bf16", shape=(None, d_in))
    d_out = W.shape[0]
    _arg(w, "mask", mask, "f32", numel=_groups(d_out, d_in, g, g_out, w))
    _arg(w, "Y", Y, "bf16", shape=(T, d_out))
    _arg(w, "ws", ws, "u8", optional=True)
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(LIB.gm_masked_linear_fwd(_ptr(X), _ptr(W), _ptr(mask), T, d_in, d_out, int(g), int(g_out), _ptr(Y),
                                    _ptr(ws), nbytes, _stream(stream)), "gm_masked_linear_fwd")


def gm_masked_linear_bwd(dY, X, W, mask, g: int, dX=None, dgate=None, ws=None, stream=None, g_out: int = 1) -> None:
    w = "gm_masked_linear_bwd"
    _arg(w, "X", X, "bf16", shape=(None, None))
    T, d_in = X.shape
    _arg(w, "W", W, "bf16", shape=(None, d_in))
    d_out = W.shape[0]
    G = _groups(d_out, d_in, g, g_out, w)
    _arg(w, "dY", dY, "bf16", shape=(T, d_out))
    _arg(w, "mask", mask, "f32", numel=G, optional=dX is None)
    _arg(w, "dX", dX, "bf16", shape=(T, d_in), optional=True)
    _arg(w, "dgate", dgate, "f32", numel=G, optional=True)
    _arg(w, "ws", ws, "u8", optional=True)
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(LIB.gm_masked_linear_bwd(_ptr(dY), _ptr(X), _ptr(W), _ptr(mask), T, d_in, d_out, int(g), int(g_out),
                                    _ptr(dX), _ptr(dgate), _ptr(ws), nbytes, _stream(stream)), "gm_masked_linear_bwd")


def gm_masked_linear_bwd_noalloc(dY, X, W, mask, g: int, dX=None, dgate=None, stream=None, g_out: int = 1) -> None:
    """gm_masked_linear_bwd with the library's fixed device scratch instead of a workspace (no allocation)."""
    w = "gm_masked_linear_bwd_noalloc"
    _arg(w, "X", X, "bf16", shape=(None, None))
    T, d_in = X.shape
    _arg(w, "W", W, "bf16", shape=(None, d_in))
    d_out = W.shape[0]
    G = _groups(d_out, d_in, g, g_out, w)
    _arg(w, "dY", dY, "bf16", shape=(T, d_out))
    _arg(w, "mask", mask, "f32", numel=G, optional=dX is None)
    _arg(w, "dX", dX, "bf16", shape=(T, d_in), optional=True)
    _arg(w, "dgate", dgate, "f32", numel=G, optional=True)
    _check(LIB.gm_masked_linear_bwd_noalloc(_ptr(dY), _ptr(X), _ptr(W), _ptr(mask), T, d_in, d_out, int(g),
                                            int(g_out), _ptr(dX), _ptr(dgate), _stream(stream)),
           "gm_masked_linear_bwd_noalloc")


GM_NOALLOC_SCRATCH_BYTES = 96 << 20


def gm_pack_rows(W, mask, g: int, capacity: int, Wp, chunk, scale, rowptr, stream=None, g_out: int = 1) -> None:
    w = "gm_pack_rows"
    _arg(w, "W", W, "bf16", shape=(None, None))
    d_out, d_in = W.shape
    _arg(w, "mask", mask, "f32", numel=_groups(d_out, d_in, g, g_out, w))
    _arg(w, "Wp", Wp, "bf16", at_least=int(capacity) * int(g))
    _arg(w, "chunk", chunk, "i32", at_least=int(capacity))
    _arg(w, "scale", scale, "f32", at_least=int(capacity))
    _arg(w, "rowptr", rowptr, "i32", numel=d_out + 1)
    _check(LIB.gm_pack_rows(_ptr(W), _ptr(mask), d_in, d_out, int(g), int(g_out), int(capacity), _ptr(Wp),
                            _ptr(chunk), _ptr(scale), _ptr(rowptr), _stream(stream)), "gm_pack_rows")


def gm_packed_linear_fwd(X, Wp, chunk, scale, rowptr, d_out: int, g: int, Y, stream=None) -> None:
    w = "gm_packed_linear_fwd"
    _arg(w, "X", X, "bf16", shape=(None, None))
    T, d_in = X.shape
    _arg(w, "Wp", Wp, "bf16", shape=(None, g))
    cap = Wp.shape[0]
    _arg(w, "chunk", chunk, "i32", numel=cap)
    _arg(w, "scale", scale, "f32", numel=cap)
    _arg(w, "rowptr", rowptr, "i32", numel=int(d_out) + 1)
    _arg(w, "Y", Y, "bf16", shape=(T, d_out))
    _check(LIB.gm_packed_linear_fwd(_ptr(X), _ptr(Wp), _ptr(chunk), _ptr(scale), _ptr(rowptr), T, d_in, int(d_out),
                                    int(g), _ptr(Y), _stream(stream)), "gm_packed_linear_fwd")


def gm_distill_workspace_size(N: int, d: int, V: int) -> int:
    out = ctypes.c_size_t(0)
    _check(LIB.gm_distill_workspace_size(int(N), int(d), int(V), ctypes.byref(out)), "gm_distill_workspace_size")
    return out.value


def gm_distill_fwd(Ht, Hs, W, valid, loss, ce, ws, stream=None) -> None:
    """Distillation loss of Eq. 4 (see gm_distill_fwd in the header); valid and ce may be None."""
    w = "gm_distill_fwd"
    _arg(w, "Ht", Ht, "bf16", shape=(None, None))
    N, d = Ht.shape
    _arg(w, "Hs", Hs, "bf16", shape=(N, d))
    _arg(w, "W", W, "bf16", shape=(None, d))
    V = W.shape[0]
    _arg(w, "valid", valid, "u8", numel=N, optional=True)
    _arg(w, "loss", loss, "f32", numel=1)
    _arg(w, "ce", ce, "f32", numel=N, optional=True)
    _arg(w, "ws", ws, "u8")
    _check(LIB.gm_distill_fwd(_ptr(Ht), _ptr(Hs), _ptr(W), _ptr(valid), N, d, V, _ptr(loss), _ptr(ce), _ptr(ws),
                              ws.numel() * ws.element_size(), _stream(stream)), "gm_distill_fwd")


def gm_distill_bwd(W, dHs, ws, stream=None) -> None:
    """Gradient of the distillation loss to the student hidden states, from the forward's workspace."""
    w = "gm_distill_bwd"
    _arg(w, "dHs", dHs, "bf16", shape=(None, None))
    N, d = dHs.shape
    _arg(w, "W", W, "bf16", shape=(None, d))
    V = W.shape[0]
    _arg(w, "ws", ws, "u8")
    _check(LIB.gm_distill_bwd(_ptr(W), N, d, V, _ptr(dHs), _ptr(ws), ws.numel() * ws.element_size(),
                              _stream(stream)), "gm_distill_bwd")


def gm_hyper_workspace_size(L: int, D: int, H: int, G_total: int) -> int:
    out = ctypes.c_size_t(0)
    _check(LIB.gm_hyper_workspace_size(int(L), int(D), int(H), int(G_total), ctypes.byref(out)),
           "gm_hyper_workspace_size")
    return out.value


def gm_hyper_fwd(z, gru, A, c, offsets, H: int, logits, ws, stream=None) -> None:
    """Selector logits from the hypernetwork (see gm_hyper_fwd in the header)."""
    w = "gm_hyper_fwd"
    _arg(w, "z", z, "f32", shape=(None, None))
    L, D = z.shape
    _arg(w, "gru", gru, "f32", numel=2 * 3 * int(H) * (D + int(H) + 2))
    _arg(w, "A", A, "f32", shape=(None, 2 * int(H)))
    G = A.shape[0]
    _arg(w, "c", c, "f32", numel=G)
    _arg(w, "offsets", offsets, "i64", numel=L + 1)
    _arg(w, "logits", logits, "f32", numel=G)
    _arg(w, "ws", ws, "u8")
    _check(LIB.gm_hyper_fwd(_ptr(z), _ptr(gru), _ptr(A), _ptr(c), _ptr(offsets), L, D, int(H), A.shape[0],
                            _ptr(logits), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)), "gm_hyper_fwd")


def gm_hyper_bwd(dlogits, z, gru, A, c, mA, vA, mc, vc, H: int, lr: float, beta1: float, beta2: float, eps: float,
                 weight_decay: float, step: int, dgru, ws, stream=None) -> None:
    """Backward of the hypernetwork with one AdamW step on its heads; the GRU gradient goes to dgru."""
    w = "gm_hyper_bwd"
    _arg(w, "z", z, "f32", shape=(None, None))
    L, D = z.shape
    P = 2 * 3 * int(H) * (D + int(H) + 2)
    _arg(w, "gru", gru, "f32", numel=P)
    _arg(w, "A", A, "f32", shape=(None, 2 * int(H)))
    G = A.shape[0]
    _arg(w, "dlogits", dlogits, "f32", numel=G)
    _arg(w, "c", c, "f32", numel=G)
    _arg(w, "mA", mA, "f32", shape=(G, 2 * int(H)))
    _arg(w, "vA", vA, "f32", shape=(G, 2 * int(H)))
    _arg(w, "mc", mc, "f32", numel=G)
    _arg(w, "vc", vc, "f32", numel=G)
    _arg(w, "dgru", dgru, "f32", numel=P)
    _arg(w, "ws", ws, "u8")
    _check(LIB.gm_hyper_bwd(_ptr(dlogits), _ptr(z), _ptr(gru), _ptr(A), _ptr(c), _ptr(mA), _ptr(vA), _ptr(mc),
                            _ptr(vc), L, D, int(H), A.shape[0], float(lr), float(beta1), float(beta2), float(eps),
                            float(weight_decay), int(step), _ptr(dgru), _ptr(ws), ws.numel() * ws.element_size(),
                            _stream(stream)), "gm_hyper_bwd")


def gm_adamw(p, g, m, v, lr: float, beta1: float, beta2: float, eps: float, weight_decay: float, step: int,
             stream=None) -> None:
    n = p.numel()
    for what, t in (("p", p), ("g", g), ("m", m), ("v", v)):
        _arg("gm_adamw", what, t, "f32", numel=n)
    _check(LIB.gm_adamw(_ptr(p), _ptr(g), _ptr(m), _ptr(v), p.numel(), float(lr), float(beta1), float(beta2),
                        float(eps), float(weight_decay), int(step), _stream(stream)), "gm_adamw")
