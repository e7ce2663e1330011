"""GPU parity of the hypernetwork (Sec. 2.2, Eq. 3) and its AdamW step
(Table 5) against the fp64 oracle.

The GPU computes in fp32.  Tolerances: logits to 1e-5 relative Frobenius;
the GRU gradient (a recurrence over the layers) to 1e-4; AdamW moments to
1e-5; the parameter update (p_new - p_old) to 1e-3 of its own norm, since it
divides by sqrt(v)."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_support import assert_close, dev_f32, empty_f32, say, sync, workspace

pytestmark = pytest.mark.gpu

OPT = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.05)


def _dev_i64(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int64)).cuda()


def _run(case, step):
    import paper_2609_33977_amd as gm
    G = int(case.offsets[-1])
    d = {k: dev_f32(getattr(case, k)) for k in ("z", "gru", "A", "c", "dlogits", "mA", "vA", "mc", "vc")}
    ws = workspace(gm.gm_hyper_workspace_size(case.L, case.D, case.H, G))
    logits = empty_f32(G)
    gm.gm_hyper_fwd(d["z"], d["gru"], d["A"], d["c"], _dev_i64(case.offsets), case.H, logits, ws)
    sync()
    logits_h = logits.cpu().numpy().astype(np.float64)
    dgru = empty_f32(case.gru.size)
    gm.gm_hyper_bwd(d["dlogits"], d["z"], d["gru"], d["A"], d["c"], d["mA"], d["vA"], d["mc"], d["vc"], case.H,
                    step=step, dgru=dgru, ws=ws, **OPT)
    sync()
    out = {k: d[k].cpu().numpy().astype(np.float64) for k in ("A", "c", "mA", "vA", "mc", "vc")}
    return logits_h, dgru.cpu().numpy().astype(np.float64), out


def _check(case, step, full_dgru=True):
    logits, dgru, out = _run(case, step)
    ref = oracle.hyper_fwd(case.z, case.gru, case.A, case.c, case.offsets, case.H)
    assert_close("logits", logits, ref, 1e-5)
    dA, dc, dgru_ref, _ = oracle.hyper_bwd(case.dlogits, case.z, case.gru, case.A, case.c, case.offsets, case.H)
    if full_dgru:
        assert_close("dgru", dgru, dgru_ref, 1e-4)
    for name, p0, g, m0, v0 in (("A", case.A, dA, case.mA, case.vA), ("c", case.c, dc, case.mc, case.vc)):
        p, m, v = oracle.adamw_step(p0, g, m0, v0, OPT["lr"], OPT["beta1"], OPT["beta2"], OPT["eps"],
                                    OPT["weight_decay"], step)
        assert_close(f"m_{name}", out["m" + name], m, 1e-5)
        assert_close(f"v_{name}", out["v" + name], v, 1e-5)
        assert_close(f"update of {name}", out[name] - p0, p - p0, 1e-3)


@pytest.mark.parametrize("H,D", [(32, 16), (64, 64), (128, 40)])
def test_hyper_parity(H, D):
    # ragged layers: a single row, an empty layer, rows across several 2048-row chunks
    sizes = [3000, 1, 0, 4100, 2048, 17, 5000]
    say(f"hypernetwork: L={len(sizes)} D={D} H={H} rows={sum(sizes)}")
    case = workloads.make_hyper_case((250, H, D), sizes, D, H)
    _check(case, step=7)


def test_hyper_first_step_from_zero_moments():
    sizes = [700, 2049, 64]
    say("hypernetwork: first AdamW step")
    case = workloads.make_hyper_case((251,), sizes, 32, 64, warm=False)
    _check(case, step=1)


def test_hyper_many_layers():
    # 224 layers as in LLaMA-2-7B, with small selector counts
    r = workloads.gen.rng_for(252)
    sizes = [int(x) for x in r.integers(1, 600, size=224)]
    say(f"hypernetwork: 224 layers, {sum(sizes)} rows")
    case = workloads.make_hyper_case((253,), sizes, 64, 64)
    _check(case, step=3)


def test_adamw_flat():
    import paper_2609_33977_amd as gm
    r = workloads.gen.rng_for(254)
    n = 100003
    p0 = r.standard_normal(n).astype(np.float32)
    g = (r.standard_normal(n) * 1e-2).astype(np.float32)
    m0 = (r.standard_normal(n) * 1e-3).astype(np.float32)
    v0 = r.uniform(1e-7, 1e-5, size=n).astype(np.float32)
    p, gg, m, v = dev_f32(p0), dev_f32(g), dev_f32(m0), dev_f32(v0)
    gm.gm_adamw(p, gg, m, v, step=5, **OPT)
    sync()
    pr, mr, vr = oracle.adamw_step(p0, g, m0, v0, OPT["lr"], OPT["beta1"], OPT["beta2"], OPT["eps"],
                                   OPT["weight_decay"], 5)
    assert_close("m", m.cpu().numpy(), mr, 1e-5)
    assert_close("v", v.cpu().numpy(), vr, 1e-5)
    assert_close("update", p.cpu().numpy().astype(np.float64) - p0, pr - p0, 1e-3)


def test_hyper_llama2_7b_selectors():
    # the 224 selector matrices of LLaMA-2-7B with 1x256 groups (25.3 M logits),
    # H = 64, D = 64; logits and the head update on sampled rows
    import torch
    import paper_2609_33977_amd as gm
    cfg = workloads.config("llama2_7b_step")
    g = cfg["g"]
    sizes = [do * di // g for _ in range(cfg["layers"]) for _, do, di in cfg["linears"]]
    L, D, H = len(sizes), 64, 64
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    G = int(offsets[-1])
    say(f"hypernetwork at LLaMA-2-7B scale: L={L} rows={G}")
    small = workloads.make_hyper_case((255,), [1] * L, D, H)  # z and GRU parameters
    gen = torch.Generator(device="cuda")
    gen.manual_seed(workloads.SEED)
    a = 1.0 / np.sqrt(2 * H)
    A = (torch.rand(G, 2 * H, device="cuda", generator=gen) * 2 - 1) * a
    c = (torch.rand(G, device="cuda", generator=gen) * 2 - 1) * a
    dl = torch.randn(G, device="cuda", generator=gen) * 0.01
    mA, vA = torch.zeros_like(A), torch.zeros_like(A)
    mc, vc = torch.zeros_like(c), torch.zeros_like(c)
    r = workloads.gen.rng_for(256)
    rows = np.sort(r.choice(G, size=2000, replace=False))
    idx = torch.from_numpy(rows).cuda()
    A0, c0, dl0 = (t[idx].cpu().numpy().astype(np.float64) for t in (A, c, dl))
    z, gru = dev_f32(small.z), dev_f32(small.gru)
    ws = workspace(gm.gm_hyper_workspace_size(L, D, H, G))
    logits = empty_f32(G)
    gm.gm_hyper_fwd(z, gru, A, c, _dev_i64(offsets), H, logits, ws)
    dgru = empty_f32(small.gru.size)
    gm.gm_hyper_bwd(dl, z, gru, A, c, mA, vA, mc, vc, H, step=1, dgru=dgru, ws=ws, **OPT)
    sync()
    o = oracle.bigru_fwd(small.z, small.gru, H)
    lay = np.searchsorted(offsets, rows, side="right") - 1
    ref = np.einsum("rk,rk->r", A0, o[lay]) + c0
    assert_close("logits (sampled rows)", logits[idx].cpu().numpy(), ref, 1e-5)
    gA = dl0[:, None] * o[lay]
    pA, mref, _ = oracle.adamw_step(A0, gA, 0.0, 0.0, OPT["lr"], OPT["beta1"], OPT["beta2"], OPT["eps"],
                                    OPT["weight_decay"], 1)
    assert_close("m_A (sampled rows)", mA[idx].cpu().numpy(), mref, 1e-5)
    assert_close("update of A (sampled rows)", A[idx].cpu().numpy().astype(np.float64) - A0, pA - A0, 1e-3)
    assert np.all(np.isfinite(dgru.cpu().numpy()))
