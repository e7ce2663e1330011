"""One whole mask-learning step of a toy model, composed only of the library's
entry points and checked stage by stage against the same composition of the
fp64 oracle (Sec. 2.2-2.4, Fig. 2):

  hypernetwork -> Gumbel-Sigmoid gate (hard, STE) -> teacher pass (all
  selectors kept) and student pass through three chained masked linears ->
  distillation loss through an LM head -> backward through the student's
  linears (dX chain, dgate per layer) -> budget regulariser folded into the
  gate backward -> hypernetwork backward with its AdamW step, and AdamW on the
  GRU parameters.

The oracle chain rounds every activation and activation gradient to bf16 where
the library stores bf16 (R11 of the readings), so the two chains stay within
fp32 accumulation error of each other; where floating point decides a gate,
the library's decisions are compared with the oracle's outside the
near-threshold band and then used by both chains."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_support import assert_close, dev_bf16, dev_f32, empty_bf16, empty_f32, host_f64_from_bf16, say, sync, workspace

pytestmark = pytest.mark.gpu


def _bf16(x):
    """fp64 -> the bf16 value the library would store (via fp32, round to nearest even)."""
    return workloads.f32_from_bf16_bits(workloads.bf16_bits_from_f32(np.asarray(x, np.float32))).astype(np.float64)


def test_mask_learning_step_end_to_end():
    import torch
    import paper_2609_33977_amd as gm
    T, d, V, g, L = 96, 512, 1000, 64, 3
    D, H = 16, 32
    tau, lam, s_t = 0.4, 16.0, 0.5
    opt = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.05)
    step = 5
    G_l = d * (d // g)
    r = workloads.gen.rng_for(260)
    X0 = workloads.bf16_bits_from_f32(r.standard_normal((T, d), dtype=np.float32))
    Ws = [workloads.bf16_bits_from_f32(r.standard_normal((d, d), dtype=np.float32) * np.float32(1.0 / np.sqrt(d)))
          for _ in range(L)]
    Wlm = workloads.bf16_bits_from_f32(r.standard_normal((V, d), dtype=np.float32) * np.float32(3.0 / np.sqrt(d)))
    hc = workloads.make_hyper_case((261,), [G_l] * L, D, H, warm=True)
    u = workloads.draw_uniform_noise(r, L * G_l)
    offsets = hc.offsets
    params = [d * d] * L
    say(f"pipeline: T={T} d={d} V={V} L={L} 1x{g} groups, hypernetwork D={D} H={H}")

    # ---------------------------------------------------------------- GPU
    dz, dgru_t = dev_f32(hc.z), dev_f32(hc.gru)
    dA, dc, dmA, dvA, dmc, dvc = (dev_f32(x) for x in (hc.A, hc.c, hc.mA, hc.vA, hc.mc, hc.vc))
    d_off = torch.from_numpy(offsets).cuda()
    d_par = torch.tensor(params, dtype=torch.int64, device="cuda")
    ws_h = workspace(gm.gm_hyper_workspace_size(L, D, H, L * G_l))
    logits = empty_f32(L * G_l)
    gm.gm_hyper_fwd(dz, dgru_t, dA, dc, d_off, H, logits, ws_h)
    mask, soft = empty_f32(L * G_l), empty_f32(L * G_l)
    gm.gm_gate(logits, dev_f32(u), tau, True, mask, soft)

    x0 = dev_bf16(X0)
    dW = [dev_bf16(w) for w in Ws]
    ones = torch.ones(d, d // g, device="cuda")
    masks = [mask[l * G_l:(l + 1) * G_l].view(d, d // g) for l in range(L)]

    def chain(ms):
        acts = [x0]
        for l in range(L):
            y = empty_bf16(T, d)
            gm.gm_masked_linear_fwd(acts[-1], dW[l], ms[l], g, y)
            acts.append(y)
        return acts

    teacher = chain([ones] * L)
    student = chain(masks)
    ws_d = workspace(gm.gm_distill_workspace_size(T, d, V))
    loss = empty_f32(1)
    w_lm = dev_bf16(Wlm)
    gm.gm_distill_fwd(teacher[-1], student[-1], w_lm, None, loss, None, ws_d)
    dHs = empty_bf16(T, d)
    gm.gm_distill_bwd(w_lm, dHs, ws_d)

    dgate = empty_f32(L * G_l)
    ws_b = workspace(gm.gm_workspace_size(gm.GM_OP_BWD, T, d, d, g))
    dy = dHs
    dys = {}
    for l in reversed(range(L)):
        dys[l] = dy
        dx = empty_bf16(T, d)
        gm.gm_masked_linear_bwd(dy, student[l], dW[l], masks[l], g, dx, dgate[l * G_l:(l + 1) * G_l].view(d, d // g),
                                ws_b)
        dy = dx
    kept = torch.empty(L, dtype=torch.int64, device="cuda")
    bloss = torch.empty(1, dtype=torch.float64, device="cuda")
    coeff = empty_f32(L)
    gm.gm_budget_loss(mask, d_off, d_par, s_t, lam, False, kept, bloss, coeff)
    dlog = empty_f32(L * G_l)
    gm.gm_gate_bwd_budget(dgate, soft, tau, d_off, coeff, dlog)
    dgru = empty_f32(hc.gru.size)
    gm.gm_hyper_bwd(dlog, dz, dgru_t, dA, dc, dmA, dvA, dmc, dvc, H, step=step, dgru=dgru, ws=ws_h, **opt)
    mg, vg = dev_f32(np.zeros_like(hc.gru)), dev_f32(np.zeros_like(hc.gru))
    gm.gm_adamw(dgru_t, dgru, mg, vg, step=1, **opt)
    sync()

    # ---------------------------------------------------------------- oracle, stage by stage
    lo = oracle.hyper_fwd(hc.z, hc.gru, hc.A, hc.c, offsets, H)
    assert_close("hypernetwork logits", logits.cpu().numpy(), lo, 1e-5)
    m_ref, y_ref = oracle.gate(lo, u, tau, True)
    mg_h = mask.cpu().numpy().astype(np.float64)
    band = oracle.near_threshold(y_ref)
    assert np.array_equal(mg_h[~band], m_ref[~band]), "hard selectors differ outside the near-threshold band"
    say(f"  selectors: {int(mg_h.sum())} of {mg_h.size} kept, {int(band.sum())} near the threshold")

    Xr = oracle.from_bf16(X0)
    Wr = [oracle.from_bf16(w) for w in Ws]
    ml = [mg_h[l * G_l:(l + 1) * G_l].reshape(d, d // g) for l in range(L)]

    def ochain(ms):
        acts = [Xr]
        for l in range(L):
            acts.append(_bf16(oracle.linear_fwd(acts[-1], Wr[l], ms[l], g)))
        return acts

    t_ref = ochain([np.ones((d, d // g))] * L)
    s_ref = ochain(ml)
    assert_close("teacher output", host_f64_from_bf16(teacher[-1]), t_ref[-1])
    assert_close("student output", host_f64_from_bf16(student[-1]), s_ref[-1])
    Wl = oracle.from_bf16(Wlm)
    L_ref, _, _, _ = oracle.distill_loss(t_ref[-1], s_ref[-1], Wl)
    say(f"  distillation loss {float(loss.item()):.6f} (oracle {L_ref:.6f})")
    assert abs(float(loss.item()) - L_ref) <= 1e-3 * abs(L_ref)
    dH_ref = _bf16(oracle.distill_loss_bwd(t_ref[-1], s_ref[-1], Wl))
    assert_close("dH_S", host_f64_from_bf16(dHs), dH_ref)

    dy_r = dH_ref
    dg_ref = np.empty(L * G_l)
    for l in reversed(range(L)):
        dx_r, dg_r = oracle.linear_bwd(dy_r, s_ref[l], Wr[l], ml[l], g)
        dg_ref[l * G_l:(l + 1) * G_l] = dg_r.reshape(-1)
        assert_close(f"dgate of linear {l}", dgate[l * G_l:(l + 1) * G_l].cpu().numpy(), dg_r.reshape(-1))
        dy_r = _bf16(dx_r)

    Lb, cb, kb = oracle.budget_loss(np.split(mg_h, L), params, s_t, lam)
    assert np.array_equal(kept.cpu().numpy(), kb)
    assert abs(float(bloss.item()) - Lb) <= 1e-12 * max(1.0, abs(Lb))
    say(f"  budget: kept {list(kb)}, loss {Lb:.6f}")
    dlog_ref = oracle.gate_bwd(dg_ref + np.repeat(cb, G_l), y_ref, tau)
    assert_close("logit gradient", dlog.cpu().numpy(), dlog_ref)

    gA, gc, gg, _ = oracle.hyper_bwd(dlog_ref, hc.z, hc.gru, hc.A, hc.c, offsets, H)
    pA, mA_ref, _ = oracle.adamw_step(hc.A, gA, hc.mA, hc.vA, opt["lr"], opt["beta1"], opt["beta2"], opt["eps"],
                                      opt["weight_decay"], step)
    assert_close("head moment m_A", dmA.cpu().numpy(), mA_ref)
    assert_close("head update", dA.cpu().numpy().astype(np.float64) - hc.A, pA - hc.A)
    assert_close("GRU gradient", dgru.cpu().numpy(), gg)
    pg, _, _ = oracle.adamw_step(hc.gru, gg, 0.0, 0.0, opt["lr"], opt["beta1"], opt["beta2"], opt["eps"],
                                 opt["weight_decay"], 1)
    # first AdamW step: lr * g / (|g| + eps) per element, so compare signs of the update
    upd, upd_ref = dgru_t.cpu().numpy().astype(np.float64) - hc.gru, pg - hc.gru
    agree = np.mean(np.sign(upd) == np.sign(upd_ref))
    say(f"  GRU update sign agreement {agree:.4f}")
    assert agree >= 0.99
