"""GPU parity of the self-distillation loss through the LM head (Sec. 2.4,
Eq. 4) and its gradient to the student hidden states, against the fp64 oracle.

Tolerances: the logits are fp32 sums of exact bf16 products, so the loss and
each token's cross-entropy match to 1e-4 (1 + |value|); dH_S is rounded to
bf16 (as is dz_S before the product), so it matches to 1e-2 relative
Frobenius."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_support import assert_close, dev_bf16, empty_bf16, empty_f32, host_bits, host_f64_from_bf16, say, sync, workspace

pytestmark = pytest.mark.gpu

CE_TOL = 1e-4


def _run(case, valid=None):
    import torch
    import paper_2609_33977_amd as gm
    Ht, Hs, W = dev_bf16(case.Ht), dev_bf16(case.Hs), dev_bf16(case.W)
    v = None if valid is None else torch.from_numpy(np.ascontiguousarray(valid, dtype=np.uint8)).cuda()
    ws = workspace(gm.gm_distill_workspace_size(case.N, case.d, case.V))
    loss, ce = empty_f32(1), empty_f32(case.N)
    gm.gm_distill_fwd(Ht, Hs, W, v, loss, ce, ws)
    dH = empty_bf16(case.N, case.d)
    gm.gm_distill_bwd(W, dH, ws)
    sync()
    return float(loss.cpu().numpy()[0]), ce.cpu().numpy().astype(np.float64), dH


def _close(name, got, ref):
    err = np.max(np.abs(np.asarray(got, np.float64) - ref) / (1.0 + np.abs(ref)))
    say(f"  {name}: max error {err:.2e}")
    assert err <= CE_TOL, f"{name}: {err:.2e} > {CE_TOL}"


def _host(case):
    return oracle.from_bf16(case.Ht), oracle.from_bf16(case.Hs), oracle.from_bf16(case.W)


SHAPES = [  # (N, d, V): ragged token and vocabulary tiles, short K loops
    (300, 256, 1000),
    (77, 96, 2056),    # the last vocabulary tile holds 8 rows: one wave row of it is empty
    (513, 512, 4096),
    (128, 1024, 768),
]


@pytest.mark.parametrize("N,d,V", SHAPES)
def test_distill_parity(N, d, V):
    say(f"distill: N={N} d={d} V={V}")
    case = workloads.make_distill_case((240, N, d, V), N, d, V)
    loss, ce, dH = _run(case)
    Ht, Hs, W = _host(case)
    L, ce_ref, _, _ = oracle.distill_loss(Ht, Hs, W)
    _close("loss", loss, L)
    _close("ce", ce, ce_ref)
    assert_close("dH_S", host_f64_from_bf16(dH), oracle.distill_loss_bwd(Ht, Hs, W))


def test_distill_valid_tokens():
    N, d, V = 260, 128, 1000
    case = workloads.make_distill_case((241,), N, d, V, valid_frac=0.6)
    say(f"distill with {int(case.valid.sum())} of {N} tokens valid")
    loss, ce, dH = _run(case, case.valid)
    Ht, Hs, W = _host(case)
    L, ce_ref, _, _ = oracle.distill_loss(Ht, Hs, W, case.valid)
    _close("loss", loss, L)
    _close("ce (every token)", ce, ce_ref)
    bits = host_bits(dH)
    assert not np.any(bits[case.valid == 0] & 0x7FFF), "invalid tokens must get an exactly zero gradient"
    assert_close("dH_S", host_f64_from_bf16(dH), oracle.distill_loss_bwd(Ht, Hs, W, case.valid))


def test_distill_no_valid_token_is_zero():
    N, d, V = 64, 64, 512
    case = workloads.make_distill_case((242,), N, d, V)
    loss, _, dH = _run(case, np.zeros(N, dtype=np.uint8))
    assert loss == 0.0
    assert not np.any(host_bits(dH) & 0x7FFF)


def test_distill_identical_passes():
    # H_S = H_T: the loss is the teacher entropy and the gradient vanishes.
    # The two passes' statistics are reduced by different code, so their
    # log-sum-exp may differ in the last bit; the gradient must stay below
    # 1e-4 of the one the same tokens get from a student that differs.
    N, d, V = 200, 256, 1000
    case = workloads.make_distill_case((243,), N, d, V)
    Ht, Hs, W = _host(case)
    scale = np.linalg.norm(oracle.distill_loss_bwd(Ht, Hs, W))
    case.Hs = case.Ht.copy()
    loss, ce, dH = _run(case)
    L, ce_ref, _, _ = oracle.distill_loss(Ht, Ht, W)
    _close("loss (teacher entropy)", loss, L)
    _close("ce", ce, ce_ref)
    ratio = np.linalg.norm(host_f64_from_bf16(dH)) / scale
    say(f"  |dH_S| / |dH_S of a differing student| = {ratio:.2e}")
    assert ratio <= 1e-4


def test_distill_llama2_7b_lm_head():
    # the LLaMA-2-7B LM head (V = 32000, d = 4096) over one mask-learning
    # batch (4096 tokens); sampled tokens against the oracle
    cfg = workloads.config("llama2_7b_step")
    N, d, V = cfg["T"], 4096, 32000
    say(f"distill llama2-7b LM head: N={N} d={d} V={V}")
    case = workloads.make_distill_case((244,), N, d, V)
    loss, ce, dH = _run(case)
    assert abs(loss - ce.mean()) <= 1e-6 * abs(loss)  # the loss is the mean of the per-token values
    r = workloads.gen.rng_for(245)
    t_s = np.sort(r.choice(N, size=48, replace=False))
    Ht, Hs, W = (oracle.from_bf16(x) for x in (case.Ht[t_s], case.Hs[t_s], case.W))
    _, ce_ref, _, _ = oracle.distill_loss(Ht, Hs, W)
    _close("ce (sampled tokens)", ce[t_s], ce_ref)
    # the sample's own mean divides by 48; the full batch by N
    ref = oracle.distill_loss_bwd(Ht, Hs, W) * (len(t_s) / N)
    assert_close("dH_S (sampled tokens)", host_f64_from_bf16(dH)[t_s], ref)
