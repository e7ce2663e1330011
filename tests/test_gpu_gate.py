"""GPU parity of the gate (Gumbel-Sigmoid + STE) against the fp64 oracle.

The hard mask must agree bit for bit except for gates whose relaxed value lies
within 1e-6 of the 1/2 threshold (counted and reported); the soft value and
the STE gradient agree within fp32 rounding."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_support import assert_close, dev_f32, empty_f32, say, sync

pytestmark = pytest.mark.gpu

BAND = 1e-6


def _run_gate(logits, noise, tau, hard):
    import paper_2609_33977_amd as gm
    n = logits.size
    d_l = dev_f32(logits.ravel())
    d_u = dev_f32(noise.ravel()) if noise is not None else None
    d_m, d_y = empty_f32(n), empty_f32(n)
    gm.gm_gate(d_l, d_u, tau, hard, d_m, d_y)
    sync()
    return d_m.cpu().numpy().astype(np.float64), d_y.cpu().numpy().astype(np.float64)


def _compare_hard(m_gpu, logits, noise, tau):
    m_ref, y_ref = oracle.gate(logits.ravel().astype(np.float64), None if noise is None else noise.ravel(), tau, True)
    near = oracle.near_threshold(y_ref, BAND)
    mism = (m_gpu != m_ref) & ~near
    say(f"  hard gate: {near.sum()} of {near.size} within {BAND} of the threshold; {mism.sum()} mismatches outside")
    assert not mism.any()
    assert set(np.unique(m_gpu)) <= {0.0, 1.0}
    return m_ref, y_ref


def test_gate_budgeted_single_layer():
    case = workloads.make_linear_case((1, 0, 0), 4, 1024, 1024, 256, 2048, tau=0.5)
    say("gate: 4096 groups, tau 0.5, budget 2048 kept")
    m, y = _run_gate(case.logits, case.noise, case.tau, True)
    m_ref, y_ref = _compare_hard(m, case.logits, case.noise, case.tau)
    assert int(m.sum()) == 2048
    assert np.array_equal(m.reshape(case.mask.shape), case.mask.astype(np.float64))
    assert_close("soft y", y, y_ref, 1e-6)


def test_gate_random_inputs_near_threshold_counted():
    r = workloads.gen.rng_for(100)
    n = 1_000_003  # not a multiple of 4: exercises the scalar tail
    logits = r.standard_normal(n).astype(np.float32)
    noise = workloads.draw_uniform_noise(r, n)
    for tau in (0.4, 0.5):
        say(f"gate: {n} random groups, tau {tau}")
        m, y = _run_gate(logits, noise, tau, True)
        _, y_ref = _compare_hard(m, logits, noise, tau)
        assert np.max(np.abs(y - y_ref)) < 1e-5


def test_gate_eval_mode_and_soft_mode():
    r = workloads.gen.rng_for(101)
    n = 4099
    logits = (r.standard_normal(n) * 2).astype(np.float32)
    logits[:3] = [0.0, -0.0, 1e-30]
    say("gate: evaluation mode (no noise)")
    m, _ = _run_gate(logits, None, 0.4, True)
    assert np.array_equal(m, (logits.astype(np.float64) > 0).astype(np.float64))
    say("gate: soft mode")
    noise = workloads.draw_uniform_noise(r, n)
    m, y = _run_gate(logits, noise, 0.5, False)
    _, y_ref = oracle.gate(logits.astype(np.float64), noise, 0.5, False)
    assert_close("soft mask", m, y_ref, 1e-6)
    assert np.array_equal(m, y)


@pytest.mark.parametrize("n", [1, 2, 3, 5, 64, 4097])
def test_gate_small_and_ragged_sizes(n):
    r = workloads.gen.rng_for(102, n)
    logits = r.standard_normal(n).astype(np.float32)
    noise = workloads.draw_uniform_noise(r, n)
    say(f"gate: n={n}")
    m, y = _run_gate(logits, noise, 0.4, True)
    _compare_hard(m, logits, noise, 0.4)


def test_gate_bwd_matches_ste_and_allows_aliasing():
    import paper_2609_33977_amd as gm
    r = workloads.gen.rng_for(103)
    n = 65539
    logits = r.standard_normal(n).astype(np.float32)
    noise = workloads.draw_uniform_noise(r, n)
    up = r.standard_normal(n).astype(np.float32)
    tau = 0.4
    say(f"gate bwd: n={n}")
    _, y = _run_gate(logits, noise, tau, True)
    d_y = dev_f32(y)
    d_up = dev_f32(up)
    d_out = empty_f32(n)
    gm.gm_gate_bwd(d_up, d_y, tau, d_out)
    sync()
    ref = oracle.gate_bwd(up, y, tau)
    assert_close("dlogits", d_out.cpu().numpy(), ref, 1e-6)
    gm.gm_gate_bwd(d_up, d_y, tau, d_up)  # in place
    sync()
    assert np.array_equal(d_up.cpu().numpy(), d_out.cpu().numpy())
