"""GPU parity of the sparsity-budget regulariser (Sec. 2.3, Eq. 2) against the fp64 oracle.

Kept counts are integers and must match exactly; the loss is accumulated in
fp64 on the device and must match to 1e-12 relative; the per-layer gradient
coefficients are stored in fp32 (relative 1e-6).  The folded gate backward
adds the coefficient of each selector's layer to dgate before the STE factor
and matches the oracle's gate_bwd of that sum within fp32 rounding."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_support import dev_f32, empty_f32, say, sync

pytestmark = pytest.mark.gpu


def _dev_i64(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int64)).cuda()


def _run_budget(flat, offsets, params, s_t, lam, uniform):
    import torch
    import paper_2609_33977_amd as gm
    L = len(params)
    kept = torch.empty(L, dtype=torch.int64, device="cuda")  # uint64 counts, far below 2^63
    loss = torch.empty(1, dtype=torch.float64, device="cuda")
    coeff = empty_f32(L)
    d_off, d_par = _dev_i64(offsets), _dev_i64(params)
    gm.gm_budget_loss(dev_f32(flat), d_off, d_par, s_t, lam, uniform, kept, loss, coeff)
    sync()
    return (kept.cpu().numpy().astype(np.int64), float(loss.cpu().numpy()[0]), coeff.cpu().numpy().astype(np.float64),
            d_off)


def _check(flat, sizes, params, s_t, lam, uniform, tag):
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    kept, loss, coeff, _ = _run_budget(flat, offsets, params, s_t, lam, uniform)
    sel = np.split(flat, offsets[1:-1])
    L_ref, c_ref, k_ref = oracle.budget_loss(sel, params, s_t, lam, uniform)
    say(f"  {tag}: {len(sizes)} layers, {flat.size} selectors, loss {loss:.9g} (oracle {L_ref:.9g})")
    assert np.array_equal(kept, k_ref)
    assert abs(loss - L_ref) <= 1e-12 * abs(L_ref) + 1e-300
    assert np.allclose(coeff, c_ref, rtol=1e-6, atol=0.0)
    return offsets, coeff


@pytest.mark.parametrize("uniform", [False, True])
def test_budget_small_layers_of_mixed_shapes(uniform):
    # Layers smaller than one 4096-selector block, one straddling many blocks,
    # odd sizes (tails that are not multiples of 4), soft values counted as kept.
    r = workloads.gen.rng_for(950, int(uniform))
    sizes = [37, 4096, 5000, 3, 12289, 640, 1]
    params = [s * 256 for s in sizes]
    params[3] = 3 * 128  # a layer with another group size
    flat = np.concatenate([(r.uniform(size=n) < p).astype(np.float32) * r.uniform(0.2, 1.0, size=n).astype(np.float32)
                           for n, p in zip(sizes, (0.5, 0.3, 0.8, 0.5, 0.45, 0.6, 0.0))])
    _check(flat, sizes, params, 0.5, 16.0, uniform, f"mixed uniform={uniform}")


def test_budget_llama2_7b_batched_selectors():
    # The 224 selector matrices of LLaMA-2-7B with Beta-law kept counts that
    # meet the 50 % budget exactly: s = s_t, so the loss and every coefficient
    # vanish; one flipped selector moves s off the target.
    cfg = workloads.config("llama2_7b_step")
    g = cfg["g"]
    shapes = [(do, di) for _ in range(cfg["layers"]) for _, do, di in cfg["linears"]]
    sizes = [do * di // g for do, di in shapes]
    params = [do * di for do, di in shapes]
    kept, _ = workloads.kept_counts_beta_law(workloads.gen.rng_for(4, 0), sizes, params)
    r = workloads.gen.rng_for(950, 7)
    flat = np.concatenate([workloads.random_kept_mask(r, n, k) for n, k in zip(sizes, kept)])
    offsets, coeff = _check(flat, sizes, params, 0.5, 16.0, False, "llama2-7b at the target")
    assert np.all(coeff == 0.0)
    flat[int(np.flatnonzero(flat == 0)[0])] = 1.0
    _check(flat, sizes, params, 0.5, 16.0, False, "llama2-7b, one more kept")
    _check(flat, sizes, params, 0.5, 16.0, True, "llama2-7b uniform")


def test_budget_all_kept_layer_is_infinite_in_the_uniform_variant():
    flat = np.concatenate([np.ones(100, np.float32), (np.arange(300) % 2).astype(np.float32)])
    offsets = np.array([0, 100, 400], np.int64)
    kept, loss, coeff, _ = _run_budget(flat, offsets, [100 * 256, 300 * 256], 0.5, 16.0, True)
    assert list(kept) == [100, 150]
    assert np.isinf(loss) and np.isinf(coeff[0]) and coeff[1] == 0.0


@pytest.mark.parametrize("alias", [False, True])
def test_gate_bwd_budget_folds_the_coefficient(alias):
    import paper_2609_33977_amd as gm
    r = workloads.gen.rng_for(951, int(alias))
    sizes = [4093, 9000, 7]
    n = sum(sizes)
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    coeff = np.array([0.37, -1.25, 4.0], np.float32)
    dgate = r.standard_normal(n).astype(np.float32)
    y = r.uniform(0.01, 0.99, size=n).astype(np.float32)
    tau = 0.4
    d_dg, d_y, d_c = dev_f32(dgate), dev_f32(y), dev_f32(coeff)
    out = d_dg if alias else empty_f32(n)
    gm.gm_gate_bwd_budget(d_dg, d_y, tau, _dev_i64(offsets), d_c, out)
    sync()
    got = out.cpu().numpy().astype(np.float64)
    c_elem = np.repeat(coeff.astype(np.float64), sizes)
    ref = oracle.gate_bwd(dgate.astype(np.float64) + c_elem, y.astype(np.float64), tau)
    # relative to the magnitude of the terms (dgate + coeff can cancel)
    scale = (np.abs(dgate) + np.abs(c_elem)) * y * (1.0 - y) / tau
    err = np.max(np.abs(got - ref) / scale)
    say(f"  gate_bwd_budget alias={alias}: max rel err {err:.2e}")
    assert err <= 2e-6
