"""Pins of the fp64 oracle against what the paper and the mathematics fix.

None of these re-types an oracle formula: each compares the oracle with an
independent route (brute-force loops, a closed form, an identity that holds only
for the correct operator, a library routine on a special case, the paper's own
printed numbers).  The mutation test at the end plants plausible mistakes in
copies of the oracle functions and checks that at least one pin catches each.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import scipy.special

import oracle
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand(shape, key, scale=1.0):
    return workloads.gen.rng_for(900, *key).standard_normal(shape) * scale


def _soft_mask(shape, key, p_zero=0.4):
    r = workloads.gen.rng_for(901, *key)
    m = r.uniform(0.05, 1.5, size=shape)
    m[r.uniform(size=shape) < p_zero] = 0.0
    return m


# ----------------------------------------------------------- brute force (loops)

def _brute_fwd(X, W, B, g, g_out=1):
    T, d_in = X.shape
    d_out = W.shape[0]
    Y = [[0.0] * d_out for _ in range(T)]
    for t in range(T):
        for o in range(d_out):
            acc = 0.0
            for i in range(d_in):
                acc += X[t][i] * W[o][i] * B[o // g_out][i // g]
            Y[t][o] = acc
    return np.array(Y)


def _brute_dx(dY, W, B, g, g_out=1):
    T, d_out = dY.shape
    d_in = W.shape[1]
    dX = [[0.0] * d_in for _ in range(T)]
    for t in range(T):
        for i in range(d_in):
            acc = 0.0
            for o in range(d_out):
                acc += dY[t][o] * W[o][i] * B[o // g_out][i // g]
            dX[t][i] = acc
    return np.array(dX)


def _brute_dgate(dY, X, W, g, g_out=1):
    T, d_out = dY.shape
    d_in = X.shape[1]
    out = [[0.0] * (d_in // g) for _ in range(d_out // g_out)]
    for u in range(d_out // g_out):
        for v in range(d_in // g):
            acc = 0.0
            for o in range(u * g_out, (u + 1) * g_out):
                for i in range(v * g, (v + 1) * g):
                    for t in range(T):
                        acc += dY[t][o] * X[t][i] * W[o][i]
            out[u][v] = acc
    return np.array(out)


# (T, d_out, G_in, g, g_out): 1 x g groups and 2-D g_out x g groups
TINY = [(3, 5, 2, 4, 1), (2, 4, 3, 2, 1), (4, 3, 1, 8, 1), (1, 6, 4, 1, 1), (3, 6, 2, 4, 3), (2, 8, 3, 2, 2),
        (2, 4, 2, 4, 4)]


@pytest.mark.parametrize("T,d_out,G_in,g,g_out", TINY)
def test_fwd_matches_brute_force(T, d_out, G_in, g, g_out):
    d_in = G_in * g
    X, W = _rand((T, d_in), (1, T)), _rand((d_out, d_in), (2, T))
    B = _soft_mask((d_out // g_out, G_in), (3, T, g_out))
    np.testing.assert_allclose(oracle.linear_fwd(X, W, B, g, g_out), _brute_fwd(X, W, B, g, g_out), rtol=1e-12,
                               atol=1e-12)


@pytest.mark.parametrize("T,d_out,G_in,g,g_out", TINY)
def test_dx_matches_brute_force(T, d_out, G_in, g, g_out):
    d_in = G_in * g
    dY, W = _rand((T, d_out), (4, T)), _rand((d_out, d_in), (5, T))
    B = _soft_mask((d_out // g_out, G_in), (6, T, g_out))
    np.testing.assert_allclose(oracle.linear_bwd_dx(dY, W, B, g, g_out), _brute_dx(dY, W, B, g, g_out), rtol=1e-12,
                               atol=1e-12)


@pytest.mark.parametrize("T,d_out,G_in,g,g_out", TINY)
def test_dgate_matches_brute_force(T, d_out, G_in, g, g_out):
    d_in = G_in * g
    dY, X, W = _rand((T, d_out), (7, T)), _rand((T, d_in), (8, T)), _rand((d_out, d_in), (9, T))
    np.testing.assert_allclose(oracle.linear_bwd_dgate(dY, X, W, g, g_out), _brute_dgate(dY, X, W, g, g_out),
                               rtol=1e-12, atol=1e-12)


def test_square_group_gradient_sums_the_row_gradients_of_its_block():
    # A g_out x g group is the union of g_out row groups 1 x g sharing one
    # selector: its gradient is the sum of theirs (Y is linear in each selector).
    T, d_out, d_in, g, g_out = 5, 12, 16, 4, 3
    dY, X, W = _rand((T, d_out), (40,)), _rand((T, d_in), (41,)), _rand((d_out, d_in), (42,))
    rows = oracle.linear_bwd_dgate(dY, X, W, g)
    np.testing.assert_allclose(oracle.linear_bwd_dgate(dY, X, W, g, g_out),
                               rows.reshape(d_out // g_out, g_out, d_in // g).sum(axis=1), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("h", [0.5, 3.0])
def test_square_group_dgate_matches_central_finite_differences(h):
    T, d_out, d_in, g, g_out = 4, 8, 12, 4, 2
    dY, X, W = _rand((T, d_out), (43,)), _rand((T, d_in), (44,)), _rand((d_out, d_in), (45,))
    B = _soft_mask((d_out // g_out, d_in // g), (46,))
    dg = oracle.linear_bwd_dgate(dY, X, W, g, g_out)
    for u, v in itertools.product(range(d_out // g_out), range(d_in // g)):
        Bp, Bm = B.copy(), B.copy()
        Bp[u, v] += h
        Bm[u, v] -= h
        fd = (np.sum(dY * oracle.linear_fwd(X, W, Bp, g, g_out)) - np.sum(dY * oracle.linear_fwd(X, W, Bm, g, g_out))) / (2 * h)
        assert abs(fd - dg[u, v]) <= 1e-10 * (1 + abs(dg[u, v]))


def test_single_square_group_scales_the_dense_layer():
    T, d_out, d_in = 3, 6, 8
    X, W = _rand((T, d_in), (47,)), _rand((d_out, d_in), (48,))
    for b in (0.0, 0.3, 1.0):
        np.testing.assert_allclose(oracle.linear_fwd(X, W, np.array([[b]]), d_in, d_out), b * np.matmul(X, W.T),
                                   rtol=1e-13, atol=1e-13)


# ----------------------------------------------------------- special cases (Eq. 1)

def test_all_ones_mask_is_dense_linear():
    # Teacher pass: B = 1 gives the dense frozen layer (Sec. 2.4).
    T, d_out, d_in, g = 7, 12, 32, 8
    X, W, dY = _rand((T, d_in), (10,)), _rand((d_out, d_in), (11,)), _rand((T, d_out), (12,))
    ones = np.ones((d_out, d_in // g))
    np.testing.assert_allclose(oracle.linear_fwd(X, W, ones, g), np.matmul(X, W.T), rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(oracle.linear_bwd_dx(dY, W, ones, g), np.matmul(dY, W), rtol=1e-13, atol=1e-13)


def test_all_zeros_mask_gives_exact_zero():
    T, d_out, d_in, g = 5, 8, 16, 4
    X, W, dY = _rand((T, d_in), (13,)), _rand((d_out, d_in), (14,)), _rand((T, d_out), (15,))
    zeros = np.zeros((d_out, d_in // g))
    assert np.all(oracle.linear_fwd(X, W, zeros, g) == 0.0)
    assert np.all(oracle.linear_bwd_dx(dY, W, zeros, g) == 0.0)


def test_group_spanning_whole_row_is_output_row_pruning():
    T, d_out, d_in = 6, 10, 24
    X, W = _rand((T, d_in), (16,)), _rand((d_out, d_in), (17,))
    keep = (np.arange(d_out) % 3 != 1).astype(float)[:, None]
    Y = oracle.linear_fwd(X, W, keep, d_in)
    dense = np.matmul(X, W.T)
    for o in range(d_out):
        if keep[o, 0]:
            np.testing.assert_allclose(Y[:, o], dense[:, o], rtol=1e-13, atol=1e-13)
        else:
            assert np.all(Y[:, o] == 0.0)


def test_unit_groups_give_textbook_mask_gradient():
    # g = 1 is an elementwise mask: d<dY, X (W*M)^T>/dM = W * (dY^T X).
    T, d_out, d_in = 9, 7, 5
    dY, X, W = _rand((T, d_out), (18,)), _rand((T, d_in), (19,)), _rand((d_out, d_in), (20,))
    ref = W * np.einsum("to,ti->oi", dY, X)
    np.testing.assert_allclose(oracle.linear_bwd_dgate(dY, X, W, 1), ref, rtol=1e-12, atol=1e-12)


def test_expand_mask_is_kronecker_block_layout():
    B = np.array([[1.0, 0.0, 2.0], [0.0, 3.0, 0.0]])
    M = oracle.expand_mask(B, 2, 3)
    assert M.shape == (6, 6)
    for r, c in itertools.product(range(6), range(6)):
        assert M[r, c] == B[r // 3, c // 2]


# --------------------------------------------------- identities of the backward

def test_dx_is_the_adjoint_of_the_forward():
    T, d_out, G_in, g = 6, 9, 3, 4
    d_in = G_in * g
    W, B, dY = _rand((d_out, d_in), (21,)), _soft_mask((d_out, G_in), (22,)), _rand((T, d_out), (23,))
    dX = oracle.linear_bwd_dx(dY, W, B, g)
    for k in range(3):
        X = _rand((T, d_in), (24, k))
        lhs = float(np.sum(dX * X))
        rhs = float(np.sum(dY * oracle.linear_fwd(X, W, B, g)))
        assert lhs == pytest.approx(rhs, rel=1e-12, abs=1e-12)


@pytest.mark.parametrize("h", [1e-3, 0.5, 3.0])
def test_dgate_matches_central_finite_differences(h):
    # <dY, Y(B)> is linear in every selector, so the central difference is exact for any h.
    T, d_out, G_in, g = 4, 5, 3, 4
    d_in = G_in * g
    dY, X, W = _rand((T, d_out), (25,)), _rand((T, d_in), (26,)), _rand((d_out, d_in), (27,))
    B = _soft_mask((d_out, G_in), (28,))
    dgate = oracle.linear_bwd_dgate(dY, X, W, g)
    for o, v in itertools.product(range(d_out), range(G_in)):
        Bp, Bm = B.copy(), B.copy()
        Bp[o, v] += h
        Bm[o, v] -= h
        fd = (np.sum(dY * oracle.linear_fwd(X, W, Bp, g)) - np.sum(dY * oracle.linear_fwd(X, W, Bm, g))) / (2 * h)
        assert fd == pytest.approx(dgate[o, v], rel=1e-9, abs=1e-9)


def test_dgate_euler_and_row_sum_identities():
    T, d_out, G_in, g = 8, 6, 4, 8
    d_in = G_in * g
    dY, X, W = _rand((T, d_out), (29,)), _rand((T, d_in), (30,)), _rand((d_out, d_in), (31,))
    B = _soft_mask((d_out, G_in), (32,))
    dgate = oracle.linear_bwd_dgate(dY, X, W, g)
    # Euler: Y is homogeneous of degree one in the selectors.
    assert float(np.sum(B * dgate)) == pytest.approx(float(np.sum(dY * oracle.linear_fwd(X, W, B, g))), rel=1e-12)
    # Summing a row's groups recovers the dense row's contribution.
    dense = np.matmul(X, W.T)
    np.testing.assert_allclose(dgate.sum(axis=1), np.sum(dY * dense, axis=0), rtol=1e-12, atol=1e-12)


def test_dgate_two_factorisations_agree():
    # sum_i W[o,i] (dY^T X)[o,i] over a group == sum_t dY[t,o] (X[t,group] . W[o,group]).
    T, d_out, G_in, g = 5, 4, 3, 8
    d_in = G_in * g
    dY, X, W = _rand((T, d_out), (33,)), _rand((T, d_in), (34,)), _rand((d_out, d_in), (35,))
    per_token = np.zeros((d_out, G_in))
    for o in range(d_out):
        for v in range(G_in):
            cols = slice(v * g, (v + 1) * g)
            per_token[o, v] = float(np.dot(dY[:, o], X[:, cols] @ W[o, cols]))
    np.testing.assert_allclose(oracle.linear_bwd_dgate(dY, X, W, g), per_token, rtol=1e-12, atol=1e-12)


# --------------------------------------------------------------- gate (Sec. 2.2)

def test_hard_gate_is_thresholded_sigmoid():
    r = workloads.gen.rng_for(40)
    logits = r.standard_normal(4096) * 3
    u = workloads.draw_uniform_noise(r, 4096).astype(np.float64)
    for tau in (0.25, 0.4, 0.5, 2.0):
        m, y = oracle.gate(logits, u, tau, hard=True)
        y_ref = scipy.special.expit((logits + scipy.special.logit(u)) / tau)
        np.testing.assert_allclose(y, y_ref, rtol=1e-12, atol=1e-15)
        assert np.array_equal(m, (y_ref > 0.5).astype(float))
        ms, ys = oracle.gate(logits, u, tau, hard=False)
        np.testing.assert_allclose(ms, y_ref, rtol=1e-12, atol=1e-15)


def test_hard_gate_does_not_depend_on_temperature():
    r = workloads.gen.rng_for(41)
    logits = r.standard_normal(2048)
    u = workloads.draw_uniform_noise(r, 2048)
    ref, _ = oracle.gate(logits, u, 1.0, True)
    for tau in (0.1, 0.4, 0.5, 7.0):
        assert np.array_equal(oracle.gate(logits, u, tau, True)[0], ref)


def test_noise_is_neutral_at_one_half_and_antisymmetric():
    assert oracle.logistic_noise(0.5) == 0.0
    u = np.array([2.0 ** -20, 0.125, 0.3125, 0.4375])  # dyadic, so 1 - u is exact
    np.testing.assert_allclose(oracle.logistic_noise(u), -oracle.logistic_noise(1 - u), rtol=1e-12)
    _, y1 = oracle.gate([0.7], [0.5], 0.4, False)
    assert y1[0] == pytest.approx(1 / (1 + math.exp(-0.7 / 0.4)), rel=1e-15)


def test_sigmoid_symmetry():
    z = np.linspace(-8, 8, 97)
    _, yp = oracle.gate(z, None, 0.5, False)
    _, ym = oracle.gate(-z, None, 0.5, False)
    np.testing.assert_allclose(yp + ym, 1.0, rtol=0, atol=1e-15)


def test_eval_mode_thresholds_logits():
    logits = np.array([-2.0, -1e-30, 0.0, 1e-30, 3.0])
    m, _ = oracle.gate(logits, None, 0.4, True)
    assert m.tolist() == [0.0, 0.0, 0.0, 1.0, 1.0]


def test_keep_probability_is_sigmoid_of_logit():
    # Binary-concrete property: with u ~ U(0,1), P(logit + ln u - ln(1-u) > 0) = sigmoid(logit).
    r = workloads.gen.rng_for(42)
    n = 200_000
    for logit in (-1.5, 0.0, 0.8):
        u = workloads.draw_uniform_noise(r, n)
        m, _ = oracle.gate(np.full(n, logit), u, 0.4, True)
        p = 1 / (1 + math.exp(-logit))
        assert abs(m.mean() - p) < 5 * math.sqrt(p * (1 - p) / n)


def test_ste_derivative_matches_finite_difference_of_relaxation():
    r = workloads.gen.rng_for(43)
    logits = r.standard_normal(64)
    u = workloads.draw_uniform_noise(r, 64)
    up = r.standard_normal(64)
    for tau in (0.4, 0.5):
        _, y = oracle.gate(logits, u, tau, False)
        dl = oracle.gate_bwd(up, y, tau)
        h = 1e-6
        yp = scipy.special.expit((logits + h + scipy.special.logit(u.astype(float))) / tau)
        ym = scipy.special.expit((logits - h + scipy.special.logit(u.astype(float))) / tau)
        np.testing.assert_allclose(dl, up * (yp - ym) / (2 * h), rtol=1e-6, atol=1e-9)


def test_near_threshold_band():
    y = np.array([0.5, 0.5 + 0.9e-6, 0.5 - 2e-6, 0.7])
    assert oracle.near_threshold(y).tolist() == [True, True, False, False]


# ------------------------------------------------- budget and sparsity (Eq. 2)

def test_budgeted_inputs_give_exact_kept_count():
    case = workloads.make_linear_case((44,), 4, 1024, 1024, 256, 2048, tau=0.5)
    m, y = oracle.gate(case.logits, case.noise, case.tau, True)
    assert oracle.kept_count(m) == 2048
    assert np.array_equal(m, case.mask.astype(float))
    assert not oracle.near_threshold(y).any()


def test_sparsity_closed_forms():
    shapes = [(4, 8), (2, 8)]
    B1 = np.ones((4, 2))
    B2 = np.zeros((2, 2))
    s_l, s = oracle.sparsity([B1, B2], shapes)
    assert s_l == [0.0, 1.0]
    assert s == pytest.approx(16 / 48)
    B1[0, 0] = 0
    s_l, s = oracle.sparsity([B1, B2], shapes)
    assert s_l[0] == pytest.approx(1 / 8)
    assert s == pytest.approx((32 / 8 + 16) / 48)


def test_paper_category_rates_reproduce_global_rate():
    """Sec. 3.5 prints 36.6 % kept for attention, 56.6 % for MLP and 49.98 % overall."""
    with open(os.path.join(GOLDEN, "paper_preserved_rates.json")) as f:
        gold = json.load(f)
    selectors, shapes = [], []
    for _layer in range(32):
        for name, d_out, d_in in workloads.LLAMA2_7B_LINEARS:
            rate = gold["attention_preserved"] if name in ("q", "k", "v", "o") else gold["mlp_preserved"]
            G = (d_out * d_in) // 256
            B = np.zeros(G)
            B[: int(round(rate * G))] = 1
            selectors.append(B)
            shapes.append((d_out, d_in))
    _, s = oracle.sparsity(selectors, shapes)
    assert abs((1 - s) - gold["global_preserved"]) <= gold["printed_precision"]


def test_preserved_rate_counts_active_weights():
    B = np.array([[1, 0, 1, 1], [0, 0, 1, 0]])
    assert oracle.preserved_rate(B, 3) == pytest.approx(4 / 8)
    with open(os.path.join(GOLDEN, "paper_decision_count.json")) as f:
        gold = json.load(f)
    d_out, d_in = 512, 1024
    B = np.ones((d_out // gold["g_out"], d_in // gold["g_in"]))
    assert (d_out * d_in) / B.size == gold["reduction_factor"]


def test_kept_count_and_preserved_rate_away_from_one_half():
    """At 3 of 8 kept, counting the pruned groups (5) or the pruned weights (5/8) instead fails."""
    B = np.array([[1, 0, 0, 1], [0, 0, 0.25, 0]])  # a fractional selector is kept too (only zeros prune)
    assert oracle.kept_count(B) == 3
    assert oracle.preserved_rate(B, 3) == pytest.approx(3 / 8)
    # 2-D groups: each selector covers g_out x g weights, so the rate is still 3 of 8 selectors
    assert oracle.preserved_rate(B, 4, 2) == pytest.approx(3 / 8)
    # element count after the Kronecker expansion, one weight at a time
    M = oracle.expand_mask((B != 0).astype(float), 5, 3)
    assert M.shape == (6, 20) and int(M.sum()) == 3 * 15
    # Eq. 2 on the same matrix: s = 1 - 3/8 (a layer of 6 x 20 weights, one layer)
    s_l, s = oracle.sparsity([B], [(6, 20)])
    assert s_l == [pytest.approx(5 / 8)] and s == pytest.approx(5 / 8)


# ------------------------------------------------------------- bf16 widening

def _bf16_closed_form(bits: int) -> float:
    """Value of a finite bf16 pattern from its fields: sign, 8-bit exponent (bias 127), 7-bit fraction."""
    sign = -1.0 if bits >> 15 else 1.0
    e, f = (bits >> 7) & 0xFF, bits & 0x7F
    if e == 0:
        return sign * math.ldexp(f / 128.0, -126)  # subnormal (and signed zero)
    return sign * math.ldexp(1.0 + f / 128.0, e - 127)


def test_from_bf16_is_exact_over_every_bit_pattern():
    """Every one of the 65,536 patterns: equal to torch's bfloat16 -> float64 widening (NaNs stay NaN),
    and every finite one equal to the value its sign, exponent and fraction fields define."""
    import torch
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    got = oracle.from_bf16(bits)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(got, ref)  # NaN positions must agree as well
    assert np.array_equal(np.signbit(got), np.signbit(ref))  # -0 stays -0
    finite = ((bits >> 7) & 0xFF) != 0xFF
    assert int(finite.sum()) == 65536 - 256  # exponent field all ones: 2 signs x 128 fractions
    closed = np.array([_bf16_closed_form(int(b)) for b in bits[finite]])
    np.testing.assert_array_equal(got[finite], closed)
    assert np.all(np.isinf(got[((bits & 0x7FFF) == 0x7F80)]))


# ------------------------------------------- sparsity-budget regulariser (Sec. 2.3)

def _budget_layers():
    """Three layers of different shapes and group sizes, about half of the groups kept."""
    r = workloads.gen.rng_for(902)
    shapes = [(48, 512, 256), (96, 1024, 256), (40, 768, 128)]  # (d_out, d_in, g)
    B = [(r.uniform(size=(do, di // g)) < p).astype(np.float64) for (do, di, g), p in zip(shapes, (0.3, 0.55, 0.7))]
    params = [do * di for do, di, _ in shapes]
    return shapes, B, params


def _with_pruned(B, target_pruned):
    """Copy of a single selector matrix with exactly target_pruned zeros (first in row-major order)."""
    flat = np.ones(np.asarray(B).size)
    flat[:target_pruned] = 0.0
    return flat.reshape(np.asarray(B).shape)


def test_budget_loss_vanishes_at_the_target():
    B = _with_pruned(np.zeros((40, 25)), 400)  # s = 0.4 exactly
    for uniform in (False, True):
        L, coeff, kept = oracle.budget_loss([B], [40 * 25 * 256], 0.4, 16.0, uniform)
        assert L == 0.0 and np.all(coeff == 0.0) and kept[0] == 600


def test_budget_loss_depends_only_on_the_ratio():
    # Sec. 2.3: s = c s_t and s = s_t / c get the same penalty.
    s_t, c, G = 0.4, 1.25, 1000
    Lhi, _, _ = oracle.budget_loss([_with_pruned(np.zeros(G), int(round(c * s_t * G)))], [G * 256], s_t, 16.0)
    Llo, _, _ = oracle.budget_loss([_with_pruned(np.zeros(G), int(round(s_t / c * G)))], [G * 256], s_t, 16.0)
    assert Lhi > 0 and abs(Lhi - Llo) <= 1e-12 * Lhi
    assert abs(Lhi - 16.0 * math.log(c)) <= 1e-12


def test_budget_global_sparsity_is_the_fraction_of_pruned_weights():
    # Eq. 2 weights s^l by d_out d_in: the result is the fraction of zero
    # weights over every element of every layer, counted after expansion.
    shapes, B, params = _budget_layers()
    zeros = sum(float(np.sum(oracle.expand_mask(b, g) == 0)) for b, (_, _, g) in zip(B, shapes))
    total = float(sum(params))
    s_elem = zeros / total
    L, _, _ = oracle.budget_loss(B, params, 0.5, 16.0)
    assert abs(L - 16.0 * abs(math.log(s_elem / 0.5))) <= 1e-12


@pytest.mark.parametrize("uniform", [False, True])
def test_budget_gradient_matches_selector_flips(uniform):
    # Central difference in the kept count: one selector of layer l goes from
    # 1 to 0 (B-) and another from 0 to 1 (B+); (L(B+) - L(B-)) / 2 is dL/dB^l
    # up to the curvature of the log over one flip, relative (ds/s)^2 / 3 with
    # ds/s below 5e-3 for these layers, so 1e-4 is a safe bound.
    shapes, B, params = _budget_layers()
    _, coeff, _ = oracle.budget_loss(B, params, 0.5, 16.0, uniform)
    for l in range(len(B)):
        flat = B[l].ravel()
        on, off = int(np.flatnonzero(flat)[0]), int(np.flatnonzero(flat == 0)[0])
        Bp = [b.copy() for b in B]
        Bm = [b.copy() for b in B]
        Bp[l].ravel()[off] = 1.0
        Bm[l].ravel()[on] = 0.0
        Lp, _, _ = oracle.budget_loss(Bp, params, 0.5, 16.0, uniform)
        Lm, _, _ = oracle.budget_loss(Bm, params, 0.5, 16.0, uniform)
        fd = (Lp - Lm) / 2.0
        assert abs(fd - coeff[l]) <= 1e-4 * abs(coeff[l]) + 1e-15, (l, fd, coeff[l])


def test_budget_uniform_variant_is_the_sum_of_single_layer_losses():
    shapes, B, params = _budget_layers()
    Lu, cu, _ = oracle.budget_loss(B, params, 0.5, 16.0, uniform=True)
    singles = [oracle.budget_loss([b], [p], 0.5, 16.0) for b, p in zip(B, params)]
    assert abs(Lu - sum(x[0] for x in singles)) <= 1e-12 * Lu
    assert np.allclose(cu, [x[1][0] for x in singles], rtol=1e-12, atol=0)


# ------------------------------------------- distillation loss (Sec. 2.4, Eq. 4)

def _distill_case(N, V, d, key, noise=0.5, w_scale=1.0):
    H_t = _rand((N, d), (60,) + key)
    H_s = H_t + noise * _rand((N, d), (61,) + key)
    W = _rand((V, d), (62,) + key, w_scale)
    return H_t, H_s, W


def test_distill_matches_brute_force_loops():
    H_t, H_s, W = _distill_case(3, 5, 4, (0,))
    total = 0.0
    for t in range(3):
        zt = [sum(H_t[t][j] * W[v][j] for j in range(4)) for v in range(5)]
        zs = [sum(H_s[t][j] * W[v][j] for j in range(4)) for v in range(5)]
        et, es = [math.exp(x) for x in zt], [math.exp(x) for x in zs]
        total -= sum(et[v] / sum(et) * math.log(es[v] / sum(es)) for v in range(5))
    L, ce, _, _ = oracle.distill_loss(H_t, H_s, W)
    assert abs(L - total / 3) <= 1e-12 * abs(total)
    assert abs(ce.mean() - total / 3) <= 1e-12 * abs(total)


def test_distill_is_kl_plus_teacher_entropy():
    # the identity stated after Eq. 4: cross-entropy = KL(p_T || p_S) + H(p_T)
    from scipy.special import entr, rel_entr, softmax
    H_t, H_s, W = _distill_case(6, 40, 16, (1,), w_scale=0.7)
    p_t, p_s = softmax(H_t @ W.T, axis=1), softmax(H_s @ W.T, axis=1)
    ref = (rel_entr(p_t, p_s).sum(axis=1) + entr(p_t).sum(axis=1)).mean()
    L, _, _, _ = oracle.distill_loss(H_t, H_s, W)
    assert abs(L - ref) <= 1e-12 * abs(ref)


def test_distill_of_identical_passes_is_teacher_entropy_with_zero_gradient():
    from scipy.special import softmax
    from scipy.stats import entropy
    H_t, H_s, W = _distill_case(5, 30, 12, (2,))
    L0, _, _, _ = oracle.distill_loss(H_t, H_t, W)
    assert abs(L0 - entropy(softmax(H_t @ W.T, axis=1), axis=1).mean()) <= 1e-12 * L0
    assert not np.any(oracle.distill_loss_bwd(H_t, H_t, W))
    L1, ce1, _, _ = oracle.distill_loss(H_t, H_s, W)
    _, ce0, _, _ = oracle.distill_loss(H_t, H_t, W)
    assert L1 > L0 and np.all(ce1 >= ce0)  # Gibbs: cross-entropy >= entropy


def test_distill_one_hot_teacher_is_cross_entropy():
    from scipy.special import log_softmax
    N, V, d = 4, 9, 64
    _, H_s, W = _distill_case(N, V, d, (3,))
    k = np.array([2, 7, 0, 7])
    H_t = 200.0 * W[k] / np.linalg.norm(W[k], axis=1, keepdims=True)  # the target row dominates by > 700 nats
    L, _, _, _ = oracle.distill_loss(H_t, H_s, W)
    ref = -log_softmax(H_s @ W.T, axis=1)[np.arange(N), k].mean()
    assert abs(L - ref) <= 1e-12 * abs(ref)


def test_distill_uniform_teacher():
    from scipy.special import logsumexp
    _, H_s, W = _distill_case(5, 17, 8, (4,))
    L, _, lse_t, lse_s = oracle.distill_loss(np.zeros_like(H_s), H_s, W)
    z = H_s @ W.T
    ref = (logsumexp(z, axis=1) - z.mean(axis=1)).mean()
    assert abs(L - ref) <= 1e-12 * abs(ref)
    assert np.allclose(lse_t, np.log(17.0), rtol=1e-15, atol=0)
    assert np.allclose(lse_s, logsumexp(z, axis=1), rtol=1e-13, atol=0)


def test_distill_gradient_matches_finite_differences():
    H_t, H_s, W = _distill_case(4, 11, 6, (5,))
    dH = oracle.distill_loss_bwd(H_t, H_s, W)
    h = 1e-5
    for t, j in itertools.product(range(4), range(6)):
        Hp, Hm = H_s.copy(), H_s.copy()
        Hp[t, j] += h
        Hm[t, j] -= h
        fd = (oracle.distill_loss(H_t, Hp, W)[0] - oracle.distill_loss(H_t, Hm, W)[0]) / (2 * h)
        assert abs(fd - dH[t, j]) <= 1e-8 * (1 + abs(dH[t, j]))


def test_distill_counts_only_valid_tokens():
    H_t, H_s, W = _distill_case(7, 13, 5, (6,))
    valid = np.array([1, 0, 1, 1, 0, 0, 1], dtype=np.uint8)
    sub = valid != 0
    L, ce, _, _ = oracle.distill_loss(H_t, H_s, W, valid)
    L_sub, ce_sub, _, _ = oracle.distill_loss(H_t[sub], H_s[sub], W)
    assert abs(L - L_sub) <= 1e-14 * abs(L_sub)
    assert np.array_equal(ce[sub], ce_sub)
    dH = oracle.distill_loss_bwd(H_t, H_s, W, valid)
    assert not np.any(dH[~sub])
    np.testing.assert_allclose(dH[sub], oracle.distill_loss_bwd(H_t[sub], H_s[sub], W), rtol=1e-14, atol=0)
    none = np.zeros(7, dtype=np.uint8)
    assert oracle.distill_loss(H_t, H_s, W, none)[0] == 0.0
    assert not np.any(oracle.distill_loss_bwd(H_t, H_s, W, none))


# ----------------------------------------------- hypernetwork (Sec. 2.2, Eq. 3)

def _hyper_case(L, D, H, sizes, key):
    P = 2 * sum(int(np.prod(shp)) for shp in oracle.gru_param_shapes(D, H))
    z = _rand((L, D), (70,) + key)
    gru = _rand((P,), (71,) + key, 0.4)
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    A = _rand((int(offsets[-1]), 2 * H), (72,) + key, 0.3)
    c = _rand((int(offsets[-1]),), (73,) + key, 0.1)
    return z, gru, A, c, offsets


def _torch_hyper(z, gru, A, c, offsets, H):
    import torch
    D = z.shape[1]
    net = torch.nn.GRU(D, H, bidirectional=True, batch_first=True).double()
    params = [net.weight_ih_l0, net.weight_hh_l0, net.bias_ih_l0, net.bias_hh_l0,
              net.weight_ih_l0_reverse, net.weight_hh_l0_reverse, net.bias_ih_l0_reverse, net.bias_hh_l0_reverse]
    pos = 0
    with torch.no_grad():
        for prm in params:
            n = prm.numel()
            prm.copy_(torch.from_numpy(gru[pos:pos + n].reshape(prm.shape)))
            pos += n
    tA = torch.tensor(A, requires_grad=True)
    tc = torch.tensor(c, requires_grad=True)
    o = net(torch.from_numpy(z)[None])[0][0]
    rows = [tA[offsets[l]:offsets[l + 1]] @ o[l] + tc[offsets[l]:offsets[l + 1]] for l in range(len(offsets) - 1)]
    return torch.cat(rows), tA, tc, params


@pytest.mark.parametrize("L,D,H", [(5, 6, 4), (9, 3, 7), (1, 4, 2)])
def test_bigru_matches_torch_gru(L, D, H):
    import torch
    z, gru, A, c, offsets = _hyper_case(L, D, H, [3] * L, (L, D, H))
    logits, _, _, _ = _torch_hyper(z, gru, A, c, offsets, H)
    np.testing.assert_allclose(oracle.hyper_fwd(z, gru, A, c, offsets, H), logits.detach().numpy(), rtol=1e-12,
                               atol=1e-13)
    del torch


def test_hyper_heads_match_loops():
    L, D, H = 3, 4, 2
    z, gru, A, c, offsets = _hyper_case(L, D, H, [2, 5, 1], (1,))
    o = oracle.bigru_fwd(z, gru, H)
    got = oracle.hyper_fwd(z, gru, A, c, offsets, H)
    for l in range(L):
        for e in range(offsets[l], offsets[l + 1]):
            ref = c[e] + sum(A[e][k] * o[l][k] for k in range(2 * H))
            assert abs(got[e] - ref) <= 1e-13


@pytest.mark.parametrize("L,D,H", [(6, 5, 3), (4, 8, 4)])
def test_hyper_gradients_match_autograd(L, D, H):
    import torch
    sizes = [7, 1, 4, 9, 2, 3, 5, 6][:L]
    z, gru, A, c, offsets = _hyper_case(L, D, H, sizes, (2, L))
    dl = _rand((int(offsets[-1]),), (74, L))
    logits, tA, tc, params = _torch_hyper(z, gru, A, c, offsets, H)
    (logits * torch.from_numpy(dl)).sum().backward()
    dA, dc, dgru, _ = oracle.hyper_bwd(dl, z, gru, A, c, offsets, H)
    np.testing.assert_allclose(dA, tA.grad.numpy(), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(dc, tc.grad.numpy(), rtol=1e-12, atol=1e-13)
    ref = np.concatenate([prm.grad.numpy().reshape(-1) for prm in params])
    np.testing.assert_allclose(dgru, ref, rtol=1e-10, atol=1e-12)


def test_hyper_gru_gradient_matches_finite_differences():
    L, D, H = 4, 3, 3
    z, gru, A, c, offsets = _hyper_case(L, D, H, [2, 3, 1, 2], (3,))
    dl = _rand((int(offsets[-1]),), (75,))
    _, _, dgru, _ = oracle.hyper_bwd(dl, z, gru, A, c, offsets, H)
    h = 1e-6
    for k in range(0, gru.size, 5):
        gp, gm_ = gru.copy(), gru.copy()
        gp[k] += h
        gm_[k] -= h
        fd = (dl @ oracle.hyper_fwd(z, gp, A, c, offsets, H) - dl @ oracle.hyper_fwd(z, gm_, A, c, offsets, H)) / (2 * h)
        assert abs(fd - dgru[k]) <= 1e-7 * (1 + abs(dgru[k]))


def test_adamw_matches_torch():
    import torch
    r = workloads.gen.rng_for(76)
    p0 = r.standard_normal(50)
    grads = [r.standard_normal(50) * 10.0 ** (-k) for k in range(4)]
    tp = torch.tensor(p0, requires_grad=True)
    opt = torch.optim.AdamW([tp], lr=1e-3, betas=(0.9, 0.999), eps=1e-8, weight_decay=0.05)
    p, m, v = p0.copy(), np.zeros(50), np.zeros(50)
    for step, gr in enumerate(grads, start=1):
        tp.grad = torch.from_numpy(gr.copy())
        opt.step()
        p, m, v = oracle.adamw_step(p, gr, m, v, 1e-3, 0.9, 0.999, 1e-8, 0.05, step)
        np.testing.assert_allclose(p, tp.detach().numpy(), rtol=1e-14, atol=1e-15)
        st = opt.state[tp]
        np.testing.assert_allclose(m, st["exp_avg"].numpy(), rtol=1e-14, atol=0)
        np.testing.assert_allclose(v, st["exp_avg_sq"].numpy(), rtol=1e-14, atol=0)


# ------------------------------------------------------- the pins catch mistakes

def _mutant_fwd_strided_groups(X, W, B, g, g_out=1):
    # selector v applied to columns v, v + G_in, v + 2 G_in, ... instead of a contiguous block
    M = np.tile(np.repeat(np.asarray(B, dtype=float), g_out, axis=0), (1, g))
    return np.asarray(X, float) @ (np.asarray(W, float) * M).T


def _mutant_fwd_strided_rows(X, W, B, g, g_out=1):
    # row block u applied to rows u, u + G_out, ... instead of g_out consecutive rows
    M = np.tile(np.repeat(np.asarray(B, dtype=float), g, axis=1), (g_out, 1))
    return np.asarray(X, float) @ (np.asarray(W, float) * M).T


def _mutant_dgate_no_weight(dY, X, W, g, g_out=1):
    d_out, d_in = np.asarray(W).shape
    G = np.asarray(dY, float).T @ np.asarray(X, float)
    return G.reshape(d_out // g_out, g_out, d_in // g, g).sum(axis=(1, 3))


def _mutant_dgate_strided_groups(dY, X, W, g, g_out=1):
    d_out, d_in = np.asarray(W).shape
    G = np.asarray(dY, float).T @ np.asarray(X, float)
    return (np.asarray(W, float) * G).reshape(d_out // g_out, g_out, g, d_in // g).sum(axis=(1, 2))


def _mutant_dgate_first_row_only(dY, X, W, g, g_out=1):
    # a 2-D group's gradient taken from the first of its rows alone
    d_out, d_in = np.asarray(W).shape
    G = np.asarray(dY, float).T @ np.asarray(X, float)
    return (np.asarray(W, float) * G).reshape(d_out // g_out, g_out, d_in // g, g)[:, 0].sum(axis=2)


def _mutant_dx_unmasked(dY, W, B, g, g_out=1):
    return np.asarray(dY, float) @ np.asarray(W, float)


def _mutant_dx_strided_rows(dY, W, B, g, g_out=1):
    M = np.tile(np.repeat(np.asarray(B, dtype=float), g, axis=1), (g_out, 1))
    return np.asarray(dY, float) @ (np.asarray(W, float) * M)


def _mutant_gate_sign(logits, noise, tau, hard):
    z = np.asarray(logits, float)
    if noise is not None:
        z = z - oracle.logistic_noise(noise)
    y = 1 / (1 + np.exp(-z / tau))
    return ((y > 0.5).astype(float) if hard else y), y


_ORIG_GATE = oracle.gate


def _mutant_gate_ge(logits, noise, tau, hard):
    m, y = _ORIG_GATE(logits, noise, tau, False)
    return ((y >= 0.5).astype(float) if hard else y), y


def _mutant_ste_no_tau(dmask, y, tau):
    y = np.asarray(y, float)
    return np.asarray(dmask, float) * y * (1 - y)


def _mutant_sparsity_unweighted(selectors, shapes):
    s_l = [1.0 - np.count_nonzero(B) / float(np.asarray(B).size) for B in selectors]
    return s_l, float(np.mean(s_l))


_ORIG_BUDGET = oracle.budget_loss


def _mutant_budget_unweighted(selectors, params, s_target, lam, uniform=False):
    return _ORIG_BUDGET(selectors, [1] * len(params), s_target, lam, uniform)


def _mutant_budget_grad_sign(selectors, params, s_target, lam, uniform=False):
    L, c, k = _ORIG_BUDGET(selectors, params, s_target, lam, uniform)
    return L, -c, k


def _mutant_budget_grad_no_inv_s(selectors, params, s_target, lam, uniform=False):
    L, c, k = _ORIG_BUDGET(selectors, params, s_target, lam, uniform)
    G = np.array([np.asarray(B).size for B in selectors], float)
    s_l = 1.0 - k / G
    s = float(np.sum(s_l * np.array(params, float)) / np.sum(np.array(params, float)))
    return L, c * (s_l if uniform else s), k


_ORIG_DISTILL = oracle.distill_loss
_ORIG_DISTILL_BWD = oracle.distill_loss_bwd


def _mutant_distill_sum(H_t, H_s, W, valid=None):
    L, ce, lt, ls = _ORIG_DISTILL(H_t, H_s, W, valid)
    n = len(ce) if valid is None else int(np.count_nonzero(valid))
    return L * n, ce, lt, ls


def _mutant_distill_reversed(H_t, H_s, W, valid=None):
    return _ORIG_DISTILL(H_s, H_t, W, valid)


def _mutant_distill_over_tokens(H_t, H_s, W, valid=None):
    # softmax over the token axis instead of the vocabulary
    z_t, z_s = np.asarray(H_t, float) @ np.asarray(W, float).T, np.asarray(H_s, float) @ np.asarray(W, float).T
    p_t = oracle.softmax_rows(z_t.T).T
    ls = z_s - np.log(np.exp(z_s).sum(axis=0, keepdims=True))
    ce = -(p_t * ls).sum(axis=1)
    _, _, lse_t, lse_s = _ORIG_DISTILL(H_t, H_s, W, valid)
    return float(ce.mean()), ce, lse_t, lse_s


def _mutant_distill_bwd_sign(H_t, H_s, W, valid=None):
    return -_ORIG_DISTILL_BWD(H_t, H_s, W, valid)


def _mutant_distill_bwd_no_teacher(H_t, H_s, W, valid=None):
    p_s = oracle.softmax_rows(np.asarray(H_s, float) @ np.asarray(W, float).T)
    return p_s / p_s.shape[0] @ np.asarray(W, float)


_ORIG_HYPER_FWD = oracle.hyper_fwd
_ORIG_HYPER_BWD = oracle.hyper_bwd
_ORIG_ADAMW = oracle.adamw_step


def _mutant_hyper_reset_inside(z, gru_flat, A, c, offsets, H):
    # the other GRU form: candidate from W_hn (r * h) instead of r * (W_hn h + b_hn)
    z = np.asarray(z, float)
    L, D = z.shape
    p = oracle.groupmask_oracle._split_gru(gru_flat, D, H)
    outs = []
    for d, order in ((0, range(L)), (1, range(L - 1, -1, -1))):
        W_ih, W_hh, b_ih, b_hh = p[d]
        h, out = np.zeros(H), np.zeros((L, H))
        for l in order:
            gi = W_ih @ z[l] + b_ih
            gh = W_hh @ h + b_hh
            r = 1 / (1 + np.exp(-(gi[:H] + gh[:H])))
            u = 1 / (1 + np.exp(-(gi[H:2 * H] + gh[H:2 * H])))
            n = np.tanh(gi[2 * H:] + W_hh[2 * H:] @ (r * h) + b_hh[2 * H:])
            h = (1 - u) * n + u * h
            out[l] = h
        outs.append(out)
    o = np.concatenate(outs, axis=1)
    return np.concatenate([np.asarray(A, float)[offsets[l]:offsets[l + 1]] @ o[l] + np.asarray(c, float)[offsets[l]:offsets[l + 1]]
                           for l in range(L)])


def _mutant_hyper_one_direction(z, gru_flat, A, c, offsets, H):
    # both halves of the output taken from the forward direction
    z = np.asarray(z, float)
    L, D = z.shape
    p = oracle.groupmask_oracle._split_gru(gru_flat, D, H)
    f, _ = oracle.groupmask_oracle._gru_dir(z, *p[0], range(L))
    o = np.concatenate([f, f], axis=1)
    return np.concatenate([np.asarray(A, float)[offsets[l]:offsets[l + 1]] @ o[l] + np.asarray(c, float)[offsets[l]:offsets[l + 1]]
                           for l in range(L)])


def _mutant_hyper_bwd_no_carry(dlogits, z, gru_flat, A, c, offsets, H):
    # the recurrent gradient is dropped between steps (truncated backpropagation)
    dA, dc, dgru, do = _ORIG_HYPER_BWD(dlogits, z, gru_flat, A, c, offsets, H)
    z = np.asarray(z, float)
    L, D = z.shape
    p = oracle.groupmask_oracle._split_gru(gru_flat, D, H)
    grads = []
    for d, order in ((0, range(L)), (1, range(L - 1, -1, -1))):
        _, cache = oracle.groupmask_oracle._gru_dir(z, *p[d], order)
        g = [np.zeros_like(x) for x in p[d]]
        for l in order:
            h, r, u, n, ghn = cache[l]
            dh = do[l, d * H:(d + 1) * H]
            dan = dh * (1 - u) * (1 - n * n)
            dar = dan * ghn * r * (1 - r)
            dau = dh * (h - n) * u * (1 - u)
            dgi = np.concatenate([dar, dau, dan])
            dgh = np.concatenate([dar, dau, dan * r])
            g[0] += np.outer(dgi, z[l]); g[1] += np.outer(dgh, h); g[2] += dgi; g[3] += dgh
        grads += g
    return dA, dc, np.concatenate([x.reshape(-1) for x in grads]), do


def _mutant_hyper_bwd_head_transposed(dlogits, z, gru_flat, A, c, offsets, H):
    dA, dc, dgru, do = _ORIG_HYPER_BWD(dlogits, z, gru_flat, A, c, offsets, H)
    return -dA, dc, dgru, do


def _mutant_adamw_no_bias_correction(p, g, m, v, lr, beta1, beta2, eps, weight_decay, step):
    return _ORIG_ADAMW(p, g, m, v, lr, beta1, beta2, eps, weight_decay, 10 ** 9)


def _mutant_adamw_coupled_decay(p, g, m, v, lr, beta1, beta2, eps, weight_decay, step):
    return _ORIG_ADAMW(p, np.asarray(g, float) + weight_decay * np.asarray(p, float), m, v, lr, beta1, beta2, eps, 0.0,
                       step)


def _mutant_from_bf16_as_half(bits):
    # the 16 bits read as IEEE half precision instead of the top half of an fp32
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float64)


def _mutant_from_bf16_shift15(bits):
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(15)
    return b.view(np.float32).astype(np.float64)


def _mutant_kept_count_pruned(B):
    B = np.asarray(B)
    return int(B.size - np.count_nonzero(B))


def _mutant_preserved_rate_pruned(B, g_in, g_out=1):
    M = oracle.expand_mask((np.asarray(B) == 0).astype(np.float64), g_in, g_out)
    return float(M.sum() / M.size)


MUTANTS = [
    ("linear_fwd", _mutant_fwd_strided_groups),
    ("linear_fwd", _mutant_fwd_strided_rows),
    ("linear_bwd_dgate", _mutant_dgate_first_row_only),
    ("linear_bwd_dx", _mutant_dx_strided_rows),
    ("linear_bwd_dgate", _mutant_dgate_no_weight),
    ("linear_bwd_dgate", _mutant_dgate_strided_groups),
    ("linear_bwd_dx", _mutant_dx_unmasked),
    ("gate", _mutant_gate_sign),
    ("gate", _mutant_gate_ge),
    ("gate_bwd", _mutant_ste_no_tau),
    ("sparsity", _mutant_sparsity_unweighted),
    ("budget_loss", _mutant_budget_unweighted),
    ("budget_loss", _mutant_budget_grad_sign),
    ("budget_loss", _mutant_budget_grad_no_inv_s),
    ("distill_loss", _mutant_distill_sum),
    ("distill_loss", _mutant_distill_reversed),
    ("distill_loss", _mutant_distill_over_tokens),
    ("distill_loss_bwd", _mutant_distill_bwd_sign),
    ("distill_loss_bwd", _mutant_distill_bwd_no_teacher),
    ("hyper_fwd", _mutant_hyper_reset_inside),
    ("hyper_fwd", _mutant_hyper_one_direction),
    ("hyper_bwd", _mutant_hyper_bwd_no_carry),
    ("hyper_bwd", _mutant_hyper_bwd_head_transposed),
    ("adamw_step", _mutant_adamw_no_bias_correction),
    ("adamw_step", _mutant_adamw_coupled_decay),
    ("from_bf16", _mutant_from_bf16_as_half),
    ("from_bf16", _mutant_from_bf16_shift15),
    ("kept_count", _mutant_kept_count_pruned),
    ("preserved_rate", _mutant_preserved_rate_pruned),
]

PIN_TESTS = [
    lambda: [test_fwd_matches_brute_force(*c) for c in TINY],
    lambda: [test_dx_matches_brute_force(*c) for c in TINY],
    lambda: [test_dgate_matches_brute_force(*c) for c in TINY],
    test_square_group_gradient_sums_the_row_gradients_of_its_block,
    lambda: test_square_group_dgate_matches_central_finite_differences(0.5),
    test_single_square_group_scales_the_dense_layer,
    test_dx_is_the_adjoint_of_the_forward,
    lambda: test_dgate_matches_central_finite_differences(0.5),
    test_dgate_euler_and_row_sum_identities,
    test_hard_gate_is_thresholded_sigmoid,
    test_eval_mode_thresholds_logits,
    test_ste_derivative_matches_finite_difference_of_relaxation,
    test_paper_category_rates_reproduce_global_rate,
    test_budgeted_inputs_give_exact_kept_count,
    test_budget_loss_depends_only_on_the_ratio,
    test_budget_global_sparsity_is_the_fraction_of_pruned_weights,
    lambda: test_budget_gradient_matches_selector_flips(False),
    lambda: test_budget_gradient_matches_selector_flips(True),
    test_distill_matches_brute_force_loops,
    test_distill_is_kl_plus_teacher_entropy,
    test_distill_of_identical_passes_is_teacher_entropy_with_zero_gradient,
    test_distill_one_hot_teacher_is_cross_entropy,
    test_distill_uniform_teacher,
    test_distill_gradient_matches_finite_differences,
    test_distill_counts_only_valid_tokens,
    lambda: test_bigru_matches_torch_gru(5, 6, 4),
    test_hyper_heads_match_loops,
    lambda: test_hyper_gradients_match_autograd(6, 5, 3),
    test_hyper_gru_gradient_matches_finite_differences,
    test_adamw_matches_torch,
    test_kept_count_and_preserved_rate_away_from_one_half,
    test_from_bf16_is_exact_over_every_bit_pattern,
]


@pytest.mark.parametrize("name,mutant", MUTANTS, ids=[m[1].__name__ for m in MUTANTS])
def test_pins_catch_planted_mistake(monkeypatch, name, mutant):
    monkeypatch.setattr(oracle, name, mutant)
    caught = 0
    for pin in PIN_TESTS:
        try:
            pin()
        except AssertionError:
            caught += 1
    assert caught > 0, f"no pin caught the planted mistake in {name}"
