"""Random draws for the synthetic workloads (no method arithmetic here)."""
from __future__ import annotations

import dataclasses
from typing import Optional, Sequence

import numpy as np

# The paper fixes its calibration seed to 42 (Appendix A, Table 5); every
# stream here is derived from it.
SEED = 42

# u = (j + 1/2) / 2^23 is a multiple of 2^-24 in (0, 1): exact in fp32, as is 1 - u,
# and never 0 or 1.
_NOISE_BITS = 23


def _rng(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED, *key])))


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (round-to-nearest-even), returned as uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return r.astype(np.uint16)


def f32_from_bf16_bits(b: np.ndarray) -> np.ndarray:
    """Widen uint16 bf16 bit patterns to fp32 (exact)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def draw_uniform_noise(rng: np.random.Generator, n: int, half: Optional[str] = None) -> np.ndarray:
    """Uniform variates u = (j + 1/2) / 2^23, j integer, exact in fp32.

    ``half`` restricts j to the upper ("hi", u > 1/2) or lower ("lo", u < 1/2)
    half of its range; None draws from the whole of (0, 1).
    """
    lo, hi = 0, 1 << _NOISE_BITS
    if half == "hi":
        lo = 1 << (_NOISE_BITS - 1)
    elif half == "lo":
        hi = 1 << (_NOISE_BITS - 1)
    j = rng.integers(lo, hi, size=n, dtype=np.int64)
    return ((j.astype(np.float64) + 0.5) / float(1 << _NOISE_BITS)).astype(np.float32)


def random_kept_mask(rng: np.random.Generator, n_groups: int, kept: int) -> np.ndarray:
    """0/1 vector of length n_groups with exactly ``kept`` ones at uniformly random positions."""
    if not 0 <= kept <= n_groups:
        raise ValueError("kept out of range")
    m = np.zeros(n_groups, dtype=np.float32)
    m[rng.permutation(n_groups)[:kept]] = 1.0
    return m


def budgeted_gate_inputs(rng: np.random.Generator, keep: np.ndarray):
    """Logits and uniform noise whose hard gate decision equals ``keep`` (for tests of the
    products given a mask; the gate itself is exercised on ``independent_gate_inputs``).

    The relaxed gate keeps a group when logit + (ln u - ln(1-u)) > 0.  The noise
    term is positive exactly when u > 1/2, so drawing |N(0,1)| logits with
    u > 1/2 for kept groups and -|N(0,1)| logits with u < 1/2 for pruned ones
    fixes every decision without evaluating the noise transform.  When half the
    groups are kept the logits are N(0,1) and u is uniform on (0,1) marginally.
    """
    keep = np.asarray(keep) != 0
    n = keep.size
    mag = np.abs(rng.standard_normal(n)).astype(np.float32)
    mag = np.maximum(mag, np.float32(2.0 ** -20))  # keep the sign of every logit strict
    logits = np.where(keep, mag, -mag).astype(np.float32)
    u_hi = draw_uniform_noise(rng, n, "hi")
    u_lo = draw_uniform_noise(rng, n, "lo")
    noise = np.where(keep, u_hi, u_lo).astype(np.float32)
    return logits, noise


def independent_gate_inputs(rng: np.random.Generator, n: int, loc=0.0):
    """Gate logits ~ N(loc, 1) and uniform noise u ~ U(0, 1), drawn independently of each other.

    ``loc`` (a scalar or one value per selector) is the caller's offset of the
    logits; it is how a caller meets a kept budget other than the one half that
    loc = 0 gives on average.  Nothing here evaluates the gate: which groups
    such inputs keep is decided by the gate itself.
    """
    z = rng.standard_normal(n)
    logits = (z + np.asarray(loc, dtype=np.float64)).astype(np.float32)
    return logits, draw_uniform_noise(rng, n)


def kept_counts_uniform_law(rng: np.random.Generator, n_groups: Sequence[int], lo: float, hi: float):
    """Per-matrix kept counts with sparsity s_j ~ U(lo, hi) (layer-adaptive budgets)."""
    s = rng.uniform(lo, hi, size=len(n_groups))
    return [int(round((1.0 - sj) * G)) for sj, G in zip(s, n_groups)], s


def kept_counts_beta_law(rng: np.random.Generator, n_groups: Sequence[int], params: Sequence[int],
                         target_sparsity: float = 0.5, a: float = 2.0, b: float = 2.0):
    """Per-matrix kept counts from a Beta(a, b) draw shifted so the parameter-weighted
    sparsity equals ``target_sparsity`` exactly in whole groups.

    r_l ~ Beta(a, b); s_l = clip(r_l + c, 0.02, 0.98) with the scalar c found by
    bisection so that sum_l s_l P_l / sum_l P_l = target; kept counts are then
    rounded with a largest-remainder fix so sum_l kept_l = (1 - target) sum_l G_l.
    All matrices are assumed to share one group size, so group counts are
    proportional to parameter counts.
    """
    G = np.asarray(n_groups, dtype=np.float64)
    P = np.asarray(params, dtype=np.float64)
    r = rng.beta(a, b, size=G.size)

    def mean_s(c):
        return float(np.sum(np.clip(r + c, 0.02, 0.98) * P) / np.sum(P))

    lo, hi = -1.0, 1.0
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        if mean_s(mid) < target_sparsity:
            lo = mid
        else:
            hi = mid
    s = np.clip(r + 0.5 * (lo + hi), 0.02, 0.98)
    want = (1.0 - s) * G
    kept = np.floor(want).astype(np.int64)
    total = int(round((1.0 - target_sparsity) * G.sum()))
    short = total - int(kept.sum())
    order = np.argsort(-(want - kept), kind="stable")
    kept[order[:short]] += 1
    return [int(k) for k in kept], s


@dataclasses.dataclass
class LinearCase:
    """Host copies of one masked linear's inputs (bf16 as uint16 bits, fp32 otherwise)."""
    T: int
    d_in: int
    d_out: int
    g: int
    tau: float
    X: np.ndarray       # uint16 [T, d_in]
    W: np.ndarray       # uint16 [d_out, d_in]
    dY: np.ndarray      # uint16 [T, d_out]
    logits: np.ndarray  # f32 [d_out/g_out, d_in/g]
    noise: np.ndarray   # f32 [d_out/g_out, d_in/g]
    mask: np.ndarray    # f32 [d_out/g_out, d_in/g], the hard decision the gate inputs encode
    kept: int
    g_out: int = 1


def make_linear_case(key: Sequence[int], T: int, d_in: int, d_out: int, g: int, kept: Optional[int],
                     tau: float = 0.5, w_std: float = 0.02, x_std: float = 1.0, dy_std: float = 1.0,
                     g_out: int = 1) -> LinearCase:
    """One masked linear: X ~ N(0, x_std), W ~ N(0, w_std), dY ~ N(0, dy_std), all rounded to bf16;
    a uniformly random kept set of ``kept`` groups of g_out x g (half when None) and gate inputs encoding it."""
    if d_in % g or d_out % g_out:
        raise ValueError("d_in must be a multiple of g and d_out of g_out")
    G_in, G_out = d_in // g, d_out // g_out
    n = G_out * G_in
    if kept is None:
        kept = n // 2
    rng = _rng(*key)
    X = bf16_bits_from_f32(rng.standard_normal((T, d_in), dtype=np.float32) * np.float32(x_std))
    W = bf16_bits_from_f32(rng.standard_normal((d_out, d_in), dtype=np.float32) * np.float32(w_std))
    dY = bf16_bits_from_f32(rng.standard_normal((T, d_out), dtype=np.float32) * np.float32(dy_std))
    mask = random_kept_mask(rng, n, kept)
    logits, noise = budgeted_gate_inputs(rng, mask)
    return LinearCase(T, d_in, d_out, g, tau, X, W, dY,
                      logits.reshape(G_out, G_in), noise.reshape(G_out, G_in),
                      mask.reshape(G_out, G_in), kept, g_out)


@dataclasses.dataclass
class DistillCase:
    """Host copies of the LM-head inputs of the distillation loss (bf16 as uint16 bits)."""
    N: int
    d: int
    V: int
    Ht: np.ndarray      # uint16 [N, d]  teacher final hidden states
    Hs: np.ndarray      # uint16 [N, d]  student final hidden states
    W: np.ndarray       # uint16 [V, d]  LM head
    valid: np.ndarray   # uint8 [N]


def make_distill_case(key: Sequence[int], N: int, d: int, V: int, student_noise: float = 0.3,
                      logit_std: float = 3.0, valid_frac: float = 1.0) -> DistillCase:
    """H_T ~ N(0, 1); H_S = H_T + student_noise N(0, 1) (the pruned pass drifts from the dense one);
    W ~ N(0, logit_std^2 / d), so logits have standard deviation about logit_std whatever d;
    each token valid with probability valid_frac (all valid at 1)."""
    rng = _rng(*key)
    ht = rng.standard_normal((N, d), dtype=np.float32)
    hs = ht + np.float32(student_noise) * rng.standard_normal((N, d), dtype=np.float32)
    w = rng.standard_normal((V, d), dtype=np.float32) * np.float32(logit_std / np.sqrt(d))
    valid = np.ones(N, dtype=np.uint8) if valid_frac >= 1.0 else (rng.uniform(size=N) < valid_frac).astype(np.uint8)
    return DistillCase(N, d, V, bf16_bits_from_f32(ht), bf16_bits_from_f32(hs), bf16_bits_from_f32(w), valid)


@dataclasses.dataclass
class HyperCase:
    """Host copies of the hypernetwork's parameters, inputs and optimiser state (fp32)."""
    L: int
    D: int
    H: int
    offsets: np.ndarray  # int64 [L + 1]
    z: np.ndarray        # [L, D]
    gru: np.ndarray      # [2 * 3H (D + H + 2)]
    A: np.ndarray        # [G, 2H]
    c: np.ndarray        # [G]
    dlogits: np.ndarray  # [G]
    mA: np.ndarray       # [G, 2H]
    vA: np.ndarray       # [G, 2H]
    mc: np.ndarray       # [G]
    vc: np.ndarray       # [G]


def make_hyper_case(key: Sequence[int], sizes: Sequence[int], D: int, H: int, warm: bool = True) -> HyperCase:
    """z ~ N(0, 1); GRU weights ~ U(-1/sqrt(H), 1/sqrt(H)) and heads ~ U(-1/sqrt(2H), 1/sqrt(2H)) (the
    default initialisation of recurrent and linear layers); logit gradients ~ N(0, 0.01^2); with warm,
    AdamW moments as after some steps (m ~ N(0, 1e-3^2), v ~ U(1e-7, 1e-5)), else zero."""
    rng = _rng(*key)
    L = len(sizes)
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    G = int(offsets[-1])
    P = 2 * 3 * H * (D + H + 2)
    f32 = np.float32
    z = rng.standard_normal((L, D), dtype=f32)
    gru = rng.uniform(-1.0, 1.0, size=P).astype(f32) * f32(1.0 / np.sqrt(H))
    a = f32(1.0 / np.sqrt(2 * H))
    A = rng.uniform(-1.0, 1.0, size=(G, 2 * H)).astype(f32) * a
    c = rng.uniform(-1.0, 1.0, size=G).astype(f32) * a
    dl = rng.standard_normal(G, dtype=f32) * f32(0.01)
    if warm:
        mA = rng.standard_normal((G, 2 * H), dtype=f32) * f32(1e-3)
        vA = rng.uniform(1e-7, 1e-5, size=(G, 2 * H)).astype(f32)
        mc = rng.standard_normal(G, dtype=f32) * f32(1e-3)
        vc = rng.uniform(1e-7, 1e-5, size=G).astype(f32)
    else:
        mA, vA = np.zeros((G, 2 * H), f32), np.zeros((G, 2 * H), f32)
        mc, vc = np.zeros(G, f32), np.zeros(G, f32)
    return HyperCase(L, D, H, offsets, z, gru, A, c, dl, mA, vA, mc, vc)


def rng_for(*key: int) -> np.random.Generator:
    """A generator for ad-hoc draws in tests, derived from the shared seed."""
    return _rng(*key)
