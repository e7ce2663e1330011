"""Plain, slow, fp64 reference of the group-masked linear layer of GroupMask.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import or call this
module: only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` do.  It shares no code with the HIP library.

Every function is the paper's definition written out in NumPy float64; bf16 and
fp32 inputs widen to fp64 exactly, so the only rounding here is fp64's.

Readings taken where the paper is silent (each is listed with its reason in the
design notes of the repository):

* Gumbel-Sigmoid (Sec. 2.2 cites the relaxation without printing it): the
  binary-concrete form y = sigmoid((logit + ln u - ln(1-u)) / tau) with one
  uniform variate u per group.  ln u - ln(1-u) is a logistic variate, i.e. the
  difference of two independent Gumbel variates, so P(z > 0) = sigmoid(logit).
  This choice of noise form is pinned only by the statistical property above,
  not by any number printed in the paper ("parity unpinned" for the exact form).
* Hard decision: keep iff y > 1/2, i.e. iff z = logit + noise > 0; z == 0 prunes.
* STE (Sec. 2.2): the forward uses the binary selector; the backward uses the
  derivative of the relaxation, d y / d logit = y (1 - y) / tau.
* Evaluation mode (Sec. 2.2, Appendix F): no noise; keep iff logit > 0.
* Soft selectors: a fractional mask value scales its group; only exact zeros
  prune.  The paper's forward is binary; this generalisation keeps the soft
  output usable.
* Groups are g_out x g blocks (Sec. 2.1): g consecutive input columns of
  g_out consecutive output rows; the default 1 x 256 has g_out = 1.
* dgate is produced for every group, pruned or kept, because the STE passes a
  gradient to every selector; it does not depend on the mask values.
* Budget regulariser (Sec. 2.3): a selector counts as kept when its mask value
  is nonzero (the discrete B).  Its gradient is the derivative of the loss
  with B taken as continuous (what the STE hands to the relaxation), with
  sign(0) = 0 at s = s_t; the uniform variant sums the per-layer terms.
* Distillation loss (Sec. 2.4, Eq. 4): teacher and student logits come from
  one frozen LM head applied to the final hidden states of the dense (teacher)
  and the masked (student) pass; N counts the valid tokens (a per-token flag);
  with no valid token the loss and its gradient are zero.  The gradient goes
  to the student's hidden states only (the teacher is detached, the LM head
  is frozen).
* Hypernetwork (Sec. 2.2, Eq. 3; no sizes are printed): the fixed input holds
  one D-vector per target layer; the bidirectional GRU uses the standard GRU
  cell (reset gate applied to the recurrent candidate term, zero initial
  state) with H units per direction, and its output for layer l is the
  concatenation [forward; backward] of size 2H; the head of layer l is an
  affine map A^l o_l + c^l onto its G^l selector logits.  The heads of all
  layers are stacked row by row in one [sum G, 2H] matrix, in the layer order
  of the flat selector array.  Parameters are trained with AdamW (Table 5):
  decoupled weight decay, bias-corrected moments.
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "from_bf16", "logistic_noise", "gate", "gate_bwd", "expand_mask", "masked_weight",
    "linear_fwd", "linear_bwd_dx", "linear_bwd_dgate", "linear_bwd", "sparsity",
    "preserved_rate", "near_threshold", "kept_count", "budget_loss",
    "softmax_rows", "distill_loss", "distill_loss_bwd",
    "gru_param_shapes", "bigru_fwd", "hyper_fwd", "hyper_bwd", "adamw_step",
]


def from_bf16(bits) -> np.ndarray:
    """bf16 bit patterns (uint16) to float64: the 16 bits are the top half of an IEEE fp32."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


# ---------------------------------------------------------------- gate (Sec. 2.2)

def logistic_noise(u) -> np.ndarray:
    """Noise term of the Gumbel-Sigmoid relaxation: ln u - ln(1 - u), for u in (0, 1)."""
    u = np.asarray(u, dtype=np.float64)
    return np.log(u) - np.log1p(-u)


def gate(logits, noise, tau: float, hard: bool):
    """Gumbel-Sigmoid gate with straight-through forward (Sec. 2.2; Appendix F for eval).

    z = logit + (ln u - ln(1-u)), or z = logit when ``noise`` is None (evaluation);
    y = sigmoid(z / tau).  Returns (mask, y): mask = [y > 1/2] when ``hard``,
    else mask = y.
    """
    z = np.asarray(logits, dtype=np.float64)
    if noise is not None:
        z = z + logistic_noise(noise)
    y = 1.0 / (1.0 + np.exp(-z / float(tau)))
    if hard:
        # sigmoid is strictly increasing with sigmoid(0) = 1/2, so y > 1/2 holds exactly
        # when z > 0; testing z keeps the decision exact where fp64 rounds y to 1/2.
        mask = (z > 0.0).astype(np.float64)
    else:
        mask = y.copy()
    return mask, y


def gate_bwd(dmask, y, tau: float) -> np.ndarray:
    """Straight-through backward (Sec. 2.2): d logit = d mask * y (1 - y) / tau."""
    y = np.asarray(y, dtype=np.float64)
    return np.asarray(dmask, dtype=np.float64) * y * (1.0 - y) / float(tau)


def near_threshold(y, band: float = 1e-6) -> np.ndarray:
    """Gates whose relaxed value lies within ``band`` of the 1/2 threshold."""
    return np.abs(np.asarray(y, dtype=np.float64) - 0.5) <= band


# ------------------------------------------------------- mask and weight (Eq. 1)

def expand_mask(B, g_in: int, g_out: int = 1) -> np.ndarray:
    """Full-resolution mask M = B (Kronecker) 1_{g_out x g_in} (Eq. 1)."""
    B = np.asarray(B, dtype=np.float64)
    return np.kron(B, np.ones((g_out, g_in), dtype=np.float64))


def masked_weight(W, B, g_in: int, g_out: int = 1) -> np.ndarray:
    """Pruned weight W_hat = W (elementwise) M (Eq. 1)."""
    W = np.asarray(W, dtype=np.float64)
    M = expand_mask(B, g_in, g_out)
    if M.shape != W.shape:
        raise ValueError(f"mask expands to {M.shape}, weight is {W.shape}")
    return W * M


# ------------------------------------------------------------ masked linear layer

def linear_fwd(X, W, B, g: int, g_out: int = 1) -> np.ndarray:
    """Student forward of one target linear: Y = X W_hat^T (Eq. 1 applied to nn.Linear).

    Groups are g_out x g (rows x input columns); B is [d_out / g_out, d_in / g].
    """
    X = np.asarray(X, dtype=np.float64)
    return X @ masked_weight(W, B, g, g_out).T


def linear_bwd_dx(dY, W, B, g: int, g_out: int = 1) -> np.ndarray:
    """Input gradient through the frozen masked weight: dX = dY W_hat."""
    return np.asarray(dY, dtype=np.float64) @ masked_weight(W, B, g, g_out)


def linear_bwd_dgate(dY, X, W, g: int, g_out: int = 1) -> np.ndarray:
    """Selector gradient: dgate[u, v] = sum over the group's entries of W * (dY^T X).

    Y is linear in each selector, so d<dY, Y>/dB[u, v] = sum_{o in block u, i in block v} W[o, i] (dY^T X)[o, i];
    the weight itself gets no gradient (frozen, Sec. 2.4).
    """
    dY = np.asarray(dY, dtype=np.float64)
    X = np.asarray(X, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    d_out, d_in = W.shape
    if d_in % g or d_out % g_out:
        raise ValueError("d_in must be a multiple of g and d_out of g_out")
    G = dY.T @ X
    return (W * G).reshape(d_out // g_out, g_out, d_in // g, g).sum(axis=(1, 3))


def linear_bwd(dY, X, W, B, g: int, g_out: int = 1):
    """(dX, dgate) of one masked linear."""
    return linear_bwd_dx(dY, W, B, g, g_out), linear_bwd_dgate(dY, X, W, g, g_out)


# ------------------------------------------------------ sparsity ratios (Eq. 2)

def kept_count(B) -> int:
    """Number of retained groups of a selector matrix."""
    return int(np.count_nonzero(np.asarray(B)))


def sparsity(selectors, shapes):
    """Layer-wise and overall sparsity (Eq. 2).

    selectors: list of B^l arrays; shapes: list of (d_out, d_in).
    s^l = 1 - sum(B^l) / (G_out G_in); s = sum_l s^l d_out d_in / sum_l d_out d_in.
    """
    s_layer = []
    for B in selectors:
        B = np.asarray(B)
        s_layer.append(1.0 - np.count_nonzero(B) / float(B.size))
    sizes = np.array([float(do) * float(di) for do, di in shapes])
    s = float(np.sum(np.array(s_layer) * sizes) / np.sum(sizes))
    return s_layer, s


def preserved_rate(B, g_in: int, g_out: int = 1) -> float:
    """Active weights / total weights after applying the binary mask (Appendix F)."""
    M = expand_mask((np.asarray(B) != 0).astype(np.float64), g_in, g_out)
    return float(M.sum() / M.size)


# ------------------------------------------ sparsity-budget regulariser (Sec. 2.3)

def budget_loss(selectors, params, s_target: float, lam: float, uniform: bool = False):
    """Sparsity-budget regulariser of Sec. 2.3 and its gradient per selector.

    selectors: list of B^l arrays (nonzero = kept); params: list of P^l, the
    weight count d_out^l d_in^l of each layer.  With G^l = B^l.size groups and
    s^l, s from Eq. 2 (evaluated exactly in rationals, then rounded once):

      global  : L = lam |log(s / s_t)|
                dL/dB^l = lam sgn(log(s/s_t)) (1/s) ds/dB^l,  ds/dB^l = -(P^l / G^l) / sum_k P^k
      uniform : L = sum_l lam |log(s^l / s_t)|
                dL/dB^l = lam sgn(log(s^l/s_t)) (1/s^l) (-1 / G^l)

    Every selector of layer l receives the same derivative coeff[l].  s = 0
    (every group kept) makes L and the derivative infinite.
    Returns (L, coeff, kept) with coeff a float64 array over layers and kept
    the integer kept counts.
    """
    from fractions import Fraction
    kept = np.array([np.count_nonzero(np.asarray(B)) for B in selectors], dtype=np.int64)
    Gi = [int(np.asarray(B).size) for B in selectors]
    Pi = [int(p) for p in params]
    G = np.array(Gi, dtype=np.float64)
    P = np.array(Pi, dtype=np.float64)
    s_layer_exact = [Fraction(g - int(k), g) for g, k in zip(Gi, kept)]
    with np.errstate(divide="ignore"):
        if uniform:
            s_layer = np.array([float(x) for x in s_layer_exact])
            logs = np.log(s_layer / s_target)
            L = float(np.sum(lam * np.abs(logs)))
            coeff = lam * np.sign(logs) / s_layer * (-1.0 / G)
        else:
            s = float(sum(x * p for x, p in zip(s_layer_exact, Pi)) / sum(Pi))
            logr = np.log(s / s_target)
            L = float(lam * abs(logr))
            coeff = lam * np.sign(logr) / s * (-(P / G) / np.sum(P))
    return L, coeff, kept


# ------------------------------------------------ distillation loss (Sec. 2.4, Eq. 4)

def softmax_rows(z) -> np.ndarray:
    """Softmax over the last axis: exp(z - max) / sum(exp(z - max))."""
    z = np.asarray(z, dtype=np.float64)
    e = np.exp(z - z.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def _lm_logits(H, W) -> np.ndarray:
    """Logits of the LM head: z[t, v] = sum_j H[t, j] W[v, j]."""
    return np.asarray(H, dtype=np.float64) @ np.asarray(W, dtype=np.float64).T


def distill_loss(H_t, H_s, W, valid=None):
    """Self-distillation loss of Eq. 4 over N valid tokens.

    L = -(1/N) sum_{valid t} sum_v p_T(t, v) log p_S(t, v), with p_T, p_S the
    softmax over the vocabulary of the teacher and student logits H W^T.
    Returns (L, ce, lse_t, lse_s): ce[t] = -sum_v p_T log p_S per token (for
    every token, valid or not) and the log-sum-exp of each token's teacher and
    student logits.
    """
    z_t, z_s = _lm_logits(H_t, W), _lm_logits(H_s, W)
    m_s = z_s.max(axis=1, keepdims=True)
    lse_s = (m_s + np.log(np.exp(z_s - m_s).sum(axis=1, keepdims=True)))[:, 0]
    m_t = z_t.max(axis=1, keepdims=True)
    lse_t = (m_t + np.log(np.exp(z_t - m_t).sum(axis=1, keepdims=True)))[:, 0]
    p_t = softmax_rows(z_t)
    log_p_s = z_s - lse_s[:, None]
    ce = -(p_t * log_p_s).sum(axis=1)
    v = np.ones(ce.shape[0], dtype=bool) if valid is None else np.asarray(valid) != 0
    n = int(v.sum())
    L = float(ce[v].sum() / n) if n else 0.0
    return L, ce, lse_t, lse_s


def distill_loss_bwd(H_t, H_s, W, valid=None) -> np.ndarray:
    """Gradient of Eq. 4 with respect to the student's hidden states.

    dL/dz_S[t, v] = (p_S(t, v) - p_T(t, v)) / N for a valid token (the teacher
    probabilities sum to one), zero otherwise; dH_S = dz_S W.
    """
    W = np.asarray(W, dtype=np.float64)
    p_t = softmax_rows(_lm_logits(H_t, W))
    p_s = softmax_rows(_lm_logits(H_s, W))
    v = np.ones(p_t.shape[0], dtype=bool) if valid is None else np.asarray(valid) != 0
    n = int(v.sum())
    dz = np.zeros_like(p_s)
    if n:
        dz[v] = (p_s[v] - p_t[v]) / n
    return dz @ W


# ------------------------------------------------------- hypernetwork (Sec. 2.2, Eq. 3)

def _sigmoid(x):
    return 1.0 / (1.0 + np.exp(-x))


def gru_param_shapes(D: int, H: int):
    """Shapes of one direction's parameters, in storage order: W_ih [3H, D], W_hh [3H, H], b_ih [3H], b_hh [3H].

    The 3H rows are the reset, update and candidate gates, in that order.
    """
    return [(3 * H, D), (3 * H, H), (3 * H,), (3 * H,)]


def _split_gru(flat, D, H):
    flat = np.asarray(flat, dtype=np.float64)
    out, pos = [], 0
    for direction in range(2):
        ps = []
        for shp in gru_param_shapes(D, H):
            n = int(np.prod(shp))
            ps.append(flat[pos:pos + n].reshape(shp))
            pos += n
        out.append(ps)
    if pos != flat.size:
        raise ValueError("GRU parameter vector has the wrong length")
    return out


def _gru_dir(z, W_ih, W_hh, b_ih, b_hh, order):
    """One GRU direction over the steps in `order`; returns outputs [L, H] and per-step caches."""
    L = z.shape[0]
    H = W_hh.shape[1]
    h = np.zeros(H)
    out = np.zeros((L, H))
    cache = {}
    for l in order:
        gi = W_ih @ z[l] + b_ih
        gh = W_hh @ h + b_hh
        r = _sigmoid(gi[:H] + gh[:H])
        u = _sigmoid(gi[H:2 * H] + gh[H:2 * H])
        n = np.tanh(gi[2 * H:] + r * gh[2 * H:])
        h_new = (1.0 - u) * n + u * h
        cache[l] = (h, r, u, n, gh[2 * H:])
        h = h_new
        out[l] = h
    return out, cache


def bigru_fwd(z, gru_flat, H: int):
    """Bidirectional GRU over the layer sequence z [L, D]: outputs [L, 2H] = [forward; backward]."""
    z = np.asarray(z, dtype=np.float64)
    L, D = z.shape
    (p0, p1) = _split_gru(gru_flat, D, H)
    f, _ = _gru_dir(z, *p0, range(L))
    b, _ = _gru_dir(z, *p1, range(L - 1, -1, -1))
    return np.concatenate([f, b], axis=1)


def hyper_fwd(z, gru_flat, A, c, offsets, H: int):
    """Selector logits of every layer (Eq. 3 before binarisation), flat in layer order.

    logits[e] = A[e] . o_{l(e)} + c[e] for e in [offsets[l], offsets[l+1]).
    """
    o = bigru_fwd(z, gru_flat, H)
    A = np.asarray(A, dtype=np.float64)
    c = np.asarray(c, dtype=np.float64)
    out = np.empty(A.shape[0])
    for l in range(len(offsets) - 1):
        a, b = int(offsets[l]), int(offsets[l + 1])
        out[a:b] = A[a:b] @ o[l] + c[a:b]
    return out


def _gru_dir_bwd(z, W_ih, W_hh, b_ih, b_hh, order, cache, dout):
    """Backpropagation through one direction; dout [L, H] is the gradient of its outputs."""
    H = W_hh.shape[1]
    g = [np.zeros_like(W_ih), np.zeros_like(W_hh), np.zeros_like(b_ih), np.zeros_like(b_hh)]
    dh = np.zeros(H)
    for l in reversed(list(order)):
        h, r, u, n, ghn = cache[l]
        dh = dh + dout[l]
        dn = dh * (1.0 - u)
        du = dh * (h - n)
        dan = dn * (1.0 - n * n)
        dar = dan * ghn * r * (1.0 - r)
        dau = du * u * (1.0 - u)
        dgi = np.concatenate([dar, dau, dan])
        dgh = np.concatenate([dar, dau, dan * r])
        g[0] += np.outer(dgi, z[l])
        g[1] += np.outer(dgh, h)
        g[2] += dgi
        g[3] += dgh
        dh = dh * u + W_hh.T @ dgh
    return g


def hyper_bwd(dlogits, z, gru_flat, A, c, offsets, H: int):
    """Gradients of <dlogits, hyper_fwd(...)> with respect to A, c and the GRU parameters (flat)."""
    z = np.asarray(z, dtype=np.float64)
    L, D = z.shape
    p0, p1 = _split_gru(gru_flat, D, H)
    f, cf = _gru_dir(z, *p0, range(L))
    b, cb = _gru_dir(z, *p1, range(L - 1, -1, -1))
    o = np.concatenate([f, b], axis=1)
    A = np.asarray(A, dtype=np.float64)
    dl = np.asarray(dlogits, dtype=np.float64)
    dA = np.empty_like(A)
    do = np.zeros_like(o)
    for l in range(L):
        a, e = int(offsets[l]), int(offsets[l + 1])
        dA[a:e] = np.outer(dl[a:e], o[l])
        do[l] = A[a:e].T @ dl[a:e]
    g0 = _gru_dir_bwd(z, *p0, range(L), cf, do[:, :H])
    g1 = _gru_dir_bwd(z, *p1, range(L - 1, -1, -1), cb, do[:, H:])
    dgru = np.concatenate([x.reshape(-1) for x in g0 + g1])
    return dA, dl.copy(), dgru, do


def adamw_step(p, g, m, v, lr, beta1, beta2, eps, weight_decay, step: int):
    """One AdamW step (decoupled weight decay, bias-corrected moments); returns (p, m, v)."""
    p = np.asarray(p, dtype=np.float64) * (1.0 - lr * weight_decay)
    g = np.asarray(g, dtype=np.float64)
    m = beta1 * np.asarray(m, dtype=np.float64) + (1.0 - beta1) * g
    v = beta2 * np.asarray(v, dtype=np.float64) + (1.0 - beta2) * g * g
    m_hat = m / (1.0 - beta1 ** step)
    v_hat = v / (1.0 - beta2 ** step)
    return p - lr * m_hat / (np.sqrt(v_hat) + eps), m, v
