"""TV loss, its gradient w.r.t. the draft logits, and the multi-step losses,
in float64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Per position n and draft step k (paper Sec. 4.1 Eq. tv_loss, Eq. tv_grad and
App. A):
  p = softmax(z_target / T)   (detached: no gradient flows into it)
  q = softmax(z_draft  / T)
  alpha = sum_v min(p_v, q_v)             L_TV = 1 - alpha
  S     = sum_v 1[q_v <= p_v] q_v
  d alpha / d z_draft_j = (1/T) q_j (1[q_j <= p_j] - S)
(the paper's gradient of L_TV carries the opposite sign and T = 1).

Per-position loss over the K steps, by mode:
  E2E      1 - (1/K) sum_j prod_{i<=j} alpha_i      (Sec. 4.2 Eq. e2e_tv)
  PROD     - prod_k alpha_k                         (the product-of-overlaps
                                                     objective, i.e. the
                                                     negated probability that
                                                     all K drafts are accepted)
  PER_STEP (1/K) sum_k (1 - alpha_k)                (Eq. tv_loss averaged)
The total is  loss = scale * sum_n L_n  and  grad = d loss / d z_draft.
The chain factors g_k = d L_n / d alpha_k are formed from prefix and suffix
products, never by dividing by an alpha (which may be 0).

The subgradient of min at a tie q_v = p_v follows the paper's indicator
1[q_v <= p_v].  No clamp is applied to the loss (the paper's optional clamp
has no stated value).
"""

import numpy as np

from .verify import softmax_t

MODE_E2E = 0
MODE_PROD = 1
MODE_PER_STEP = 2


def chain_factors(alpha, mode):
    """g[n, k] = d L_n / d alpha[n, k] and the per-position loss L[n].

    alpha: [N, K] float64.  Returns (g [N, K], L [N]).
    """
    alpha = np.asarray(alpha, dtype=np.float64)
    N, K = alpha.shape
    if mode == MODE_PER_STEP:
        L = (1.0 - alpha).sum(axis=1) / K
        g = np.full((N, K), -1.0 / K)
        return g, L
    # prefix[k] = prod_{i<k} alpha_i ; suffix[k] = prod_{i>=k} alpha_i
    prefix = np.ones((N, K + 1))
    suffix = np.ones((N, K + 1))
    for k in range(K):
        prefix[:, k + 1] = prefix[:, k] * alpha[:, k]
    for k in range(K - 1, -1, -1):
        suffix[:, k] = suffix[:, k + 1] * alpha[:, k]
    if mode == MODE_PROD:
        L = -prefix[:, K]
        g = -(prefix[:, :K] * suffix[:, 1:])
        return g, L
    if mode == MODE_E2E:
        # sum_j prod_{i<=j} alpha_i = sum_j prefix[j+1]
        L = 1.0 - prefix[:, 1:].sum(axis=1) / K
        # tail[k] = sum_{j>=k} prod_{k<i<=j} alpha_i = 1 + alpha_{k+1} tail[k+1]
        tail = np.ones((N, K))
        for k in range(K - 2, -1, -1):
            tail[:, k] = 1.0 + alpha[:, k + 1] * tail[:, k + 1]
        g = -(prefix[:, :K] * tail) / K
        return g, L
    raise ValueError("unknown mode %r" % (mode,))


def tv_ref(target_logits, draft_logits, temperature, mode=MODE_E2E, scale=1.0,
           want_grad=True):
    """Float64 TV loss forward and gradient.

    target_logits, draft_logits: [N, K, V]; temperature: positive scalar.
    Returns dict with loss (float), loss_per_position [N], overlap [N, K],
    S [N, K], g [N, K] (chain factors including ``scale``), scale, grad
    [N, K, V] (or None), and with the gradient also q [N, K, V], grad_weight
    [N, K, V] = g q / T (grad = grad_weight (1[q <= p] - S)) and tie_margin
    [N, K, V] = |log q - log p| with tie_condition [N, K, V], the size of
    the terms log q - log p is formed from, which locate the elements whose
    indicator is decided by rounding and how far that moves S.
    """
    zt = np.asarray(target_logits, dtype=np.float64)
    zd = np.asarray(draft_logits, dtype=np.float64)
    N, K, V = zt.shape
    assert zd.shape == (N, K, V)
    T = float(temperature)
    p, lzt = softmax_t(zt, T)
    q, lzd = softmax_t(zd, T)
    alpha = np.minimum(p, q).sum(axis=-1)
    ind = q <= p
    S = np.where(ind, q, 0.0).sum(axis=-1)
    g, L = chain_factors(alpha, mode)
    g = g * scale
    out = {
        "loss": float(scale * L.sum()),
        "loss_per_position": scale * L,
        "overlap": alpha,
        "S": S,
        "g": g,
        "grad": None,
        "logz_target": lzt,
        "logz_draft": lzd,
    }
    out["scale"] = float(scale)
    if want_grad:
        out["q"] = q
        out["grad_weight"] = g[:, :, None] * (1.0 / T) * q
        out["grad"] = g[:, :, None] * (1.0 / T) * q * (ind.astype(np.float64) - S[:, :, None])
        with np.errstate(divide="ignore", invalid="ignore"):
            out["tie_margin"] = np.abs((zd / T - lzd[..., None]) - (zt / T - lzt[..., None]))
            # size of the terms ln q - ln p is formed from: an evaluation with
            # unit roundoff u decides 1[q <= p] correctly once tie_margin
            # exceeds a small multiple of u times this
            out["tie_condition"] = (np.abs(zd) + np.abs(zt)) / T + np.abs(lzd)[..., None] + np.abs(lzt)[..., None]
    return out
