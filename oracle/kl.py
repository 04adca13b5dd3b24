"""Cross-entropy, forward-KL and reverse-KL losses of the draft distribution
against the target, and their gradients w.r.t. the draft logits, in float64:
the training objectives the TV loss is compared against.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Per position n and draft step k (paper Sec. 4.1 with its footnote, Table
grad_comparison, App. B and App. C), with p = softmax(z_target / T)
(detached) and q = softmax(z_draft / T):

  forward KL  L = sum_v p_v (log p_v - log q_v)      dL/dz_j = (q_j - p_j) / T
  CE          L = -sum_v p_v log q_v                 same gradient (CE = H(p) + KL)
  reverse KL  L = sum_v q_v (log q_v - log p_v)      dL/dz_j = q_j (log q_j - log p_j - L) / T

A term whose weight is zero (p_v = 0 for forward KL and CE, q_v = 0 for
reverse KL) is zero.  Over the K steps: L_n = (1/K) sum_k L_{n,k};
loss = scale * sum_n L_n; grad = d loss / d z_draft.

Readings: the K draft steps are averaged (each MTP head has its own
objective, as for the per-step TV loss); the paper derives the gradients at
T = 1 and the 1/T factor of softmax(z / T) is included here.
"""

import numpy as np

KIND_FORWARD = 0
KIND_CE = 1
KIND_REVERSE = 2


def log_softmax_t(z, T):
    """log softmax(z / T) along the last axis, float64."""
    a = np.asarray(z, dtype=np.float64) / T
    m = np.max(a, axis=-1, keepdims=True)
    with np.errstate(invalid="ignore", over="ignore", divide="ignore"):
        lse = m + np.log(np.sum(np.exp(a - m), axis=-1, keepdims=True))
        return a - lse


def kl_ref(target_logits, draft_logits, temperature, kind, scale=1.0):
    """target_logits, draft_logits: [N, K, V].  Returns per_step [N, K]
    (L_{n,k}), loss (float) and grad [N, K, V] (d loss / d z_draft)."""
    zt = np.asarray(target_logits, dtype=np.float64)
    zd = np.asarray(draft_logits, dtype=np.float64)
    N, K, V = zd.shape
    T = float(temperature)
    lp = log_softmax_t(zt, T)
    lq = log_softmax_t(zd, T)
    p = np.exp(lp)
    q = np.exp(lq)
    with np.errstate(invalid="ignore"):
        if kind == KIND_FORWARD:
            L = np.where(p > 0, p * (lp - lq), 0.0).sum(axis=-1)
            g = (q - p) / T
        elif kind == KIND_CE:
            L = np.where(p > 0, -p * lq, 0.0).sum(axis=-1)
            g = (q - p) / T
        elif kind == KIND_REVERSE:
            L = np.where(q > 0, q * (lq - lp), 0.0).sum(axis=-1)
            g = np.where(q > 0, q * (lq - lp - L[..., None]), 0.0) / T
        else:
            raise ValueError(kind)
    loss_pos = L.mean(axis=1)
    return {"per_step": L, "loss": float(scale * loss_pos.sum()), "loss_pos": scale * loss_pos,
            "grad": g * (scale / K)}
