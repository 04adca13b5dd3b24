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

Precision: the gradients are differences of probabilities (q - p) and of
log-probabilities (log q - log p - L).  Where one token holds all but 1e-10
of both distributions, q - p of that token is a difference of two numbers
within 1e-10 of 1, and float64 keeps only about six of its digits.  The
softmax, the differences and the sums are therefore evaluated in extended
precision (numpy.longdouble, a 64-bit significand on x86-64), then returned
as float64.
"""

import numpy as np

KIND_FORWARD = 0
KIND_CE = 1
KIND_REVERSE = 2


XP = np.longdouble


def log_softmax_t(z, T):
    """log softmax(z / T) along the last axis, in extended precision."""
    a = np.asarray(z, dtype=XP) / XP(T)
    m = np.max(a, axis=-1, keepdims=True)
    with np.errstate(invalid="ignore", over="ignore", divide="ignore"):
        lse = m + np.log(np.sum(np.exp(a - m), axis=-1, keepdims=True))
        return a - lse


def kl_ref(target_logits, draft_logits, temperature, kind, scale=1.0):
    """target_logits, draft_logits: [N, K, V].  Returns per_step [N, K]
    (L_{n,k}), loss (float) and grad [N, K, V] (d loss / d z_draft), float64."""
    zt = np.asarray(target_logits, dtype=np.float64)
    zd = np.asarray(draft_logits, dtype=np.float64)
    N, K, V = zd.shape
    T = XP(float(temperature))
    lp = log_softmax_t(zt, T)
    lq = log_softmax_t(zd, T)
    p = np.exp(lp)
    q = np.exp(lq)
    with np.errstate(invalid="ignore"):
        if kind == KIND_FORWARD:
            L = np.where(p > 0, p * (lp - lq), XP(0)).sum(axis=-1)
            g = (q - p) / T
        elif kind == KIND_CE:
            L = np.where(p > 0, -p * lq, XP(0)).sum(axis=-1)
            g = (q - p) / T
        elif kind == KIND_REVERSE:
            L = np.where(q > 0, q * (lq - lp), XP(0)).sum(axis=-1)
            g = np.where(q > 0, q * (lq - lp - L[..., None]), XP(0)) / T
        else:
            raise ValueError(kind)
    loss_pos = L.mean(axis=1)
    sc = XP(float(scale))
    return {"per_step": L.astype(np.float64), "loss": float(sc * loss_pos.sum()),
            "loss_pos": (sc * loss_pos).astype(np.float64), "grad": (g * (sc / K)).astype(np.float64)}
