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
log-probabilities (log q - log p - L).  Where one token holds all but 1e-14
of both distributions, q - p of that token is a difference of two numbers
within 1e-14 of 1; where two tokens share the mass of two nearly equal
distributions, log q - log p of each is the small difference of two log
partition functions.  So every quantity is evaluated in extended precision
(numpy.longdouble, a 64-bit significand on x86-64), and the log ratio of one
element is formed without subtracting two separately rounded log partition
functions:

  log q_v - log p_v = w_v - log(1 + X / Z_t'),  w_v = ((zd_v - zt_v) - (max zd - max zt)) / T,
  Z_t' = sum_v e^(zt_v / T - max zt / T),  X = Z_d' - Z_t' = sum_v e^(zt_v / T - max zt / T) (e^(w_v) - 1),

with e^w - 1 and log(1 + x) evaluated by expm1 and log1p, and
q - p = p (e^(log q - log p) - 1).  For reverse KL, with d = log q - log p
and the q_u summing to 1, d_v - L = (d_v - d_r) + sum_u q_u (d_r - d_u) for
any element r; r is the draft's first largest element and each d_v - d_r =
((zd_v - zt_v) - (zd_r - zt_r)) / T comes from the logits (the partition
functions cancel), so no term is a small difference of two large log ratios
where the draft's mass sits on tokens whose log ratios nearly agree (one
token holding nearly all of q, or several with nearly equal d).  Results
are returned as float64.
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
    dl = log_ratio(zt, zd, T)  # log q - log p
    with np.errstate(invalid="ignore"):
        # q - p: p (e^dl - 1) where p > 0 (dl = -inf gives -p), q where p = 0
        qmp = np.where(p > 0, p * np.expm1(dl), q)
        if kind == KIND_FORWARD:
            L = np.where(p > 0, -p * dl, XP(0)).sum(axis=-1)
            g = qmp / T
        elif kind == KIND_CE:
            L = np.where(p > 0, -p * lq, XP(0)).sum(axis=-1)
            g = qmp / T
        elif kind == KIND_REVERSE:
            qdl = np.where(q > 0, q * dl, XP(0))
            L = qdl.sum(axis=-1)
            # dl_v - L = (dl_v - dl_r) + sum_u q_u (dl_r - dl_u), r the
            # draft's first largest element, dl_v - dl_r from the logits;
            # rows where that sum is not finite (a token with p = 0 and
            # q > 0) keep q (dl - L)
            r = np.argmax(zd, axis=-1)[..., None]
            x = (np.asarray(zd, dtype=XP) - np.asarray(zt, dtype=XP)) / T
            dv = x - np.take_along_axis(x, r, axis=-1)
            comp = np.where(q > 0, -q * dv, XP(0)).sum(axis=-1, keepdims=True)
            g_ref = np.where(q > 0, q * (dv + comp), XP(0))
            g_plain = np.where(q > 0, q * (dl - L[..., None]), XP(0))
            g = np.where(np.isfinite(comp), g_ref, g_plain) / T
        else:
            raise ValueError(kind)
    loss_pos = L.mean(axis=1)
    sc = XP(float(scale))
    return {"per_step": L.astype(np.float64), "loss": float(sc * loss_pos.sum()),
            "loss_pos": (sc * loss_pos).astype(np.float64), "grad": (g * (sc / K)).astype(np.float64)}


def log_ratio(target_logits, draft_logits, T):
    """log q_v - log p_v along the last axis in extended precision, from the
    exact logit differences and the pairwise difference X = Z_d' - Z_t' of
    the two partition sums taken relative to each row's largest logit (see
    the module docstring).  Elements whose p or q is zero get -inf / +inf
    (both zero: NaN, never used)."""
    zt = np.asarray(target_logits, dtype=XP)
    zd = np.asarray(draft_logits, dtype=XP)
    T = XP(T)
    mt = np.max(zt, axis=-1, keepdims=True)
    md = np.max(zd, axis=-1, keepdims=True)
    with np.errstate(invalid="ignore", over="ignore", divide="ignore"):
        ea = np.exp((zt - mt) / T)
        eb = np.exp((zd - md) / T)
        w = ((zd - zt) - (md - mt)) / T
        both = (ea > 0) & (eb > 0)
        # e^(b') - e^(a') per element: ea (e^w - 1) where both are non-zero,
        # else the one non-zero term
        diff = np.where(both, ea * np.expm1(np.where(both, w, XP(0))), eb - ea)
        X = diff.sum(axis=-1, keepdims=True)
        Zt = ea.sum(axis=-1, keepdims=True)
        return np.where(both, w - np.log1p(X / Zt), np.log(eb) - np.log(ea) - np.log1p(X / Zt))
