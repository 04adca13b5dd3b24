"""Chain rejection-sampling verification of K draft tokens, in float64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What is computed, per batch row b (paper Sec. 2.2 "Rejection Sampling",
Eq. reject_sample; App. G.1 and its Alg. rs_multinomial):

  p_i = softmax(z_target[b, i, :] / T_b)   for i = 0..K   (row K: bonus position)
  q_i = softmax(z_draft[b, i, :]  / T_b)   for i = 0..K-1
  alpha_i = sum_v min(p_i(v), q_i(v))      (= 1 - d_TV(p_i, q_i), Eq. rs_tv)
  step i accepts draft x_i iff  u_i * q_i(x_i) < p_i(x_i)   (no division),
  u_i = U24(word 0 of Philox((b, i, offset, 0); (seed, 0)))
  n = first rejected step, or K if none (sequential early exit)
  residual r = max(0, p_n - q_n) if n < K, else p_K (bonus token)
  Z = sum_v r(v),  C = cumulative sum of r in vocabulary order
  y* = smallest v with C[v] > u' * Z,  u' = U24(word 1 of the block at (b, n))
  emitted = x_0..x_{n-1}, y*, then -1 padding;  accept_len = n

Readings taken where the paper is silent or inconsistent:
  * the bonus token comes from target row K, the position after the last
    draft (the algorithm writes p_gamma with gamma 1-based);
  * the CDF inversion uses a strict ">" ("first exceeds" in App. G.1) so a
    zero-mass token can never be emitted;
  * one temperature per row applies to both target and draft logits;
  * if Z underflows to exactly 0 the sample is drawn from p_n instead;
  * alpha is reported for every draft step, also those after the first
    rejection, since it is a property of (p_i, q_i) only.

Row data errors (NaN or +inf logits, a row that is entirely -inf, a draft id
outside [0, V), a temperature that is not a positive finite number) mark the
whole batch row: accept_len = -1, emitted = -1, every float output NaN.
-inf entries are legal and mean probability 0.
"""

import numpy as np

from .philox import draw_words, u24


def softmax_t(z, T):
    """Temperature softmax along the last axis in float64.

    z: [..., V] logits; T: scalar or array broadcastable to z[..., :1].
    Returns (prob, log_normaliser) where log_normaliser = max(z/T) +
    log(sum exp(z/T - max)) is the natural-log partition function of z/T.
    """
    a = np.asarray(z, dtype=np.float64) / T
    m = np.max(a, axis=-1, keepdims=True)
    with np.errstate(invalid="ignore", over="ignore"):
        e = np.exp(a - m)
    d = np.sum(e, axis=-1, keepdims=True)
    with np.errstate(invalid="ignore", divide="ignore"):
        prob = e / d
        logz = (m + np.log(d))[..., 0]
    return prob, logz


def inverse_cdf(r, t):
    """Smallest index v with cumsum(r)[v] > t, for each leading row.

    r: [R, V] non-negative masses; t: [R] thresholds.  Returns (index [R],
    cumulative sums [R, V]).  Equivalent to searchsorted(C, t, side='right').
    """
    C = np.cumsum(r, axis=-1)
    above = C > t[:, None]
    idx = np.where(above.any(axis=-1), above.argmax(axis=-1), r.shape[-1] - 1)
    return idx, C


def residual_sample(p, q, u):
    """Residual / bonus resample for a batch of rows.

    p: [R, V] target probabilities; q: [R, V] draft probabilities, or None
    for the bonus case (residual = p).  u: [R] uniforms in [0, 1).
    Returns (token [R], Z [R], C [R, V], zero_mass_fallback [R] bool).
    """
    if q is None:
        r = p.copy()
    else:
        r = np.maximum(0.0, p - q)
    Z = r.sum(axis=-1)
    zero = Z <= 0.0
    if np.any(zero):
        r[zero] = p[zero]
        Z = r.sum(axis=-1)
    tok, C = inverse_cdf(r, u * Z)
    return tok, Z, C, zero


def _row_errors(zt, zd, ids, T, V):
    bad = ~(np.isfinite(T) & (T > 0))
    bad |= np.any((ids < 0) | (ids >= V), axis=-1)
    for z in (zt, zd):
        bad |= np.any(np.isnan(z) | (z == np.inf), axis=(-2, -1))
        bad |= np.any(np.all(z == -np.inf, axis=-1), axis=-1)
    return bad


def verify_ref(target_logits, draft_logits, draft_ids, temperature, seed, offset=0,
               rows=None):
    """Float64 verification of one batch.

    target_logits: [R, K+1, V] (any real dtype; widened exactly to float64)
    draft_logits:  [R, K, V]
    draft_ids:     [R, K] integer
    temperature:   scalar or [R]
    seed, offset:  Philox key word 0 and counter word 2
    rows:          the batch-row index b of each of the R given rows (the
                   Philox counter uses it); default 0..R-1.  Lets the oracle
                   check a sample of rows taken out of a large batch.

    Returns a dict of numpy arrays:
      accept_len [R] int32, emitted [R, K+1] int32, overlap [R, K],
      p_at_draft / q_at_draft [R, K], logz_target [R, K+1], logz_draft [R, K]
      (natural-log partition functions of z/T), and diagnostics used to
      classify boundary draws: u_accept [R, K], ratio [R, K] = p(x)/q(x),
      u_resample [R], resample_margin [R] (distance of u' to the nearest
      CDF step C/Z bracketing it), zero_mass [R], row_error [R], and
      logit_range [R, K]: the larger of the target and draft rows' spans of
      finite logits over T (the size of the exponent differences that a
      float32 temperature scale multiplies).
    """
    zt = np.asarray(target_logits, dtype=np.float64)
    zd = np.asarray(draft_logits, dtype=np.float64)
    ids = np.asarray(draft_ids, dtype=np.int64)
    R, K1, V = zt.shape
    K = K1 - 1
    assert zd.shape == (R, K, V) and ids.shape == (R, K) and K >= 1
    T = np.broadcast_to(np.asarray(temperature, dtype=np.float64), (R,)).copy()
    rows = np.arange(R) if rows is None else np.asarray(rows, dtype=np.int64)

    out = {
        "accept_len": np.full(R, -1, np.int32),
        "emitted": np.full((R, K + 1), -1, np.int32),
        "overlap": np.full((R, K), np.nan),
        "p_at_draft": np.full((R, K), np.nan),
        "q_at_draft": np.full((R, K), np.nan),
        "logz_target": np.full((R, K + 1), np.nan),
        "logz_draft": np.full((R, K), np.nan),
        "u_accept": np.full((R, K), np.nan),
        "ratio": np.full((R, K), np.nan),
        "u_resample": np.full(R, np.nan),
        "resample_margin": np.full(R, np.nan),
        "zero_mass": np.zeros(R, bool),
        "row_error": np.zeros(R, bool),
    }
    with np.errstate(invalid="ignore", divide="ignore"):
        def span(z):
            f = np.isfinite(z)
            hi = np.where(f, z, -np.inf).max(axis=-1)
            lo = np.where(f, z, np.inf).min(axis=-1)
            return np.where(f.any(axis=-1), hi - lo, 0.0)
        out["logit_range"] = np.maximum(span(zt[:, :K]), span(zd)) / T[:, None]
    words = draw_words(seed, rows, np.arange(K + 1), offset)      # [R, K+1, 4]
    u_acc_all = u24(words[..., 0])
    u_res_all = u24(words[..., 1])

    chunk = max(1, (1 << 22) // ((2 * K + 1) * V))
    for s in range(0, R, chunk):
        sl = slice(s, min(R, s + chunk))
        r_n = sl.stop - sl.start
        bad = _row_errors(zt[sl], zd[sl], ids[sl], T[sl], V)
        out["row_error"][sl] = bad
        good = np.nonzero(~bad)[0]
        if good.size == 0:
            continue
        g = good + s
        Tg = T[g][:, None, None]
        p, lzt = softmax_t(zt[g], Tg)                               # [G, K+1, V]
        q, lzd = softmax_t(zd[g], Tg)                               # [G, K, V]
        alpha = np.minimum(p[:, :K], q).sum(axis=-1)                # [G, K]
        xi = ids[g]
        gi = np.arange(g.size)[:, None]
        ki = np.arange(K)[None, :]
        px = p[gi, ki, xi]
        qx = q[gi, ki, xi]
        u = u_acc_all[g, :K]
        reject = u * qx >= px                                       # Alg. rs_multinomial
        n = np.where(reject.any(axis=1), reject.argmax(axis=1), K)
        # residual at step n (rejected draft) or the bonus row K
        pn = p[np.arange(g.size), n]
        qn = np.where((n < K)[:, None], q[np.arange(g.size), np.minimum(n, K - 1)], 0.0)
        r = np.where((n < K)[:, None], np.maximum(0.0, pn - qn), pn)
        Z = r.sum(axis=-1)
        zero = Z <= 0.0
        r[zero] = pn[zero]
        Z = r.sum(axis=-1)
        u2 = u_res_all[g, n]
        y, C = inverse_cdf(r, u2 * Z)
        Cn = C / Z[:, None]
        hi = Cn[np.arange(g.size), y]
        lo = np.where(y > 0, Cn[np.arange(g.size), np.maximum(y - 1, 0)], 0.0)
        margin = np.minimum(np.abs(u2 - hi), np.abs(u2 - lo))

        em = np.full((g.size, K + 1), -1, np.int32)
        for j in range(K):
            em[:, j] = np.where(j < n, xi[:, j], -1)
        em[np.arange(g.size), n] = y
        out["accept_len"][g] = n
        out["emitted"][g] = em
        out["overlap"][g] = alpha
        out["p_at_draft"][g] = px
        out["q_at_draft"][g] = qx
        out["logz_target"][g] = lzt
        out["logz_draft"][g] = lzd
        out["u_accept"][g] = u
        with np.errstate(divide="ignore", invalid="ignore"):
            out["ratio"][g] = px / qx
        out["u_resample"][g] = u2
        out["resample_margin"][g] = margin
        out["zero_mass"][g] = zero
        del r_n
    return out
