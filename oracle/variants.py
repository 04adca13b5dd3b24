"""Target-only verification, the draft-stage sampler and per-step diagnostics,
in float64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Target-only verification (paper Sec. 2.2 "Target-Only Sampling", Eq.
target_only).  The draft token of step i is the draft's greedy choice
x_i = argmax q_i (given as input here, like the draft ids of rejection
sampling); it is accepted with probability p_i(x_i), the target's own
probability, and q plays no other part.  Per batch row b:

  p_i = softmax(z_target[b, i, :] / T_b)        i = 0..K
  step i accepts x_i iff u_i < p_i(x_i),  u_i = U24(word 0 of Philox((b, i, offset, 0); (seed, 0)))
  n = first rejected step, or K
  residual r = p_n with x_n removed (r(v) = p_n(v) 1[v != x_n]) if n < K, else p_K
  y* = smallest v with cumsum(r)[v] > u' * sum(r),  u' = U24(word 1 of the block at (b, n))

The emitted token is then distributed exactly as p_n: x_n with probability
p_n(x_n), any other v with (1 - p_n(x_n)) * p_n(v) / (1 - p_n(x_n)).
Readings: the uniforms are those of rejection sampling (same Philox stream,
so switching the acceptance rule changes nothing else); if the residual is
exactly 0 (p_n is one-hot on x_n, which then cannot be rejected) the sample
falls back to p_n.

Draft-stage sampler (the step before verification, App. G.1: each draft head
samples its token from softmax(z / T) of its logits): for row r with T > 0,
  token = smallest v with cumsum(p)[v] > u,  u = U24(word 0 of Philox((r, 0, offset, 1); (seed, 0))),
and with T == 0 the greedy token, the smallest index of the largest logit
(the draft choice target-only verification assumes).  Readings: counter word
3 = 1 keeps the sampler's stream apart from verification's (word 3 = 0);
T == 0 selecting greedy decoding is the usual serving convention, not the
paper's.

Per-step diagnostics (Sec. 3.1-3.3 and App. E), for i < K:
  H(p_i), H(q_i)              entropies in nats
  max p_i                     (= alpha^TO of a draft whose greedy token is the target's top-1, Prop. to_entropy)
  x^g_i = argmax q_i          the draft's greedy token (smallest index among ties)
  alpha^TO_i = p_i(x^g_i)     Eq. target_only
  alpha^RS_i = sum min(p, q)  Eq. reject_sample
  alpha_{p>q} = sum_{v: p(v) > q(v)} q(v),  alpha_{q>p} = sum_{v: q(v) >= p(v)} p(v)
                              (the overlap split by which side is larger; the
                              paper plots both without defining them; ties
                              go to the second so the two add up to alpha^RS)
  rs_preferred_i = alpha^RS_i > alpha^TO_i   (App. E: d_TV(p, q) < 1 - p(x^g))
"""

import numpy as np

from .philox import philox4x64_10, draw_words, u24
from .verify import inverse_cdf, softmax_t

_MASK64 = (1 << 64) - 1


def _bad_rows(z, T_ok, V, ids=None):
    """Rows with a data error: NaN or +inf logits, a (sub)row that is all
    -inf, a draft id outside [0, V), or T_ok False."""
    R = z.shape[0]
    zz = z.reshape(R, -1, z.shape[-1])
    bad = ~np.asarray(T_ok, dtype=bool)
    bad |= np.any(np.isnan(zz) | (zz == np.inf), axis=(1, 2))
    bad |= np.any(np.all(zz == -np.inf, axis=-1), axis=1)
    if ids is not None:
        bad |= np.any((ids < 0) | (ids >= V), axis=-1)
    return bad


def _positive(T):
    return np.isfinite(T) & (T > 0)


def verify_target_only_ref(target_logits, draft_ids, temperature, seed, offset=0, rows=None):
    """Float64 target-only verification of one batch.

    target_logits: [R, K+1, V]; draft_ids: [R, K]; temperature: scalar or [R].
    Returns accept_len [R], emitted [R, K+1], p_at_draft [R, K],
    logz_target [R, K+1], and boundary diagnostics u_accept [R, K],
    u_resample [R], resample_margin [R], zero_mass [R], row_error [R].
    Rows with a data error get accept_len = -1, emitted = -1, NaN floats.
    """
    zt = np.asarray(target_logits, dtype=np.float64)
    ids = np.asarray(draft_ids, dtype=np.int64)
    R, K1, V = zt.shape
    K = K1 - 1
    assert ids.shape == (R, K) and K >= 1
    T = np.broadcast_to(np.asarray(temperature, dtype=np.float64), (R,)).copy()
    rows = np.arange(R) if rows is None else np.asarray(rows, dtype=np.int64)
    out = {
        "accept_len": np.full(R, -1, np.int32),
        "emitted": np.full((R, K + 1), -1, np.int32),
        "p_at_draft": np.full((R, K), np.nan),
        "logz_target": np.full((R, K + 1), np.nan),
        "u_accept": np.full((R, K), np.nan),
        "u_resample": np.full(R, np.nan),
        "resample_margin": np.full(R, np.nan),
        "zero_mass": np.zeros(R, bool),
        "row_error": np.zeros(R, bool),
    }
    words = draw_words(seed, rows, np.arange(K + 1), offset)
    u_acc = u24(words[..., 0])
    u_res = u24(words[..., 1])
    bad = _bad_rows(zt, _positive(T), V, ids)
    out["row_error"][:] = bad
    for r in np.nonzero(~bad)[0]:
        p, lz = softmax_t(zt[r], T[r])                 # [K+1, V]
        px = p[np.arange(K), ids[r]]
        n = K
        for i in range(K):
            if not u_acc[r, i] < px[i]:                # accepted with probability p_i(x_i)
                n = i
                break
        res = p[n].copy()
        if n < K:
            res[ids[r, n]] = 0.0                       # residual: p_n without the rejected token
        Z = res.sum()
        zero = Z <= 0.0
        if zero:
            res = p[n].copy()
            Z = res.sum()
        u2 = u_res[r, n]
        y, C = inverse_cdf(res[None, :], np.array([u2 * Z]))
        y = int(y[0])
        Cn = C[0] / Z
        lo = Cn[y - 1] if y > 0 else 0.0
        out["accept_len"][r] = n
        em = np.full(K + 1, -1, np.int32)
        em[:n] = ids[r, :n]
        em[n] = y
        out["emitted"][r] = em
        out["p_at_draft"][r] = px
        out["logz_target"][r] = lz
        out["u_accept"][r] = u_acc[r, :K]
        out["u_resample"][r] = u2
        out["resample_margin"][r] = min(abs(u2 - Cn[y]), abs(u2 - lo))
        out["zero_mass"][r] = zero
    return out


def sampler_words(seed, rows, offset):
    """Philox blocks of the draft-stage sampler: counter (r, 0, offset, 1)."""
    rows = np.asarray(rows, dtype=np.uint64)
    ctr = np.zeros((rows.shape[0], 4), dtype=np.uint64)
    ctr[:, 0] = rows
    ctr[:, 2] = np.uint64(int(offset) & _MASK64)
    ctr[:, 3] = np.uint64(1)
    key = np.array([int(seed) & _MASK64, 0], dtype=np.uint64)
    return philox4x64_10(ctr, key)


def sample_ref(logits, temperature, seed, offset=0, rows=None):
    """Draft-stage token choice for R rows of logits [R, V].

    A row with temperature T > 0 draws by inverse CDF of softmax(z / T) at u
    (see the module docstring); a row with T == 0 takes the greedy token, the
    smallest index of the largest logit.  Returns token [R] int32, logz [R]
    (natural-log partition function of z / T; NaN for greedy rows), u [R],
    margin [R] (distance of u to the nearest CDF step bracketing the token;
    NaN for greedy rows) and row_error [R].  Rows with a data error (NaN or
    +inf logits, all -inf, T negative or not finite) give token -1.
    """
    z = np.asarray(logits, dtype=np.float64)
    R, V = z.shape
    T = np.broadcast_to(np.asarray(temperature, dtype=np.float64), (R,)).copy()
    rows = np.arange(R) if rows is None else np.asarray(rows, dtype=np.int64)
    u = u24(sampler_words(seed, rows, offset)[:, 0])
    tok = np.full(R, -1, np.int32)
    logz = np.full(R, np.nan)
    margin = np.full(R, np.nan)
    bad = _bad_rows(z, np.isfinite(T) & (T >= 0), V)
    for r in np.nonzero(~bad)[0]:
        if T[r] == 0:
            tok[r] = int(np.argmax(z[r]))              # first index of the maximum
            continue
        p, lz = softmax_t(z[r], T[r])
        logz[r] = lz
        y, C = inverse_cdf(p[None, :], np.array([u[r]]))
        y = int(y[0])
        tok[r] = y
        lo = C[0, y - 1] if y > 0 else 0.0
        margin[r] = min(abs(u[r] - C[0, y]), abs(u[r] - lo))
    return {"token": tok, "logz": logz, "u": u, "margin": margin, "row_error": bad}


DIAG_COLUMNS = ("entropy_target", "entropy_draft", "max_p", "alpha_to", "alpha_rs", "alpha_p_gt_q", "alpha_q_ge_p")


def diagnostics_ref(target_logits, draft_logits, temperature, tie_window=1e-5):
    """Per-step diagnostics for target [R, K(+1), V] (the first K rows are
    used) and draft [R, K, V] logits.  Returns a dict with float arrays
    [R, K] named by DIAG_COLUMNS, greedy_draft [R, K] int32, rs_preferred
    [R, K] bool, and tie_mass [R, K]: sum of min(p, q) over the tokens with
    |p - q| <= tie_window * max(p, q), the most that alpha_{p>q} and
    alpha_{q>p} can move when p and q are known only to that relative
    precision.  Rows with a data error give NaN / -1 / False.
    """
    zt = np.asarray(target_logits, dtype=np.float64)
    zd = np.asarray(draft_logits, dtype=np.float64)
    R, K, V = zd.shape
    zt = zt[:, :K]
    T = np.broadcast_to(np.asarray(temperature, dtype=np.float64), (R,)).copy()
    out = {c: np.full((R, K), np.nan) for c in DIAG_COLUMNS}
    out["greedy_draft"] = np.full((R, K), -1, np.int32)
    out["rs_preferred"] = np.zeros((R, K), bool)
    out["tie_mass"] = np.full((R, K), np.nan)
    bad = _bad_rows(zt, _positive(T), V) | _bad_rows(zd, _positive(T), V)
    out["row_error"] = bad
    for r in np.nonzero(~bad)[0]:
        p, _ = softmax_t(zt[r], T[r])
        q, _ = softmax_t(zd[r], T[r])
        with np.errstate(divide="ignore", invalid="ignore"):
            hp = -np.sum(np.where(p > 0, p * np.log(p), 0.0), axis=-1)
            hq = -np.sum(np.where(q > 0, q * np.log(q), 0.0), axis=-1)
        g = np.argmax(zd[r], axis=-1)                  # first index of the maximum
        a_to = p[np.arange(K), g]
        mn = np.minimum(p, q)
        a_rs = mn.sum(axis=-1)
        out["entropy_target"][r] = hp
        out["entropy_draft"][r] = hq
        out["max_p"][r] = p.max(axis=-1)
        out["alpha_to"][r] = a_to
        out["alpha_rs"][r] = a_rs
        out["alpha_p_gt_q"][r] = np.where(p > q, q, 0.0).sum(axis=-1)
        out["alpha_q_ge_p"][r] = np.where(q >= p, p, 0.0).sum(axis=-1)
        out["greedy_draft"][r] = g
        out["rs_preferred"][r] = a_rs > a_to
        out["tie_mass"][r] = np.where(np.abs(p - q) <= tie_window * np.maximum(p, q), mn, 0.0).sum(axis=-1)
    return out
