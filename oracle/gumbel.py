"""Gumbel-max verification and the Gumbel-max draft sampler, in float64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Paper App. G.2 (Alg. rs_gumbel): the acceptance loop is that of rejection
sampling (u_i q_i(x_i) < p_i(x_i), first rejection ends the chain); the token
at the emitting position n is drawn by the Gumbel-max trick instead of a CDF
inversion:

  z_resid(v) = log max(0, p_n(v) - q_n(v))   if n < K  (-inf where p_n <= q_n)
  z_resid(v) = z_target[K](v) / T            if n = K  (the bonus)
  y* = argmax_v [ z_resid(v) + G_v ],  G_v = -log(-log U_v)  i.i.d. Gumbel(0, 1)

The draft stage of the same appendix samples x = argmax_v [z(v) / T + G_v].

Readings:
  * the bonus uses the temperature-scaled target logits z/T (the appendix
    writes the raw logits; with T = 1 they coincide, and only z/T makes the
    bonus follow p_K);
  * the V uniforms of a row come from Philox4x64-10 with key (seed, 0) and
    counter (row, v >> 3, offset, tag): element v takes word (v >> 1) & 3 of
    that block, its top 24 bits for even v and bits 8..31 for odd v, as
    U = (bits + 1/2) 2^-24, strictly inside (0, 1); tag 2 for verification,
    tag 3 for the draft sampler (tags 0 and 1 are the accept / resample and
    multinomial-sampler streams);
  * if the residual has no mass the sample is drawn from p_n (as in the
    multinomial variant);
  * ties in the score go to the smallest index (argmax's first maximum);
  * T = 0 in the draft sampler selects the greedy token.
"""

import numpy as np

from .philox import philox4x64_10
from .verify import softmax_t, verify_ref

_MASK64 = (1 << 64) - 1
TAG_VERIFY = 2
TAG_SAMPLE = 3


def gumbel_uniforms(seed, rows, V, offset, tag):
    """U [R, V] in (0, 1) for the given batch rows (see the module docstring)."""
    rows = np.asarray(rows, dtype=np.uint64)
    nblk = (V + 7) // 8
    ctr = np.zeros((rows.shape[0], nblk, 4), dtype=np.uint64)
    ctr[..., 0] = rows[:, None]
    ctr[..., 1] = np.arange(nblk, dtype=np.uint64)[None, :]
    ctr[..., 2] = np.uint64(int(offset) & _MASK64)
    ctr[..., 3] = np.uint64(tag)
    key = np.array([int(seed) & _MASK64, 0], dtype=np.uint64)
    w = philox4x64_10(ctr, key)                            # [R, nblk, 4]
    hi = w >> np.uint64(40)                                # top 24 bits: even elements
    lo = (w >> np.uint64(8)) & np.uint64(0xFFFFFF)         # bits 8..31: odd elements
    bits = np.stack([hi, lo], axis=-1).reshape(rows.shape[0], nblk * 8)[:, :V]
    return (bits.astype(np.float64) + 0.5) * 2.0 ** -24


def gumbel_noise(U):
    return -np.log(-np.log(U))


def _argmax_first(score):
    return int(np.argmax(score))                           # first index of the maximum


def verify_gumbel_ref(target_logits, draft_logits, draft_ids, temperature, seed, offset=0, rows=None):
    """Alg. rs_gumbel for one batch.  Same arguments and outputs as
    verify_ref, with emitted[n] drawn by the Gumbel-max trick; adds
    gumbel_score [R, V] (the float64 scores of the emitting row),
    gumbel_sens [R, V] ((p + q) / r for residual rows, 1 for bonus and
    fallback rows: how strongly the relative rounding of p and q moves each
    token's log residual) and gumbel_fallback [R]."""
    zt = np.asarray(target_logits, dtype=np.float64)
    zd = np.asarray(draft_logits, dtype=np.float64)
    R, K1, V = zt.shape
    K = K1 - 1
    rows = np.arange(R) if rows is None else np.asarray(rows, dtype=np.int64)
    T = np.broadcast_to(np.asarray(temperature, dtype=np.float64), (R,)).copy()
    out = verify_ref(zt, zd, draft_ids, T, seed, offset, rows=rows)
    U = gumbel_uniforms(seed, rows, V, offset, TAG_VERIFY)
    G = gumbel_noise(U)
    out["gumbel_score"] = np.full((R, V), np.nan)
    out["gumbel_sens"] = np.full((R, V), np.nan)
    out["gumbel_fallback"] = np.zeros(R, bool)
    for r in range(R):
        n = int(out["accept_len"][r])
        if n < 0:
            continue
        if n < K:
            p, _ = softmax_t(zt[r, n], T[r])
            q, _ = softmax_t(zd[r, n], T[r])
            res = np.maximum(0.0, p - q)
            if res.sum() > 0.0:
                with np.errstate(divide="ignore"):
                    z_resid = np.log(res)
                    sens = np.where(res > 0, (p + q) / np.where(res > 0, res, 1.0), np.inf)
            else:                                          # no residual mass: draw from p_n
                z_resid = zt[r, n] / T[r]
                sens = np.ones(V)
                out["gumbel_fallback"][r] = True
        else:
            z_resid = zt[r, K] / T[r]
            sens = np.ones(V)
        score = z_resid + G[r]
        out["emitted"][r, n] = _argmax_first(score)
        out["gumbel_score"][r] = score
        out["gumbel_sens"][r] = sens
    return out


def sample_gumbel_ref(logits, temperature, seed, offset=0, rows=None):
    """Gumbel-max draft sampler for logits [R, V]: token [R] int32 (-1 on a
    row error), score [R, V] float64 (NaN for greedy and error rows)."""
    z = np.asarray(logits, dtype=np.float64)
    R, V = z.shape
    T = np.broadcast_to(np.asarray(temperature, dtype=np.float64), (R,)).copy()
    rows = np.arange(R) if rows is None else np.asarray(rows, dtype=np.int64)
    G = gumbel_noise(gumbel_uniforms(seed, rows, V, offset, TAG_SAMPLE))
    tok = np.full(R, -1, np.int32)
    score = np.full((R, V), np.nan)
    bad = ~(np.isfinite(T) & (T >= 0))
    bad |= np.any(np.isnan(z) | (z == np.inf), axis=-1)
    bad |= np.all(z == -np.inf, axis=-1)
    for r in np.nonzero(~bad)[0]:
        if T[r] == 0:
            tok[r] = _argmax_first(z[r])
            continue
        score[r] = z[r] / T[r] + G[r]
        tok[r] = _argmax_first(score[r])
    return {"token": tok, "score": score, "row_error": bad}
