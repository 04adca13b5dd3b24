"""Philox4x64-10, written from its published definition.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Definition (Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers: As Easy as
1, 2, 3", SC'11, Sec. 3.2 "Philox"): a 4-word counter (c0, c1, c2, c3) of
64-bit words and a 2-word key (k0, k1).  One round maps

    (hi0, lo0) = full 128-bit product  M0 * c0
    (hi1, lo1) = full 128-bit product  M1 * c2
    c' = (hi1 ^ c1 ^ k0,  lo1,  hi0 ^ c3 ^ k1,  lo0)

and between rounds the key is bumped by the Weyl constants (W0, W1) modulo
2^64.  Ten rounds are applied; the first uses the key as given.  The
multipliers and Weyl constants are the ones the paper's authors published
for the 4x64 variant.

Stream used by the verification method (the paper only says the uniforms
are seeded by the request's seed and position, App. G.2): key = (seed, 0),
counter = (row, step, offset, 0).  Word 0 of that block drives the accept
test of draft step ``step``; word 1 drives the residual / bonus resample when
``step`` is the emitting position.  U24(w) = (w >> 40) * 2^-24 in [0, 1),
exactly representable in float32.
"""

import numpy as np

_MASK64 = (1 << 64) - 1
PHILOX_M0 = 0xD2E7470EE14C6C93
PHILOX_M1 = 0xCA5A826395121157
PHILOX_W0 = 0x9E3779B97F4A7C15
PHILOX_W1 = 0xBB67AE8584CAA73B
_LO32 = np.uint64(0xFFFFFFFF)
_S32 = np.uint64(32)


def _mulhilo(a, m):
    """Full 64x64 -> 128-bit product of uint64 array ``a`` and constant ``m``,
    returned as (hi, lo) uint64 arrays.  Done in 32-bit limbs so that every
    partial product fits in 64 bits."""
    a = np.asarray(a, dtype=np.uint64)
    m_lo = np.uint64(m & 0xFFFFFFFF)
    m_hi = np.uint64(m >> 32)
    a_lo = a & _LO32
    a_hi = a >> _S32
    p0 = a_lo * m_lo
    p1 = a_lo * m_hi
    p2 = a_hi * m_lo
    p3 = a_hi * m_hi
    mid = (p0 >> _S32) + (p1 & _LO32) + (p2 & _LO32)
    hi = p3 + (p1 >> _S32) + (p2 >> _S32) + (mid >> _S32)
    lo = a * np.uint64(m)  # wraps modulo 2^64
    return hi, lo


def philox4x64_10(counter, key):
    """Philox4x64 with 10 rounds.

    counter: array-like of shape [..., 4] (uint64 words c0..c3)
    key:     array-like of shape [..., 2] (uint64 words k0, k1), broadcastable
    returns: uint64 array of shape [..., 4]
    """
    with np.errstate(over="ignore"):
        c = np.array(counter, dtype=np.uint64, copy=True)
        k = np.array(key, dtype=np.uint64, copy=True)
        c0, c1, c2, c3 = c[..., 0], c[..., 1], c[..., 2], c[..., 3]
        k0 = np.broadcast_to(k[..., 0], c0.shape).copy()
        k1 = np.broadcast_to(k[..., 1], c0.shape).copy()
        for rnd in range(10):
            if rnd > 0:
                k0 = k0 + np.uint64(PHILOX_W0)
                k1 = k1 + np.uint64(PHILOX_W1)
            hi0, lo0 = _mulhilo(c0, PHILOX_M0)
            hi1, lo1 = _mulhilo(c2, PHILOX_M1)
            c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
        return np.stack([c0, c1, c2, c3], axis=-1)


def u24(word):
    """Top 24 bits of a 64-bit word as a uniform on the 2^-24 grid in [0, 1).
    Returned as float64 (the value is exact in float32 as well)."""
    w = np.asarray(word, dtype=np.uint64)
    return (w >> np.uint64(40)).astype(np.float64) * (2.0 ** -24)


def draw_words(seed, rows, steps, offset):
    """Philox blocks for every (row, step) pair of the verification stream.

    rows:  1-D array of row indices b;  steps: 1-D array of step indices i.
    Returns uint64 [len(rows), len(steps), 4] = Philox((b, i, offset, 0); (seed, 0)).
    """
    rows = np.asarray(rows, dtype=np.uint64)
    steps = np.asarray(steps, dtype=np.uint64)
    R, S = rows.shape[0], steps.shape[0]
    ctr = np.zeros((R, S, 4), dtype=np.uint64)
    ctr[..., 0] = rows[:, None]
    ctr[..., 1] = steps[None, :]
    ctr[..., 2] = np.uint64(int(offset) & _MASK64)
    key = np.array([int(seed) & _MASK64, 0], dtype=np.uint64)
    return philox4x64_10(ctr, key)
