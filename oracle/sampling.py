"""Oracle: categorical sampling of the draft tokens with temperature (Gumbel-max).

TEST INFRASTRUCTURE ONLY (see the package docstring).  Float64 numpy.

Paper passages this follows:

* Sec. 5.2 (Mode B) "Sampling from categorical distribution": with a positive
  temperature, Gumbel noise is added to the logits to sample from the
  categorical distribution; Sec. 5.1 (Mode A) step 3 names the same Gumbel
  sampling and the temperature.  Gumbel-max: the token
  argmax_v (z_v / T + G_v) with independent standard Gumbel G_v is distributed
  as softmax(z / T).
* Sec. 5.2 "Draft phase": the confidence of a slot is the probability of its
  first token -- with sampling, of the token actually drafted.

Random numbers: Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random
numbers: as easy as 1, 2, 3", SC 2011), written here from its published
definition and checked against the published known-answer vectors.  The
uniform for vocabulary entry v of row i comes from the block with counter
(v >> 2, i, offset_lo, offset_hi) and key (seed_lo, seed_hi), output word
v & 3: u = ((x >> 9) + 1/2) * 2^-23, strictly inside (0, 1) and exactly
representable in float32.  G = -ln(-ln u).

Readings where the paper is silent (each listed in the design notes): the
counter layout above; the reported probability of the drafted token is its
model probability softmax(z)[x] (temperature 1), the same quantity the greedy
path reports as max_prob; ties of the perturbed scores go to the lowest id.
A row whose logits include a NaN or an infinity has no distribution to draw
from (its log-sum-exp is not finite): it reports sample id -1 and NaN
probabilities, as the greedy confidence does.
"""

from __future__ import annotations

import numpy as np

PHILOX_M0 = 0xD2511F53
PHILOX_M1 = 0xCD9E8D57
PHILOX_W0 = 0x9E3779B9
PHILOX_W1 = 0xBB67AE85
_MASK = np.uint64(0xFFFFFFFF)


def philox4x32(counter, key, rounds=10):
    """Philox4x32 on arrays: counter [..., 4] and key [..., 2] of uint32 values
    (broadcast together).  Returns the four output words [..., 4] as uint32."""
    c = np.asarray(counter, dtype=np.uint64)
    k = np.asarray(key, dtype=np.uint64)
    c0, c1, c2, c3 = (c[..., j] & _MASK for j in range(4))
    k0, k1 = k[..., 0] & _MASK, k[..., 1] & _MASK
    for _ in range(rounds):
        p0 = np.uint64(PHILOX_M0) * c0  # < 2^64: the full 64-bit product
        p1 = np.uint64(PHILOX_M1) * c2
        hi0, lo0 = p0 >> np.uint64(32), p0 & _MASK
        hi1, lo1 = p1 >> np.uint64(32), p1 & _MASK
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
        k0 = (k0 + np.uint64(PHILOX_W0)) & _MASK
        k1 = (k1 + np.uint64(PHILOX_W1)) & _MASK
    return np.stack([c0, c1, c2, c3], axis=-1).astype(np.uint32)


def uniforms(rows, vocab, seed, offset):
    """u[i, v] in (0, 1) for the given row indices and ids 0..vocab-1 (float64)."""
    seed, offset = int(seed), int(offset)
    rows = np.asarray(rows, dtype=np.uint64).reshape(-1)
    nb = (vocab + 3) // 4
    ctr = np.empty((rows.size, nb, 4), dtype=np.uint64)
    ctr[..., 0] = np.arange(nb, dtype=np.uint64)[None, :]
    ctr[..., 1] = rows[:, None]
    ctr[..., 2] = offset & 0xFFFFFFFF
    ctr[..., 3] = (offset >> 32) & 0xFFFFFFFF
    key = np.array([seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF], dtype=np.uint64)
    x = philox4x32(ctr, key).reshape(rows.size, nb * 4)[:, :vocab]
    return ((x >> 9).astype(np.float64) + 0.5) * 2.0 ** -23


def gumbel(u):
    """Standard Gumbel variates from uniforms in (0, 1)."""
    return -np.log(-np.log(u))


def slot_sample(hidden, w_vocab, temperature, seed, offset, row_chunk=256, row_ids=None):
    """Gumbel-max sample of every row of logits = hidden . w_vocab^T.

    ``row_ids`` are the rows' indices in the random stream (default 0..M-1;
    given when ``hidden`` holds a subset of a larger batch).
    Returns a dict: ``sample_id`` (int64), ``sample_prob`` = softmax(z)[id],
    ``lse``, ``score_gap`` (top-2 gap of the perturbed scores z/T + G, to tell
    decided rows from near-ties), ``sample_logit`` and ``best_score`` (the
    largest perturbed score).
    """
    h = np.asarray(hidden, dtype=np.float64)
    w = np.asarray(w_vocab, dtype=np.float64)
    M, V = h.shape[0], w.shape[0]
    ids = np.arange(M) if row_ids is None else np.asarray(row_ids).reshape(M)
    T = float(temperature)
    assert T > 0
    out = {k: np.empty(M) for k in ("sample_prob", "lse", "score_gap", "sample_logit", "best_score")}
    out["sample_id"] = np.empty(M, dtype=np.int64)
    for r0 in range(0, M, row_chunk):
        r1 = min(M, r0 + row_chunk)
        with np.errstate(invalid="ignore", over="ignore"):
            z = h[r0:r1] @ w.T
            u = uniforms(ids[r0:r1], V, seed, offset)
            score = z / T + gumbel(u)
            idx = np.argmax(score, axis=1)  # first (lowest) id on ties
            m = z.max(axis=1)
            lse = m + np.log(np.exp(z - m[:, None]).sum(axis=1))
            bad = ~np.isfinite(lse)  # a NaN or infinite logit: no distribution to draw from
            zx = z[np.arange(r1 - r0), idx]
            if V > 1:
                top2 = np.sort(score, axis=1)[:, -2:]
                gap = np.where(bad, np.inf, top2[:, 1] - top2[:, 0])
            else:
                gap = np.full(r1 - r0, np.inf)
            out["sample_id"][r0:r1] = np.where(bad, -1, idx)
            out["best_score"][r0:r1] = np.where(bad, np.nan, score[np.arange(r1 - r0), idx])
            out["sample_logit"][r0:r1] = np.where(bad, np.nan, zx)
            out["lse"][r0:r1] = np.where(bad, np.nan, lse)
            out["sample_prob"][r0:r1] = np.where(bad, np.nan, np.exp(zx - lse))
            out["score_gap"][r0:r1] = gap
    return out
