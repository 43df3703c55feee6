"""Oracle: full-vocabulary softmax statistics of the LM head, float64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Paper passages this follows:

* Sec. 5.2 "Draft phase": the confidence of a slot is the probability of its
  first token; "Verification phase": a token is accepted when its probability
  exceeds ``token_threshold``.  Both are the softmax of the LM-head logits.
* Sec. 5.1 step 3: the model yields logits for the masked positions.
* Table 1: every model ties its embedding, so the LM head is the token
  embedding matrix W of shape [V, H] and logits = h . W^T.

Readings where the paper is silent: the probability is taken at temperature 1
with no sampling noise; the argmax takes the lowest vocabulary id among equal
maxima.  A row whose logits include a NaN or an infinity (a NaN or infinite
hidden value, say) has no softmax: its log-sum-exp is not finite, and such a
row reports argmax -1 and NaN for every probability and the log-sum-exp.

For each row of ``hidden`` the oracle returns the max logit, its id, the
log-sum-exp of the row, the largest softmax probability ``exp(m - lse)``, the
optional probability of a given target id, and the gap between the largest
and second-largest logit (the tests use it to find rows whose argmax is
decided by rounding).
"""

from __future__ import annotations

import math

import numpy as np


def slot_confidence(hidden, w_vocab, target_ids=None, row_chunk=256):
    """Per-row softmax statistics of logits = hidden . w_vocab^T in float64.

    hidden [M, H], w_vocab [V, H], target_ids [M] (or None).
    Returns a dict of float64/int64 arrays of length M: ``max_prob``,
    ``argmax``, ``lse``, ``max_logit``, ``top2_gap`` and, when target ids are
    given, ``target_prob``.
    """
    h = np.asarray(hidden)
    w = np.asarray(w_vocab, dtype=np.float64)
    M = h.shape[0]
    out = {
        "max_prob": np.empty(M),
        "argmax": np.empty(M, dtype=np.int64),
        "lse": np.empty(M),
        "max_logit": np.empty(M),
        "top2_gap": np.empty(M),
    }
    if target_ids is not None:
        target_ids = np.asarray(target_ids, dtype=np.int64)
        out["target_prob"] = np.empty(M)
    for r0 in range(0, M, row_chunk):
        r1 = min(M, r0 + row_chunk)
        with np.errstate(invalid="ignore", over="ignore"):
            logits = np.asarray(h[r0:r1], dtype=np.float64) @ w.T
            idx = np.argmax(logits, axis=1)  # first occurrence: lowest id on ties
            m = logits[np.arange(r1 - r0), idx]
            lse = m + np.log(np.exp(logits - m[:, None]).sum(axis=1))
            bad = ~np.isfinite(lse)  # a NaN or infinite logit: no softmax
            out["argmax"][r0:r1] = np.where(bad, -1, idx)
            out["max_logit"][r0:r1] = np.where(bad, np.nan, m)
            out["lse"][r0:r1] = np.where(bad, np.nan, lse)
            out["max_prob"][r0:r1] = np.where(bad, np.nan, np.exp(m - lse))
            if logits.shape[1] > 1:
                second = np.partition(logits, -2, axis=1)[:, -2]
                out["top2_gap"][r0:r1] = np.where(bad, np.inf, m - second)
            else:
                out["top2_gap"][r0:r1] = np.inf
            if target_ids is not None:
                t = target_ids[r0:r1]
                out["target_prob"][r0:r1] = np.where(bad, np.nan, np.exp(logits[np.arange(r1 - r0), t] - lse))
    return out


def slot_confidence_loops(hidden, w_vocab, target_ids=None):
    """Brute force for small V and H: scalar loops and an exactly rounded sum."""
    M, H = np.shape(hidden)
    V = np.shape(w_vocab)[0]
    res = {k: [] for k in ("max_prob", "argmax", "lse", "target_prob")}
    for i in range(M):
        row = [float(x) for x in hidden[i]]
        logits = []
        for v in range(V):
            logits.append(math.fsum(a * float(b) for a, b in zip(row, w_vocab[v])))
        best, best_id = logits[0], 0
        for v in range(1, V):
            if logits[v] > best:
                best, best_id = logits[v], v
        lse = best + math.log(math.fsum(math.exp(x - best) for x in logits))
        if not math.isfinite(lse):  # a NaN or infinite logit: no softmax
            lse, best_id = math.nan, -1
        res["max_prob"].append(math.exp(best - lse))
        res["argmax"].append(best_id)
        res["lse"].append(lse)
        if target_ids is not None:
            res["target_prob"].append(math.exp(logits[int(target_ids[i])] - lse))
    out = {k: np.array(v) for k, v in res.items() if v}
    return out
