"""Oracle: masked softmax attention of draft slots against a reused prefix cache.

TEST INFRASTRUCTURE ONLY (see the package docstring). Float64 numpy.

Paper passages this follows:

* Sec. 5.2 (Mode B, "Reordering"): before the first forward pass the masked
  tokens are placed after the unmasked ones, so one scoring call sees the
  committed prefix (P tokens, already in the KV cache) followed by the S draft
  slots of L tokens each, slot 0 first.
* Sec. 5.1 (closing paragraph, the KV-reuse argument): tokens fixed at a step
  precede the masked positions, so under causal attention the cached prefix
  states never change; every draft token therefore sees the whole prefix and
  the prefix itself is read-only.
* Sec. 5.2 "Draft phase": one forward pass drafts all slots of the block in
  parallel.  Read here as the DIFFUSION pass: a draft token sees the prefix and
  every token of its own slot (bidirectional inside the slot).
* Sec. 5.2 "Verification phase": the selected slots get an autoregressive
  forward pass.  Read here as the AR_INFILL pass: a token sees the prefix and
  the tokens of its own slot at or before it (causal inside the slot).
* Sec. 3.1 (causal masked reconstruction) and Sec. 1 (clean slots precede
  masked ones, both groups permuted): in the reordered training layout the
  backbone keeps causal attention.  ``cross_slot=CAUSAL`` adds the earlier
  slots to what a token sees, which with every slot in the AR_INFILL pass is
  ordinary causal attention in physical order.

* Sec. 5.2 "KV cache update": accepted tokens are appended to the cache, so
  after a verification step the batch rows of one call can hold prefixes of
  different lengths.  ``prefix_len`` is either one length for every row or one
  length per batch row.

Readings where the paper is silent (each listed in the design notes):
draft slots do not see each other in the scoring pass (``cross_slot=NONE``);
query head h uses KV head floor(h / (Hq / Hkv)); the softmax scale is an
argument (1/sqrt(head_dim) in the workloads).
"""

from __future__ import annotations

import math

import numpy as np

PASS_DIFFUSION = 0
PASS_AR_INFILL = 1
CROSS_SLOT_NONE = 0
CROSS_SLOT_CAUSAL = 1


def prefix_lengths(prefix_len, batch):
    """Per-batch-row prefix lengths from one int or a length-``batch`` sequence."""
    if np.ndim(prefix_len) == 0:
        return [int(prefix_len)] * batch
    pl = [int(x) for x in np.asarray(prefix_len).reshape(-1)]
    assert len(pl) == batch
    return pl


def _slot_passes(n_slots, pass_, slot_pass):
    """Pass of every slot: the per-slot override if given, else the call's pass."""
    if slot_pass is None:
        return np.full(n_slots, pass_, dtype=np.int64)
    sp = np.asarray(slot_pass, dtype=np.int64).reshape(n_slots)
    return sp


def visibility(prefix_len, n_slots, slot_len, pass_, cross_slot=CROSS_SLOT_NONE, slot_pass=None):
    """Boolean mask [T, P + T]: may draft token t see key j?

    Keys 0..P-1 are the cached prefix, keys P..P+T-1 are the draft tokens in
    slot-major order (slot s, position r at index P + s*L + r).
    """
    P, S, L = int(prefix_len), int(n_slots), int(slot_len)
    T = S * L
    passes = _slot_passes(S, pass_, slot_pass)
    mask = np.zeros((T, P + T), dtype=bool)
    mask[:, :P] = True  # the whole committed prefix is visible (Sec. 5.1 KV reuse)
    for s in range(S):
        rows = slice(s * L, (s + 1) * L)
        own = slice(P + s * L, P + (s + 1) * L)
        if passes[s] == PASS_DIFFUSION:
            mask[rows, own] = True  # bidirectional inside the slot
        else:
            mask[rows, own] = np.tril(np.ones((L, L), dtype=bool))  # causal inside the slot
        if cross_slot == CROSS_SLOT_CAUSAL and s > 0:
            mask[rows, P : P + s * L] = True  # every earlier slot
    return mask


def slot_attention(
    q,
    k_cache,
    v_cache,
    k_slot,
    v_slot,
    prefix_len,
    n_slots,
    slot_len,
    scale,
    pass_,
    cross_slot=CROSS_SLOT_NONE,
    slot_pass=None,
    return_probs=False,
):
    """Masked softmax attention, float64.

    q       [B, Hq, T, D]       draft-token queries, rows (slot, position)
    k_cache [B, Hkv, C, D]      prefix keys (first ``prefix_len`` rows valid;
                                ``prefix_len`` is an int or one length per row)
    v_cache [B, Hkv, C, D]
    k_slot  [B, Hkv, T, D]      the draft tokens' own keys
    v_slot  [B, Hkv, T, D]
    slot_pass: optional [B, S] per-slot pass (overrides ``pass_``)

    Returns O [B, Hq, T, D] and LSE [B, Hq, T] (natural log of the softmax
    denominator including the max shift), and the probabilities
    [B, Hq, T, P + T] when ``return_probs``.
    """
    q = np.asarray(q, dtype=np.float64)
    B, Hq, T, D = q.shape
    Hkv = k_slot.shape[1]
    assert Hq % Hkv == 0 and T == n_slots * slot_len
    G = Hq // Hkv
    plens = prefix_lengths(prefix_len, B)
    out = np.empty((B, Hq, T, D), dtype=np.float64)
    lse = np.empty((B, Hq, T), dtype=np.float64)
    if return_probs:
        assert len(set(plens)) == 1, "probabilities are returned for one common prefix length"
    probs = np.empty((B, Hq, T, plens[0] + T), dtype=np.float64) if return_probs else None
    for b in range(B):
        P = plens[b]
        sp = None if slot_pass is None else np.asarray(slot_pass)[b]
        mask = visibility(P, n_slots, slot_len, pass_, cross_slot, sp)
        for g in range(Hkv):
            keys = np.concatenate(
                [np.asarray(k_cache[b, g, :P], dtype=np.float64), np.asarray(k_slot[b, g], dtype=np.float64)]
            )
            vals = np.concatenate(
                [np.asarray(v_cache[b, g, :P], dtype=np.float64), np.asarray(v_slot[b, g], dtype=np.float64)]
            )
            for h in range(g * G, (g + 1) * G):
                scores = scale * (q[b, h] @ keys.T)
                scores = np.where(mask, scores, -np.inf)
                m = scores.max(axis=1, keepdims=True)
                p = np.exp(scores - m)
                denom = p.sum(axis=1, keepdims=True)
                out[b, h] = (p @ vals) / denom
                lse[b, h] = m[:, 0] + np.log(denom[:, 0])
                if return_probs:
                    probs[b, h] = p / denom
    if return_probs:
        return out, lse, probs
    return out, lse


def slot_attention_loops(
    q, k_cache, v_cache, k_slot, v_slot, prefix_len, n_slots, slot_len, scale, pass_,
    cross_slot=CROSS_SLOT_NONE, slot_pass=None,
):
    """Brute force for tiny shapes: scalar Python loops, one key at a time.

    Visibility is decided per (query, key) from the physical position of each
    token, independently of :func:`visibility`.
    """
    B, Hq, T, D = np.shape(q)
    Hkv = np.shape(k_slot)[1]
    G = Hq // Hkv
    plens, L = prefix_lengths(prefix_len, B), int(slot_len)
    out = np.zeros((B, Hq, T, D))
    lse = np.zeros((B, Hq, T))
    for b in range(B):
        P = plens[b]
        for h in range(Hq):
            g = h // G
            for t in range(T):
                s_q, r_q = t // L, t % L
                qp = pass_ if slot_pass is None else int(slot_pass[b][s_q])
                scores = []
                values = []
                for j in range(P + T):
                    if j < P:
                        ok, kv = True, (k_cache[b][g][j], v_cache[b][g][j])
                    else:
                        s_k, r_k = (j - P) // L, (j - P) % L
                        if s_k == s_q:
                            ok = qp == PASS_DIFFUSION or r_k <= r_q
                        else:
                            ok = cross_slot == CROSS_SLOT_CAUSAL and s_k < s_q
                        kv = (k_slot[b][g][j - P], v_slot[b][g][j - P])
                    if not ok:
                        continue
                    dot = 0.0
                    for d in range(D):
                        dot += float(q[b][h][t][d]) * float(kv[0][d])
                    scores.append(scale * dot)
                    values.append(kv[1])
                mx = max(scores)
                w = [math.exp(x - mx) for x in scores]
                tot = sum(w)
                for d in range(D):
                    acc = 0.0
                    for wi, vi in zip(w, values):
                        acc += wi * float(vi[d])
                    out[b, h, t, d] = acc / tot
                lse[b, h, t] = mx + math.log(tot)
    return out, lse
