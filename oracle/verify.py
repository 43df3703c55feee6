"""Oracle: token acceptance after the verification pass, and the KV-cache append.

TEST INFRASTRUCTURE ONLY (see the package docstring).  Plain numpy; the
acceptance is a comparison of float32 probabilities with a float32 threshold,
the append is a copy, so both are exact.

Paper passages this follows (Sec. 5.2, Mode B: slotted speculative decoding):

* "Verification phase": the selected slots get an autoregressive forward pass;
  a draft token whose probability under that pass exceeds ``token_threshold``
  is accepted, the others go back into the speculative loop to be refined.
  Sec. 6 runs the evaluation with ``token_threshold = 0.4``.
* "KV cache update": the cache grows incrementally by the accepted tokens, so
  that verified prefixes are never recomputed.
* "Reordering" (same list) and Sec. 5.1 (KV reuse): committed tokens precede
  the undecided ones, so accepted tokens join the committed prefix.

Readings where the paper is silent (each listed in the design notes):

* ``ACCEPT_PREFIX`` (default): in a slot, the accepted tokens are the longest
  run from the slot's first token whose probabilities all exceed the
  threshold.  An autoregressive pass scores token r given tokens 0..r-1 of the
  slot, so once a token is rejected the scores of the tokens after it no longer
  hold.  ``ACCEPT_PER_TOKEN`` is the literal per-token reading: every token
  above the threshold is accepted on its own.
* "Exceeding" is strict: p > threshold.
* Only selected slots are verified; every token of an unselected slot is
  rejected.
* Accepted tokens are appended slot by slot in the given order (the selection
  order), positions inside a slot in order.  Attention over the cache does not
  depend on the order of the keys, so any fixed order works; this one keeps a
  slot's tokens contiguous.  A slot listed again in the order is skipped: the
  cache grows by the accepted tokens, each committed once.
"""

from __future__ import annotations

import numpy as np

ACCEPT_PREFIX = 0
ACCEPT_PER_TOKEN = 1


def accept_tokens(token_prob, selected, threshold, rule=ACCEPT_PREFIX):
    """Accepted draft tokens of the verified slots.

    token_prob [B, S, L] float32: probability of each draft token under the
               verification pass
    selected   [B, S] int: the verified slots; the first -1 ends the list and
               ids past S are skipped
    threshold  float32 token threshold (a token is accepted if p > threshold)

    Returns accepted [B, S, L] uint8 (1 = accepted), n_accepted [B, S] int32
    and n_total [B] int32.
    """
    tp = np.asarray(token_prob, dtype=np.float32)
    B, S, L = tp.shape
    thr = np.float32(threshold)
    sel = np.asarray(selected).reshape(B, S)
    accepted = np.zeros((B, S, L), dtype=np.uint8)
    for b in range(B):
        for i in range(S):
            s = int(sel[b, i])
            if s < 0:
                break  # the rest of the row is padding
            if s >= S:
                continue  # not a slot id
            above = tp[b, s] > thr
            if rule == ACCEPT_PREFIX:
                r = 0
                while r < L and above[r]:
                    r += 1
                accepted[b, s, :r] = 1
            else:
                accepted[b, s] = above.astype(np.uint8)
    n_accepted = accepted.sum(axis=2, dtype=np.int64).astype(np.int32)
    return accepted, n_accepted, n_accepted.sum(axis=1, dtype=np.int64).astype(np.int32)


def kv_append(k_cache, v_cache, prefix_lens, k_slot, v_slot, accepted, order):
    """Append the accepted draft tokens' keys and values after each prefix.

    k_cache, v_cache [B, Hkv, C, D]   cache (not modified; copies are returned)
    prefix_lens      [B]              valid prefix length of each batch row
    k_slot, v_slot   [B, Hkv, T, D]   the draft tokens' own K/V, T = S*L
    accepted         [B, S, L]        1 = accepted
    order            [B, S]           slots in append order; the first -1 ends it,
                                      ids past S are skipped, and a slot listed
                                      again is skipped (its tokens are committed once)

    A batch row whose appended length would exceed the capacity C is left
    unchanged.  Returns (k_cache', v_cache', prefix_lens').
    """
    kc = np.array(k_cache, copy=True)
    vc = np.array(v_cache, copy=True)
    B, Hkv, C, D = kc.shape
    acc = np.asarray(accepted).astype(bool)
    _, S, L = acc.shape
    plens = np.array(prefix_lens, dtype=np.int64).reshape(B)
    out_lens = plens.copy()
    ordr = np.asarray(order).reshape(B, S)
    for b in range(B):
        tokens = []
        listed = set()
        for i in range(S):
            s = int(ordr[b, i])
            if s < 0:
                break
            if s >= S or s in listed:
                continue  # not a slot id, or a slot already appended
            listed.add(s)
            tokens += [s * L + r for r in range(L) if acc[b, s, r]]
        p0 = int(plens[b])
        if p0 < 0 or p0 + len(tokens) > C:
            continue
        for i, t in enumerate(tokens):
            kc[b, :, p0 + i] = k_slot[b, :, t]
            vc[b, :, p0 + i] = v_slot[b, :, t]
        out_lens[b] = p0 + len(tokens)
    return kc, vc, out_lens.astype(np.int32)
