"""Oracle: slot confidence and first-hitting slot selection.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Paper passages this follows:

* Sec. 5.2 "Draft phase": the confidence of a slot is the probability of its
  first token (rule ``FIRST_TOKEN``).  The mean over the slot's tokens (rule
  ``MEAN``) is the alternative the 1.7B-scale workload asks for.
* Sec. 5.2 "Slot selection": slots whose confidence exceeds
  ``slot_threshold`` are accepted; if none does, the single most confident slot
  is taken, so at least one slot always goes on (rule ``THRESHOLD``).
  Sec. 6 evaluates with ``slot_threshold = 0.9``.
* Top-k selection (rule ``TOP_K``) takes the k most confident open slots.

Readings where the paper is silent: "exceeding" is a strict comparison; the
fallback takes the lowest slot index among equally confident slots; the
output lists the chosen slots in first-hitting order, i.e. by descending
confidence with ties going to the lower slot index.  A NaN slot confidence
(for instance from a NaN token probability) counts as -inf: it ranks after
every other open slot, never exceeds the threshold, and is reported as -inf.

Precision: the selection is an integer decision taken from floating point, so
this oracle takes it in the precision of the kernel it checks: slot
confidences are float32, a mean is summed in float64 in increasing token order,
divided by L in float64 and rounded once to float32, and every comparison is
made between float32 values.
"""

from __future__ import annotations

import numpy as np

CONF_FIRST_TOKEN = 0
CONF_MEAN = 1
SELECT_THRESHOLD = 0
SELECT_TOP_K = 1


def slot_conf(token_conf, conf_rule):
    """Slot confidence [B, S] float32 from token confidences [B, S, L]."""
    tc = np.asarray(token_conf, dtype=np.float32)
    if conf_rule == CONF_FIRST_TOKEN:
        return tc[:, :, 0].copy()
    if conf_rule == CONF_MEAN:
        L = tc.shape[2]
        acc = np.zeros(tc.shape[:2], dtype=np.float64)
        for r in range(L):  # sequential order, as the definition above fixes
            acc = acc + tc[:, :, r].astype(np.float64)
        return (acc / np.float64(L)).astype(np.float32)
    raise ValueError(f"unknown confidence rule {conf_rule}")


def select_slots(token_conf, slot_open=None, conf_rule=CONF_FIRST_TOKEN, rule=SELECT_THRESHOLD,
                 threshold=0.9, k=1):
    """First-hitting slot selection.

    token_conf [B, S, L] float32 (per-token max probability), slot_open [B, S]
    (nonzero = slot still undecided; None = all open).
    Returns (slot_conf [B, S] float32 with -1 for closed slots,
    selected [B, S] int32 in first-hitting order padded with -1,
    n_selected [B] int32).
    """
    conf = slot_conf(token_conf, conf_rule)
    conf = np.where(np.isnan(conf), np.float32(-np.inf), conf).astype(np.float32)  # NaN ranks as -inf
    B, S = conf.shape
    is_open = np.ones((B, S), dtype=bool) if slot_open is None else (np.asarray(slot_open) != 0)
    tau = np.float32(threshold)
    out_conf = np.where(is_open, conf, np.float32(-1.0)).astype(np.float32)
    selected = np.full((B, S), -1, dtype=np.int32)
    n_sel = np.zeros(B, dtype=np.int32)
    for b in range(B):
        open_ids = [s for s in range(S) if is_open[b, s]]
        # first-hitting order: descending confidence, then ascending slot index
        ranked = sorted(open_ids, key=lambda s: (-float(conf[b, s]), s))
        if rule == SELECT_THRESHOLD:
            picks = [s for s in ranked if conf[b, s] > tau]
            if not picks and ranked:
                picks = ranked[:1]  # most confident open slot, lowest index on ties
        elif rule == SELECT_TOP_K:
            picks = ranked[: max(0, int(k))]
        else:
            raise ValueError(f"unknown selection rule {rule}")
        n_sel[b] = len(picks)
        selected[b, : len(picks)] = picks
    return out_conf, selected, n_sel
