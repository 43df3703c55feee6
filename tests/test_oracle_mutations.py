"""Plant plausible mistakes in copies of the oracle (CPU only) and show the pins catch each.

A pin set that a dropped term, a wrong sign or index, or a transposed operand
survives would not pin anything; every mutant below must fail at least one
check of the set that covers its function.
"""

import numpy as np
import pytest

import oracle
import oracle.attention as oatt
import oracle_pins as pins


_ORIG_VIS = oatt.visibility


def _with_visibility(bad_visibility):
    """An attention oracle whose mask comes from ``bad_visibility``."""

    def attn(*args, **kw):
        saved = oatt.visibility
        oatt.visibility = bad_visibility
        try:
            return oracle.slot_attention(*args, **kw)
        finally:
            oatt.visibility = saved

    return attn


def _vis_flipped_causal(P, S, L, pass_, cross_slot=0, slot_pass=None):
    m = _ORIG_VIS(P, S, L, pass_, cross_slot, slot_pass)
    for s in range(S):
        rows = slice(s * L, (s + 1) * L)
        own = slice(P + s * L, P + (s + 1) * L)
        sp = pass_ if slot_pass is None else slot_pass[s]
        if sp == oracle.PASS_AR_INFILL:
            m[rows, own] = np.triu(np.ones((L, L), bool))  # looks forward instead of back
    return m


def _vis_diffusion_as_causal(P, S, L, pass_, cross_slot=0, slot_pass=None):
    return _ORIG_VIS(P, S, L, oracle.PASS_AR_INFILL, cross_slot, None)


def _vis_no_prefix(P, S, L, pass_, cross_slot=0, slot_pass=None):
    m = _ORIG_VIS(P, S, L, pass_, cross_slot, slot_pass)
    m[:, :P] = False
    return m


def _vis_slots_leak(P, S, L, pass_, cross_slot=0, slot_pass=None):
    m = _ORIG_VIS(P, S, L, pass_, cross_slot, slot_pass)
    m[:, P:] = True  # every slot sees every other slot
    return m


def _vis_boundary_off_by_one(P, S, L, pass_, cross_slot=0, slot_pass=None):
    m = _ORIG_VIS(P, S, L, pass_, cross_slot, slot_pass)
    return np.roll(m, 1, axis=1) | np.eye(S * L, P + S * L, k=P, dtype=bool)


def _vis_excludes_diagonal(P, S, L, pass_, cross_slot=0, slot_pass=None):
    m = _ORIG_VIS(P, S, L, pass_, cross_slot, slot_pass)
    if P > 0:
        idx = np.arange(S * L)
        m[idx, P + idx] = False
    return m


def _attn_no_scale(q, kc, vc, ks, vs, P, S, L, scale, pass_, **kw):
    return oracle.slot_attention(q, kc, vc, ks, vs, P, S, L, 1.0, pass_, **kw)


def _attn_gqa_modulo(q, kc, vc, ks, vs, P, S, L, scale, pass_, **kw):
    # query head h reads KV head h % Hkv instead of h // G
    Hq, Hkv = q.shape[1], ks.shape[1]
    perm = sorted(range(Hq), key=lambda h: (h % Hkv, h))
    O, lse = oracle.slot_attention(q[:, perm], kc, vc, ks, vs, P, S, L, scale, pass_, **kw)
    Om, lsem = np.empty_like(O), np.empty_like(lse)
    Om[:, perm], lsem[:, perm] = O, lse
    return Om, lsem


def _attn_lse_without_max(q, kc, vc, ks, vs, P, S, L, scale, pass_, **kw):
    O, lse = oracle.slot_attention(q, kc, vc, ks, vs, P, S, L, scale, pass_, **kw)
    s = scale * np.einsum("bhtd,bhtd->bht", q, np.repeat(ks, q.shape[1] // ks.shape[1], axis=1))
    return O, lse - np.maximum(s, 0)  # forgot part of the max shift


def _attn_values_from_keys(q, kc, vc, ks, vs, P, S, L, scale, pass_, **kw):
    return oracle.slot_attention(q, kc, kc, ks, ks, P, S, L, scale, pass_, **kw)


ATTENTION_MUTANTS = {
    "no softmax scale": _attn_no_scale,
    "AR_INFILL looks forward": _with_visibility(_vis_flipped_causal),
    "DIFFUSION treated as causal": _with_visibility(_vis_diffusion_as_causal),
    "prefix dropped": _with_visibility(_vis_no_prefix),
    "slots see each other": _with_visibility(_vis_slots_leak),
    "slot boundary off by one": _with_visibility(_vis_boundary_off_by_one),
    "token does not see itself": _with_visibility(_vis_excludes_diagonal),
    "GQA head mapping h % Hkv": _attn_gqa_modulo,
    "LSE missing the max shift": _attn_lse_without_max,
    "values taken from keys": _attn_values_from_keys,
}


def _conf_wrong_tie(h, w, target_ids=None, row_chunk=256):
    r = oracle.slot_confidence(h, w, target_ids, row_chunk)
    logits = np.asarray(h, np.float64) @ np.asarray(w, np.float64).T
    r["argmax"] = logits.shape[1] - 1 - np.argmax(logits[:, ::-1], axis=1)  # highest id on ties
    return r


def _conf_lse_missing_max(h, w, target_ids=None, row_chunk=256):
    r = oracle.slot_confidence(h, w, target_ids, row_chunk)
    r["lse"] = r["lse"] - r["max_logit"]
    return r


def _conf_shuffled_vocab(h, w, target_ids=None, row_chunk=256):
    w = np.asarray(w)
    perm = np.roll(np.arange(w.shape[0]), 1)
    return oracle.slot_confidence(h, w[perm], target_ids, row_chunk)


def _conf_target_is_argmax(h, w, target_ids=None, row_chunk=256):
    r = oracle.slot_confidence(h, w, target_ids, row_chunk)
    if target_ids is not None:
        r["target_prob"] = r["max_prob"].copy()
    return r


def _conf_prob_without_normaliser(h, w, target_ids=None, row_chunk=256):
    r = oracle.slot_confidence(h, w, target_ids, row_chunk)
    r["max_prob"] = 1.0 / (1.0 + np.exp(-r["max_logit"]))
    return r


def _conf_nonfinite_keeps_argmax(h, w, target_ids=None, row_chunk=256):
    r = oracle.slot_confidence(h, w, target_ids, row_chunk)
    with np.errstate(invalid="ignore", over="ignore"):
        logits = np.asarray(h, np.float64) @ np.asarray(w, np.float64).T
    bad = r["argmax"] < 0
    r["argmax"][bad] = np.argmax(logits[bad], axis=1)  # numpy's id of the first NaN
    return r


def _conf_nonfinite_rows_dropped_nan(h, w, target_ids=None, row_chunk=256):
    # NaN hidden values treated as zero
    return oracle.slot_confidence(np.nan_to_num(np.asarray(h, np.float64), nan=0.0, posinf=0.0), w, target_ids,
                                  row_chunk)


CONFIDENCE_MUTANTS = {
    "non-finite row keeps numpy's argmax": _conf_nonfinite_keeps_argmax,
    "non-finite hidden values read as zero": _conf_nonfinite_rows_dropped_nan,
    "argmax takes the highest id on ties": _conf_wrong_tie,
    "lse without the max": _conf_lse_missing_max,
    "vocab rows shifted by one": _conf_shuffled_vocab,
    "target prob is the max prob": _conf_target_is_argmax,
    "sigmoid instead of softmax": _conf_prob_without_normaliser,
}


def _sel_non_strict(tc, op=None, cr=0, rule=0, threshold=0.9, k=1):
    return oracle.select_slots(tc, op, cr, rule, np.nextafter(np.float32(threshold), np.float32(0)), k)


def _sel_fallback_highest_index(tc, op=None, cr=0, rule=0, threshold=0.9, k=1):
    c, sel, n = oracle.select_slots(tc, op, cr, rule, threshold, k)
    conf = oracle.slot_conf(tc, cr)
    for b in range(sel.shape[0]):
        if n[b] == 1 and not conf[b, sel[b, 0]] > np.float32(threshold) and rule == 0:
            is_open = np.ones(conf.shape[1], bool) if op is None else op[b] != 0
            cand = [s for s in range(conf.shape[1]) if is_open[s] and conf[b, s] == conf[b, sel[b, 0]]]
            sel[b, 0] = max(cand)
    return c, sel, n


def _sel_slot_order(tc, op=None, cr=0, rule=0, threshold=0.9, k=1):
    c, sel, n = oracle.select_slots(tc, op, cr, rule, threshold, k)
    for b in range(sel.shape[0]):
        sel[b, : n[b]] = np.sort(sel[b, : n[b]])
    return c, sel, n


def _sel_mean_is_first(tc, op=None, cr=0, rule=0, threshold=0.9, k=1):
    return oracle.select_slots(tc, op, oracle.CONF_FIRST_TOKEN, rule, threshold, k)


def _sel_ignores_open(tc, op=None, cr=0, rule=0, threshold=0.9, k=1):
    return oracle.select_slots(tc, None, cr, rule, threshold, k)


def _sel_no_fallback(tc, op=None, cr=0, rule=0, threshold=0.9, k=1):
    c, sel, n = oracle.select_slots(tc, op, cr, rule, threshold, k)
    conf = oracle.slot_conf(tc, cr)
    for b in range(sel.shape[0]):
        if rule == 0 and n[b] == 1 and not conf[b, sel[b, 0]] > np.float32(threshold):
            sel[b, 0], n[b] = -1, 0
    return c, sel, n


def _attn_ragged_uses_max(q, kc, vc, ks, vs, P, S, L, scale, pass_, **kw):
    # every row uses the longest prefix of the batch
    return oracle.slot_attention(q, kc, vc, ks, vs, int(np.max(P)), S, L, scale, pass_, **kw)


def _attn_ragged_first_row(q, kc, vc, ks, vs, P, S, L, scale, pass_, **kw):
    # every row uses the first row's prefix length
    return oracle.slot_attention(q, kc, vc, ks, vs, int(np.ravel(P)[0]), S, L, scale, pass_, **kw)


ATTENTION_MUTANTS["ragged prefix: longest for every row"] = _attn_ragged_uses_max
ATTENTION_MUTANTS["ragged prefix: first row's for every row"] = _attn_ragged_first_row


def _sel_nan_first(tc, op=None, cr=0, rule=0, threshold=0.9, k=1):
    tc = np.array(tc, dtype=np.float32)
    # NaN read as +inf: NaN slots rank first and pass the threshold
    if cr == oracle.CONF_FIRST_TOKEN:
        tc[..., 0] = np.where(np.isnan(tc[..., 0]), np.float32(np.inf), tc[..., 0])
    else:
        tc = np.where(np.isnan(tc).any(axis=2, keepdims=True), np.float32(np.inf), tc)
    return oracle.select_slots(tc, op, cr, rule, threshold, k)


def _sel_nan_reported(tc, op=None, cr=0, rule=0, threshold=0.9, k=1):
    c, sel, n = oracle.select_slots(tc, op, cr, rule, threshold, k)
    conf = oracle.slot_conf(tc, cr)
    c = np.where(np.isnan(conf) & (c != -1.0), conf, c)  # reports the NaN itself
    return c, sel, n


SELECTION_MUTANTS = {
    "NaN confidence ranks first": _sel_nan_first,
    "NaN confidence reported as NaN": _sel_nan_reported,
    "threshold compared with >=": _sel_non_strict,
    "fallback takes the highest index on ties": _sel_fallback_highest_index,
    "output in slot order": _sel_slot_order,
    "mean rule uses the first token": _sel_mean_is_first,
    "closed slots ignored": _sel_ignores_open,
    "no fallback": _sel_no_fallback,
}


def _caught(fn, checks):
    failed = []
    for check in checks:
        try:
            check(fn)
        except (AssertionError, ValueError, IndexError) as e:  # noqa: PERF203
            failed.append((check.__name__, str(e)[:80]))
    return failed


@pytest.mark.parametrize("name", list(ATTENTION_MUTANTS))
def test_attention_mutant_is_caught(name):
    assert _caught(ATTENTION_MUTANTS[name], pins.ATTENTION_CHECKS), f"mutant '{name}' passed every pin"


@pytest.mark.parametrize("name", list(CONFIDENCE_MUTANTS))
def test_confidence_mutant_is_caught(name):
    assert _caught(CONFIDENCE_MUTANTS[name], pins.CONFIDENCE_CHECKS), f"mutant '{name}' passed every pin"


@pytest.mark.parametrize("name", list(SELECTION_MUTANTS))
def test_selection_mutant_is_caught(name):
    assert _caught(SELECTION_MUTANTS[name], pins.SELECTION_CHECKS), f"mutant '{name}' passed every pin"


def _acc_non_strict(tp, sel, thr, rule=0):
    return oracle.accept_tokens(tp, sel, np.nextafter(np.float32(thr), np.float32(-1)), rule)


def _acc_prefix_is_per_token(tp, sel, thr, rule=0):
    return oracle.accept_tokens(tp, sel, thr, oracle.ACCEPT_PER_TOKEN)


def _acc_ignores_selection(tp, sel, thr, rule=0):
    S = np.shape(tp)[1]
    return oracle.accept_tokens(tp, np.tile(np.arange(S), (np.shape(tp)[0], 1)), thr, rule)


def _acc_padding_skipped(tp, sel, thr, rule=0):
    # a -1 entry is skipped instead of ending the list
    sel = np.asarray(sel).copy()
    for b in range(sel.shape[0]):
        keep = [s for s in sel[b] if s >= 0]
        sel[b] = keep + [-1] * (sel.shape[1] - len(keep))
    return oracle.accept_tokens(tp, sel, thr, rule)


def _acc_run_off_by_one(tp, sel, thr, rule=0):
    acc, n, t = oracle.accept_tokens(tp, sel, thr, rule)
    if rule == oracle.ACCEPT_PREFIX:
        for b, s in zip(*np.nonzero(n)):
            acc[b, s, n[b, s] - 1] = 0  # drops the last token of the run
        n = acc.sum(axis=2).astype(np.int32)
        t = n.sum(axis=1).astype(np.int32)
    return acc, n, t


ACCEPT_MUTANTS = {
    "threshold compared with >=": _acc_non_strict,
    "prefix rule accepts per token": _acc_prefix_is_per_token,
    "unselected slots verified": _acc_ignores_selection,
    "padding skipped instead of ending the list": _acc_padding_skipped,
    "accepted run one short": _acc_run_off_by_one,
}


def _app_slot_order_ignored(kc, vc, pl, ks, vs, acc, order):
    order = np.sort(np.where(np.asarray(order) < 0, 1 << 30, order), axis=1)
    order = np.where(order == 1 << 30, -1, order)
    return oracle.kv_append(kc, vc, pl, ks, vs, acc, order)


def _app_off_by_one(kc, vc, pl, ks, vs, acc, order):
    return oracle.kv_append(kc, vc, np.asarray(pl) + 1, ks, vs, acc, order)


def _app_whole_slots(kc, vc, pl, ks, vs, acc, order):
    acc = np.asarray(acc).copy()
    acc[acc.any(axis=2)] = 1  # a partly accepted slot is appended whole
    return oracle.kv_append(kc, vc, pl, ks, vs, acc, order)


def _app_keys_for_values(kc, vc, pl, ks, vs, acc, order):
    return oracle.kv_append(kc, vc, pl, ks, ks, acc, order)


def _app_repeats_appended(kc, vc, pl, ks, vs, acc, order):
    # a slot listed twice is appended twice: repeats become distinct copies of the slot
    order = np.asarray(order)
    B, S = order.shape
    L = np.asarray(acc).shape[2]
    acc2 = np.zeros((B, 2 * S, L), dtype=np.uint8)
    ks2 = np.concatenate([ks, ks], axis=2)
    vs2 = np.concatenate([vs, vs], axis=2)
    order2 = np.full((B, 2 * S), -1, dtype=np.int64)
    for b in range(B):
        seen = set()
        for i, s in enumerate(order[b]):
            if s < 0:
                break
            if s >= S:
                order2[b, i] = 2 * S
                continue
            s2 = int(s) + (S if s in seen else 0)
            seen.add(int(s))
            order2[b, i] = s2
            acc2[b, s2] = np.asarray(acc)[b, s]
    # slot s2 of the widened layout holds tokens s2*L.., so ks2 must hold slot s at s and s+S
    return oracle.kv_append(kc, vc, pl, ks2, vs2, acc2, order2)


APPEND_MUTANTS = {
    "a repeated slot appended twice": _app_repeats_appended,
    "slots appended in slot order": _app_slot_order_ignored,
    "appended one position late": _app_off_by_one,
    "partly accepted slots appended whole": _app_whole_slots,
    "keys written as values": _app_keys_for_values,
}


@pytest.mark.parametrize("name", list(ACCEPT_MUTANTS))
def test_accept_mutant_is_caught(name):
    assert _caught(ACCEPT_MUTANTS[name], pins.ACCEPT_CHECKS), f"mutant '{name}' passed every pin"


@pytest.mark.parametrize("name", list(APPEND_MUTANTS))
def test_append_mutant_is_caught(name):
    assert _caught(APPEND_MUTANTS[name], pins.APPEND_CHECKS), f"mutant '{name}' passed every pin"


import oracle.sampling as osm  # noqa: E402

_ORIG_PHILOX = osm.philox4x32
_ORIG_UNIF = osm.uniforms
_ORIG_GUMBEL = osm.gumbel


def _philox_rounds9(c, k, rounds=10):
    return _ORIG_PHILOX(c, k, rounds=9)


def _philox_swapped_multipliers(c, k, rounds=10):
    saved = osm.PHILOX_M0, osm.PHILOX_M1
    osm.PHILOX_M0, osm.PHILOX_M1 = saved[1], saved[0]
    try:
        return _ORIG_PHILOX(c, k, rounds)
    finally:
        osm.PHILOX_M0, osm.PHILOX_M1 = saved


def _philox_no_key_schedule(c, k, rounds=10):
    saved = osm.PHILOX_W0, osm.PHILOX_W1
    osm.PHILOX_W0, osm.PHILOX_W1 = 0, 0
    try:
        return _ORIG_PHILOX(c, k, rounds)
    finally:
        osm.PHILOX_W0, osm.PHILOX_W1 = saved


PHILOX_MUTANTS = {
    "nine rounds": _philox_rounds9,
    "multipliers swapped": _philox_swapped_multipliers,
    "key never bumped": _philox_no_key_schedule,
}


def _unif_block_word0(rows, vocab, seed, offset):
    u = _ORIG_UNIF(rows, ((vocab + 3) // 4) * 4, seed, offset)
    return np.repeat(u[:, ::4], 4, axis=1)[:, :vocab]  # one word for the four ids of a block


def _unif_row_ignored(rows, vocab, seed, offset):
    return np.repeat(_ORIG_UNIF([0], vocab, seed, offset), len(np.ravel(rows)), axis=0)


def _unif_low_bits(rows, vocab, seed, offset):
    u = _ORIG_UNIF(rows, vocab, seed, offset)
    return np.mod(u * 256.0, 1.0) * 0.5  # a biased, squeezed uniform


UNIFORM_MUTANTS = {
    "one word for a whole block": _unif_block_word0,
    "row not in the counter": _unif_row_ignored,
    "biased uniforms": _unif_low_bits,
}


def _with_sampling(unif=None, gum=None):
    def sample(*a, **kw):
        saved = osm.uniforms, osm.gumbel
        if unif is not None:
            osm.uniforms = unif
        if gum is not None:
            osm.gumbel = gum
        try:
            return osm.slot_sample(*a, **kw)
        finally:
            osm.uniforms, osm.gumbel = saved
    return sample


def _sample_temperature_multiplied(h, w, T, seed, offset, row_chunk=256):
    return osm.slot_sample(h, w, 1.0 / T, seed, offset, row_chunk)


def _sample_prob_of_argmax(h, w, T, seed, offset, row_chunk=256):
    r = osm.slot_sample(h, w, T, seed, offset, row_chunk)
    z = np.asarray(h, np.float64) @ np.asarray(w, np.float64).T
    r["sample_prob"] = np.exp(z.max(axis=1) - r["lse"])
    return r


def _sample_nonfinite_drawn(h, w, T, seed, offset, row_chunk=256):
    # a row without a distribution still reports the id of its best score
    r = osm.slot_sample(h, w, T, seed, offset, row_chunk)
    with np.errstate(invalid="ignore", over="ignore"):
        z = np.asarray(h, np.float64) @ np.asarray(w, np.float64).T
        u = osm.uniforms(np.arange(z.shape[0]), z.shape[1], seed, offset)
        score = z / T + osm.gumbel(u)
    bad = r["sample_id"] < 0
    r["sample_id"][bad] = np.argmax(score[bad], axis=1)
    return r


SAMPLING_MUTANTS = {
    "row without a distribution still sampled": _sample_nonfinite_drawn,
    "noise sign flipped": _with_sampling(gum=lambda u: np.log(-np.log(u))),
    "exponential instead of Gumbel noise": _with_sampling(gum=lambda u: -np.log(u)),
    "one word for a whole block": _with_sampling(unif=_unif_block_word0),
    "row not in the counter": _with_sampling(unif=_unif_row_ignored),
    "temperature multiplies": _sample_temperature_multiplied,
    "probability of the argmax reported": _sample_prob_of_argmax,
}


@pytest.mark.parametrize("name", list(PHILOX_MUTANTS))
def test_philox_mutant_is_caught(name):
    assert _caught(PHILOX_MUTANTS[name], pins.PHILOX_CHECKS), f"mutant '{name}' passed every pin"


@pytest.mark.parametrize("name", list(UNIFORM_MUTANTS))
def test_uniform_mutant_is_caught(name):
    assert _caught(UNIFORM_MUTANTS[name], pins.UNIFORM_CHECKS), f"mutant '{name}' passed every pin"


@pytest.mark.parametrize("name", list(SAMPLING_MUTANTS))
def test_sampling_mutant_is_caught(name):
    assert _caught(SAMPLING_MUTANTS[name], pins.SAMPLING_CHECKS), f"mutant '{name}' passed every pin"


import oracle.mdm as omd  # noqa: E402


def _budget_t0_rounds_down(N, T, a, seed):
    if T == 0 and N > 0:
        t = max(1, N // 4)
        base, extra = divmod(N, t)
        return np.array([base + (1 if i < extra else 0) for i in range(t)]), t
    return omd.mask_budget(N, T, a, seed)


def _budget_drops_sequential(N, T, a, seed):
    counts, t = omd.mask_budget(N, T, a, seed)
    return counts[:t], t


def _budget_complement(N, T, a, seed):
    return omd.mask_budget(N, T, 1.0 - a if T > 0 else a, seed)


def _budget_extra_last(N, T, a, seed):
    counts, t = omd.mask_budget(N, T, a, seed)
    return np.concatenate([counts[:t][::-1], counts[t:]]), t


def _budget_t0_binomial(N, T, a, seed):
    if T == 0 and N > 0:
        return omd.mask_budget(N, -(-N // 4), a, seed)
    return omd.mask_budget(N, T, a, seed)


BUDGET_MUTANTS = {
    "T = 0 rounds the step count down": _budget_t0_rounds_down,
    "sequential tokens dropped": _budget_drops_sequential,
    "binomial with 1 - alpha_0": _budget_complement,
    "extra tokens to the last steps": _budget_extra_last,
    "T = 0 still draws the binomial": _budget_t0_binomial,
}


def _rev_ties_high(conf, op, k, rule=0, seed=0, offset=0, tokens=None, sample_id=None):
    if rule != omd.REVEAL_CONFIDENCE:
        return omd.reveal(conf, op, k, rule, seed, offset, tokens, sample_id)
    c = np.asarray(conf, np.float32)
    N = c.shape[1]
    # reverse the positions, so equal confidences favour the higher index
    o, n, op2, tok = omd.reveal(c[:, ::-1], np.asarray(op)[:, ::-1], k, rule, seed, offset)
    o = np.where(o >= 0, N - 1 - o, -1).astype(np.int32)
    tok2 = None
    if tokens is not None:
        tok2 = np.array(tokens, copy=True)
        for b in range(c.shape[0]):
            for i in o[b, : n[b]]:
                tok2[b, i] = sample_id[b][i]
    return o, n, op2[:, ::-1], tok2


def _rev_lowest_first(conf, op, k, rule=0, seed=0, offset=0, tokens=None, sample_id=None):
    c = np.asarray(conf, np.float32)
    return omd.reveal(-c if rule == omd.REVEAL_CONFIDENCE else c, op, k, rule, seed, offset, tokens, sample_id)


def _rev_ignores_open(conf, op, k, rule=0, seed=0, offset=0, tokens=None, sample_id=None):
    o, n, _, tok = omd.reveal(conf, np.ones_like(np.asarray(op, bool)), k, rule, seed, offset, tokens, sample_id)
    op2 = np.asarray(op, bool).copy()
    for b in range(op2.shape[0]):
        op2[b, o[b, : n[b]]] = False
    return o, n, op2, tok


def _rev_rightmost(conf, op, k, rule=0, seed=0, offset=0, tokens=None, sample_id=None):
    if rule != omd.REVEAL_LEFTMOST:
        return omd.reveal(conf, op, k, rule, seed, offset, tokens, sample_id)
    N = np.asarray(op).shape[1]
    return omd.reveal(np.tile(np.arange(N, dtype=np.float32), (np.asarray(op).shape[0], 1)), op, k,
                      omd.REVEAL_CONFIDENCE, seed, offset, tokens, sample_id)


def _rev_random_row_ignored(conf, op, k, rule=0, seed=0, offset=0, tokens=None, sample_id=None):
    if rule != omd.REVEAL_RANDOM:
        return omd.reveal(conf, op, k, rule, seed, offset, tokens, sample_id)
    saved = omd.uniforms
    omd.uniforms = lambda rows, vocab, s, o: saved([0] * len(np.ravel(rows)), vocab, s, o)
    try:
        return omd.reveal(conf, op, k, rule, seed, offset, tokens, sample_id)
    finally:
        omd.uniforms = saved


def _rev_random_offset_ignored(conf, op, k, rule=0, seed=0, offset=0, tokens=None, sample_id=None):
    return omd.reveal(conf, op, k, rule, seed, 0, tokens, sample_id)


REVEAL_MUTANTS = {
    "confidence ties to the higher index": _rev_ties_high,
    "lowest confidence first": _rev_lowest_first,
    "open mask ignored": _rev_ignores_open,
    "sequential phase from the right": _rev_rightmost,
    "random choice not keyed by row": _rev_random_row_ignored,
    "random choice ignores the step offset": _rev_random_offset_ignored,
}


@pytest.mark.parametrize("name", list(BUDGET_MUTANTS))
def test_budget_mutant_is_caught(name):
    assert _caught(BUDGET_MUTANTS[name], pins.BUDGET_CHECKS), f"mutant '{name}' passed every pin"


@pytest.mark.parametrize("name", list(REVEAL_MUTANTS))
def test_reveal_mutant_is_caught(name):
    assert _caught(REVEAL_MUTANTS[name], pins.REVEAL_CHECKS), f"mutant '{name}' passed every pin"
