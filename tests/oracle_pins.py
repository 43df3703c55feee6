"""Pins of the oracle to facts outside itself.

Each ``check_*`` function takes the function under test (the oracle, or a
deliberately broken copy of it in the mutation tests) and raises
AssertionError when the pin does not hold.  The pins are textbook special
cases computed by library routines (torch's scaled_dot_product_attention on
the CPU in float64, scipy's logsumexp/softmax, numpy's argmax), closed forms,
invariants, brute force on tiny inputs, and the paper's selection rule.
"""

from __future__ import annotations

import json
import os

import numpy as np
import scipy.special
import torch
import torch.nn.functional as F

import oracle
from oracle import (
    CROSS_SLOT_CAUSAL,
    CROSS_SLOT_NONE,
    PASS_AR_INFILL,
    PASS_DIFFUSION,
)

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
TOL = 1e-11


def _inputs(seed, B, Hq, Hkv, D, P, S, L, C=None):
    rng = np.random.default_rng(seed)
    C = P if C is None else C
    T = S * L
    return dict(
        q=rng.standard_normal((B, Hq, T, D)),
        k_cache=rng.standard_normal((B, Hkv, C, D)),
        v_cache=rng.standard_normal((B, Hkv, C, D)),
        k_slot=rng.standard_normal((B, Hkv, T, D)),
        v_slot=rng.standard_normal((B, Hkv, T, D)),
    )


def _sdpa(q, k, v, scale, is_causal=False):
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64))
    gqa = q.shape[1] != k.shape[1]
    return F.scaled_dot_product_attention(t(q), t(k), t(v), scale=scale, is_causal=is_causal, enable_gqa=gqa).numpy()


def _close(a, b, tol=TOL, what=""):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    assert a.shape == b.shape, f"{what}: shape {a.shape} vs {b.shape}"
    err = np.max(np.abs(a - b)) if a.size else 0.0
    assert err <= tol, f"{what}: max |diff| {err:.3e} > {tol:.1e}"


def _call(attn, x, P, S, L, scale, pass_, cross=CROSS_SLOT_NONE, slot_pass=None):
    return attn(x["q"], x["k_cache"], x["v_cache"], x["k_slot"], x["v_slot"], P, S, L, scale, pass_,
                cross_slot=cross, slot_pass=slot_pass)


# ---------------------------------------------------------------- attention


def check_decode_l1(attn):
    """L = 1: both passes equal ordinary decode of each token over prefix + itself."""
    B, Hq, Hkv, D, P, S, L = 2, 4, 2, 8, 7, 5, 1
    x = _inputs(11, B, Hq, Hkv, D, P, S, L)
    scale = 0.37
    outs = []
    for pass_ in (PASS_DIFFUSION, PASS_AR_INFILL):
        O, lse = _call(attn, x, P, S, L, scale, pass_)
        for s in range(S):
            k = np.concatenate([x["k_cache"][:, :, :P], x["k_slot"][:, :, s : s + 1]], axis=2)
            v = np.concatenate([x["v_cache"][:, :, :P], x["v_slot"][:, :, s : s + 1]], axis=2)
            ref = _sdpa(x["q"][:, :, s : s + 1], k, v, scale)
            _close(O[:, :, s : s + 1], ref, what=f"decode O pass={pass_} slot={s}")
            kk = np.repeat(k, Hq // Hkv, axis=1)
            scores = scale * np.einsum("bhd,bhjd->bhj", x["q"][:, :, s], kk)
            _close(lse[:, :, s], scipy.special.logsumexp(scores, axis=-1), what="decode LSE")
        outs.append((O, lse))
    _close(outs[0][0], outs[1][0], what="L=1 passes agree")


def check_prefill_s1(attn):
    """S = 1, AR_INFILL: a chunked causal prefill of L tokens after P cached ones.

    The cache has slack rows beyond P that must be ignored.
    """
    B, Hq, Hkv, D, P, S, L = 2, 6, 3, 8, 5, 1, 6
    x = _inputs(12, B, Hq, Hkv, D, P, S, L, C=P + 3)
    scale = 0.41
    O, _ = _call(attn, x, P, S, L, scale, PASS_AR_INFILL)
    rng = np.random.default_rng(5)
    q_full = np.concatenate([rng.standard_normal((B, Hq, P, D)), x["q"]], axis=2)
    k_full = np.concatenate([x["k_cache"][:, :, :P], x["k_slot"]], axis=2)
    v_full = np.concatenate([x["v_cache"][:, :, :P], x["v_slot"]], axis=2)
    ref = _sdpa(q_full, k_full, v_full, scale, is_causal=True)[:, :, P:]
    _close(O, ref, what="S=1 causal prefill")


def check_blockdiag_p0(attn):
    """P = 0, DIFFUSION: every slot is an independent full (unmasked) attention."""
    B, Hq, Hkv, D, P, S, L = 2, 2, 1, 8, 0, 3, 4
    x = _inputs(13, B, Hq, Hkv, D, P, S, L)
    scale = 0.5
    O, _ = _call(attn, x, P, S, L, scale, PASS_DIFFUSION)
    for s in range(S):
        sl = slice(s * L, (s + 1) * L)
        ref = _sdpa(x["q"][:, :, sl], x["k_slot"][:, :, sl], x["v_slot"][:, :, sl], scale)
        _close(O[:, :, sl], ref, what=f"block-diagonal slot {s}")


def check_cross_causal(attn):
    """cross_slot = CAUSAL with every slot AR_INFILL is causal attention in physical order."""
    for P in (0, 3):
        B, Hq, Hkv, D, S, L = 1, 4, 2, 8, 4, 3
        x = _inputs(14 + P, B, Hq, Hkv, D, P, S, L)
        scale = 0.3
        O, _ = _call(attn, x, P, S, L, scale, PASS_AR_INFILL, cross=CROSS_SLOT_CAUSAL)
        rng = np.random.default_rng(6)
        q_full = np.concatenate([rng.standard_normal((B, Hq, P, D)), x["q"]], axis=2)
        k_full = np.concatenate([x["k_cache"][:, :, :P], x["k_slot"]], axis=2)
        v_full = np.concatenate([x["v_cache"][:, :, :P], x["v_slot"]], axis=2)
        ref = _sdpa(q_full, k_full, v_full, scale, is_causal=True)[:, :, P:]
        _close(O, ref, what=f"cross-slot causal P={P}")


def check_slot_permutation(attn):
    """Permuting whole draft slots (queries and their K/V) permutes the outputs."""
    B, Hq, Hkv, D, P, S, L = 2, 4, 2, 8, 6, 5, 3
    x = _inputs(15, B, Hq, Hkv, D, P, S, L)
    perm = np.array([3, 0, 4, 2, 1])
    rows = (perm[:, None] * L + np.arange(L)[None, :]).reshape(-1)
    xp = dict(x)
    for key in ("q", "k_slot", "v_slot"):
        xp[key] = x[key][:, :, rows]
    for pass_ in (PASS_DIFFUSION, PASS_AR_INFILL):
        O, lse = _call(attn, x, P, S, L, 0.35, pass_)
        Op, lsep = _call(attn, xp, P, S, L, 0.35, pass_)
        _close(Op, O[:, :, rows], what=f"slot permutation O pass={pass_}")
        _close(lsep, lse[:, :, rows], what=f"slot permutation LSE pass={pass_}")


def check_token_permutation_diffusion(attn):
    """DIFFUSION: permuting the tokens inside a slot permutes that slot's outputs."""
    B, Hq, Hkv, D, P, S, L = 1, 2, 1, 8, 4, 3, 5
    x = _inputs(16, B, Hq, Hkv, D, P, S, L)
    rng = np.random.default_rng(3)
    rows = np.concatenate([s * L + rng.permutation(L) for s in range(S)])
    xp = dict(x)
    for key in ("q", "k_slot", "v_slot"):
        xp[key] = x[key][:, :, rows]
    O, _ = _call(attn, x, P, S, L, 0.35, PASS_DIFFUSION)
    Op, _ = _call(attn, xp, P, S, L, 0.35, PASS_DIFFUSION)
    _close(Op, O[:, :, rows], what="in-slot token permutation")


def check_last_token_same(attn):
    """The last token of every slot sees the same keys in both passes."""
    B, Hq, Hkv, D, P, S, L = 2, 2, 2, 8, 5, 4, 4
    x = _inputs(17, B, Hq, Hkv, D, P, S, L)
    Od, ld = _call(attn, x, P, S, L, 0.3, PASS_DIFFUSION)
    Oa, la = _call(attn, x, P, S, L, 0.3, PASS_AR_INFILL)
    last = np.arange(S) * L + L - 1
    _close(Od[:, :, last], Oa[:, :, last], what="last token O")
    _close(ld[:, :, last], la[:, :, last], what="last token LSE")
    assert np.max(np.abs(Od[:, :, 0::L] - Oa[:, :, 0::L])) > 1e-3, "first tokens should differ between passes"


def check_constant_v(attn):
    """Constant values: the output equals that value (probabilities sum to 1)."""
    B, Hq, Hkv, D, P, S, L = 2, 4, 2, 8, 6, 3, 4
    x = _inputs(18, B, Hq, Hkv, D, P, S, L)
    rng = np.random.default_rng(9)
    c = rng.standard_normal((B, Hkv, 1, D))
    x["v_cache"] = np.broadcast_to(c, x["v_cache"].shape).copy()
    x["v_slot"] = np.broadcast_to(c, x["v_slot"].shape).copy()
    for pass_ in (PASS_DIFFUSION, PASS_AR_INFILL):
        O, _ = _call(attn, x, P, S, L, 0.8, pass_)
        ref = np.repeat(c, Hq // Hkv, axis=1)
        _close(O, np.broadcast_to(ref, O.shape), tol=1e-12, what=f"constant V pass={pass_}")


def n_visible(P, S, L, pass_, cross=CROSS_SLOT_NONE):
    """Number of keys a token (s, r) sees, counted from the paper's rule."""
    counts = np.empty(S * L, dtype=np.int64)
    for s in range(S):
        for r in range(L):
            own = L if pass_ == PASS_DIFFUSION else r + 1
            counts[s * L + r] = P + own + (s * L if cross == CROSS_SLOT_CAUSAL else 0)
    return counts


def check_identical_keys(attn):
    """All keys equal: O is the mean of the visible values, LSE = s0 + ln(#visible)."""
    B, Hq, Hkv, D, P, S, L = 1, 2, 1, 8, 5, 3, 4
    for pass_ in (PASS_DIFFUSION, PASS_AR_INFILL):
        for cross in (CROSS_SLOT_NONE, CROSS_SLOT_CAUSAL):
            x = _inputs(19, B, Hq, Hkv, D, P, S, L)
            k0 = x["k_slot"][:, :, :1]
            x["k_cache"] = np.broadcast_to(k0, x["k_cache"].shape).copy()
            x["k_slot"] = np.broadcast_to(k0, x["k_slot"].shape).copy()
            scale = 0.45
            O, lse = _call(attn, x, P, S, L, scale, pass_, cross=cross)
            cnt = n_visible(P, S, L, pass_, cross)
            vals = np.concatenate([x["v_cache"][0, 0, :P], x["v_slot"][0, 0]])
            for h in range(Hq):
                s0 = scale * (x["q"][0, h] @ k0[0, 0, 0])
                _close(lse[0, h], s0 + np.log(cnt), what=f"identical keys LSE pass={pass_} cross={cross}")
                for t in range(S * L):
                    s, r = divmod(t, L)
                    idx = list(range(P))
                    own = range(s * L, s * L + (L if pass_ == PASS_DIFFUSION else r + 1))
                    earlier = range(0, s * L) if cross == CROSS_SLOT_CAUSAL else range(0)
                    idx += [P + j for j in earlier] + [P + j for j in own]
                    _close(O[0, h, t], vals[idx].mean(axis=0), what="identical keys O")


def check_bruteforce(attn):
    """Agreement with the scalar-loop brute force on tiny random inputs."""
    cases = [
        (1, 2, 1, 4, 3, 2, 3, None, CROSS_SLOT_NONE),
        (2, 4, 2, 4, 0, 3, 2, None, CROSS_SLOT_NONE),
        (1, 3, 1, 4, 2, 3, 2, [[0, 1, 0]], CROSS_SLOT_NONE),
        (2, 2, 2, 4, 0, 4, 2, [[1, 0, 1, 0], [0, 0, 1, 1]], CROSS_SLOT_CAUSAL),
        (1, 2, 1, 4, 3, 2, 2, None, CROSS_SLOT_CAUSAL),
    ]
    for i, (B, Hq, Hkv, D, P, S, L, sp, cross) in enumerate(cases):
        x = _inputs(40 + i, B, Hq, Hkv, D, P, S, L, C=P + 1)
        for pass_ in (PASS_DIFFUSION, PASS_AR_INFILL):
            O, lse = _call(attn, x, P, S, L, 0.6, pass_, cross=cross, slot_pass=sp)
            Ob, lseb = oracle.slot_attention_loops(
                x["q"], x["k_cache"], x["v_cache"], x["k_slot"], x["v_slot"], P, S, L, 0.6, pass_,
                cross_slot=cross, slot_pass=sp)
            _close(O, Ob, tol=1e-12, what=f"brute force O case {i}")
            _close(lse, lseb, tol=1e-12, what=f"brute force LSE case {i}")


def check_ragged_rows(attn):
    """Per-row prefix lengths (Sec. 5.2 KV cache update): each batch row equals
    the same call made on that row alone with its own prefix length; cache rows
    past a row's length (random here) never matter."""
    B, Hq, Hkv, D, S, L, C = 3, 4, 2, 8, 2, 3, 9
    x = _inputs(60, B, Hq, Hkv, D, C, S, L, C=C)
    plens = [5, 0, 9]
    for pass_ in (PASS_DIFFUSION, PASS_AR_INFILL):
        O, lse = _call(attn, x, plens, S, L, 0.45, pass_)
        for b, P in enumerate(plens):
            xb = {k: v[b:b + 1] for k, v in x.items()}
            Ob, lseb = _call(attn, xb, P, S, L, 0.45, pass_)
            _close(O[b:b + 1], Ob, tol=1e-13, what=f"ragged row {b} O")
            _close(lse[b:b + 1], lseb, tol=1e-13, what=f"ragged row {b} LSE")
        # a row whose prefix is empty sees only draft tokens: the cache may be anything
        x2 = dict(x, k_cache=x["k_cache"].copy(), v_cache=x["v_cache"].copy())
        x2["k_cache"][1] = 1e3
        x2["v_cache"][1] = -7.0
        O2, _ = _call(attn, x2, plens, S, L, 0.45, pass_)
        _close(O2[1], O[1], tol=0.0, what="cache of an empty-prefix row")


def check_ragged_bruteforce(attn):
    """Per-row prefix lengths against the scalar-loop brute force."""
    x = _inputs(61, 2, 2, 1, 4, 4, 2, 2, C=4)
    for pass_ in (PASS_DIFFUSION, PASS_AR_INFILL):
        O, lse = _call(attn, x, [3, 1], 2, 2, 0.7, pass_)
        Ob, lseb = oracle.slot_attention_loops(x["q"], x["k_cache"], x["v_cache"], x["k_slot"], x["v_slot"],
                                               [3, 1], 2, 2, 0.7, pass_)
        _close(O, Ob, tol=1e-12, what="ragged brute force O")
        _close(lse, lseb, tol=1e-12, what="ragged brute force LSE")


ATTENTION_CHECKS = [
    check_ragged_rows,
    check_ragged_bruteforce,
    check_decode_l1,
    check_prefill_s1,
    check_blockdiag_p0,
    check_cross_causal,
    check_slot_permutation,
    check_token_permutation_diffusion,
    check_last_token_same,
    check_constant_v,
    check_identical_keys,
    check_bruteforce,
]


# --------------------------------------------------------------- confidence


def check_conf_library(conf):
    """Random rows against scipy's logsumexp/softmax and numpy's argmax."""
    rng = np.random.default_rng(21)
    for V in (512, 500):
        h = rng.standard_normal((9, 32))
        w = 0.3 * rng.standard_normal((V, 32))
        t = rng.integers(0, V, 9)
        r = conf(h, w, target_ids=t)
        logits = h @ w.T
        sm = scipy.special.softmax(logits, axis=1)
        _close(r["lse"], scipy.special.logsumexp(logits, axis=1), what="lse vs scipy")
        _close(r["max_prob"], sm.max(axis=1), what="max_prob vs softmax")
        _close(r["target_prob"], sm[np.arange(9), t], what="target_prob vs softmax")
        assert np.array_equal(r["argmax"], np.argmax(logits, axis=1)), "argmax vs numpy"


def check_conf_bruteforce(conf):
    """Agreement with scalar loops and exactly rounded sums (V = 512 and 500)."""
    rng = np.random.default_rng(22)
    for V in (512, 500):
        h = rng.standard_normal((4, 16))
        w = 0.5 * rng.standard_normal((V, 16))
        t = rng.integers(0, V, 4)
        r = conf(h, w, target_ids=t)
        b = oracle.slot_confidence_loops(h, w, target_ids=t)
        for key in ("max_prob", "lse", "target_prob"):
            _close(r[key], b[key], tol=1e-12, what=f"brute force {key}")
        assert np.array_equal(r["argmax"], b["argmax"])


def check_conf_zero_hidden(conf):
    """h = 0: every logit is 0, so lse = ln V, max_prob = 1/V, argmax = 0."""
    V = 777
    w = np.random.default_rng(23).standard_normal((V, 24))
    r = conf(np.zeros((3, 24)), w)
    _close(r["lse"], np.full(3, np.log(V)), what="zero h lse")
    _close(r["max_prob"], np.full(3, 1.0 / V), what="zero h max_prob")
    assert np.all(r["argmax"] == 0)


def check_conf_planted(conf):
    """h = a * W[v]/|W[v]| makes v the argmax; max_prob rises towards 1 with a."""
    rng = np.random.default_rng(24)
    V, H = 300, 64
    w = 0.02 * rng.standard_normal((V, H))
    v_star = 137
    u = w[v_star] / np.linalg.norm(w[v_star])
    alphas = np.array([5.0, 15.0, 25.0, 35.0, 60.0])
    r = conf(alphas[:, None] * u[None, :], w)
    assert np.all(r["argmax"] == v_star), r["argmax"]
    assert np.all(np.diff(r["max_prob"]) > 0), r["max_prob"]
    assert r["max_prob"][-1] > 0.95 and r["max_prob"][0] < 0.05


def check_conf_sums_to_one(conf):
    """Summing the target probability over every vocabulary id gives 1."""
    rng = np.random.default_rng(25)
    V, H = 257, 16
    w = rng.standard_normal((V, H))
    h = np.repeat(rng.standard_normal((1, H)), V, axis=0)
    r = conf(h, w, target_ids=np.arange(V))
    _close(r["target_prob"].sum(), 1.0, tol=1e-12, what="softmax sums to 1")
    _close(r["max_prob"][0], r["target_prob"].max(), what="max_prob is the largest probability")
    assert r["argmax"][0] == int(np.argmax(r["target_prob"]))


def check_conf_ties(conf):
    """Equal maximal logits: the lowest vocabulary id wins and the top-2 gap is 0."""
    rng = np.random.default_rng(26)
    V, H = 64, 8
    w = rng.standard_normal((V, H))
    h = rng.standard_normal((1, H))
    best = int(np.argmax(h @ w.T))
    w2 = w.copy()
    lo = max(0, best - 5)
    w2[lo] = w[best]
    r = conf(h, w2)
    assert r["argmax"][0] == min(lo, best)
    assert r["top2_gap"][0] == 0.0


def check_conf_nonfinite_rows(conf):
    """Rows with a NaN or infinite hidden value: IEEE arithmetic makes some of
    their logits NaN or infinite, scipy's logsumexp of such a row is not
    finite, and the row reports argmax -1 and NaN probabilities (the rule the
    header states).  Every other row keeps the values it has without them."""
    rng = np.random.default_rng(27)
    V, H, M = 300, 16, 6
    w = 0.3 * rng.standard_normal((V, H))
    h = rng.standard_normal((M, H))
    t = rng.integers(0, V, M)
    clean = conf(h, w, target_ids=t)
    h2 = h.copy()
    h2[1, 3] = np.nan
    h2[4, 0] = np.inf
    with np.errstate(invalid="ignore", over="ignore"):
        lse_scipy = scipy.special.logsumexp(h2 @ w.T, axis=1)
    bad = ~np.isfinite(lse_scipy)
    assert bad.tolist() == [False, True, False, False, True, False], bad
    r = conf(h2, w, target_ids=t)
    assert np.all(r["argmax"][bad] == -1), r["argmax"]
    for key in ("max_prob", "lse", "target_prob"):
        assert np.all(np.isnan(r[key][bad])), (key, r[key])
        assert np.array_equal(r[key][~bad], clean[key][~bad]), key
    assert np.array_equal(r["argmax"][~bad], clean["argmax"][~bad])


CONFIDENCE_CHECKS = [
    check_conf_library,
    check_conf_bruteforce,
    check_conf_zero_hidden,
    check_conf_planted,
    check_conf_sums_to_one,
    check_conf_ties,
    check_conf_nonfinite_rows,
]


# ---------------------------------------------------------------- selection


def load_selection_golden():
    with open(os.path.join(GOLDEN, "select_slots_cases.json")) as f:
        return json.load(f)["cases"]


def check_select_golden(select):
    """Hand cases of the paper's selection rule (Sec. 5.2, tau from Sec. 6)."""
    for case in load_selection_golden():
        tc = np.array(case["token_conf"], dtype=np.float32)[None]
        is_open = None if case.get("open") is None else np.array(case["open"], dtype=np.uint8)[None]
        _, sel, n = select(tc, is_open, case["conf_rule"], case["rule"], case.get("threshold", 0.9), case.get("k", 1))
        got = [int(s) for s in sel[0, : n[0]]]
        assert got == case["expect"], f"{case['name']}: got {got}, expected {case['expect']}"
        assert np.all(sel[0, n[0]:] == -1), f"{case['name']}: padding"


def check_select_nan_reported(select):
    """A NaN slot confidence is reported as -inf and selects like -inf, for
    both confidence rules; closed slots still report -1."""
    rng = np.random.default_rng(31)
    B, S, L = 3, 7, 3
    tc = rng.random((B, S, L)).astype(np.float32)
    tc[0, 2, 0] = np.nan  # first token NaN: the slot's confidence under both rules
    tc[1, 4, 1] = np.nan  # a later token NaN: only the mean is NaN
    tc[2, :, 0] = np.nan
    op = np.ones((B, S), dtype=np.uint8)
    op[2, 5] = 0
    for cr in (0, 1):
        minus = tc.copy()
        minus[np.isnan(minus)] = -np.inf
        for rule, k in ((0, 1), (1, 4), (1, S)):
            sc, sel, n = select(tc, op, cr, rule, 0.5, k)
            sc2, sel2, n2 = select(minus, op, cr, rule, 0.5, k)
            assert np.array_equal(sel, sel2) and np.array_equal(n, n2), (cr, rule, k)
            assert np.array_equal(sc, sc2), (cr, rule, k)
            assert not np.isnan(sc).any()
            assert sc[2, 5] == -1.0
    sc, _, _ = select(tc, op, 0, 0, 0.5, 1)
    assert sc[0, 2] == -np.inf and np.isfinite(sc[1, 4])
    sc, _, _ = select(tc, op, 1, 0, 0.5, 1)
    assert sc[0, 2] == -np.inf and sc[1, 4] == -np.inf


SELECTION_CHECKS = [check_select_golden, check_select_nan_reported]


# ------------------------------------------------------- verification


def load_accept_golden():
    with open(os.path.join(GOLDEN, "accept_cases.json")) as f:
        return json.load(f)["cases"]


def check_accept_golden(accept):
    """Hand cases of the acceptance rule (Sec. 5.2 verification, threshold from Sec. 6)."""
    for case in load_accept_golden():
        tp = np.array(case["token_prob"], dtype=np.float32)[None]
        sel = np.array(case["selected"], dtype=np.int32)[None]
        acc, n, tot = accept(tp, sel, np.float32(case["threshold"]), case["rule"])
        exp = np.array(case["expect"], dtype=np.uint8)
        assert np.array_equal(acc[0], exp), f"{case['name']}: got {acc[0].tolist()}, expected {exp.tolist()}"
        assert np.array_equal(n[0], exp.sum(axis=1)), f"{case['name']}: per-slot counts"
        assert int(tot[0]) == int(exp.sum()), f"{case['name']}: total"


def check_accept_invariants(accept):
    """Random batches: accepted tokens pass the threshold, lie in selected
    slots, form a leading run under the prefix rule, and the prefix rule
    accepts a subset of what the per-token rule accepts."""
    rng = np.random.default_rng(70)
    B, S, L = 40, 6, 5
    tp = rng.random((B, S, L)).astype(np.float32)
    tp[rng.random((B, S, L)) < 0.1] = np.float32(0.4)
    sel = np.full((B, S), -1, dtype=np.int32)
    for b in range(B):
        k = int(rng.integers(0, S + 1))
        sel[b, :k] = rng.permutation(S)[:k]
    thr = np.float32(0.4)
    a_pre, n_pre, t_pre = accept(tp, sel, thr, oracle.ACCEPT_PREFIX)
    a_tok, n_tok, t_tok = accept(tp, sel, thr, oracle.ACCEPT_PER_TOKEN)
    for b in range(B):
        chosen = set(int(s) for s in sel[b] if s >= 0)
        for s in range(S):
            if s not in chosen:
                assert not a_pre[b, s].any() and not a_tok[b, s].any(), "unselected slot accepted"
                continue
            above = tp[b, s] > thr
            assert np.array_equal(a_tok[b, s].astype(bool), above), "per-token rule"
            run = 0
            while run < L and above[run]:
                run += 1
            assert a_pre[b, s].tolist() == [1] * run + [0] * (L - run), "prefix rule is the leading run"
    assert np.all(a_pre <= a_tok)
    assert np.array_equal(n_pre, a_pre.sum(axis=2)) and np.array_equal(t_pre, n_pre.sum(axis=1))
    assert np.array_equal(t_tok, a_tok.sum(axis=(1, 2)))


def check_append_hand(append):
    """A worked append: prefix of 2, slots taken in the order [1, 0]."""
    B, Hkv, C, D, S, L = 1, 2, 7, 2, 2, 2
    kc = np.full((B, Hkv, C, D), -1.0)
    vc = np.full((B, Hkv, C, D), -2.0)
    ks = np.arange(B * Hkv * S * L * D, dtype=np.float64).reshape(B, Hkv, S * L, D)
    vs = 100.0 + ks
    acc = np.array([[[1, 0], [1, 1]]], dtype=np.uint8)
    kc2, vc2, lens = append(kc, vc, [2], ks, vs, acc, np.array([[1, 0]]))
    assert lens.tolist() == [5]
    # positions 2, 3, 4 take tokens 2, 3 (slot 1) then 0 (slot 0, position 0)
    for g in range(Hkv):
        assert np.array_equal(kc2[0, g, 2:5], ks[0, g, [2, 3, 0]])
        assert np.array_equal(vc2[0, g, 2:5], vs[0, g, [2, 3, 0]])
        assert np.all(kc2[0, g, :2] == -1.0) and np.all(kc2[0, g, 5:] == -1.0)
        assert np.all(vc2[0, g, :2] == -2.0) and np.all(vc2[0, g, 5:] == -2.0)
    # a slot listed again is committed once: the order [1, 1] appends slot 1's two tokens once
    kc4, vc4, lens4 = append(kc, vc, [2], ks, vs, acc, np.array([[1, 1]]))
    assert lens4.tolist() == [4]
    for g in range(Hkv):
        assert np.array_equal(kc4[0, g, 2:4], ks[0, g, [2, 3]]) and np.all(kc4[0, g, 4:] == -1.0)
        assert np.array_equal(vc4[0, g, 2:4], vs[0, g, [2, 3]]) and np.all(vc4[0, g, 4:] == -2.0)
    # the same append into a cache of capacity 4 does not fit: the row is left as it was
    kc3, vc3, lens3 = append(kc[:, :, :4], vc[:, :, :4], [2], ks, vs, acc, np.array([[1, 0]]))
    assert lens3.tolist() == [2] and np.all(kc3 == -1.0) and np.all(vc3 == -2.0)


def check_append_invariants(append):
    """Random appends: the prefix and the tail of every row are untouched and
    the appended rows are the accepted draft tokens, slot order then position
    order."""
    rng = np.random.default_rng(71)
    B, Hkv, D, S, L, C = 5, 3, 4, 4, 3, 30
    T = S * L
    kc = rng.standard_normal((B, Hkv, C, D))
    vc = rng.standard_normal((B, Hkv, C, D))
    ks = rng.standard_normal((B, Hkv, T, D))
    vs = rng.standard_normal((B, Hkv, T, D))
    acc = (rng.random((B, S, L)) < 0.5).astype(np.uint8)
    order = np.full((B, S), -1, dtype=np.int32)
    for b in range(B):
        k = int(rng.integers(0, S + 1))
        order[b, :k] = rng.permutation(S)[:k]
    plens = rng.integers(0, C - T + 1, B)
    kc2, vc2, lens = append(kc, vc, plens, ks, vs, acc, order)
    for b in range(B):
        toks = [s * L + r for s in order[b] if s >= 0 for r in range(L) if acc[b, s, r]]
        p0, n = int(plens[b]), len(toks)
        assert int(lens[b]) == p0 + n
        assert np.array_equal(kc2[b, :, :p0], kc[b, :, :p0]) and np.array_equal(kc2[b, :, p0 + n:], kc[b, :, p0 + n:])
        assert np.array_equal(vc2[b, :, :p0], vc[b, :, :p0]) and np.array_equal(vc2[b, :, p0 + n:], vc[b, :, p0 + n:])
        assert np.array_equal(kc2[b, :, p0:p0 + n], ks[b][:, toks]) and np.array_equal(vc2[b, :, p0:p0 + n], vs[b][:, toks])


ACCEPT_CHECKS = [check_accept_golden, check_accept_invariants]
APPEND_CHECKS = [check_append_hand, check_append_invariants]


# ------------------------------------------------------------------ sampling

# Known-answer vectors of Philox4x32-10 published with the generator (Salmon,
# Moraes, Dror, Shaw, SC 2011; the Random123 distribution): (counter, key) ->
# output words.
PHILOX_KAT = [
    ((0x00000000, 0x00000000, 0x00000000, 0x00000000), (0x00000000, 0x00000000),
     (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)),
    ((0xFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF), (0xFFFFFFFF, 0xFFFFFFFF),
     (0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)),
    ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0),
     (0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1)),
]


def check_philox_kat(philox):
    for ctr, key, want in PHILOX_KAT:
        got = tuple(int(x) for x in philox(np.array(ctr), np.array(key)))
        assert got == want, f"Philox4x32-10 {ctr} {key}: {[hex(x) for x in got]}"


def check_uniform_moments(unif):
    """u strictly inside (0, 1), mean 1/2 and variance 1/12 within 5 sigma,
    and different rows / offsets / seeds give different streams."""
    u = unif(np.arange(1000), 1000, seed=7, offset=3)
    n = u.size
    assert u.min() > 0.0 and u.max() < 1.0
    assert abs(u.mean() - 0.5) < 5 * np.sqrt(1 / 12 / n)
    assert abs(u.var() - 1 / 12) < 5 * np.sqrt(1 / 180 / n)  # var of (u - 1/2)^2 is 1/180
    assert not np.array_equal(u[0], u[1]), "rows share a stream"
    assert not np.array_equal(unif([0], 1000, 7, 4), u[:1]), "offsets share a stream"
    assert not np.array_equal(unif([0], 1000, 8, 3), u[:1]), "seeds share a stream"
    # neighbouring ids are uncorrelated
    assert abs(np.corrcoef(u[:, :-1].ravel(), u[:, 1:].ravel())[0, 1]) < 5 / np.sqrt(n)


def check_gumbel_moments(unif):
    """-ln(-ln u) has the standard Gumbel mean (Euler's gamma) and variance pi^2/6."""
    g = oracle.gumbel(unif(np.arange(500), 2000, seed=11, offset=0))
    n = g.size
    assert abs(g.mean() - np.euler_gamma) < 5 * np.sqrt(np.pi ** 2 / 6 / n)
    assert abs(g.var() - np.pi ** 2 / 6) < 0.02 * np.pi ** 2 / 6


def _logit_rows(z, M):
    """hidden / W such that every one of M rows has logits z (W = identity)."""
    z = np.asarray(z, dtype=np.float64)
    return np.tile(z, (M, 1)), np.eye(z.size)


def check_sampling_distribution(sample):
    """Gumbel-max: over many rows the drafted ids follow softmax(z / T)."""
    z = np.array([1.2, -0.3, 0.0, 2.1, 0.7])
    for T in (0.6, 1.7):
        h, w = _logit_rows(z, 20000)
        ids = sample(h, w, T, seed=5, offset=9)["sample_id"]
        freq = np.bincount(ids, minlength=z.size) / ids.size
        p = scipy.special.softmax(z / T)
        sd = np.sqrt(p * (1 - p) / ids.size)
        assert np.all(np.abs(freq - p) < 5 * sd), f"T={T}: frequencies {freq} vs softmax {p}"


def check_sampling_cold_and_prob(sample):
    """A tiny temperature gives the argmax; the reported probability is the
    model's own softmax probability of the drafted id."""
    rng = np.random.default_rng(12)
    h = rng.standard_normal((40, 16))
    w = rng.standard_normal((300, 16))
    z = h @ w.T
    r = sample(h, w, 1e-5, seed=1, offset=2)
    assert np.array_equal(r["sample_id"], np.argmax(z, axis=1))
    r = sample(h, w, 1.0, seed=1, offset=2)
    p = scipy.special.softmax(z, axis=1)[np.arange(40), r["sample_id"]]
    _close(r["sample_prob"], p, tol=1e-12, what="sample_prob")
    _close(r["lse"], scipy.special.logsumexp(z, axis=1), tol=1e-12, what="sampling lse")
    assert not np.array_equal(r["sample_id"], np.argmax(z, axis=1)), "T = 1 should not be greedy on 40 rows"


PHILOX_CHECKS = [check_philox_kat]
UNIFORM_CHECKS = [check_uniform_moments, check_gumbel_moments]
def check_sampling_nonfinite_rows(sample):
    """A row with a NaN or infinite hidden value has no distribution to draw
    from (scipy's logsumexp of its logits is not finite): sample id -1 and NaN
    probabilities; the other rows draw what they draw without it."""
    rng = np.random.default_rng(13)
    h = rng.standard_normal((5, 16))
    w = rng.standard_normal((200, 16))
    clean = sample(h, w, 0.8, seed=3, offset=4)
    h2 = h.copy()
    h2[2, 7] = np.nan
    h2[3, 1] = -np.inf
    with np.errstate(invalid="ignore", over="ignore"):
        bad = ~np.isfinite(scipy.special.logsumexp(h2 @ w.T, axis=1))
    assert bad.tolist() == [False, False, True, True, False]
    r = sample(h2, w, 0.8, seed=3, offset=4)
    assert np.all(r["sample_id"][bad] == -1)
    assert np.all(np.isnan(r["sample_prob"][bad])) and np.all(np.isnan(r["lse"][bad]))
    assert np.array_equal(r["sample_id"][~bad], clean["sample_id"][~bad])
    assert np.array_equal(r["sample_prob"][~bad], clean["sample_prob"][~bad])


SAMPLING_CHECKS = [check_sampling_distribution, check_sampling_cold_and_prob, check_sampling_nonfinite_rows]


# ---------------------------------------------------------------- Mode A (Sec. 5.1)

def load_mdm_golden():
    with open(os.path.join(GOLDEN, "mdm_cases.json")) as f:
        return json.load(f)


def check_budget_golden(budget):
    """Hand cases of the mask budget (Sec. 5.1 step 1 and its readings)."""
    for case in load_mdm_golden()["budget"]:
        counts, t = budget(case["n_masked"], case["n_steps"], case["alpha0"], seed=3)
        assert list(map(int, counts)) == case["expect"], f"{case['name']}: got {list(counts)}"
        assert t == case["n_diffusion_steps"], f"{case['name']}: {t} diffusion steps"


def check_budget_structure(budget):
    """Every plan reveals each mask exactly once; diffusion steps are as even
    as possible; sequential steps reveal one token; T = 0 gives steps of at
    most four."""
    rng = np.random.default_rng(80)
    for _ in range(200):
        N = int(rng.integers(0, 300))
        T = int(rng.integers(0, 12))
        a = float(rng.choice([0.0, 0.1, 0.25, 0.5, 0.9, 1.0]))
        counts, t = budget(N, T, a, seed=int(rng.integers(0, 2**63)))
        counts = np.asarray(counts)
        assert counts.sum() == N, (N, T, a)
        if N == 0:
            assert counts.size == 0 and t == 0
            continue
        assert t == (T if T > 0 else -(-N // 4))
        diff, seq = counts[:t], counts[t:]
        assert diff.size == t and np.all(seq == 1)
        assert diff.max() - diff.min() <= 1 and np.all(np.diff(diff) <= 0)
        if T == 0:
            assert seq.size == 0 and diff.max() <= 4
        if T > 0 and a == 0.0:  # T = 0 skips the binomial draw
            assert diff.sum() == 0
        if a == 1.0:
            assert seq.size == 0


def check_budget_binomial(budget):
    """The number of diffusion tokens follows Binomial(N, alpha_0) over seeds
    (chi-square against scipy's pmf, bins with expectation >= 5)."""
    import scipy.stats

    N, a, runs = 40, 0.3, 4000
    n_diff = np.array([int(np.asarray(budget(N, 5, a, seed=s)[0])[:5].sum()) for s in range(runs)])
    obs = np.bincount(n_diff, minlength=N + 1).astype(np.float64)
    exp = scipy.stats.binom.pmf(np.arange(N + 1), N, a) * runs
    keep = exp >= 5
    o = np.append(obs[keep], obs[~keep].sum())
    e = np.append(exp[keep], exp[~keep].sum())
    chi2 = float(((o - e) ** 2 / e).sum())
    assert chi2 < scipy.stats.chi2.ppf(1 - 1e-4, o.size - 1), f"chi2 {chi2:.1f} over {o.size - 1} dof"
    assert abs(n_diff.mean() - N * a) < 5 * np.sqrt(N * a * (1 - a) / runs)


def _reveal_conf(values):
    return np.array([np.nan if v == "nan" else v for v in values], dtype=np.float32)


def check_reveal_golden(reveal):
    """Hand cases of the reveal rules."""
    for case in load_mdm_golden()["reveal"]:
        conf = _reveal_conf(case["conf"])[None]
        op = np.array(case["open"], dtype=bool)[None]
        order, n, op2, _ = reveal(conf, op, [case["k"]], case["rule"])
        exp = case["expect"]
        assert order[0, : len(exp)].tolist() == exp and np.all(order[0, len(exp):] == -1), \
            f"{case['name']}: got {order[0].tolist()}"
        assert int(n[0]) == len(exp)
        want = op[0].copy()
        want[exp] = False
        assert np.array_equal(op2[0], want), f"{case['name']}: open mask"


def check_reveal_invariants(reveal):
    """Random rows, all three rules: revealed positions were open and are now
    closed, n = min(k, open count), tokens change only there; the confidence
    rule matches a stable descending sort of the open positions, the leftmost
    rule the lowest open indices."""
    rng = np.random.default_rng(81)
    B, N = 30, 17
    conf = rng.random((B, N)).astype(np.float32)
    conf[rng.random((B, N)) < 0.2] = np.float32(0.5)  # ties
    op = rng.random((B, N)) < 0.7
    k = rng.integers(0, N + 3, B)
    tokens = rng.integers(0, 1000, (B, N))
    sid = rng.integers(0, 1000, (B, N))
    for rule in (oracle.REVEAL_CONFIDENCE, oracle.REVEAL_LEFTMOST, oracle.REVEAL_RANDOM):
        order, n, op2, tok = reveal(conf, op, k, rule, seed=5, offset=6, tokens=tokens, sample_id=sid)
        for b in range(B):
            cnt = int(n[b])
            opened = np.flatnonzero(op[b])
            assert cnt == min(int(k[b]), opened.size)
            pick = order[b, :cnt]
            assert np.all(order[b, cnt:] == -1) and len(set(pick.tolist())) == cnt
            assert np.all(op[b, pick]) and not np.any(op2[b, pick])
            assert np.array_equal(op2[b] | np.isin(np.arange(N), pick), op[b])
            assert np.array_equal(tok[b, pick], sid[b, pick])
            rest = np.setdiff1d(np.arange(N), pick)
            assert np.array_equal(tok[b, rest], tokens[b, rest])
            if rule == oracle.REVEAL_CONFIDENCE:
                ranked = opened[np.argsort(-conf[b, opened].astype(np.float64), kind="stable")]
                assert np.array_equal(pick, ranked[:cnt])
            if rule == oracle.REVEAL_LEFTMOST:
                assert np.array_equal(pick, opened[:cnt])


def check_reveal_random_uniform(reveal):
    """REVEAL_RANDOM chooses a uniformly random subset: over many offsets each
    open position is revealed with probability k / #open and is the first
    pick with probability 1 / #open; batch rows draw independently."""
    N, k, runs = 6, 2, 3000
    op = np.ones((2, N), dtype=bool)
    op[:, 4] = False  # 5 open positions
    hits = np.zeros(N)
    first = np.zeros(N)
    same = 0
    for off in range(runs):
        order, n, _, _ = reveal(np.zeros((2, N), np.float32), op, [k, k], oracle.REVEAL_RANDOM, seed=9, offset=off)
        hits[order[0, :k]] += 1
        first[order[0, 0]] += 1
        same += int(set(order[0, :k].tolist()) == set(order[1, :k].tolist()))
    assert hits[4] == 0 and first[4] == 0
    p = k / 5
    assert np.all(np.abs(hits[op[0]] / runs - p) < 5 * np.sqrt(p * (1 - p) / runs)), hits
    q = 1 / 5
    assert np.all(np.abs(first[op[0]] / runs - q) < 5 * np.sqrt(q * (1 - q) / runs)), first
    # two rows agree on the subset with probability 1 / C(5, 2) = 0.1
    assert abs(same / runs - 0.1) < 5 * np.sqrt(0.09 / runs), same


BUDGET_CHECKS = [check_budget_golden, check_budget_structure, check_budget_binomial]
REVEAL_CHECKS = [check_reveal_golden, check_reveal_invariants, check_reveal_random_uniform]
