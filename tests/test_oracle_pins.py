"""The oracle against what the paper and the mathematics fix (CPU only)."""

import numpy as np
import pytest

import oracle
import oracle_pins as pins


@pytest.mark.parametrize("check", pins.ATTENTION_CHECKS, ids=lambda f: f.__name__)
def test_attention_pin(check):
    check(oracle.slot_attention)


@pytest.mark.parametrize("check", pins.CONFIDENCE_CHECKS, ids=lambda f: f.__name__)
def test_confidence_pin(check):
    check(oracle.slot_confidence)


@pytest.mark.parametrize("check", pins.SELECTION_CHECKS, ids=lambda f: f.__name__)
def test_selection_pin(check):
    check(oracle.select_slots)


@pytest.mark.parametrize("check", pins.ACCEPT_CHECKS, ids=lambda f: f.__name__)
def test_accept_pin(check):
    check(oracle.accept_tokens)


@pytest.mark.parametrize("check", pins.APPEND_CHECKS, ids=lambda f: f.__name__)
def test_append_pin(check):
    check(oracle.kv_append)


def test_attention_probabilities_sum_to_one():
    x = pins._inputs(31, 2, 4, 2, 8, 5, 3, 4)
    for pass_ in (oracle.PASS_DIFFUSION, oracle.PASS_AR_INFILL):
        _, _, p = oracle.slot_attention(x["q"], x["k_cache"], x["v_cache"], x["k_slot"], x["v_slot"],
                                        5, 3, 4, 0.5, pass_, return_probs=True)
        np.testing.assert_allclose(p.sum(axis=-1), 1.0, atol=1e-13)
        mask = oracle.visibility(5, 3, 4, pass_)
        assert np.all(p[..., ~mask] == 0.0)


def test_visibility_counts_match_rule():
    for pass_ in (oracle.PASS_DIFFUSION, oracle.PASS_AR_INFILL):
        for cross in (oracle.CROSS_SLOT_NONE, oracle.CROSS_SLOT_CAUSAL):
            m = oracle.visibility(3, 4, 5, pass_, cross)
            assert np.array_equal(m.sum(axis=1), pins.n_visible(3, 4, 5, pass_, cross))
            assert np.all(m[np.arange(20), 3 + np.arange(20)]), "a token always sees itself"


def test_l1_prefix_zero_is_self_attention():
    # P = 0 and L = 1: a token sees only itself, so O equals its own value row.
    x = pins._inputs(32, 1, 2, 1, 8, 0, 6, 1)
    O, lse = oracle.slot_attention(x["q"], x["k_cache"], x["v_cache"], x["k_slot"], x["v_slot"],
                                   0, 6, 1, 0.5, oracle.PASS_DIFFUSION)
    np.testing.assert_allclose(O, np.repeat(x["v_slot"], 2, axis=1), atol=1e-15)
    s = 0.5 * np.einsum("bhtd,bhtd->bht", x["q"], np.repeat(x["k_slot"], 2, axis=1))
    np.testing.assert_allclose(lse, s, atol=1e-13)


def test_select_first_token_equals_column_zero():
    rng = np.random.default_rng(1)
    tc = rng.random((3, 7, 4)).astype(np.float32)
    np.testing.assert_array_equal(oracle.slot_conf(tc, oracle.CONF_FIRST_TOKEN), tc[:, :, 0])


def test_select_mean_is_rounded_exact_mean():
    # values with few significant bits: the float64 sum is exact, so the mean is
    # the correctly rounded float32 of the exact rational mean
    rng = np.random.default_rng(2)
    tc = (rng.integers(0, 1 << 10, (4, 5, 6)) / 1024.0).astype(np.float32)
    exact = tc.astype(np.float64).sum(axis=2) / 6.0
    np.testing.assert_array_equal(oracle.slot_conf(tc, oracle.CONF_MEAN), exact.astype(np.float32))


def test_select_threshold_always_returns_one_when_open():
    rng = np.random.default_rng(3)
    tc = rng.random((50, 6, 2)).astype(np.float32) * 0.5
    _, sel, n = oracle.select_slots(tc, None, oracle.CONF_FIRST_TOKEN, oracle.SELECT_THRESHOLD, 0.9, 1)
    assert np.all(n == 1)
    np.testing.assert_array_equal(sel[:, 0], np.argmax(tc[:, :, 0], axis=1))


@pytest.mark.parametrize("check", pins.PHILOX_CHECKS, ids=lambda f: f.__name__)
def test_philox_pin(check):
    check(oracle.philox4x32)


@pytest.mark.parametrize("check", pins.UNIFORM_CHECKS, ids=lambda f: f.__name__)
def test_uniform_pin(check):
    check(oracle.uniforms)


@pytest.mark.parametrize("check", pins.SAMPLING_CHECKS, ids=lambda f: f.__name__)
def test_sampling_pin(check):
    check(oracle.slot_sample)


@pytest.mark.parametrize("check", pins.BUDGET_CHECKS, ids=lambda f: f.__name__)
def test_budget_pin(check):
    check(oracle.mask_budget)


@pytest.mark.parametrize("check", pins.REVEAL_CHECKS, ids=lambda f: f.__name__)
def test_reveal_pin(check):
    check(oracle.reveal)
