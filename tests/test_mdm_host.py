"""Mode A host logic through the C ABI, no GPU needed: the mask budget
(zarya_mdm_budget runs on the host only) against the oracle, exactly, and
the argument checks of zarya_mdm_reveal (rejected before any launch)."""

import ctypes

import numpy as np
import pytest

import oracle

import paper_2609_19868_amd as Z
from paper_2609_19868_amd import _lib


def test_budget_matches_the_oracle():
    rng = np.random.default_rng(83)
    cases = [(0, 0, 0.25), (1, 0, 0.25), (10, 0, 0.5), (5, 2, 0.0), (7, 3, 1.0), (2, 4, 1.0), (4096, 16, 0.25),
             (1000, 1, 0.999)]
    cases += [(int(rng.integers(0, 600)), int(rng.integers(0, 20)), float(rng.random())) for _ in range(150)]
    for i, (N, T, a) in enumerate(cases):
        seed = int(rng.integers(0, 2**64, dtype=np.uint64))
        counts, t = Z.mdm_budget(N, T, a, seed)
        ref, t_ref = oracle.mask_budget(N, T, a, seed)
        assert counts == [int(c) for c in ref] and t == t_ref, (N, T, a, seed)


def test_budget_argument_checks():
    L = _lib.lib()
    n, t = ctypes.c_int32(0), ctypes.c_int32(0)
    for args in [(-1, 0, 0.5), (5, -1, 0.5), (5, 2, -0.1), (5, 2, 1.5), (5, 2, float("nan"))]:
        assert L.zarya_mdm_budget(*args, 1, None, 0, ctypes.byref(n), ctypes.byref(t)) == _lib.ERR_INVALID_ARGUMENT
    assert L.zarya_mdm_budget(5, 2, 0.5, 1, None, 0, None, None) == _lib.ERR_INVALID_ARGUMENT
    # the length query, then a buffer one step too short
    assert L.zarya_mdm_budget(10, 0, 0.5, 1, None, 0, ctypes.byref(n), None) == _lib.OK and n.value == 3
    buf = (ctypes.c_int32 * 2)()
    assert L.zarya_mdm_budget(10, 0, 0.5, 1, buf, 2, ctypes.byref(n), None) == _lib.ERR_INVALID_ARGUMENT


@pytest.mark.parametrize("args,code", [
    (dict(batch=0), _lib.ERR_INVALID_ARGUMENT),
    (dict(n=0), _lib.ERR_INVALID_ARGUMENT),
    (dict(n=8193), _lib.ERR_UNSUPPORTED),
    (dict(rule=3), _lib.ERR_INVALID_ARGUMENT),
    (dict(conf=None), _lib.ERR_INVALID_ARGUMENT),
    (dict(mask=None), _lib.ERR_INVALID_ARGUMENT),
    (dict(k=None), _lib.ERR_INVALID_ARGUMENT),
    (dict(order=None), _lib.ERR_INVALID_ARGUMENT),
    (dict(tokens=None), _lib.ERR_INVALID_ARGUMENT),  # sample_id given without tokens
])
def test_reveal_argument_checks(args, code):
    p = ctypes.c_void_p(1)
    a = dict(batch=2, n=100, conf=p, mask=p, k=p, rule=0, seed=1, offset=2, sample_id=p, tokens=p, order=p,
             n_revealed=None)
    a.update(args)
    assert _lib.lib().zarya_mdm_reveal(*a.values(), None) == code
    assert len(_lib.lib().zarya_last_error()) > 0
