"""zarya_slot_confidence_noalloc (static device scratch, no workspace) against
zarya_slot_confidence (caller's workspace): the same kernels on the same
inputs, so results must be bit-identical.  Two calls in a row, the second on
a smaller problem (the scratch keeps the first call's partials), then the
first problem again."""

import ctypes

import numpy as np
import pytest
import torch

import workloads as W
from gpu_helpers import require_gpu, say, to_dev

import paper_2609_19868_amd as Z
from paper_2609_19868_amd import _lib

pytestmark = pytest.mark.gpu


def _noalloc(hd, wd, td):
    """The allocation-free call through the C ABI (outputs allocated here,
    by the caller)."""
    M, H = hd.shape
    V = wd.shape[0]
    dev = hd.device
    out = {k: torch.full((M,), -7.0, dtype=torch.float32, device=dev) for k in ("max_prob", "lse", "target_prob")}
    out["argmax"] = torch.full((M,), -7, dtype=torch.int32, device=dev)
    desc = _lib.ConfDesc(n_rows=M, hidden=H, vocab=V, dtype=_lib.DTYPE_BF16)
    ptr = lambda t: ctypes.c_void_p(t.data_ptr())
    with torch.cuda.device(dev):
        _lib.check(_lib.lib().zarya_slot_confidence_noalloc(
            ctypes.byref(desc), ptr(hd), ptr(wd), ptr(td), ptr(out["max_prob"]), ptr(out["argmax"]), ptr(out["lse"]),
            ptr(out["target_prob"]), ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)))
    return out


CASES = [
    ("qwen0.6b rows", dict(batch=16, n_slots=8, slot_len=8, hidden=1024, vocab=151936)),
    ("smaller", dict(batch=1, n_slots=60, slot_len=5, hidden=256, vocab=5003)),
    ("few rows (64-row tile)", dict(batch=1, n_slots=9, slot_len=5, hidden=512, vocab=20011)),
    # 1024 rows x 2560: the hidden rows do not fit in L2, W is loaded with plain loads
    ("4B-scale rows", dict(batch=8, n_slots=8, slot_len=16, hidden=2560, vocab=30011)),
]


def test_noalloc_matches_the_workspace_call():
    dev = require_gpu()
    for i, (name, over) in enumerate(CASES + CASES[:1]):
        wl = W.WORKLOADS["qwen0.6b"].replace(**over, seed=400 + i)
        c = W.confidence_inputs(wl)
        hd, wd = to_dev(c["hidden"], "bf16", dev), to_dev(c["w_vocab"], "bf16", dev)
        td = torch.from_numpy(c["target_ids"]).to(dev)
        say(f"slot_confidence_noalloc call {i}: {name} M={wl.M} H={wl.hidden} V={wl.vocab}")
        got = _noalloc(hd, wd, td)
        ref = Z.slot_confidence(hd, wd, target_ids=td)
        torch.cuda.synchronize()
        for k in ("max_prob", "lse", "target_prob"):
            assert torch.equal(got[k].view(torch.int32), ref[k].view(torch.int32)), (name, k)
        assert torch.equal(got["argmax"], ref["argmax"]), name


def test_noalloc_refuses_partials_beyond_its_scratch():
    """float32, 1400 rows over a 131072-entry vocabulary: 64 vocabulary groups
    of 12-byte partials per row need more than the 1 MiB scratch; the call
    fails before launching anything."""
    dev = require_gpu()
    M, H, V = 1400, 8, 131072
    hd = torch.zeros((M, H), dtype=torch.float32, device=dev)
    wd = torch.zeros((V, H), dtype=torch.float32, device=dev)
    mp = torch.full((M,), -7.0, dtype=torch.float32, device=dev)
    am = torch.full((M,), -7, dtype=torch.int32, device=dev)
    desc = _lib.ConfDesc(n_rows=M, hidden=H, vocab=V, dtype=_lib.DTYPE_F32)
    ptr = lambda t: ctypes.c_void_p(t.data_ptr())
    st = _lib.lib().zarya_slot_confidence_noalloc(ctypes.byref(desc), ptr(hd), ptr(wd), None, ptr(mp), ptr(am), None,
                                                 None, ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream))
    torch.cuda.synchronize()
    assert st == _lib.ERR_UNSUPPORTED
    assert torch.all(mp == -7.0) and torch.all(am == -7)
