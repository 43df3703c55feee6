"""The C-ABI library: it loads, exports every declared symbol, and validates
arguments on the host before any launch (CPU only: no call here reaches HIP)."""

import ctypes
import os
import re
import subprocess

import pytest

import workloads as W

from paper_2609_19868_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "zarya.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(zarya_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_the_binding_exports():
    assert declared_functions() == sorted(_lib.EXPORTS)


def test_library_exports_every_declared_symbol():
    L = _lib.lib()
    out = subprocess.run(["nm", "-D", "--defined-only", _lib.LIB_PATH], capture_output=True, text=True, check=True).stdout
    dyn = set(re.findall(r"\sT\s(\S+)", out))
    for name in declared_functions():
        assert name in dyn, f"{name} is not exported"
        assert hasattr(L, name)


def test_version_and_status_strings():
    L = _lib.lib()
    assert L.zarya_version() == 5
    for code, name in [(0, "ZARYA_OK"), (1, "ZARYA_ERR_INVALID_ARGUMENT"), (2, "ZARYA_ERR_UNSUPPORTED"),
                       (3, "ZARYA_ERR_WORKSPACE_TOO_SMALL"), (4, "ZARYA_ERR_HIP")]:
        assert L.zarya_status_string(code).decode() == name


def _desc(**kw):
    base = dict(batch=2, n_q_heads=4, n_kv_heads=2, head_dim=128, prefix_len=100, kv_capacity=128, n_slots=4,
                slot_len=8, softmax_scale=0.088, pass_=0, cross_slot=0, dtype=1, prefix_splits=0)
    base.update(kw)
    return _lib.SlotAttnDesc(**base)


def _attn_status(desc, ptr=1, ws=None, ws_bytes=0):
    p = ctypes.c_void_p(ptr) if ptr else None
    return _lib.lib().zarya_slot_attn(ctypes.byref(desc), p, p, p, p, p, None, None, p, None, ws, ws_bytes, None)


@pytest.mark.parametrize("bad,code", [
    (dict(batch=0), _lib.ERR_INVALID_ARGUMENT),
    (dict(n_q_heads=3), _lib.ERR_INVALID_ARGUMENT),
    (dict(n_kv_heads=0), _lib.ERR_INVALID_ARGUMENT),
    (dict(prefix_len=-1), _lib.ERR_INVALID_ARGUMENT),
    (dict(kv_capacity=50), _lib.ERR_INVALID_ARGUMENT),
    (dict(n_slots=0), _lib.ERR_INVALID_ARGUMENT),
    (dict(slot_len=0), _lib.ERR_INVALID_ARGUMENT),
    (dict(softmax_scale=0.0), _lib.ERR_INVALID_ARGUMENT),
    (dict(softmax_scale=float("nan")), _lib.ERR_INVALID_ARGUMENT),
    (dict(pass_=2), _lib.ERR_INVALID_ARGUMENT),
    (dict(cross_slot=5), _lib.ERR_INVALID_ARGUMENT),
    (dict(dtype=7), _lib.ERR_INVALID_ARGUMENT),
    (dict(prefix_splits=65), _lib.ERR_INVALID_ARGUMENT),
    (dict(head_dim=96), _lib.ERR_UNSUPPORTED),
    (dict(batch=1 << 20, n_q_heads=64, n_kv_heads=64), _lib.ERR_UNSUPPORTED),
])
def test_slot_attn_rejects_bad_descriptors(bad, code):
    d = _desc(**bad)
    assert _attn_status(d) == code
    assert len(_lib.lib().zarya_last_error()) > 0
    n = ctypes.c_size_t(0)
    assert _lib.lib().zarya_slot_attn_workspace_size(ctypes.byref(d), ctypes.byref(n)) == code


def test_slot_attn_rejects_null_pointers_and_small_workspace():
    d = _desc()
    assert _attn_status(d, ptr=0) == _lib.ERR_INVALID_ARGUMENT
    need = _lib.slot_attn_workspace_size(d)
    if need > 0:
        assert _attn_status(d, ws=ctypes.c_void_p(1), ws_bytes=need - 1) == _lib.ERR_WORKSPACE_TOO_SMALL
        assert _attn_status(d, ws=None, ws_bytes=need) == _lib.ERR_INVALID_ARGUMENT
    # a prefix needs the cache pointers
    p = ctypes.c_void_p(1)
    assert _lib.lib().zarya_slot_attn(ctypes.byref(d), p, None, None, p, p, None, None, p, None, p, 1 << 40,
                                      None) == _lib.ERR_INVALID_ARGUMENT


def test_slot_attn_plan_reports_the_decomposition():
    """The planner's choice, as zarya_slot_attn_plan reports it, is consistent
    with the workspace it asks for and covers every GQA group."""
    for name in ("qwen0.6b", "qwen1.7b", "qwen4b"):
        wl = W.WORKLOADS[name]
        d = _lib.SlotAttnDesc(batch=wl.batch, n_q_heads=wl.n_q_heads, n_kv_heads=wl.n_kv_heads, head_dim=128,
                              prefix_len=wl.prefix_len, kv_capacity=wl.prefix_len, n_slots=wl.n_slots,
                              slot_len=wl.slot_len, softmax_scale=0.088, pass_=0, cross_slot=0, dtype=1)
        plan = _lib.slot_attn_plan(d)
        groups = wl.batch * wl.n_kv_heads
        rows = wl.n_q_heads // wl.n_kv_heads * wl.T
        rb = -(-rows // plan["rows_per_workgroup"])
        assert plan["workgroups"] == groups * rb * plan["prefix_splits"], (name, plan)
        assert 1 <= plan["prefix_splits"] <= 64 and plan["kernels"] in (1, 2)
        assert (_lib.slot_attn_workspace_size(d) > 0) == (plan["prefix_splits"] > 1)
    d = _lib.SlotAttnDesc(batch=1, n_q_heads=2, n_kv_heads=1, head_dim=64, prefix_len=64, kv_capacity=64,
                          n_slots=4, slot_len=4, softmax_scale=0.125, pass_=0, cross_slot=0, dtype=0)
    assert _lib.slot_attn_plan(d) == {"prefix_splits": 1, "rows_per_workgroup": 32, "workgroups": 1, "kernels": 1}
    assert _lib.lib().zarya_slot_attn_plan(ctypes.byref(d), None) == _lib.ERR_INVALID_ARGUMENT


def test_noalloc_confidence_rejects_before_touching_a_device():
    """The allocation-free confidence call validates its descriptor and the
    size of its partials first: on this host, without a GPU, a bad or
    oversized call returns its status without reaching the runtime."""
    L = _lib.lib()
    d = _lib.ConfDesc(n_rows=0, hidden=64, vocab=100, dtype=_lib.DTYPE_BF16)
    p = ctypes.c_void_p(16)
    assert L.zarya_slot_confidence_noalloc(ctypes.byref(d), p, p, None, p, p, None, None, None) == \
        _lib.ERR_INVALID_ARGUMENT
    d = _lib.ConfDesc(n_rows=8, hidden=64, vocab=100, dtype=_lib.DTYPE_BF16)
    assert L.zarya_slot_confidence_noalloc(ctypes.byref(d), p, None, None, p, p, None, None, None) == \
        _lib.ERR_INVALID_ARGUMENT
    # float32, 1400 rows x 64 vocabulary groups of 12-byte partials: more than the 1 MiB scratch
    d = _lib.ConfDesc(n_rows=1400, hidden=8, vocab=131072, dtype=_lib.DTYPE_F32)
    assert L.zarya_slot_confidence_noalloc(ctypes.byref(d), p, p, None, p, p, None, None, None) == \
        _lib.ERR_UNSUPPORTED
    assert b"scratch" in L.zarya_last_error()


def test_slot_attn_workspace_sizes():
    # one split needs no workspace; several splits need fp32 partials of O and LSE
    d1 = _desc(prefix_splits=1)
    assert _lib.slot_attn_workspace_size(d1) == 0
    d4 = _desc(prefix_len=1024, kv_capacity=1024, prefix_splits=4)
    rows = 2 * 4 * 32
    assert _lib.slot_attn_workspace_size(d4) >= 4 * rows * (128 + 1) * 4
    assert _lib.slot_attn_workspace_size(_desc(dtype=0)) == 0  # float32 path has no splits
    assert _lib.slot_attn_workspace_size(_desc(prefix_len=0, kv_capacity=0)) == 0


def _conf_status(desc, ptr=1, ws_bytes=1 << 40):
    p = ctypes.c_void_p(ptr) if ptr else None
    return _lib.lib().zarya_slot_confidence(ctypes.byref(desc), p, p, None, p, p, None, None, p, ws_bytes, None)


@pytest.mark.parametrize("bad,code", [
    (dict(n_rows=0), _lib.ERR_INVALID_ARGUMENT),
    (dict(hidden=0), _lib.ERR_INVALID_ARGUMENT),
    (dict(vocab=0), _lib.ERR_INVALID_ARGUMENT),
    (dict(dtype=3), _lib.ERR_INVALID_ARGUMENT),
    (dict(hidden=1001), _lib.ERR_UNSUPPORTED),
    (dict(dtype=0, hidden=10000), _lib.ERR_UNSUPPORTED),
    (dict(hidden=4194304 + 8), _lib.ERR_UNSUPPORTED),  # 256-row W tiles need 32-bit offsets
])
def test_slot_confidence_rejects_bad_descriptors(bad, code):
    base = dict(n_rows=64, hidden=1024, vocab=151936, dtype=1)
    base.update(bad)
    assert _conf_status(_lib.ConfDesc(**base)) == code


def test_slot_confidence_workspace_checks():
    d = _lib.ConfDesc(n_rows=1024, hidden=1024, vocab=151936, dtype=1)
    need = _lib.slot_confidence_workspace_size(d)
    assert need >= 64 * 1024 * 12
    assert _conf_status(d, ws_bytes=need - 1) == _lib.ERR_WORKSPACE_TOO_SMALL
    assert _conf_status(d, ptr=0) == _lib.ERR_INVALID_ARGUMENT


def _sample_status(desc, temperature=1.0, ptr=1, ws_bytes=1 << 40, params=True, out_null=None, rows=None,
                   hidden_rows=0):
    p = ctypes.c_void_p(ptr) if ptr else None
    sp = _lib.SampleParams(temperature=temperature, seed=1, offset=2)
    outs = [p, p]
    if out_null is not None:
        outs[out_null] = None
    return _lib.lib().zarya_slot_sample(ctypes.byref(desc), ctypes.byref(sp) if params else None, p, rows,
                                        hidden_rows, p, *outs, None, None, p, ws_bytes, None)


@pytest.mark.parametrize("temperature", [0.0, -1.0, float("nan"), float("inf"), 1e-31])
def test_slot_sample_rejects_bad_temperatures(temperature):
    d = _lib.ConfDesc(n_rows=64, hidden=1024, vocab=151936, dtype=1)
    assert _sample_status(d, temperature=temperature) == _lib.ERR_INVALID_ARGUMENT
    assert "temperature" in _lib.lib().zarya_last_error().decode()


def test_slot_sample_argument_checks():
    d = _lib.ConfDesc(n_rows=1024, hidden=1024, vocab=151936, dtype=1)
    need = _lib.slot_sample_workspace_size(d)
    # two more partial arrays than the greedy reduction: best perturbed score and its id
    assert need > _lib.slot_confidence_workspace_size(d)
    assert need >= 64 * 1024 * 20
    assert _sample_status(d, ws_bytes=need - 1) == _lib.ERR_WORKSPACE_TOO_SMALL
    assert _sample_status(d, ptr=0) == _lib.ERR_INVALID_ARGUMENT
    assert _sample_status(d, params=False) == _lib.ERR_INVALID_ARGUMENT
    assert _sample_status(d, out_null=0) == _lib.ERR_INVALID_ARGUMENT  # sample_id is required
    assert _sample_status(d, out_null=1) == _lib.ERR_INVALID_ARGUMENT  # sample_prob is required
    # a row selection needs the hidden row count, and its bytes must stay below 4 GiB
    r = ctypes.c_void_p(1)
    assert _sample_status(d, rows=r, hidden_rows=0) == _lib.ERR_INVALID_ARGUMENT
    assert _sample_status(d, rows=r, hidden_rows=1 << 21) == _lib.ERR_UNSUPPORTED
    for bad, code in [(dict(n_rows=0), _lib.ERR_INVALID_ARGUMENT), (dict(hidden=1001), _lib.ERR_UNSUPPORTED)]:
        base = dict(n_rows=64, hidden=1024, vocab=151936, dtype=1)
        base.update(bad)
        assert _sample_status(_lib.ConfDesc(**base)) == code


@pytest.mark.parametrize("args,code", [
    (dict(batch=0), _lib.ERR_INVALID_ARGUMENT),
    (dict(n_slots=0), _lib.ERR_INVALID_ARGUMENT),
    (dict(n_slots=2048), _lib.ERR_UNSUPPORTED),
    (dict(slot_len=0), _lib.ERR_INVALID_ARGUMENT),
    (dict(conf_rule=2), _lib.ERR_INVALID_ARGUMENT),
    (dict(rule=9), _lib.ERR_INVALID_ARGUMENT),
    (dict(rule=1, k=-1), _lib.ERR_INVALID_ARGUMENT),
    (dict(ptr=0), _lib.ERR_INVALID_ARGUMENT),
])
def test_select_slots_rejects_bad_arguments(args, code):
    a = dict(batch=4, n_slots=8, slot_len=4, conf_rule=0, rule=0, threshold=0.9, k=1, ptr=1)
    a.update(args)
    p = ctypes.c_void_p(a["ptr"]) if a["ptr"] else None
    st = _lib.lib().zarya_select_slots(a["batch"], a["n_slots"], a["slot_len"], p, None, a["conf_rule"], a["rule"],
                                       a["threshold"], a["k"], p, p, p, None)
    assert st == code


@pytest.mark.parametrize("args,code", [
    (dict(batch=0), _lib.ERR_INVALID_ARGUMENT),
    (dict(n_slots=0), _lib.ERR_INVALID_ARGUMENT),
    (dict(slot_len=0), _lib.ERR_INVALID_ARGUMENT),
    (dict(n_slots=2048), _lib.ERR_UNSUPPORTED),
    (dict(slot_len=5000), _lib.ERR_UNSUPPORTED),
    (dict(rule=2), _lib.ERR_INVALID_ARGUMENT),
    (dict(threshold=float("nan")), _lib.ERR_INVALID_ARGUMENT),
    (dict(ptr=0), _lib.ERR_INVALID_ARGUMENT),
])
def test_verify_accept_rejects_bad_arguments(args, code):
    a = dict(batch=4, n_slots=8, slot_len=4, threshold=0.4, rule=0, ptr=1)
    a.update(args)
    p = ctypes.c_void_p(a["ptr"]) if a["ptr"] else None
    st = _lib.lib().zarya_verify_accept(a["batch"], a["n_slots"], a["slot_len"], p, p, a["threshold"], a["rule"],
                                        p, p, None, None)
    assert st == code
    assert len(_lib.lib().zarya_last_error()) > 0


@pytest.mark.parametrize("bad,code", [
    (dict(batch=0), _lib.ERR_INVALID_ARGUMENT),
    (dict(n_kv_heads=0), _lib.ERR_INVALID_ARGUMENT),
    (dict(n_slots=0), _lib.ERR_INVALID_ARGUMENT),
    (dict(kv_capacity=-1), _lib.ERR_INVALID_ARGUMENT),
    (dict(dtype=5), _lib.ERR_INVALID_ARGUMENT),
    (dict(head_dim=80), _lib.ERR_UNSUPPORTED),
    (dict(n_slots=1025, slot_len=1), _lib.ERR_UNSUPPORTED),
    (dict(n_slots=512, slot_len=32), _lib.ERR_UNSUPPORTED),
    (dict(batch=4096, n_kv_heads=64, kv_capacity=1 << 14), _lib.ERR_UNSUPPORTED),
])
def test_kv_append_rejects_bad_descriptors(bad, code):
    base = dict(batch=2, n_kv_heads=8, head_dim=128, kv_capacity=4096, n_slots=8, slot_len=8, dtype=1)
    base.update(bad)
    d = _lib.KvAppendDesc(**base)
    p = ctypes.c_void_p(1)
    assert _lib.lib().zarya_kv_append(ctypes.byref(d), p, p, p, p, p, p, p, None) == code
    assert len(_lib.lib().zarya_last_error()) > 0


def test_kv_append_requires_every_tensor():
    d = _lib.KvAppendDesc(batch=2, n_kv_heads=8, head_dim=128, kv_capacity=4096, n_slots=8, slot_len=8, dtype=1)
    p = ctypes.c_void_p(1)
    for i in range(7):
        args = [p] * 7
        args[i] = None
        assert _lib.lib().zarya_kv_append(ctypes.byref(d), *args, None) == _lib.ERR_INVALID_ARGUMENT


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(_lib, "_lib", None)
    monkeypatch.setattr(_lib, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(ImportError):
        _lib.lib()


def test_library_has_no_undefined_own_symbols():
    out = subprocess.run(["nm", "-D", "--undefined-only", _lib.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    assert "zarya" not in out, out


def test_binding_refuses_host_tensors():
    """Host (CPU) tensors never reach the library: the binding runs each call
    with the tensors' GPU current, and a CPU device is refused."""
    import torch
    import paper_2609_19868_amd as Z

    h = torch.zeros(4, 64, dtype=torch.bfloat16)
    w = torch.zeros(100, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="cuda"):
        Z.slot_confidence(h, w)
    with pytest.raises(ValueError, match="cuda"):
        Z.select_slots(torch.zeros(2, 3, 4))
    # caller-supplied outputs and workspaces are checked like the inputs
    with pytest.raises(ValueError, match="cuda"):
        Z._need(torch.zeros(4), "out['max_prob']", (4,), torch.float32, torch.device("cpu"))
    with pytest.raises(ValueError, match="cuda"):
        Z._need_workspace(torch.zeros(64, dtype=torch.uint8), 16, torch.device("cpu"))


def test_binding_checks_workspace_shape_and_size():
    """A workspace must be a contiguous 1-D uint8 tensor of at least the
    reported size (its element count is passed as the byte count).  The
    checks are exercised on a stand-in device object, since this host has no
    HIP device: only their logic is under test."""
    import torch
    import paper_2609_19868_amd as Z

    class FakeCuda:
        """Tensor stand-in whose device reads as cuda:0."""

        def __init__(self, t):
            self.t = t
            self.device = torch.device("cuda:0")
            self.dtype = t.dtype
            self.shape = t.shape

        def dim(self):
            return self.t.dim()

        def is_contiguous(self):
            return self.t.is_contiguous()

        def numel(self):
            return self.t.numel()

    dev = torch.device("cuda:0")
    Z._need_workspace(FakeCuda(torch.zeros(64, dtype=torch.uint8)), 64, dev)  # accepted
    with pytest.raises(ValueError, match="uint8"):
        Z._need_workspace(FakeCuda(torch.zeros(64, dtype=torch.float32)), 16, dev)
    with pytest.raises(ValueError, match="required"):
        Z._need_workspace(FakeCuda(torch.zeros(15, dtype=torch.uint8)), 16, dev)
    with pytest.raises(ValueError, match="uint8"):
        Z._need_workspace(FakeCuda(torch.zeros(4, 16, dtype=torch.uint8)), 16, dev)
    with pytest.raises(ValueError, match="uint8"):
        Z._need_workspace(FakeCuda(torch.zeros(64, dtype=torch.uint8)[::2]), 16, dev)
    with pytest.raises(ValueError, match="expected contiguous"):
        Z._need(FakeCuda(torch.zeros(5, dtype=torch.float32)), "out['lse']", (4,), torch.float32, dev)
    with pytest.raises(ValueError, match="expected contiguous"):
        Z._need(FakeCuda(torch.zeros(4, dtype=torch.int64)), "out['argmax']", (4,), torch.int32, dev)
