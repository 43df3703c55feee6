"""ctypes binding of libzarya.so: argument marshalling only.

Every step of the slot-scoring path runs in the HIP kernels behind the C ABI
declared in include/zarya.h; this module only checks tensor metadata, passes
device pointers and torch's current HIP stream, and turns status codes into
exceptions.  There is no fallback: if the library is missing, loading fails.
"""

from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libzarya.so")

OK = 0
ERR_INVALID_ARGUMENT = 1
ERR_UNSUPPORTED = 2
ERR_WORKSPACE_TOO_SMALL = 3
ERR_HIP = 4

DTYPE_F32 = 0
DTYPE_BF16 = 1
PASS_DIFFUSION = 0
PASS_AR_INFILL = 1
CROSS_SLOT_NONE = 0
CROSS_SLOT_CAUSAL = 1
SLOT_CONF_FIRST_TOKEN = 0
SLOT_CONF_MEAN = 1
SELECT_THRESHOLD = 0
SELECT_TOP_K = 1
ACCEPT_PREFIX = 0
ACCEPT_PER_TOKEN = 1
REVEAL_CONFIDENCE = 0
REVEAL_LEFTMOST = 1
REVEAL_RANDOM = 2

# every symbol include/zarya.h declares
EXPORTS = (
    "zarya_slot_attn_workspace_size",
    "zarya_slot_attn_plan",
    "zarya_slot_attn",
    "zarya_slot_confidence_workspace_size",
    "zarya_slot_confidence",
    "zarya_slot_confidence_noalloc",
    "zarya_select_slots",
    "zarya_verify_accept",
    "zarya_kv_append",
    "zarya_slot_sample_workspace_size",
    "zarya_slot_sample",
    "zarya_mdm_budget",
    "zarya_mdm_reveal",
    "zarya_status_string",
    "zarya_last_error",
    "zarya_version",
)


class SlotAttnDesc(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("n_q_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("prefix_len", ctypes.c_int32),
        ("kv_capacity", ctypes.c_int32),
        ("n_slots", ctypes.c_int32),
        ("slot_len", ctypes.c_int32),
        ("softmax_scale", ctypes.c_float),
        ("pass_", ctypes.c_int32),
        ("cross_slot", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("prefix_splits", ctypes.c_int32),
    ]


class SlotAttnPlanInfo(ctypes.Structure):
    _fields_ = [
        ("prefix_splits", ctypes.c_int32),
        ("rows_per_workgroup", ctypes.c_int32),
        ("workgroups", ctypes.c_int32),
        ("kernels", ctypes.c_int32),
    ]


class ConfDesc(ctypes.Structure):
    _fields_ = [
        ("n_rows", ctypes.c_int32),
        ("hidden", ctypes.c_int32),
        ("vocab", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
    ]


class SampleParams(ctypes.Structure):
    _fields_ = [
        ("temperature", ctypes.c_float),
        ("seed", ctypes.c_uint64),
        ("offset", ctypes.c_uint64),
    ]


class KvAppendDesc(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("kv_capacity", ctypes.c_int32),
        ("n_slots", ctypes.c_int32),
        ("slot_len", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
    ]


class ZaryaError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{status_name(status)}: {message}")
        self.status = status


_lib = None


def lib():
    """Load libzarya.so once; raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(
                f"{LIB_PATH} is missing: build it with `python -m paper_2609_19868_amd.build` "
                "(the HIP library is the only implementation)"
            )
        L = ctypes.CDLL(LIB_PATH)
        vp, sz, i32, f32 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32, ctypes.c_float
        L.zarya_slot_attn_workspace_size.argtypes = [ctypes.POINTER(SlotAttnDesc), ctypes.POINTER(sz)]
        L.zarya_slot_attn_workspace_size.restype = ctypes.c_int
        L.zarya_slot_attn_plan.argtypes = [ctypes.POINTER(SlotAttnDesc), ctypes.POINTER(SlotAttnPlanInfo)]
        L.zarya_slot_attn_plan.restype = ctypes.c_int
        L.zarya_slot_attn.argtypes = [ctypes.POINTER(SlotAttnDesc), vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.zarya_slot_attn.restype = ctypes.c_int
        L.zarya_slot_confidence_workspace_size.argtypes = [ctypes.POINTER(ConfDesc), ctypes.POINTER(sz)]
        L.zarya_slot_confidence_workspace_size.restype = ctypes.c_int
        L.zarya_slot_confidence.argtypes = [ctypes.POINTER(ConfDesc), vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.zarya_slot_confidence.restype = ctypes.c_int
        L.zarya_slot_confidence_noalloc.argtypes = [ctypes.POINTER(ConfDesc), vp, vp, vp, vp, vp, vp, vp, vp]
        L.zarya_slot_confidence_noalloc.restype = ctypes.c_int
        L.zarya_select_slots.argtypes = [i32, i32, i32, vp, vp, i32, i32, f32, i32, vp, vp, vp, vp]
        L.zarya_select_slots.restype = ctypes.c_int
        L.zarya_verify_accept.argtypes = [i32, i32, i32, vp, vp, f32, i32, vp, vp, vp, vp]
        L.zarya_verify_accept.restype = ctypes.c_int
        L.zarya_kv_append.argtypes = [ctypes.POINTER(KvAppendDesc), vp, vp, vp, vp, vp, vp, vp, vp]
        L.zarya_kv_append.restype = ctypes.c_int
        L.zarya_slot_sample_workspace_size.argtypes = [ctypes.POINTER(ConfDesc), ctypes.POINTER(sz)]
        L.zarya_slot_sample_workspace_size.restype = ctypes.c_int
        L.zarya_slot_sample.argtypes = [ctypes.POINTER(ConfDesc), ctypes.POINTER(SampleParams), vp, vp, i32, vp, vp,
                                        vp, vp, vp, vp, sz, vp]
        L.zarya_slot_sample.restype = ctypes.c_int
        u64, ip = ctypes.c_uint64, ctypes.POINTER(i32)
        L.zarya_mdm_budget.argtypes = [i32, i32, ctypes.c_double, u64, ip, i32, ip, ip]
        L.zarya_mdm_budget.restype = ctypes.c_int
        L.zarya_mdm_reveal.argtypes = [i32, i32, vp, vp, vp, i32, u64, u64, vp, vp, vp, vp, vp]
        L.zarya_mdm_reveal.restype = ctypes.c_int
        L.zarya_status_string.argtypes = [ctypes.c_int]
        L.zarya_status_string.restype = ctypes.c_char_p
        L.zarya_last_error.argtypes = []
        L.zarya_last_error.restype = ctypes.c_char_p
        L.zarya_version.argtypes = []
        L.zarya_version.restype = i32
        _lib = L
    return _lib


def status_name(status):
    return lib().zarya_status_string(status).decode()


def check(status):
    if status != OK:
        raise ZaryaError(status, lib().zarya_last_error().decode())


def slot_attn_workspace_size(desc: SlotAttnDesc) -> int:
    n = ctypes.c_size_t(0)
    check(lib().zarya_slot_attn_workspace_size(ctypes.byref(desc), ctypes.byref(n)))
    return n.value


def slot_attn_plan(desc: SlotAttnDesc) -> dict:
    """The work decomposition zarya_slot_attn chooses for desc."""
    info = SlotAttnPlanInfo()
    check(lib().zarya_slot_attn_plan(ctypes.byref(desc), ctypes.byref(info)))
    return {name: int(getattr(info, name)) for name, _ in SlotAttnPlanInfo._fields_}


def slot_confidence_workspace_size(desc: ConfDesc) -> int:
    n = ctypes.c_size_t(0)
    check(lib().zarya_slot_confidence_workspace_size(ctypes.byref(desc), ctypes.byref(n)))
    return n.value


def slot_sample_workspace_size(desc: ConfDesc) -> int:
    n = ctypes.c_size_t(0)
    check(lib().zarya_slot_sample_workspace_size(ctypes.byref(desc), ctypes.byref(n)))
    return n.value
