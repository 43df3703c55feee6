"""Zarya slot-scoring step on MI355X: Python binding of libzarya (HIP, gfx950).

The three calls of one scoring step of slotted speculative decoding
(Zarya, Sec. 5.2):

* :func:`slot_attn`        -- slot-parallel attention against the prefix cache
* :func:`slot_confidence`  -- LM-head softmax statistics, logits kept on chip
* :func:`select_slots`     -- first-hitting slot selection

and the verification step after it (Sec. 5.2 "Verification phase", "KV cache
update"):

* :func:`verify_accept`    -- accepted tokens of the verified slots
* :func:`kv_append`        -- the accepted tokens' K/V appended to the cache

Each function marshals torch tensors (device memory) and torch's current
stream into the C ABI of ``include/zarya.h``; all arithmetic runs in the HIP
kernels.  Outputs and workspaces are allocated with torch unless passed in.
"""

from __future__ import annotations

import ctypes
import math

import torch

from . import _lib
from ._lib import (  # noqa: F401
    ACCEPT_PER_TOKEN,
    ACCEPT_PREFIX,
    CROSS_SLOT_CAUSAL,
    CROSS_SLOT_NONE,
    DTYPE_BF16,
    DTYPE_F32,
    PASS_AR_INFILL,
    PASS_DIFFUSION,
    REVEAL_CONFIDENCE,
    REVEAL_LEFTMOST,
    REVEAL_RANDOM,
    SELECT_THRESHOLD,
    SELECT_TOP_K,
    SLOT_CONF_FIRST_TOKEN,
    SLOT_CONF_MEAN,
    ZaryaError,
)

__all__ = [
    "slot_attn",
    "slot_attn_desc",
    "slot_confidence",
    "slot_sample",
    "mdm_budget",
    "mdm_reveal",
    "REVEAL_CONFIDENCE",
    "REVEAL_LEFTMOST",
    "REVEAL_RANDOM",
    "select_slots",
    "verify_accept",
    "kv_append",
    "ZaryaError",
    "ACCEPT_PREFIX",
    "ACCEPT_PER_TOKEN",
    "PASS_DIFFUSION",
    "PASS_AR_INFILL",
    "CROSS_SLOT_NONE",
    "CROSS_SLOT_CAUSAL",
    "SLOT_CONF_FIRST_TOKEN",
    "SLOT_CONF_MEAN",
    "SELECT_THRESHOLD",
    "SELECT_TOP_K",
]

_DT = {torch.bfloat16: DTYPE_BF16, torch.float32: DTYPE_F32}


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(dev):
    """The current stream of `dev` (calls run inside `torch.cuda.device(dev)`,
    so that the library launches on the tensors' device)."""
    return ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)


def _need(t, name, shape, dtype, device):
    if t.device.type != "cuda":
        raise ValueError(f"{name}: expected a cuda (HIP) device tensor, got one on {t.device}")
    if t.device != device or t.dtype != dtype or tuple(t.shape) != tuple(shape) or not t.is_contiguous():
        raise ValueError(
            f"{name}: expected contiguous {dtype} {tuple(shape)} on {device}, "
            f"got {t.dtype} {tuple(t.shape)} on {t.device} (contiguous={t.is_contiguous()})"
        )


def _need_opt(t, name, shape, dtype, device):
    if t is not None:
        _need(t, name, shape, dtype, device)


def _need_workspace(ws, n_bytes, device):
    """A caller's workspace: a contiguous 1-D uint8 device tensor of at least n_bytes."""
    if ws is None:
        return
    if ws.device.type != "cuda":
        raise ValueError(f"workspace: expected a cuda (HIP) device tensor, got one on {ws.device}")
    if ws.device != device or ws.dtype != torch.uint8 or ws.dim() != 1 or not ws.is_contiguous():
        raise ValueError(f"workspace: expected a contiguous 1-D torch.uint8 tensor on {device}, "
                         f"got {ws.dtype} {tuple(ws.shape)} on {ws.device} (contiguous={ws.is_contiguous()})")
    if ws.numel() < n_bytes:
        raise ValueError(f"workspace: {ws.numel()} bytes, {n_bytes} required")


def slot_attn_desc(q, k_cache, k_slot, n_slots, slot_len, pass_=PASS_DIFFUSION, cross_slot=CROSS_SLOT_NONE,
                   prefix_len=None, softmax_scale=None, prefix_splits=0):
    B, Hq, T, D = q.shape
    Hkv = k_slot.shape[1]
    C = 0 if k_cache is None else k_cache.shape[2]
    P = C if prefix_len is None else int(prefix_len)
    if q.dtype not in _DT:
        raise ValueError(f"unsupported dtype {q.dtype}")
    return _lib.SlotAttnDesc(
        batch=B, n_q_heads=Hq, n_kv_heads=Hkv, head_dim=D, prefix_len=P, kv_capacity=C,
        n_slots=int(n_slots), slot_len=int(slot_len),
        softmax_scale=float(1.0 / math.sqrt(D) if softmax_scale is None else softmax_scale),
        pass_=int(pass_), cross_slot=int(cross_slot), dtype=_DT[q.dtype], prefix_splits=int(prefix_splits),
    )


def slot_attn(q, k_cache, v_cache, k_slot, v_slot, n_slots, slot_len, pass_=PASS_DIFFUSION,
              cross_slot=CROSS_SLOT_NONE, slot_pass=None, prefix_len=None, softmax_scale=None,
              out=None, lse=None, want_lse=True, workspace=None, prefix_splits=0, prefix_lens=None):
    """Attention of S draft slots x L tokens against a prefix KV cache.

    q [B,Hq,T,D], k_cache/v_cache [B,Hkv,C,D] (or None when there is no
    prefix), k_slot/v_slot [B,Hkv,T,D], slot_pass [B,S] uint8 or None,
    prefix_lens [B] int32 per-row prefix lengths (each at most prefix_len,
    which defaults to C) or None.
    Returns (out [B,Hq,T,D], lse [B,Hq,T] float32 or None).
    """
    B, Hq, T, D = q.shape
    dev, dt = q.device, q.dtype
    Hkv = k_slot.shape[1]
    desc = slot_attn_desc(q, k_cache, k_slot, n_slots, slot_len, pass_, cross_slot, prefix_len, softmax_scale,
                          prefix_splits)
    _need(q, "q", (B, Hq, T, D), dt, dev)
    _need(k_slot, "k_slot", (B, Hkv, T, D), dt, dev)
    _need(v_slot, "v_slot", (B, Hkv, T, D), dt, dev)
    if k_cache is not None:
        _need(k_cache, "k_cache", (B, Hkv, desc.kv_capacity, D), dt, dev)
        _need(v_cache, "v_cache", (B, Hkv, desc.kv_capacity, D), dt, dev)
    if slot_pass is not None:
        _need(slot_pass, "slot_pass", (B, n_slots), torch.uint8, dev)
    if prefix_lens is not None:
        _need(prefix_lens, "prefix_lens", (B,), torch.int32, dev)
    if out is None:
        out = torch.empty((B, Hq, T, D), dtype=dt, device=dev)
    _need(out, "out", (B, Hq, T, D), dt, dev)
    if lse is None and want_lse:
        lse = torch.empty((B, Hq, T), dtype=torch.float32, device=dev)
    if lse is not None:
        _need(lse, "lse", (B, Hq, T), torch.float32, dev)
    ws_bytes = _lib.slot_attn_workspace_size(desc)
    _need_workspace(workspace, ws_bytes, dev)
    if workspace is None and ws_bytes > 0:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    with torch.cuda.device(dev):  # the library launches on the current device
        _lib.check(_lib.lib().zarya_slot_attn(
            ctypes.byref(desc), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(k_slot), _ptr(v_slot), _ptr(slot_pass),
            _ptr(prefix_lens), _ptr(out), _ptr(lse), _ptr(workspace), 0 if workspace is None else workspace.numel(),
            _stream(dev)))
    return out, lse


def slot_confidence(hidden, w_vocab, target_ids=None, out=None, workspace=None):
    """Per-row softmax statistics of hidden . w_vocab^T over the full vocabulary.

    hidden [M,H], w_vocab [V,H] (bf16 or float32), target_ids [M] int32 or None.
    Returns a dict with ``max_prob``, ``argmax``, ``lse`` (float32/int32 [M])
    and ``target_prob`` when target ids are given.
    """
    M, H = hidden.shape
    V = w_vocab.shape[0]
    dev, dt = hidden.device, hidden.dtype
    _need(hidden, "hidden", (M, H), dt, dev)
    _need(w_vocab, "w_vocab", (V, H), dt, dev)
    if target_ids is not None:
        _need(target_ids, "target_ids", (M,), torch.int32, dev)
    desc = _lib.ConfDesc(n_rows=M, hidden=H, vocab=V, dtype=_DT[dt])
    if out is None:
        out = {
            "max_prob": torch.empty(M, dtype=torch.float32, device=dev),
            "argmax": torch.empty(M, dtype=torch.int32, device=dev),
            "lse": torch.empty(M, dtype=torch.float32, device=dev),
        }
        if target_ids is not None:
            out["target_prob"] = torch.empty(M, dtype=torch.float32, device=dev)
    _need(out["max_prob"], "out['max_prob']", (M,), torch.float32, dev)
    _need(out["argmax"], "out['argmax']", (M,), torch.int32, dev)
    _need_opt(out.get("lse"), "out['lse']", (M,), torch.float32, dev)
    _need_opt(out.get("target_prob"), "out['target_prob']", (M,), torch.float32, dev)
    ws_bytes = _lib.slot_confidence_workspace_size(desc)
    _need_workspace(workspace, ws_bytes, dev)
    if workspace is None:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    with torch.cuda.device(dev):  # the library launches on the current device
        _lib.check(_lib.lib().zarya_slot_confidence(
            ctypes.byref(desc), _ptr(hidden), _ptr(w_vocab), _ptr(target_ids), _ptr(out["max_prob"]),
            _ptr(out["argmax"]), _ptr(out.get("lse")), _ptr(out.get("target_prob")), _ptr(workspace),
            workspace.numel(), _stream(dev)))
    return out


def slot_sample(hidden, w_vocab, temperature, seed, offset=0, rows=None, out=None, workspace=None):
    """Gumbel-max sample of every row of hidden . w_vocab^T at temperature T.

    hidden [N,H], w_vocab [V,H] (bf16 or float32); seed and offset are the
    64-bit Philox key and counter words (advance offset between draft steps).
    rows: optional int32 [M] hidden-row indices (output row i samples hidden
    row rows[i]); without it M = N.
    Returns a dict with ``sample_id`` int32 [M], ``sample_prob`` (the sampled
    token's probability at T = 1), ``max_prob`` and ``lse`` (float32 [M]).
    """
    N, H = hidden.shape
    V = w_vocab.shape[0]
    dev, dt = hidden.device, hidden.dtype
    _need(hidden, "hidden", (N, H), dt, dev)
    _need(w_vocab, "w_vocab", (V, H), dt, dev)
    M = N
    if rows is not None:
        M = rows.shape[0]
        _need(rows, "rows", (M,), torch.int32, dev)
    desc = _lib.ConfDesc(n_rows=M, hidden=H, vocab=V, dtype=_DT[dt])
    params = _lib.SampleParams(temperature=float(temperature), seed=int(seed) & (2**64 - 1),
                               offset=int(offset) & (2**64 - 1))
    if out is None:
        out = {k: torch.empty(M, dtype=torch.float32, device=dev) for k in ("sample_prob", "max_prob", "lse")}
        out["sample_id"] = torch.empty(M, dtype=torch.int32, device=dev)
    _need(out["sample_id"], "out['sample_id']", (M,), torch.int32, dev)
    _need(out["sample_prob"], "out['sample_prob']", (M,), torch.float32, dev)
    _need_opt(out.get("max_prob"), "out['max_prob']", (M,), torch.float32, dev)
    _need_opt(out.get("lse"), "out['lse']", (M,), torch.float32, dev)
    ws_bytes = _lib.slot_sample_workspace_size(desc)
    _need_workspace(workspace, ws_bytes, dev)
    if workspace is None:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    with torch.cuda.device(dev):  # the library launches on the current device
        _lib.check(_lib.lib().zarya_slot_sample(
            ctypes.byref(desc), ctypes.byref(params), _ptr(hidden), _ptr(rows), N, _ptr(w_vocab), _ptr(out["sample_id"]),
            _ptr(out["sample_prob"]), _ptr(out.get("max_prob")), _ptr(out.get("lse")), _ptr(workspace),
            workspace.numel(), _stream(dev)))
    return out


def mdm_budget(n_masked, n_steps, alpha0, seed):
    """Mode A mask budget (host): (counts per step, number of diffusion steps)."""
    L = _lib.lib()
    n, t = ctypes.c_int32(0), ctypes.c_int32(0)
    args = (int(n_masked), int(n_steps), float(alpha0), int(seed) & (2**64 - 1))
    _lib.check(L.zarya_mdm_budget(*args, None, 0, ctypes.byref(n), ctypes.byref(t)))
    counts = (ctypes.c_int32 * max(1, n.value))()
    _lib.check(L.zarya_mdm_budget(*args, counts, n.value, ctypes.byref(n), ctypes.byref(t)))
    return [int(c) for c in counts[: n.value]], t.value


def mdm_reveal(mask, k, rule=REVEAL_CONFIDENCE, conf=None, seed=0, offset=0, sample_id=None, tokens=None,
               out=None):
    """Reveal positions of a Mode A step.

    mask [B,N] uint8 (nonzero = masked; cleared where revealed, in place),
    k [B] int32, conf [B,N] float32 (confidence rule), sample_id / tokens
    [B,N] int32 (optional pair; tokens updated in place).
    Returns (order [B,N] int32: revealed positions then -1, n_revealed [B] int32).
    """
    B, N = mask.shape
    dev = mask.device
    _need(mask, "mask", (B, N), torch.uint8, dev)
    _need(k, "k", (B,), torch.int32, dev)
    if conf is not None:
        _need(conf, "conf", (B, N), torch.float32, dev)
    if sample_id is not None:
        _need(sample_id, "sample_id", (B, N), torch.int32, dev)
    if tokens is not None:
        _need(tokens, "tokens", (B, N), torch.int32, dev)
    if out is None:
        out = (torch.empty((B, N), dtype=torch.int32, device=dev), torch.empty((B,), dtype=torch.int32, device=dev))
    order, n = out
    _need(order, "out[0] (order)", (B, N), torch.int32, dev)
    _need_opt(n, "out[1] (n_revealed)", (B,), torch.int32, dev)
    with torch.cuda.device(dev):  # the library launches on the current device
        _lib.check(_lib.lib().zarya_mdm_reveal(
            B, N, _ptr(conf), _ptr(mask), _ptr(k), int(rule), int(seed) & (2**64 - 1), int(offset) & (2**64 - 1),
            _ptr(sample_id), _ptr(tokens), _ptr(order), _ptr(n), _stream(dev)))
    return order, n


def select_slots(token_conf, slot_open=None, conf_rule=SLOT_CONF_FIRST_TOKEN, rule=SELECT_THRESHOLD,
                 threshold=0.9, k=1, out=None):
    """First-hitting slot selection from per-token confidences [B,S,L] float32.

    Returns (slot_conf [B,S] float32, selected [B,S] int32, n_selected [B] int32).
    """
    B, S, L = token_conf.shape
    dev = token_conf.device
    _need(token_conf, "token_conf", (B, S, L), torch.float32, dev)
    if slot_open is not None:
        _need(slot_open, "slot_open", (B, S), torch.uint8, dev)
    if out is None:
        out = (
            torch.empty((B, S), dtype=torch.float32, device=dev),
            torch.empty((B, S), dtype=torch.int32, device=dev),
            torch.empty((B,), dtype=torch.int32, device=dev),
        )
    slot_conf, selected, n_selected = out
    _need(slot_conf, "out[0] (slot_conf)", (B, S), torch.float32, dev)
    _need(selected, "out[1] (selected)", (B, S), torch.int32, dev)
    _need(n_selected, "out[2] (n_selected)", (B,), torch.int32, dev)
    with torch.cuda.device(dev):  # the library launches on the current device
        _lib.check(_lib.lib().zarya_select_slots(
            B, S, L, _ptr(token_conf), _ptr(slot_open), int(conf_rule), int(rule), float(threshold), int(k),
            _ptr(slot_conf), _ptr(selected), _ptr(n_selected), _stream(dev)))
    return slot_conf, selected, n_selected


def verify_accept(token_prob, selected, token_threshold=0.4, rule=ACCEPT_PREFIX, out=None):
    """Accepted draft tokens of the verified slots.

    token_prob [B,S,L] float32 (probability of each draft token under the
    verification pass), selected [B,S] int32 (verified slots, the first -1
    ends the list).  Returns (accepted [B,S,L] uint8, n_accepted [B,S] int32,
    n_total [B] int32).
    """
    B, S, L = token_prob.shape
    dev = token_prob.device
    _need(token_prob, "token_prob", (B, S, L), torch.float32, dev)
    _need(selected, "selected", (B, S), torch.int32, dev)
    if out is None:
        out = (
            torch.empty((B, S, L), dtype=torch.uint8, device=dev),
            torch.empty((B, S), dtype=torch.int32, device=dev),
            torch.empty((B,), dtype=torch.int32, device=dev),
        )
    accepted, n_accepted, n_total = out
    _need(accepted, "out[0] (accepted)", (B, S, L), torch.uint8, dev)
    _need(n_accepted, "out[1] (n_accepted)", (B, S), torch.int32, dev)
    _need_opt(n_total, "out[2] (n_total)", (B,), torch.int32, dev)
    with torch.cuda.device(dev):  # the library launches on the current device
        _lib.check(_lib.lib().zarya_verify_accept(
            B, S, L, _ptr(token_prob), _ptr(selected), float(token_threshold), int(rule), _ptr(accepted),
            _ptr(n_accepted), _ptr(n_total), _stream(dev)))
    return accepted, n_accepted, n_total


def kv_append(k_cache, v_cache, prefix_lens, k_slot, v_slot, accepted, order):
    """Append the accepted draft tokens' K/V after each row's prefix, in place.

    k_cache/v_cache [B,Hkv,C,D] (updated), prefix_lens [B] int32 (updated),
    k_slot/v_slot [B,Hkv,S*L,D], accepted [B,S,L] uint8, order [B,S] int32
    (slots in append order, the first -1 ends it).
    """
    B, Hkv, C, D = k_cache.shape
    _, S, L = accepted.shape
    dev, dt = k_cache.device, k_cache.dtype
    _need(k_cache, "k_cache", (B, Hkv, C, D), dt, dev)
    _need(v_cache, "v_cache", (B, Hkv, C, D), dt, dev)
    _need(k_slot, "k_slot", (B, Hkv, S * L, D), dt, dev)
    _need(v_slot, "v_slot", (B, Hkv, S * L, D), dt, dev)
    _need(accepted, "accepted", (B, S, L), torch.uint8, dev)
    _need(order, "order", (B, S), torch.int32, dev)
    _need(prefix_lens, "prefix_lens", (B,), torch.int32, dev)
    desc = _lib.KvAppendDesc(batch=B, n_kv_heads=Hkv, head_dim=D, kv_capacity=C, n_slots=S, slot_len=L,
                             dtype=_DT[dt])
    with torch.cuda.device(dev):  # the library launches on the current device
        _lib.check(_lib.lib().zarya_kv_append(
            ctypes.byref(desc), _ptr(k_slot), _ptr(v_slot), _ptr(accepted), _ptr(order), _ptr(prefix_lens),
            _ptr(k_cache), _ptr(v_cache), _stream(dev)))
    return k_cache, v_cache, prefix_lens
