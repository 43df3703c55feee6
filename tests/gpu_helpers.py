"""Shared helpers of the GPU tests: device transfer and tolerance checks."""

from __future__ import annotations

import sys

import numpy as np
import torch

import workloads as W


def run_parallel(fn, items, workers=8):
    """fn over items on a thread pool, results in order.  The oracle's numpy
    work (BLAS products, ufuncs over large arrays) releases the GIL, so
    independent batch rows or row blocks run side by side; BLAS is held to
    two threads per worker meanwhile."""
    from concurrent.futures import ThreadPoolExecutor

    from threadpoolctl import threadpool_limits

    with threadpool_limits(limits=2):
        with ThreadPoolExecutor(max_workers=workers) as ex:
            return list(ex.map(fn, items))


def oracle_attention_by_row(xf, prefix_len, n_slots, slot_len, scale, pass_, cross=0, slot_pass=None):
    """oracle.slot_attention over every batch row, one row per task (the
    oracle treats batch rows independently)."""
    import oracle

    B = xf["q"].shape[0]
    plens = np.broadcast_to(np.asarray(prefix_len), (B,))

    def one(b):
        return oracle.slot_attention(xf["q"][b:b + 1], xf["k_cache"][b:b + 1], xf["v_cache"][b:b + 1],
                                     xf["k_slot"][b:b + 1], xf["v_slot"][b:b + 1], [int(plens[b])], n_slots,
                                     slot_len, scale, pass_, cross_slot=cross,
                                     slot_pass=None if slot_pass is None else slot_pass[b:b + 1])

    res = run_parallel(one, range(B))
    return np.concatenate([r[0] for r in res]), np.concatenate([r[1] for r in res])


def _by_blocks(fn, M, block=128):
    blocks = [(r0, min(M, r0 + block)) for r0 in range(0, M, block)]
    parts = run_parallel(fn, blocks)
    return {k: np.concatenate([p[k] for p in parts]) for k in parts[0]}


def oracle_confidence_by_block(hf, wf, target_ids=None):
    """oracle.slot_confidence over every row, blocks of rows side by side (the
    oracle treats rows independently)."""
    import oracle

    return _by_blocks(lambda r: oracle.slot_confidence(
        hf[r[0]:r[1]], wf, target_ids=None if target_ids is None else target_ids[r[0]:r[1]]), hf.shape[0])


def oracle_sample_by_block(hf, wf, T, seed, offset, row_ids=None):
    """oracle.slot_sample over every row, blocks of rows side by side; each
    row keeps its own index in the random stream."""
    import oracle

    ids = np.arange(hf.shape[0]) if row_ids is None else np.asarray(row_ids)
    return _by_blocks(lambda r: oracle.slot_sample(hf[r[0]:r[1]], wf, T, seed, offset, row_ids=ids[r[0]:r[1]]),
                      hf.shape[0])


_FULL_CACHE = {}


def full_attention_inputs(wl, dev):
    """(storage arrays, device tensors, float64 arrays) of a workload's
    attention inputs; the last workload drawn is kept, so the tests of its two
    passes draw it once."""
    key = (wl, str(dev))
    if key not in _FULL_CACHE:
        _FULL_CACHE.clear()
        x = W.attention_inputs(wl)
        xd = {k: to_dev(v, wl.dtype, dev) for k, v in x.items()}
        xf = {k: W.as_f64(v, wl.dtype) for k, v in x.items()}
        _FULL_CACHE[key] = (x, xd, xf)
    return _FULL_CACHE[key]


def require_gpu():
    if not torch.cuda.is_available():
        raise RuntimeError("this test needs an MI355X (HIP device); run the CPU suite with -m 'not gpu'")
    return torch.device("cuda:0")


def say(msg):
    """Name the case before each GPU step, flushed, so a crash still reports it."""
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


def to_dev(x, dtype, dev):
    """Storage array (float32, or uint16 bf16 bits) -> device tensor."""
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).to(dev)
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(dev)


def to_f64(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def attn_inputs_dev(wl, dev, q_scale=1.0, rng=None):
    x = W.attention_inputs(wl, rng=rng, q_scale=q_scale)
    xd = {k: to_dev(v, wl.dtype, dev) for k, v in x.items()}
    xf = {k: W.as_f64(v, wl.dtype) for k, v in x.items()}
    return xd, xf


def check_attn(O_gpu, lse_gpu, O_ref, lse_ref, dtype, what=""):
    """Elementwise, per-(b,h) relative-L2 and LSE checks (bounds in the test docstrings)."""
    O_gpu = np.asarray(O_gpu, np.float64)
    err = np.abs(O_gpu - O_ref)
    if dtype == "bf16":
        bound = 2e-2 + 1e-2 * np.abs(O_ref)
        lse_tol = 1e-3
        rel_l2_tol = 1e-2
    else:
        bound = 1e-4 + 1e-4 * np.abs(O_ref)
        lse_tol = 1e-4
        rel_l2_tol = 1e-4
    bad = err > bound
    assert not bad.any(), f"{what}: {bad.sum()} elements out of tolerance, max err {err.max():.3e}"
    axes = tuple(range(2, O_ref.ndim))
    rel = np.sqrt((err ** 2).sum(axis=axes)) / np.maximum(np.sqrt((O_ref ** 2).sum(axis=axes)), 1e-30)
    assert rel.max() <= rel_l2_tol, f"{what}: relative L2 {rel.max():.3e} > {rel_l2_tol}"
    if lse_gpu is not None:
        le = np.abs(np.asarray(lse_gpu, np.float64) - lse_ref)
        assert le.max() <= lse_tol, f"{what}: LSE err {le.max():.3e} > {lse_tol}"
    return float(rel.max())


def check_conf(res_gpu, ref, rows=None, what="", f32=False, logit_of=None):
    """max_prob abs and relative, lse abs, argmax exact unless the top-2 gap is tiny."""
    sel = slice(None) if rows is None else rows
    mp = res_gpu["max_prob"].cpu().numpy().astype(np.float64)[sel]
    lse = res_gpu["lse"].cpu().numpy().astype(np.float64)[sel]
    am = res_gpu["argmax"].cpu().numpy()[sel]
    tol = 1e-4 if f32 else 1e-3
    e_mp = np.abs(mp - ref["max_prob"])
    assert e_mp.max() <= tol, f"{what}: max_prob abs err {e_mp.max():.3e}"
    assert np.all(e_mp <= tol * ref["max_prob"] + 1e-7), f"{what}: max_prob rel err {(e_mp / ref['max_prob']).max():.3e}"
    e_lse = np.abs(lse - ref["lse"])
    assert e_lse.max() <= tol, f"{what}: lse err {e_lse.max():.3e}"
    decided = ref["top2_gap"] >= 1e-3
    mism = (am != ref["argmax"]) & decided
    assert not mism.any(), f"{what}: {mism.sum()} argmax mismatches on rows with a clear maximum"
    if logit_of is not None:
        # rows without a clear maximum: the GPU's id must be one of the near-maximal ids
        for i in np.flatnonzero(~decided):
            z = logit_of(i, int(am[i]))
            assert ref["max_logit"][i] - z <= 1e-3, f"{what}: row {i} argmax {am[i]} is not near-maximal"
    if "target_prob" in ref:
        tp = res_gpu["target_prob"].cpu().numpy().astype(np.float64)[sel]
        e_tp = np.abs(tp - ref["target_prob"])
        assert np.all(e_tp <= tol * ref["target_prob"] + 1e-12), f"{what}: target_prob rel err {(e_tp / ref['target_prob']).max():.3e}"
    return int((~decided).sum())
