"""Shared helpers of the GPU tests: device transfer and tolerance checks."""

from __future__ import annotations

import sys

import numpy as np
import torch

import workloads as W


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
