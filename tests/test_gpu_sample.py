"""zarya_slot_sample on the GPU (through the C ABI) against the float64 oracle.

The sampled id is a decision taken on float32 perturbed scores (kernel) and
float64 ones (oracle), so ids must agree exactly wherever the oracle's top-2
gap of the perturbed scores z/T + G is >= g = 1e-3 / min(T, 1) (the logit
error is divided by T); elsewhere the GPU's id must be a valid near-winner:
its oracle score within g of the best.  Both
sides draw the same Philox uniforms (integer work, exact), so the noise
itself is not a source of disagreement.  sample_prob, max_prob and lse carry
the tolerances of the greedy reduction (1e-3; float32 path 1e-4).
"""

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_helpers import oracle_confidence_by_block, oracle_sample_by_block, require_gpu, say, to_dev

import paper_2609_19868_amd as Z

pytestmark = pytest.mark.gpu

SEED, OFFSET = 0x1234_5678_9ABC_DEF0, 0x0000_0003_0000_0011


def _planted(M, V, n, seed):
    rng = np.random.default_rng(seed)
    rows = rng.choice(M, size=min(n, M), replace=False)
    return rows, rng.integers(0, V, size=len(rows)), rng.uniform(0.0, 120.0, size=len(rows))


def _check(res, hf, wf, T, seed, offset, rows, f32, what, row_ids=None, parallel=False):
    """Compare the GPU results of `rows` with the oracle on the same rows
    (`row_ids`: the rows' indices in the random stream, default `rows`);
    `parallel` runs the oracle on blocks of rows side by side."""
    row_ids = rows if row_ids is None else row_ids
    if parallel:
        ref = oracle_sample_by_block(hf, wf, T, seed, offset, row_ids=row_ids)
        conf = oracle_confidence_by_block(hf, wf)
    else:
        ref = oracle.slot_sample(hf, wf, T, seed, offset, row_ids=row_ids)
        conf = oracle.slot_confidence(hf, wf)
    tol = 1e-4 if f32 else 1e-3
    sid = res["sample_id"].cpu().numpy()[rows].astype(np.int64)
    sp = res["sample_prob"].cpu().numpy().astype(np.float64)[rows]
    mp = res["max_prob"].cpu().numpy().astype(np.float64)[rows]
    lse = res["lse"].cpu().numpy().astype(np.float64)[rows]
    V = wf.shape[0]
    assert np.all((sid >= 0) & (sid < V)), f"{what}: sampled id out of range"
    gap_tol = 1e-3 / min(T, 1.0)
    decided = ref["score_gap"] >= gap_tol
    mism = decided & (sid != ref["sample_id"])
    assert not mism.any(), f"{what}: {mism.sum()} of {decided.sum()} decided rows sampled a different id"
    for i in np.flatnonzero(~decided):  # near-ties: the GPU's pick must be a near-winner
        u = oracle.uniforms([row_ids[i]], V, seed, offset)[0, sid[i]]
        score = float(hf[i] @ wf[sid[i]]) / T + float(oracle.gumbel(u))
        assert ref["best_score"][i] - score <= gap_tol, f"{what}: row {rows[i]} id {sid[i]} is not a near-winner"
    # probability of the id the GPU drew, from the oracle's logits
    z_pick = np.einsum("ih,ih->i", hf, wf[sid])
    p_ref = np.exp(z_pick - ref["lse"])
    e = np.abs(sp - p_ref)
    assert np.all(e <= tol * p_ref + 1e-12), f"{what}: sample_prob rel err {(e / p_ref).max():.3e}"
    assert np.abs(lse - ref["lse"]).max() <= tol, f"{what}: lse err"
    e_mp = np.abs(mp - conf["max_prob"])
    assert np.all(e_mp <= tol * conf["max_prob"] + 1e-7), f"{what}: max_prob err {e_mp.max():.3e}"
    return int((~decided).sum()), ref, conf


def _run(wl, dev, T, rows=None, plant=None, what="", seed=SEED, offset=OFFSET, parallel=False):
    c = W.confidence_inputs(wl, plant=plant)
    hd, wd = to_dev(c["hidden"], wl.dtype, dev), to_dev(c["w_vocab"], wl.dtype, dev)
    say(f"slot_sample {what} T={T}")
    res = Z.slot_sample(hd, wd, T, seed, offset)
    torch.cuda.synchronize()
    rows = np.arange(hd.shape[0]) if rows is None else np.asarray(rows)
    hf = W.as_f64(c["hidden"][rows], wl.dtype)
    wf = W.as_f64(c["w_vocab"], wl.dtype)
    say(f"slot_sample {what} T={T}: oracle")
    n_near, ref, conf = _check(res, hf, wf, T, seed, offset, rows, wl.dtype == "f32", what, parallel=parallel)
    return res, ref, conf, n_near


def test_tiny_fp32():
    dev = require_gpu()
    wl = W.WORKLOADS["tiny"]
    for T in (1.0, 0.5):
        _run(wl, dev, T, plant=_planted(wl.M, wl.vocab, 6, 1), what="tiny f32")


SMALL = [
    ("m300_v5000_h256", dict(batch=1, n_slots=60, slot_len=5, hidden=256, vocab=5000)),
    ("m40_v2049_h136", dict(batch=1, n_slots=8, slot_len=5, hidden=136, vocab=2049)),
    ("m1_v100_h64", dict(batch=1, n_slots=1, slot_len=1, hidden=64, vocab=100)),
    ("m513_v33000_h1024", dict(batch=1, n_slots=27, slot_len=19, hidden=1024, vocab=33000)),
    ("m128_v7001_h512", dict(batch=1, n_slots=16, slot_len=8, hidden=512, vocab=7001)),  # largest 64-row-tile case
    ("m129_v7001_h512", dict(batch=1, n_slots=43, slot_len=3, hidden=512, vocab=7001)),  # smallest 256-row-tile case
    ("m3_v1_h8", dict(batch=1, n_slots=3, slot_len=1, hidden=8, vocab=1)),  # a one-token vocabulary
    # 256-row tile with a partial last k-stage (200 = 3*64 + 8) and last vocab tiles of a few rows
    ("m260_v3001_h200", dict(batch=1, n_slots=52, slot_len=5, hidden=200, vocab=3001)),
    ("m257_v257_h72", dict(batch=1, n_slots=257, slot_len=1, hidden=72, vocab=257)),
]


@pytest.mark.parametrize("T", [1.0, 0.7, 25.0], ids=["T1", "T0.7", "T25"])
@pytest.mark.parametrize("name,over", SMALL, ids=[s[0] for s in SMALL])
def test_bf16_small_shapes(name, over, T):
    dev = require_gpu()
    wl = W.WORKLOADS["qwen0.6b"].replace(**over, seed=93)
    _, ref, _, _ = _run(wl, dev, T, plant=_planted(wl.M, wl.vocab, wl.M // 3 + 1, 2), what=name)
    if wl.M >= 20 and T == 1.0:
        assert ref["sample_prob"].max() > 0.9 and ref["sample_prob"].min() < 0.01, "planted rows should span (0, 1)"


def test_cold_limit_is_the_argmax():
    """(z1 - z2) / T beyond the whole range of the Gumbel noise (< 19.5 for
    these uniforms): the draw must be the greedy argmax."""
    dev = require_gpu()
    wl = W.WORKLOADS["qwen0.6b"].replace(batch=1, n_slots=64, slot_len=4, hidden=512, vocab=7000, seed=94)
    T = 1e-3
    res, ref, conf, _ = _run(wl, dev, T, plant=_planted(wl.M, wl.vocab, 64, 5), what="cold")
    clear = conf["top2_gap"] / T > 20.0
    assert clear.sum() > wl.M // 2
    assert np.array_equal(res["sample_id"].cpu().numpy()[clear], conf["argmax"][clear])


def test_stream_is_deterministic_and_keyed():
    dev = require_gpu()
    wl = W.WORKLOADS["qwen0.6b"].replace(batch=1, n_slots=64, slot_len=5, hidden=512, vocab=20000, seed=95)
    c = W.confidence_inputs(wl)
    hd, wd = to_dev(c["hidden"], "bf16", dev), to_dev(c["w_vocab"], "bf16", dev)
    a = Z.slot_sample(hd, wd, 1.0, SEED, OFFSET)
    b = Z.slot_sample(hd, wd, 1.0, SEED, OFFSET)
    o = Z.slot_sample(hd, wd, 1.0, SEED, OFFSET + 1)
    s = Z.slot_sample(hd, wd, 1.0, SEED + (1 << 32), OFFSET)
    torch.cuda.synchronize()
    for k in ("sample_id", "sample_prob", "max_prob", "lse"):
        assert torch.equal(a[k], b[k]), k
    # near-flat logits: a fresh stream changes almost every draw
    assert (a["sample_id"] != o["sample_id"]).float().mean().item() > 0.9
    assert (a["sample_id"] != s["sample_id"]).float().mean().item() > 0.9
    assert torch.equal(a["max_prob"], o["max_prob"]) and torch.equal(a["lse"], o["lse"])


def test_draws_follow_the_tempered_softmax():
    """Many rows with the same hidden state: the ids' frequencies must match
    softmax(z / T) (chi-square, 31 degrees of freedom, 1e-4 tail)."""
    dev = require_gpu()
    rng = np.random.default_rng(96)
    V, H, M, T = 32, 64, 60000, 0.8
    w = W.bf16_bits(rng.standard_normal((V, H)).astype(np.float32) * 0.2)
    h = np.repeat(W.bf16_bits(rng.standard_normal((1, H)).astype(np.float32)), M, axis=0)
    res = Z.slot_sample(to_dev(h, "bf16", dev), to_dev(w, "bf16", dev), T, 7, 0)
    torch.cuda.synchronize()
    z = W.as_f64(w, "bf16") @ W.as_f64(h[0], "bf16")
    p = np.exp((z - z.max()) / T)
    p /= p.sum()
    counts = np.bincount(res["sample_id"].cpu().numpy(), minlength=V)
    chi2 = float(((counts - M * p) ** 2 / (M * p)).sum())
    assert chi2 < 70.0, chi2  # P(chi2_31 > 70) < 1e-4
    zs = z[res["sample_id"].cpu().numpy()]
    sp = res["sample_prob"].cpu().numpy()
    lse = z.max() + np.log(np.exp(z - z.max()).sum())
    assert np.allclose(sp, np.exp(zs - lse), rtol=1e-3)


@pytest.mark.parametrize("name", ["qwen0.6b", "qwen1.7b", "qwen4b"])
def test_full_size_every_row(name):
    """Full vocabulary and row count in the benchmark's launch configuration:
    every row against the oracle (every vocab entry of each)."""
    dev = require_gpu()
    wl = W.WORKLOADS[name]
    plant = _planted(wl.M, wl.vocab, 64, 4)
    say(f"slot_sample full {name}: generating inputs")
    _run(wl, dev, 1.0, plant=plant, what=f"full {name}", parallel=True)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_row_selection(dtype):
    """Output row i samples hidden row rows[i] (duplicates allowed) with the
    stream of output row i; indices outside the hidden rows give -1 / NaN."""
    dev = require_gpu()
    base = W.WORKLOADS["qwen0.6b"] if dtype == "bf16" else W.WORKLOADS["tiny"]
    wl = base.replace(batch=1, n_slots=60, slot_len=5, hidden=256 if dtype == "bf16" else 128,
                      vocab=33000 if dtype == "bf16" else 700, seed=97)
    c = W.confidence_inputs(wl, plant=_planted(wl.M, wl.vocab, 40, 6))
    N = wl.M
    rng = np.random.default_rng(98)
    rows = rng.integers(0, N, 130).astype(np.int32)
    rows[[3, 77]] = rows[5]  # duplicates
    rows[10], rows[100] = -1, N  # out of range
    hd, wd = to_dev(c["hidden"], dtype, dev), to_dev(c["w_vocab"], dtype, dev)
    say(f"slot_sample row selection {dtype} N={N} M={rows.size}")
    res = Z.slot_sample(hd, wd, 0.8, SEED, OFFSET, rows=torch.from_numpy(rows).to(dev))
    torch.cuda.synchronize()
    bad = (rows < 0) | (rows >= N)
    sid = res["sample_id"].cpu().numpy()
    assert np.all(sid[bad] == -1)
    for k in ("sample_prob", "max_prob", "lse"):
        assert np.all(np.isnan(res[k].cpu().numpy()[bad])), k
    ok = np.flatnonzero(~bad)
    hf = W.as_f64(c["hidden"][rows[ok]], dtype)
    wf = W.as_f64(c["w_vocab"], dtype)
    # the oracle on the selected hidden rows, each with its output row's stream
    sub = {k: v[torch.from_numpy(ok).to(dev)] for k, v in res.items()}
    _check(sub, hf, wf, 0.8, SEED, OFFSET, np.arange(ok.size), dtype == "f32", f"row selection {dtype}",
           row_ids=ok)
