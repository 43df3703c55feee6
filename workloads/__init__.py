"""Seeded synthetic inputs for the slot-scoring step.

This module only draws random numbers and rounds them to the storage dtype.
It holds none of the method's arithmetic, and it is the one module both the
HIP path's callers (tests, benchmark) and the oracle's callers share.

Workloads (shapes from Table 1 of the paper for heads and hidden size; head
dim 128, vocab 151936 and the slot shapes are workload choices):

  tiny      fp32  B=1  Hq/Hkv=2/1   D=64  P=64    S=4  L=4   H=128  V=512
  qwen0.6b  bf16  B=16 Hq/Hkv=16/8  D=128 P=2048  S=8  L=8   H=1024 V=151936
  qwen1.7b  bf16  B=32 Hq/Hkv=16/8  D=128 P=4096  S=16 L=4   H=2048 V=151936
  qwen4b    bf16  B=8  Hq/Hkv=32/8  D=128 P=16384 S=8  L=16  H=2560 V=151936
  layout    bf16  B=8  Hq/Hkv=16/8  D=128 P=0     S=128 L=32 (training layout)
  modeA     bf16  B=16 Hq/Hkv=16/8  D=128 P=2048  S=260 L=1  H=1024 V=151936
            (a Mode A denoising step: the 4 tokens revealed at the previous
            step and the 256 still masked, one causal run after the prompt;
            the LM head runs on the 256 masked rows of each batch row)

Distributions: Q, K, V ~ N(0, 1); hidden ~ N(0, 1); W ~ N(0, 0.02^2).  Values
are drawn in float32 and, for bf16 workloads, rounded to bfloat16 with
round-to-nearest-even; the same bits go to the GPU and (upcast) to the oracle.
Draw order from ``numpy.random.default_rng(seed)``: Q, K_cache, V_cache,
K_slot, V_slot, hidden, then W in 8192-row chunks.  The training layout uses
the child generator ``default_rng((seed, 1))``.
"""

from __future__ import annotations

import dataclasses
import math

import numpy as np

W_CHUNK_ROWS = 8192


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    dtype: str  # "f32" or "bf16"
    batch: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    prefix_len: int
    n_slots: int
    slot_len: int
    hidden: int
    vocab: int
    kv_capacity: int = 0  # 0: equal to prefix_len
    seed: int = 1000

    @property
    def T(self):
        return self.n_slots * self.slot_len

    @property
    def M(self):
        return self.batch * self.T

    @property
    def capacity(self):
        return self.kv_capacity if self.kv_capacity else self.prefix_len

    @property
    def scale(self):
        return 1.0 / math.sqrt(self.head_dim)

    def replace(self, **kw):
        return dataclasses.replace(self, **kw)


WORKLOADS = {
    "tiny": Workload("tiny", "f32", 1, 2, 1, 64, 64, 4, 4, 128, 512, seed=1000),
    "qwen0.6b": Workload("qwen0.6b", "bf16", 16, 16, 8, 128, 2048, 8, 8, 1024, 151936, seed=1001),
    "qwen1.7b": Workload("qwen1.7b", "bf16", 32, 16, 8, 128, 4096, 16, 4, 2048, 151936, seed=1002),
    "qwen4b": Workload("qwen4b", "bf16", 8, 32, 8, 128, 16384, 8, 16, 2560, 151936, seed=1003),
    "layout": Workload("layout", "bf16", 8, 16, 8, 128, 0, 128, 32, 0, 0, seed=1004),
    "modeA": Workload("modeA", "bf16", 16, 16, 8, 128, 2048, 260, 1, 1024, 151936, seed=1005),
}
WORKLOAD_ORDER = ["tiny", "qwen0.6b", "qwen1.7b", "qwen4b", "layout", "modeA"]
MODE_A_REVEALED = 4  # rows of the modeA step revealed at the previous step


def bf16_bits(x):
    """float32 array -> uint16 bfloat16 bits, round to nearest even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def bf16_to_f32(bits):
    """uint16 bfloat16 bits -> float32 (exact)."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def _draw(rng, shape, std, dtype):
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return bf16_bits(x) if dtype == "bf16" else x


def attention_inputs(wl: Workload, rng=None, q_scale=1.0):
    """Q [B,Hq,T,D], K/V cache [B,Hkv,C,D], K/V slot [B,Hkv,T,D].

    Returns float32 arrays for f32 workloads, uint16 bf16 bits otherwise.
    ``q_scale`` > 1 sharpens the attention ("peaked" test inputs).
    Cache rows at or beyond ``prefix_len`` (capacity slack) are drawn too.
    """
    rng = np.random.default_rng(wl.seed) if rng is None else rng
    B, Hq, Hkv, D, T, C = wl.batch, wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.T, wl.capacity
    q = rng.standard_normal(size=(B, Hq, T, D), dtype=np.float32)
    if q_scale != 1.0:
        q *= np.float32(q_scale)
    q = bf16_bits(q) if wl.dtype == "bf16" else q
    k_cache = _draw(rng, (B, Hkv, C, D), 1.0, wl.dtype)
    v_cache = _draw(rng, (B, Hkv, C, D), 1.0, wl.dtype)
    k_slot = _draw(rng, (B, Hkv, T, D), 1.0, wl.dtype)
    v_slot = _draw(rng, (B, Hkv, T, D), 1.0, wl.dtype)
    return {"q": q, "k_cache": k_cache, "v_cache": v_cache, "k_slot": k_slot, "v_slot": v_slot}


def confidence_inputs(wl: Workload, rng=None, n_rows=None, plant=None):
    """hidden [M,H] ~ N(0,1), W [V,H] ~ N(0, 0.02^2), target ids [M].

    ``plant`` = (row_ids, vocab_ids, alphas): those hidden rows become
    alpha * W[v] / |W[v]| so that v is their argmax with a chosen margin.
    """
    rng = np.random.default_rng(wl.seed + 7_000_000) if rng is None else rng
    M = wl.M if n_rows is None else n_rows
    H, V = wl.hidden, wl.vocab
    h = rng.standard_normal(size=(M, H), dtype=np.float32)
    w = np.empty((V, H), dtype=np.uint16 if wl.dtype == "bf16" else np.float32)
    for r0 in range(0, V, W_CHUNK_ROWS):
        r1 = min(V, r0 + W_CHUNK_ROWS)
        w[r0:r1] = _draw(rng, (r1 - r0, H), 0.02, wl.dtype)
    target = rng.integers(0, V, size=M, dtype=np.int64).astype(np.int32)
    if plant is not None:
        rows, vids, alphas = plant
        wf = bf16_to_f32(w) if wl.dtype == "bf16" else w
        for r, v, a in zip(rows, vids, alphas):
            vec = wf[v].astype(np.float64)
            h[r] = (a * vec / np.linalg.norm(vec)).astype(np.float32)
    h = bf16_bits(h) if wl.dtype == "bf16" else h
    return {"hidden": h, "w_vocab": w, "target_ids": target}


def training_layout(wl: Workload, seed=None):
    """Reordered training layout of the paper's Sec. 1 / Sec. 4.1 recipe.

    Each of the S slots of each batch row is masked with probability 1/2
    (independently); the physical order puts the clean slots first and the
    masked slots after them, each group in a random order.
    Returns (order [B,S] original slot id at each physical position,
    masked_phys [B,S] bool: is the slot at this physical position masked).
    """
    seed = wl.seed if seed is None else seed
    rng = np.random.default_rng((seed, 1))
    B, S = wl.batch, wl.n_slots
    order = np.empty((B, S), dtype=np.int64)
    masked_phys = np.empty((B, S), dtype=bool)
    for b in range(B):
        masked = rng.random(S) < 0.5
        clean_ids = np.flatnonzero(~masked)
        masked_ids = np.flatnonzero(masked)
        clean_perm = rng.permutation(clean_ids)
        masked_perm = rng.permutation(masked_ids)
        order[b] = np.concatenate([clean_perm, masked_perm])
        masked_phys[b] = np.concatenate([np.zeros(len(clean_perm), bool), np.ones(len(masked_perm), bool)])
    return order, masked_phys


def as_f64(x, dtype):
    """Storage array (float32 or bf16 bits) -> float64 values."""
    if dtype == "bf16":
        return bf16_to_f32(x).astype(np.float64)
    return np.asarray(x, dtype=np.float64)
