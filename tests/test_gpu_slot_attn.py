"""slot_attn on the GPU (through the C ABI) against the float64 oracle.

Tolerances: bf16 outputs |diff| <= 2e-2 + 1e-2*|ref| elementwise, relative L2
per (batch, head) <= 1e-2 (the bf16 rounding of P and of O gives ~3e-3), LSE
|diff| <= 1e-3; float32 path: 1e-4 + 1e-4*|ref| and LSE 1e-4.  Inputs are the
seeded workloads (bf16 bits shared by both sides), also with queries scaled by
4 ("peaked") so that the softmax is far from uniform.
"""

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_helpers import (attn_inputs_dev, check_attn, full_attention_inputs, oracle_attention_by_row, require_gpu,
                         say, to_dev, to_f64)

import paper_2609_19868_amd as Z

pytestmark = pytest.mark.gpu

PASSES = [(Z.PASS_DIFFUSION, "diffusion"), (Z.PASS_AR_INFILL, "ar_infill")]


def _run(xd, wl, pass_, cross=Z.CROSS_SLOT_NONE, slot_pass=None, splits=0):
    out, lse = Z.slot_attn(xd["q"], xd["k_cache"] if wl.capacity else None, xd["v_cache"] if wl.capacity else None,
                           xd["k_slot"], xd["v_slot"], wl.n_slots, wl.slot_len, pass_=pass_, cross_slot=cross,
                           slot_pass=slot_pass, prefix_len=wl.prefix_len, softmax_scale=wl.scale,
                           prefix_splits=splits)
    torch.cuda.synchronize()
    return out, lse


def _oracle(xf, wl, pass_, cross=oracle.CROSS_SLOT_NONE, slot_pass=None):
    return oracle.slot_attention(xf["q"], xf["k_cache"], xf["v_cache"], xf["k_slot"], xf["v_slot"], wl.prefix_len,
                                 wl.n_slots, wl.slot_len, wl.scale, pass_, cross_slot=cross, slot_pass=slot_pass)


def test_tiny_fp32_both_passes():
    dev = require_gpu()
    wl = W.WORKLOADS["tiny"]
    xd, xf = attn_inputs_dev(wl, dev)
    for pass_, name in PASSES:
        say(f"slot_attn tiny f32 {name}")
        out, lse = _run(xd, wl, pass_)
        O, L = _oracle(xf, wl, pass_)
        check_attn(to_f64(out), to_f64(lse), O, L, "f32", f"tiny {name}")


SMALL_BF16 = [
    # name, workload overrides: several key tiles, ragged prefix and token counts
    ("p300_s5l7", dict(batch=2, n_q_heads=4, n_kv_heads=2, prefix_len=300, kv_capacity=320, n_slots=5, slot_len=7)),
    ("g4_two_row_blocks", dict(batch=1, n_q_heads=8, n_kv_heads=2, prefix_len=200, n_slots=6, slot_len=8)),
    ("no_prefix", dict(batch=2, n_q_heads=2, n_kv_heads=1, prefix_len=0, n_slots=9, slot_len=5)),
    ("l1_decode", dict(batch=2, n_q_heads=4, n_kv_heads=4, prefix_len=130, n_slots=16, slot_len=1)),
    ("one_slot", dict(batch=1, n_q_heads=4, n_kv_heads=1, prefix_len=64, n_slots=1, slot_len=33)),
    ("d64", dict(batch=2, n_q_heads=4, n_kv_heads=2, head_dim=64, prefix_len=257, n_slots=4, slot_len=6)),
    # one key past a tile, and slots longer than several key tiles
    ("p65_long_slots", dict(batch=1, n_q_heads=2, n_kv_heads=1, prefix_len=65, n_slots=2, slot_len=200)),
    ("p1", dict(batch=3, n_q_heads=2, n_kv_heads=2, prefix_len=1, n_slots=3, slot_len=4)),
    # 256-row (eight-wave) workgroups: two of them, the second with 112 padding rows; D = 64;
    # and 260 rows, which stay on three 128-row workgroups
    ("wide_two_blocks", dict(batch=2, n_q_heads=8, n_kv_heads=2, prefix_len=333, n_slots=10, slot_len=10)),
    ("d64_wide", dict(batch=1, n_q_heads=8, n_kv_heads=2, head_dim=64, prefix_len=300, n_slots=8, slot_len=8)),
    ("g2_three_row_blocks", dict(batch=1, n_q_heads=4, n_kv_heads=2, prefix_len=190, n_slots=10, slot_len=13)),
    # three query heads per KV head: the rows of a token are split across row blocks
    ("g3_token_split", dict(batch=2, n_q_heads=6, n_kv_heads=2, prefix_len=200, n_slots=7, slot_len=11)),
]


@pytest.mark.parametrize("name,over", SMALL_BF16, ids=[c[0] for c in SMALL_BF16])
@pytest.mark.parametrize("q_scale", [1.0, 4.0], ids=["normal", "peaked"])
def test_bf16_small_shapes(name, over, q_scale):
    dev = require_gpu()
    wl = W.WORKLOADS["qwen0.6b"].replace(**over, hidden=0, vocab=0, seed=77)
    xd, xf = attn_inputs_dev(wl, dev, q_scale=q_scale)
    for pass_, pname in PASSES:
        say(f"slot_attn bf16 {name} q_scale={q_scale} {pname}")
        out, lse = _run(xd, wl, pass_)
        O, L = _oracle(xf, wl, pass_)
        check_attn(to_f64(out), to_f64(lse), O, L, "bf16", f"{name} {pname}")


def test_bf16_per_slot_pass_and_cross_causal():
    dev = require_gpu()
    wl = W.WORKLOADS["qwen0.6b"].replace(batch=2, n_q_heads=4, n_kv_heads=2, prefix_len=150, n_slots=6, slot_len=8,
                                         hidden=0, vocab=0, seed=78)
    xd, xf = attn_inputs_dev(wl, dev)
    sp = (np.random.default_rng(4).random((2, 6)) < 0.5).astype(np.uint8)
    for cross in (Z.CROSS_SLOT_NONE, Z.CROSS_SLOT_CAUSAL):
        say(f"slot_attn bf16 slot_pass cross={cross}")
        out, lse = _run(xd, wl, Z.PASS_DIFFUSION, cross=cross, slot_pass=torch.from_numpy(sp).to(dev))
        O, L = _oracle(xf, wl, oracle.PASS_DIFFUSION, cross=cross, slot_pass=sp)
        check_attn(to_f64(out), to_f64(lse), O, L, "bf16", f"slot_pass cross={cross}")


@pytest.mark.parametrize("over", [dict(n_q_heads=8, n_kv_heads=4), dict(n_q_heads=8, n_kv_heads=4, head_dim=64),
                                  dict(n_q_heads=12, n_kv_heads=4)], ids=["g2", "g2_d64", "g3"])
def test_bf16_cross_causal_with_prefix_heavy_first(over):
    """Cross-slot causal order after a prefix, one split and 8 GQA groups:
    the launch that dispatches row blocks heaviest first (D = 128 and 64;
    three heads per group, whose token rows straddle row blocks); both
    passes, every head against the oracle."""
    dev = require_gpu()
    wl = W.WORKLOADS["qwen0.6b"].replace(batch=2, prefix_len=300, n_slots=16, slot_len=16, hidden=0, vocab=0,
                                         seed=82, **over)
    xd, xf = attn_inputs_dev(wl, dev)
    for pass_, pname in PASSES:
        say(f"slot_attn cross causal heavy-first {pname}")
        out, lse = _run(xd, wl, pass_, cross=Z.CROSS_SLOT_CAUSAL, splits=1)
        O, L = _oracle(xf, wl, pass_, cross=oracle.CROSS_SLOT_CAUSAL)
        check_attn(to_f64(out), to_f64(lse), O, L, "bf16", f"cross causal heavy-first {pname}")


@pytest.mark.parametrize("over", [dict(), dict(n_q_heads=8, n_kv_heads=2)], ids=["rows128", "rows256_wide"])
def test_bf16_split_counts_agree_and_runs_are_bitwise_identical(over):
    dev = require_gpu()
    wl = W.WORKLOADS["qwen0.6b"].replace(batch=2, prefix_len=1000, hidden=0, vocab=0, seed=79, **over)
    xd, xf = attn_inputs_dev(wl, dev)
    O, L = _oracle(xf, wl, oracle.PASS_DIFFUSION)
    outs = {}
    for splits in (1, 2, 4, 8, 16):  # 16 (one key tile each): the merge's path past its first 8 splits
        say(f"slot_attn bf16 splits={splits}")
        out, lse = _run(xd, wl, Z.PASS_DIFFUSION, splits=splits)
        check_attn(to_f64(out), to_f64(lse), O, L, "bf16", f"splits={splits}")
        out2, lse2 = _run(xd, wl, Z.PASS_DIFFUSION, splits=splits)
        assert torch.equal(out.view(torch.int16), out2.view(torch.int16)), "rerun differs"
        assert torch.equal(lse, lse2), "rerun LSE differs"
        outs[splits] = (to_f64(out), to_f64(lse))
    for splits in (2, 4, 8, 16):
        # each split rounds its probabilities to bf16 against its own running
        # maximum, so splits agree to that rounding (2^-9 relative per term of a
        # convex combination of |v| <= ~5), not bit for bit; LSE is float32 only
        d = np.abs(outs[splits][0] - outs[1][0])
        assert d.max() <= 4e-3 and d.mean() <= 2e-4, f"split {splits} vs 1: max {d.max():.3e} mean {d.mean():.3e}"
        assert np.abs(outs[splits][1] - outs[1][1]).max() < 1e-5


RAGGED = [
    # name, dtype, overrides: per-row prefix lengths after KV-cache appends
    ("bf16_p300", "bf16", dict(batch=4, n_q_heads=4, n_kv_heads=2, prefix_len=300, kv_capacity=320, n_slots=5,
                               slot_len=7)),
    ("bf16_d64", "bf16", dict(batch=3, n_q_heads=4, n_kv_heads=2, head_dim=64, prefix_len=257, n_slots=4,
                              slot_len=6)),
    ("f32", "f32", dict(batch=3, n_q_heads=2, n_kv_heads=1, head_dim=64, prefix_len=70, n_slots=3, slot_len=4)),
    ("bf16_wide", "bf16", dict(batch=3, n_q_heads=8, n_kv_heads=2, prefix_len=300, n_slots=8, slot_len=8)),
]


@pytest.mark.parametrize("name,dtype,over", RAGGED, ids=[c[0] for c in RAGGED])
def test_ragged_prefix_lengths(name, dtype, over):
    """Rows with different prefix lengths (0, full, and between), with 1 and 3
    prefix splits: every row against the oracle with its own length."""
    dev = require_gpu()
    wl = W.WORKLOADS["qwen0.6b"].replace(**over, dtype=dtype, hidden=0, vocab=0, seed=80)
    xd, xf = attn_inputs_dev(wl, dev)
    P = wl.prefix_len
    plens = np.array([P, 0, P // 2 + 3, 1][: wl.batch], dtype=np.int32)
    pl_dev = torch.from_numpy(plens).to(dev)
    for pass_, pname in PASSES:
        O, L = oracle.slot_attention(xf["q"], xf["k_cache"], xf["v_cache"], xf["k_slot"], xf["v_slot"], plens,
                                     wl.n_slots, wl.slot_len, wl.scale, pass_)
        for splits in (1, 3):
            say(f"slot_attn ragged {name} {pname} splits={splits} plens={plens.tolist()}")
            out, lse = Z.slot_attn(xd["q"], xd["k_cache"], xd["v_cache"], xd["k_slot"], xd["v_slot"], wl.n_slots,
                                   wl.slot_len, pass_=pass_, prefix_len=P, softmax_scale=wl.scale,
                                   prefix_splits=splits, prefix_lens=pl_dev)
            torch.cuda.synchronize()
            check_attn(to_f64(out), to_f64(lse), O, L, dtype, f"ragged {name} {pname} splits={splits}")
    # out-of-range lengths are clamped to [0, prefix_len]
    say(f"slot_attn ragged {name} clamped lengths")
    wild = torch.tensor(([P + 50, -7, P, 0] * 2)[: wl.batch], dtype=torch.int32, device=dev)
    out, lse = Z.slot_attn(xd["q"], xd["k_cache"], xd["v_cache"], xd["k_slot"], xd["v_slot"], wl.n_slots,
                           wl.slot_len, prefix_len=P, softmax_scale=wl.scale, prefix_lens=wild)
    torch.cuda.synchronize()
    cl = np.clip(wild.cpu().numpy(), 0, P)
    O, L = oracle.slot_attention(xf["q"], xf["k_cache"], xf["v_cache"], xf["k_slot"], xf["v_slot"], cl,
                                 wl.n_slots, wl.slot_len, wl.scale, oracle.PASS_DIFFUSION)
    check_attn(to_f64(out), to_f64(lse), O, L, dtype, f"ragged {name} clamped")


def test_bf16_outputs_stay_inside_their_buffers():
    dev = require_gpu()
    wl = W.WORKLOADS["qwen0.6b"].replace(batch=1, n_q_heads=4, n_kv_heads=2, prefix_len=100, n_slots=3, slot_len=5,
                                         hidden=0, vocab=0, seed=80)
    xd, xf = attn_inputs_dev(wl, dev)
    B, Hq, T, D = xd["q"].shape
    n = B * Hq * T * D
    guard = 4096
    buf = torch.full((n + 2 * guard,), 7.0, dtype=torch.bfloat16, device=dev)
    lbuf = torch.full((B * Hq * T + 2 * guard,), 7.0, dtype=torch.float32, device=dev)
    out = buf[guard:guard + n].view(B, Hq, T, D)
    lse = lbuf[guard:guard + B * Hq * T].view(B, Hq, T)
    for splits in (1, 3):
        say(f"slot_attn guard canaries splits={splits}")
        Z.slot_attn(xd["q"], xd["k_cache"], xd["v_cache"], xd["k_slot"], xd["v_slot"], wl.n_slots, wl.slot_len,
                    prefix_len=wl.prefix_len, out=out, lse=lse, prefix_splits=splits)
        torch.cuda.synchronize()
        assert torch.all(buf[:guard] == 7.0) and torch.all(buf[guard + n:] == 7.0)
        assert torch.all(lbuf[:guard] == 7.0) and torch.all(lbuf[guard + B * Hq * T:] == 7.0)
    O, L = _oracle(xf, wl, oracle.PASS_DIFFUSION)
    check_attn(to_f64(out), to_f64(lse), O, L, "bf16", "guarded")


@pytest.mark.parametrize("pass_,pname", PASSES, ids=[p[1] for p in PASSES])
@pytest.mark.parametrize("name", ["qwen0.6b", "qwen1.7b", "qwen4b"])
def test_full_size_every_head(name, pass_, pname):
    """Full workload shapes in the launch configuration the benchmark times
    (the library's own prefix split): every (batch, head) pair and every token
    against the oracle, and the last token of each slot identical across the
    two passes (it sees the same keys in both)."""
    dev = require_gpu()
    wl = W.WORKLOADS[name].replace(hidden=0, vocab=0)
    say(f"slot_attn full {name} {pname}: generating inputs")
    x, xd, xf = full_attention_inputs(wl, dev)
    say(f"slot_attn full {name} {pname}")
    out, lse = _run(xd, wl, pass_)
    Og, Lg = to_f64(out), to_f64(lse)
    say(f"slot_attn full {name} {pname}: oracle over every head")
    O, L = oracle_attention_by_row(xf, wl.prefix_len, wl.n_slots, wl.slot_len, wl.scale, pass_)
    check_attn(Og, Lg, O, L, "bf16", f"{name} {pname}")
    other = Z.PASS_AR_INFILL if pass_ == Z.PASS_DIFFUSION else Z.PASS_DIFFUSION
    out2, lse2 = _run(xd, wl, other)
    last = np.arange(wl.n_slots) * wl.slot_len + wl.slot_len - 1
    assert np.abs(to_f64(out2)[:, :, last] - Og[:, :, last]).max() <= 1e-2
    assert np.abs(to_f64(lse2)[:, :, last] - Lg[:, :, last]).max() <= 1e-4


def _layout_case(wl, dev, variant):
    """Training-layout attention: P = 0, every slot sees the earlier slots.
    Paper-literal reading: causal in physical order (every slot AR_INFILL).
    Variant: the masked slots (after the clean ones) are bidirectional inside."""
    x = W.attention_inputs(wl)
    xd = {k: to_dev(v, wl.dtype, dev) for k, v in x.items()}
    order, masked_phys = W.training_layout(wl)
    sp = masked_phys.astype(np.uint8) * 0 + 1  # all AR_INFILL
    if variant:
        sp = np.where(masked_phys, 0, 1).astype(np.uint8)  # masked slots DIFFUSION
    say(f"layout attention N={wl.T} variant={variant}")
    out, lse = Z.slot_attn(xd["q"], None, None, xd["k_slot"], xd["v_slot"], wl.n_slots, wl.slot_len,
                           pass_=Z.PASS_AR_INFILL, cross_slot=Z.CROSS_SLOT_CAUSAL,
                           slot_pass=torch.from_numpy(sp).to(dev))
    torch.cuda.synchronize()
    Og, Lg = to_f64(out), to_f64(lse)
    xf = {k: W.as_f64(v, "bf16") for k, v in x.items()}
    say(f"layout attention N={wl.T} variant={variant}: oracle over every head")
    O, L = oracle_attention_by_row(xf, 0, wl.n_slots, wl.slot_len, wl.scale, oracle.PASS_AR_INFILL,
                                   cross=oracle.CROSS_SLOT_CAUSAL, slot_pass=sp)
    check_attn(Og, Lg, O, L, "bf16", f"layout variant={variant}")


@pytest.mark.parametrize("variant", [False, True], ids=["causal", "masked_bidirectional"])
@pytest.mark.parametrize("shape", [dict(batch=2, n_q_heads=4, n_kv_heads=2, n_slots=16, slot_len=32),
                                   # 8 GQA groups, one split: the heaviest-first dispatch
                                   dict(batch=2, n_q_heads=8, n_kv_heads=4, n_slots=8, slot_len=32)],
                         ids=["four_groups", "eight_groups_heavy_first"])
def test_training_layout_small(variant, shape):
    dev = require_gpu()
    wl = W.WORKLOADS["layout"].replace(**shape, seed=81)
    _layout_case(wl, dev, variant)


def test_training_layout_full_size():
    """The full training layout (B = 8, 16 heads, 4096 tokens), every (batch,
    head) pair against the oracle."""
    dev = require_gpu()
    wl = W.WORKLOADS["layout"]
    _layout_case(wl, dev, False)
