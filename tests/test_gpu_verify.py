"""Verification step on the GPU (through the C ABI) against the oracle.

zarya_verify_accept and zarya_kv_append are integer and copy work: the bar is
bit-exact (accepted flags, counts, cache bytes and lengths).  The acceptance
decision compares float32 probabilities with a float32 threshold on both
sides.  The last test chains a whole verification step on the GPU -- AR_INFILL
attention, confidence with the draft ids as targets, acceptance, append, and
the next draft pass over the now ragged prefixes -- and checks each stage
against the oracle fed with the stage's GPU inputs.
"""

import zlib

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_helpers import attn_inputs_dev, check_attn, require_gpu, say, to_dev, to_f64

import paper_2609_19868_amd as Z

pytestmark = pytest.mark.gpu


def _selection(rng, B, S, invalid=False, repeats=False):
    sel = np.full((B, S), -1, dtype=np.int32)
    for b in range(B):
        k = int(rng.integers(0, S + 1))
        sel[b, :k] = rng.permutation(S)[:k]
        if invalid and k < S and rng.random() < 0.5:
            sel[b, k] = S + 3  # not a slot id: skipped
            if k + 1 < S:
                sel[b, k + 1] = int(rng.integers(0, S))  # after an invalid id the list goes on
        if repeats and k >= 2 and rng.random() < 0.7:
            i = int(rng.integers(1, k))
            sel[b, i] = sel[b, int(rng.integers(0, i))]  # an earlier slot listed again: skipped
    return sel


ACCEPT_SHAPES = [(16, 8, 8), (3, 1, 5), (5, 7, 1), (2, 1024, 3), (4, 6, 300)]


@pytest.mark.parametrize("B,S,L", ACCEPT_SHAPES, ids=[f"B{b}_S{s}_L{l}" for b, s, l in ACCEPT_SHAPES])
@pytest.mark.parametrize("rule", [Z.ACCEPT_PREFIX, Z.ACCEPT_PER_TOKEN], ids=["prefix", "per_token"])
def test_accept_bit_exact(B, S, L, rule):
    dev = require_gpu()
    rng = np.random.default_rng(1000 * B + S + L + rule)
    tp = rng.random((B, S, L)).astype(np.float32)
    tp[rng.random((B, S, L)) < 0.05] = np.float32(0.4)  # exactly at the threshold: rejected
    tp[rng.random((B, S, L)) < 0.3] = np.float32(0.9)
    sel = _selection(rng, B, S, invalid=True)
    say(f"verify_accept B={B} S={S} L={L} rule={rule}")
    acc, n, tot = Z.verify_accept(torch.from_numpy(tp).to(dev), torch.from_numpy(sel).to(dev), 0.4, rule)
    torch.cuda.synchronize()
    a_ref, n_ref, t_ref = oracle.accept_tokens(tp, sel, np.float32(0.4), rule)
    assert np.array_equal(acc.cpu().numpy(), a_ref)
    assert np.array_equal(n.cpu().numpy(), n_ref)
    assert np.array_equal(tot.cpu().numpy(), t_ref)


APPEND_CASES = [
    # name, dtype, B, Hkv, D, C, S, L
    ("bf16_d128", "bf16", 6, 8, 128, 200, 8, 8),
    ("bf16_d64", "bf16", 3, 2, 64, 90, 4, 16),
    ("f32_d64", "f32", 4, 3, 64, 50, 5, 3),
    ("bf16_long_slots", "bf16", 2, 1, 128, 5000, 8, 512),
    ("bf16_max_tokens", "bf16", 3, 1, 64, 9000, 1024, 8),  # S*L = 8192 draft tokens, the largest accepted
]


@pytest.mark.parametrize("name,dtype,B,Hkv,D,C,S,L", APPEND_CASES, ids=[c[0] for c in APPEND_CASES])
def test_append_bit_exact(name, dtype, B, Hkv, D, C, S, L):
    dev = require_gpu()
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    T = S * L

    def draw(shape):
        x = rng.standard_normal(shape, dtype=np.float32)
        return W.bf16_bits(x) if dtype == "bf16" else x

    kc, vc, ks, vs = draw((B, Hkv, C, D)), draw((B, Hkv, C, D)), draw((B, Hkv, T, D)), draw((B, Hkv, T, D))
    acc = (rng.random((B, S, L)) < 0.6).astype(np.uint8)
    order = _selection(rng, B, S, invalid=True, repeats=True)
    plens = rng.integers(0, max(1, C - T), B).astype(np.int32)
    plens[0] = C - 1 if B > 1 else plens[0]  # cannot fit unless nothing is appended
    if B > 2:
        plens[1] = -5  # negative: left alone
    kd, vd = to_dev(kc, dtype, dev), to_dev(vc, dtype, dev)
    pl = torch.from_numpy(plens.copy()).to(dev)
    say(f"kv_append {name} plens={plens.tolist()}")
    Z.kv_append(kd, vd, pl, to_dev(ks, dtype, dev), to_dev(vs, dtype, dev), torch.from_numpy(acc).to(dev),
                torch.from_numpy(order).to(dev))
    torch.cuda.synchronize()
    kr, vr, lr = oracle.kv_append(kc, vc, plens, ks, vs, acc, order)
    assert np.array_equal(pl.cpu().numpy(), lr)
    view = np.int16 if dtype == "bf16" else np.int32
    assert np.array_equal(kd.cpu().view(torch.int16 if dtype == "bf16" else torch.int32).numpy(), kr.view(view))
    assert np.array_equal(vd.cpu().view(torch.int16 if dtype == "bf16" else torch.int32).numpy(), vr.view(view))


def test_verification_step_chain():
    """Select -> AR_INFILL attention -> confidence of the draft ids -> accept ->
    append -> next DIFFUSION draft pass over the ragged prefixes (bf16)."""
    dev = require_gpu()
    wl = W.WORKLOADS["qwen0.6b"].replace(batch=4, n_q_heads=4, n_kv_heads=2, prefix_len=200, kv_capacity=300,
                                         n_slots=6, slot_len=4, hidden=256, vocab=3000, seed=90)
    xd, xf = attn_inputs_dev(wl, dev)
    B, S, L, T = wl.batch, wl.n_slots, wl.slot_len, wl.T
    rng = np.random.default_rng(91)

    say("chain: AR_INFILL verification attention")
    out, lse = Z.slot_attn(xd["q"], xd["k_cache"], xd["v_cache"], xd["k_slot"], xd["v_slot"], S, L,
                           pass_=Z.PASS_AR_INFILL, prefix_len=wl.prefix_len, softmax_scale=wl.scale)
    torch.cuda.synchronize()
    O, Lr = oracle.slot_attention(xf["q"], xf["k_cache"], xf["v_cache"], xf["k_slot"], xf["v_slot"], wl.prefix_len,
                                  S, L, wl.scale, oracle.PASS_AR_INFILL)
    check_attn(to_f64(out), to_f64(lse), O, Lr, "bf16", "chain verification attention")

    say("chain: confidence with the draft ids as targets")
    c = W.confidence_inputs(wl, rng=rng, n_rows=B * T)
    h, w = to_dev(c["hidden"], "bf16", dev), to_dev(c["w_vocab"], "bf16", dev)
    draft_ids = rng.integers(0, wl.vocab, B * T).astype(np.int32)
    # make about half of the draft ids the model's own argmax so that some tokens pass
    ref = oracle.slot_confidence(W.as_f64(c["hidden"], "bf16"), W.as_f64(c["w_vocab"], "bf16"))
    keep = rng.random(B * T) < 0.5
    draft_ids[keep] = ref["argmax"][keep]
    res = Z.slot_confidence(h, w, target_ids=torch.from_numpy(draft_ids).to(dev))
    torch.cuda.synchronize()
    ref_t = oracle.slot_confidence(W.as_f64(c["hidden"], "bf16"), W.as_f64(c["w_vocab"], "bf16"), draft_ids)
    tp = res["target_prob"].cpu().numpy()
    assert np.all(np.abs(tp - ref_t["target_prob"]) <= 1e-3 * ref_t["target_prob"] + 1e-12)

    say("chain: selection, acceptance and append")
    conf = res["max_prob"].view(B, S, L)
    _, sel, nsel = Z.select_slots(conf, threshold=0.9)
    tp_dev = res["target_prob"].view(B, S, L).contiguous()
    # with these random weights the probabilities are small; a threshold at their
    # median gives a mix of accepted and rejected tokens
    thr = float(np.median(tp))
    acc, nacc, ntot = Z.verify_accept(tp_dev, sel, thr, Z.ACCEPT_PREFIX)
    torch.cuda.synchronize()
    a_ref, n_ref, t_ref = oracle.accept_tokens(tp.reshape(B, S, L), sel.cpu().numpy(), np.float32(thr))
    assert np.array_equal(acc.cpu().numpy(), a_ref) and np.array_equal(ntot.cpu().numpy(), t_ref)
    plens = torch.full((B,), wl.prefix_len, dtype=torch.int32, device=dev)
    kc, vc = xd["k_cache"].clone(), xd["v_cache"].clone()
    Z.kv_append(kc, vc, plens, xd["k_slot"], xd["v_slot"], acc, sel)
    torch.cuda.synchronize()
    kr, vr, lr = oracle.kv_append(x_bits(xd["k_cache"]), x_bits(xd["v_cache"]), [wl.prefix_len] * B,
                                  x_bits(xd["k_slot"]), x_bits(xd["v_slot"]), a_ref, sel.cpu().numpy())
    assert np.array_equal(plens.cpu().numpy(), lr)
    assert np.array_equal(x_bits(kc), kr) and np.array_equal(x_bits(vc), vr)

    say(f"chain: next draft pass over ragged prefixes {lr.tolist()}")
    out2, lse2 = Z.slot_attn(xd["q"], kc, vc, xd["k_slot"], xd["v_slot"], S, L, pass_=Z.PASS_DIFFUSION,
                             prefix_len=int(lr.max()), softmax_scale=wl.scale, prefix_lens=plens)
    torch.cuda.synchronize()
    O2, L2 = oracle.slot_attention(xf["q"], W.as_f64(kr, "bf16"), W.as_f64(vr, "bf16"), xf["k_slot"], xf["v_slot"],
                                   lr, S, L, wl.scale, oracle.PASS_DIFFUSION)
    check_attn(to_f64(out2), to_f64(lse2), O2, L2, "bf16", "chain next draft pass")


def x_bits(t):
    """bf16 device tensor -> uint16 bits on the host."""
    return t.detach().cpu().view(torch.int16).numpy().view(np.uint16)
