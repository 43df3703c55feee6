"""Mode A (MDM sampling with first-hitting denoising) on the GPU, through the
C ABI, against the oracle.

zarya_mdm_reveal is integer work (keys built from float32 confidences by
integer operations, or from Philox words): the bar is bit-exact order, counts,
mask flags and tokens.  The chained test runs a whole small generation --
budget, then per step causal attention of the previous step's revealed
tokens and the masked tail after the cache, Gumbel-max sampling of the masked
rows, the reveal, and the cache append of the tokens revealed the step
before -- and checks every stage against the oracle fed with that stage's GPU
inputs (attention and sampling to the tolerances of their own tests).
"""

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_helpers import (check_attn, oracle_attention_by_row, oracle_sample_by_block, require_gpu, say, to_dev,
                         to_f64)

import paper_2609_19868_amd as Z

pytestmark = pytest.mark.gpu

RULES = [(Z.REVEAL_CONFIDENCE, "confidence"), (Z.REVEAL_LEFTMOST, "leftmost"), (Z.REVEAL_RANDOM, "random")]
SHAPES = [(4, 1), (8, 17), (5, 257), (3, 1000), (2, 4096), (2, 8192)]


def _reveal_inputs(rng, B, N):
    conf = rng.random((B, N)).astype(np.float32)
    conf[rng.random((B, N)) < 0.15] = np.float32(0.5)  # ties
    conf[rng.random((B, N)) < 0.02] = np.float32(np.nan)
    zero = rng.random((B, N)) < 0.05
    conf[zero] = np.where(rng.random(zero.sum()) < 0.5, np.float32(0.0), np.float32(-0.0))
    mask = (rng.random((B, N)) < 0.7).astype(np.uint8)
    mask[0] = 1  # every position open
    if B > 2:
        mask[1] = 0  # nothing open
    k = rng.integers(-2, N + 3, B).astype(np.int32)
    k[-1] = min(N, 3)
    sid = rng.integers(0, 151936, (B, N)).astype(np.int32)
    tok = rng.integers(0, 151936, (B, N)).astype(np.int32)
    return conf, mask, k, sid, tok


@pytest.mark.parametrize("B,N", SHAPES, ids=[f"B{b}_N{n}" for b, n in SHAPES])
@pytest.mark.parametrize("rule,rname", RULES, ids=[r[1] for r in RULES])
def test_reveal_bit_exact(B, N, rule, rname):
    dev = require_gpu()
    rng = np.random.default_rng(100 * B + N + rule)
    conf, mask, k, sid, tok = _reveal_inputs(rng, B, N)
    seed, offset = 0xDEADBEEF12345678, 77 + N
    say(f"mdm_reveal {rname} B={B} N={N}")
    md = torch.from_numpy(mask).to(dev)
    td = torch.from_numpy(tok).to(dev)
    order, n = Z.mdm_reveal(md, torch.from_numpy(k).to(dev), rule, conf=torch.from_numpy(conf).to(dev), seed=seed,
                            offset=offset, sample_id=torch.from_numpy(sid).to(dev), tokens=td)
    torch.cuda.synchronize()
    o_ref, n_ref, m_ref, t_ref = oracle.reveal(conf, mask.astype(bool), np.maximum(k, 0), rule, seed, offset,
                                               tokens=tok, sample_id=sid)
    assert np.array_equal(n.cpu().numpy(), n_ref)
    assert np.array_equal(order.cpu().numpy(), o_ref)
    assert np.array_equal(md.cpu().numpy().astype(bool), m_ref)
    assert np.array_equal(td.cpu().numpy(), t_ref)


def test_reveal_without_tokens_or_counts():
    dev = require_gpu()
    rng = np.random.default_rng(7)
    conf, mask, k, _, _ = _reveal_inputs(rng, 3, 50)
    md = torch.from_numpy(mask).to(dev)
    order = torch.full((3, 50), 99, dtype=torch.int32, device=dev)
    from paper_2609_19868_amd import _lib
    _lib.check(_lib.lib().zarya_mdm_reveal(3, 50, None, md.data_ptr(), torch.from_numpy(k).to(dev).data_ptr(),
                                           Z.REVEAL_LEFTMOST, 0, 0, None, None, order.data_ptr(), None, None))
    torch.cuda.synchronize()
    o_ref, _, m_ref, _ = oracle.reveal(conf, mask.astype(bool), np.maximum(k, 0), oracle.REVEAL_LEFTMOST)
    assert np.array_equal(order.cpu().numpy(), o_ref) and np.array_equal(md.cpu().numpy().astype(bool), m_ref)


def _x_bits(t):
    return t.detach().cpu().view(torch.int16).numpy().view(np.uint16)


@pytest.mark.parametrize("rule,rname", RULES[::2], ids=[r[1] for r in RULES[::2]])
def test_generation_chain(rule, rname):
    """A whole Mode A generation: 2 rows of 30 masks after a 100-token prompt,
    T = 0 (steps of at most four), every stage against the oracle.  The
    confidence rule samples every masked row, then reveals; the random rule
    (first-hitting sampler) reveals first and samples only the chosen rows."""
    dev = require_gpu()
    B, Hq, Hkv, D, P0, N0, H, V = 2, 4, 2, 128, 100, 30, 256, 3000
    scale = 1.0 / np.sqrt(D)
    rng = np.random.default_rng(200 + rule)
    counts, n_diff_steps = Z.mdm_budget(N0, 0, 0.25, seed=5)
    ref_counts, _ = oracle.mask_budget(N0, 0, 0.25, 5)
    assert counts == [int(c) for c in ref_counts] and sum(counts) == N0

    C = P0 + N0
    kc = W.bf16_bits(rng.standard_normal((B, Hkv, C, D)).astype(np.float32))
    vc = W.bf16_bits(rng.standard_normal((B, Hkv, C, D)).astype(np.float32))
    kcd, vcd = to_dev(kc, "bf16", dev), to_dev(vc, "bf16", dev)
    plens = torch.full((B,), P0, dtype=torch.int32, device=dev)
    w = W.bf16_bits(rng.standard_normal((V, H)).astype(np.float32) * 0.05)
    wd = to_dev(w, "bf16", dev)
    # the masked tail in its current order, as original positions (host bookkeeping)
    tail = [list(range(N0)) for _ in range(B)]
    tokens = np.full((B, N0), -1, dtype=np.int64)
    prev = 0  # tokens revealed at the previous step (the first rows of this step)
    for t, k_t in enumerate(counts + [0]):
        Nt = len(tail[0])
        R = prev + Nt
        if R == 0:
            break
        say(f"mode A {rname} step {t}: {prev} revealed + {Nt} masked rows, prefix {int(plens[0])}")
        q = W.bf16_bits(rng.standard_normal((B, Hq, R, D)).astype(np.float32))
        ks = W.bf16_bits(rng.standard_normal((B, Hkv, R, D)).astype(np.float32))
        vs = W.bf16_bits(rng.standard_normal((B, Hkv, R, D)).astype(np.float32))
        ksd, vsd = to_dev(ks, "bf16", dev), to_dev(vs, "bf16", dev)
        out, lse = Z.slot_attn(to_dev(q, "bf16", dev), kcd, vcd, ksd, vsd, R, 1, pass_=Z.PASS_AR_INFILL,
                               cross_slot=Z.CROSS_SLOT_CAUSAL, prefix_len=int(plens.max()), softmax_scale=scale,
                               prefix_lens=plens)
        torch.cuda.synchronize()
        pl = plens.cpu().numpy()
        O, L = oracle.slot_attention(W.as_f64(q, "bf16"), W.as_f64(_x_bits(kcd), "bf16"),
                                     W.as_f64(_x_bits(vcd), "bf16"), W.as_f64(ks, "bf16"), W.as_f64(vs, "bf16"),
                                     pl, R, 1, scale, oracle.PASS_AR_INFILL, cross_slot=oracle.CROSS_SLOT_CAUSAL)
        check_attn(to_f64(out), to_f64(lse), O, L, "bf16", f"step {t} attention")

        # the revealed tokens of the previous step join the cache
        if prev > 0:
            acc = np.zeros((B, R, 1), dtype=np.uint8)
            acc[:, :prev] = 1
            ordr = np.tile(np.arange(R, dtype=np.int32), (B, 1))
            kc_before, vc_before = _x_bits(kcd), _x_bits(vcd)
            Z.kv_append(kcd, vcd, plens, ksd, vsd, torch.from_numpy(acc).to(dev), torch.from_numpy(ordr).to(dev))
            torch.cuda.synchronize()
            kr, vr, lr = oracle.kv_append(kc_before, vc_before, pl, ks, vs, acc, ordr)
            assert np.array_equal(_x_bits(kcd), kr) and np.array_equal(_x_bits(vcd), vr)
            assert np.array_equal(plens.cpu().numpy(), lr)
        if Nt == 0:
            break

        hid = W.bf16_bits(rng.standard_normal((B * Nt, H)).astype(np.float32))
        hd = to_dev(hid, "bf16", dev)
        mask = torch.ones((B, Nt), dtype=torch.uint8, device=dev)
        kk = torch.full((B,), k_t, dtype=torch.int32, device=dev)
        if rule == Z.REVEAL_RANDOM:
            # first-hitting sampler: choose the positions, then draw only their tokens
            order, n = Z.mdm_reveal(mask, kk, rule, seed=13, offset=t)
            torch.cuda.synchronize()
            o_ref, n_ref, m_ref, _ = oracle.reveal(None, np.ones((B, Nt), bool), [k_t] * B, rule, 13, t)
            assert np.array_equal(order.cpu().numpy(), o_ref) and np.array_equal(n.cpu().numpy(), n_ref)
            assert np.array_equal(mask.cpu().numpy().astype(bool), m_ref)
            sel = np.concatenate([b * Nt + o_ref[b, : n_ref[b]] for b in range(B)]).astype(np.int32)
            res = Z.slot_sample(hd, wd, 1.0, seed=11, offset=t, rows=torch.from_numpy(sel).to(dev))
            torch.cuda.synchronize()
            ref = oracle.slot_sample(W.as_f64(hid[sel], "bf16"), W.as_f64(w, "bf16"), 1.0, 11, t)
            sid_sel = res["sample_id"].cpu().numpy()
            decided = ref["score_gap"] >= 1e-3
            assert np.array_equal(sid_sel[decided], ref["sample_id"][decided]), f"step {t} sampling"
            drawn = np.full((B, Nt), -1, dtype=np.int64)
            drawn.reshape(-1)[sel] = sid_sel
        else:
            # LM head with Gumbel-max sampling on every masked row (row i = b * Nt + j)
            res = Z.slot_sample(hd, wd, 1.0, seed=11, offset=t)
            torch.cuda.synchronize()
            ref = oracle.slot_sample(W.as_f64(hid, "bf16"), W.as_f64(w, "bf16"), 1.0, 11, t)
            sid = res["sample_id"].cpu().numpy()
            decided = ref["score_gap"] >= 1e-3
            assert np.array_equal(sid[decided], ref["sample_id"][decided]), f"step {t} sampling"
            sp = res["sample_prob"].view(B, Nt).contiguous()
            # reveal the k_t most confident of the masked tail, writing their tokens
            tok_t = torch.full((B, Nt), -1, dtype=torch.int32, device=dev)
            sid_t = res["sample_id"].view(B, Nt).contiguous()
            order, n = Z.mdm_reveal(mask, kk, rule, conf=sp, seed=13, offset=t, sample_id=sid_t, tokens=tok_t)
            torch.cuda.synchronize()
            o_ref, n_ref, m_ref, t_ref = oracle.reveal(sp.cpu().numpy(), np.ones((B, Nt), bool), [k_t] * B, rule,
                                                       13, t, tokens=np.full((B, Nt), -1),
                                                       sample_id=sid.reshape(B, Nt))
            assert np.array_equal(order.cpu().numpy(), o_ref) and np.array_equal(n.cpu().numpy(), n_ref)
            assert np.array_equal(mask.cpu().numpy().astype(bool), m_ref)
            assert np.array_equal(tok_t.cpu().numpy(), t_ref)
            drawn = sid.reshape(B, Nt)
        o = order.cpu().numpy()
        for b in range(B):
            picked = [tail[b][j] for j in o[b, : n_ref[b]]]
            for j, pos in zip(o[b, : n_ref[b]], picked):
                assert tokens[b, pos] == -1 and drawn[b, j] >= 0
                tokens[b, pos] = drawn[b, j]
            tail[b] = [tail[b][j] for j in range(Nt) if m_ref[b, j]]
        prev = int(n_ref[0])
    assert np.all(tokens >= 0), "every masked position is revealed exactly once"
    assert np.all(plens.cpu().numpy() == P0 + N0)


def test_mode_a_full_step():
    """The Mode A step at its full shape in the benchmark's launch
    configuration: attention of 4 revealed + 256 masked rows after a
    2048-token prompt (every (batch, head) pair), sampling of the 4096 masked
    rows (every row), the reveal of all rows bit-exact."""
    dev = require_gpu()
    wl = W.WORKLOADS["modeA"]
    B, Hq, Hkv, R = wl.batch, wl.n_q_heads, wl.n_kv_heads, wl.T
    Nt = R - W.MODE_A_REVEALED
    say("mode A full step: generating inputs")
    x = W.attention_inputs(wl)
    xd = {k: to_dev(v, "bf16", dev) for k, v in x.items()}
    out, lse = Z.slot_attn(xd["q"], xd["k_cache"], xd["v_cache"], xd["k_slot"], xd["v_slot"], R, 1,
                           pass_=Z.PASS_AR_INFILL, cross_slot=Z.CROSS_SLOT_CAUSAL, softmax_scale=wl.scale)
    torch.cuda.synchronize()
    Og, Lg = to_f64(out), to_f64(lse)
    say("mode A full step: oracle attention over every head")
    xf = {kk: W.as_f64(v, "bf16") for kk, v in x.items()}
    O, L = oracle_attention_by_row(xf, wl.prefix_len, R, 1, wl.scale, oracle.PASS_AR_INFILL,
                                   cross=oracle.CROSS_SLOT_CAUSAL)
    check_attn(Og, Lg, O, L, "bf16", "mode A attention")
    del xf, O, L

    c = W.confidence_inputs(wl, n_rows=B * Nt)
    hd, wd = to_dev(c["hidden"], "bf16", dev), to_dev(c["w_vocab"], "bf16", dev)
    say("mode A full step: sampling")
    res = Z.slot_sample(hd, wd, 1.0, seed=21, offset=3)
    torch.cuda.synchronize()
    say("mode A full step: oracle sampling of every row")
    ref = oracle_sample_by_block(W.as_f64(c["hidden"], "bf16"), W.as_f64(c["w_vocab"], "bf16"), 1.0, 21, 3)
    sid = res["sample_id"].cpu().numpy()
    decided = ref["score_gap"] >= 1e-3
    assert decided.mean() > 0.99
    assert np.array_equal(sid[decided], ref["sample_id"][decided])
    sp_ref = np.exp(ref["sample_logit"] - ref["lse"])
    e = np.abs(res["sample_prob"].cpu().numpy()[decided] - sp_ref[decided])
    assert np.all(e <= 1e-3 * sp_ref[decided] + 1e-12)

    say("mode A full step: reveal")
    mask = torch.ones((B, Nt), dtype=torch.uint8, device=dev)
    kk = torch.full((B,), 4, dtype=torch.int32, device=dev)
    sp = res["sample_prob"].view(B, Nt).contiguous()
    order, n = Z.mdm_reveal(mask, kk, Z.REVEAL_CONFIDENCE, conf=sp)
    torch.cuda.synchronize()
    o_ref, n_ref, _, _ = oracle.reveal(sp.cpu().numpy(), np.ones((B, Nt), bool), [4] * B)
    assert np.array_equal(order.cpu().numpy(), o_ref) and np.array_equal(n.cpu().numpy(), n_ref)
