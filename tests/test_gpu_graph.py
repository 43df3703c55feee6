"""The scoring step captured in a HIP graph (torch.cuda.CUDAGraph over the
library's launches on the capturing stream) and replayed.

Every kernel of the step is deterministic, so each replay must equal an
eager run on the same inputs bit for bit.  The test replays several times
with new inputs copied into the captured buffers and eager work between the
replays, and checks every replay.
"""

import numpy as np
import pytest
import torch

import workloads as W
from gpu_helpers import require_gpu, say, to_dev

import paper_2609_19868_amd as Z

pytestmark = pytest.mark.gpu


def _inputs(wl, seed, dev):
    w2 = wl.replace(seed=seed)
    x = W.attention_inputs(w2)
    c = W.confidence_inputs(w2)
    d = {k: to_dev(v, "bf16", dev) for k, v in x.items()}
    d["hidden"] = to_dev(c["hidden"], "bf16", dev)
    d["w_vocab"] = to_dev(c["w_vocab"], "bf16", dev)
    return d


def _step(s, wl, out):
    B, S, L = wl.batch, wl.n_slots, wl.slot_len
    Z.slot_attn(s["q"], s["k_cache"], s["v_cache"], s["k_slot"], s["v_slot"], S, L, pass_=Z.PASS_DIFFUSION,
                out=out["attn"], lse=out["attn_lse"], workspace=out["attn_ws"])
    Z.slot_confidence(s["hidden"], s["w_vocab"], out=out["conf"], workspace=out["conf_ws"])
    Z.select_slots(out["conf"]["max_prob"].view(B, S, L), threshold=0.9, out=out["sel"])


def _buffers(wl, s, dev):
    from paper_2609_19868_amd import _lib

    B, Hq, S, L, D, M = wl.batch, wl.n_q_heads, wl.n_slots, wl.slot_len, wl.head_dim, wl.M
    desc = Z.slot_attn_desc(s["q"], s["k_cache"], s["k_slot"], S, L, Z.PASS_DIFFUSION)
    cdesc = _lib.ConfDesc(n_rows=M, hidden=wl.hidden, vocab=wl.vocab, dtype=1)
    return {
        "attn": torch.empty((B, Hq, wl.T, D), dtype=torch.bfloat16, device=dev),
        "attn_lse": torch.empty((B, Hq, wl.T), dtype=torch.float32, device=dev),
        "attn_ws": torch.empty(max(1, _lib.slot_attn_workspace_size(desc)), dtype=torch.uint8, device=dev),
        "conf": {"max_prob": torch.empty(M, dtype=torch.float32, device=dev),
                 "argmax": torch.empty(M, dtype=torch.int32, device=dev),
                 "lse": torch.empty(M, dtype=torch.float32, device=dev)},
        "conf_ws": torch.empty(_lib.slot_confidence_workspace_size(cdesc), dtype=torch.uint8, device=dev),
        "sel": (torch.empty((B, S), dtype=torch.float32, device=dev), torch.empty((B, S), dtype=torch.int32, device=dev),
                torch.empty((B,), dtype=torch.int32, device=dev)),
    }


def _flat(out):
    return [out["attn"], out["attn_lse"], *out["conf"].values(), *out["sel"]]


@pytest.mark.parametrize("batch", [1, 4])
def test_graph_replays_match_eager(batch):
    dev = require_gpu()
    wl = W.WORKLOADS["qwen0.6b"].replace(batch=batch, prefix_len=300, n_slots=4, slot_len=8, hidden=256,
                                         vocab=5000, seed=120)
    static = _inputs(wl, 120, dev)
    gout = _buffers(wl, static, dev)
    eout = _buffers(wl, static, dev)
    say(f"graph capture, batch {batch}")
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for _ in range(2):
            _step(static, wl, gout)
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        _step(static, wl, gout)
    torch.cuda.synchronize()
    for trial in range(4):
        fresh = _inputs(wl, 121 + trial, dev)
        for k, v in fresh.items():
            static[k].copy_(v)
        say(f"graph replay {trial}")
        g.replay()
        torch.cuda.synchronize()
        _step(fresh, wl, eout)  # eager work between replays, on the same inputs
        torch.cuda.synchronize()
        for a, b in zip(_flat(gout), _flat(eout)):
            assert torch.equal(a, b), f"replay {trial} differs from the eager step"
        assert int(gout["sel"][2].sum()) >= batch  # at least one slot per row is selected
