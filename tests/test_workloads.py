"""Input generators: bf16 rounding, seeds, the training layout (CPU only)."""

import numpy as np
import torch

import workloads as W


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.standard_normal(100000).astype(np.float32),
        (rng.standard_normal(1000) * 1e-30).astype(np.float32),
        np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -1.0 - 2 ** -8, 65504.0, 3.3895314e38, 0.0, -0.0], np.float32),
    ])
    ours = W.bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    np.testing.assert_array_equal(W.bf16_to_f32(ours), torch.from_numpy(ref.view(np.int16)).view(torch.bfloat16).float().numpy())


def test_seeds_reproduce_and_differ():
    wl = W.WORKLOADS["qwen0.6b"].replace(batch=1, prefix_len=64, vocab=300, hidden=64)
    a = W.attention_inputs(wl)
    b = W.attention_inputs(wl)
    for k in a:
        np.testing.assert_array_equal(a[k], b[k])
    c = W.attention_inputs(wl.replace(seed=5))
    assert not np.array_equal(a["q"], c["q"])
    ca = W.confidence_inputs(wl)
    cb = W.confidence_inputs(wl)
    np.testing.assert_array_equal(ca["w_vocab"], cb["w_vocab"])


def test_distributions():
    wl = W.WORKLOADS["qwen0.6b"].replace(batch=2, vocab=20000)
    x = W.attention_inputs(wl)
    kc = W.bf16_to_f32(x["k_cache"])
    assert x["k_cache"].shape == (2, 8, 2048, 128) and x["q"].shape == (2, 16, 64, 128)
    assert abs(kc.mean()) < 0.01 and abs(kc.std() - 1.0) < 0.01
    c = W.confidence_inputs(wl)
    w = W.bf16_to_f32(c["w_vocab"])
    assert c["hidden"].shape == (128, 1024) and w.shape == (20000, 1024)
    assert abs(w.std() - 0.02) < 2e-4


def test_training_layout():
    wl = W.WORKLOADS["layout"]
    order, masked = W.training_layout(wl)
    order2, masked2 = W.training_layout(wl)
    np.testing.assert_array_equal(order, order2)
    B, S = order.shape
    assert (B, S) == (8, 128)
    for b in range(B):
        assert sorted(order[b]) == list(range(S))  # a permutation of the slots
        n_clean = int((~masked[b]).sum())
        assert not masked[b, :n_clean].any() and masked[b, n_clean:].all()  # clean first
        assert order[b, :n_clean].tolist() != sorted(order[b, :n_clean]) or n_clean < 3  # permuted
    frac = masked.mean()
    assert 0.4 < frac < 0.6
