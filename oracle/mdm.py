"""Oracle: Mode A (MDM sampling with first-hitting denoising) -- the mask
budget of a generation and the choice of the positions revealed at a step.

TEST INFRASTRUCTURE ONLY (see the package docstring).  Integer work on
float32 / float64 comparisons; exact.

Paper passages this follows (Sec. 5.1, Mode A):

* Step 1, "Mask budget planning": with a positive number T of discretization
  steps, exactly T diffusion steps are used; a binomial draw decides how many
  of the masked tokens are denoised by the diffusion process (alpha_0 is the
  expected fraction) and the tokens left over are denoised sequentially.  With
  T = 0 the noise calculation is skipped and T is set to a quarter of the
  number of masked tokens.
* Step 2, "Reordering": masked tokens always come after unmasked ones, so the
  positions revealed at a step join the committed prefix (Sec. 5.1 closing
  paragraph: the cached prefix states never change).
* Step 3: per step the model yields logits for the masked positions and the
  revealed tokens are drawn from them (the sampling oracle).
* The first-hitting denoising process (cited there) reveals masked positions
  one draw at a time.

Readings where the paper is silent (each listed in the design notes):

* Binomial(N, alpha_0) is drawn as the number of i < N with u_i < alpha_0, u_i
  the uniforms of row 0, ids 0..N-1, offset 0 of the sampling oracle's Philox
  stream under the budget's own seed (compared in float64; u is exact).
* T = 0: T = ceil(N / 4), every masked token goes through diffusion.
* The diffusion tokens are spread over the T steps as evenly as possible, the
  first (n_diff mod T) steps taking one more; then one step per sequential
  token.  Steps that reveal nothing (n_diff < T) are kept: T is exact.
* Which positions a step reveals: rule ``REVEAL_CONFIDENCE`` takes the k most
  confident open positions (descending confidence, ties to the lower index --
  first-hitting order; NaN counts as -inf); ``REVEAL_LEFTMOST`` the k lowest
  open positions (the sequential phase, left to right); ``REVEAL_RANDOM`` a
  uniformly random set of k open positions, the first-hitting sampler's choice:
  the k smallest uniforms u(b, pos) of the sampling stream (row b, id pos)
  under the step's seed and offset, ties to the lower index.  A row with fewer
  than k open positions reveals all of them.
"""

from __future__ import annotations

import numpy as np

from .sampling import uniforms

REVEAL_CONFIDENCE = 0
REVEAL_LEFTMOST = 1
REVEAL_RANDOM = 2


def mask_budget(n_masked, n_steps, alpha0, seed):
    """Tokens revealed per step for a generation with ``n_masked`` masks.

    Returns (counts, n_diffusion_steps): ``counts`` lists the diffusion steps
    first, then one entry of 1 per sequentially denoised token.
    """
    N, T = int(n_masked), int(n_steps)
    assert N >= 0 and T >= 0 and 0.0 <= float(alpha0) <= 1.0
    if N == 0:
        return np.zeros(0, dtype=np.int64), 0
    if T == 0:
        T = -(-N // 4)
        n_diff = N
    else:
        u = uniforms([0], N, seed, 0)[0]
        n_diff = int(np.count_nonzero(u < float(alpha0)))
    base, extra = divmod(n_diff, T)
    diff = [base + (1 if t < extra else 0) for t in range(T)]
    return np.array(diff + [1] * (N - n_diff), dtype=np.int64), T


def reveal(conf, open_, k, rule=REVEAL_CONFIDENCE, seed=0, offset=0, tokens=None, sample_id=None):
    """Positions revealed at one Mode A step, per batch row.

    conf   [B, N] float32   confidence of each position's drawn token
                            (REVEAL_CONFIDENCE only)
    open_  [B, N] bool      still masked
    k      [B] int          how many to reveal (>= 0)
    tokens [B, N] int, sample_id [B, N] int: optional; the revealed positions
           of ``tokens`` receive their ``sample_id``.

    Returns (order [B, N] int32: revealed positions in reveal order, then -1;
    n [B] int32; open' [B, N] bool; tokens' or None).
    """
    op = np.asarray(open_, dtype=bool)
    B, N = op.shape
    kk = np.asarray(k, dtype=np.int64).reshape(B)
    order = np.full((B, N), -1, dtype=np.int32)
    n = np.zeros(B, dtype=np.int32)
    op2 = op.copy()
    tok = None if tokens is None else np.array(tokens, copy=True)
    if rule == REVEAL_CONFIDENCE:
        c = np.asarray(conf, dtype=np.float32).reshape(B, N).astype(np.float64)
        c = np.where(np.isnan(c), -np.inf, c)
    for b in range(B):
        cand = [i for i in range(N) if op[b, i]]
        if rule == REVEAL_CONFIDENCE:
            cand.sort(key=lambda i: (-c[b, i], i))
        elif rule == REVEAL_LEFTMOST:
            pass  # already in index order
        elif rule == REVEAL_RANDOM:
            u = uniforms([b], N, seed, offset)[0]
            cand.sort(key=lambda i: (u[i], i))
        else:
            raise ValueError(f"unknown rule {rule}")
        pick = cand[: max(0, min(int(kk[b]), len(cand)))]
        order[b, : len(pick)] = pick
        n[b] = len(pick)
        for i in pick:
            op2[b, i] = False
            if tok is not None:
                tok[b, i] = sample_id[b][i]
    return order, n, op2, tok
