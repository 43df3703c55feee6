"""Float64 CPU oracle for the Zarya slot-scoring step.

TEST INFRASTRUCTURE ONLY. Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package. The product path (the
HIP library and its Python binding) never imports, calls or links anything
here, and nothing here imports the product path.

What it computes, each function citing the passage of the paper it follows
(Sinev, Koziev, Leshchuk, "Zarya: A Hybrid Autoregressive--Masked Diffusion
Language Model with Flexible Training and Dual-Mode Inference"):

* ``attention``   -- masked softmax attention of S draft slots x L tokens
  against a reused prefix KV cache (Sec. 5.1 KV-reuse argument, Sec. 5.2
  draft and verification phases, Sec. 3.1 causal masked reconstruction).
* ``confidence``  -- full-vocabulary softmax statistics of the LM head
  (Sec. 5.2: a slot's confidence is its first token's probability; Table 1
  tied embedding).
* ``selection``   -- slot confidence and first-hitting slot selection
  (Sec. 5.2 slot selection, Sec. 6 inference settings).
* ``sampling``    -- Gumbel-max sampling with temperature from a Philox4x32-10
  stream (Sec. 5.2 "Sampling from categorical distribution", Sec. 5.1 step 3).
* ``verify``      -- token acceptance after the verification pass and the
  KV-cache append of the accepted tokens (Sec. 5.2 "Verification phase",
  "KV cache update").
* ``mdm``         -- Mode A: the mask budget of a generation and the positions
  revealed at a denoising step (Sec. 5.1 steps 1-3).

Every function is the plain definition written out in float64 numpy; there is
no blocking, fusion or reordering beyond what the definition states.
"""

from .attention import (
    PASS_DIFFUSION,
    PASS_AR_INFILL,
    CROSS_SLOT_NONE,
    CROSS_SLOT_CAUSAL,
    visibility,
    prefix_lengths,
    slot_attention,
    slot_attention_loops,
)
from .confidence import slot_confidence, slot_confidence_loops
from .selection import (
    CONF_FIRST_TOKEN,
    CONF_MEAN,
    SELECT_THRESHOLD,
    SELECT_TOP_K,
    slot_conf,
    select_slots,
)

from .sampling import gumbel, philox4x32, slot_sample, uniforms
from .verify import ACCEPT_PREFIX, ACCEPT_PER_TOKEN, accept_tokens, kv_append
from .mdm import REVEAL_CONFIDENCE, REVEAL_LEFTMOST, REVEAL_RANDOM, mask_budget, reveal

__all__ = [
    "PASS_DIFFUSION",
    "PASS_AR_INFILL",
    "CROSS_SLOT_NONE",
    "CROSS_SLOT_CAUSAL",
    "visibility",
    "slot_attention",
    "slot_attention_loops",
    "slot_confidence",
    "slot_confidence_loops",
    "CONF_FIRST_TOKEN",
    "CONF_MEAN",
    "SELECT_THRESHOLD",
    "SELECT_TOP_K",
    "slot_conf",
    "select_slots",
    "prefix_lengths",
    "ACCEPT_PREFIX",
    "ACCEPT_PER_TOKEN",
    "accept_tokens",
    "kv_append",
    "philox4x32",
    "uniforms",
    "gumbel",
    "slot_sample",
    "REVEAL_CONFIDENCE",
    "REVEAL_LEFTMOST",
    "REVEAL_RANDOM",
    "mask_budget",
    "reveal",
]
