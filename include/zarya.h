/*
 * zarya.h -- C ABI of the Zarya slot-scoring step on AMD Instinct MI355X (gfx950).
 *
 * One scoring step of slotted speculative decoding (paper: Zarya, Sec. 5.2,
 * "Mode B: Slotted Speculative Decoding") is
 *
 *   1. zarya_slot_attn        attention of S draft slots x L tokens against the
 *                             reused prefix KV cache (Sec. 5.1 KV-reuse argument,
 *                             Sec. 5.2 draft and verification phases);
 *   2. zarya_slot_confidence  LM-head projection reduced on the fly to per-token
 *                             softmax statistics (Sec. 5.2 "probability of its
 *                             first token"; Table 1 tied embedding);
 *   3. zarya_select_slots     slot confidence and first-hitting slot selection
 *                             (Sec. 5.2 "Slot selection"; Sec. 6 threshold 0.9).
 *
 * and the verification step that follows it (Sec. 5.2 "Verification phase",
 * "KV cache update") adds
 *
 *   4. zarya_verify_accept    token acceptance of the verified slots against the
 *                             token threshold (Sec. 6: 0.4);
 *   5. zarya_kv_append        the accepted tokens' K/V appended to the cache,
 *                             after which the rows of a batch may hold prefixes
 *                             of different lengths (zarya_slot_attn's
 *                             prefix_lens).
 *
 * With a positive temperature the draft tokens are sampled instead of taken
 * greedily (Sec. 5.2 "Sampling from categorical distribution"; Sec. 5.1):
 *
 *   6. zarya_slot_sample      Gumbel-max sampling fused into the LM-head
 *                             reduction of 2.
 *
 * Mode A, MDM sampling with first-hitting denoising (Sec. 5.1), runs the same
 * kernels on a masked tail (zarya_slot_attn with slot_len 1 and cross_slot
 * CAUSAL, then zarya_slot_sample) plus
 *
 *   7. zarya_mdm_budget       host-side plan of how many masks each step
 *                             reveals (Sec. 5.1 step 1);
 *   8. zarya_mdm_reveal       the positions revealed at a step, their tokens
 *                             written and their mask flags cleared.
 *
 * Conventions for every entry point:
 *  - Tensor arguments are DEVICE pointers to dense row-major (C-contiguous)
 *    arrays whose shapes are given in the comments; the caller owns every
 *    buffer, including the workspace.  The library never allocates or frees
 *    device memory and keeps no state between calls.
 *  - Calls only enqueue work on `stream` (0 = the null stream); nothing waits
 *    for the GPU.  Results are ready when the stream is.
 *  - Arguments are validated on the host before anything is launched.  A
 *    non-OK status means nothing was enqueued, except ZARYA_ERR_HIP, which
 *    reports a failed launch.  zarya_last_error() returns a message for the
 *    last non-OK status returned on the calling thread.
 *  - Results are bit-identical from run to run for the same arguments (no
 *    floating-point atomics; every reduction has a fixed order).
 *  - Entry points are reentrant.  Calls that share an output or workspace
 *    buffer must be ordered by the caller (same stream or events).
 */
#ifndef ZARYA_H
#define ZARYA_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ZARYA_VERSION_MAJOR 0
#define ZARYA_VERSION_MINOR 5

typedef enum zarya_status {
  ZARYA_OK = 0,
  ZARYA_ERR_INVALID_ARGUMENT = 1,    /* NULL pointer, bad size, inconsistent shape      */
  ZARYA_ERR_UNSUPPORTED = 2,         /* valid request this build does not implement     */
  ZARYA_ERR_WORKSPACE_TOO_SMALL = 3, /* workspace_bytes below the *_workspace_size value */
  ZARYA_ERR_HIP = 4                  /* a HIP launch or runtime call failed              */
} zarya_status;

typedef enum zarya_dtype {
  ZARYA_DTYPE_F32 = 0,  /* IEEE float32 storage and arithmetic                    */
  ZARYA_DTYPE_BF16 = 1  /* bfloat16 storage, float32 accumulation (Sec. 6: BF16) */
} zarya_dtype;

/* In-slot attention pattern of a pass (Sec. 5.2). */
typedef enum zarya_pass {
  ZARYA_PASS_DIFFUSION = 0, /* draft phase: a token sees every token of its own slot   */
  ZARYA_PASS_AR_INFILL = 1  /* verification phase: a token sees its own slot up to itself */
} zarya_pass;

/* Whether a draft slot sees earlier slots (Sec. 3.1 causal layout). */
typedef enum zarya_cross_slot {
  ZARYA_CROSS_SLOT_NONE = 0,  /* scoring path: prefix + own slot only (slots are parallel) */
  ZARYA_CROSS_SLOT_CAUSAL = 1 /* every earlier slot is visible too (reordered training layout) */
} zarya_cross_slot;

/* ------------------------------------------------------------------------ */
/* 1. Slot-parallel attention against the prefix KV cache                    */
/* ------------------------------------------------------------------------ */
/*
 * Physical order of one sequence (Sec. 5.2 "Reordering": masked tokens follow
 * the unmasked ones): the P_b committed prefix tokens, whose K/V live in the
 * cache, then the draft slots 0..S-1 of L tokens each (T = S*L tokens), whose
 * own K/V are passed separately.  Draft token t = s*L + r (slot s, position r)
 * of query head h (KV head g = h / (Hq/Hkv)) attends to
 *   - every prefix key j < P_b (the cache is read-only; Sec. 5.1 KV reuse),
 *     where P_b = prefix_lens[b] if given, else desc->prefix_len,
 *   - the keys of its own slot: all L of them in the DIFFUSION pass, those at
 *     positions r' <= r in the AR_INFILL pass,
 *   - with cross_slot = CAUSAL, also every key of slots s' < s.
 * Softmax scale `softmax_scale` is applied to q.k before the softmax.
 *
 * Output O[b,h,t,:] = sum_j p_j v_j with p the masked softmax, and
 * lse[b,h,t] = ln(sum_j exp(scale * q.k_j)) over the visible keys (natural log).
 */
typedef struct zarya_slot_attn_desc {
  int32_t batch;         /* B >= 1                                              */
  int32_t n_q_heads;     /* Hq >= 1                                             */
  int32_t n_kv_heads;    /* Hkv >= 1, Hq % Hkv == 0                             */
  int32_t head_dim;      /* D: 64 or 128                                        */
  int32_t prefix_len;    /* P >= 0 valid cache rows (the largest, with prefix_lens) */
  int32_t kv_capacity;   /* C >= P: row count (token stride) of the cache arrays */
  int32_t n_slots;       /* S >= 1                                              */
  int32_t slot_len;      /* L >= 1                                              */
  float softmax_scale;   /* finite, > 0 (1/sqrt(D) in the usual model)          */
  int32_t pass;          /* zarya_pass, used for slots without a slot_pass entry */
  int32_t cross_slot;    /* zarya_cross_slot                                    */
  int32_t dtype;         /* zarya_dtype of q, caches, slot K/V and out          */
  int32_t prefix_splits; /* 0 = library's choice; 1..64 = split the prefix keys
                            into at most this many ranges processed by
                            separate workgroups and merged exactly (results
                            agree to float32 rounding for every choice; the
                            F32 path ignores it)                             */
} zarya_slot_attn_desc;

/* Bytes of device workspace zarya_slot_attn needs for `desc` (may be 0). */
zarya_status zarya_slot_attn_workspace_size(const zarya_slot_attn_desc* desc, size_t* bytes);

/* Work decomposition zarya_slot_attn chooses for `desc` (diagnostics only;
 * nothing is launched).  Host memory `info` is filled on ZARYA_OK. */
typedef struct zarya_slot_attn_plan_info {
  int32_t prefix_splits;      /* ranges of prefix keys given to separate workgroups (1 = none) */
  int32_t rows_per_workgroup; /* query rows (of one GQA group) per workgroup                 */
  int32_t workgroups;         /* workgroups of the attention kernel                          */
  int32_t kernels;            /* kernels one call enqueues                                   */
} zarya_slot_attn_plan_info;

zarya_status zarya_slot_attn_plan(const zarya_slot_attn_desc* desc, zarya_slot_attn_plan_info* info);

/*
 * q         [B, Hq, T, D]  dtype   draft-token queries, T = S*L, row t = s*L + r
 * k_cache   [B, Hkv, C, D] dtype   prefix keys; rows >= P are never read;
 * v_cache   [B, Hkv, C, D] dtype   may be NULL only when P == 0
 * k_slot    [B, Hkv, T, D] dtype   the draft tokens' own keys
 * v_slot    [B, Hkv, T, D] dtype   the draft tokens' own values
 * slot_pass [B, S] uint8 or NULL   per-slot zarya_pass overriding desc->pass
 * prefix_lens [B] int32 or NULL    per-row prefix length P_b (after zarya_kv_append
 *                                  rows differ); values are clamped on the GPU to
 *                                  [0, desc->prefix_len]; NULL = desc->prefix_len
 * out       [B, Hq, T, D]  dtype   attention output (bf16: round to nearest even)
 * lse       [B, Hq, T] float32 or NULL
 * workspace device buffer of at least zarya_slot_attn_workspace_size bytes
 *           (may be NULL when that size is 0); contents on entry do not matter
 *
 * slot_pass entries: 0 = DIFFUSION, any other value = AR_INFILL.
 *
 * ZARYA_ERR_UNSUPPORTED: head_dim not 64 or 128; B*Hq*T or B*Hkv*C at or above 2^31.
 */
zarya_status zarya_slot_attn(const zarya_slot_attn_desc* desc, const void* q, const void* k_cache,
                             const void* v_cache, const void* k_slot, const void* v_slot,
                             const uint8_t* slot_pass, const int32_t* prefix_lens, void* out, float* lse,
                             void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* 2. LM-head confidence: logits = hidden . W^T reduced per row on the fly   */
/* ------------------------------------------------------------------------ */
/*
 * For every row i of `hidden` (rows ordered (b, s, r)) with logits
 * z_v = hidden[i,:] . w_vocab[v,:] over the whole vocabulary v < V:
 *   argmax_id[i]   = the smallest v with z_v = max_v z_v
 *   lse[i]         = ln sum_v exp(z_v)
 *   max_prob[i]    = exp(max_v z_v - lse[i])   (largest softmax probability)
 *   target_prob[i] = exp(z_{target_ids[i]} - lse[i])
 * Logits are computed in float32 and never written to memory.  A row whose
 * logits include a NaN or an infinity (a NaN or infinite value in its hidden
 * state, say) has no softmax -- its log-sum-exp is not finite -- and reports
 * argmax_id -1 and NaN for max_prob, lse and target_prob.
 */
typedef struct zarya_conf_desc {
  int32_t n_rows; /* M >= 1                                              */
  int32_t hidden; /* H >= 1; for BF16 a multiple of 8 and <= 4194304      */
  int32_t vocab;  /* V >= 1                                              */
  int32_t dtype;  /* zarya_dtype of hidden and w_vocab                   */
} zarya_conf_desc;

zarya_status zarya_slot_confidence_workspace_size(const zarya_conf_desc* desc, size_t* bytes);

/*
 * hidden      [M, H] dtype      final hidden states of the draft tokens
 * w_vocab     [V, H] dtype      LM-head weight = tied token embedding (Table 1)
 * target_ids  [M] int32 or NULL ids in [0, V) (checked on the GPU: an id out of
 *                               range gives target_prob = NaN); NULL skips target_prob
 * max_prob    [M] float32       required
 * argmax_id   [M] int32         required
 * lse         [M] float32 or NULL
 * target_prob [M] float32 or NULL (ignored when target_ids is NULL)
 * workspace   at least zarya_slot_confidence_workspace_size bytes
 */
zarya_status zarya_slot_confidence(const zarya_conf_desc* desc, const void* hidden, const void* w_vocab,
                                   const int32_t* target_ids, float* max_prob, int32_t* argmax_id,
                                   float* lse, float* target_prob, void* workspace,
                                   size_t workspace_bytes, hipStream_t stream);

/*
 * zarya_slot_confidence without a workspace, for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc.  Same arguments and results as
 * zarya_slot_confidence (bit-identical); the partials live in a static device
 * array of the library, 1 MiB per GPU (loaded with the library's code, held
 * until the process ends), whose address is looked up on the first call on
 * each device.  Every bf16 call with n_rows <= 65536 fits; a call whose
 * partials need more returns ZARYA_ERR_UNSUPPORTED before anything is
 * launched.  All calls on one GPU share that array: calls that overlap on one
 * GPU (different streams without ordering, or different host threads) race
 * and give wrong results; calls ordered on one stream are safe.  Nothing in
 * the array needs to start at any value.  No device memory is allocated.
 */
zarya_status zarya_slot_confidence_noalloc(const zarya_conf_desc* desc, const void* hidden, const void* w_vocab,
                                           const int32_t* target_ids, float* max_prob, int32_t* argmax_id,
                                           float* lse, float* target_prob, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* 3. First-hitting slot selection                                           */
/* ------------------------------------------------------------------------ */
typedef enum zarya_slot_conf_rule {
  ZARYA_SLOT_CONF_FIRST_TOKEN = 0, /* confidence of the slot's first token (Sec. 5.2) */
  ZARYA_SLOT_CONF_MEAN = 1         /* mean over the slot's L tokens: summed in float64
                                      in token order, divided by L, rounded once to float32 */
} zarya_slot_conf_rule;

typedef enum zarya_select_rule {
  ZARYA_SELECT_THRESHOLD = 0, /* every open slot with confidence > threshold (strict);
                                 if none, the single most confident open slot (Sec. 5.2) */
  ZARYA_SELECT_TOP_K = 1      /* the k most confident open slots                      */
} zarya_select_rule;

/*
 * token_conf  [B, S, L] float32   per-token confidence (max_prob of slot_confidence)
 * slot_open   [B, S] uint8 or NULL  nonzero = slot still undecided; NULL = all open
 * slot_conf   [B, S] float32 out  slot confidence; -1 for closed slots
 * selected    [B, S] int32 out    chosen slot ids in first-hitting order (descending
 *                                 confidence, ties to the lower slot index), then -1
 * n_selected  [B] int32 out       number of chosen slots
 * Comparisons are made between float32 values; `threshold` is used as given.
 * A NaN slot confidence counts as -inf: it ranks after every other open slot
 * (ties among such slots go to the lower index), never exceeds the threshold,
 * and is reported as -inf in slot_conf.
 * Requires 1 <= S <= 1024 and k >= 0 for TOP_K.
 */
zarya_status zarya_select_slots(int32_t batch, int32_t n_slots, int32_t slot_len, const float* token_conf,
                                const uint8_t* slot_open, int32_t conf_rule, int32_t rule, float threshold,
                                int32_t k, float* slot_conf, int32_t* selected, int32_t* n_selected,
                                hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* 4. Verification: token acceptance                                         */
/* ------------------------------------------------------------------------ */
typedef enum zarya_accept_rule {
  ZARYA_ACCEPT_PREFIX = 0,   /* the longest run of passing tokens from the slot's first token:
                                an autoregressive pass scores token r given tokens < r, so a
                                rejected token voids the scores after it                       */
  ZARYA_ACCEPT_PER_TOKEN = 1 /* every passing token on its own                                   */
} zarya_accept_rule;

/*
 * Sec. 5.2 "Verification phase": the selected slots get an autoregressive
 * verification pass (zarya_slot_attn with AR_INFILL, then
 * zarya_slot_confidence with the draft ids as target_ids); a draft token of a
 * verified slot passes when its probability exceeds the token threshold
 * (strict; Sec. 6 uses 0.4).  Tokens of slots not listed in `selected` are
 * rejected.
 *
 * token_prob [B, S, L] float32    probability of each draft token (target_prob)
 * selected   [B, S] int32         verified slots; the first -1 ends the list
 *                                 (zarya_select_slots output); ids outside [0, S)
 *                                 are skipped
 * accepted   [B, S, L] uint8 out  1 = accepted
 * n_accepted [B, S] int32 out     accepted tokens per slot
 * n_total    [B] int32 out or NULL  accepted tokens per batch row
 * Comparisons are made between float32 values.  Requires 1 <= S <= 1024 and
 * 1 <= L <= 4096.
 */
zarya_status zarya_verify_accept(int32_t batch, int32_t n_slots, int32_t slot_len, const float* token_prob,
                                 const int32_t* selected, float token_threshold, int32_t rule,
                                 uint8_t* accepted, int32_t* n_accepted, int32_t* n_total, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* 5. KV-cache update: append the accepted tokens                            */
/* ------------------------------------------------------------------------ */
typedef struct zarya_kv_append_desc {
  int32_t batch;       /* B >= 1                                              */
  int32_t n_kv_heads;  /* Hkv >= 1                                            */
  int32_t head_dim;    /* D: 64 or 128                                        */
  int32_t kv_capacity; /* C: row count (token stride) of the cache arrays     */
  int32_t n_slots;     /* S >= 1                                              */
  int32_t slot_len;    /* L >= 1, S*L <= 8192                                 */
  int32_t dtype;       /* zarya_dtype of the caches and the slot K/V          */
} zarya_kv_append_desc;

/*
 * Sec. 5.2 "KV cache update": accepted tokens join the committed prefix, so
 * they are never recomputed.  For each batch row b the K and V rows of its
 * accepted draft tokens are copied to cache positions prefix_lens[b],
 * prefix_lens[b] + 1, ... -- slots in the order given by `order` (the first -1
 * ends it), positions in slot order -- and prefix_lens[b] grows by their
 * number.  Attention over the cache does not depend on the order of its keys.
 *
 * k_slot, v_slot   [B, Hkv, S*L, D] dtype  the draft tokens' own K/V
 * accepted         [B, S, L] uint8         nonzero = append
 * order            [B, S] int32            slots in append order (e.g. `selected`);
 *                                          ids outside [0, S) are skipped, and
 *                                          so is a slot listed a second time
 *                                          (its tokens are appended once)
 * prefix_lens      [B] int32 in/out
 * k_cache, v_cache [B, Hkv, C, D] dtype in/out
 * A row whose prefix_lens[b] is negative or whose append would pass C is left
 * unchanged, its length included (checked on the GPU).  The slot K/V must not
 * overlap the caches (the copies read and write them concurrently).
 */
zarya_status zarya_kv_append(const zarya_kv_append_desc* desc, const void* k_slot, const void* v_slot,
                             const uint8_t* accepted, const int32_t* order, int32_t* prefix_lens,
                             void* k_cache, void* v_cache, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* 6. Sampled draft tokens: Gumbel-max inside the LM-head reduction          */
/* ------------------------------------------------------------------------ */
/*
 * Sec. 5.2 "Sampling from categorical distribution" (and Sec. 5.1 step 3):
 * with temperature T > 0 each draft token is drawn from softmax(z / T) by
 * Gumbel-max, z_v = hidden[i,:] . w_vocab[v,:]:
 *   sample_id[i]   = argmax_v (z_v / T + G_iv), ties to the smallest v
 *   sample_prob[i] = exp(z_{sample_id[i]} - lse[i])  (model probability at
 *                    T = 1: the drafted token's confidence, Sec. 5.2)
 *   max_prob[i], lse[i] as in zarya_slot_confidence
 * G_iv = -ln(-ln u_iv) with u_iv = ((x >> 9) + 1/2) * 2^-23, where x is word
 * v & 3 of the Philox4x32-10 block (Salmon et al., SC 2011) with counter
 * (v >> 2, i, offset_lo, offset_hi) and key (seed_lo, seed_hi) -- 32-bit
 * halves of `seed` and `offset`.  The stream is fully determined by (seed,
 * offset, i, v): advance `offset` between draft steps for fresh noise.  The
 * perturbed scores are compared in float32 (in base 2:
 * z log2(e) / T - log2(-log2 u), the same order).  Logits are never written to
 * memory.  A row whose logits include a NaN or an infinity has no
 * distribution to draw from: sample_id -1, NaN sample_prob, max_prob and lse.
 */
typedef struct zarya_sample_params {
  float temperature; /* T: finite, > 0                                      */
  uint64_t seed;     /* Philox key                                          */
  uint64_t offset;   /* Philox counter words 2 and 3                        */
} zarya_sample_params;

zarya_status zarya_slot_sample_workspace_size(const zarya_conf_desc* desc, size_t* bytes);

/*
 * hidden      [M, H] dtype, or [hidden_rows, H] with row_index
 * row_index   [M] int32 or NULL: output row i samples hidden row row_index[i]
 *             (the first-hitting sampler draws only the positions it reveals);
 *             an index outside [0, hidden_rows) gives sample_id -1 and NaN
 *             probabilities for that row (checked on the GPU).  The random
 *             stream's row is the output row i in both cases.
 * hidden_rows rows of hidden when row_index is given (ignored otherwise)
 * w_vocab     [V, H] dtype
 * sample_id   [M] int32       required
 * sample_prob [M] float32     required
 * max_prob    [M] float32 or NULL
 * lse         [M] float32 or NULL
 * workspace   at least zarya_slot_sample_workspace_size bytes
 * M = desc->n_rows.  Requires 1/T <= 1e30 (T not denormal-small).
 */
zarya_status zarya_slot_sample(const zarya_conf_desc* desc, const zarya_sample_params* params, const void* hidden,
                               const int32_t* row_index, int32_t hidden_rows, const void* w_vocab,
                               int32_t* sample_id, float* sample_prob, float* max_prob, float* lse, void* workspace,
                               size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* 7. Mode A: mask budget (host)                                             */
/* ------------------------------------------------------------------------ */
/*
 * Sec. 5.1 step 1 "Mask budget planning" for a generation with n_masked masks.
 * n_steps T > 0: n_diff ~ Binomial(n_masked, alpha0) tokens go through exactly
 * T diffusion steps, spread as evenly as possible (the first n_diff mod T
 * steps take one more; steps may reveal 0), then n_masked - n_diff sequential
 * steps reveal one token each.  T = 0: the binomial draw is skipped, T =
 * ceil(n_masked / 4) and every token goes through diffusion.  The binomial
 * draw counts the i < n_masked with u_i < alpha0 (in double), u_i the uniform
 * of row 0, id i, offset 0 of the Philox stream of zarya_slot_sample under
 * key `seed`.
 *
 * counts             HOST int32 [capacity] out: tokens revealed per step,
 *                    diffusion steps first; NULL only asks for the length
 * n_plan_steps       HOST out: number of steps of the plan (required)
 * n_diffusion_steps  HOST out or NULL
 * Requires n_masked >= 0, n_steps >= 0, 0 <= alpha0 <= 1, capacity >= the plan
 * length when counts is given.  Runs on the host only; touches no device.
 */
zarya_status zarya_mdm_budget(int32_t n_masked, int32_t n_steps, double alpha0, uint64_t seed, int32_t* counts,
                              int32_t capacity, int32_t* n_plan_steps, int32_t* n_diffusion_steps);

/* ------------------------------------------------------------------------ */
/* 8. Mode A: positions revealed at a denoising step                         */
/* ------------------------------------------------------------------------ */
typedef enum zarya_reveal_rule {
  ZARYA_REVEAL_CONFIDENCE = 0, /* the k most confident open positions: descending conf,
                                  ties to the lower index, NaN as -inf                   */
  ZARYA_REVEAL_LEFTMOST = 1,   /* the k lowest open positions (sequential phase)          */
  ZARYA_REVEAL_RANDOM = 2      /* a uniformly random k-subset (first-hitting sampler): the
                                  k smallest uniforms u(b, pos) of the zarya_slot_sample
                                  stream (row b, id pos) under seed/offset, ties to the
                                  lower index                                            */
} zarya_reveal_rule;

/*
 * For each batch row b, reveal min(k[b], open count) of the N positions whose
 * mask flag is set (Sec. 5.1 steps 2-3: revealed tokens join the committed part
 * of the sequence, the rest stay masked).
 *
 * conf       [B, N] float32     confidence of each position's drawn token
 *                               (sample_prob); used by CONFIDENCE, else may be NULL
 * mask       [B, N] uint8 in/out  nonzero = still masked; cleared where revealed
 * k          [B] int32          tokens to reveal in row b (negative counts as 0)
 * sample_id  [B, N] int32 or NULL  drawn token of each position
 * tokens     [B, N] int32 in/out or NULL  receives sample_id at revealed
 *                               positions (both or neither of the two)
 * order      [B, N] int32 out   revealed positions in reveal order, then -1
 * n_revealed [B] int32 out or NULL
 * Requires 1 <= N <= 8192.  Integer work: bit-identical to the rule.
 */
zarya_status zarya_mdm_reveal(int32_t batch, int32_t n, const float* conf, uint8_t* mask, const int32_t* k,
                              int32_t rule, uint64_t seed, uint64_t offset, const int32_t* sample_id, int32_t* tokens,
                              int32_t* order, int32_t* n_revealed, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Diagnostics                                                               */
/* ------------------------------------------------------------------------ */
/* Static name of a status code; never NULL. */
const char* zarya_status_string(zarya_status status);
/* Message for the last non-OK status returned on this thread ("" if none).
   The pointer stays valid until the next zarya_* call on the same thread. */
const char* zarya_last_error(void);
/* ZARYA_VERSION_MAJOR * 1000 + ZARYA_VERSION_MINOR of the built library. */
int32_t zarya_version(void);

#ifdef __cplusplus
}
#endif

#endif /* ZARYA_H */
