// Kernel parameter blocks and launchers of libzarya (host <-> device contract).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace zarya {

// bf16 slot attention.  Rows of a GQA group (G heads x T tokens) are
// contiguous in q and out, so a group is addressed as one [R = G*T, D] block.
struct AttnParams {
  const uint16_t* q;        // [B, Hq, T, D]
  const uint16_t* k_cache;  // [B, Hkv, C, D]
  const uint16_t* v_cache;
  const uint16_t* k_slot;  // [B, Hkv, T, D]
  const uint16_t* v_slot;
  const uint8_t* slot_pass;    // [B, S] or null
  const int32_t* prefix_lens;  // [B] or null (then P for every row)
  uint16_t* out;               // [B, Hq, T, D]
  float* lse;                // [B, Hq, T] or null (natural log)
  float* part_o;             // [n_split, rows_total, D]  (n_split > 1)
  float* part_lse;           // [n_split, rows_total]     (n_split > 1, log2 units)
  int B, Hq, Hkv, P, C, S, L, T, G, R;
  int pass, cross;
  float scale_log2;  // softmax scale * log2(e)
  int n_split, n_rb, tiles_per_split, n_prefix_tiles;
  int per_xcd, n_items;
  int rows_total;      // B * Hq * T
  int rows_per_block;  // kAttnRowsPerBlock or kAttnWideRowsPerBlock
  // causal launch, one split, 8 | B*Hkv: every XCD holds B*Hkv/8 whole
  // groups and takes their row blocks heaviest first
  int heavy_first;
};

struct AttnParams32 {
  const float* q;
  const float* k_cache;
  const float* v_cache;
  const float* k_slot;
  const float* v_slot;
  const uint8_t* slot_pass;
  const int32_t* prefix_lens;
  float* out;
  float* lse;
  int B, Hq, Hkv, P, C, S, L, T, G;
  int pass, cross;
  float scale;
  int rows_total;
};

// LM-head confidence.  Partials are per (vocab group, row): m = max logit,
// s = sum of exp(logit - m), idx = lowest id at the max.
struct ConfParams {
  const void* hidden;   // [M, H]
  const void* w_vocab;  // [V, H]
  int M, H, V;
  int n_vg;        // vocabulary groups (partials per row)
  int n_rt;        // row tiles (bf16 path)
  int per_xcd, n_items;
  float* part_m;   // [M, n_vg]
  float* part_s;   // [M, n_vg]
  int* part_idx;   // [M, n_vg]
  // Gumbel-max sampling (null part_g: no sampling).  Per (row, group): best
  // perturbed score z*log2(e)/T - log2(-log2 u) and its id.  The bf16 path
  // does not track the argmax when sampling (part_idx then holds INT_MAX).
  float* part_g;
  int* part_gi;
  float c2t;  // log2(e) / temperature
  uint32_t seed_lo, seed_hi, off_lo, off_hi;
  // Row selection (null: row i of the output is hidden row i): output row i
  // is hidden row row_index[i] of hidden_rows (clamped into range here; the
  // merge marks out-of-range rows).
  const int32_t* row_index;
  int hidden_rows;
  // bf16 path: W is loaded non-temporally (the hidden rows an XCD's work
  // items re-read fit in its L2 beside the W stream; see kConfXResidentBytes)
  int w_stream;
};

// Hidden row of output row r.
__device__ __forceinline__ int conf_hidden_row(const int32_t* row_index, int hidden_rows, int r) {
  return row_index ? min(max(row_index[r], 0), hidden_rows - 1) : r;
}

struct ConfMergeParams {
  const float* part_m;
  const float* part_s;
  const int* part_idx;
  int n_vg, M, H, V;
  int bf16;
  const void* hidden;
  const void* w_vocab;
  const int32_t* target_ids;
  float* max_prob;
  int32_t* argmax_id;
  float* lse;
  float* target_prob;
  const float* part_g;  // sampling partials, or null
  const int* part_gi;
  int32_t* sample_id;
  float* sample_prob;
  const int32_t* row_index;  // as in ConfParams
  int hidden_rows;
};

struct SelectParams {
  int B, S, L;
  const float* token_conf;
  const uint8_t* slot_open;
  int conf_rule, rule;
  float threshold;
  int k;
  float* slot_conf;
  int32_t* selected;
  int32_t* n_selected;
};

struct AcceptParams {
  int B, S, L;
  const float* token_prob;
  const int32_t* selected;
  float threshold;
  int rule;
  uint8_t* accepted;
  int32_t* n_accepted;
  int32_t* n_total;
};

struct AppendParams {
  int B, Hkv, C, S, L, row_bytes;  // row_bytes = head_dim * element size, a multiple of 16
  const void* k_slot;
  const void* v_slot;
  const uint8_t* accepted;
  const int32_t* order;
  int32_t* prefix_lens;
  void* k_cache;
  void* v_cache;
};

// Mode A reveal: one workgroup per batch row sorts the row's N keys in LDS.
struct RevealParams {
  int B, N, NP;  // NP = N rounded up to a power of two (>= 2)
  int rule;      // 0 confidence, 1 leftmost, 2 random
  const float* conf;
  uint8_t* mask;
  const int32_t* k;
  uint32_t seed_lo, seed_hi, off_lo, off_hi;
  const int32_t* sample_id;
  int32_t* tokens;
  int32_t* order;
  int32_t* n_revealed;
};
constexpr int kRevealMaxN = 8192;

// Mode A mask budget on the host: fills counts (if not null) and returns the
// plan length; *n_diff_steps gets the number of diffusion steps.
int64_t mask_budget_plan(int32_t n_masked, int32_t n_steps, double alpha0, uint64_t seed, int32_t* counts,
                         int32_t* n_diff_steps);

// largest S*L the append kernel stages in LDS
constexpr int kAppendMaxTokens = 8192;

constexpr int kAttnKeysPerTile = 64;
constexpr int kAttnF32RowsPerBlock = 32;    // float32 path: query rows per workgroup (D/16 lanes each)
constexpr int kAttnRowsPerBlock = 128;      // four waves
constexpr int kAttnWideRowsPerBlock = 256;  // eight waves: every K/V tile staged once for 256 rows
// Tile configuration of the bf16 LM-head reduction (measured on MI355X over
// the 0.6B/1.7B/4B shapes): 8 waves over a 256 x 256 tile, 64-deep stages,
// three W and two hidden LDS buffers (160 KB), one workgroup per compute
// unit.  With few rows (a single sequence's draft tokens, the tokens a
// first-hitting step reveals) most of a 256-row tile would be padding and the
// reduction is bound by the W stream instead: 4 waves over a 256 x 64 tile,
// up to 128 rows (the measured crossover).  The vocabulary is split into
// groups until row tiles x groups reaches kConfTargetWGs (one per CU).
constexpr int kConfNW = 8, kConfBR = 256, kConfBK = 64, kConfNSW = 3, kConfNSX = 2;
constexpr int kConfSmallNW = 4, kConfSmallBR = 64, kConfSmallMaxRows = 128;
constexpr int kConfTargetWGs = 256;
// Device scratch of zarya_slot_confidence_noalloc: room for the partials of
// every bf16 call up to 65536 rows (row tiles x vocabulary groups <= 256, 12
// bytes per row and group).
constexpr size_t kConfScratchBytes = (size_t)1 << 20;
// Largest hidden-row footprint per XCD (rows of the row tiles among its work
// items x H x 2 bytes) for which W is loaded non-temporally: up to this size
// the hidden tiles, re-read once per vocab tile, stay in the 4 MB L2 instead
// of being evicted by the W stream (measured on MI355X: at 2 MB the LM head's
// L2-miss traffic falls from 1.61x to 1.11x its algorithmic bytes and the
// kernel gains 2-4%; at 3 MB 1.15x and equal time; from 4 MB the hidden rows
// no longer fit either way and non-temporal W costs traffic and 1% of time).
constexpr size_t kConfXResidentBytes = (size_t)3 << 20;
constexpr int conf_tile_rows(int n_rows) { return n_rows <= kConfSmallMaxRows ? kConfSmallBR : kConfBR; }

hipError_t launch_slot_attn_bf16(const AttnParams& p, int head_dim, hipStream_t stream);
hipError_t launch_slot_attn_f32(const AttnParams32& p, int head_dim, hipStream_t stream);
hipError_t launch_slot_conf_bf16(const ConfParams& p, hipStream_t stream);
hipError_t launch_slot_conf_f32(const ConfParams& p, hipStream_t stream);
hipError_t launch_slot_conf_merge(const ConfMergeParams& p, hipStream_t stream);
hipError_t launch_select_slots(const SelectParams& p, hipStream_t stream);
hipError_t launch_verify_accept(const AcceptParams& p, hipStream_t stream);
hipError_t launch_kv_append(const AppendParams& p, hipStream_t stream);
hipError_t launch_mdm_reveal(const RevealParams& p, hipStream_t stream);

}  // namespace zarya
