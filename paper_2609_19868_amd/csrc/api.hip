// Host side of the libzarya C ABI: argument validation, workspace sizing,
// work decomposition and kernel launches.  Nothing is launched unless every
// argument passes validation.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>

#include <algorithm>
#include <cmath>
#include <mutex>
#include <string>

#include "kernels.hpp"
#include "zarya.h"

using namespace zarya;

// Partials of zarya_slot_confidence_noalloc.  Every GPU the library runs on
// holds its own copy (allocated when the code object is loaded, kept until
// the process ends).  In host code this name is a host-side stand-in, not a
// device address: the device address comes from hipGetSymbolAddress.
static __device__ __align__(256) uint8_t scratch[kConfScratchBytes];

namespace {

thread_local std::string g_last_error;

zarya_status fail(zarya_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

zarya_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return ZARYA_OK;
  return fail(ZARYA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

constexpr int64_t kI32Max = 2147483647;

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// ------------------------------------------------------------- attention plan

struct AttnPlan {
  int T, G, R;
  int n_split, tiles_per_split, n_prefix_tiles, n_rb, rows_per_block;
  int64_t rows_total;
  size_t ws_bytes;
};

zarya_status check_attn_desc(const zarya_slot_attn_desc* d) {
  if (!d) return fail(ZARYA_ERR_INVALID_ARGUMENT, "desc is NULL");
  if (d->batch < 1 || d->n_q_heads < 1 || d->n_kv_heads < 1)
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "batch, n_q_heads and n_kv_heads must be >= 1");
  if (d->n_q_heads % d->n_kv_heads != 0)
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "n_q_heads (%d) is not a multiple of n_kv_heads (%d)", d->n_q_heads,
                d->n_kv_heads);
  if (d->prefix_len < 0) return fail(ZARYA_ERR_INVALID_ARGUMENT, "prefix_len must be >= 0");
  if (d->kv_capacity < d->prefix_len)
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "kv_capacity (%d) < prefix_len (%d)", d->kv_capacity, d->prefix_len);
  if (d->n_slots < 1 || d->slot_len < 1) return fail(ZARYA_ERR_INVALID_ARGUMENT, "n_slots and slot_len must be >= 1");
  if (!(isfinite(d->softmax_scale) && d->softmax_scale > 0.f))
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "softmax_scale must be finite and > 0");
  if (d->pass != ZARYA_PASS_DIFFUSION && d->pass != ZARYA_PASS_AR_INFILL)
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "unknown pass %d", d->pass);
  if (d->cross_slot != ZARYA_CROSS_SLOT_NONE && d->cross_slot != ZARYA_CROSS_SLOT_CAUSAL)
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "unknown cross_slot %d", d->cross_slot);
  if (d->dtype != ZARYA_DTYPE_F32 && d->dtype != ZARYA_DTYPE_BF16)
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "unknown dtype %d", d->dtype);
  if (d->prefix_splits < 0 || d->prefix_splits > 64)
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "prefix_splits must be in [0, 64]");
  if (d->head_dim != 64 && d->head_dim != 128)
    return fail(ZARYA_ERR_UNSUPPORTED, "head_dim %d is not supported (64 or 128)", d->head_dim);
  const int64_t T = (int64_t)d->n_slots * d->slot_len;
  const int64_t rows = (int64_t)d->batch * d->n_q_heads * T;
  const int64_t cache_rows = (int64_t)d->batch * d->n_kv_heads * d->kv_capacity;
  if (T > kI32Max || rows > kI32Max || cache_rows > kI32Max)
    return fail(ZARYA_ERR_UNSUPPORTED, "problem too large: batch*heads*tokens must stay below 2^31");
  return ZARYA_OK;
}

AttnPlan plan_attn(const zarya_slot_attn_desc* d) {
  AttnPlan pl{};
  pl.T = d->n_slots * d->slot_len;
  pl.G = d->n_q_heads / d->n_kv_heads;
  pl.R = pl.G * pl.T;
  pl.rows_total = (int64_t)d->batch * d->n_q_heads * pl.T;
  pl.n_prefix_tiles = (d->prefix_len + kAttnKeysPerTile - 1) / kAttnKeysPerTile;
  // 256-row workgroups (each K/V tile staged once for twice the rows) when
  // they add no padding waves over 128-row ones and the prefix holds at least
  // as many key tiles as the draft tokens (4B shape: 358 against 372-379 us;
  // on the 4096-token training layout, all draft tokens under a causal mask,
  // they are 6% slower)
  const int n_narrow = (pl.R + kAttnRowsPerBlock - 1) / kAttnRowsPerBlock;
  const int n_wide = (pl.R + kAttnWideRowsPerBlock - 1) / kAttnWideRowsPerBlock;
  const bool wide = d->dtype == ZARYA_DTYPE_BF16 && 2 * n_wide <= n_narrow &&
                    (int64_t)pl.n_prefix_tiles * kAttnKeysPerTile >= pl.T;
  pl.rows_per_block = wide ? kAttnWideRowsPerBlock : kAttnRowsPerBlock;
  pl.n_rb = wide ? n_wide : n_narrow;
  int ns = 1;
  if (d->dtype == ZARYA_DTYPE_BF16 && pl.n_prefix_tiles > 0) {
    if (d->prefix_splits > 0) {
      ns = d->prefix_splits;
    } else {
      // aim for about one workgroup per compute unit (measured best on the
      // 0.6B/1.7B/4B shapes), with at least two key tiles per split so the
      // partial traffic stays small, and at most 8 splits: past that the
      // merge of the partials costs more than the extra workgroups save
      // (single-sequence batches: 8 splits 19.7 us, 16 splits 22.9 us)
      const int64_t base = (int64_t)d->batch * d->n_kv_heads * pl.n_rb;
      int64_t want = (256 + base - 1) / base;
      // long prefixes: two workgroups per compute unit when every split
      // still walks at least 64 key tiles, so that one workgroup's softmax
      // overlaps the other's MFMAs (4B shape, 256 tiles: 383 us with two
      // splits against 424-435 us with one; at 64 tiles the extra split
      // costs more than it overlaps)
      // (256-row workgroups already hold two waves per SIMD and fit once per
      // compute unit)
      if (pl.rows_per_block == kAttnRowsPerBlock && pl.n_prefix_tiles >= 128 * want) want *= 2;
      ns = (int)std::min<int64_t>(8, std::max<int64_t>(1, want));
      ns = std::max(1, std::min(ns, pl.n_prefix_tiles / 2));
    }
    ns = std::min(ns, pl.n_prefix_tiles);
    pl.tiles_per_split = (pl.n_prefix_tiles + ns - 1) / ns;
    ns = (pl.n_prefix_tiles + pl.tiles_per_split - 1) / pl.tiles_per_split;
  } else {
    pl.tiles_per_split = pl.n_prefix_tiles;
  }
  pl.n_split = ns;
  pl.ws_bytes = 0;
  if (ns > 1) {
    pl.ws_bytes = align256((size_t)ns * pl.rows_total * d->head_dim * 4) + align256((size_t)ns * pl.rows_total * 4);
  }
  return pl;
}

// ------------------------------------------------------------ confidence plan

struct ConfPlan {
  int n_vg, n_rt;
  size_t ws_bytes;
};

zarya_status check_conf_desc(const zarya_conf_desc* d) {
  if (!d) return fail(ZARYA_ERR_INVALID_ARGUMENT, "desc is NULL");
  if (d->n_rows < 1 || d->hidden < 1 || d->vocab < 1)
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "n_rows, hidden and vocab must be >= 1");
  if (d->dtype != ZARYA_DTYPE_F32 && d->dtype != ZARYA_DTYPE_BF16)
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "unknown dtype %d", d->dtype);
  if (d->dtype == ZARYA_DTYPE_BF16 && d->hidden % 8 != 0)
    return fail(ZARYA_ERR_UNSUPPORTED, "bf16 hidden size %d is not a multiple of 8", d->hidden);
  // a 256-row W tile is addressed with 32-bit byte offsets
  if (d->dtype == ZARYA_DTYPE_BF16 && d->hidden > 4194304)
    return fail(ZARYA_ERR_UNSUPPORTED, "bf16 hidden size %d exceeds 4194304", d->hidden);
  if (d->dtype == ZARYA_DTYPE_F32 && d->hidden > 8192)
    return fail(ZARYA_ERR_UNSUPPORTED, "f32 hidden size %d exceeds 8192", d->hidden);
  if (d->dtype == ZARYA_DTYPE_F32 && d->n_rows > 65535)
    return fail(ZARYA_ERR_UNSUPPORTED, "f32 path supports at most 65535 rows");
  if ((int64_t)d->n_rows * d->hidden * 2 >= ((int64_t)1 << 32))
    return fail(ZARYA_ERR_UNSUPPORTED, "hidden states of %lld bytes exceed 4 GiB",
                (long long)d->n_rows * d->hidden * 2);
  return ZARYA_OK;
}

ConfPlan plan_conf(const zarya_conf_desc* d) {
  ConfPlan pl{};
  if (d->dtype == ZARYA_DTYPE_BF16) {
    const int br = conf_tile_rows(d->n_rows);
    pl.n_rt = (d->n_rows + br - 1) / br;
    const int nblk = (d->vocab + 31) / 32;
    // split the vocabulary so that row tiles x vocabulary groups reaches the
    // workgroup count the kernel is tuned for
    pl.n_vg = std::max(1, std::min(nblk, kConfTargetWGs / pl.n_rt));
  } else {
    pl.n_rt = 1;
    pl.n_vg = std::max(1, std::min(64, d->vocab / 2048));
  }
  pl.ws_bytes = 3 * align256((size_t)pl.n_vg * d->n_rows * 4);
  return pl;
}

// Sampling keeps two more partial arrays (best perturbed score and its id).
size_t sample_ws_bytes(const zarya_conf_desc* d) {
  const ConfPlan pl = plan_conf(d);
  return pl.ws_bytes + 2 * align256((size_t)pl.n_vg * d->n_rows * 4);
}

// Device address of `scratch` on the current device, looked up once per
// device (with that device current) and kept.
constexpr int kMaxDevices = 256;
void* g_scratch_addr[kMaxDevices];
std::mutex g_scratch_mutex;

zarya_status current_device_scratch(void** addr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(ZARYA_ERR_UNSUPPORTED, "device index %d", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_status(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(ZARYA_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_addr[dev] = p;
  }
  *addr = g_scratch_addr[dev];
  return ZARYA_OK;
}

// Enqueues the LM-head reduction and its merge; with `sp` also the sampling.
// Arguments are already validated.
zarya_status run_conf(const zarya_conf_desc* d, const zarya_sample_params* sp, const void* hidden,
                      const int32_t* row_index, int32_t hidden_rows, const void* w_vocab, const int32_t* target_ids,
                      float* max_prob, int32_t* argmax_id, float* lse, float* target_prob, int32_t* sample_id,
                      float* sample_prob, void* workspace, hipStream_t stream) {
  const ConfPlan pl = plan_conf(d);
  (void)hipGetLastError();
  const size_t part = align256((size_t)pl.n_vg * d->n_rows * 4);
  char* ws = static_cast<char*>(workspace);
  ConfParams p{};
  p.hidden = hidden;
  p.w_vocab = w_vocab;
  p.M = d->n_rows;
  p.H = d->hidden;
  p.V = d->vocab;
  p.n_vg = pl.n_vg;
  p.n_rt = pl.n_rt;
  p.n_items = pl.n_vg * pl.n_rt;
  p.per_xcd = (p.n_items + 7) / 8;
  p.part_m = reinterpret_cast<float*>(ws);
  p.part_s = reinterpret_cast<float*>(ws + part);
  p.part_idx = reinterpret_cast<int*>(ws + 2 * part);
  p.row_index = row_index;
  p.hidden_rows = hidden_rows;
  if (d->dtype == ZARYA_DTYPE_BF16) {
    // the row tiles present among one XCD's work items (a contiguous run of
    // per_xcd items, row tile fastest) and the hidden rows they re-read
    const int64_t br = conf_tile_rows(d->n_rows);
    const int64_t rows_on_xcd = std::min<int64_t>(d->n_rows, std::min(pl.n_rt, p.per_xcd) * br);
    p.w_stream = (size_t)rows_on_xcd * d->hidden * 2 <= kConfXResidentBytes ? 1 : 0;
  }
  if (sp) {
    p.part_g = reinterpret_cast<float*>(ws + 3 * part);
    p.part_gi = reinterpret_cast<int*>(ws + 4 * part);
    p.c2t = (float)(1.4426950408889634 / (double)sp->temperature);
    p.seed_lo = (uint32_t)sp->seed;
    p.seed_hi = (uint32_t)(sp->seed >> 32);
    p.off_lo = (uint32_t)sp->offset;
    p.off_hi = (uint32_t)(sp->offset >> 32);
  }
  hipError_t e = d->dtype == ZARYA_DTYPE_BF16 ? launch_slot_conf_bf16(p, stream) : launch_slot_conf_f32(p, stream);
  if (e != hipSuccess) return hip_status(e, "LM-head reduction launch");

  ConfMergeParams mp{};
  mp.part_m = p.part_m;
  mp.part_s = p.part_s;
  mp.part_idx = p.part_idx;
  mp.n_vg = pl.n_vg;
  mp.M = d->n_rows;
  mp.H = d->hidden;
  mp.V = d->vocab;
  mp.bf16 = d->dtype == ZARYA_DTYPE_BF16;
  mp.hidden = hidden;
  mp.w_vocab = w_vocab;
  mp.target_ids = target_ids;
  mp.max_prob = max_prob;
  mp.argmax_id = argmax_id;
  mp.lse = lse;
  mp.target_prob = target_prob;
  mp.part_g = p.part_g;
  mp.part_gi = p.part_gi;
  mp.sample_id = sample_id;
  mp.sample_prob = sample_prob;
  mp.row_index = row_index;
  mp.hidden_rows = hidden_rows;
  return hip_status(launch_slot_conf_merge(mp, stream), "LM-head merge launch");
}

}  // namespace

extern "C" {

const char* zarya_status_string(zarya_status s) {
  switch (s) {
    case ZARYA_OK: return "ZARYA_OK";
    case ZARYA_ERR_INVALID_ARGUMENT: return "ZARYA_ERR_INVALID_ARGUMENT";
    case ZARYA_ERR_UNSUPPORTED: return "ZARYA_ERR_UNSUPPORTED";
    case ZARYA_ERR_WORKSPACE_TOO_SMALL: return "ZARYA_ERR_WORKSPACE_TOO_SMALL";
    case ZARYA_ERR_HIP: return "ZARYA_ERR_HIP";
  }
  return "ZARYA_STATUS_UNKNOWN";
}

const char* zarya_last_error(void) { return g_last_error.c_str(); }

int32_t zarya_version(void) { return ZARYA_VERSION_MAJOR * 1000 + ZARYA_VERSION_MINOR; }

zarya_status zarya_slot_attn_workspace_size(const zarya_slot_attn_desc* desc, size_t* bytes) {
  if (!bytes) return fail(ZARYA_ERR_INVALID_ARGUMENT, "bytes is NULL");
  zarya_status st = check_attn_desc(desc);
  if (st != ZARYA_OK) return st;
  *bytes = plan_attn(desc).ws_bytes;
  return ZARYA_OK;
}

zarya_status zarya_slot_attn_plan(const zarya_slot_attn_desc* desc, zarya_slot_attn_plan_info* info) {
  if (!info) return fail(ZARYA_ERR_INVALID_ARGUMENT, "info is NULL");
  zarya_status st = check_attn_desc(desc);
  if (st != ZARYA_OK) return st;
  const AttnPlan pl = plan_attn(desc);
  if (desc->dtype == ZARYA_DTYPE_F32) {
    info->prefix_splits = 1;
    info->rows_per_workgroup = kAttnF32RowsPerBlock;
    info->workgroups = (int32_t)((pl.rows_total + kAttnF32RowsPerBlock - 1) / kAttnF32RowsPerBlock);
    info->kernels = 1;
    return ZARYA_OK;
  }
  info->prefix_splits = pl.n_split;
  info->rows_per_workgroup = pl.rows_per_block;
  info->workgroups = (int32_t)((int64_t)desc->batch * desc->n_kv_heads * pl.n_split * pl.n_rb);
  info->kernels = pl.n_split > 1 ? 2 : 1;
  return ZARYA_OK;
}

zarya_status zarya_slot_attn(const zarya_slot_attn_desc* d, const void* q, const void* k_cache, const void* v_cache,
                             const void* k_slot, const void* v_slot, const uint8_t* slot_pass,
                             const int32_t* prefix_lens, void* out, float* lse, void* workspace,
                             size_t workspace_bytes, hipStream_t stream) {
  zarya_status st = check_attn_desc(d);
  if (st != ZARYA_OK) return st;
  if (!q || !k_slot || !v_slot || !out) return fail(ZARYA_ERR_INVALID_ARGUMENT, "q, k_slot, v_slot and out are required");
  if (d->prefix_len > 0 && (!k_cache || !v_cache))
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "k_cache and v_cache are required when prefix_len > 0");
  const AttnPlan pl = plan_attn(d);
  if (workspace_bytes < pl.ws_bytes)
    return fail(ZARYA_ERR_WORKSPACE_TOO_SMALL, "workspace of %zu bytes is below the %zu required", workspace_bytes,
                pl.ws_bytes);
  if (pl.ws_bytes > 0 && !workspace) return fail(ZARYA_ERR_INVALID_ARGUMENT, "workspace is NULL");
  (void)hipGetLastError();  // drop a stale error so the status below is ours

  if (d->dtype == ZARYA_DTYPE_F32) {
    AttnParams32 p{};
    p.q = static_cast<const float*>(q);
    p.k_cache = static_cast<const float*>(k_cache);
    p.v_cache = static_cast<const float*>(v_cache);
    p.k_slot = static_cast<const float*>(k_slot);
    p.v_slot = static_cast<const float*>(v_slot);
    p.slot_pass = slot_pass;
    p.prefix_lens = prefix_lens;
    p.out = static_cast<float*>(out);
    p.lse = lse;
    p.B = d->batch;
    p.Hq = d->n_q_heads;
    p.Hkv = d->n_kv_heads;
    p.P = d->prefix_len;
    p.C = d->kv_capacity;
    p.S = d->n_slots;
    p.L = d->slot_len;
    p.T = pl.T;
    p.G = pl.G;
    p.pass = d->pass;
    p.cross = d->cross_slot;
    p.scale = d->softmax_scale;
    p.rows_total = (int)pl.rows_total;
    return hip_status(launch_slot_attn_f32(p, d->head_dim, stream), "slot_attn f32 launch");
  }

  AttnParams p{};
  p.q = static_cast<const uint16_t*>(q);
  p.k_cache = static_cast<const uint16_t*>(k_cache);
  p.v_cache = static_cast<const uint16_t*>(v_cache);
  p.k_slot = static_cast<const uint16_t*>(k_slot);
  p.v_slot = static_cast<const uint16_t*>(v_slot);
  p.slot_pass = slot_pass;
  p.prefix_lens = prefix_lens;
  p.out = static_cast<uint16_t*>(out);
  p.lse = lse;
  if (pl.n_split > 1) {
    p.part_o = static_cast<float*>(workspace);
    p.part_lse = reinterpret_cast<float*>(static_cast<char*>(workspace) +
                                          align256((size_t)pl.n_split * pl.rows_total * d->head_dim * 4));
  }
  p.B = d->batch;
  p.Hq = d->n_q_heads;
  p.Hkv = d->n_kv_heads;
  p.P = d->prefix_len;
  p.C = d->kv_capacity;
  p.S = d->n_slots;
  p.L = d->slot_len;
  p.T = pl.T;
  p.G = pl.G;
  p.R = pl.R;
  p.pass = d->pass;
  p.cross = d->cross_slot;
  p.scale_log2 = d->softmax_scale * 1.4426950408889634f;
  p.n_split = pl.n_split;
  p.n_rb = pl.n_rb;
  p.tiles_per_split = pl.tiles_per_split;
  p.n_prefix_tiles = pl.n_prefix_tiles;
  const int64_t items = (int64_t)d->batch * d->n_kv_heads * pl.n_split * pl.n_rb;
  if (items > kI32Max / 2) return fail(ZARYA_ERR_UNSUPPORTED, "too many workgroups");
  p.n_items = (int)items;
  p.per_xcd = (p.n_items + 7) / 8;
  p.rows_total = (int)pl.rows_total;
  p.rows_per_block = pl.rows_per_block;
  // with a causal cross-slot order the row blocks' key ranges grow with
  // their tokens: dispatch the longest first where the grid allows it
  const int64_t n_bg = (int64_t)d->batch * d->n_kv_heads;
  p.heavy_first = d->cross_slot == ZARYA_CROSS_SLOT_CAUSAL && pl.n_split == 1 && n_bg % 8 == 0;
  return hip_status(launch_slot_attn_bf16(p, d->head_dim, stream), "slot_attn bf16 launch");
}

zarya_status zarya_slot_confidence_workspace_size(const zarya_conf_desc* desc, size_t* bytes) {
  if (!bytes) return fail(ZARYA_ERR_INVALID_ARGUMENT, "bytes is NULL");
  zarya_status st = check_conf_desc(desc);
  if (st != ZARYA_OK) return st;
  *bytes = plan_conf(desc).ws_bytes;
  return ZARYA_OK;
}

zarya_status zarya_slot_confidence(const zarya_conf_desc* d, const void* hidden, const void* w_vocab,
                                   const int32_t* target_ids, float* max_prob, int32_t* argmax_id, float* lse,
                                   float* target_prob, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  zarya_status st = check_conf_desc(d);
  if (st != ZARYA_OK) return st;
  if (!hidden || !w_vocab || !max_prob || !argmax_id)
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "hidden, w_vocab, max_prob and argmax_id are required");
  const ConfPlan pl = plan_conf(d);
  if (workspace_bytes < pl.ws_bytes)
    return fail(ZARYA_ERR_WORKSPACE_TOO_SMALL, "workspace of %zu bytes is below the %zu required", workspace_bytes,
                pl.ws_bytes);
  if (!workspace) return fail(ZARYA_ERR_INVALID_ARGUMENT, "workspace is NULL");
  return run_conf(d, nullptr, hidden, nullptr, d->n_rows, w_vocab, target_ids, max_prob, argmax_id, lse, target_prob,
                  nullptr, nullptr, workspace, stream);
}

zarya_status zarya_slot_confidence_noalloc(const zarya_conf_desc* d, const void* hidden, const void* w_vocab,
                                           const int32_t* target_ids, float* max_prob, int32_t* argmax_id,
                                           float* lse, float* target_prob, hipStream_t stream) {
  zarya_status st = check_conf_desc(d);
  if (st != ZARYA_OK) return st;
  if (!hidden || !w_vocab || !max_prob || !argmax_id)
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "hidden, w_vocab, max_prob and argmax_id are required");
  const ConfPlan pl = plan_conf(d);
  if (pl.ws_bytes > kConfScratchBytes)
    return fail(ZARYA_ERR_UNSUPPORTED, "the partials of this call need %zu bytes; the library's scratch holds %zu",
                pl.ws_bytes, kConfScratchBytes);
  void* ws = nullptr;
  st = current_device_scratch(&ws);
  if (st != ZARYA_OK) return st;
  return run_conf(d, nullptr, hidden, nullptr, d->n_rows, w_vocab, target_ids, max_prob, argmax_id, lse, target_prob,
                  nullptr, nullptr, ws, stream);
}

zarya_status zarya_slot_sample_workspace_size(const zarya_conf_desc* desc, size_t* bytes) {
  if (!bytes) return fail(ZARYA_ERR_INVALID_ARGUMENT, "bytes is NULL");
  zarya_status st = check_conf_desc(desc);
  if (st != ZARYA_OK) return st;
  *bytes = sample_ws_bytes(desc);
  return ZARYA_OK;
}

zarya_status zarya_slot_sample(const zarya_conf_desc* d, const zarya_sample_params* sp, const void* hidden,
                               const int32_t* row_index, int32_t hidden_rows, const void* w_vocab, int32_t* sample_id,
                               float* sample_prob, float* max_prob, float* lse, void* workspace,
                               size_t workspace_bytes, hipStream_t stream) {
  zarya_status st = check_conf_desc(d);
  if (st != ZARYA_OK) return st;
  if (!sp) return fail(ZARYA_ERR_INVALID_ARGUMENT, "params is NULL");
  const float T = sp->temperature;
  if (!(T > 0.f) || !std::isfinite(T) || !(1.0 / (double)T <= 1e30))
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "temperature %g must be finite, > 0 and >= 1e-30", (double)T);
  if (!hidden || !w_vocab || !sample_id || !sample_prob)
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "hidden, w_vocab, sample_id and sample_prob are required");
  if (row_index) {
    if (hidden_rows < 1) return fail(ZARYA_ERR_INVALID_ARGUMENT, "hidden_rows must be >= 1 with a row_index");
    if ((int64_t)hidden_rows * d->hidden * 2 >= ((int64_t)1 << 32))
      return fail(ZARYA_ERR_UNSUPPORTED, "hidden states of %lld bytes exceed 4 GiB",
                  (long long)hidden_rows * d->hidden * 2);
  } else {
    hidden_rows = d->n_rows;
  }
  const size_t need = sample_ws_bytes(d);
  if (workspace_bytes < need)
    return fail(ZARYA_ERR_WORKSPACE_TOO_SMALL, "workspace of %zu bytes is below the %zu required", workspace_bytes,
                need);
  if (!workspace) return fail(ZARYA_ERR_INVALID_ARGUMENT, "workspace is NULL");
  return run_conf(d, sp, hidden, row_index, hidden_rows, w_vocab, nullptr, max_prob, nullptr, lse, nullptr, sample_id,
                  sample_prob, workspace, stream);
}

zarya_status zarya_mdm_budget(int32_t n_masked, int32_t n_steps, double alpha0, uint64_t seed, int32_t* counts,
                              int32_t capacity, int32_t* n_plan_steps, int32_t* n_diffusion_steps) {
  if (n_masked < 0 || n_steps < 0)
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "n_masked (%d) and n_steps (%d) must be >= 0", n_masked, n_steps);
  if (!(alpha0 >= 0.0 && alpha0 <= 1.0)) return fail(ZARYA_ERR_INVALID_ARGUMENT, "alpha0 %g is not in [0, 1]", alpha0);
  if (!n_plan_steps) return fail(ZARYA_ERR_INVALID_ARGUMENT, "n_plan_steps is NULL");
  int32_t t = 0;
  const int64_t len = mask_budget_plan(n_masked, n_steps, alpha0, seed, nullptr, &t);
  if (len > kI32Max) return fail(ZARYA_ERR_UNSUPPORTED, "plan of %lld steps", (long long)len);
  if (counts) {
    if (capacity < len)
      return fail(ZARYA_ERR_INVALID_ARGUMENT, "counts holds %d steps, the plan has %lld", capacity, (long long)len);
    mask_budget_plan(n_masked, n_steps, alpha0, seed, counts, &t);
  }
  *n_plan_steps = (int32_t)len;
  if (n_diffusion_steps) *n_diffusion_steps = t;
  return ZARYA_OK;
}

zarya_status zarya_mdm_reveal(int32_t batch, int32_t n, const float* conf, uint8_t* mask, const int32_t* k,
                              int32_t rule, uint64_t seed, uint64_t offset, const int32_t* sample_id, int32_t* tokens,
                              int32_t* order, int32_t* n_revealed, hipStream_t stream) {
  if (batch < 1 || n < 1) return fail(ZARYA_ERR_INVALID_ARGUMENT, "batch and n must be >= 1");
  if (n > kRevealMaxN) return fail(ZARYA_ERR_UNSUPPORTED, "n %d exceeds %d", n, kRevealMaxN);
  if (rule != ZARYA_REVEAL_CONFIDENCE && rule != ZARYA_REVEAL_LEFTMOST && rule != ZARYA_REVEAL_RANDOM)
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "unknown reveal rule %d", rule);
  if (!mask || !k || !order) return fail(ZARYA_ERR_INVALID_ARGUMENT, "mask, k and order are required");
  if (rule == ZARYA_REVEAL_CONFIDENCE && !conf)
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "the confidence rule needs conf");
  if ((tokens == nullptr) != (sample_id == nullptr))
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "tokens and sample_id go together");
  if ((int64_t)batch * n > kI32Max) return fail(ZARYA_ERR_UNSUPPORTED, "batch * n exceeds 2^31");
  (void)hipGetLastError();
  RevealParams p{};
  p.B = batch;
  p.N = n;
  p.NP = 2;
  while (p.NP < n) p.NP <<= 1;
  p.rule = rule;
  p.conf = conf;
  p.mask = mask;
  p.k = k;
  p.seed_lo = (uint32_t)seed;
  p.seed_hi = (uint32_t)(seed >> 32);
  p.off_lo = (uint32_t)offset;
  p.off_hi = (uint32_t)(offset >> 32);
  p.sample_id = sample_id;
  p.tokens = tokens;
  p.order = order;
  p.n_revealed = n_revealed;
  return hip_status(launch_mdm_reveal(p, stream), "mdm_reveal launch");
}

zarya_status zarya_select_slots(int32_t batch, int32_t n_slots, int32_t slot_len, const float* token_conf,
                                const uint8_t* slot_open, int32_t conf_rule, int32_t rule, float threshold, int32_t k,
                                float* slot_conf, int32_t* selected, int32_t* n_selected, hipStream_t stream) {
  if (batch < 1 || batch > 65535) return fail(ZARYA_ERR_INVALID_ARGUMENT, "batch must be in [1, 65535]");
  if (n_slots < 1) return fail(ZARYA_ERR_INVALID_ARGUMENT, "n_slots must be >= 1");
  if (n_slots > 1024) return fail(ZARYA_ERR_UNSUPPORTED, "n_slots %d exceeds 1024", n_slots);
  if (slot_len < 1) return fail(ZARYA_ERR_INVALID_ARGUMENT, "slot_len must be >= 1");
  if (conf_rule != ZARYA_SLOT_CONF_FIRST_TOKEN && conf_rule != ZARYA_SLOT_CONF_MEAN)
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "unknown conf_rule %d", conf_rule);
  if (rule != ZARYA_SELECT_THRESHOLD && rule != ZARYA_SELECT_TOP_K)
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "unknown rule %d", rule);
  if (rule == ZARYA_SELECT_TOP_K && k < 0) return fail(ZARYA_ERR_INVALID_ARGUMENT, "k must be >= 0");
  if (!token_conf || !slot_conf || !selected || !n_selected)
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "token_conf, slot_conf, selected and n_selected are required");
  (void)hipGetLastError();
  SelectParams p{};
  p.B = batch;
  p.S = n_slots;
  p.L = slot_len;
  p.token_conf = token_conf;
  p.slot_open = slot_open;
  p.conf_rule = conf_rule;
  p.rule = rule;
  p.threshold = threshold;
  p.k = k;
  p.slot_conf = slot_conf;
  p.selected = selected;
  p.n_selected = n_selected;
  return hip_status(launch_select_slots(p, stream), "select_slots launch");
}

zarya_status zarya_verify_accept(int32_t batch, int32_t n_slots, int32_t slot_len, const float* token_prob,
                                 const int32_t* selected, float token_threshold, int32_t rule, uint8_t* accepted,
                                 int32_t* n_accepted, int32_t* n_total, hipStream_t stream) {
  if (batch < 1 || batch > 65535) return fail(ZARYA_ERR_INVALID_ARGUMENT, "batch must be in [1, 65535]");
  if (n_slots < 1 || slot_len < 1) return fail(ZARYA_ERR_INVALID_ARGUMENT, "n_slots and slot_len must be >= 1");
  if (n_slots > 1024) return fail(ZARYA_ERR_UNSUPPORTED, "n_slots %d exceeds 1024", n_slots);
  if (slot_len > 4096) return fail(ZARYA_ERR_UNSUPPORTED, "slot_len %d exceeds 4096", slot_len);
  if (rule != ZARYA_ACCEPT_PREFIX && rule != ZARYA_ACCEPT_PER_TOKEN)
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "unknown acceptance rule %d", rule);
  if (isnan(token_threshold)) return fail(ZARYA_ERR_INVALID_ARGUMENT, "token_threshold is NaN");
  if (!token_prob || !selected || !accepted || !n_accepted)
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "token_prob, selected, accepted and n_accepted are required");
  (void)hipGetLastError();
  AcceptParams p{};
  p.B = batch;
  p.S = n_slots;
  p.L = slot_len;
  p.token_prob = token_prob;
  p.selected = selected;
  p.threshold = token_threshold;
  p.rule = rule;
  p.accepted = accepted;
  p.n_accepted = n_accepted;
  p.n_total = n_total;
  return hip_status(launch_verify_accept(p, stream), "verify_accept launch");
}

zarya_status zarya_kv_append(const zarya_kv_append_desc* d, const void* k_slot, const void* v_slot,
                             const uint8_t* accepted, const int32_t* order, int32_t* prefix_lens, void* k_cache,
                             void* v_cache, hipStream_t stream) {
  if (!d) return fail(ZARYA_ERR_INVALID_ARGUMENT, "desc is NULL");
  if (d->batch < 1 || d->batch > 65535) return fail(ZARYA_ERR_INVALID_ARGUMENT, "batch must be in [1, 65535]");
  if (d->n_kv_heads < 1 || d->n_slots < 1 || d->slot_len < 1 || d->kv_capacity < 0)
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "n_kv_heads, n_slots and slot_len must be >= 1, kv_capacity >= 0");
  if (d->dtype != ZARYA_DTYPE_F32 && d->dtype != ZARYA_DTYPE_BF16)
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "unknown dtype %d", d->dtype);
  if (d->head_dim != 64 && d->head_dim != 128)
    return fail(ZARYA_ERR_UNSUPPORTED, "head_dim %d is not supported (64 or 128)", d->head_dim);
  if (d->n_slots > 1024) return fail(ZARYA_ERR_UNSUPPORTED, "n_slots %d exceeds 1024", d->n_slots);
  if ((int64_t)d->n_slots * d->slot_len > kAppendMaxTokens)
    return fail(ZARYA_ERR_UNSUPPORTED, "n_slots * slot_len exceeds %d", kAppendMaxTokens);
  if ((int64_t)d->batch * d->n_kv_heads * std::max<int64_t>(d->kv_capacity, (int64_t)d->n_slots * d->slot_len) >
      kI32Max)
    return fail(ZARYA_ERR_UNSUPPORTED, "problem too large: batch*heads*tokens must stay below 2^31");
  if (!k_slot || !v_slot || !accepted || !order || !prefix_lens || !k_cache || !v_cache)
    return fail(ZARYA_ERR_INVALID_ARGUMENT, "every tensor argument is required");
  (void)hipGetLastError();
  AppendParams p{};
  p.B = d->batch;
  p.Hkv = d->n_kv_heads;
  p.C = d->kv_capacity;
  p.S = d->n_slots;
  p.L = d->slot_len;
  p.row_bytes = d->head_dim * (d->dtype == ZARYA_DTYPE_BF16 ? 2 : 4);
  p.k_slot = k_slot;
  p.v_slot = v_slot;
  p.accepted = accepted;
  p.order = order;
  p.prefix_lens = prefix_lens;
  p.k_cache = k_cache;
  p.v_cache = v_cache;
  return hip_status(launch_kv_append(p, stream), "kv_append launch");
}

}  // extern "C"
