// Host-side checks of libzarya's C ABI, built with AddressSanitizer and
// UndefinedBehaviorSanitizer on the host code (tests/test_host_sanitize.py).
//
// The library's host sources (argument validation, work planning, parameter
// set-up, the Mode A budget) are linked against stub launchers that launch
// nothing: they check the parameters the host code built -- the partial
// arrays lie inside the caller's workspace, the work decomposition covers the
// problem -- and report a launch failure, so every valid call must come back
// as ZARYA_ERR_HIP with a message.  Device pointers are fake addresses that
// nothing dereferences; no GPU is touched.
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <string>
#include <vector>

#include "kernels.hpp"
#include "zarya.h"

static int g_fail = 0;
static int g_checks = 0;
#define CHECK(c)                                                        \
  do {                                                                  \
    ++g_checks;                                                         \
    if (!(c)) {                                                         \
      std::printf("FAIL %s:%d: %s\n", __FILE__, __LINE__, #c);          \
      ++g_fail;                                                         \
    }                                                                   \
  } while (0)

// The fake workspace of the current call: [lo, hi).
static uintptr_t g_ws_lo = 0, g_ws_hi = 0;
static bool in_ws(const void* p, size_t bytes) {
  const uintptr_t a = reinterpret_cast<uintptr_t>(p);
  return a >= g_ws_lo && a + bytes <= g_ws_hi;
}
static int g_launches = 0;

namespace zarya {
static AttnParams g_last_attn;  // the parameters of the last bf16 attention launch

hipError_t launch_slot_attn_bf16(const AttnParams& p, int head_dim, hipStream_t) {
  ++g_launches;
  g_last_attn = p;
  CHECK(p.n_split >= 1 && p.n_split <= 64);
  CHECK((int64_t)p.tiles_per_split * p.n_split >= p.n_prefix_tiles);
  CHECK(p.n_split == 1 || (int64_t)p.tiles_per_split * (p.n_split - 1) < p.n_prefix_tiles);
  CHECK(p.rows_per_block == kAttnRowsPerBlock || p.rows_per_block == kAttnWideRowsPerBlock);
  CHECK((int64_t)p.n_rb * p.rows_per_block >= p.R && (int64_t)(p.n_rb - 1) * p.rows_per_block < p.R &&
        p.R == p.G * p.T);
  CHECK(p.n_items == p.B * p.Hkv * p.n_split * p.n_rb);
  // heavy-first dispatch only where every XCD holds whole groups of one split
  CHECK(!p.heavy_first || (p.cross == 1 && p.n_split == 1 && (p.B * p.Hkv) % 8 == 0 && p.per_xcd * 8 == p.n_items &&
                           p.per_xcd % p.n_rb == 0));
  CHECK(p.per_xcd * 8 >= p.n_items && (p.per_xcd - 1) * 8 < p.n_items);
  if (p.n_split > 1) {
    CHECK(in_ws(p.part_o, (size_t)p.n_split * p.rows_total * head_dim * 4));
    CHECK(in_ws(p.part_lse, (size_t)p.n_split * p.rows_total * 4));
    CHECK(reinterpret_cast<uintptr_t>(p.part_lse) >=
          reinterpret_cast<uintptr_t>(p.part_o) + (size_t)p.n_split * p.rows_total * head_dim * 4);
  }
  return hipErrorNoDevice;
}

hipError_t launch_slot_attn_f32(const AttnParams32& p, int, hipStream_t) {
  ++g_launches;
  CHECK(p.rows_total == p.B * p.Hq * p.T);
  return hipErrorNoDevice;
}

static void check_conf(const ConfParams& p) {
  const size_t n = (size_t)p.n_vg * p.M * 4;
  CHECK(in_ws(p.part_m, n) && in_ws(p.part_s, n) && in_ws(p.part_idx, n));
  if (p.part_g) CHECK(in_ws(p.part_g, n) && in_ws(p.part_gi, n));
  CHECK(p.n_vg >= 1);
  CHECK(p.n_items == p.n_vg * p.n_rt);
  CHECK(p.per_xcd * 8 >= p.n_items);
  CHECK(p.row_index != nullptr || p.hidden_rows == p.M);
}

static ConfParams g_last_conf;  // the parameters of the last bf16 LM-head launch

hipError_t launch_slot_conf_bf16(const ConfParams& p, hipStream_t) {
  ++g_launches;
  g_last_conf = p;
  check_conf(p);
  CHECK(p.w_stream == 0 || p.w_stream == 1);
  CHECK((int64_t)p.n_rt * conf_tile_rows(p.M) >= p.M);
  CHECK(p.n_vg <= (p.V + 31) / 32);
  return hipErrorNoDevice;
}

hipError_t launch_slot_conf_f32(const ConfParams& p, hipStream_t) {
  ++g_launches;
  check_conf(p);
  CHECK(p.n_rt == 1 && p.n_vg <= 64);
  return hipErrorNoDevice;
}

hipError_t launch_slot_conf_merge(const ConfMergeParams&, hipStream_t) { return hipErrorNoDevice; }

hipError_t launch_select_slots(const SelectParams&, hipStream_t) {
  ++g_launches;
  return hipErrorNoDevice;
}

hipError_t launch_verify_accept(const AcceptParams& p, hipStream_t) {
  ++g_launches;
  CHECK(p.S >= 1 && p.S <= 1024 && p.L >= 1);
  return hipErrorNoDevice;
}

hipError_t launch_kv_append(const AppendParams& p, hipStream_t) {
  ++g_launches;
  CHECK(p.row_bytes % 16 == 0 && p.S * p.L <= kAppendMaxTokens);
  return hipErrorNoDevice;
}

hipError_t launch_mdm_reveal(const RevealParams& p, hipStream_t) {
  ++g_launches;
  CHECK(p.NP >= p.N && p.NP >= 2 && (p.NP & (p.NP - 1)) == 0 && p.NP <= kRevealMaxN);
  CHECK(p.NP < 2 * p.N || p.NP == 2);
  return hipErrorNoDevice;
}

}  // namespace zarya

static void* fake(uintptr_t a) { return reinterpret_cast<void*>(a); }

// A valid call must reach its launcher and report the launch failure.
static void expect_launch(zarya_status st, int launches_before, const char* what) {
  if (st != ZARYA_ERR_HIP || g_launches != launches_before + 1 || std::strlen(zarya_last_error()) == 0) {
    std::printf("FAIL %s: status %s, launches %d -> %d\n", what, zarya_status_string(st), launches_before,
                g_launches);
    ++g_fail;
  }
  ++g_checks;
}

static void attn_cases(std::mt19937_64& rng) {
  const int dims[2] = {64, 128};
  for (int it = 0; it < 400; ++it) {
    zarya_slot_attn_desc d{};
    d.batch = 1 + (int)(rng() % 32);
    d.n_kv_heads = 1 + (int)(rng() % 8);
    d.n_q_heads = d.n_kv_heads * (1 + (int)(rng() % 4));
    d.head_dim = dims[rng() % 2];
    d.prefix_len = (rng() % 4 == 0) ? 0 : (int)(rng() % 20000);
    d.kv_capacity = d.prefix_len + (int)(rng() % 300);
    d.n_slots = 1 + (int)(rng() % 64);
    d.slot_len = 1 + (int)(rng() % 32);
    d.softmax_scale = 0.088f;
    d.pass = (int)(rng() % 2);
    d.cross_slot = (int)(rng() % 2);
    d.dtype = (rng() % 5 == 0) ? ZARYA_DTYPE_F32 : ZARYA_DTYPE_BF16;
    d.prefix_splits = (rng() % 3 == 0) ? (int)(rng() % 9) : 0;
    size_t ws = 0;
    CHECK(zarya_slot_attn_workspace_size(&d, &ws) == ZARYA_OK);
    g_ws_lo = 0x100000000ull;
    g_ws_hi = g_ws_lo + ws;
    void* p = fake(0x200000000ull);
    const int before = g_launches;
    expect_launch(zarya_slot_attn(&d, p, p, p, p, p, nullptr, nullptr, p, nullptr, ws ? fake(g_ws_lo) : nullptr, ws,
                                  nullptr),
                  before, "slot_attn");
    if (ws > 0) {
      CHECK(zarya_slot_attn(&d, p, p, p, p, p, nullptr, nullptr, p, nullptr, fake(g_ws_lo), ws - 1, nullptr) ==
            ZARYA_ERR_WORKSPACE_TOO_SMALL);
    }
  }
}

// The work decomposition the planner picks for the named workloads (rows per
// workgroup, row blocks, prefix splits): 256-row blocks only where they add no
// padding and the prefix dominates, two splits per group where that reaches
// about one workgroup per compute unit, and a doubling for 128-row blocks on
// long prefixes.
static void named_plans() {
  struct Case {
    const char* name;
    int B, Hq, Hkv, P, S, L, cross;
    int rows_per_block, n_rb, n_split;
  };
  const Case cases[] = {
      {"qwen0.6b", 16, 16, 8, 2048, 8, 8, 0, 128, 1, 2},
      {"qwen1.7b", 32, 16, 8, 4096, 16, 4, 0, 128, 1, 1},
      {"qwen4b", 8, 32, 8, 16384, 8, 16, 0, 256, 2, 2},
      {"qwen4b with 17-token slots: 128-row blocks pad less", 8, 32, 8, 16384, 8, 17, 0, 128, 5, 2},
      {"qwen0.6b batch 1", 1, 16, 8, 2048, 8, 8, 0, 128, 1, 8},
      {"layout", 8, 16, 8, 0, 128, 32, 1, 128, 64, 1},
      {"modeA", 16, 16, 8, 2048, 260, 1, 1, 128, 5, 1},
      {"128-row blocks, 256 prefix tiles: two splits doubled", 16, 16, 8, 16384, 8, 8, 0, 128, 1, 4},
      {"128-row blocks, 128 prefix tiles: two splits kept", 16, 16, 8, 8192, 8, 8, 0, 128, 1, 2},
  };
  for (const Case& c : cases) {
    zarya_slot_attn_desc d{};
    d.batch = c.B;
    d.n_q_heads = c.Hq;
    d.n_kv_heads = c.Hkv;
    d.head_dim = 128;
    d.prefix_len = c.P;
    d.kv_capacity = c.P;
    d.n_slots = c.S;
    d.slot_len = c.L;
    d.softmax_scale = 0.088f;
    d.pass = 0;
    d.cross_slot = c.cross;
    d.dtype = ZARYA_DTYPE_BF16;
    size_t ws = 0;
    CHECK(zarya_slot_attn_workspace_size(&d, &ws) == ZARYA_OK);
    g_ws_lo = 0x100000000ull;
    g_ws_hi = g_ws_lo + ws;
    void* p = fake(0x200000000ull);
    const int before = g_launches;
    expect_launch(zarya_slot_attn(&d, p, p, p, p, p, nullptr, nullptr, p, nullptr, ws ? fake(g_ws_lo) : nullptr, ws,
                                  nullptr),
                  before, c.name);
    const zarya::AttnParams& a = zarya::g_last_attn;
    // the causal launches over 8 x 8 groups (training layout) and 16 x 8
    // (Mode A) dispatch heaviest first
    const bool hf = std::string(c.name) == "layout" || std::string(c.name) == "modeA";
    if ((a.heavy_first != 0) != hf) {
      std::printf("FAIL plan %s: heavy_first %d\n", c.name, a.heavy_first);
      ++g_fail;
    }
    if (a.rows_per_block != c.rows_per_block || a.n_rb != c.n_rb || a.n_split != c.n_split) {
      std::printf("FAIL plan %s: rows/block %d, row blocks %d, splits %d (expected %d, %d, %d)\n", c.name,
                  a.rows_per_block, a.n_rb, a.n_split, c.rows_per_block, c.n_rb, c.n_split);
      ++g_fail;
    }
    ++g_checks;
  }
}

static void conf_cases(std::mt19937_64& rng) {
  for (int it = 0; it < 400; ++it) {
    zarya_conf_desc d{};
    d.dtype = (rng() % 4 == 0) ? ZARYA_DTYPE_F32 : ZARYA_DTYPE_BF16;
    d.n_rows = 1 + (int)(rng() % 5000);
    d.hidden = 8 * (1 + (int)(rng() % 512));
    d.vocab = 1 + (int)(rng() % 200000);
    size_t ws = 0, ws_s = 0;
    CHECK(zarya_slot_confidence_workspace_size(&d, &ws) == ZARYA_OK);
    CHECK(zarya_slot_sample_workspace_size(&d, &ws_s) == ZARYA_OK && ws_s > ws);
    void* p = fake(0x200000000ull);
    g_ws_lo = 0x100000000ull;
    g_ws_hi = g_ws_lo + ws;
    int before = g_launches;
    expect_launch(zarya_slot_confidence(&d, p, p, nullptr, (float*)p, (int32_t*)p, nullptr, nullptr, fake(g_ws_lo),
                                        ws, nullptr),
                  before, "slot_confidence");
    CHECK(zarya_slot_confidence(&d, p, p, nullptr, (float*)p, (int32_t*)p, nullptr, nullptr, fake(g_ws_lo), ws - 1,
                                nullptr) == ZARYA_ERR_WORKSPACE_TOO_SMALL);
    g_ws_hi = g_ws_lo + ws_s;
    zarya_sample_params sp{0.7f, 12345, 6};
    const bool rows = rng() % 2 == 0;
    before = g_launches;
    expect_launch(zarya_slot_sample(&d, &sp, p, rows ? (const int32_t*)p : nullptr, rows ? 1 + (int)(rng() % 9000) : 0,
                                    p, (int32_t*)p, (float*)p, nullptr, nullptr, fake(g_ws_lo), ws_s, nullptr),
                  before, "slot_sample");
  }
}

static void small_call_cases() {
  void* p = fake(0x300000000ull);
  int before = g_launches;
  expect_launch(zarya_select_slots(4, 1024, 3, (const float*)p, nullptr, 1, 1, 0.9f, 5, (float*)p, (int32_t*)p,
                                   (int32_t*)p, nullptr),
                before, "select_slots");
  before = g_launches;
  expect_launch(zarya_verify_accept(4, 1024, 4096, (const float*)p, (const int32_t*)p, 0.4f, 0, (uint8_t*)p,
                                    (int32_t*)p, nullptr, nullptr),
                before, "verify_accept");
  zarya_kv_append_desc a{2, 8, 128, 4096, 64, 128, ZARYA_DTYPE_BF16};
  before = g_launches;
  expect_launch(zarya_kv_append(&a, p, p, (const uint8_t*)p, (const int32_t*)p, (int32_t*)p, p, p, nullptr), before,
                "kv_append");
  for (int n : {1, 2, 3, 64, 65, 4097, 8192}) {
    for (int rule = 0; rule < 3; ++rule) {
      before = g_launches;
      expect_launch(zarya_mdm_reveal(3, n, (const float*)p, (uint8_t*)p, (const int32_t*)p, rule, 1, 2, nullptr,
                                     nullptr, (int32_t*)p, nullptr, nullptr),
                    before, "mdm_reveal");
    }
  }
  // rejected before any launch
  before = g_launches;
  CHECK(zarya_mdm_reveal(3, 8193, (const float*)p, (uint8_t*)p, (const int32_t*)p, 0, 1, 2, nullptr, nullptr,
                         (int32_t*)p, nullptr, nullptr) == ZARYA_ERR_UNSUPPORTED);
  CHECK(zarya_select_slots(4, 1025, 3, (const float*)p, nullptr, 0, 0, 0.9f, 1, (float*)p, (int32_t*)p, (int32_t*)p,
                           nullptr) == ZARYA_ERR_UNSUPPORTED);
  zarya_kv_append_desc big{2, 8, 128, 4096, 512, 32, ZARYA_DTYPE_BF16};
  CHECK(zarya_kv_append(&big, p, p, (const uint8_t*)p, (const int32_t*)p, (int32_t*)p, p, p, nullptr) ==
        ZARYA_ERR_UNSUPPORTED);
  CHECK(g_launches == before);
}

// The plan is written into a buffer of exactly the reported length, so any
// write past it is caught by the sanitizer.
static void budget_cases(std::mt19937_64& rng) {
  for (int it = 0; it < 300; ++it) {
    const int n = (int)(rng() % 3000);
    const int t = (int)(rng() % 40);
    const double a = (double)(rng() % 1001) / 1000.0;
    const uint64_t seed = rng();
    int32_t len = -1, diff = -1;
    CHECK(zarya_mdm_budget(n, t, a, seed, nullptr, 0, &len, &diff) == ZARYA_OK);
    std::vector<int32_t>* buf = new std::vector<int32_t>((size_t)len);
    int32_t len2 = -1;
    CHECK(zarya_mdm_budget(n, t, a, seed, buf->data(), len, &len2, &diff) == ZARYA_OK && len2 == len);
    long long sum = 0;
    for (int32_t c : *buf) sum += c;
    CHECK(sum == n);
    CHECK(diff == (n == 0 ? 0 : (t > 0 ? t : (n + 3) / 4)));
    if (len > 0) CHECK(zarya_mdm_budget(n, t, a, seed, buf->data(), len - 1, &len2, &diff) == ZARYA_ERR_INVALID_ARGUMENT);
    delete buf;
  }
}

// W is loaded non-temporally exactly when the hidden rows among one XCD's
// work items (all of them for every shape here: each XCD holds whole vocab
// groups) fit in 3 MB: the 0.6B-scale head (1024 x 1024: 2 MB) and single
// sequences, not the 1.7B (2048 x 2048) or 4B (1024 x 2560) heads.
static void conf_named_plans() {
  struct Case {
    int M, H, w_stream;
  };
  const Case cases[] = {{1024, 1024, 1}, {2048, 2048, 0}, {1024, 2560, 0}, {1024, 1536, 1}, {1024, 2048, 0},
                        {64, 1024, 1},   {128, 2560, 1},  {2048, 1024, 0}};
  for (const Case& c : cases) {
    zarya_conf_desc d{};
    d.n_rows = c.M;
    d.hidden = c.H;
    d.vocab = 151936;
    d.dtype = ZARYA_DTYPE_BF16;
    size_t ws = 0;
    CHECK(zarya_slot_confidence_workspace_size(&d, &ws) == ZARYA_OK);
    g_ws_lo = 0x100000000ull;
    g_ws_hi = g_ws_lo + ws;
    void* p = fake(0x200000000ull);
    const int before = g_launches;
    expect_launch(zarya_slot_confidence(&d, p, p, nullptr, (float*)p, (int32_t*)p, nullptr, nullptr, fake(g_ws_lo), ws,
                                        nullptr),
                  before, "conf named plan");
    if (zarya::g_last_conf.w_stream != c.w_stream) {
      std::printf("FAIL conf plan %d x %d: w_stream %d (expected %d)\n", c.M, c.H, zarya::g_last_conf.w_stream,
                  c.w_stream);
      ++g_fail;
    }
    ++g_checks;
  }
}

int main() {
  std::mt19937_64 rng(20260);
  attn_cases(rng);
  named_plans();
  conf_named_plans();
  conf_cases(rng);
  small_call_cases();
  budget_cases(rng);
  std::printf("%d checks, %d failures, %d launches reached\n", g_checks, g_fail, g_launches);
  return g_fail == 0 ? 0 : 1;
}
