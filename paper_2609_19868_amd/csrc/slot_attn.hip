// Slot-parallel attention against a reused prefix KV cache (gfx950).
//
// What is computed (Zarya, Sec. 5.1 KV-reuse argument and Sec. 5.2 draft /
// verification phases): every draft token t = s*L + r of query head h attends
// to all P prefix keys of KV head g = h / G and to a contiguous range of the
// draft tokens' own keys -- its own slot (all of it in the DIFFUSION pass, up
// to itself in the AR_INFILL pass), preceded by every earlier slot when
// cross_slot = CAUSAL.
//
// bf16 kernel design (one workgroup = 4 or 8 waves = up to 128 or 256 query
// rows of one GQA group, i.e. G heads x T tokens flattened token-major, so a
// block holds every head of a contiguous token range; one split of the
// prefix keys):
//  * K/V tiles of 64 keys are staged in LDS once and shared by every query
//    row of the group (the prefix is read from HBM once per group and split).
//  * Scores are computed transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16:
//    each lane then owns one query row, so the online-softmax row statistics
//    need a single cross-lane exchange (lane ^ 32) per tile.
//  * O^T += V^T P^T reuses the score accumulators directly as the B operand
//    (the MFMA k-order is chosen to match the accumulator layout); V^T is read
//    from the row-major LDS tile with ds_read_b64_tr_b16.
//  * LDS rows are XOR-swizzled in 16-byte chunks so that both the row reads of
//    K and the transposing reads of V are free of bank conflicts.
//  * The prefix is split into `n_split` ranges handled by separate workgroups
//    (split-K, flash-decoding style); each writes a float32 partial (O, LSE)
//    and a merge kernel combines them exactly.  With one split the kernel
//    writes the final bf16 output itself.  The draft tokens' own keys are
//    processed by the last split, with the mask applied per element.
#include "common.hpp"
#include "kernels.hpp"

namespace zarya {

#ifndef ZARYA_ATTN_NS
#define ZARYA_ATTN_NS 2  // LDS stages of the bf16 kernel (2 x 32 KB: two workgroups per CU)
#endif
#ifndef ZARYA_ATTN_WPE
#define ZARYA_ATTN_WPE 2  // waves per SIMD the register budget is sized for
#endif

namespace {

constexpr int KT = 64;          // keys per tile
constexpr float kRescaleLog2 = 8.f;  // growth of a row maximum (log2 units) that forces a rescale

// XOR swizzle of the 16-byte chunk index of LDS row `kr` (D = 128: 16 chunks
// per row; D = 64: 8).  Any 16 consecutive rows (the rows one pass of a
// K-fragment ds_read_b128 serves) get distinct bank groups, and the aligned
// chunk pairs of 4 consecutive rows (one transposing V read) stay aligned
// pairs on distinct banks: the pair index takes the low row bits, the chunk's
// low bit the next one.
template <int D>
__host__ __device__ constexpr int swz(int kr) {
  if constexpr (D == 128) {
    return ((kr & 7) << 1) | ((kr >> 3) & 1);
  } else {
    return (((kr >> 1) & 3) << 1) | ((kr >> 3) & 1);
  }
}

}  // namespace

// NS: LDS stages (prefetch distance NS - 1 tiles).  NWAVE: waves per
// workgroup, 32 query rows each; every wave stages its share of each K/V tile.
template <int D, int NS, int NWAVE>
__global__ __launch_bounds__(NWAVE * 64) __attribute__((amdgpu_waves_per_eu(ZARYA_ATTN_WPE))) void slot_attn_bf16_kernel(AttnParams p) {
  constexpr int RB = NWAVE * 32;        // query rows per workgroup
  constexpr int ROWB = D * 2;           // bytes per key row
  constexpr int TILEB = KT * ROWB;      // bytes of one K (or V) tile
  constexpr int CPW = TILEB / 1024 / NWAVE;  // 1 KB direct loads per wave per tile (K; same for V)
  constexpr int LPR = ROWB / 16;        // lanes per row in a direct load
  constexpr int RPC = 1024 / ROWB;      // rows per 1 KB chunk
  constexpr int NDB = D / 32;           // 32-wide blocks of the head dim
  constexpr int NKS = D / 16;           // k-steps of the QK^T contraction
  constexpr int LPT = 2 * CPW;          // direct loads per wave per tile
  static_assert(CPW * NWAVE * 1024 == TILEB, "tile must split into 1 KB chunks per wave");
  __shared__ __attribute__((aligned(16))) uint8_t lds[NS][2][TILEB];

  int rb, split, bg;  // row block, prefix split, b * Hkv + g
  if (p.heavy_first) {
    // Causal launch whose XCDs each hold whole GQA groups (one split): an
    // XCD walks its groups' row blocks heaviest first (the last tokens see
    // the most keys), so the longest work items start first and the short
    // ones fill the tail.
    const int x = blockIdx.x & 7, k = blockIdx.x >> 3;
    const int gpx = p.per_xcd / p.n_rb;  // groups per XCD
    rb = p.n_rb - 1 - k / gpx;
    split = 0;
    bg = x * gpx + k % gpx;
  } else {
    const int w = xcd_work_index(blockIdx.x, p.per_xcd, p.n_items);
    if (w < 0) return;
    rb = w % p.n_rb;
    split = (w / p.n_rb) % p.n_split;
    bg = w / (p.n_rb * p.n_split);
  }
  const int b = bg / p.Hkv;
  // this batch row's prefix length (rows differ after KV-cache appends)
  const int Pb = p.prefix_lens ? min(max(p.prefix_lens[b], 0), p.P) : p.P;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  const int n = lane & 31, hh = lane >> 5;

  // ---- this lane's query row and its visible range [vis_lo, vis_hi) of
  // draft-token keys.  A group's G*T rows are taken token-major (row = t*G +
  // h), so a block's rows cover a contiguous token range of every head of
  // the group and share one visible key range; mrow is the row's place in
  // the head-major [G, T] layout of q and out.
  const int row = rb * RB + wave * 32 + n;
  const bool row_ok = row < p.R;
  const int mrow = (row % p.G) * p.T + row / p.G;
  int vis_lo = 0, vis_hi = 0;
  if (row_ok) {
    const int t = row / p.G;
    const int s = t / p.L, r = t - s * p.L;
    const int pass = p.slot_pass ? (int)p.slot_pass[b * p.S + s] : p.pass;
    const int own_lo = s * p.L;
    vis_hi = own_lo + (pass == 0 ? p.L : r + 1);
    vis_lo = p.cross ? 0 : own_lo;
  }

  // ---- key tiles of this workgroup: a range of prefix tiles, then (last
  // split only) the draft-token tiles covering every row's visible range.
  const int pre_begin = split * p.tiles_per_split;
  const int pre_end = min((Pb + KT - 1) / KT, pre_begin + p.tiles_per_split);
  const int n_pre = max(0, pre_end - pre_begin);
  int slot_lo = 0, n_slot = 0;
  if (split == p.n_split - 1) {
    const int t0 = rb * RB / p.G;                   // tokens of this block's rows
    const int t1 = (min(p.R, rb * RB + RB) - 1) / p.G;
    const int lo = p.cross ? 0 : (t0 / p.L) * p.L;
    const int hi = min(p.T, (t1 / p.L + 1) * p.L);
    slot_lo = (lo / KT) * KT;
    n_slot = (hi - slot_lo + KT - 1) / KT;
  }
  const int nt = n_pre + n_slot;

  // ---- Q fragments (B operand of S^T = K Q^T), kept in registers; loaded
  // and waited for before the direct-load pipeline starts so that the
  // pipeline's counted waits see only its own loads
  bf16x8 qf[NKS];
  {
    const uint4* qrow = reinterpret_cast<const uint4*>(p.q + ((size_t)bg * p.R + (row_ok ? mrow : 0)) * D);
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      uint4 v = row_ok ? qrow[2 * ks + hh] : make_uint4(0, 0, 0, 0);
      qf[ks] = __builtin_bit_cast(bf16x8, v);
    }
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) lds_tie(qf[ks]);
    wait_vmcnt<0>();
  }

  // ---- direct-to-LDS staging of K and V tiles: load j of a wave fills 1 KB
  // chunk c = NWAVE*j + wave (RPC rows); lane l lands at row RPC*c + l/LPR,
  // physical 16-byte column l%LPR and fetches the logical column the swizzle
  // puts there.  Rows past the valid keys are clamped to the last valid row
  // (their scores are masked, so they contribute exact zeros).
  int my_r[CPW];
  uint32_t my_off[CPW];
#pragma unroll
  for (int j = 0; j < CPW; ++j) {
    my_r[j] = RPC * (NWAVE * j + wave_u) + lane / LPR;
    my_off[j] = (uint32_t)(my_r[j] * ROWB + (((lane % LPR) ^ swz<D>(my_r[j])) << 4));
  }
  const char* kc = reinterpret_cast<const char*>(p.k_cache + (size_t)bg * p.C * D);
  const char* vc = reinterpret_cast<const char*>(p.v_cache + (size_t)bg * p.C * D);
  const char* ks_ = reinterpret_cast<const char*>(p.k_slot + (size_t)bg * p.T * D);
  const char* vs_ = reinterpret_cast<const char*>(p.v_slot + (size_t)bg * p.T * D);
  auto issue = [&](int i, int buf) {
    const char *kp, *vp;
    int key0, valid;
    if (i < n_pre) {
      key0 = (pre_begin + i) * KT;
      kp = kc;
      vp = vc;
      valid = Pb - key0;
    } else {
      key0 = slot_lo + (i - n_pre) * KT;
      kp = ks_;
      vp = vs_;
      valid = p.T - key0;
    }
    kp += (size_t)key0 * ROWB;
    vp += (size_t)key0 * ROWB;
    uint8_t* kd = &lds[buf][0][wave_u * 1024];
    uint8_t* vd = &lds[buf][1][wave_u * 1024];
    if (valid >= KT) {
#pragma unroll
      for (int j = 0; j < CPW; ++j) {
        dma16(kp + my_off[j], kd + NWAVE * j * 1024);
        dma16(vp + my_off[j], vd + NWAVE * j * 1024);
      }
    } else {
#pragma unroll
      for (int j = 0; j < CPW; ++j) {
        const int dr = min(my_r[j], valid - 1) - my_r[j];  // <= 0: clamp to the last valid row
        dma16(kp + my_off[j] + dr * ROWB, kd + NWAVE * j * 1024);
        dma16(vp + my_off[j] + dr * ROWB, vd + NWAVE * j * 1024);
      }
    }
  };

  f32x16 oacc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) oacc[db] = f32x16{};
  float m_run = kNegBig, l_run = 0.f;  // running max of raw scores; sum of 2^(scaled score - scaled max)
  const float c2 = p.scale_log2;

  // lane-dependent parts of the LDS fragment addresses (the swizzle of every
  // row a lane reads depends on the lane only)
  const uint32_t lds0 = lds_addr(&lds[0][0][0]);
  // K fragment of k-step ks: row n, logical chunk 2*ks + hh, i.e. physical
  // chunk (2*ks) ^ (hh ^ swz(n)) (2*ks is even, hh the low bit)
  const uint32_t k_row = n * ROWB;
  const uint32_t k_cx = (uint32_t)((hh ^ swz<D>(n)) << 4);
  auto k_col = [&](int ks) { return k_row + (k_cx ^ ((uint32_t)ks << 5)); };
  const int q16 = lane >> 4, rr = lane & 15;
  const int vrow = 4 * hh + (rr >> 2);  // first key row of this lane's transposing reads (+16*st, +8)
  // Rows vrow + 16 * step and vrow + 8 + 16 * step: the swizzle repeats every
  // 16 rows and, for vrow < 8, swz(vrow + 8) = swz(vrow) ^ 1, which flips bit
  // 4 of the address (the chunk's low bit): the second half of a step is read
  // at (v_col ^ 16) + 8 rows.
  uint32_t v_col[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) {
    const int d = db * 32 + (q16 & 1) * 16 + 4 * (rr & 3);
    v_col[db] = vrow * ROWB + (((d >> 3) ^ swz<D>(vrow)) << 4) + (d & 7) * 2;
  }
  static_assert((swz<D>(8) ^ swz<D>(0)) == 1, "second V half-step addressing assumes swz(r + 8) = swz(r) ^ 1");

  f32x16 sacc[2];   // scores of the tile between its QK^T and its softmax
  bf16x8 pb[4];      // its probabilities (bf16, B operands of the PV steps)
  v4i16 vf[2][NDB][2];  // V^T fragments, double-buffered across PV steps

  // ---- S^T = K Q^T of tile i for two 32-key blocks; register v of block kb
  // holds key kb*32 + 8*(v/4) + 4*hh + v%4 of the tile.  K fragments are read
  // one k-step ahead of their MFMAs (deeper read-ahead measured no faster).
  auto qk = [&](int i) {
    const uint32_t kb_addr = lds0 + (i % NS) * (2 * TILEB);
    sacc[0] = f32x16{};
    sacc[1] = f32x16{};
    bf16x8 kf[2][2];
    kf[0][0] = lds_read_b128<0>(kb_addr + k_col(0));
    kf[0][1] = lds_read_b128<32 * ROWB>(kb_addr + k_col(0));
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const int sl = ks & 1;
      if (ks + 1 < NKS) {
        kf[sl ^ 1][0] = lds_read_b128<0>(kb_addr + k_col(ks + 1));
        kf[sl ^ 1][1] = lds_read_b128<32 * ROWB>(kb_addr + k_col(ks + 1));
        lds_wait<2>();
      } else {
        lds_wait<0>();
      }
      lds_tie(kf[sl][0]);
      lds_tie(kf[sl][1]);
      sacc[0] = mfma32x32x16(kf[sl][0], qf[ks], sacc[0]);
      sacc[1] = mfma32x32x16(kf[sl][1], qf[ks], sacc[1]);
    }
  };

  // ---- V^T fragments of the first PV step of tile i
  auto pv_start = [&](int i) {
    const uint32_t vb_addr = lds0 + (i % NS) * (2 * TILEB) + TILEB;
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      vf[0][db][0] = lds_read_tr16_b64<0>(vb_addr + v_col[db]);
      vf[0][db][1] = lds_read_tr16_b64<8 * ROWB>(vb_addr + (v_col[db] ^ 16u));
    }
  };

  // ---- online softmax of tile i's scores; masks only on tiles that need them
  auto softmax = [&](int i) {
    const bool is_slot = i >= n_pre;
    const int key0 = is_slot ? slot_lo + (i - n_pre) * KT : (pre_begin + i) * KT;
    const bool full = !is_slot && key0 + KT <= Pb;
    const int lim_lo = is_slot ? vis_lo : key0;
    const int lim_n = is_slot ? vis_hi - vis_lo : Pb - key0;
    if (!full) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int key = key0 + kb * 32 + 8 * (v >> 2) + 4 * hh + (v & 3);
          if ((unsigned)(key - lim_lo) >= (unsigned)lim_n) sacc[kb][v] = -INFINITY;
        }
    }
    // tile maximum of this lane's row: a max3 tree (depth 3 instead of a
    // 16-long chain), then the other lane half of the row
    float mt;
    {
      float t[11];
#pragma unroll
      for (int j = 0; j < 5; ++j) t[j] = max3f(sacc[0][3 * j], sacc[0][3 * j + 1], sacc[0][3 * j + 2]);
      t[5] = max3f(sacc[0][15], sacc[1][0], sacc[1][1]);
#pragma unroll
      for (int j = 0; j < 4; ++j) t[6 + j] = max3f(sacc[1][3 * j + 2], sacc[1][3 * j + 3], sacc[1][3 * j + 4]);
      t[10] = max3f(sacc[1][14], sacc[1][15], sacc[1][15]);
      const float u0 = max3f(t[0], t[1], t[2]), u1 = max3f(t[3], t[4], t[5]);
      const float u2 = max3f(t[6], t[7], t[8]), u3 = max3f(t[9], t[10], t[10]);
      mt = max_xor32(max3f(max3f(u0, u1, u2), u3, u3));
    }
    const float m_new = fmaxf(m_run, mt);
    // Rescale only when the maximum of some row moved by more than 2^8 in
    // probability: until then the exponentials below are taken against the
    // stale maximum and stay <= 2^8 (exact in the float32 sums, same relative
    // rounding in bf16), and the final O / l and LSE do not depend on which
    // maximum was used.  Random scores raise a row's maximum on most early
    // tiles, each time by little; this skips those rescales.  Every PV of the
    // earlier tiles is in oacc before this (the callers keep that order).
    if (__any((m_new - m_run) * c2 > kRescaleLog2)) {
      const float alpha = fast_exp2((m_run - m_new) * c2);
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) oacc[db][v] *= alpha;
      m_run = m_new;
    }
    const float mc = m_run * c2;
    float ps[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        uint32_t pk[4];
#pragma unroll
        for (int j = 0; j < 8; j += 2) {
          const int v = half * 8 + j;
          const float e0 = fast_exp2(fmaf(sacc[kb][v], c2, -mc));
          const float e1 = fast_exp2(fmaf(sacc[kb][v + 1], c2, -mc));
          ps[j >> 1] += e0 + e1;
          pk[j >> 1] = pack_bf16x2_hw(e0, e1);
        }
        // B operand of PV step 2*kb + half: slot j = accumulator register 8*half + j
        pb[2 * kb + half] = __builtin_bit_cast(bf16x8, make_uint4(pk[0], pk[1], pk[2], pk[3]));
      }
    l_run += (ps[0] + ps[1]) + (ps[2] + ps[3]);
  };

  // ---- O^T += V^T P^T of tile i (after pv_start(i)).  Step st covers keys
  // 16*st + 4*hh + {0..3} (slots 0-3) and 16*st + 8 + 4*hh + {0..3} (slots
  // 4-7); V^T fragments are read one step ahead with the transposing LDS read.
  auto pv_finish = [&](int i) {
    const uint32_t vb_addr = lds0 + (i % NS) * (2 * TILEB) + TILEB;
#pragma unroll
    for (int stp = 0; stp < 4; ++stp) {
      const int sl = stp & 1;
      if (stp + 1 < 4) {
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          vf[sl ^ 1][db][0] = lds_read_tr16_b64<0>(vb_addr + v_col[db] + 16 * (stp + 1) * ROWB);
          vf[sl ^ 1][db][1] = lds_read_tr16_b64<8 * ROWB>(vb_addr + (v_col[db] ^ 16u) + 16 * (stp + 1) * ROWB);
        }
        lds_wait<2 * NDB>();
      } else {
        lds_wait<0>();
      }
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        lds_tie(vf[sl][db][0]);
        lds_tie(vf[sl][db][1]);
        const uint2 l2 = __builtin_bit_cast(uint2, vf[sl][db][0]);
        const uint2 h2 = __builtin_bit_cast(uint2, vf[sl][db][1]);
        const bf16x8 a = __builtin_bit_cast(bf16x8, make_uint4(l2.x, l2.y, h2.x, h2.y));
        oacc[db] = mfma32x32x16(a, pb[stp], oacc[db]);
      }
    }
  };

  for (int st = 0; st < NS - 1 && st < nt; ++st) issue(st, st);
  for (int i = 0; i < nt; ++i) {
    const int ahead = min(nt - 1, i + NS - 2) - i;  // later tiles whose loads may still fly
    if constexpr (NS >= 4) {
      if (ahead >= 2) {
        wait_vmcnt<2 * LPT>();
      } else if (ahead == 1) {
        wait_vmcnt<LPT>();
      } else {
        wait_vmcnt<0>();
      }
    } else if constexpr (NS == 3) {
      if (ahead >= 1) {
        wait_vmcnt<LPT>();
      } else {
        wait_vmcnt<0>();
      }
    } else {
      wait_vmcnt<0>();
    }
    block_barrier();
    if (i + NS - 1 < nt) issue(i + NS - 1, (i + NS - 1) % NS);
    qk(i);
    pv_start(i);  // in flight during the softmax
    softmax(i);
    pv_finish(i);
  }

  // ---- finalize: combine the two lane halves' partial sums
  const float l_tot = sum_xor32(l_run);
  if (!row_ok) return;
  const size_t grow = (size_t)bg * p.R + mrow;  // row of the [B*Hq*T] output
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  const float lse2 = m_run * c2 + __log2f(l_tot);  // log2 units
  if (p.n_split == 1) {
    uint16_t* orow = p.out + grow * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int d = db * 32 + 8 * u + 4 * hh;
        uint2 pk;
        pk.x = pack_bf16x2_hw(oacc[db][4 * u] * inv, oacc[db][4 * u + 1] * inv);
        pk.y = pack_bf16x2_hw(oacc[db][4 * u + 2] * inv, oacc[db][4 * u + 3] * inv);
        *reinterpret_cast<uint2*>(orow + d) = pk;
      }
    if (p.lse && hh == 0) p.lse[grow] = lse2 * kLn2;
  } else {
    float* orow = p.part_o + ((size_t)split * p.rows_total + grow) * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int d = db * 32 + 8 * u + 4 * hh;
        float4 o4 = make_float4(oacc[db][4 * u] * inv, oacc[db][4 * u + 1] * inv, oacc[db][4 * u + 2] * inv,
                                oacc[db][4 * u + 3] * inv);
        *reinterpret_cast<float4*>(orow + d) = o4;
      }
    if (hh == 0) p.part_lse[(size_t)split * p.rows_total + grow] = l_tot > 0.f ? lse2 : -INFINITY;
  }
}

// Exact merge of the prefix splits: O = sum_i w_i O_i / sum_i w_i with
// w_i = 2^(lse_i - max_j lse_j); lse = max + log2(sum w) (natural log on output).
template <int D>
__global__ __launch_bounds__(256) void slot_attn_merge_kernel(const float* __restrict__ part_o,
                                                              const float* __restrict__ part_lse, int n_split,
                                                              int rows_total, uint16_t* __restrict__ out,
                                                              float* __restrict__ lse) {
  // a lane merges 4 consecutive elements of one row: D/4 lanes per row
  constexpr int LPR = D / 4, RPW = 64 / LPR;
  constexpr int MAXS = 8;  // splits whose loads are all issued before any arithmetic
  const int lane = threadIdx.x & 63;
  const int row = (blockIdx.x * 4 + (threadIdx.x >> 6)) * RPW + lane / LPR;
  const int c = (lane % LPR) * 4;
  if (row >= rows_total) return;
  float l[MAXS];
  float4 o[MAXS];
  const int ns = min(n_split, MAXS);
#pragma unroll
  for (int i = 0; i < MAXS; ++i) {  // every load in flight at once
    if (i < ns) {
      l[i] = part_lse[(size_t)i * rows_total + row];
      o[i] = *reinterpret_cast<const float4*>(part_o + ((size_t)i * rows_total + row) * D + c);
    }
  }
  float mx = -INFINITY;
#pragma unroll
  for (int i = 0; i < MAXS; ++i)
    if (i < ns) mx = fmaxf(mx, l[i]);
  for (int i = MAXS; i < n_split; ++i) mx = fmaxf(mx, part_lse[(size_t)i * rows_total + row]);
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  float wsum = 0.f;
#pragma unroll
  for (int i = 0; i < MAXS; ++i) {
    if (i < ns) {
      const float wi = l[i] == -INFINITY ? 0.f : fast_exp2(l[i] - mx);
      wsum += wi;
      acc[0] += wi * o[i].x;
      acc[1] += wi * o[i].y;
      acc[2] += wi * o[i].z;
      acc[3] += wi * o[i].w;
    }
  }
  for (int i = MAXS; i < n_split; ++i) {
    const float li = part_lse[(size_t)i * rows_total + row];
    const float wi = li == -INFINITY ? 0.f : fast_exp2(li - mx);
    wsum += wi;
    const float4 oi = *reinterpret_cast<const float4*>(part_o + ((size_t)i * rows_total + row) * D + c);
    acc[0] += wi * oi.x;
    acc[1] += wi * oi.y;
    acc[2] += wi * oi.z;
    acc[3] += wi * oi.w;
  }
  const float inv = 1.f / wsum;
  *reinterpret_cast<uint2*>(out + (size_t)row * D + c) =
      make_uint2(pack_bf16x2_hw(acc[0] * inv, acc[1] * inv), pack_bf16x2_hw(acc[2] * inv, acc[3] * inv));
  if (lse && c == 0) lse[row] = (mx + __log2f(wsum)) * kLn2;
}

// float32 path: LPR = D/16 lanes per query row, each holding 16 elements of
// the row's q and output; a score is the lanes' partial dot products summed
// across the group (then taken from the group's first lane, so every lane
// of a row follows the same online softmax, with expf).  Plain FMA
// arithmetic; serves small float32 problems and every mask variant.
template <int D>
__global__ __launch_bounds__(kAttnF32RowsPerBlock * (D / 16)) void slot_attn_f32_kernel(AttnParams32 p) {
  constexpr int LPR = D / 16;  // lanes per row
  static_assert(LPR >= 1 && (LPR & (LPR - 1)) == 0 && 64 % LPR == 0, "a row's lanes are a power of two in a wave");
  const int sub = threadIdx.x % LPR;  // this lane's 16-element slice of the row
  const int gid = blockIdx.x * kAttnF32RowsPerBlock + threadIdx.x / LPR;
  const bool row_ok = gid < p.rows_total;
  // lanes past the last row follow a valid row (the shuffles need every lane
  // of a group) and store nothing
  const int grow = row_ok ? gid : p.rows_total - 1;
  const int t = grow % p.T;
  const int h = (grow / p.T) % p.Hq;
  const int b = grow / (p.T * p.Hq);
  const int g = h / p.G;
  const int s = t / p.L, r = t - s * p.L;
  const int pass = p.slot_pass ? (int)p.slot_pass[b * p.S + s] : p.pass;
  const int vis_hi = s * p.L + (pass == 0 ? p.L : r + 1);
  const int vis_lo = p.cross ? 0 : s * p.L;
  const int lead = (int)(threadIdx.x % 64) & ~(LPR - 1);  // the group's first lane in the wave

  float qv[16], o[16];
  const float* qrow = p.q + (size_t)grow * D + sub * 16;
#pragma unroll
  for (int d = 0; d < 16; ++d) {
    qv[d] = qrow[d] * p.scale;
    o[d] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  auto visit = [&](const float* krow, const float* vrow) {
    float part = 0.f;
#pragma unroll
    for (int d = 0; d < 16; ++d) part = fmaf(qv[d], krow[sub * 16 + d], part);
#pragma unroll
    for (int off = LPR / 2; off > 0; off >>= 1) part += __shfl_xor(part, off);
    const float sc = __shfl(part, lead);
    const float m_new = fmaxf(m, sc);
    const float c = expf(m - m_new);
    const float e = expf(sc - m_new);
    l = l * c + e;
#pragma unroll
    for (int d = 0; d < 16; ++d) o[d] = fmaf(e, vrow[sub * 16 + d], o[d] * c);
    m = m_new;
  };
  const size_t cbase = ((size_t)b * p.Hkv + g) * p.C * D;
  const int Pb = p.prefix_lens ? min(max(p.prefix_lens[b], 0), p.P) : p.P;
  for (int j = 0; j < Pb; ++j) visit(p.k_cache + cbase + (size_t)j * D, p.v_cache + cbase + (size_t)j * D);
  const size_t sbase = ((size_t)b * p.Hkv + g) * p.T * D;
  for (int j = vis_lo; j < vis_hi; ++j) visit(p.k_slot + sbase + (size_t)j * D, p.v_slot + sbase + (size_t)j * D);
  if (!row_ok) return;
  float* orow = p.out + (size_t)gid * D + sub * 16;
  const float inv = 1.f / l;
#pragma unroll
  for (int d = 0; d < 16; ++d) orow[d] = o[d] * inv;
  if (p.lse && sub == 0) p.lse[gid] = m + logf(l);
}

// ------------------------------------------------------------------ launchers

hipError_t launch_slot_attn_bf16(const AttnParams& p, int head_dim, hipStream_t stream) {
  const int grid = 8 * p.per_xcd;
  const bool wide = p.rows_per_block == kAttnWideRowsPerBlock;
  if (head_dim == 128) {
    if (wide) {
      slot_attn_bf16_kernel<128, ZARYA_ATTN_NS, 8><<<dim3(grid), dim3(512), 0, stream>>>(p);
    } else {
      slot_attn_bf16_kernel<128, ZARYA_ATTN_NS, 4><<<dim3(grid), dim3(256), 0, stream>>>(p);
    }
  } else {
    if (wide) {
      slot_attn_bf16_kernel<64, ZARYA_ATTN_NS, 8><<<dim3(grid), dim3(512), 0, stream>>>(p);
    } else {
      slot_attn_bf16_kernel<64, ZARYA_ATTN_NS, 4><<<dim3(grid), dim3(256), 0, stream>>>(p);
    }
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.n_split == 1) return e;
  const int rows_per_wg = 4 * (64 / (head_dim / 4));  // four waves, 64 / (D/4) rows each
  const int mgrid = (p.rows_total + rows_per_wg - 1) / rows_per_wg;
  if (head_dim == 128) {
    hipLaunchKernelGGL(slot_attn_merge_kernel<128>, dim3(mgrid), dim3(256), 0, stream, p.part_o, p.part_lse,
                       p.n_split, p.rows_total, p.out, p.lse);
  } else {
    hipLaunchKernelGGL(slot_attn_merge_kernel<64>, dim3(mgrid), dim3(256), 0, stream, p.part_o, p.part_lse,
                       p.n_split, p.rows_total, p.out, p.lse);
  }
  return hipGetLastError();
}

hipError_t launch_slot_attn_f32(const AttnParams32& p, int head_dim, hipStream_t stream) {
  const int grid = (p.rows_total + kAttnF32RowsPerBlock - 1) / kAttnF32RowsPerBlock;
  if (head_dim == 128) {
    hipLaunchKernelGGL(slot_attn_f32_kernel<128>, dim3(grid), dim3(kAttnF32RowsPerBlock * 8), 0, stream, p);
  } else {
    hipLaunchKernelGGL(slot_attn_f32_kernel<64>, dim3(grid), dim3(kAttnF32RowsPerBlock * 4), 0, stream, p);
  }
  return hipGetLastError();
}

}  // namespace zarya
