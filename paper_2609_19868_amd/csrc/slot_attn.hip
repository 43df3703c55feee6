// Slot-parallel attention against a reused prefix KV cache (gfx950).
//
// What is computed (Zarya, Sec. 5.1 KV-reuse argument and Sec. 5.2 draft /
// verification phases): every draft token t = s*L + r of query head h attends
// to all P prefix keys of KV head g = h / G and to a contiguous range of the
// draft tokens' own keys -- its own slot (all of it in the DIFFUSION pass, up
// to itself in the AR_INFILL pass), preceded by every earlier slot when
// cross_slot = CAUSAL.
//
// bf16 kernel design (one workgroup = 4 waves = up to 128 query rows of one
// GQA group, i.e. G heads x T tokens flattened; one split of the prefix keys):
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

namespace {

constexpr int KT = 64;      // keys per tile
constexpr int NWAVE = 4;    // waves per workgroup
constexpr int RB = NWAVE * 32;  // query rows per workgroup

// XOR swizzle of the 16-byte chunk index of LDS row `kr`.
template <int D>
__device__ __forceinline__ int swz(int kr) {
  if constexpr (D == 128) {
    return (kr & 7) << 1;
  } else {
    return ((kr >> 1) & 3) << 1;
  }
}

template <int D>
__device__ __forceinline__ int lds_off(int kr, int chunk) {
  return kr * (D * 2) + ((chunk ^ swz<D>(kr)) << 4);
}

}  // namespace

template <int D>
__global__ __launch_bounds__(256) void slot_attn_bf16_kernel(AttnParams p) {
  constexpr int NCH = D / 8;           // 16-byte chunks per key row
  constexpr int TILEB = KT * D * 2;    // bytes of one K (or V) tile
  constexpr int NLD = TILEB / (256 * 16);  // 16-byte loads per thread per tile
  constexpr int NDB = D / 32;          // 32-wide blocks of the head dim
  constexpr int NKS = D / 16;          // k-steps of the QK^T contraction
  __shared__ __attribute__((aligned(16))) uint8_t lds[2][2][TILEB];

  const int w = xcd_work_index(blockIdx.x, p.per_xcd, p.n_items);
  if (w < 0) return;
  const int rb = w % p.n_rb;
  const int split = (w / p.n_rb) % p.n_split;
  const int bg = w / (p.n_rb * p.n_split);  // b * Hkv + g
  const int b = bg / p.Hkv;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int n = lane & 31, hh = lane >> 5;

  // ---- this lane's query row and its visible range of draft-token keys
  const int row = rb * RB + wave * 32 + n;  // row of the GQA group, [0, G*T)
  const bool row_ok = row < p.R;
  int vis_lo = 0, vis_hi = 0;
  if (row_ok) {
    const int t = row % p.T;
    const int s = t / p.L, r = t - s * p.L;
    const int pass = p.slot_pass ? (int)p.slot_pass[b * p.S + s] : p.pass;
    const int own_lo = s * p.L;
    vis_hi = own_lo + (pass == 0 ? p.L : r + 1);
    vis_lo = p.cross ? 0 : own_lo;
  }

  // ---- key tiles of this workgroup: a range of prefix tiles, then (last
  // split only) the draft-token tiles covering every row's visible range.
  const int pre_begin = split * p.tiles_per_split;
  const int pre_end = min(p.n_prefix_tiles, pre_begin + p.tiles_per_split);
  const int n_pre = max(0, pre_end - pre_begin);
  int slot_lo = 0, n_slot = 0;
  if (split == p.n_split - 1) {
    const int r0 = rb * RB;
    const int r1 = min(p.R, r0 + RB) - 1;
    int lo = 0, hi = p.T;
    if (r0 / p.T == r1 / p.T) {  // rows of one head: tokens r0%T .. r1%T
      const int t0 = r0 % p.T, t1 = r1 % p.T;
      lo = p.cross ? 0 : (t0 / p.L) * p.L;
      hi = min(p.T, (t1 / p.L + 1) * p.L);
    }
    slot_lo = (lo / KT) * KT;
    n_slot = (hi - slot_lo + KT - 1) / KT;
  }
  const int nt = n_pre + n_slot;

  const size_t cache_base = (size_t)bg * p.C * D;
  const size_t slot_base = (size_t)bg * p.T * D;

  // ---- Q fragments (B operand of S^T = K Q^T), kept in registers
  bf16x8 qf[NKS];
  {
    const uint4* qrow = reinterpret_cast<const uint4*>(p.q + ((size_t)bg * p.R + (row_ok ? row : 0)) * D);
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      uint4 v = row_ok ? qrow[2 * ks + hh] : make_uint4(0, 0, 0, 0);
      qf[ks] = __builtin_bit_cast(bf16x8, v);
    }
  }

  uint4 kreg[NLD], vreg[NLD];
  auto load_tile = [&](int i) {
    const uint16_t *kp, *vp;
    int valid;
    if (i < n_pre) {
      const int key0 = (pre_begin + i) * KT;
      kp = p.k_cache + cache_base + (size_t)key0 * D;
      vp = p.v_cache + cache_base + (size_t)key0 * D;
      valid = min(KT, p.P - key0);
    } else {
      const int key0 = slot_lo + (i - n_pre) * KT;
      kp = p.k_slot + slot_base + (size_t)key0 * D;
      vp = p.v_slot + slot_base + (size_t)key0 * D;
      valid = min(KT, p.T - key0);
    }
#pragma unroll
    for (int j = 0; j < NLD; ++j) {
      const int c = j * 256 + tid;
      const int kr = c / NCH, ch = c % NCH;
      if (kr < valid) {
        kreg[j] = reinterpret_cast<const uint4*>(kp + (size_t)kr * D)[ch];
        vreg[j] = reinterpret_cast<const uint4*>(vp + (size_t)kr * D)[ch];
      } else {  // rows past the end: zeros, so masked probabilities multiply finite values
        kreg[j] = make_uint4(0, 0, 0, 0);
        vreg[j] = make_uint4(0, 0, 0, 0);
      }
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int j = 0; j < NLD; ++j) {
      const int c = j * 256 + tid;
      const int kr = c / NCH, ch = c % NCH;
      *reinterpret_cast<uint4*>(&lds[buf][0][lds_off<D>(kr, ch)]) = kreg[j];
      *reinterpret_cast<uint4*>(&lds[buf][1][lds_off<D>(kr, ch)]) = vreg[j];
    }
  };

  f32x16 oacc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) oacc[db] = f32x16{};
  float m_run = kNegBig, l_run = 0.f;

  if (nt > 0) {
    load_tile(0);
    store_tile(0);
  }
  __syncthreads();

  for (int i = 0; i < nt; ++i) {
    const int buf = i & 1;
    if (i + 1 < nt) load_tile(i + 1);
    const uint8_t* kl = lds[buf][0];
    const uint8_t* vl = lds[buf][1];

    // S^T for two 32-key blocks: reg v of block kb is key kb*32 + 8*(v/4) + 4*hh + v%4
    f32x16 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      sacc[kb] = f32x16{};
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(kl + lds_off<D>(kb * 32 + n, 2 * ks + hh));
        sacc[kb] = mfma32x32x16(a, qf[ks], sacc[kb]);
      }
    }

    // scale into the log2 domain and mask
    float sv[2][16];
    const bool is_slot = i >= n_pre;
    int key0, lim_lo, lim_n;
    if (!is_slot) {
      key0 = (pre_begin + i) * KT;
      lim_lo = key0;
      lim_n = p.P - key0;  // keys [key0, P) valid
    } else {
      key0 = slot_lo + (i - n_pre) * KT;
      lim_lo = vis_lo;
      lim_n = vis_hi - vis_lo;
    }
    float mt = kNegBig;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int key = key0 + kb * 32 + 8 * (v >> 2) + 4 * hh + (v & 3);
        const bool vis = (unsigned)(key - lim_lo) < (unsigned)lim_n;
        const float x = vis ? sacc[kb][v] * p.scale_log2 : -INFINITY;
        sv[kb][v] = x;
        mt = fmaxf(mt, x);
      }
    }
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    const float m_new = fmaxf(m_run, mt);
    const float alpha = fast_exp2(m_run - m_new);
    m_run = m_new;
    float psum = 0.f;
    // B operand of PV step st, slot j = accumulator register 8*(st%2) + j of key
    // block st/2; packed two bf16 per dword and bit-cast as whole vectors
    uint32_t pk[4][4];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int v = 0; v < 16; v += 2) {
        const float e0 = fast_exp2(sv[kb][v] - m_new);
        const float e1 = fast_exp2(sv[kb][v + 1] - m_new);
        psum += e0 + e1;
        pk[2 * kb + (v >> 3)][(v & 7) >> 1] = pack_bf16x2(e0, e1);
      }
    }
    bf16x8 pb[4];
#pragma unroll
    for (int st = 0; st < 4; ++st) pb[st] = __builtin_bit_cast(bf16x8, make_uint4(pk[st][0], pk[st][1], pk[st][2], pk[st][3]));
    l_run = l_run * alpha + psum;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int v = 0; v < 16; ++v) oacc[db][v] *= alpha;

    // O^T += V^T P^T.  Step st covers keys 16*st + 4*hh + {0..3} (slots 0-3)
    // and 16*st + 8 + 4*hh + {0..3} (slots 4-7); lane-group row rr = lane%16
    // reads 4 d-values of key (.. + rr/4) for the transposing load.
    const int q16 = lane >> 4, rr = lane & 15;
    const int dgrp = q16 & 1;
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const int d = db * 32 + dgrp * 16 + 4 * (rr & 3);
      const int chunk = d >> 3, half = (d & 7) * 2;
#pragma unroll
      for (int st = 0; st < 4; ++st) {
        const int k0 = 16 * st + 4 * hh + (rr >> 2);
        const int k1 = k0 + 8;
        v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(vl + lds_off<D>(k0, chunk) + half));
        v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(vl + lds_off<D>(k1, chunk) + half));
        const uint2 l2 = __builtin_bit_cast(uint2, lo);
        const uint2 h2 = __builtin_bit_cast(uint2, hi);
        const bf16x8 a = __builtin_bit_cast(bf16x8, make_uint4(l2.x, l2.y, h2.x, h2.y));
        oacc[db] = mfma32x32x16(a, pb[st], oacc[db]);
      }
    }

    if (i + 1 < nt) store_tile(buf ^ 1);
    __syncthreads();
  }

  // ---- finalize: combine the two lane halves' partial sums
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (!row_ok) return;
  const size_t grow = (size_t)bg * p.R + row;  // row of the [B*Hq*T] output
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  if (p.n_split == 1) {
    uint16_t* orow = p.out + grow * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int d = db * 32 + 8 * u + 4 * hh;
        uint2 pk;
        pk.x = pack_bf16x2(oacc[db][4 * u] * inv, oacc[db][4 * u + 1] * inv);
        pk.y = pack_bf16x2(oacc[db][4 * u + 2] * inv, oacc[db][4 * u + 3] * inv);
        *reinterpret_cast<uint2*>(orow + d) = pk;
      }
    if (p.lse && hh == 0) p.lse[grow] = (m_run + __log2f(l_tot)) * kLn2;
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
    if (hh == 0) p.part_lse[(size_t)split * p.rows_total + grow] = l_tot > 0.f ? m_run + __log2f(l_tot) : -INFINITY;
  }
}

// Exact merge of the prefix splits: O = sum_i w_i O_i / sum_i w_i with
// w_i = 2^(lse_i - max_j lse_j); lse = max + log2(sum w) (natural log on output).
template <int D>
__global__ __launch_bounds__(256) void slot_attn_merge_kernel(const float* __restrict__ part_o,
                                                              const float* __restrict__ part_lse, int n_split,
                                                              int rows_total, uint16_t* __restrict__ out,
                                                              float* __restrict__ lse) {
  constexpr int PER = D / 64;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows_total) return;
  float mx = -INFINITY;
  for (int i = 0; i < n_split; ++i) mx = fmaxf(mx, part_lse[(size_t)i * rows_total + row]);
  float acc[PER] = {};
  float wsum = 0.f;
  for (int i = 0; i < n_split; ++i) {
    const float li = part_lse[(size_t)i * rows_total + row];
    const float wi = li == -INFINITY ? 0.f : fast_exp2(li - mx);
    wsum += wi;
    const float* po = part_o + ((size_t)i * rows_total + row) * D + lane * PER;
#pragma unroll
    for (int e = 0; e < PER; ++e) acc[e] += wi * po[e];
  }
  const float inv = 1.f / wsum;
  uint16_t* orow = out + (size_t)row * D + lane * PER;
  if constexpr (PER == 2) {
    *reinterpret_cast<uint32_t*>(orow) = pack_bf16x2(acc[0] * inv, acc[1] * inv);
  } else {
    orow[0] = f32_to_bf16(acc[0] * inv);
  }
  if (lse && lane == 0) lse[row] = (mx + __log2f(wsum)) * kLn2;
}

// float32 path: one thread per query row, plain FMA arithmetic, online softmax
// with expf.  Serves small float32 problems and every mask variant.
template <int D>
__global__ __launch_bounds__(64) void slot_attn_f32_kernel(AttnParams32 p) {
  const int gid = blockIdx.x * 64 + threadIdx.x;
  if (gid >= p.rows_total) return;
  const int t = gid % p.T;
  const int h = (gid / p.T) % p.Hq;
  const int b = gid / (p.T * p.Hq);
  const int g = h / p.G;
  const int s = t / p.L, r = t - s * p.L;
  const int pass = p.slot_pass ? (int)p.slot_pass[b * p.S + s] : p.pass;
  const int vis_hi = s * p.L + (pass == 0 ? p.L : r + 1);
  const int vis_lo = p.cross ? 0 : s * p.L;

  float qv[D], o[D];
  const float* qrow = p.q + (size_t)gid * D;
#pragma unroll
  for (int d = 0; d < D; ++d) {
    qv[d] = qrow[d] * p.scale;
    o[d] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  auto visit = [&](const float* krow, const float* vrow) {
    float sc = 0.f;
#pragma unroll
    for (int d = 0; d < D; ++d) sc = fmaf(qv[d], krow[d], sc);
    const float m_new = fmaxf(m, sc);
    const float c = expf(m - m_new);
    const float e = expf(sc - m_new);
    l = l * c + e;
#pragma unroll
    for (int d = 0; d < D; ++d) o[d] = fmaf(e, vrow[d], o[d] * c);
    m = m_new;
  };
  const size_t cbase = ((size_t)b * p.Hkv + g) * p.C * D;
  for (int j = 0; j < p.P; ++j) visit(p.k_cache + cbase + (size_t)j * D, p.v_cache + cbase + (size_t)j * D);
  const size_t sbase = ((size_t)b * p.Hkv + g) * p.T * D;
  for (int j = vis_lo; j < vis_hi; ++j) visit(p.k_slot + sbase + (size_t)j * D, p.v_slot + sbase + (size_t)j * D);
  float* orow = p.out + (size_t)gid * D;
  const float inv = 1.f / l;
#pragma unroll
  for (int d = 0; d < D; ++d) orow[d] = o[d] * inv;
  if (p.lse) p.lse[gid] = m + logf(l);
}

// ------------------------------------------------------------------ launchers

hipError_t launch_slot_attn_bf16(const AttnParams& p, int head_dim, hipStream_t stream) {
  const int grid = 8 * p.per_xcd;
  if (head_dim == 128) {
    hipLaunchKernelGGL(slot_attn_bf16_kernel<128>, dim3(grid), dim3(256), 0, stream, p);
  } else {
    hipLaunchKernelGGL(slot_attn_bf16_kernel<64>, dim3(grid), dim3(256), 0, stream, p);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.n_split == 1) return e;
  const int mgrid = (p.rows_total + 3) / 4;
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
  const int grid = (p.rows_total + 63) / 64;
  if (head_dim == 128) {
    hipLaunchKernelGGL(slot_attn_f32_kernel<128>, dim3(grid), dim3(64), 0, stream, p);
  } else {
    hipLaunchKernelGGL(slot_attn_f32_kernel<64>, dim3(grid), dim3(64), 0, stream, p);
  }
  return hipGetLastError();
}

}  // namespace zarya
