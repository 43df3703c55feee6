// LM-head confidence reduction (gfx950): logits = hidden . W^T reduced per row
// to (max, log-sum-exp, argmax) without writing logits to memory.
//
// What is computed (Zarya, Sec. 5.2: the slot confidence is the probability of
// its first token and verification compares token probabilities with a
// threshold; Table 1: the LM head is the tied embedding W[V, H]): for every
// row, the largest softmax probability, its token id (lowest on ties), the
// log-sum-exp and optionally the probability of a given target id.
//
// bf16 design: a workgroup owns a tile of rows of `hidden` (256 by default)
// and a contiguous vocabulary range, walked in 256-wide tiles.  The product is
// computed transposed, logits^T = W h^T, with v_mfma_f32_32x32x16_bf16 (each
// wave owns 128 vocab ids x 64 rows), so every lane holds values of a single
// row and the per-row reduction runs inside the lane.  After each vocab tile
// the epilogue folds the tile into running (max, sum exp(x - max), argmax)
// statistics; at the end of the range the two lane halves and the two vocab
// halves are combined and one partial per (row, range) is written.
// Operands are streamed into a ring of XOR-swizzled LDS stages with direct
// global->LDS loads (no register staging), one workgroup barrier per stage;
// the MFMA operand fragments are read from LDS one k-step ahead of their use.
// Workgroups that share a vocabulary range are mapped to the same XCD so each
// W tile is fetched from HBM once and reused from that XCD's L2.
#include <limits.h>

#include "common.hpp"
#include "kernels.hpp"

namespace zarya {

namespace {

constexpr int BV = 256;  // vocab entries per tile


// Merge two (max logit, sum exp(logit - max), argmax) statistics.  On equal
// maxima the lower id wins, which keeps the result independent of the merge
// order.
__device__ __forceinline__ void stat_merge(float& m, float& s, int& idx, float m2, float s2, int idx2) {
  const float mn = fmaxf(m, m2);
  const float sa = s == 0.f ? 0.f : s * fast_exp2((m - mn) * kLog2e);
  const float sb = s2 == 0.f ? 0.f : s2 * fast_exp2((m2 - mn) * kLog2e);
  int in;
  if (m2 > m) {
    in = idx2;
  } else if (m > m2) {
    in = idx;
  } else {
    in = min(idx, idx2);
  }
  m = mn;
  s = sa + sb;
  idx = in;
}

// XOR swizzle of the 16-byte column of row r in a [rows][BK] bf16 LDS tile:
// keeps the 32 rows read by one MFMA operand load (and the rows one direct
// load writes) on distinct LDS banks.
template <int BK>
__device__ __forceinline__ int cswz(int r) {
  if constexpr (BK == 64) {
    return (r >> 1) & 7;
  } else {
    return (r >> 2) & 3;
  }
}

}  // namespace

// Fold one vocab tile into the running (max, sum exp(x - max), argmax)
// statistics of a lane's rows.  Register v of block (ib, jb) holds the logit
// of vocab id id0 + c(ib, v), c = 32*ib + 8*(v/4) + v%4, for the lane's row of
// row block jb; offsets c >= lim are past the vocabulary range.  The argmax
// is searched only when the tile raises the running maximum; the lowest id at
// the maximum wins (earlier tiles hold lower ids).  ARGMAX = false skips it.
template <int JB, bool ARGMAX = true>
__device__ __forceinline__ void fold_tile(const f32x16 (&acc)[4][JB], int lim, int id0, float (&m_run)[JB],
                                          float (&s_run)[JB], int (&i_run)[JB]) {
  constexpr int IB = 4;
  const bool full = lim >= 128;
#pragma unroll
  for (int jb = 0; jb < JB; ++jb) {
    float mt = -INFINITY;
    if (full) {
      float mq[IB];
#pragma unroll
      for (int ib = 0; ib < IB; ++ib) {
        const f32x16& x = acc[ib][jb];
        float t = max3f(x[0], x[1], x[2]);
#pragma unroll
        for (int v = 3; v < 15; v += 2) t = max3f(t, x[v], x[v + 1]);
        mq[ib] = max3f(t, x[15], x[15]);
      }
      mt = max3f(max3f(mq[0], mq[1], mq[2]), mq[3], mq[3]);
    } else {
#pragma unroll
      for (int ib = 0; ib < IB; ++ib)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int c = ib * 32 + 8 * (v >> 2) + (v & 3);
          mt = fmaxf(mt, c < lim ? acc[ib][jb][v] : -INFINITY);
        }
    }
    if (ARGMAX && mt > m_run[jb]) {
      int it = 0;
      if (full) {
#pragma unroll
        for (int ib = IB - 1; ib >= 0; --ib)
#pragma unroll
          for (int v = 15; v >= 0; --v) it = acc[ib][jb][v] == mt ? ib * 32 + 8 * (v >> 2) + (v & 3) : it;
      } else {
#pragma unroll
        for (int ib = IB - 1; ib >= 0; --ib)
#pragma unroll
          for (int v = 15; v >= 0; --v) {
            const int c = ib * 32 + 8 * (v >> 2) + (v & 3);
            it = (acc[ib][jb][v] == mt && c < lim) ? c : it;
          }
      }
      i_run[jb] = id0 + it;
    }
    const float mn = fmaxf(m_run[jb], mt);
    const float mn2 = mn * kLog2e;
    float e = 0.f;
    if (full) {
#pragma unroll
      for (int ib = 0; ib < IB; ++ib) {
        float e4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int v = 0; v < 16; ++v) e4[v & 3] += fast_exp2(fmaf(acc[ib][jb][v], kLog2e, -mn2));
        e += (e4[0] + e4[1]) + (e4[2] + e4[3]);
        __builtin_amdgcn_sched_barrier(0);  // keep the live ranges short
      }
    } else {
#pragma unroll
      for (int ib = 0; ib < IB; ++ib)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int c = ib * 32 + 8 * (v >> 2) + (v & 3);
          const float pe = fast_exp2(fmaf(acc[ib][jb][v], kLog2e, -mn2));
          e += c < lim ? pe : 0.f;
        }
    }
    s_run[jb] = s_run[jb] * fast_exp2((m_run[jb] - mn) * kLog2e) + e;
    m_run[jb] = mn;
  }
}

// Sampling: fold one vocab tile into the running best perturbed score of the
// lane's rows (same register layout as fold_tile; `row` = the lane's row of
// row block 0, block jb holds row + 32*jb).  The uniforms of vocab ids
// 4q..4q+3 of a row are the four words of the Philox block with counter
// (q, row, off_lo, off_hi); a lane's ids come in aligned runs of four, so each
// block is drawn once.  The strict comparison keeps the lowest id of equal
// scores (ids grow along the scan).  Only the id is kept: the merge recomputes
// the winner's logit.  The row blocks are the inner loop so that each range
// test on the vocab offset serves all of them (hoisted across row blocks, the
// tests' lane masks overflow the scalar registers).
template <int JB>
__device__ __forceinline__ void sample_fold(const f32x16 (&acc)[4][JB], int lim, int id0, int row,
                                            const ConfParams& p, float (&g_best)[JB], int (&g_id)[JB]) {
  const bool full = lim >= 128;
#pragma unroll
  for (int ib = 0; ib < 4; ++ib) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int c0 = ib * 32 + 8 * q;  // offsets c0 .. c0+3 hold ids id0 + c0 .. + 3
#pragma unroll
      for (int jb = 0; jb < JB; ++jb) {
        const uint4 r = philox4x32_10_dev((uint32_t)(id0 + c0) >> 2, (uint32_t)(row + 32 * jb), p.off_lo, p.off_hi,
                                      p.seed_lo, p.seed_hi);
        const uint32_t words[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const float sc = fmaf(acc[ib][jb][4 * q + w], p.c2t, gumbel_log2(words[w]));
          if ((full || c0 + w < lim) && sc > g_best[jb]) {
            g_best[jb] = sc;
            g_id[jb] = id0 + c0 + w;
          }
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

// Merge two sampling candidates: the higher score wins, the lower id on ties.
__device__ __forceinline__ void sample_merge(float& g, int& gi, float g2, int gi2) {
  if (g2 > g || (g2 == g && gi2 < gi)) {
    g = g2;
    gi = gi2;
  }
}

// Combine the statistics of a workgroup's rows and write one partial per
// (vocabulary group, row).  Lanes n and n+32 hold disjoint vocab ids of the
// same row (merged by a shuffle); the waves of vocab halves 0 and 1 hold the
// same rows (merged through `scratch`, 20 bytes per row).  With SAMPLE the
// sampling candidates are combined and written the same way (and the argmax,
// not tracked then, is not written).  Contains a
// workgroup barrier; `scratch` must be free of pending reads.
template <int JB, int BR, bool SAMPLE>
__device__ __forceinline__ void store_partials(const ConfParams& p, int vg, int row0, int rbase, int wv, int hh, int n,
                                               float (&m_run)[JB], float (&s_run)[JB], int (&i_run)[JB],
                                               float (&g_best)[JB], int (&g_id)[JB], uint8_t* scratch) {
#pragma unroll
  for (int jb = 0; jb < JB; ++jb) {
    const float m2 = __shfl_xor(m_run[jb], 32);
    const float s2 = __shfl_xor(s_run[jb], 32);
    const int i2 = __shfl_xor(i_run[jb], 32);
    stat_merge(m_run[jb], s_run[jb], i_run[jb], m2, s2, i2);
    if constexpr (SAMPLE) {
      const float g2 = __shfl_xor(g_best[jb], 32);
      const int gi2 = __shfl_xor(g_id[jb], 32);
      sample_merge(g_best[jb], g_id[jb], g2, gi2);
    }
  }
  float* xm = reinterpret_cast<float*>(scratch);
  float* xs = xm + BR;
  int* xi = reinterpret_cast<int*>(xs + BR);
  float* xg = reinterpret_cast<float*>(xi + BR);
  int* xgi = reinterpret_cast<int*>(xg + BR);
  if (wv == 1 && hh == 0) {
#pragma unroll
    for (int jb = 0; jb < JB; ++jb) {
      const int lr = rbase + jb * 32 + n;
      xm[lr] = m_run[jb];
      xs[lr] = s_run[jb];
      xi[lr] = i_run[jb];
      if constexpr (SAMPLE) {
        xg[lr] = g_best[jb];
        xgi[lr] = g_id[jb];
      }
    }
  }
  __syncthreads();
  if (wv == 0 && hh == 0) {
#pragma unroll
    for (int jb = 0; jb < JB; ++jb) {
      const int lr = rbase + jb * 32 + n;
      stat_merge(m_run[jb], s_run[jb], i_run[jb], xm[lr], xs[lr], xi[lr]);
      const int row = row0 + lr;
      const size_t o = (size_t)row * p.n_vg + vg;
      if (row < p.M) {
        p.part_m[o] = m_run[jb];
        p.part_s[o] = s_run[jb];
        p.part_idx[o] = i_run[jb];
      }
      if constexpr (SAMPLE) {
        sample_merge(g_best[jb], g_id[jb], xg[lr], xgi[lr]);
        if (row < p.M) {
          p.part_g[o] = g_best[jb];
          p.part_gi[o] = g_id[jb];
        }
      }
    }
  }
}

// One workgroup: NW waves as a 2 (vocab) x NW/2 (rows) grid over a
// 256-vocab x BR-row tile; each wave owns 128 vocab ids x 2*BR/NW rows.
// BK: contraction depth per stage.  The W tile streams from HBM through a
// ring of NSW LDS buffers (prefetch distance NSW - 1 stages), the hidden tile
// (re-read for every vocab tile, so served from L2) through a ring of NSX.
// W_NT: the W loads are non-temporal, so that the W stream does not evict the
// hidden tiles from L2 (for launches whose hidden rows fit there).  Partials
// are written per (vocabulary group, row).
template <int NW, int BR, int BK, int NSW, int NSX, bool SAMPLE, bool W_NT>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(NW / 4))) void slot_conf_bf16_kernel(
    ConfParams p) {
  constexpr int ATB = BV * BK * 2;    // bytes of the W tile of one stage
  constexpr int BTB = BR * BK * 2;    // bytes of the hidden tile of one stage
  constexpr int CPA = ATB / 1024 / NW;  // 1 KB direct-load chunks per wave: W
  constexpr int CPB = BTB / 1024 / NW;  // ... hidden
  constexpr int LPR = BK / 8;           // 16-byte columns per row
  constexpr int RPC = 1024 / (BK * 2);  // rows per 1 KB chunk
  constexpr int IB = 4;                 // 32-wide vocab blocks per wave
  constexpr int WROWS = 2 * BR / NW;    // rows per wave
  constexpr int JB = WROWS / 32;        // 32-wide row blocks per wave
  constexpr int NKS = BK / 16;          // MFMA k-steps per stage
  static_assert(CPA * NW * 1024 == ATB && CPB * NW * 1024 == BTB, "chunks must divide over the waves");
  static_assert(JB * 32 == WROWS, "rows per wave must be a multiple of 32");
  static_assert(NSX == 2 && (NSW == 2 || NSW == 3), "the load waits below are written for these ring depths");
  static_assert(NSW * ATB + NSX * BTB <= 160 * 1024, "LDS rings exceed 160 KB");
  __shared__ __attribute__((aligned(16))) uint8_t lds_w[NSW][ATB];
  __shared__ __attribute__((aligned(16))) uint8_t lds_x[NSX][BTB];

  const int w = xcd_work_index(blockIdx.x, p.per_xcd, p.n_items);
  if (w < 0) return;
  const int rt = w % p.n_rt, vg = w / p.n_rt;
  const int nblk = (p.V + 31) / 32;
  const int vb_lo = (int)((long long)vg * nblk / p.n_vg);
  const int vb_hi = (int)((long long)(vg + 1) * nblk / p.n_vg);
  const int v_lo = vb_lo * 32, v_hi = min(p.V, vb_hi * 32);
  const int n_vt = (vb_hi - vb_lo + 7) / 8;
  const int row0 = rt * BR;
  const int H = p.H;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = lane & 31, hh = lane >> 5;
  const int wv = wave & 1, wr = wave >> 1;  // vocab half, row slice
  const int rbase = wr * WROWS;

  const uint16_t* W = static_cast<const uint16_t*>(p.w_vocab);
  const uint16_t* X = static_cast<const uint16_t*>(p.hidden);

  // Direct-to-LDS staging: load j of a wave fills 1 KB chunk c = NW*j + wave
  // of an operand tile; lane l lands at byte 16*l of it, i.e. row RPC*c + l/LPR
  // and physical column l%LPR, and fetches the logical column the swizzle puts
  // there.  The swizzle repeats every 16 rows and chunk j starts RPC*NW*j rows
  // after chunk 0, so a lane's column is the same in every chunk.  W rows are
  // read through a buffer resource covering the current vocab tile's rows:
  // chunk j is chunk 0 moved by a_step bytes, and rows past the vocabulary
  // fall outside the buffer and read as zeros (their logits are masked).  The
  // row offset is part of the per-lane offset, which the hardware checks
  // against the buffer's size; the scalar offset (the stage's k column) is not
  // checked and stays inside a row.  Hidden
  // rows past the row count are clamped to a valid row (never stored); columns
  // past H are clamped and zeroed in LDS before use.
  const int nks = (H + BK - 1) / BK;
  const int n_st = n_vt * nks;
  const bool k_ragged = (H % BK) != 0;
  const int lcol = lane % LPR, lrow = lane / LPR;
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);  // wave index in a scalar register
  static_assert((RPC * NW) % 16 == 0, "chunks must keep the swizzle phase");
  const int l_row = RPC * wave_u + lrow;                        // row of this lane in chunk 0
  const int l_col = 8 * (lcol ^ cswz<BK>(l_row));               // its logical column, every chunk
  const uint32_t a_off = (uint32_t)(l_row * H + l_col) * 2u;    // in the W tile, chunk 0
  const uint32_t a_step = (uint32_t)(RPC * NW) * (uint32_t)H * 2u;  // bytes from chunk j to j+1
  uint32_t b_off[CPB];  // in the hidden states, per chunk (rows may be gathered)
#pragma unroll
  for (int j = 0; j < CPB; ++j) {
    const int r = l_row + RPC * NW * j;
    const int xr = conf_hidden_row(p.row_index, p.hidden_rows, min(row0 + r, p.M - 1));
    b_off[j] = (uint32_t)((size_t)xr * H + l_col) * 2u;
  }
  // Stage cursors: (vocab tile, k-stage, ring slot) of the next W and hidden
  // stage to load and of the stage being consumed, advanced by one stage at a
  // time (no integer division in the loop).
  struct Cursor {
    int st, vt, kq, slot;
  };
  auto advance = [&](Cursor& c, int ring) {
    ++c.st;
    if (++c.kq == nks) {
      c.kq = 0;
      ++c.vt;
    }
    if (++c.slot == ring) c.slot = 0;
  };
  Cursor cw{0, 0, 0, 0}, cx{0, 0, 0, 0};
  int cur_vt = -1;
  __amdgpu_buffer_rsrc_t rsrc_w = buffer_rsrc(W, 0);  // the current vocab tile's rows of W
  const __amdgpu_buffer_rsrc_t rsrc_x =
      buffer_rsrc(X, (uint32_t)((size_t)(p.row_index ? p.hidden_rows : p.M) * H * 2));
  // byte shift of this lane's column in the last, partial k-stage, whose
  // columns past H are clamped (and zeroed in LDS before use)
  auto ragged_shift = [&](int kk) { return 2 * (min(kk + l_col, H - 8) - (kk + l_col)); };
  auto issue_w = [&]() {  // the W tile of stage cw.st
    const int vt = cw.vt, kk = cw.kq * BK;
    if (vt != cur_vt) {
      const int vb = v_lo + vt * BV;
      rsrc_w = buffer_rsrc(W + (size_t)vb * H, (uint32_t)((size_t)(min(p.V, vb + BV) - vb) * H * 2));
      cur_vt = vt;
    }
    uint8_t* dst = &lds_w[cw.slot][wave_u * 1024];
    const uint32_t off = (!k_ragged || kk + BK <= H) ? a_off : a_off + ragged_shift(kk);
#pragma unroll
    for (int j = 0; j < CPA; ++j) dmab16<W_NT ? kLoadNonTemporal : 0>(rsrc_w, dst + NW * j * 1024, off + j * a_step, 2u * kk);
    advance(cw, NSW);
  };
  auto issue_x = [&]() {  // the hidden tile of stage cx.st
    const int kk = cx.kq * BK;
    uint8_t* dst = &lds_x[cx.slot][wave_u * 1024];
    const int dk = (!k_ragged || kk + BK <= H) ? 0 : ragged_shift(kk);
#pragma unroll
    for (int j = 0; j < CPB; ++j) dmab16(rsrc_x, dst + NW * j * 1024, b_off[j] + dk, 2u * kk);
    advance(cx, NSX);
  };
  auto zero_k_tail = [&](const Cursor& c) {
    if (c.kq * BK + l_col < H) return;  // this lane's column is inside H in every chunk
    const int sw = c.st % NSW, sx = c.st % NSX;
#pragma unroll
    for (int j = 0; j < CPA; ++j)
      *reinterpret_cast<uint4*>(&lds_w[sw][(NW * j + wave) * 1024 + lane * 16]) = make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int j = 0; j < CPB; ++j)
      *reinterpret_cast<uint4*>(&lds_x[sx][(NW * j + wave) * 1024 + lane * 16]) = make_uint4(0, 0, 0, 0);
  };

  f32x16 acc[IB][JB];  // set by the first k-step of every vocab tile
  float m_run[JB], s_run[JB];
  int i_run[JB];
  float g_best[JB];  // sampling: best perturbed score and its id
  int g_id[JB];
#pragma unroll
  for (int j = 0; j < JB; ++j) {
    m_run[j] = kNegBig;
    s_run[j] = 0.f;
    i_run[j] = INT_MAX;
    g_best[j] = -INFINITY;
    g_id[j] = INT_MAX;
  }

  // Load order: iteration i issues the hidden tile of stage i+NSX-1, then the
  // W tile of stage i+NSW-1; the prologue issues what iterations before 0
  // would have.  Loads complete in issue order, so when the hidden tile of
  // stage i has landed so has its W tile, and with NSW = 3 only the W tile of
  // stage i+1 (CPA loads) may still be in flight.  Waves with work issue the W
  // tile after the MFMAs of the stage's first k-step, so that its address
  // arithmetic runs while the matrix pipe is busy.
  for (int j = -(NSW - 1); j < 0; ++j) {
    if (j + NSX - 1 >= 0 && cx.st < n_st) issue_x();
    if (cw.st < n_st) issue_w();
  }

  // The kernel arguments' scalar loads have all landed: without this the
  // compiler, which cannot see the LDS waits in inline assembly, re-waits for
  // them (lgkmcnt(0), also draining the fragment reads) inside the loop.
  __builtin_amdgcn_s_waitcnt(0xc07f);
  Cursor cc{0, 0, 0, 0};  // the stage consumed by this iteration (slot: W ring)
  int sx_c = 0;           // its slot in the hidden ring
  for (int i = 0; i < n_st; ++i) {
    if (NSW == 3 && i + 1 < n_st) {
      wait_vmcnt<CPA>();
    } else {
      wait_vmcnt<0>();
    }
    if (k_ragged && cc.kq == nks - 1) zero_k_tail(cc);
    block_barrier();
    // the buffers consumed in the previous iteration are free
    if (cx.st < n_st) issue_x();
    const bool load_w = cw.st < n_st;

    const int vt = cc.vt;
    // first vocab id of this wave's half, from the wave index in a scalar
    // register so that `active` (and the stage cursors updated under it) stays
    // wave-uniform for the compiler
    const int vbase = v_lo + vt * BV + (wave_u & 1) * 128;
    const bool active = vbase < v_hi;
    const bool fresh = cc.kq == 0;
    if (!active && load_w) issue_w();
    if (active) {
      // Operand fragments are double-buffered across k-steps: the LDS reads of
      // step ks+1 are issued before the MFMAs of step ks, which wait only for
      // their own reads.  The swizzle of every row a lane reads depends on the
      // lane alone, so one base address per step plus immediate offsets
      // address all fragments of that step.
      const uint32_t wsb = lds_addr(lds_w[cc.slot]), xsb = lds_addr(lds_x[sx_c]);
      bf16x8 a[2][IB], bfr[2][JB];
      auto frag_load = [&](int ks, int sl) {
        const uint32_t col = ((2 * ks + hh) ^ cswz<BK>(n)) << 4;
        const uint32_t pa = wsb + (wv * 128 + n) * (BK * 2) + col;
        const uint32_t pb = xsb + (rbase + n) * (BK * 2) + col;
        a[sl][0] = lds_read_b128<0 * 32 * BK * 2>(pa);
        a[sl][1] = lds_read_b128<1 * 32 * BK * 2>(pa);
        a[sl][2] = lds_read_b128<2 * 32 * BK * 2>(pa);
        a[sl][3] = lds_read_b128<3 * 32 * BK * 2>(pa);
        bfr[sl][0] = lds_read_b128<0>(pb);
        if constexpr (JB > 1) bfr[sl][1] = lds_read_b128<1 * 32 * BK * 2>(pb);
        if constexpr (JB > 2) bfr[sl][2] = lds_read_b128<2 * 32 * BK * 2>(pb);
        if constexpr (JB > 3) bfr[sl][3] = lds_read_b128<3 * 32 * BK * 2>(pb);
      };
      static_assert(IB == 4 && JB <= 4, "fragment loads are written out for IB = 4, JB <= 4");
      frag_load(0, 0);
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        const int sl = ks & 1;
        if (ks + 1 < NKS) {
          frag_load(ks + 1, sl ^ 1);
          lds_wait<IB + JB>();  // this step's reads are done, the next step's may fly
        } else {
          lds_wait<0>();
        }
#pragma unroll
        for (int ib = 0; ib < IB; ++ib) lds_tie(a[sl][ib]);
#pragma unroll
        for (int jb = 0; jb < JB; ++jb) lds_tie(bfr[sl][jb]);
        if (ks == 0 && fresh) {  // the tile's first k-step starts the accumulators from zero
#pragma unroll
          for (int ib = 0; ib < IB; ++ib)
#pragma unroll
            for (int jb = 0; jb < JB; ++jb) acc[ib][jb] = mfma32x32x16(a[sl][ib], bfr[sl][jb], f32x16{});
        } else {
#pragma unroll
          for (int ib = 0; ib < IB; ++ib)
#pragma unroll
            for (int jb = 0; jb < JB; ++jb) acc[ib][jb] = mfma32x32x16(a[sl][ib], bfr[sl][jb], acc[ib][jb]);
        }
        // keep this step's MFMAs ahead of the next step's reads and waits
        __builtin_amdgcn_sched_barrier(0);
        if (ks == 0 && load_w) {
          issue_w();
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
    if (cc.kq == nks - 1) {
      if (active) {
        fold_tile<JB, !SAMPLE>(acc, v_hi - vbase - 4 * hh, vbase + 4 * hh, m_run, s_run, i_run);
        if constexpr (SAMPLE)
          sample_fold<JB>(acc, v_hi - vbase - 4 * hh, vbase + 4 * hh, row0 + rbase + n, p, g_best, g_id);
      }
    }
    advance(cc, NSW);
    if (++sx_c == NSX) sx_c = 0;
  }
  block_barrier();  // every wave is done with the stage buffers (reused below)
  store_partials<JB, BR, SAMPLE>(p, vg, row0, rbase, wv, hh, n, m_run, s_run, i_run, g_best, g_id, &lds_w[0][0]);
}

// float32 path: one workgroup per (vocabulary group, row); plain FMA dot products.
__global__ __launch_bounds__(256) void slot_conf_f32_kernel(ConfParams p) {
  extern __shared__ float hs[];  // [H] hidden row, then reduction scratch
  const int vg = blockIdx.x, row = blockIdx.y;
  const int tid = threadIdx.x;
  const float* X = static_cast<const float*>(p.hidden);
  const float* W = static_cast<const float*>(p.w_vocab);
  const size_t xrow = (size_t)conf_hidden_row(p.row_index, p.hidden_rows, row);
  for (int k = tid; k < p.H; k += 256) hs[k] = X[xrow * p.H + k];
  __syncthreads();
  const int v_lo = (int)((long long)vg * p.V / p.n_vg);
  const int v_hi = (int)((long long)(vg + 1) * p.V / p.n_vg);
  float m = kNegBig, s = 0.f;
  int idx = INT_MAX;
  float g = -INFINITY;  // sampling candidate
  int gi = INT_MAX;
  for (int v = v_lo + tid; v < v_hi; v += 256) {
    const float* wr = W + (size_t)v * p.H;
    float z = 0.f;
    for (int k = 0; k < p.H; ++k) z = fmaf(hs[k], wr[k], z);
    if (p.part_g) {
      const uint4 r = philox4x32_10_dev((uint32_t)v >> 2, (uint32_t)row, p.off_lo, p.off_hi, p.seed_lo, p.seed_hi);
      const uint32_t words[4] = {r.x, r.y, r.z, r.w};
      const float sc = fmaf(z, p.c2t, gumbel_log2(words[v & 3]));
      if (sc > g) {
        g = sc;
        gi = v;
      }
    }
    if (z > m) {
      s = s * fast_exp2((m - z) * kLog2e) + 1.f;
      m = z;
      idx = v;
    } else {
      s += fast_exp2((z - m) * kLog2e);
    }
  }
  float* rm = hs + p.H;
  float* rs = rm + 256;
  int* ri = reinterpret_cast<int*>(rs + 256);
  float* rg = reinterpret_cast<float*>(ri + 256);
  int* rgi = reinterpret_cast<int*>(rg + 256);
  rm[tid] = m;
  rs[tid] = s;
  ri[tid] = idx;
  rg[tid] = g;
  rgi[tid] = gi;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if (tid < off) {
      float a = rm[tid], b = rs[tid];
      int c = ri[tid];
      stat_merge(a, b, c, rm[tid + off], rs[tid + off], ri[tid + off]);
      rm[tid] = a;
      rs[tid] = b;
      ri[tid] = c;
      float g1 = rg[tid];
      int i1 = rgi[tid];
      sample_merge(g1, i1, rg[tid + off], rgi[tid + off]);
      rg[tid] = g1;
      rgi[tid] = i1;
    }
    __syncthreads();
  }
  if (tid == 0) {
    const size_t o = (size_t)row * p.n_vg + vg;
    p.part_m[o] = rm[0];
    p.part_s[o] = rs[0];
    p.part_idx[o] = ri[0];
    if (p.part_g) {
      p.part_g[o] = rg[0];
      p.part_gi[o] = rgi[0];
    }
  }
}

// Logit of vocab id v for a row, hidden . w_vocab[v], as a float32 dot
// product spread over the 64 lanes of a wave (every lane gets the sum).
__device__ float row_logit(const ConfMergeParams& p, int hrow, int v, int lane) {
  float z = 0.f;
  if (p.bf16) {  // 16-byte loads (H is a multiple of 8): one or two load rounds for H <= 1024
    const uint16_t* hr = static_cast<const uint16_t*>(p.hidden) + (size_t)hrow * p.H;
    const uint16_t* wr = static_cast<const uint16_t*>(p.w_vocab) + (size_t)v * p.H;
#pragma unroll 4
    for (int k = lane * 8; k < p.H; k += 512) {
      const uint4 hv = *reinterpret_cast<const uint4*>(hr + k);
      const uint4 wv = *reinterpret_cast<const uint4*>(wr + k);
      const uint32_t hw[4] = {hv.x, hv.y, hv.z, hv.w}, ww[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        z = fmaf(__uint_as_float(hw[e] << 16), __uint_as_float(ww[e] << 16), z);
        z = fmaf(__uint_as_float(hw[e] & 0xffff0000u), __uint_as_float(ww[e] & 0xffff0000u), z);
      }
    }
  } else {
    const float* hr = static_cast<const float*>(p.hidden) + (size_t)hrow * p.H;
    const float* wr = static_cast<const float*>(p.w_vocab) + (size_t)v * p.H;
    for (int k = lane; k < p.H; k += 64) z = fmaf(hr[k], wr[k], z);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) z += __shfl_xor(z, off);
  return z;
}

// Per row (one wave): merge the vocabulary-group partials in a fixed order
// and finish max_prob = 1 / sum exp(x - max), lse, the target probability
// and, when sampling, the sampled id and its probability.
__global__ __launch_bounds__(256) void slot_conf_merge_kernel(ConfMergeParams p) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= p.M) return;
  // loads that do not depend on the partials go first, so that their latency
  // overlaps the partials' (the target logit needs the target id)
  const int tgt = p.target_ids ? p.target_ids[row] : -1;
  const int hrow = conf_hidden_row(p.row_index, p.hidden_rows, row);
  float m = kNegBig, s = 0.f;
  int idx = INT_MAX;
  float sg = -INFINITY;
  int sgi = INT_MAX;
  for (int g = lane; g < p.n_vg; g += 64) {
    const size_t o = (size_t)row * p.n_vg + g;  // a row's partials are contiguous
    stat_merge(m, s, idx, p.part_m[o], p.part_s[o], p.part_idx[o]);
    if (p.part_g) sample_merge(sg, sgi, p.part_g[o], p.part_gi[o]);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const float m2 = __shfl_xor(m, off);
    const float s2 = __shfl_xor(s, off);
    const int i2 = __shfl_xor(idx, off);
    stat_merge(m, s, idx, m2, s2, i2);
    if (p.part_g) {
      const float g2 = __shfl_xor(sg, off);
      const int gi2 = __shfl_xor(sgi, off);
      sample_merge(sg, sgi, g2, gi2);
    }
  }
  const float lse2 = m * kLog2e + __log2f(s);
  // A row whose logits include a NaN or an infinity has no softmax: its sum
  // is NaN (or 0 when every logit is -inf), so its log-sum-exp is not finite.
  // Such a row reports id -1 and NaN probabilities, and no logit is recomputed
  // for it (its ids are not meaningful).  Every lane holds the same merged
  // statistics, so these conditions are uniform over the wave, as the dot
  // products' shuffles need.
  const bool no_softmax = !(fabsf(lse2) < INFINITY);
  const bool tgt_ok = tgt >= 0 && tgt < p.V && !no_softmax;
  const bool idx_ok = idx >= 0 && idx < p.V && !no_softmax;
  const bool sgi_ok = sgi >= 0 && sgi < p.V && !no_softmax;
  const float zt = tgt_ok ? row_logit(p, hrow, tgt, lane) : 0.f;
  const float zs = p.part_g && sgi_ok ? row_logit(p, hrow, sgi, lane) : 0.f;
  if (lane != 0) return;
  // a row index outside the hidden rows was clamped for the loads: mark its results
  const bool bad = no_softmax || (p.row_index && (p.row_index[row] < 0 || p.row_index[row] >= p.hidden_rows));
  const float nan = __builtin_nanf("");
  if (p.max_prob) p.max_prob[row] = bad ? nan : 1.f / s;
  if (p.argmax_id) p.argmax_id[row] = bad || !idx_ok ? -1 : idx;
  if (p.lse) p.lse[row] = bad ? nan : lse2 * kLn2;
  if (p.part_g) {
    p.sample_id[row] = bad || !sgi_ok ? -1 : sgi;
    p.sample_prob[row] = bad || !sgi_ok ? nan : fast_exp2(zs * kLog2e - lse2);
  }
  if (p.target_ids && p.target_prob) p.target_prob[row] = tgt_ok && !bad ? fast_exp2(zt * kLog2e - lse2) : nan;
}

template <int NW, int BR, bool SAMPLE>
void launch_conf_tile(const ConfParams& p, hipStream_t stream) {
  const dim3 grid(8 * p.per_xcd);
  if (p.w_stream) {
    slot_conf_bf16_kernel<NW, BR, kConfBK, kConfNSW, kConfNSX, SAMPLE, true><<<grid, dim3(NW * 64), 0, stream>>>(p);
  } else {
    slot_conf_bf16_kernel<NW, BR, kConfBK, kConfNSW, kConfNSX, SAMPLE, false><<<grid, dim3(NW * 64), 0, stream>>>(p);
  }
}

hipError_t launch_slot_conf_bf16(const ConfParams& p, hipStream_t stream) {
  if (conf_tile_rows(p.M) == kConfSmallBR) {
    if (p.part_g) {
      launch_conf_tile<kConfSmallNW, kConfSmallBR, true>(p, stream);
    } else {
      launch_conf_tile<kConfSmallNW, kConfSmallBR, false>(p, stream);
    }
  } else if (p.part_g) {
    launch_conf_tile<kConfNW, kConfBR, true>(p, stream);
  } else {
    launch_conf_tile<kConfNW, kConfBR, false>(p, stream);
  }
  return hipGetLastError();
}

hipError_t launch_slot_conf_f32(const ConfParams& p, hipStream_t stream) {
  const size_t shm = (size_t)p.H * 4 + 256 * 20;
  hipLaunchKernelGGL(slot_conf_f32_kernel, dim3(p.n_vg, p.M), dim3(256), shm, stream, p);
  return hipGetLastError();
}

hipError_t launch_slot_conf_merge(const ConfMergeParams& p, hipStream_t stream) {
  hipLaunchKernelGGL(slot_conf_merge_kernel, dim3((p.M + 3) / 4), dim3(256), 0, stream, p);
  return hipGetLastError();
}

}  // namespace zarya
