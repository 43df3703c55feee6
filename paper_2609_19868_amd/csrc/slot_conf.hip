// LM-head confidence reduction (gfx950): logits = hidden . W^T reduced per row
// to (max, log-sum-exp, argmax) without writing logits to memory.
//
// What is computed (Zarya, Sec. 5.2: the slot confidence is the probability of
// its first token and verification compares token probabilities with a
// threshold; Table 1: the LM head is the tied embedding W[V, H]): for every
// row, the largest softmax probability, its token id (lowest on ties), the
// log-sum-exp and optionally the probability of a given target id.
//
// bf16 design: a workgroup owns a 256-row tile of `hidden` and a contiguous
// vocabulary range, walked in 256-wide tiles.  The product is computed
// transposed, logits^T = W h^T, with v_mfma_f32_32x32x16_bf16 (each of the 8
// waves owns 128 vocab x 64 rows), so every lane holds values of a single
// row and the per-row reduction runs inside the lane.  After each vocab tile
// the epilogue folds the tile into running (max, sum 2^(x-max), argmax)
// statistics in the log2 domain; at the end of the range the two lane halves
// and the two vocab halves are combined and one partial per (row, range) is
// written.  Operands go through double-buffered, XOR-swizzled LDS tiles.
// Workgroups that share a vocabulary range are mapped to the same XCD so each
// W tile is fetched from HBM once and reused from that XCD's L2.
#include <limits.h>

#include "common.hpp"
#include "kernels.hpp"

namespace zarya {

namespace {

constexpr int BV = kConfTileV;     // vocab entries per tile
constexpr int BR = kConfTileRows;  // hidden rows per tile
constexpr int BK = 32;             // contraction depth per LDS stage
constexpr int ROWB = BK * 2;       // bytes per LDS row

__device__ __forceinline__ int coff(int row, int ch) { return row * ROWB + ((ch ^ ((row >> 2) & 3)) << 4); }

// Merge two (max, sum, argmax) statistics in the log2 domain.  On equal maxima
// the lower id wins, which keeps the result independent of the merge order.
__device__ __forceinline__ void stat_merge(float& m, float& s, int& idx, float m2, float s2, int idx2) {
  const float mn = fmaxf(m, m2);
  const float sa = s == 0.f ? 0.f : s * fast_exp2(m - mn);
  const float sb = s2 == 0.f ? 0.f : s2 * fast_exp2(m2 - mn);
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

}  // namespace

__global__ __launch_bounds__(512) void slot_conf_bf16_kernel(ConfParams p) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[2][2][BV * ROWB];  // [buf][W | hidden]
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
  const int wv = wave & 1, wr = wave >> 1;  // vocab half, row quarter

  const uint16_t* W = static_cast<const uint16_t*>(p.w_vocab);
  const uint16_t* X = static_cast<const uint16_t*>(p.hidden);

  uint4 areg[2], breg[2];
  auto load = [&](int vt, int kk) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int c = j * 512 + tid;
      const int r = c >> 2, ch = c & 3;
      const int k = kk + ch * 8;
      const int vid = v_lo + vt * BV + r;
      const int hr = row0 + r;
      areg[j] = (vid < v_hi && k < H) ? *reinterpret_cast<const uint4*>(W + (size_t)vid * H + k) : make_uint4(0, 0, 0, 0);
      breg[j] = (hr < p.M && k < H) ? *reinterpret_cast<const uint4*>(X + (size_t)hr * H + k) : make_uint4(0, 0, 0, 0);
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int c = j * 512 + tid;
      const int r = c >> 2, ch = c & 3;
      *reinterpret_cast<uint4*>(&lds[buf][0][coff(r, ch)]) = areg[j];
      *reinterpret_cast<uint4*>(&lds[buf][1][coff(r, ch)]) = breg[j];
    }
  };

  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};
  float m_run[2], s_run[2];
  int i_run[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    m_run[j] = kNegBig;
    s_run[j] = 0.f;
    i_run[j] = INT_MAX;
  }

  const int nks = (H + BK - 1) / BK;
  const int n_st = n_vt * nks;
  load(0, 0);
  store(0);
  __syncthreads();

  for (int i = 0; i < n_st; ++i) {
    const int buf = i & 1;
    if (i + 1 < n_st) load((i + 1) / nks, ((i + 1) % nks) * BK);
    const int vt = i / nks;
    const int vbase = v_lo + vt * BV + wv * 128;  // first vocab id of this wave's half
    const bool active = vbase < v_hi;
    if (active) {
      const uint8_t* la = lds[buf][0];
      const uint8_t* lb = lds[buf][1];
#pragma unroll
      for (int ks = 0; ks < BK / 16; ++ks) {
        bf16x8 a[4], bfr[2];
#pragma unroll
        for (int ib = 0; ib < 4; ++ib)
          a[ib] = *reinterpret_cast<const bf16x8*>(la + coff(wv * 128 + ib * 32 + n, 2 * ks + hh));
#pragma unroll
        for (int jb = 0; jb < 2; ++jb)
          bfr[jb] = *reinterpret_cast<const bf16x8*>(lb + coff(wr * 64 + jb * 32 + n, 2 * ks + hh));
#pragma unroll
        for (int ib = 0; ib < 4; ++ib)
#pragma unroll
          for (int jb = 0; jb < 2; ++jb) acc[ib][jb] = mfma32x32x16(a[ib], bfr[jb], acc[ib][jb]);
      }
    }
    if (i % nks == nks - 1) {
      if (active) {
        // fold this vocab tile into the running statistics of the lane's 2 rows;
        // register v of block ib holds vocab id vbase + 32*ib + 8*(v/4) + 4*hh + v%4.
        // Ids are visited in increasing order, so a strict '>' keeps the lowest id.
        const int nvalid = v_hi - vbase;  // ids at local offset >= nvalid are masked
#pragma unroll
        for (int jb = 0; jb < 2; ++jb) {
          float mt = kNegBig;
          int it = INT_MAX;
#pragma unroll
          for (int ib = 0; ib < 4; ++ib)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
              const int off = ib * 32 + 8 * (v >> 2) + 4 * hh + (v & 3);
              const float x = off < nvalid ? acc[ib][jb][v] : -INFINITY;
              if (x > mt) {
                mt = x;
                it = off;
              }
            }
          mt *= kLog2e;
          const float mn = fmaxf(m_run[jb], mt);
          float e = 0.f;
#pragma unroll
          for (int ib = 0; ib < 4; ++ib)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
              const int off = ib * 32 + 8 * (v >> 2) + 4 * hh + (v & 3);
              const float pe = fast_exp2(fmaf(acc[ib][jb][v], kLog2e, -mn));
              e += off < nvalid ? pe : 0.f;
            }
          s_run[jb] = s_run[jb] * fast_exp2(m_run[jb] - mn) + e;
          if (mt > m_run[jb]) i_run[jb] = vbase + it;
          m_run[jb] = mn;
        }
      }
#pragma unroll
      for (int ib = 0; ib < 4; ++ib)
#pragma unroll
        for (int jb = 0; jb < 2; ++jb) acc[ib][jb] = f32x16{};
    }
    if (i + 1 < n_st) store(buf ^ 1);
    __syncthreads();
  }

  // combine the lane halves (disjoint vocab ids of the same rows)
#pragma unroll
  for (int jb = 0; jb < 2; ++jb) {
    const float m2 = __shfl_xor(m_run[jb], 32);
    const float s2 = __shfl_xor(s_run[jb], 32);
    const int i2 = __shfl_xor(i_run[jb], 32);
    stat_merge(m_run[jb], s_run[jb], i_run[jb], m2, s2, i2);
  }
  // combine the two vocab halves through LDS (the tiles are no longer needed)
  float* xm = reinterpret_cast<float*>(&lds[0][0][0]);
  float* xs = xm + 256;
  int* xi = reinterpret_cast<int*>(xs + 256);
  if (wv == 1 && hh == 0) {
#pragma unroll
    for (int jb = 0; jb < 2; ++jb) {
      const int lr = wr * 64 + jb * 32 + n;
      xm[lr] = m_run[jb];
      xs[lr] = s_run[jb];
      xi[lr] = i_run[jb];
    }
  }
  __syncthreads();
  if (wv == 0 && hh == 0) {
#pragma unroll
    for (int jb = 0; jb < 2; ++jb) {
      const int lr = wr * 64 + jb * 32 + n;
      stat_merge(m_run[jb], s_run[jb], i_run[jb], xm[lr], xs[lr], xi[lr]);
      const int row = row0 + lr;
      if (row < p.M) {
        const size_t o = (size_t)vg * p.M + row;
        p.part_m[o] = m_run[jb];
        p.part_s[o] = s_run[jb];
        p.part_idx[o] = i_run[jb];
      }
    }
  }
}

// float32 path: one workgroup per (vocabulary group, row); plain FMA dot products.
__global__ __launch_bounds__(256) void slot_conf_f32_kernel(ConfParams p) {
  extern __shared__ float hs[];  // [H] hidden row, then reduction scratch
  const int vg = blockIdx.x, row = blockIdx.y;
  const int tid = threadIdx.x;
  const float* X = static_cast<const float*>(p.hidden);
  const float* W = static_cast<const float*>(p.w_vocab);
  for (int k = tid; k < p.H; k += 256) hs[k] = X[(size_t)row * p.H + k];
  __syncthreads();
  const int v_lo = (int)((long long)vg * p.V / p.n_vg);
  const int v_hi = (int)((long long)(vg + 1) * p.V / p.n_vg);
  float m = kNegBig, s = 0.f;
  int idx = INT_MAX;
  for (int v = v_lo + tid; v < v_hi; v += 256) {
    const float* wr = W + (size_t)v * p.H;
    float z = 0.f;
    for (int k = 0; k < p.H; ++k) z = fmaf(hs[k], wr[k], z);
    const float x = z * kLog2e;
    if (x > m) {
      s = s * fast_exp2(m - x) + 1.f;
      m = x;
      idx = v;
    } else {
      s += fast_exp2(x - m);
    }
  }
  float* rm = hs + p.H;
  float* rs = rm + 256;
  int* ri = reinterpret_cast<int*>(rs + 256);
  rm[tid] = m;
  rs[tid] = s;
  ri[tid] = idx;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if (tid < off) {
      float a = rm[tid], b = rs[tid];
      int c = ri[tid];
      stat_merge(a, b, c, rm[tid + off], rs[tid + off], ri[tid + off]);
      rm[tid] = a;
      rs[tid] = b;
      ri[tid] = c;
    }
    __syncthreads();
  }
  if (tid == 0) {
    const size_t o = (size_t)vg * p.M + row;
    p.part_m[o] = rm[0];
    p.part_s[o] = rs[0];
    p.part_idx[o] = ri[0];
  }
}

// Per row: merge the vocabulary-group partials in a fixed order and finish
// max_prob = 1 / sum 2^(x - max), lse and the target probability.
__global__ __launch_bounds__(256) void slot_conf_merge_kernel(ConfMergeParams p) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= p.M) return;
  float m = kNegBig, s = 0.f;
  int idx = INT_MAX;
  for (int g = lane; g < p.n_vg; g += 64) {
    const size_t o = (size_t)g * p.M + row;
    stat_merge(m, s, idx, p.part_m[o], p.part_s[o], p.part_idx[o]);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const float m2 = __shfl_xor(m, off);
    const float s2 = __shfl_xor(s, off);
    const int i2 = __shfl_xor(idx, off);
    stat_merge(m, s, idx, m2, s2, i2);
  }
  const float lse2 = m + __log2f(s);
  float z = 0.f;
  int tgt = -1;
  if (p.target_ids) {
    tgt = p.target_ids[row];
    if (tgt >= 0 && tgt < p.V) {
      if (p.bf16) {
        const uint16_t* hr = static_cast<const uint16_t*>(p.hidden) + (size_t)row * p.H;
        const uint16_t* wr = static_cast<const uint16_t*>(p.w_vocab) + (size_t)tgt * p.H;
        for (int k = lane; k < p.H; k += 64) z = fmaf(bf16_to_f32(hr[k]), bf16_to_f32(wr[k]), z);
      } else {
        const float* hr = static_cast<const float*>(p.hidden) + (size_t)row * p.H;
        const float* wr = static_cast<const float*>(p.w_vocab) + (size_t)tgt * p.H;
        for (int k = lane; k < p.H; k += 64) z = fmaf(hr[k], wr[k], z);
      }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) z += __shfl_xor(z, off);
  }
  if (lane != 0) return;
  p.max_prob[row] = 1.f / s;
  p.argmax_id[row] = idx;
  if (p.lse) p.lse[row] = lse2 * kLn2;
  if (p.target_ids && p.target_prob) {
    p.target_prob[row] = (tgt >= 0 && tgt < p.V) ? fast_exp2(z * kLog2e - lse2) : __builtin_nanf("");
  }
}

hipError_t launch_slot_conf_bf16(const ConfParams& p, hipStream_t stream) {
  hipLaunchKernelGGL(slot_conf_bf16_kernel, dim3(8 * p.per_xcd), dim3(512), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_slot_conf_f32(const ConfParams& p, hipStream_t stream) {
  const size_t shm = (size_t)p.H * 4 + 256 * 12;
  hipLaunchKernelGGL(slot_conf_f32_kernel, dim3(p.n_vg, p.M), dim3(256), shm, stream, p);
  return hipGetLastError();
}

hipError_t launch_slot_conf_merge(const ConfMergeParams& p, hipStream_t stream) {
  hipLaunchKernelGGL(slot_conf_merge_kernel, dim3((p.M + 3) / 4), dim3(256), 0, stream, p);
  return hipGetLastError();
}

}  // namespace zarya
