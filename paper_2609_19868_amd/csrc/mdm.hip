// Mode A of Zarya (MDM sampling with first-hitting denoising, Sec. 5.1):
// the positions a denoising step reveals (gfx950).  The mask budget of a
// generation is host code, in mdm_plan.hip.
//
// What is computed (Sec. 5.1 steps 1-3): a generation with N masks runs T
// diffusion steps that together reveal a Binomial(N, alpha_0) share of the
// masks, then reveals the rest one per step; with T = 0 the draw is skipped
// and T is a quarter of N.  At each step the model's drawn tokens of some
// masked positions are committed -- the most confident ones, the leftmost ones
// (sequential phase) or a uniformly random set (the first-hitting sampler) --
// and those positions join the committed part of the sequence.
//
// The reveal is integer work on at most 8192 positions per row: each key packs
// the rule's ordering (confidence, position, or a Philox uniform) above the
// position, so one ascending bitonic sort in LDS yields the reveal order with
// ties broken by the lower position.
#include "common.hpp"
#include "kernels.hpp"

namespace zarya {

namespace {

constexpr int kThreads = 1024;
constexpr uint64_t kClosed = ~0ull;  // sorts after every open position

// Float32 confidence -> 32-bit key that increases as the confidence falls
// (NaN counts as -inf, -0 as +0), by integer operations only.
__device__ __forceinline__ uint32_t conf_desc_key(float c) {
  uint32_t b = __float_as_uint(c);
  if ((b & 0x7F800000u) == 0x7F800000u && (b & 0x007FFFFFu) != 0) b = 0xFF800000u;  // NaN -> -inf
  if (b == 0x80000000u) b = 0;                                                        // -0 -> +0
  const uint32_t asc = (b & 0x80000000u) ? ~b : (b | 0x80000000u);  // increases with the value
  return ~asc;
}

// Philox uniform of (row, position) as its 23-bit integer (x >> 9): the same
// order as u = ((x >> 9) + 1/2) * 2^-23.
__device__ __forceinline__ uint32_t uniform_bits(const RevealParams& p, int row, int pos) {
  const uint4 r = philox4x32_10_dev((uint32_t)pos >> 2, (uint32_t)row, p.off_lo, p.off_hi, p.seed_lo, p.seed_hi);
  const uint32_t w[4] = {r.x, r.y, r.z, r.w};
  return w[pos & 3] >> 9;
}

}  // namespace

__global__ __launch_bounds__(kThreads) void mdm_reveal_kernel(RevealParams p) {
  __shared__ uint64_t keys[kRevealMaxN];
  __shared__ int n_open;
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const size_t base = (size_t)b * p.N;
  if (tid == 0) n_open = 0;
  __syncthreads();
  int mine = 0;
  for (int i = tid; i < p.NP; i += kThreads) {
    uint64_t key = kClosed;
    if (i < p.N && p.mask[base + i] != 0) {
      uint32_t hi = 0;
      if (p.rule == 0) {
        hi = conf_desc_key(p.conf[base + i]);
      } else if (p.rule == 2) {
        hi = uniform_bits(p, b, i);
      }
      key = ((uint64_t)hi << 32) | (uint32_t)i;
      ++mine;
    }
    keys[i] = key;
  }
  atomicAdd(&n_open, mine);  // integer sum: order-free
  __syncthreads();
  // ascending bitonic sort of NP keys (NP a power of two)
  for (int size = 2; size <= p.NP; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int t = tid; t < p.NP / 2; t += kThreads) {
        const int lo = 2 * t - (t & (stride - 1));  // first element of the pair
        const int hi = lo + stride;
        const bool up = (lo & size) == 0;
        const uint64_t a = keys[lo], c = keys[hi];
        if ((a > c) == up) {
          keys[lo] = c;
          keys[hi] = a;
        }
      }
      __syncthreads();
    }
  }
  const int n = min(max(p.k[b], 0), n_open);
  for (int j = tid; j < p.N; j += kThreads) {
    const int pos = j < n ? (int)(uint32_t)keys[j] : -1;
    p.order[base + j] = pos;
    if (j < n) {
      p.mask[base + pos] = 0;
      if (p.tokens) p.tokens[base + pos] = p.sample_id[base + pos];
    }
  }
  if (tid == 0 && p.n_revealed) p.n_revealed[b] = n;
}

hipError_t launch_mdm_reveal(const RevealParams& p, hipStream_t stream) {
  mdm_reveal_kernel<<<dim3(p.B), dim3(kThreads), 0, stream>>>(p);
  return hipGetLastError();
}

}  // namespace zarya
