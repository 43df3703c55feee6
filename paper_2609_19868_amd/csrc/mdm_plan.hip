// Mode A mask budget (Zarya, Sec. 5.1 step 1 "Mask budget planning"): how
// many masks each denoising step of a generation reveals.  Host code only.
//
// With T > 0 discretization steps, a Binomial(N, alpha_0) share of the N masks
// is denoised by exactly T diffusion steps and the rest one per step after
// them; with T = 0 the draw is skipped and T is a quarter of N (rounded up).
#include "common.hpp"
#include "kernels.hpp"

namespace zarya {

int64_t mask_budget_plan(int32_t n_masked, int32_t n_steps, double alpha0, uint64_t seed, int32_t* counts,
                         int32_t* n_diff_steps) {
  const int64_t N = n_masked;
  if (N == 0) {
    *n_diff_steps = 0;
    return 0;
  }
  int64_t T = n_steps, n_diff = N;
  if (T == 0) {
    T = (N + 3) / 4;
  } else {
    // Binomial(N, alpha0) as the count of N Bernoulli draws u_i < alpha0;
    // u_i = uniform of row 0, id i, offset 0: ((x >> 9) + 1/2) * 2^-23, exact
    // in double
    n_diff = 0;
    const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    for (int64_t q = 0; q * 4 < N; ++q) {
      const uint4 r = philox4x32_10((uint32_t)q, 0u, 0u, 0u, k0, k1);
      const uint32_t w[4] = {r.x, r.y, r.z, r.w};
      for (int j = 0; j < 4 && q * 4 + j < N; ++j) {
        const double u = ((double)(w[j] >> 9) + 0.5) * 0x1p-23;
        n_diff += u < alpha0 ? 1 : 0;
      }
    }
  }
  const int64_t len = T + (N - n_diff);
  if (counts) {
    const int64_t base = n_diff / T, extra = n_diff % T;
    for (int64_t t = 0; t < T; ++t) counts[t] = (int32_t)(base + (t < extra ? 1 : 0));
    for (int64_t t = T; t < len; ++t) counts[t] = 1;
  }
  *n_diff_steps = (int32_t)T;
  return len;
}

}  // namespace zarya
