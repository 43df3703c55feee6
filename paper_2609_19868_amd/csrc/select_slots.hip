// First-hitting slot selection (Zarya, Sec. 5.2 "Slot selection"; Sec. 6 uses
// slot_threshold = 0.9).  One workgroup per batch row.
//
// Slot confidence is the first token's probability (the paper's rule) or the
// mean over the slot, summed in float64 in token order, divided by L and
// rounded once to float32.  Every open slot gets its rank in first-hitting
// order: the number of open slots with a higher confidence, or an equal one
// and a lower index.  THRESHOLD keeps the open slots whose confidence exceeds
// the threshold (strictly) -- exactly the first ranks -- or, when none does,
// the rank-0 slot; TOP_K keeps ranks below k.  A kept slot is written at its
// rank, so the output is in first-hitting order without a sort.
#include "common.hpp"
#include "kernels.hpp"

namespace zarya {

__global__ __launch_bounds__(256) void select_slots_kernel(SelectParams p) {
  __shared__ float conf[1024];
  __shared__ uint8_t is_open[1024];
  __shared__ int n_open, n_above;
  const int b = blockIdx.x, tid = threadIdx.x;
  const float tau = p.threshold;
  if (tid == 0) {
    n_open = 0;
    n_above = 0;
  }
  __syncthreads();
  for (int s = tid; s < p.S; s += 256) {
    const float* tc = p.token_conf + ((size_t)b * p.S + s) * p.L;
    float c;
    if (p.conf_rule == 0) {
      c = tc[0];
    } else {
      double acc = 0.0;
      for (int r = 0; r < p.L; ++r) acc = acc + (double)tc[r];
      c = (float)(acc / (double)p.L);
    }
    if (c != c) c = -INFINITY;  // a NaN confidence ranks last and never passes the threshold
    const bool op = p.slot_open ? p.slot_open[(size_t)b * p.S + s] != 0 : true;
    conf[s] = c;
    is_open[s] = op;
    p.slot_conf[(size_t)b * p.S + s] = op ? c : -1.f;
    if (op) {
      atomicAdd(&n_open, 1);
      if (c > tau) atomicAdd(&n_above, 1);
    }
  }
  __syncthreads();
  const int n_sel = p.rule == 0 ? (n_above > 0 ? n_above : (n_open > 0 ? 1 : 0)) : min(p.k, n_open);
  int32_t* sel = p.selected + (size_t)b * p.S;
  for (int s = tid; s < p.S; s += 256) {
    if (!is_open[s]) continue;
    const float c = conf[s];
    int rank = 0;
    for (int o = 0; o < p.S; ++o) {
      if (!is_open[o]) continue;
      const float co = conf[o];
      rank += (co > c) || (co == c && o < s);
    }
    if (rank < n_sel) sel[rank] = s;
  }
  for (int pos = n_sel + tid; pos < p.S; pos += 256) sel[pos] = -1;
  if (tid == 0) p.n_selected[b] = n_sel;
}

hipError_t launch_select_slots(const SelectParams& p, hipStream_t stream) {
  hipLaunchKernelGGL(select_slots_kernel, dim3(p.B), dim3(256), 0, stream, p);
  return hipGetLastError();
}

}  // namespace zarya
