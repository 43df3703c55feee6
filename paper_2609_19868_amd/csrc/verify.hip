// Verification step of slotted speculative decoding (gfx950): token acceptance
// and the KV-cache append of the accepted tokens.
//
// What is computed (Zarya, Sec. 5.2 "Verification phase" and "KV cache
// update"; Sec. 6 token threshold 0.4): in every slot listed as verified, a
// draft token whose probability under the autoregressive verification pass
// exceeds the threshold is accepted -- with the prefix rule only the leading
// run of such tokens -- and the accepted tokens' keys and values are appended
// to the cache after the committed prefix, which grows by their number.
//
// Both kernels are tiny next to the attention and the LM head (integer and
// copy work on a few KB per batch row); one workgroup per batch row.
#include "common.hpp"
#include "kernels.hpp"

namespace zarya {

namespace {

constexpr int kThreads = 256;

// Marks the slots of row b listed in `list` (the first negative entry ends the
// list, ids >= S are skipped) in flags[0..S).  Ends with a barrier.
__device__ void mark_listed(const int32_t* list, int S, int* flags) {
  __shared__ int end;
  if (threadIdx.x == 0) end = S;
  for (int s = threadIdx.x; s < S; s += kThreads) flags[s] = 0;
  __syncthreads();
  for (int i = threadIdx.x; i < S; i += kThreads)
    if (list[i] < 0) atomicMin(&end, i);  // LDS integer minimum: order-free
  __syncthreads();
  for (int i = threadIdx.x; i < end; i += kThreads) {
    const int s = list[i];
    if (s < S) flags[s] = 1;
  }
  __syncthreads();
}

}  // namespace

// One workgroup per batch row; one thread per slot walks the slot's tokens.
__global__ __launch_bounds__(kThreads) void verify_accept_kernel(AcceptParams p) {
  __shared__ int flags[1024];
  __shared__ int total;
  const int b = blockIdx.x;
  if (threadIdx.x == 0) total = 0;
  mark_listed(p.selected + (size_t)b * p.S, p.S, flags);
  int mine = 0;
  for (int s = threadIdx.x; s < p.S; s += kThreads) {
    const float* tp = p.token_prob + ((size_t)b * p.S + s) * p.L;
    uint8_t* acc = p.accepted + ((size_t)b * p.S + s) * p.L;
    int n = 0;
    bool run = flags[s] != 0;  // prefix rule: still inside the leading run
    for (int r = 0; r < p.L; ++r) {
      const bool pass = flags[s] != 0 && tp[r] > p.threshold;
      run = run && pass;
      const bool a = p.rule == 0 ? run : pass;
      acc[r] = a ? 1 : 0;
      n += a ? 1 : 0;
    }
    p.n_accepted[(size_t)b * p.S + s] = n;
    mine += n;
  }
  atomicAdd(&total, mine);  // integer sum: order-free
  __syncthreads();
  if (threadIdx.x == 0 && p.n_total) p.n_total[b] = total;
}

// One workgroup per batch row: list the accepted tokens in append order in
// LDS (a slot listed twice counts at its first position only), check that
// they fit, then copy their K and V rows of every KV head in 16-byte pieces
// and move the row's prefix length.
__global__ __launch_bounds__(kThreads) void kv_append_kernel(AppendParams p) {
  __shared__ int slot_of[1024];   // order position -> slot id (or -1)
  __shared__ int count_of[1024];  // order position -> accepted tokens of that slot
  __shared__ int start_of[1024];  // order position -> first index in `tokens`
  __shared__ int first_pos[1024];  // slot id -> first order position listing it
  __shared__ int tokens[kAppendMaxTokens];
  __shared__ int n_tok, p0, ok;
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int32_t* ord = p.order + (size_t)b * p.S;
  if (tid == 0) n_tok = p.S;
  for (int s = tid; s < p.S; s += kThreads) first_pos[s] = p.S;
  __syncthreads();
  for (int i = tid; i < p.S; i += kThreads)
    if (ord[i] < 0) atomicMin(&n_tok, i);  // end of the order list
  __syncthreads();
  const int n_pos = n_tok;
  for (int i = tid; i < n_pos; i += kThreads) {
    const int s = ord[i];
    if (s < p.S) atomicMin(&first_pos[s], i);  // LDS integer minimum: order-free
  }
  __syncthreads();
  for (int i = tid; i < p.S; i += kThreads) {
    const int s = i < n_pos ? ord[i] : -1;
    // a slot listed again is skipped: its tokens are committed once
    const bool valid = s >= 0 && s < p.S && first_pos[s] == i;
    int c = 0;
    if (valid) {
      const uint8_t* a = p.accepted + ((size_t)b * p.S + s) * p.L;
      for (int r = 0; r < p.L; ++r) c += a[r] != 0 ? 1 : 0;
    }
    slot_of[i] = valid ? s : -1;
    count_of[i] = c;
  }
  __syncthreads();
  if (tid == 0) {  // exclusive scan over at most 1024 entries, in order
    int acc = 0;
    for (int i = 0; i < p.S; ++i) {
      start_of[i] = acc;
      acc += count_of[i];
    }
    n_tok = acc;
    p0 = p.prefix_lens[b];
    ok = p0 >= 0 && (long long)p0 + acc <= p.C;
  }
  __syncthreads();
  if (!ok) return;  // uniform: the row does not fit and stays unchanged
  for (int i = tid; i < p.S; i += kThreads) {
    const int s = slot_of[i];
    if (s < 0) continue;
    const uint8_t* a = p.accepted + ((size_t)b * p.S + s) * p.L;
    int k = start_of[i];
    for (int r = 0; r < p.L; ++r)
      if (a[r] != 0) tokens[k++] = s * p.L + r;
  }
  __syncthreads();
  const int T = p.S * p.L;
  const int pieces = p.row_bytes / 16;
  const int n = n_tok;
  // one flat loop over (head, token, 16-byte piece): every thread's loads are
  // independent of its stores (the slot K/V and the cache never overlap), so
  // many are in flight at once
  const char* __restrict__ ks = static_cast<const char*>(p.k_slot);
  const char* __restrict__ vs = static_cast<const char*>(p.v_slot);
  char* __restrict__ kc = static_cast<char*>(p.k_cache);
  char* __restrict__ vc = static_cast<char*>(p.v_cache);
  const int per_head = n * pieces;
  for (int e = tid; e < p.Hkv * per_head; e += kThreads) {
    const int g = e / per_head, r = e - g * per_head;
    const int i = r / pieces, c = r - i * pieces;
    const size_t src = (((size_t)b * p.Hkv + g) * T + tokens[i]) * p.row_bytes + (size_t)c * 16;
    const size_t dst = (((size_t)b * p.Hkv + g) * p.C + p0 + i) * p.row_bytes + (size_t)c * 16;
    const uint4 kv = *reinterpret_cast<const uint4*>(ks + src);
    const uint4 vv = *reinterpret_cast<const uint4*>(vs + src);
    *reinterpret_cast<uint4*>(kc + dst) = kv;
    *reinterpret_cast<uint4*>(vc + dst) = vv;
  }
  if (tid == 0) p.prefix_lens[b] = p0 + n;
}

hipError_t launch_verify_accept(const AcceptParams& p, hipStream_t stream) {
  verify_accept_kernel<<<dim3(p.B), dim3(kThreads), 0, stream>>>(p);
  return hipGetLastError();
}

hipError_t launch_kv_append(const AppendParams& p, hipStream_t stream) {
  kv_append_kernel<<<dim3(p.B), dim3(kThreads), 0, stream>>>(p);
  return hipGetLastError();
}

}  // namespace zarya
