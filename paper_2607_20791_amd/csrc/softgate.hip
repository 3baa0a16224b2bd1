// Soft compatibility gate (Appendix C): one probe step with the relaxed rule.
//
// The greedy token y is appended when the probe stays compatible.  Otherwise,
// on a soft step (the first soft_steps tokens of the probe), the K most
// probable next tokens are examined: those that keep the probe compatible
// carry a probability mass m under softmax(z) (temperature 1, whole
// vocabulary); if there is one and m >= rho, the most probable of them is
// appended and the probe goes on, else y is recorded and the prompt is
// sampled (INCOMPAT).  Later steps follow the hard rule.
//
// Two kernels.  The chunk pass (one workgroup per row and 4096-logit chunk)
// writes the chunk's K largest logits as (value, -index) keys in descending
// order, its maximum and sum of exp(z - max).  The decision (one workgroup per
// row) merges the chunk lists into the row's top K (equal logits: lower id
// first), forms the softmax denominator from the chunk sums, checks the
// candidates against the table and updates the probe state.  The mass is
// summed in candidate order, so the result does not depend on the launch.
#include "gatecheck.hpp"
#include "kernels.hpp"

namespace rgd {

namespace {

constexpr int kPer = 16;  // logits per thread of the chunk pass (chunk <= 4096)

RGD_DEV unsigned long long pack_key(float v, int idx) {
  return ((unsigned long long)ordered_u32(v) << 32) | (unsigned long long)(0xFFFFFFFFu - uint32_t(idx));
}
RGD_DEV int key_index(unsigned long long k) { return int(0xFFFFFFFFu - uint32_t(k & 0xFFFFFFFFull)); }
RGD_DEV float key_value(unsigned long long k) { return from_ordered_u32(uint32_t(k >> 32)); }

RGD_DEV unsigned long long block_max_key(unsigned long long k, unsigned long long* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const unsigned long long t = __shfl_xor(k, o, 64);
    k = t > k ? t : k;
  }
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = k;
  __syncthreads();
  unsigned long long t = red[0];
  for (int i = 1; i < int(blockDim.x >> 6); ++i) t = red[i] > t ? red[i] : t;
  return t;
}

__global__ __launch_bounds__(256) void topk_chunk_kernel(SoftArgs a) {
  __shared__ float red[4];
  __shared__ unsigned long long redk[4];
  const int c = blockIdx.x, r = blockIdx.y;
  const float* zr = a.z + r * a.ldz;
  const int lo = c * a.chunk, hi = min(a.V, lo + a.chunk);
  unsigned long long key[kPer];
  float v[kPer];
  float mx = -INFINITY;
#pragma unroll
  for (int e = 0; e < kPer; ++e) {
    const int i = lo + threadIdx.x + e * 256;
    v[e] = i < hi ? zr[i] : -INFINITY;
    key[e] = i < hi ? pack_key(v[e], i) : 0ull;  // 0: no logit
    mx = fmaxf(mx, v[e]);
  }
  mx = block_max(mx, red);
  float sum = 0.f;
#pragma unroll
  for (int e = 0; e < kPer; ++e)
    if (key[e]) sum += expf(v[e] - mx);
  sum = block_sum(sum, red);
  const long long rc = (long long)r * a.nchunks + c;
  if (threadIdx.x == 0) {
    a.cmax[rc] = mx;
    a.csum[rc] = sum;
  }
  // the chunk's K largest keys, largest first (0 past the chunk's length)
  unsigned long long prev = ~0ull;
  for (int t = 0; t < a.K; ++t) {
    unsigned long long best = 0ull;
#pragma unroll
    for (int e = 0; e < kPer; ++e) best = (key[e] < prev && key[e] > best) ? key[e] : best;
    best = block_max_key(best, redk);
    if (threadIdx.x == 0) a.keys[rc * a.K + t] = best;
    prev = best;
  }
}

__global__ __launch_bounds__(256) void soft_decide_kernel(SoftArgs a) {
  __shared__ float red[4];
  __shared__ unsigned long long redk[4];
  __shared__ unsigned long long top[kMaxTopK];
  __shared__ int flag[kMaxTopK];
  __shared__ int sh_tok, sh_fail;
  const GateArgs& g = a.g;
  const int r = blockIdx.x, b = g.row_prompt[r];
  if (g.event[b] != -1) return;  // decided earlier (uniform over the workgroup)
  const int nch = a.nchunks, K = a.K;
  // row maximum and softmax denominator from the chunk summaries (fixed order)
  const long long r0 = (long long)r * nch;
  const float mc = (int)threadIdx.x < nch ? a.cmax[r0 + threadIdx.x] : -INFINITY;
  const float M = block_max(mc, red);
  const float sc = (int)threadIdx.x < nch ? a.csum[r0 + threadIdx.x] * expf(mc - M) : 0.f;
  const float S = block_sum(sc, red);
  // the row's K largest keys: K rounds over the chunk lists
  const unsigned long long* kr = a.keys + r0 * K;
  unsigned long long prev = ~0ull;
  for (int t = 0; t < K; ++t) {
    unsigned long long best = 0ull;
    for (int i = threadIdx.x; i < nch * K; i += 256) {
      const unsigned long long k = kr[i];
      best = (k < prev && k > best) ? k : best;
    }
    best = block_max_key(best, redk);
    if (threadIdx.x == 0) top[t] = best;
    prev = best;
  }
  if ((int)threadIdx.x < kMaxTopK) flag[threadIdx.x] = 0;
  __syncthreads();
  const int j = g.probe_len[b];
  const int* q = g.probe_tokens + (long long)b * g.k;
  const int y = key_index(top[0]);
  bool m = false;
  for (int e = threadIdx.x; e < g.n_entries; e += 256) m = m || entry_matches(g, e, b, q, j, y);
  const bool compat = g.all_compatible || __syncthreads_or(m);
  if (threadIdx.x == 0) {
    sh_tok = y;
    sh_fail = compat ? 0 : 1;
  }
  if (!compat && j < a.soft_steps) {
    // which of the K candidates keep the probe compatible
    for (int p = threadIdx.x; p < K * g.n_entries; p += 256) {
      const int t = p / g.n_entries, e = p % g.n_entries;
      if (top[t] && entry_matches(g, e, b, q, j, key_index(top[t]))) atomicOr(&flag[t], 1);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      float mass = 0.f;
      int first = -1;
      for (int t = 0; t < K; ++t)
        if (flag[t]) {
          mass += expf(key_value(top[t]) - M) / S;
          if (first < 0) first = t;
        }
      if (first >= 0 && mass >= a.rho) {
        sh_tok = key_index(top[first]);
        sh_fail = 0;
      }
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const int tok = sh_tok;
    g.probe_tokens[(long long)b * g.k + j] = tok;
    g.probe_len[b] = j + 1;
    if (g.cur_tok) g.cur_tok[r] = tok;
    g.event[b] = sh_fail ? 0 : (g.eos >= 0 && tok == g.eos) ? 1 : (j + 1 >= g.k) ? 2 : -1;
  }
}

}  // namespace

hipError_t probe_update_soft(const SoftArgs& a, hipStream_t s) {
  if (a.g.R <= 0) return hipSuccess;
  if (a.K < 1 || a.K > kMaxTopK || a.chunk > kPer * 256 || a.nchunks > 256 ||
      (long long)a.nchunks * a.chunk < a.V)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(topk_chunk_kernel, dim3(a.nchunks, a.g.R), dim3(256), 0, s, a);
  hipLaunchKernelGGL(soft_decide_kernel, dim3(a.g.R), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace rgd
