// Token selection and the refusal gate.
//
// min-p sampling (temperature first): with m the row maximum, a token is kept
// when w_i = exp2((z_i - m) * log2(e) / T) >= p_min, and the draw returns the
// smallest kept id whose running kept-weight sum exceeds u * W.  Two kernels:
// the first has one workgroup per (row, chunk of logits) and writes the
// chunk's kept-weight sum; the second has one workgroup per row, forms the
// chunk prefix in chunk order, locates u * W and rescans that one chunk with a
// block-wide prefix scan.  Logits are read once per draw from HBM (plus the
// one rescanned chunk); the row maximum comes in as partial maxima from the
// LM-head epilogue.  Standalone rows have no such maxima: the chunk pass keeps
// each chunk's maximum and its sum relative to it, and only chunks inside the
// min-p window below the row maximum are summed again; with many rows one
// workgroup per row does all of it in one launch.  No cross-workgroup
// synchronisation: a release/acquire handshake between the workgroups of a
// row (the last to arrive makes the draw) writes back the whole L2 at every
// release and measured ten times slower.
#include "gatecheck.hpp"
#include "kernels.hpp"
#include "philox.hpp"
#include "rownorm.hpp"

namespace rgd {

namespace {

constexpr float kLog2e = 1.4426950408889634f;

// Standalone rows: from this many rows on, one workgroup per row (one launch)
// keeps every CU streaming; below it, chunk workgroups (two launches) spread a
// few rows over the whole chip.  Measured on the 152064-logit sweep rows:
// 256 rows 39 us vs 41 us; 16 rows 25 us vs 16 us.
constexpr int kRowKernelMinRows = 128;

// Kept-weight of one logit.  The hardware 2^x (no denormal range fix-up: a
// weight below 2^-126 flushes to 0); the chunk sums and the rescan use this
// same expression so both see the same kept set.
RGD_DEV float kept_weight(float z, float mx, float kT, float p_min) {
  const float w = __builtin_amdgcn_exp2f((z - mx) * kT);
  return w >= p_min ? w : -1.f;  // -1 marks a dropped token
}

__global__ void fill_u32_kernel(uint32_t* p, uint32_t v, long long n) {
  for (long long i = blockIdx.x * 256ll + threadIdx.x; i < n; i += 256ll * gridDim.x) p[i] = v;
}

// Per-chunk maxima; chunk is a multiple of 1024 (4 float4 per thread per
// 1024 logits) and V a multiple of 4.
__global__ __launch_bounds__(256) void chunk_max_kernel(const float* z, long long ldz, int V, int chunk,
                                                        float* cmax) {
  __shared__ float red[4];
  const int c = blockIdx.x, r = blockIdx.y;
  const float* zr = z + r * ldz;
  const int lo = c * chunk, hi = min(V, lo + chunk);
  float mx = -INFINITY;
  for (int i0 = lo; i0 < hi; i0 += 4096) {
    float4 v[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int i = i0 + (threadIdx.x + k * 256) * 4;
      v[k] = i < hi ? *(const float4*)(zr + i) : float4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) mx = fmaxf(mx, fmaxf(fmaxf(v[k].x, v[k].y), fmaxf(v[k].z, v[k].w)));
  }
  mx = block_max(mx, red);
  if (threadIdx.x == 0) cmax[(long long)r * gridDim.x + c] = mx;
}

RGD_DEV unsigned long long pack_key(float v, int idx) {
  return ((unsigned long long)ordered_u32(v) << 32) | (unsigned long long)(0xFFFFFFFFu - uint32_t(idx));
}

// VEC: float4 loads (V and ldz multiples of 4, rows 16-byte aligned);
// otherwise one logit per thread and step.
template <bool VEC>
__global__ __launch_bounds__(256) void argmax_kernel(const float* z, long long ldz, int V, int chunk,
                                                     unsigned long long* best) {
  __shared__ unsigned long long red[4];
  const int c = blockIdx.x, r = blockIdx.y;
  const float* zr = z + r * ldz;
  const int lo = c * chunk, hi = min(V, lo + chunk);
  unsigned long long k = 0;
  if (VEC) {
    for (int i0 = lo; i0 < hi; i0 += 4096) {
      float4 v[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int i = i0 + (threadIdx.x + j * 256) * 4;
        v[j] = i < hi ? *(const float4*)(zr + i) : float4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int i = i0 + (threadIdx.x + j * 256) * 4;
        if (i < hi) {
          unsigned long long t = pack_key(v[j].x, i);
          k = t > k ? t : k;
          t = pack_key(v[j].y, i + 1);
          k = t > k ? t : k;
          t = pack_key(v[j].z, i + 2);
          k = t > k ? t : k;
          t = pack_key(v[j].w, i + 3);
          k = t > k ? t : k;
        }
      }
    }
  } else {
    for (int i = lo + threadIdx.x; i < hi; i += 256) {
      const unsigned long long t = pack_key(zr[i], i);
      k = t > k ? t : k;
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const unsigned long long t = __shfl_xor(k, o, 64);
    k = t > k ? t : k;
  }
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = k;
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned long long t = red[0];
    for (int i = 1; i < 4; ++i) t = red[i] > t ? red[i] : t;
    atomicMax(best + r, t);
  }
}

RGD_DEV float row_max_from_partials(const float* pmax, int npmax, int r, float* red) {
  const float* p = pmax + (long long)r * npmax;
  float mx = -INFINITY;
  const int n4 = npmax & ~3;
  if ((((uintptr_t)p) & 15) == 0 && npmax <= 1024 && n4 >= 4) {
    // one float4 and one scalar per thread, loaded unconditionally from
    // clamped indices and masked afterwards (a predicated load makes the
    // compiler wait for it where the branches join)
    const int i = threadIdx.x * 4, j = n4 + threadIdx.x;
    const float4 v = *(const float4*)(p + min(i, n4 - 4));
    const float t = p[min(j, npmax - 1)];
    if (i < n4) mx = fmaxf(fmaxf(v.x, v.y), fmaxf(v.z, v.w));
    if (j < npmax) mx = fmaxf(mx, t);
  } else {
    for (int i = threadIdx.x; i < npmax; i += 256) mx = fmaxf(mx, p[i]);
  }
  return block_max(mx, red);
}

// Inclusive block scan (256 threads) of one float per thread.
RGD_DEV float block_inclusive_scan(float v, float* wsum) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const float t = __shfl_up(v, o, 64);
    if (lane >= o) v += t;
  }
  __syncthreads();
  if (lane == 63) wsum[w] = v;
  __syncthreads();
  float off = 0.f;
  for (int i = 0; i < w; ++i) off += wsum[i];
  return v + off;
}

// Selects the token of row r for target u (in [0,1)); `mine` is chunk
// threadIdx.x's kept sum (0 past the last chunk).  NTH threads; chunk / NTH
// must be a multiple of 4 and at most 16.  Returns the token id (valid in every
// thread).
template <int NTH>
RGD_DEV int select_token(const SampleArgs& a, int r, float mx, float u, float mine) {
  constexpr int NW = NTH / 64, PMAX = 4096 / NTH;
  __shared__ float csum[256];
  __shared__ int sh_chunk, sh_last_nz;
  __shared__ float sh_base, sh_target;
  __shared__ float wsum[NW];
  __shared__ int red_i[NW];
  const float kT = kLog2e / a.T;
  const float thr = a.row_thr ? a.row_thr[r] : a.p_min;  // kept: w >= thr
  // running sum over chunks in chunk order (one chunk per thread)
  const int c = threadIdx.x;
  const float incl_c = block_inclusive_scan(mine, wsum);
  if (c < 256) csum[c] = incl_c;
  if (c == 0) {
    sh_chunk = 0x7FFFFFFF;
    sh_last_nz = 0;
  }
  __syncthreads();
  const float total = csum[a.nchunks - 1];
  const float target = u * total;
  if (c < a.nchunks) {
    const float prev = c ? csum[c - 1] : 0.f;
    if (incl_c > prev) atomicMax(&sh_last_nz, c);
    if (incl_c > target && prev <= target) atomicMin(&sh_chunk, c);
  }
  __syncthreads();
  if (c == 0) {
    if (sh_chunk == 0x7FFFFFFF) sh_chunk = sh_last_nz;
    sh_base = sh_chunk ? csum[sh_chunk - 1] : 0.f;
    sh_target = target;
  }
  __syncthreads();
  // rescan of the chosen chunk: thread t owns `per` consecutive logits
  // (per = chunk / NTH <= PMAX, a multiple of 4; V is a multiple of 4)
  const int lo = sh_chunk * a.chunk, hi = min(a.V, lo + a.chunk);
  const int per = a.chunk / NTH;
  const int e0 = lo + threadIdx.x * per, e1 = min(hi, e0 + per);
  const float* zr = a.z + r * a.ldz;
  float4 zv[PMAX / 4];
#pragma unroll
  for (int k = 0; k < PMAX / 4; ++k)
    zv[k] = (4 * k < per && e0 + 4 * k < e1) ? *(const float4*)(zr + e0 + 4 * k) : float4{0.f, 0.f, 0.f, 0.f};
  float wv[PMAX];
  float ts = 0.f;
#pragma unroll
  for (int i = 0; i < PMAX; ++i) {
    const float zi = i % 4 == 0 ? zv[i / 4].x : i % 4 == 1 ? zv[i / 4].y : i % 4 == 2 ? zv[i / 4].z : zv[i / 4].w;
    const float w = (i < per && e0 + i < e1) ? kept_weight(zi, mx, kT, thr) : -1.f;
    wv[i] = w;
    ts += w > 0.f ? w : 0.f;
  }
  const float incl = block_inclusive_scan(ts, wsum);
  float run = sh_base + (incl - ts);
  int found = 0x7FFFFFFF, last = -1;
#pragma unroll
  for (int i = 0; i < PMAX; ++i) {
    if (wv[i] >= 0.f) {
      run += wv[i];
      last = e0 + i;
      if (found == 0x7FFFFFFF && run > sh_target) found = e0 + i;
    }
  }
  // smallest found index, else the last kept index of the chunk
  int f = found;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) f = min(f, __shfl_xor(f, o, 64));
  int l = last;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) l = max(l, __shfl_xor(l, o, 64));
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red_i[threadIdx.x >> 6] = f;
  __syncthreads();
  int fb = red_i[0];
  for (int i = 1; i < NW; ++i) fb = min(fb, red_i[i]);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red_i[threadIdx.x >> 6] = l;
  __syncthreads();
  int lb = red_i[0];
  for (int i = 1; i < NW; ++i) lb = max(lb, red_i[i]);
  return fb != 0x7FFFFFFF ? fb : lb;
}

// Kept sums of chunk c of row r from each thread's four float4 partials
// (part[k]: logits (threadIdx.x + 256 k) * 4 .. +3 of the chunk).  With
// sub_sums, the 16 sub-chunks of 256 logits: wave w's partials at step k cover
// sub-chunk 4k + w exactly, so each is one wave reduction (no barrier);
// otherwise the chunk's sum.
RGD_DEV void store_kept_sums(const SampleArgs& a, int r, int c, const float (&part)[4], float* red) {
  if (a.sub_sums) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    float* dst = a.sub_sums + ((long long)r * a.nchunks + c) * 16 + w;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float t = wave_sum(part[k]);
      if (lane == 0) dst[4 * k] = t;
    }
  } else {
    float sum = 0.f;
#pragma unroll
    for (int k = 0; k < 4; ++k) sum += part[k];
    sum = block_sum(sum, red);
    if (threadIdx.x == 0) a.chunk_sums[(long long)r * a.nchunks + c] = sum;
  }
}

__global__ __launch_bounds__(256) void minp_sum_kernel(SampleArgs a) {
  __shared__ float red[4];
  const int c = blockIdx.x, r = blockIdx.y;
  const float* zr = a.z + r * a.ldz;
  const int lo = c * a.chunk, hi = min(a.V, lo + a.chunk);
  // the chunk's logits (chunk <= 4096: at most 4 float4 per thread) are
  // requested before the row maximum is formed, so the two latencies overlap
  float4 v[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int i = lo + (threadIdx.x + k * 256) * 4;  // V and chunk are multiples of 4
    v[k] = i < hi ? *(const float4*)(zr + i) : float4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
  }
  const float mx = row_max_from_partials(a.pmax, a.npmax, r, red);
  const float kT = kLog2e / a.T;
  float part[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const float w0 = kept_weight(v[k].x, mx, kT, a.p_min), w1 = kept_weight(v[k].y, mx, kT, a.p_min);
    const float w2 = kept_weight(v[k].z, mx, kT, a.p_min), w3 = kept_weight(v[k].w, mx, kT, a.p_min);
    part[k] = (w0 > 0.f ? w0 : 0.f) + (w1 > 0.f ? w1 : 0.f) + (w2 > 0.f ? w2 : 0.f) + (w3 > 0.f ? w3 : 0.f);
  }
  store_kept_sums(a, r, c, part, red);
  if (threadIdx.x == 0 && c == 0 && a.status && !(mx > -INFINITY && mx < INFINITY)) atomicOr(a.status, 1);
}

// Standalone rows (no partial maxima from a producer): one read of the
// logits.  Pass 1 writes each chunk's maximum m_c and its kept sum relative
// to m_c.  With m the row maximum, a chunk whose m_c == m has the exact sum,
// a chunk whose best weight exp2((m_c - m) kT) is below p_min keeps nothing,
// and only the chunks in between are read again (by the second kernel, which
// then makes the draw) to sum the weights relative to m.
__global__ __launch_bounds__(256) void minp_cand_kernel(SampleArgs a, float* cmax) {
  __shared__ float red[4];
  const int c = blockIdx.x, r = blockIdx.y;
  const float* zr = a.z + r * a.ldz;
  const int lo = c * a.chunk, hi = min(a.V, lo + a.chunk);
  float4 v[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int i = lo + (threadIdx.x + k * 256) * 4;
    v[k] = i < hi ? *(const float4*)(zr + i) : float4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
  }
  float mc = -INFINITY;
#pragma unroll
  for (int k = 0; k < 4; ++k) mc = fmaxf(mc, fmaxf(fmaxf(v[k].x, v[k].y), fmaxf(v[k].z, v[k].w)));
  mc = block_max(mc, red);
  const float kT = kLog2e / a.T;
  float sum = 0.f;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const float w0 = kept_weight(v[k].x, mc, kT, a.p_min), w1 = kept_weight(v[k].y, mc, kT, a.p_min);
    const float w2 = kept_weight(v[k].z, mc, kT, a.p_min), w3 = kept_weight(v[k].w, mc, kT, a.p_min);
    sum += (w0 > 0.f ? w0 : 0.f) + (w1 > 0.f ? w1 : 0.f) + (w2 > 0.f ? w2 : 0.f) + (w3 > 0.f ? w3 : 0.f);
  }
  sum = block_sum(sum, red);
  if (threadIdx.x == 0) {
    cmax[(long long)r * a.nchunks + c] = mc;
    a.chunk_sums[(long long)r * a.nchunks + c] = sum;
  }
}

// Standalone rows, second kernel (one workgroup of 1024 threads per row): the
// row maximum from the chunk maxima, the kept sums of the chunks pass 1 could
// not settle, then the draw.  Each wave recomputes whole chunks (16 KB, 16
// float4 per lane) so that up to 16 of them are in flight at once.  The
// settled sums are written back for further draws from the same row.
__global__ __launch_bounds__(1024) void minp_fixsel_kernel(SampleArgs a) {
  __shared__ float red[16];
  __shared__ float fixed[256];
  __shared__ int wlist[256];
  __shared__ int nwin;
  const int r = blockIdx.x, c = threadIdx.x;
  const long long r0 = (long long)r * a.nchunks;
  const bool own = c < a.nchunks;
  const float mc = own ? a.pmax[r0 + c] : -INFINITY;
  float mine = own ? a.chunk_sums[r0 + c] : 0.f;
  if (c == 0) nwin = 0;
  const float mx = block_max(mc, red);  // its barriers also publish nwin = 0
  const float kT = kLog2e / a.T;
  const bool exact = mc == mx;
  const bool empty = !exact && kept_weight(mc, mx, kT, a.p_min) < 0.f;
  if (own && !exact && !empty) wlist[atomicAdd(&nwin, 1)] = c;
  __syncthreads();
  const int nw = nwin, wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const float* zr = a.z + r * a.ldz;
  for (int i = wave; i < nw; i += 16) {
    const int ch = wlist[i];
    const int lo = ch * a.chunk, hi = min(a.V, lo + a.chunk);
    float4 v[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const int e = lo + (lane + k * 64) * 4;
      v[k] = e < hi ? *(const float4*)(zr + e) : float4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
    }
    float sum = 0.f;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const float w0 = kept_weight(v[k].x, mx, kT, a.p_min), w1 = kept_weight(v[k].y, mx, kT, a.p_min);
      const float w2 = kept_weight(v[k].z, mx, kT, a.p_min), w3 = kept_weight(v[k].w, mx, kT, a.p_min);
      sum += (w0 > 0.f ? w0 : 0.f) + (w1 > 0.f ? w1 : 0.f) + (w2 > 0.f ? w2 : 0.f) + (w3 > 0.f ? w3 : 0.f);
    }
    sum = wave_sum(sum);
    if (lane == 0) fixed[ch] = sum;
  }
  __syncthreads();
  if (own && !exact) {
    mine = empty ? 0.f : fixed[c];
    a.chunk_sums[r0 + c] = mine;
  }
  const float u = philox_uniform(a.seeds[r], a.ctr, a.stream);
  const int tok = select_token<1024>(a, r, mx, u, mine);
  if (threadIdx.x == 0) {
    a.out[r * a.out_stride + a.out_col] = tok;
    if (a.cur_tok) a.cur_tok[r] = tok;
  }
}

// Standalone rows in one launch: one workgroup of 1024 threads per row.  Each
// wave streams whole 4096-logit chunks (16 float4 per lane, one coalesced
// 1 KiB request per load instruction) and keeps the chunk's maximum m_c and
// its kept sum relative to m_c in LDS.  After a barrier the row maximum is
// known; the chunks whose maximum lies inside the min-p window below it are
// summed again relative to it (rereads), and the draw follows.  The chunk
// maxima and settled sums are also written out for further draws.
__global__ __launch_bounds__(1024) void minp_row_kernel(SampleArgs a, float* cmax) {
  __shared__ float cm[256], cs[256];
  __shared__ float red[16];
  __shared__ int wlist[256];
  __shared__ int nwin;
  const int r = blockIdx.x, wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const float* zr = a.z + r * a.ldz;
  const float kT = kLog2e / a.T;
  for (int c = wave; c < a.nchunks; c += 16) {
    const int lo = c * a.chunk, hi = min(a.V, lo + a.chunk);
    float4 v[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const int e = lo + (lane + k * 64) * 4;
      v[k] = e < hi ? *(const float4*)(zr + e) : float4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
    }
    float mc = -INFINITY;
#pragma unroll
    for (int k = 0; k < 16; ++k) mc = fmaxf(mc, fmaxf(fmaxf(v[k].x, v[k].y), fmaxf(v[k].z, v[k].w)));
    mc = wave_max(mc);
    float sum = 0.f;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const float w0 = kept_weight(v[k].x, mc, kT, a.p_min), w1 = kept_weight(v[k].y, mc, kT, a.p_min);
      const float w2 = kept_weight(v[k].z, mc, kT, a.p_min), w3 = kept_weight(v[k].w, mc, kT, a.p_min);
      sum += (w0 > 0.f ? w0 : 0.f) + (w1 > 0.f ? w1 : 0.f) + (w2 > 0.f ? w2 : 0.f) + (w3 > 0.f ? w3 : 0.f);
    }
    sum = wave_sum(sum);
    if (lane == 0) {
      cm[c] = mc;
      cs[c] = sum;
    }
  }
  if (threadIdx.x == 0) nwin = 0;
  __syncthreads();
  const int c = threadIdx.x;
  const bool own = c < a.nchunks;
  const float mc = own ? cm[c] : -INFINITY;
  float mine = own ? cs[c] : 0.f;
  const float mx = block_max(mc, red);
  const bool exact = mc == mx;
  const bool empty = !exact && kept_weight(mc, mx, kT, a.p_min) < 0.f;
  if (own && !exact && !empty) wlist[atomicAdd(&nwin, 1)] = c;
  __syncthreads();
  const int nw = nwin;
  for (int i = wave; i < nw; i += 16) {
    const int ch = wlist[i];
    const int lo = ch * a.chunk, hi = min(a.V, lo + a.chunk);
    float4 v[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const int e = lo + (lane + k * 64) * 4;
      v[k] = e < hi ? *(const float4*)(zr + e) : float4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
    }
    float sum = 0.f;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const float w0 = kept_weight(v[k].x, mx, kT, a.p_min), w1 = kept_weight(v[k].y, mx, kT, a.p_min);
      const float w2 = kept_weight(v[k].z, mx, kT, a.p_min), w3 = kept_weight(v[k].w, mx, kT, a.p_min);
      sum += (w0 > 0.f ? w0 : 0.f) + (w1 > 0.f ? w1 : 0.f) + (w2 > 0.f ? w2 : 0.f) + (w3 > 0.f ? w3 : 0.f);
    }
    sum = wave_sum(sum);
    if (lane == 0) cs[ch] = sum;
  }
  __syncthreads();
  if (own) {
    if (!exact) mine = empty ? 0.f : cs[c];
    const long long rc = (long long)r * a.nchunks + c;
    cmax[rc] = mc;
    a.chunk_sums[rc] = mine;
  }
  const float u = philox_uniform(a.seeds[r], a.ctr, a.stream);
  const int tok = select_token<1024>(a, r, mx, u, mine);
  if (threadIdx.x == 0) {
    a.out[r * a.out_stride + a.out_col] = tok;
    if (a.cur_tok) a.cur_tok[r] = tok;
  }
}

// ------------------------------------------------------------------ p-less --
// p-less truncation (temperature first): with w_i = exp2((z_i - m) log2(e)/T),
// S1 = sum w_i and S2 = sum w_i^2, softmax(z/T) gives p_i = w_i / S1 and
// sum_j p_j^2 = S2 / S1^2, so p_i >= sum_j p_j^2 iff w_i >= S2 / S1.  The
// threshold depends on the whole row, so the chunk sums need one more pass
// than min-p: (1) per chunk, its maximum m_c and S1, S2 relative to m_c;
// (2) per chunk, the row's m, S1, S2 combined from all chunk statistics in one
// fixed order (so every workgroup of the row and the draw see the same
// threshold), then the chunk's kept sum relative to m (chunks whose best
// weight is under the threshold are not read); (3) the min-p draw kernel with
// the per-row threshold.

__global__ __launch_bounds__(256) void pless_stats_kernel(SampleArgs a, float* cmax, float* s1, float* s2) {
  __shared__ float red[4];
  const int c = blockIdx.x, r = blockIdx.y;
  const float* zr = a.z + r * a.ldz;
  const int lo = c * a.chunk, hi = min(a.V, lo + a.chunk);
  float4 v[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int i = lo + (threadIdx.x + k * 256) * 4;
    v[k] = i < hi ? *(const float4*)(zr + i) : float4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
  }
  float mc = -INFINITY;
#pragma unroll
  for (int k = 0; k < 4; ++k) mc = fmaxf(mc, fmaxf(fmaxf(v[k].x, v[k].y), fmaxf(v[k].z, v[k].w)));
  mc = block_max(mc, red);
  const float kT = kLog2e / a.T;
  float t1 = 0.f, t2 = 0.f;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const float w0 = __builtin_amdgcn_exp2f((v[k].x - mc) * kT), w1 = __builtin_amdgcn_exp2f((v[k].y - mc) * kT);
    const float w2 = __builtin_amdgcn_exp2f((v[k].z - mc) * kT), w3 = __builtin_amdgcn_exp2f((v[k].w - mc) * kT);
    t1 += (w0 + w1) + (w2 + w3);
    t2 += (w0 * w0 + w1 * w1) + (w2 * w2 + w3 * w3);
  }
  t1 = block_sum(t1, red);
  t2 = block_sum(t2, red);
  if (threadIdx.x == 0) {
    const long long rc = (long long)r * a.nchunks + c;
    cmax[rc] = mc;
    s1[rc] = t1;
    s2[rc] = t2;
  }
}

__global__ __launch_bounds__(256) void pless_sum_kernel(SampleArgs a, const float* cmax, const float* s1,
                                                        const float* s2, float* thr_out) {
  __shared__ float red[4];
  const int c = blockIdx.x, r = blockIdx.y, t = threadIdx.x;
  const long long r0 = (long long)r * a.nchunks;
  // every chunk's statistics, one chunk per thread (nchunks <= 256)
  const bool own = t < a.nchunks;
  const float mt = own ? cmax[r0 + t] : -INFINITY;
  const float a1 = own ? s1[r0 + t] : 0.f, a2 = own ? s2[r0 + t] : 0.f;
  const float m = block_max(mt, red);
  const float kT = kLog2e / a.T;
  const float e = own ? __builtin_amdgcn_exp2f((mt - m) * kT) : 0.f;
  const float S1 = block_sum(a1 * e, red);
  const float S2 = block_sum(a2 * e * e, red);
  const float thr = S2 / S1;
  if (c == 0 && t == 0) {
    thr_out[r] = thr;
    if (a.status && !(m > -INFINITY && m < INFINITY)) atomicOr(a.status, 1);
  }
  float part[4] = {0.f, 0.f, 0.f, 0.f};
  if (kept_weight(cmax[r0 + c], m, kT, thr) >= 0.f) {  // uniform: one value per workgroup
    const float* zr = a.z + r * a.ldz;
    const int lo = c * a.chunk, hi = min(a.V, lo + a.chunk);
    float4 v[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int i = lo + (t + k * 256) * 4;
      v[k] = i < hi ? *(const float4*)(zr + i) : float4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float w0 = kept_weight(v[k].x, m, kT, thr), w1 = kept_weight(v[k].y, m, kT, thr);
      const float w2 = kept_weight(v[k].z, m, kT, thr), w3 = kept_weight(v[k].w, m, kT, thr);
      part[k] = (w0 > 0.f ? w0 : 0.f) + (w1 > 0.f ? w1 : 0.f) + (w2 > 0.f ? w2 : 0.f) + (w3 > 0.f ? w3 : 0.f);
    }
  }
  store_kept_sums(a, r, c, part, red);
}

// The draw from sub-chunk kept sums (decode path): wave 0 makes the draw in
// two dependent reads and no barrier.  Each lane takes SP = nsub / 64
// consecutive sub-chunk sums (a lane-local running sum, then a wave scan of
// the lane totals gives every sub-chunk's running sum in id order); the first
// sub-chunk whose running sum exceeds u * W is rescanned, four logits per
// lane, with a second wave scan.  The token (the smallest kept id whose
// running sum exceeds u * W; else the sub-chunk's last kept id) then goes
// through LDS to all four waves for the next step's embedding row and
// RMSNorm.
__global__ __launch_bounds__(256) void minp_select_sub_kernel(SampleArgs a) {
  constexpr int kMaxSP = 16;
  __shared__ int sh_tok;
  const int r = blockIdx.x;
  const int lane = threadIdx.x & 63;
  if (threadIdx.x < 64) {
    const int nsub = a.nchunks * 16;
    const int SP = (nsub + 63) / 64;
    const float* ss = a.sub_sums + (long long)r * nsub;
    // Every load is issued unconditionally from a clamped index and its
    // value is used on every path: a load whose value is only used under a
    // condition is sunk into a branch by the compiler, which then waits for
    // it where the branches join, one memory round trip per load.
    float loc[kMaxSP];
#pragma unroll
    for (int i = 0; i < kMaxSP; ++i) {
      const int j = lane * SP + i;
      // sub-chunk sums are finite and non-negative, so a 0/1 factor masks them
      loc[i] = ss[min(j, nsub - 1)] * ((i < SP && j < nsub) ? 1.f : 0.f);
    }
    const float* pm = a.pmax + (long long)r * a.npmax;
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < 16; ++i)  // npmax <= 1024 (checked by the launcher)
      mx = fmaxf(mx, pm[min(lane + 64 * i, a.npmax - 1)]);  // a repeated entry leaves the maximum unchanged
    const float u = philox_uniform(a.seeds[r], a.ctr, a.stream);
    const float thr = a.row_thr ? a.row_thr[r] : a.p_min;
    mx = wave_max(mx);
#pragma unroll
    for (int i = 1; i < kMaxSP; ++i) loc[i] += loc[i - 1];
    const float tl = loc[kMaxSP - 1];
    float incl = tl;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const float t = __shfl_up(incl, o, 64);
      if (lane >= o) incl += t;
    }
    float excl = __shfl_up(incl, 1, 64);
    if (lane == 0) excl = 0.f;
    const float W = __shfl(incl, 63, 64);
    const float target = u * W;
    // first sub-chunk whose running sum passes the target; the last non-empty one
    int jf = 0x7FFFFFFF, jl = -1;
    float prev = excl;
#pragma unroll
    for (int i = 0; i < kMaxSP; ++i) {
      const int j = lane * SP + i;
      if (i < SP && j < nsub) {
        const float run = excl + loc[i];
        if (run > prev) jl = j;
        if (jf == 0x7FFFFFFF && run > target) jf = j;
        prev = run;
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      jf = min(jf, __shfl_xor(jf, o, 64));
      jl = max(jl, __shfl_xor(jl, o, 64));
    }
    const int js = jf != 0x7FFFFFFF ? jf : max(jl, 0);
    // running sum before sub-chunk js, from the lane that holds it
    const int ow = js / SP, oi = js - ow * SP;
    float b = excl;
#pragma unroll
    for (int i = 1; i < kMaxSP; ++i)
      if (i == oi) b = excl + loc[i - 1];
    const float base = __shfl(b, ow, 64);
    // rescan: lane l holds logits js * 256 + 4 l .. +3 (V is a multiple of 4)
    const int e0 = js * 256 + lane * 4;
    const float* zr = a.z + r * a.ldz;
    const float4 zv = e0 < a.V ? *(const float4*)(zr + e0) : float4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
    const float kT = kLog2e / a.T;
    float wv[4] = {kept_weight(zv.x, mx, kT, thr), kept_weight(zv.y, mx, kT, thr), kept_weight(zv.z, mx, kT, thr),
                   kept_weight(zv.w, mx, kT, thr)};
    if (e0 >= a.V) wv[0] = wv[1] = wv[2] = wv[3] = -1.f;
    const float ts = (wv[0] > 0.f ? wv[0] : 0.f) + (wv[1] > 0.f ? wv[1] : 0.f) + (wv[2] > 0.f ? wv[2] : 0.f) +
                     (wv[3] > 0.f ? wv[3] : 0.f);
    float inc2 = ts;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const float t = __shfl_up(inc2, o, 64);
      if (lane >= o) inc2 += t;
    }
    float run = base + (inc2 - ts);
    int found = 0x7FFFFFFF, last = -1;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (wv[i] >= 0.f) {
        run += wv[i];
        last = e0 + i;
        if (found == 0x7FFFFFFF && run > target) found = e0 + i;
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      found = min(found, __shfl_xor(found, o, 64));
      last = max(last, __shfl_xor(last, o, 64));
    }
    const int tok = found != 0x7FFFFFFF ? found : (last >= 0 ? last : js * 256);
    if (lane == 0) {
      sh_tok = tok;
      a.out[r * a.out_stride + a.out_col] = tok;
      if (a.cur_tok) a.cur_tok[r] = tok;
    }
  }
  if (!a.embed) return;
  __syncthreads();
  const int tok = sh_tok;
  float* x = a.x + (long long)r * a.d;
  if (a.embed_bf16)
    embed_norm_row(tok, (const bf16_t*)a.embed, a.d, a.vocab, a.gain, a.eps, x, (bf16_t*)a.xn + (long long)r * a.d);
  else
    embed_norm_row(tok, (const float*)a.embed, a.d, a.vocab, a.gain, a.eps, x, (float*)a.xn + (long long)r * a.d);
}

__global__ __launch_bounds__(256) void minp_select_kernel(SampleArgs a) {
  __shared__ float red[4];
  const int r = blockIdx.x;
  // chunk sums and partial maxima are requested together
  const float mine = (int)threadIdx.x < a.nchunks ? a.chunk_sums[(long long)r * a.nchunks + threadIdx.x] : 0.f;
  const float mx = row_max_from_partials(a.pmax, a.npmax, r, red);
  const float u = philox_uniform(a.seeds[r], a.ctr, a.stream);
  const int tok = select_token<256>(a, r, mx, u, mine);
  if (threadIdx.x == 0) {
    a.out[r * a.out_stride + a.out_col] = tok;
    if (a.cur_tok) a.cur_tok[r] = tok;
  }
  // the next step's first kernel (embedding gather + RMSNorm) for this row
  if (a.embed) {
    float* x = a.x + (long long)r * a.d;
    if (a.embed_bf16)
      embed_norm_row(tok, (const bf16_t*)a.embed, a.d, a.vocab, a.gain, a.eps, x, (bf16_t*)a.xn + (long long)r * a.d);
    else
      embed_norm_row(tok, (const float*)a.embed, a.d, a.vocab, a.gain, a.eps, x, (float*)a.xn + (long long)r * a.d);
  }
}

__global__ __launch_bounds__(256) void minp_multi_kernel(SampleArgs a, unsigned stream0, int draws,
                                                         int* out) {
  __shared__ float red[4];
  const int d = blockIdx.x, r = blockIdx.y;
  const float mine = (int)threadIdx.x < a.nchunks ? a.chunk_sums[(long long)r * a.nchunks + threadIdx.x] : 0.f;
  const float mx = row_max_from_partials(a.pmax, a.npmax, r, red);
  const float u = philox_uniform(a.seeds[r], a.ctr, stream0 + unsigned(d));
  const int tok = select_token<256>(a, r, mx, u, mine);
  if (threadIdx.x == 0) out[(long long)r * draws + d] = tok;
}

// ------------------------------------------------------------------ gate ----
// One probe step of row r (prompt b): the greedy token (the argmax key of the
// row, from the argmax pass or the LM head's tile keys), the compatibility of
// the probe extended by it against every table entry, the event.  Wave 0 does
// the update; with a.embed all four waves then write the next step's input
// row (embedding of the token the next step feeds, RMSNorm).
// Returns the token appended (every lane of the wave), or -1 when the row's
// prompt was already decided.
RGD_DEV int probe_update_row(const GateArgs& a, int r) {
  const int b = a.row_prompt[r];
  unsigned long long key;
  if (a.tilekeys) {
    key = 0ull;
    const unsigned long long* tk = a.tilekeys + (long long)r * a.ntiles;
    // four unconditional loads per lane and round (clamped indices, masked)
    for (int i0 = 0; i0 < a.ntiles; i0 += 256) {
      unsigned long long v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = tk[min(i0 + (int)threadIdx.x + 64 * u, a.ntiles - 1)];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (i0 + (int)threadIdx.x + 64 * u < a.ntiles) key = v[u] > key ? v[u] : key;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const unsigned long long ko = __shfl_xor(key, o, 64);
      key = ko > key ? ko : key;
    }
  } else {
    key = a.best[r];
    if (threadIdx.x == 0) a.best_reset[r] = 0ull;
  }
  if (a.event[b] != -1) return -1;
  const int tok = int(0xFFFFFFFFu - uint32_t(key & 0xFFFFFFFFull));
  const int j = a.probe_len[b];
  const int* q = a.probe_tokens + (long long)b * a.k;
  bool any = false;
  for (int e = threadIdx.x; e < a.n_entries; e += 64) any = any || entry_matches(a, e, b, q, j, tok);
  const bool compat = a.all_compatible || __any(any);
  if (threadIdx.x == 0) {
    a.probe_tokens[(long long)b * a.k + j] = tok;
    a.probe_len[b] = j + 1;
    if (a.cur_tok) a.cur_tok[r] = tok;
    const bool stop = a.eos >= 0 && tok == a.eos, full = j + 1 >= a.k;
    if (a.no_early_exit) {
      // the detector judges the finished probe: incompatibility is sticky
      // (prefix closure), so one failed token decides it
      const bool failed = a.failed[b] || !compat;
      a.failed[b] = failed;
      a.event[b] = !(stop || full) ? -1 : failed ? 0 : stop ? 1 : 2;
    } else {
      a.event[b] = !compat ? 0 : stop ? 1 : full ? 2 : -1;
    }
  }
  return tok;
}

__global__ __launch_bounds__(256) void probe_update_kernel(GateArgs a) {
  __shared__ int sh_tok, sh_held;
  const int r = blockIdx.x;
  if (threadIdx.x < 64) {
    const int t = probe_update_row(a, r);
    if (threadIdx.x == 0) sh_tok = t;
  } else if (threadIdx.x == 64) {
    // meanwhile, the token the row's probe holds at feed_col (what a prompt
    // decided earlier feeds; both loads are in range whatever feed_col)
    const int b = a.row_prompt[r];
    sh_held = a.probe_tokens[(long long)b * a.k + min(max(a.feed_col, 0), a.k - 1)];
  }
  if (!a.embed) return;
  __syncthreads();
  // the token the next step feeds: the one just appended (column feed_col),
  // or for a prompt decided earlier what its probe holds there
  const int tok = sh_tok >= 0 ? sh_tok : sh_held;
  float* x = a.x + (long long)r * a.d;
  if (a.embed_bf16)
    embed_norm_row(tok, (const bf16_t*)a.embed, a.d, a.vocab, a.gain, a.eps, x, (bf16_t*)a.xn + (long long)r * a.d);
  else
    embed_norm_row(tok, (const float*)a.embed, a.d, a.vocab, a.gain, a.eps, x, (float*)a.xn + (long long)r * a.d);
}

__global__ void gate_decide_kernel(const int* event, int B, int* decision, int* n_miss, int* miss_idx) {
  if (threadIdx.x != 0) return;
  int n = 0;
  for (int b = 0; b < B; ++b) {
    const int hit = (event[b] == 1 || event[b] == 2) ? 1 : 0;
    decision[b] = hit;
    if (!hit) miss_idx[n++] = b;
  }
  *n_miss = n;
}

}  // namespace

hipError_t fill_u32(uint32_t* p, uint32_t v, long long n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int blocks = int(min(1024ll, (n + 255) / 256));
  hipLaunchKernelGGL(fill_u32_kernel, dim3(blocks), dim3(256), 0, s, p, v, n);
  return hipGetLastError();
}

hipError_t chunk_max(const float* z, long long ldz, int R, int V, int chunk, float* cmax, hipStream_t s) {
  if (chunk % 1024 || V % 4 || ldz % 4) return hipErrorInvalidValue;
  hipLaunchKernelGGL(chunk_max_kernel, dim3((V + chunk - 1) / chunk, R), dim3(256), 0, s, z, ldz, V, chunk,
                     cmax);
  return hipGetLastError();
}

hipError_t argmax_rows(const float* z, long long ldz, int R, int V, unsigned long long* best,
                       hipStream_t s) {
  const int chunk = 4096;
  const dim3 grid((V + chunk - 1) / chunk, R);
  if (V % 4 == 0 && ldz % 4 == 0 && (uintptr_t)z % 16 == 0)
    hipLaunchKernelGGL(argmax_kernel<true>, grid, dim3(256), 0, s, z, ldz, V, chunk, best);
  else
    hipLaunchKernelGGL(argmax_kernel<false>, grid, dim3(256), 0, s, z, ldz, V, chunk, best);
  return hipGetLastError();
}

hipError_t minp_sample(const SampleArgs& a, hipStream_t s) {
  if (a.chunk % 1024 || a.chunk > 4096 || a.V % 4 || a.nchunks > 256 ||
      a.nchunks * a.chunk < a.V || !(a.T > 0.f))
    return hipErrorInvalidValue;
  if (a.sub_sums && (a.nchunks * 16 > 1024 || a.npmax > 1024)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(minp_sum_kernel, dim3(a.nchunks, a.R), dim3(256), 0, s, a);
  if (a.sub_sums)
    hipLaunchKernelGGL(minp_select_sub_kernel, dim3(a.R), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(minp_select_kernel, dim3(a.R), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t minp_sample_standalone(const SampleArgs& a0, float* cmax, hipStream_t s) {
  if (a0.chunk != 4096 || a0.V % 4 || a0.ldz % 4 || a0.nchunks > 256 || a0.nchunks * a0.chunk < a0.V ||
      !(a0.T > 0.f))
    return hipErrorInvalidValue;
  SampleArgs a = a0;
  a.pmax = cmax;
  a.npmax = a.nchunks;
  if (a.R >= kRowKernelMinRows) {
    hipLaunchKernelGGL(minp_row_kernel, dim3(a.R), dim3(1024), 0, s, a, cmax);
  } else {
    hipLaunchKernelGGL(minp_cand_kernel, dim3(a.nchunks, a.R), dim3(256), 0, s, a, cmax);
    hipLaunchKernelGGL(minp_fixsel_kernel, dim3(a.R), dim3(1024), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t pless_sample(const SampleArgs& a0, float* stats, float* thr, hipStream_t s) {
  if (a0.chunk != 4096 || a0.V % 4 || a0.ldz % 4 || a0.nchunks > 256 || a0.nchunks * a0.chunk < a0.V ||
      !(a0.T > 0.f))
    return hipErrorInvalidValue;
  SampleArgs a = a0;
  const long long n = (long long)a.R * a.nchunks;
  float* cmax = stats;
  a.pmax = cmax;
  a.npmax = a.nchunks;
  a.row_thr = thr;
  hipLaunchKernelGGL(pless_stats_kernel, dim3(a.nchunks, a.R), dim3(256), 0, s, a, cmax, stats + n, stats + 2 * n);
  if (a.sub_sums && (a.nchunks * 16 > 1024 || a.nchunks > 1024)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(pless_sum_kernel, dim3(a.nchunks, a.R), dim3(256), 0, s, a, cmax, stats + n, stats + 2 * n, thr);
  if (a.sub_sums)
    hipLaunchKernelGGL(minp_select_sub_kernel, dim3(a.R), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(minp_select_kernel, dim3(a.R), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t minp_multi_draw(const SampleArgs& a, int draws, unsigned int stream0, int* out, hipStream_t s) {
  if (draws <= 0) return hipSuccess;
  hipLaunchKernelGGL(minp_multi_kernel, dim3(draws, a.R), dim3(256), 0, s, a, stream0, draws, out);
  return hipGetLastError();
}

hipError_t probe_update(const GateArgs& a, hipStream_t s) {
  if (a.R <= 0) return hipSuccess;
  if (a.embed && (a.d % 4 || a.d > 4096)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(probe_update_kernel, dim3(a.R), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t gate_decide(const int* event, int B, int* decision, int* n_miss, int* miss_idx, hipStream_t s) {
  hipLaunchKernelGGL(gate_decide_kernel, dim3(1), dim3(64), 0, s, event, B, decision, n_miss, miss_idx);
  return hipGetLastError();
}

}  // namespace rgd
