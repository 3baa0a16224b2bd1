// Decode attention over a shared prompt KV plus per-row tails.
//
// The prompt KV of one prompt is read by every row (probe or branch) of that
// prompt.  The shared part is split over (prefix split, KV head, row block):
// a workgroup loads each 32-position K/V tile of its split once into LDS and
// all query vectors of the row block (rows x the G query heads of the KV head,
// up to 64) consume it with MFMA.  Scores are computed transposed,
// S^T = K Q^T, so that each lane ends up holding eight probabilities of one
// query vector; those feed O^T += V^T P^T directly as the B operand.  The V
// cache is kept head-dim-major (transposed per KV head), so the V^T tile is a
// plain copy into LDS.  The next tile is fetched into registers while the
// current one is consumed.  Online softmax runs in the exp2 domain with the
// row statistics reduced by lane shuffles across the four lane groups.
//
// Each row's own tail (paged) is handled by a vector kernel, and a combine
// kernel merges the (o, log-sum-exp) partials in a fixed order.
#include "kernels.hpp"

namespace rgd {

namespace {

constexpr float kLn2 = 0.6931471805599453f;
constexpr float kLog2e = 1.4426950408889634f;

RGD_DEV f32x4 mfma16x16x32(const u32x4& a, const u32x4& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

RGD_DEV uint32_t pack2(float lo, float hi) { return pack_bf16x2(lo, hi); }

// NWAVE waves; PAGED selects the row's paged tail (one row per workgroup)
// instead of the shared prompt prefix (a block of rows of one prompt).
// Tiles hold TP = 64 positions; the next tile is fetched into registers while
// the current one is consumed from LDS.
template <int NWAVE, bool PAGED>
__global__ __launch_bounds__(NWAVE * 64) void attn_mfma_kernel(AttnArgs a) {
  constexpr int D = 128, NT = NWAVE * 64, TP = 64;
  constexpr int KSEG = TP * 16 / NT, VSEG = D * (TP / 8) / NT;  // 16-byte segments per thread
  const int s = blockIdx.x, g = blockIdx.y;
  int r0, nr, b, maxlen, lo, hi, part;
  if (PAGED) {
    r0 = blockIdx.z;
    nr = 1;
    b = 0;
    maxlen = a.tail_len;
    lo = s * a.tail_chunk;
    hi = min(lo + a.tail_chunk, maxlen);
    part = a.splits + s;
  } else {
    const int4 rb = a.rblocks[blockIdx.z];
    r0 = rb.x;
    nr = rb.y;
    b = rb.z;
    maxlen = rb.w;
    lo = s * a.split_len;
    hi = min(lo + a.split_len, maxlen);
    part = s;
  }
  const int G = a.Hq / a.Hkv;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l16 = lane & 15, grp = lane >> 4;
  const int nq = nr * G;
  const int v = wave * 16 + l16;
  const bool vok = v < nq;
  const bool wave_active = wave * 16 < nq;
  const int row = r0 + (vok ? v / G : 0);
  const int head = g * G + (vok ? v % G : 0);
  const int my_end = PAGED ? hi : (vok ? min(a.rows.plen[row], hi) : lo);

  u32x4 qf[4];
  {
    const bf16_t* qp = (const bf16_t*)a.q + ((long long)row * a.Hq + head) * D + grp * 8;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
      qf[ks] = vok ? *(const u32x4*)(qp + ks * 32) : u32x4{0u, 0u, 0u, 0u};
  }

  __shared__ __attribute__((aligned(16))) bf16_t ks_lds[TP][136];
  __shared__ __attribute__((aligned(16))) bf16_t vt_lds[D][TP + 8];

  const long long pstride = (long long)a.Hkv * D;
  const int ps = a.kv.page_size;
  const bf16_t* kbase;
  const bf16_t* vbase;
  if (PAGED) {
    kbase = (const bf16_t*)a.kv.pool_k + g * D;
    vbase = (const bf16_t*)a.kv.pool_v + (long long)g * D * ps;
  } else {
    kbase = (const bf16_t*)a.kv.prefix_k + (long long)b * a.kv.P * pstride + g * D;
    vbase = (const bf16_t*)a.kv.prefix_v + ((long long)b * a.Hkv + g) * D * a.kv.VP;
  }
  const int* pages = PAGED ? a.rows.pages + (long long)r0 * a.rows.max_pages : nullptr;
  const float scale = rsqrtf(float(D)) * kLog2e;

  float m = -INFINITY, lsum = 0.f;
  f32x4 o[8];
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};

  constexpr int NSET = 1;  // tile sets in registers (one tile in flight while one is consumed)
  u32x4 kreg[NSET][KSEG], vreg[NSET][VSEG];
  auto load_tile = [&](int t0, int set) {
#pragma unroll
    for (int i = 0; i < KSEG; ++i) {
      const int seg = threadIdx.x + i * NT;
      const int pos = t0 + (seg >> 4), pc = (seg & 15) * 8;
      u32x4 kk = {0u, 0u, 0u, 0u};
      if (pos < hi) {
        const long long ro = PAGED ? ((long long)pages[pos / ps] * ps + pos % ps) * pstride : (long long)pos * pstride;
        kk = *(const u32x4*)(kbase + ro + pc);
      }
      kreg[set][i] = kk;
    }
#pragma unroll
    for (int i = 0; i < VSEG; ++i) {
      const int seg = threadIdx.x + i * NT;
      const int d = seg >> 3, p0 = t0 + (seg & 7) * 8;
      const int nv = hi - p0;
      u32x4 vv = {0u, 0u, 0u, 0u};
      if (nv > 0) {
        const long long vo = PAGED ? ((long long)pages[p0 / ps] * a.Hkv * D + d) * ps + p0 % ps
                                   : (long long)d * a.kv.VP + p0;
        vv = *(const u32x4*)(vbase + vo);
        if (nv < 8) {  // positions past the range read as 0
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            if (2 * w >= nv) vv[w] = 0u;
            else if (2 * w + 1 >= nv) vv[w] &= 0xFFFFu;
          }
        }
      }
      vreg[set][i] = vv;
    }
  };

  auto consume = [&](int t0, int set) {
    __syncthreads();
#pragma unroll
    for (int i = 0; i < KSEG; ++i) {
      const int seg = threadIdx.x + i * NT;
      *(u32x4*)&ks_lds[seg >> 4][(seg & 15) * 8] = kreg[set][i];
    }
#pragma unroll
    for (int i = 0; i < VSEG; ++i) {
      const int seg = threadIdx.x + i * NT;
      *(u32x4*)&vt_lds[seg >> 3][(seg & 7) * 8] = vreg[set][i];
    }
    if (t0 + NSET * TP < hi) load_tile(t0 + NSET * TP, set);
    __syncthreads();
    if (!wave_active) return;
    // S^T = K Q^T: 4 position blocks of 16; lane holds positions 16*mt + 4*grp + i
    f32x4 sc[4];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      sc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const u32x4 ka = *(const u32x4*)&ks_lds[mt * 16 + l16][ks * 32 + grp * 8];
        sc[mt] = mfma16x16x32(ka, qf[ks], sc[mt]);
      }
    }
    float tmax = -INFINITY;
    const bool full = t0 + TP <= my_end;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float val = sc[mt][i] * scale;
        if (!full && t0 + mt * 16 + grp * 4 + i >= my_end) val = -INFINITY;
        sc[mt][i] = val;
        tmax = fmaxf(tmax, val);
      }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16, 64));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    const float mnew = fmaxf(m, tmax);
    // a query with nothing visible yet (only possible past a causal end) keeps
    // m = -inf: its probabilities are 0 and its state is left unscaled
    const bool none = mnew == -INFINITY;
    const float alpha = none ? 1.f : exp2f(m - mnew);
    const float msub = none ? 0.f : mnew;
    m = mnew;
    float ps_ = 0.f;
    u32x4 pb[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      float p[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        p[i] = exp2f(sc[2 * h][i] - msub);
        p[4 + i] = exp2f(sc[2 * h + 1][i] - msub);
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) ps_ += p[i];
      pb[h] = u32x4{pack2(p[0], p[1]), pack2(p[2], p[3]), pack2(p[4], p[5]), pack2(p[6], p[7])};
    }
    lsum = lsum * alpha + ps_;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      o[dt] *= alpha;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const bf16_t* vr = &vt_lds[dt * 16 + l16][h * 32 + grp * 4];
        const u32x2 a0 = *(const u32x2*)vr;
        const u32x2 a1 = *(const u32x2*)(vr + 16);
        o[dt] = mfma16x16x32(u32x4{a0.x, a0.y, a1.x, a1.y}, pb[h], o[dt]);
      }
    }
  };

#pragma unroll
  for (int k = 0; k < NSET; ++k)
    if (lo + k * TP < hi) load_tile(lo + k * TP, k);
  for (int t0 = lo; t0 < hi; t0 += NSET * TP) {
#pragma unroll
    for (int k = 0; k < NSET; ++k)
      if (t0 + k * TP < hi) consume(t0 + k * TP, k);
  }

  float lt = lsum + __shfl_xor(lsum, 16, 64);
  lt += __shfl_xor(lt, 32, 64);
  if (vok) {
    const long long idx = ((long long)part * a.rows.R + row) * a.Hq + head;
    float* po = a.part_o + idx * D;
    const float inv = lt > 0.f ? 1.0f / lt : 0.f;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) po[dt * 16 + grp * 4 + i] = o[dt][i] * inv;
    if (grp == 0) a.part_lse[idx] = lt > 0.f ? (m + __log2f(lt)) * kLn2 : -INFINITY;
  }
}

// Vector path: one workgroup per (chunk, KV head, row); one position per
// thread for the scores, one (head, dim) pair per thread for the weighted sum.
// PREFIX selects the shared prompt KV, otherwise the row's paged tail.
constexpr int kChunk = 256;

template <typename T, bool PREFIX>
__global__ __launch_bounds__(256) void attn_vec_kernel(AttnArgs a) {
  const int c = blockIdx.x, g = blockIdx.y, r = blockIdx.z;
  const int D = a.D, G = a.Hq / a.Hkv;
  __shared__ float qs[8][256];
  __shared__ float sc[8][kChunk];
  __shared__ float red[4];
  const int end = PREFIX ? a.rows.plen[r] : a.tail_len;
  const int clen = PREFIX ? a.split_len : a.tail_chunk;
  const int lo = c * clen;
  const int hi = min(lo + clen, end);
  const long long pstride = (long long)a.Hkv * D;
  for (int i = threadIdx.x; i < G * D; i += 256)
    qs[i / D][i % D] = load_f((const T*)a.q + ((long long)r * a.Hq + g * G) * D + i);
  __syncthreads();

  auto k_row = [&](int pos) -> const T* {
    if (PREFIX) return (const T*)a.kv.prefix_k + ((long long)a.rows.prompt[r] * a.kv.P + pos) * pstride + g * D;
    const int page = a.rows.pages[(long long)r * a.rows.max_pages + pos / a.kv.page_size];
    return (const T*)a.kv.pool_k + ((long long)page * a.kv.page_size + pos % a.kv.page_size) * pstride + g * D;
  };
  auto v_at = [&](int pos, int d) -> float {
    if (PREFIX)
      return load_f((const T*)a.kv.prefix_v + (((long long)a.rows.prompt[r] * a.Hkv + g) * D + d) * a.kv.VP + pos);
    const int ps = a.kv.page_size;
    const int page = a.rows.pages[(long long)r * a.rows.max_pages + pos / ps];
    return load_f((const T*)a.kv.pool_v + (((long long)page * a.Hkv + g) * D + d) * ps + pos % ps);
  };

  const float scale = rsqrtf(float(D));
  const int t = threadIdx.x;
  const int pos = lo + t;
  if (t < kChunk) {
    if (pos < hi) {
      const T* kr = k_row(pos);
      float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      for (int d = 0; d < D; ++d) {
        const float kd = load_f(kr + d);
        for (int h = 0; h < G; ++h) acc[h] += qs[h][d] * kd;
      }
      for (int h = 0; h < G; ++h) sc[h][t] = acc[h] * scale;
    } else {
      for (int h = 0; h < G; ++h) sc[h][t] = -INFINITY;
    }
  }
  __syncthreads();
  float mh[8], lh[8];
  for (int h = 0; h < G; ++h) {
    const float mx = block_max(sc[h][t], red);
    const float e = mx == -INFINITY ? 0.f : __expf(sc[h][t] - mx);
    __syncthreads();
    sc[h][t] = e;
    mh[h] = mx;
    lh[h] = block_sum(e, red);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < G * D; i += 256) {
    const int h = i / D, d = i % D;
    float acc = 0.f;
    for (int p = lo; p < hi; ++p) acc += sc[h][p - lo] * v_at(p, d);
    const long long idx = ((long long)c + (PREFIX ? 0 : a.splits)) * a.rows.R + r;
    const int head = g * G + h;
    a.part_o[(idx * a.Hq + head) * D + d] = lh[h] > 0.f ? acc / lh[h] : 0.f;
    if (d == 0) a.part_lse[idx * a.Hq + head] = lh[h] > 0.f ? mh[h] + __logf(lh[h]) : -INFINITY;
  }
}

// Tail attention fused with the merge of all partials: one workgroup per
// (row, KV head).  The row's own tail positions are attended on the vector
// units (each K row and each V value is loaded once and used by all G query
// heads of the KV head), then the prefix-split partials of those heads are
// merged with the tail in log-sum-exp form and the final output is written.
constexpr int kTailBlk = 256;
constexpr int kMaxSplits = 40;

// 8 consecutive elements starting at p (16-byte aligned for bf16, 32 for fp32)
RGD_DEV void load8(const bf16_t* p, float* out) {
  const u32x4 v = *(const u32x4*)p;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    out[2 * w] = __uint_as_float(v[w] << 16);
    out[2 * w + 1] = __uint_as_float(v[w] & 0xFFFF0000u);
  }
}
RGD_DEV void load8(const float* p, float* out) {
  const float4 a = *(const float4*)p, b = *(const float4*)(p + 4);
  out[0] = a.x; out[1] = a.y; out[2] = a.z; out[3] = a.w;
  out[4] = b.x; out[5] = b.y; out[6] = b.z; out[7] = b.w;
}

template <typename T>
__global__ __launch_bounds__(256) void attn_tail_combine_kernel(AttnArgs a, T* out) {
  const int r = blockIdx.x, g = blockIdx.y;
  const int D = a.D, G = a.Hq / a.Hkv;
  const long long R = a.rows.R;
  __shared__ __attribute__((aligned(16))) float qs[8][256];
  __shared__ float sc[8][kTailBlk];
  __shared__ float red[4];
  __shared__ float accx[2048];  // [part][head][dim], part * D == 256
  for (int i = threadIdx.x; i < G * D; i += 256)
    qs[i / D][i % D] = load_f((const T*)a.q + ((long long)r * a.Hq + g * G) * D + i) * rsqrtf(float(D));
  // the prefix-split partials do not depend on the tail: request them now so
  // their latency overlaps the tail attention (first 16 splits, 2 pairs/thread)
  constexpr int kPre = 16;
  const int S = a.splits;
  const long long pstep = R * a.Hq * D;
  float pre[2][kPre];
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int i = threadIdx.x + k * 256;
    const int h = i / D, dd = i % D;
    const float* po = a.part_o + ((long long)r * a.Hq + g * G + h) * D + dd;
#pragma unroll
    for (int sp = 0; sp < kPre; ++sp) pre[k][sp] = (i < G * D && sp < S) ? po[sp * pstep] : 0.f;
  }
  __syncthreads();

  // tail attention, online softmax over blocks of 256 positions
  const int ps = a.kv.page_size;
  const int* pages = a.rows.pages ? a.rows.pages + (long long)r * a.rows.max_pages : nullptr;
  const long long pstride = (long long)a.Hkv * D;
  // weighted sum layout: thread = (part, d); part handles 8-position blocks
  const int nparts = 256 / D;
  const int d = threadIdx.x % D, part = threadIdx.x / D;
  float mh[8], lh[8], acc[8];
#pragma unroll
  for (int h = 0; h < 8; ++h) {
    mh[h] = -INFINITY;
    lh[h] = 0.f;
    acc[h] = 0.f;
  }
  for (int c0 = 0; c0 < a.tail_len; c0 += kTailBlk) {
    const int n = min(kTailBlk, a.tail_len - c0);
    const int j = threadIdx.x;
    float dot[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (j < n) {
      const int pos = c0 + j;
      const T* kr = (const T*)a.kv.pool_k + ((long long)pages[pos / ps] * ps + pos % ps) * pstride + g * D;
      for (int e0 = 0; e0 < D; e0 += 8) {
        float kv[8];
        load8(kr + e0, kv);
#pragma unroll
        for (int h = 0; h < 8; ++h) {
          if (h < G) {
            const float4 q0 = *(const float4*)&qs[h][e0], q1 = *(const float4*)&qs[h][e0 + 4];
            dot[h] += q0.x * kv[0] + q0.y * kv[1] + q0.z * kv[2] + q0.w * kv[3] + q1.x * kv[4] + q1.y * kv[5] +
                      q1.z * kv[6] + q1.w * kv[7];
          }
        }
      }
    }
#pragma unroll
    for (int h = 0; h < 8; ++h)
      if (h < G) sc[h][j] = j < n ? dot[h] : -INFINITY;
    __syncthreads();
    float alpha[8];
#pragma unroll
    for (int h = 0; h < 8; ++h) {
      if (h >= G) break;
      const float cm = block_max(sc[h][j], red);
      const float mnew = fmaxf(mh[h], cm);
      const float e = sc[h][j] == -INFINITY ? 0.f : __expf(sc[h][j] - mnew);
      __syncthreads();
      sc[h][j] = e;
      const float bs = block_sum(e, red);
      alpha[h] = mh[h] == -INFINITY ? 0.f : __expf(mh[h] - mnew);
      lh[h] = lh[h] * alpha[h] + bs;
      mh[h] = mnew;
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < 8; ++h)
      if (h < G) acc[h] *= alpha[h];
    for (int b0 = part * 8; b0 < n; b0 += nparts * 8) {
      const int pos = c0 + b0;  // 8 positions inside one page (pages hold a multiple of 8)
      float v[8];
      load8((const T*)a.kv.pool_v + (((long long)pages[pos / ps] * a.Hkv + g) * D + d) * ps + pos % ps, v);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float ve = b0 + e < n ? v[e] : 0.f;
#pragma unroll
        for (int h = 0; h < 8; ++h)
          if (h < G) acc[h] += sc[h][b0 + e < n ? b0 + e : 0] * ve;
      }
    }
    __syncthreads();
  }
  // tail outputs per (head, dim): sum of the position parts in fixed order
  __shared__ float wts[8][kMaxSplits + 1];  // merge weights; column `splits` is the tail
  __syncthreads();
#pragma unroll
  for (int h = 0; h < 8; ++h)
    if (h < G) accx[(part * 8 + h) * D + d] = acc[h];
  // log-sum-exp of every prefix split of the G heads, loaded in parallel
  for (int i = threadIdx.x; i < G * S; i += 256) {
    const int h = i / S, sp = i % S;
    wts[h][sp] = a.part_lse[(sp * R + r) * a.Hq + g * G + h];
  }
  __syncthreads();
  if (threadIdx.x < G) {
    const int h = threadIdx.x;
    const float lt = lh[h] > 0.f ? mh[h] + __logf(lh[h]) : -INFINITY;
    float M = lt;
    for (int sp = 0; sp < S; ++sp) M = fmaxf(M, wts[h][sp]);
    float den = 0.f;
    for (int sp = 0; sp < S; ++sp) {
      const float w = wts[h][sp] == -INFINITY ? 0.f : __expf(wts[h][sp] - M);
      wts[h][sp] = w;
      den += w;
    }
    const float wt = lt == -INFINITY ? 0.f : __expf(lt - M);
    den += wt;
    const float inv = den > 0.f ? 1.0f / den : 0.f;
    for (int sp = 0; sp < S; ++sp) wts[h][sp] *= inv;
    wts[h][S] = lh[h] > 0.f ? wt * inv / lh[h] : 0.f;  // applied to the unnormalised tail sum
  }
  __syncthreads();
  for (int k = 0; k * 256 < G * D; ++k) {
    const int i = threadIdx.x + k * 256;
    if (i >= G * D) break;
    const int h = i / D, dd = i % D;
    const int head = g * G + h;
    float tail = 0.f;
    for (int pp = 0; pp < nparts; ++pp) tail += accx[(pp * 8 + h) * D + dd];
    float o = wts[h][S] * tail;
    if (k < 2) {
#pragma unroll
      for (int sp = 0; sp < kPre; ++sp)
        if (sp < S) o += wts[h][sp] * pre[k & 1][sp];
    }
    const float* po = a.part_o + ((long long)r * a.Hq + head) * D + dd;
#pragma unroll 4
    for (int sp = k < 2 ? kPre : 0; sp < S; ++sp) o += wts[h][sp] * po[sp * pstep];
    store_f(out + ((long long)r * a.Hq + head) * D + dd, o);
  }
}

template <typename T>
__global__ __launch_bounds__(128) void attn_combine_kernel(AttnArgs a, T* out) {
  const int r = blockIdx.x, h = blockIdx.y;
  const int D = a.D;
  const long long R = a.rows.R;
  float m = -INFINITY;
  for (int p = 0; p < a.nparts; ++p) m = fmaxf(m, a.part_lse[(p * R + r) * a.Hq + h]);
  for (int d = threadIdx.x; d < D; d += blockDim.x) {
    float num = 0.f, den = 0.f;
    for (int p = 0; p < a.nparts; ++p) {
      const float l = a.part_lse[(p * R + r) * a.Hq + h];
      if (l == -INFINITY) continue;
      const float w = __expf(l - m);
      num += w * a.part_o[((p * R + r) * a.Hq + h) * D + d];
      den += w;
    }
    store_f(out + ((long long)r * a.Hq + h) * D + d, den > 0.f ? num / den : 0.f);
  }
}

}  // namespace

hipError_t attn_prefix_mfma_bf16(const AttnArgs& a, hipStream_t s) {
  if (a.D != 128 || a.Hq / a.Hkv > 64 || a.split_len % 64 || a.kv.VP % 16) return hipErrorInvalidValue;
  if (a.splits <= 0 || a.nrblocks <= 0) return hipSuccess;
  hipLaunchKernelGGL((attn_mfma_kernel<4, false>), dim3(a.splits, a.Hkv, a.nrblocks), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t attn_tail_mfma_bf16(const AttnArgs& a, hipStream_t s) {
  if (a.D != 128 || a.Hq / a.Hkv > 16 || a.tail_chunk % 64 || a.kv.page_size % 16) return hipErrorInvalidValue;
  if (a.tail_chunks <= 0) return hipSuccess;
  hipLaunchKernelGGL((attn_mfma_kernel<1, true>), dim3(a.tail_chunks, a.Hkv, a.rows.R), dim3(64), 0, s, a);
  return hipGetLastError();
}

template <typename T>
hipError_t attn_prefix_vec(const AttnArgs& a, hipStream_t s) {
  if (a.D > 256 || a.Hq / a.Hkv > 8 || a.split_len > kChunk) return hipErrorInvalidValue;
  if (a.splits <= 0) return hipSuccess;
  hipLaunchKernelGGL((attn_vec_kernel<T, true>), dim3(a.splits, a.Hkv, a.rows.R), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <typename T>
hipError_t attn_tail_vec(const AttnArgs& a, hipStream_t s) {
  if (a.D > 256 || a.Hq / a.Hkv > 8 || a.tail_chunk > kChunk) return hipErrorInvalidValue;
  if (a.tail_chunks <= 0) return hipSuccess;
  hipLaunchKernelGGL((attn_vec_kernel<T, false>), dim3(a.tail_chunks, a.Hkv, a.rows.R), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <typename T>
hipError_t attn_tail_combine(const AttnArgs& a, T* out, hipStream_t s) {
  if (a.D > 128 || a.D < 8 || 256 % a.D || a.Hq / a.Hkv > 8 || (a.tail_len > 0 && !a.rows.pages) ||
      (a.tail_len > 0 && a.kv.page_size % 8) || a.splits > kMaxSplits)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(attn_tail_combine_kernel<T>, dim3(a.rows.R, a.Hkv), dim3(256), 0, s, a, out);
  return hipGetLastError();
}

template <typename T>
hipError_t attn_combine(const AttnArgs& a, T* out, hipStream_t s) {
  hipLaunchKernelGGL(attn_combine_kernel<T>, dim3(a.rows.R, a.Hq), dim3(128), 0, s, a, out);
  return hipGetLastError();
}

template hipError_t attn_prefix_vec<float>(const AttnArgs&, hipStream_t);
template hipError_t attn_prefix_vec<bf16_t>(const AttnArgs&, hipStream_t);
template hipError_t attn_tail_vec<float>(const AttnArgs&, hipStream_t);
template hipError_t attn_tail_vec<bf16_t>(const AttnArgs&, hipStream_t);
template hipError_t attn_combine<float>(const AttnArgs&, float*, hipStream_t);
template hipError_t attn_tail_combine<float>(const AttnArgs&, float*, hipStream_t);
template hipError_t attn_tail_combine<bf16_t>(const AttnArgs&, bf16_t*, hipStream_t);
template hipError_t attn_combine<bf16_t>(const AttnArgs&, bf16_t*, hipStream_t);

}  // namespace rgd
