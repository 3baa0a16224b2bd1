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

RGD_DEV uint32_t pack2(float lo, float hi) {
  return uint32_t(f32_to_bf16(lo)) | (uint32_t(f32_to_bf16(hi)) << 16);
}

// NWAVE waves; PAGED selects the row's paged tail (one row per workgroup)
// instead of the shared prompt prefix (a block of rows of one prompt).
template <int NWAVE, bool PAGED>
__global__ __launch_bounds__(NWAVE * 64) void attn_mfma_kernel(AttnArgs a) {
  constexpr int D = 128, NT = NWAVE * 64, SEGS = 512 / NT;
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
  const int nq = nr * G;
  const int v = wave * 16 + (lane & 15);
  const bool vok = v < nq;
  const bool wave_active = wave * 16 < nq;
  const int row = r0 + (vok ? v / G : 0);
  const int head = g * G + (vok ? v % G : 0);
  const int my_end = PAGED ? hi : (vok ? min(a.rows.plen[row], hi) : lo);

  u32x4 qf[4];
  {
    const bf16_t* qp = (const bf16_t*)a.q + ((long long)row * a.Hq + head) * D + (lane >> 4) * 8;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
      qf[ks] = vok ? *(const u32x4*)(qp + ks * 32) : u32x4{0u, 0u, 0u, 0u};
  }

  __shared__ __attribute__((aligned(16))) bf16_t ks_lds[32][136];
  __shared__ __attribute__((aligned(16))) bf16_t vt_lds[128][40];

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
  auto krow_off = [&](int pos) -> long long {
    if (PAGED) return ((long long)pages[pos / ps] * ps + pos % ps) * pstride;
    return (long long)pos * pstride;
  };
  // start of the 8 V values (d, pos0 .. pos0+7); pos0 is a multiple of 8
  auto v_off = [&](int d, int pos0) -> long long {
    if (PAGED) return ((long long)pages[pos0 / ps] * a.Hkv * D + d) * ps + pos0 % ps;
    return (long long)d * a.kv.VP + pos0;
  };
  const float scale = rsqrtf(float(D)) * kLog2e;

  float m = -INFINITY, lsum = 0.f;
  f32x4 o[8];
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};

  u32x4 kreg[SEGS], vreg[SEGS];
  auto load_tile = [&](int t0) {
#pragma unroll
    for (int i = 0; i < SEGS; ++i) {
      const int seg = threadIdx.x + i * NT;
      // K: 32 positions x 16 segments of 8 dims
      const int pos = t0 + (seg >> 4), pc = (seg & 15) * 8;
      kreg[i] = u32x4{0u, 0u, 0u, 0u};
      if (pos < hi) kreg[i] = *(const u32x4*)(kbase + krow_off(pos) + pc);
      // V^T: 128 dims x 4 segments of 8 positions; positions >= hi read as 0
      const int d = seg >> 2, p0 = t0 + (seg & 3) * 8;
      const int nv = hi - p0;
      u32x4 vv = {0u, 0u, 0u, 0u};
      if (nv > 0) {
        vv = *(const u32x4*)(vbase + v_off(d, p0));
        if (nv < 8) {
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            if (2 * w >= nv) vv[w] = 0u;
            else if (2 * w + 1 >= nv) vv[w] &= 0xFFFFu;
          }
        }
      }
      vreg[i] = vv;
    }
  };

  if (lo < hi) load_tile(lo);
  for (int t0 = lo; t0 < hi; t0 += 32) {
    __syncthreads();
#pragma unroll
    for (int i = 0; i < SEGS; ++i) {
      const int seg = threadIdx.x + i * NT;
      *(u32x4*)&ks_lds[seg >> 4][(seg & 15) * 8] = kreg[i];
      *(u32x4*)&vt_lds[seg >> 2][(seg & 3) * 8] = vreg[i];
    }
    if (t0 + 32 < hi) load_tile(t0 + 32);
    __syncthreads();
    if (wave_active) {
      f32x4 sc[2];
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) {
        sc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          const u32x4 ka = *(const u32x4*)&ks_lds[mt * 16 + (lane & 15)][ks * 32 + (lane >> 4) * 8];
          sc[mt] = mfma16x16x32(ka, qf[ks], sc[mt]);
        }
      }
      float x[8];
      float tmax = -INFINITY;
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int pos = t0 + mt * 16 + (lane >> 4) * 4 + i;
          const float val = pos < my_end ? sc[mt][i] * scale : -INFINITY;
          x[mt * 4 + i] = val;
          tmax = fmaxf(tmax, val);
        }
      tmax = fmaxf(tmax, __shfl_xor(tmax, 16, 64));
      tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
      const float mnew = fmaxf(m, tmax);
      float p[8];
      float alpha = 1.f, ps = 0.f;
      if (mnew == -INFINITY) {
#pragma unroll
        for (int j = 0; j < 8; ++j) p[j] = 0.f;
      } else {
        alpha = exp2f(m - mnew);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          p[j] = exp2f(x[j] - mnew);
          ps += p[j];
        }
      }
      m = mnew;
      lsum = lsum * alpha + ps;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) o[dt] *= alpha;
      const u32x4 pb = {pack2(p[0], p[1]), pack2(p[2], p[3]), pack2(p[4], p[5]), pack2(p[6], p[7])};
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) {
        const bf16_t* vr = &vt_lds[dt * 16 + (lane & 15)][0];
        const u32x2 a0 = *(const u32x2*)(vr + (lane >> 4) * 4);
        const u32x2 a1 = *(const u32x2*)(vr + 16 + (lane >> 4) * 4);
        o[dt] = mfma16x16x32(u32x4{a0.x, a0.y, a1.x, a1.y}, pb, o[dt]);
      }
    }
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
      for (int i = 0; i < 4; ++i) po[dt * 16 + (lane >> 4) * 4 + i] = o[dt][i] * inv;
    if ((lane >> 4) == 0) a.part_lse[idx] = lt > 0.f ? (m + __log2f(lt)) * kLn2 : -INFINITY;
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
  if (a.D != 128 || a.Hq / a.Hkv > 64 || a.split_len % 32 || a.kv.VP % 16) return hipErrorInvalidValue;
  if (a.splits <= 0 || a.nrblocks <= 0) return hipSuccess;
  hipLaunchKernelGGL((attn_mfma_kernel<4, false>), dim3(a.splits, a.Hkv, a.nrblocks), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t attn_tail_mfma_bf16(const AttnArgs& a, hipStream_t s) {
  if (a.D != 128 || a.Hq / a.Hkv > 16 || a.tail_chunk % 32 || a.kv.page_size % 16) return hipErrorInvalidValue;
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
hipError_t attn_combine(const AttnArgs& a, T* out, hipStream_t s) {
  hipLaunchKernelGGL(attn_combine_kernel<T>, dim3(a.rows.R, a.Hq), dim3(128), 0, s, a, out);
  return hipGetLastError();
}

template hipError_t attn_prefix_vec<float>(const AttnArgs&, hipStream_t);
template hipError_t attn_prefix_vec<bf16_t>(const AttnArgs&, hipStream_t);
template hipError_t attn_tail_vec<float>(const AttnArgs&, hipStream_t);
template hipError_t attn_tail_vec<bf16_t>(const AttnArgs&, hipStream_t);
template hipError_t attn_combine<float>(const AttnArgs&, float*, hipStream_t);
template hipError_t attn_combine<bf16_t>(const AttnArgs&, bf16_t*, hipStream_t);

}  // namespace rgd
