// Per-row kernels of the decode step: embedding gather fused with the first
// RMSNorm, RMSNorm of the residual stream, and the Q/K/V epilogue (rotary
// embedding, store of q, append of k/v to the shared prefix or to the row's
// paged tail).
#include "kernels.hpp"
#include "rownorm.hpp"

namespace rgd {

namespace {

constexpr int kNormThreads = 1024;

template <typename T>
__global__ __launch_bounds__(kNormThreads) void embed_rmsnorm_kernel(const int* tok, int tok_stride,
                                                                   const int* tok_map, const T* E, int d, int V,
                                                                   float* x, const float* g, float eps, T* xn) {
  const int r = blockIdx.x;
  const long long src = tok_map ? tok_map[r] : r;
  embed_norm_row(tok[src * tok_stride], E, d, V, g, eps, x + (long long)r * d, xn + (long long)r * d);
}

// Logistic readout of one residual row per workgroup (fixed reduction order).
__global__ __launch_bounds__(256) void residual_readout_kernel(const float* x, long long row0, long long stride,
                                                               int d, const float* w, float b, float* out) {
  __shared__ float red[4];
  const int r = blockIdx.x;
  const float* xr = x + (row0 + r * stride) * d;
  float acc = 0.f;
  for (int i = threadIdx.x; i < d; i += 256) acc = fmaf(xr[i], w[i], acc);
  acc = block_sum(acc, red);
  if (threadIdx.x == 0) out[r] = 1.0f / (1.0f + expf(-(acc + b)));
}

template <typename T>
__global__ __launch_bounds__(kNormThreads) void residual_rmsnorm_kernel(float* x, const float* parts, int nparts,
                                                                      long long part_stride, const float* g,
                                                                      float eps, int d, T* xn) {
  const int r = blockIdx.x;
  float* xr = x + (long long)r * d;
  const float* pr = parts + (long long)r * d;
  float4 v[kChunks], gg[kChunks];
#pragma unroll
  for (int c = 0; c < kChunks; ++c) {
    const int i = (threadIdx.x + c * blockDim.x) * 4;
    v[c] = gg[c] = float4{0.f, 0.f, 0.f, 0.f};
    if (i < d) {
      float4 q[kMaxSplitK];
#pragma unroll
      for (int p = 0; p < kMaxSplitK; ++p)
        if (p < nparts) q[p] = *(const float4*)(pr + p * part_stride + i);
      v[c] = *(const float4*)(xr + i);
      gg[c] = *(const float4*)(g + i);
#pragma unroll
      for (int p = 0; p < kMaxSplitK; ++p)
        if (p < nparts) {
          v[c].x += q[p].x;
          v[c].y += q[p].y;
          v[c].z += q[p].z;
          v[c].w += q[p].w;
        }
      if (nparts > 0) store4(xr + i, v[c]);
    }
  }
  norm_store(v, gg, d, eps, xn + (long long)r * d);
}

// One workgroup per (row, group of 8 heads of the fused q|k|v output).  The
// rotation of position pos, pair j is (cos, sin) = rope_cs[pos][j] (a table
// computed once on the host in fp64).
// NP >= nparts: the loads of all NP split partials (clamped to the last one,
// masked by a 0/1 factor) and of the rotation are issued before any of them is
// used, so the kernel waits for memory once (a partial or a table load used
// only under a condition is moved into a branch by the compiler, which then
// waits for it where the branches join, one memory round trip each).
template <typename T, int NP>
__global__ __launch_bounds__(1024) void qkv_rope_kernel(const float* parts, int nparts, long long part_stride,
                                                       Rows rows, int Hq, int Hkv, int D, const float2* rope_cs,
                                                       int max_pos, T* q, KVLayout kv) {
  const int r = blockIdx.x;
  const int h0 = blockIdx.y * 8, h1 = min(h0 + 8, Hq + 2 * Hkv);
  const int half = D / 2;
  const int pos = min(rows.prefill ? rows.base_pos[r] : rows.base_pos[r] + rows.t, max_pos);
  const float2* cs = rope_cs + (long long)pos * half;
  const int nqkv = (Hq + 2 * Hkv) * D;
  const float* pr = parts + (long long)r * nqkv;
  // columns c and c + D/2, summed over the splits in split order (split-K
  // partials are finite, so the 0/1 factor masks them exactly)
  auto cols = [&](int c, float& v1, float& v2) {
    float a1[NP], a2[NP];
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      const float* pp = pr + min(p, nparts - 1) * part_stride;
      a1[p] = pp[c];
      a2[p] = pp[c + half];
    }
    v1 = a1[0];
    v2 = a2[0];
#pragma unroll
    for (int p = 1; p < NP; ++p) {
      const float f = p < nparts ? 1.f : 0.f;
      v1 += a1[p] * f;
      v2 += a2[p] * f;
    }
  };
  const int b = rows.prompt[r];
  // destinations: K of head h at kd + h * kstride; V of head h, dim d at
  // vd + h * vhstride + d * vdstride
  T* kd;
  T* vd;
  long long kstride, vhstride, vdstride;
  if (rows.prefill) {
    kd = (T*)kv.prefix_k + ((long long)b * Hkv * kv.P + pos) * D;
    kstride = (long long)kv.P * D;
    vd = (T*)kv.prefix_v + ((long long)b * Hkv * (kv.VP / 64) + pos / 64) * D * 64 + pos % 64;
    vhstride = (long long)kv.VP * D;
    vdstride = 64;
  } else {
    const int ps = kv.page_size;
    const int page = rows.pages[(long long)r * rows.max_pages + rows.t / ps];
    const int slot = rows.t % ps;
    kd = (T*)kv.pool_k + ((long long)page * Hkv * ps + slot) * D;
    kstride = (long long)ps * D;
    vd = (T*)kv.pool_v + (long long)page * Hkv * D * ps + slot;
    vhstride = (long long)D * ps;
    vdstride = ps;
  }
  const int nh = h1 - h0;
  for (int i = threadIdx.x; i < nh * half; i += blockDim.x) {
    const int h = h0 + i / half, j = i % half;
    const int base = h * D;
    float x1, x2;
    cols(base + j, x1, x2);
    // q and k pairs (j, j + D/2) are rotated, v passes through (cos 1, sin 0)
    const float2 cj = cs[j];
    const float kq = h < Hq + Hkv ? 1.f : 0.f;
    const float c = cj.x * kq + (1.f - kq), sn = cj.y * kq;
    const float y1 = x1 * c - x2 * sn;
    const float y2 = x2 * c + x1 * sn;
    if (h < Hq + Hkv) {
      T* dst = h < Hq ? q + ((long long)r * Hq + h) * D : kd + (long long)(h - Hq) * kstride;
      store_f(dst + j, y1);
      store_f(dst + j + half, y2);
    } else {             // v: dims j and j + D/2 of head h - Hq - Hkv
      const int hv = h - Hq - Hkv;
      store_f(vd + hv * vhstride + (long long)j * vdstride, y1);
      store_f(vd + hv * vhstride + (long long)(j + half) * vdstride, y2);
    }
  }
}

}  // namespace

template <typename T>
hipError_t embed_rmsnorm(const int* tok, int tok_stride, const int* tok_map, int R, const T* E, int d, int V,
                         float* x, const float* g, float eps, T* xn, hipStream_t s) {
  if (d % 4 || d > kChunks * 4 * kNormThreads) return hipErrorInvalidValue;
  hipLaunchKernelGGL(embed_rmsnorm_kernel<T>, dim3(R), dim3(kNormThreads), 0, s, tok, tok_stride, tok_map, E, d,
                     V, x, g, eps, xn);
  return hipGetLastError();
}

hipError_t residual_readout(const float* x, long long row0, long long stride, int nrows, int d, const float* w,
                            float b, float* out, hipStream_t s) {
  if (nrows <= 0) return hipSuccess;
  hipLaunchKernelGGL(residual_readout_kernel, dim3(nrows), dim3(256), 0, s, x, row0, stride, d, w, b, out);
  return hipGetLastError();
}

template <typename T>
hipError_t residual_rmsnorm(float* x, const float* parts, int nparts, long long part_stride, const float* g,
                            float eps, int R, int d, T* xn, hipStream_t s) {
  if (d % 4 || d > kChunks * 4 * kNormThreads || nparts < 0 || nparts > kMaxSplitK) return hipErrorInvalidValue;
  hipLaunchKernelGGL(residual_rmsnorm_kernel<T>, dim3(R), dim3(kNormThreads), 0, s, x, parts, nparts, part_stride,
                     g, eps, d, xn);
  return hipGetLastError();
}

template <typename T>
hipError_t qkv_rope_store(const float* parts, int nparts, long long part_stride, const Rows& rows, int Hq,
                          int Hkv, int D, const float* rope_cs, int max_pos, T* q, const KVLayout& kv,
                          hipStream_t s) {
  if (D > 256 || (D & 1) || nparts < 1 || nparts > kMaxSplitK) return hipErrorInvalidValue;
  // one thread per (head of the group of 8, rotation pair)
  const int threads = std::max(64, 8 * (D / 2));
  const dim3 grid(rows.R, (Hq + 2 * Hkv + 7) / 8);
  if (nparts <= 4)
    hipLaunchKernelGGL((qkv_rope_kernel<T, 4>), grid, dim3(threads), 0, s, parts, nparts, part_stride, rows, Hq, Hkv,
                       D, (const float2*)rope_cs, max_pos, q, kv);
  else if (nparts <= 8)
    hipLaunchKernelGGL((qkv_rope_kernel<T, 8>), grid, dim3(threads), 0, s, parts, nparts, part_stride, rows, Hq, Hkv,
                       D, (const float2*)rope_cs, max_pos, q, kv);
  else
    hipLaunchKernelGGL((qkv_rope_kernel<T, kMaxSplitK>), grid, dim3(threads), 0, s, parts, nparts, part_stride, rows,
                       Hq, Hkv, D, (const float2*)rope_cs, max_pos, q, kv);
  return hipGetLastError();
}

template hipError_t embed_rmsnorm<float>(const int*, int, const int*, int, const float*, int, int, float*, const float*,
                                         float, float*, hipStream_t);
template hipError_t embed_rmsnorm<bf16_t>(const int*, int, const int*, int, const bf16_t*, int, int, float*, const float*,
                                          float, bf16_t*, hipStream_t);
template hipError_t residual_rmsnorm<float>(float*, const float*, int, long long, const float*, float, int, int,
                                            float*, hipStream_t);
template hipError_t residual_rmsnorm<bf16_t>(float*, const float*, int, long long, const float*, float, int, int,
                                             bf16_t*, hipStream_t);
template hipError_t qkv_rope_store<float>(const float*, int, long long, const Rows&, int, int, int, const float*, int, float*,
                                          const KVLayout&, hipStream_t);
template hipError_t qkv_rope_store<bf16_t>(const float*, int, long long, const Rows&, int, int, int, const float*, int,
                                           bf16_t*, const KVLayout&, hipStream_t);

}  // namespace rgd
