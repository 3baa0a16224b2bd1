// Row helpers shared by the per-row kernels: a row of d values is spread over
// the threads of one workgroup in float4 chunks held in registers.
#pragma once
#include "common.hpp"

namespace rgd {
namespace {

// Each thread owns up to kChunks float4 chunks of a row (chunk c of thread t
// covers elements (t + c * blockDim) * 4 .. +3), keeps them in registers
// through the residual update and the norm, and issues all its loads (x,
// split partials, gain) before using any: one round trip to memory per row.
constexpr int kChunks = 4;  // d <= kChunks * 4 * blockDim.x

RGD_DEV float4 load4(const float* p) { return *(const float4*)p; }
RGD_DEV float4 load4(const bf16_t* p) {
  const uint2 u = *(const uint2*)p;
  return float4{__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u), __uint_as_float(u.y << 16),
                __uint_as_float(u.y & 0xFFFF0000u)};
}
RGD_DEV void store4(float* p, float4 v) { *(float4*)p = v; }
RGD_DEV void store4(bf16_t* p, float4 v) { *(uint2*)p = uint2{pack_bf16x2(v.x, v.y), pack_bf16x2(v.z, v.w)}; }

// xn = v / sqrt(mean(v^2) + eps) * g for the chunks held in registers
template <typename T>
RGD_DEV void norm_store(const float4 (&v)[kChunks], const float4 (&gg)[kChunks], int d, float eps, T* xn) {
  __shared__ float red[16];
  float ss = 0.f;
  // chunks past d do not count (a per-lane select, not a branch: a value used
  // only inside a branch makes the compiler move its load there and wait)
#pragma unroll
  for (int c = 0; c < kChunks; ++c) {
    const int i = (threadIdx.x + c * blockDim.x) * 4;
    const float q = v[c].x * v[c].x + v[c].y * v[c].y + v[c].z * v[c].z + v[c].w * v[c].w;
    ss += i < d ? q : 0.f;
  }
  ss = block_sum(ss, red);
  const float inv = rsqrtf(ss / float(d) + eps);
#pragma unroll
  for (int c = 0; c < kChunks; ++c) {
    const int i = (threadIdx.x + c * blockDim.x) * 4;
    if (i < d)
      store4(xn + i, float4{v[c].x * inv * gg[c].x, v[c].y * inv * gg[c].y, v[c].z * inv * gg[c].z,
                            v[c].w * inv * gg[c].w});
  }
}

// x = E[t] (fp32) and xn = x / sqrt(mean(x^2) + eps) * g for one row, with the
// id clamped into [0, V) so that a bad id cannot read outside the table.
// Needs d % 4 == 0 and d <= kChunks * 4 * blockDim.x.
template <typename T>
RGD_DEV void embed_norm_row(int tok, const T* E, int d, int V, const float* g, float eps, float* x, T* xn) {
  const long long t = min(max(tok, 0), V - 1);
  float4 v[kChunks], gg[kChunks];
  // unconditional loads from clamped addresses (chunks past d are left out
  // of the norm and not stored)
#pragma unroll
  for (int c = 0; c < kChunks; ++c) {
    const int i = min((int)(threadIdx.x + c * blockDim.x) * 4, d - 4);
    v[c] = load4(E + t * d + i);
    gg[c] = load4(g + i);
  }
#pragma unroll
  for (int c = 0; c < kChunks; ++c) {
    const int i = (threadIdx.x + c * blockDim.x) * 4;
    if (i < d) store4(x + i, v[c]);
  }
  norm_store(v, gg, d, eps, xn);
}

}  // namespace
}  // namespace rgd
