// Shared device/host helpers for the refusal-gated decoding library (gfx950).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#define RGD_DEV __device__ __forceinline__

typedef uint16_t bf16_t;  // bf16 storage (bit pattern)
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

namespace rgd {

constexpr int kWave = 64;

RGD_DEV float bf16_to_f32(bf16_t b) { return __uint_as_float(uint32_t(b) << 16); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// round-to-nearest-even float -> bf16 (v_cvt_pk_bf16_f32 on gfx950)
RGD_DEV bf16_t f32_to_bf16(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }

// two floats -> packed bf16 pair (lo in bits 0..15)
RGD_DEV uint32_t pack_bf16x2(float lo, float hi) {
  const bf16x2_t v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

template <typename T> RGD_DEV float load_f(const T* p);
template <> RGD_DEV float load_f<float>(const float* p) { return *p; }
template <> RGD_DEV float load_f<bf16_t>(const bf16_t* p) { return bf16_to_f32(*p); }

template <typename T> RGD_DEV void store_f(T* p, float v);
template <> RGD_DEV void store_f<float>(float* p, float v) { *p = v; }
template <> RGD_DEV void store_f<bf16_t>(bf16_t* p, float v) { *p = f32_to_bf16(v); }

// Order-preserving map float -> uint32 (for max via integer atomics).
RGD_DEV uint32_t ordered_u32(float f) {
  uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
RGD_DEV float from_ordered_u32(uint32_t o) {
  uint32_t u = (o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o;
  return __uint_as_float(u);
}

RGD_DEV float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}
RGD_DEV float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// Block-wide reductions for blockDim.x a multiple of 64 (<= 1024).  `scratch`
// must hold blockDim.x/64 floats; the result is broadcast to every thread.
RGD_DEV float block_sum(float v, float* scratch) {
  v = wave_sum(v);
  const int w = threadIdx.x / kWave, nw = blockDim.x / kWave;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) scratch[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < nw; ++i) t += scratch[i];
  return t;
}
RGD_DEV float block_max(float v, float* scratch) {
  v = wave_max(v);
  const int w = threadIdx.x / kWave, nw = blockDim.x / kWave;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) scratch[w] = v;
  __syncthreads();
  float t = -INFINITY;
  for (int i = 0; i < nw; ++i) t = fmaxf(t, scratch[i]);
  return t;
}

}  // namespace rgd
