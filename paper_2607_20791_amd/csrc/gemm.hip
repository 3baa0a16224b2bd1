// Skinny-M GEMMs for the decode step: Y = X W^T.
//
// bf16 path: one workgroup (4 waves) owns 64 output columns and MT*16 rows.
// Each wave streams its 16 weight rows straight from HBM into registers (a
// lane reads 64 contiguous bytes of one row per 128-wide k block, prefetched
// one block ahead) while the X rows of the block are staged once per k block
// in LDS and shared by the four waves.  The product runs on
// v_mfma_f32_16x16x32_bf16 with fp32 accumulation.  Because the contraction
// index only has to be permuted the same way for both operands, each lane's
// 32-element k slice is taken contiguously, which keeps every global load
// 64 B wide.
#include "kernels.hpp"

namespace rgd {

namespace {

RGD_DEV f32x4 mfma16x16x32(const u32x4& a, const u32x4& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

RGD_DEV float silu(float g) { return g / (1.0f + __expf(-g)); }

template <int MT, int MODE>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(GemmArgs a) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int tile = blockIdx.x;
  const int m0 = blockIdx.y * (MT * 16);
  const int split = blockIdx.z;
  const int K = a.K;
  const int nkb = K >> 7;
  const int kb0 = int((long long)split * nkb / a.splits);
  const int kb1 = int((long long)(split + 1) * nkb / a.splits);

  // the weight row (output column) feeding this lane's B operand
  int n;
  const bf16_t* wrow;
  if (MODE == GEMM_SILU) {
    n = tile * 32 + (wave & 1) * 16 + (lane & 15);
    const GemmSeg& sg = a.seg[wave >> 1];
    wrow = (const bf16_t*)sg.w + (long long)min(n, a.N - 1) * K;
  } else {
    n = tile * 64 + wave * 16 + (lane & 15);
    const int c0 = tile * 64;
    int si = 0;
    if (a.nseg > 1 && c0 >= a.seg[1].n0) si = 1;
    if (a.nseg > 2 && c0 >= a.seg[2].n0) si = 2;
    const GemmSeg& sg = a.seg[si];
    wrow = (const bf16_t*)sg.w + (long long)(min(n, a.N - 1) - sg.n0) * K;
  }

  __shared__ __attribute__((aligned(16))) bf16_t xs[MT * 16][136];
  f32x4 acc[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};

  const bf16_t* X = (const bf16_t*)a.x;
  const int kq = (lane >> 4) * 32;
  u32x4 wb[4], wn[4];
  if (kb0 < kb1) {
    const u32x4* p = (const u32x4*)(wrow + (kb0 << 7) + kq);
#pragma unroll
    for (int j = 0; j < 4; ++j) wb[j] = __builtin_nontemporal_load(p + j);
  }
  for (int kb = kb0; kb < kb1; ++kb) {
    for (int i = threadIdx.x; i < MT * 16 * 16; i += 256) {
      const int r = i >> 4, c = (i & 15) * 8, m = m0 + r;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (m < a.M) v = *(const u32x4*)(X + (long long)m * a.ldx + (kb << 7) + c);
      *(u32x4*)&xs[r][c] = v;
    }
    if (kb + 1 < kb1) {
      const u32x4* p = (const u32x4*)(wrow + ((kb + 1) << 7) + kq);
#pragma unroll
      for (int j = 0; j < 4; ++j) wn[j] = __builtin_nontemporal_load(p + j);
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 4; ++j) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const u32x4 av = *(const u32x4*)&xs[mt * 16 + (lane & 15)][kq + j * 8];
        acc[mt] = mfma16x16x32(av, wb[j], acc[mt]);
      }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 4; ++j) wb[j] = wn[j];
  }

  // D layout of the 16x16 MFMA: lane holds rows 4*(lane/16)+i of column lane%16
  const int rq = (lane >> 4) * 4;
  if (MODE == GEMM_PARTIAL) {
    float* Y = (float*)a.y + (long long)split * a.split_stride;
    if (n < a.N) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = m0 + mt * 16 + rq + i;
          if (m < a.M) Y[(long long)m * a.ldy + n] = acc[mt][i];
        }
    }
  } else if (MODE == GEMM_LOGITS) {
    float* Y = (float*)a.y;
    __shared__ float red[4][MT * 16];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = m0 + mt * 16 + rq + i;
        const bool ok = (m < a.M) && (n < a.N);
        if (ok) Y[(long long)m * a.ldy + n] = acc[mt][i];
        float v = ok ? acc[mt][i] : -INFINITY;
        v = fmaxf(v, __shfl_xor(v, 1, 64));
        v = fmaxf(v, __shfl_xor(v, 2, 64));
        v = fmaxf(v, __shfl_xor(v, 4, 64));
        v = fmaxf(v, __shfl_xor(v, 8, 64));
        if ((lane & 15) == 0) red[wave][mt * 16 + rq + i] = v;
      }
    __syncthreads();
    if (threadIdx.x < MT * 16) {
      const int m = m0 + threadIdx.x;
      const float v = fmaxf(fmaxf(red[0][threadIdx.x], red[1][threadIdx.x]),
                            fmaxf(red[2][threadIdx.x], red[3][threadIdx.x]));
      if (m < a.M) a.tilemax[(long long)m * a.ntiles + tile] = v;
    }
  } else {  // GEMM_SILU: waves 2,3 hold the up projection of waves 0,1's features
    __shared__ float up[MT * 16][33];
    if (wave >= 2) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) up[mt * 16 + rq + i][(wave - 2) * 16 + (lane & 15)] = acc[mt][i];
    }
    __syncthreads();
    if (wave < 2 && n < a.N) {
      bf16_t* Y = (bf16_t*)a.y;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = m0 + mt * 16 + rq + i;
          const float u = up[mt * 16 + rq + i][wave * 16 + (lane & 15)];
          if (m < a.M) Y[(long long)m * a.ldy + n] = f32_to_bf16(silu(acc[mt][i]) * u);
        }
    }
  }
}

template <int MODE>
hipError_t launch_bf16(const GemmArgs& a, hipStream_t s) {
  const int ntile = MODE == GEMM_SILU ? (a.N + 31) / 32 : (a.N + 63) / 64;
  const int splits = MODE == GEMM_PARTIAL ? a.splits : 1;
  GemmArgs b = a;
  b.splits = splits;
  if (a.M <= 16) {
    hipLaunchKernelGGL((gemm_bf16_kernel<1, MODE>), dim3(ntile, 1, splits), dim3(256), 0, s, b);
  } else if (a.M <= 32) {
    hipLaunchKernelGGL((gemm_bf16_kernel<2, MODE>), dim3(ntile, 1, splits), dim3(256), 0, s, b);
  } else {
    hipLaunchKernelGGL((gemm_bf16_kernel<4, MODE>), dim3(ntile, (a.M + 63) / 64, splits), dim3(256),
                       0, s, b);
  }
  return hipGetLastError();
}

// ----------------------------------------------------------------- fp32 ----
// Plain fp32 path for small fp32 models: one thread per output element.
template <int MODE>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs a) {
  const int n = blockIdx.x * 256 + threadIdx.x;
  const int m = blockIdx.y;
  const float* x = (const float*)a.x + (long long)m * a.ldx;
  const int K = a.K;
  const bool ok = n < a.N;
  const int nc = min(n, a.N - 1);
  float acc = 0.f, acc2 = 0.f;
  if (MODE == GEMM_SILU) {
    const float* wg = (const float*)a.seg[0].w + (long long)nc * K;
    const float* wu = (const float*)a.seg[1].w + (long long)nc * K;
    for (int k = 0; k < K; ++k) { acc += x[k] * wg[k]; acc2 += x[k] * wu[k]; }
    if (ok) ((float*)a.y)[(long long)m * a.ldy + n] = silu(acc) * acc2;
    return;
  }
  int si = 0;
  if (a.nseg > 1 && nc >= a.seg[1].n0) si = 1;
  if (a.nseg > 2 && nc >= a.seg[2].n0) si = 2;
  const float* w = (const float*)a.seg[si].w + (long long)(nc - a.seg[si].n0) * K;
  for (int k = 0; k < K; ++k) acc += x[k] * w[k];
  if (MODE == GEMM_PARTIAL) {
    if (ok) ((float*)a.y)[(long long)m * a.ldy + n] = acc;
  } else {
    if (ok) ((float*)a.y)[(long long)m * a.ldy + n] = acc;
    // 64 consecutive columns form one wave: its max is that tile's max
    const float v = wave_max(ok ? acc : -INFINITY);
    if ((threadIdx.x & 63) == 0 && ok) a.tilemax[(long long)m * a.ntiles + n / 64] = v;
  }
}

}  // namespace

hipError_t gemm_bf16(const GemmArgs& a, hipStream_t s) {
  if (a.K % 128 != 0) return hipErrorInvalidValue;
  switch (a.mode) {
    case GEMM_PARTIAL: return launch_bf16<GEMM_PARTIAL>(a, s);
    case GEMM_SILU: return launch_bf16<GEMM_SILU>(a, s);
    default: return launch_bf16<GEMM_LOGITS>(a, s);
  }
}

hipError_t gemm_f32(const GemmArgs& a, hipStream_t s) {
  dim3 grid((a.N + 255) / 256, a.M);
  switch (a.mode) {
    case GEMM_PARTIAL:
      hipLaunchKernelGGL(gemm_f32_kernel<GEMM_PARTIAL>, grid, dim3(256), 0, s, a); break;
    case GEMM_SILU:
      hipLaunchKernelGGL(gemm_f32_kernel<GEMM_SILU>, grid, dim3(256), 0, s, a); break;
    default:
      hipLaunchKernelGGL(gemm_f32_kernel<GEMM_LOGITS>, grid, dim3(256), 0, s, a); break;
  }
  return hipGetLastError();
}

}  // namespace rgd
