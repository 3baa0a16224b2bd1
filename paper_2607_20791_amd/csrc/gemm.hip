// Skinny-M GEMMs of the decode step: Y = X W^T with X [M][K] (bf16) and W
// [N][K].
//
// At decode sizes every GEMM is bound by streaming W from HBM.  Weights are
// repacked once, at model creation, into 16-row panels: panel p holds rows
// [16p, 16p+16) as 2 KiB blocks of 64 k values.  A block is two dense 1 KiB
// halves, one per MFMA of the 64-k step, each in the order the MFMA B operand
// is loaded: lane l = 16q + r reads 16 contiguous bytes, row r, k values
// 16q + 8h + {0..7} of the block (h = half).  Every weight load instruction of
// a wave is thus one dense 1 KiB read.  The blocks of a group of G panels are
// interleaved step by step (block (p, st) at ((p/G)*steps + st)*G + p%G), G
// being the panels one wave streams: G = 1 (each panel one contiguous run) for
// the projections, G = kHeadGroup for the LM head, whose waves then read one
// contiguous 8 KiB run per step instead of four 2 KiB blocks 128 KiB apart
// (measured with the weights evicted: 165 against 173 us for the one-row LM
// head, 174 against 177 us at 64 rows; a weight-only stream in this layout
// matches a flat read of the same bytes).
//
// A workgroup owns NW*NT panels (waves split N; for SwiGLU the first half of
// the waves computes the gate panels and the second half the matching up
// panels) and one K range (split-K across workgroups when N alone gives too
// few workgroups).  The X rows of the current 64-wide k step are staged once
// in a two-slot LDS ring shared by all waves; each wave keeps SW steps of its
// weight panels in flight in registers.  Products run on
// v_mfma_f32_16x16x32_bf16 with fp32 accumulation; X and W take the same
// permutation of the contraction index.
#include "kernels.hpp"

namespace rgd {

namespace {

RGD_DEV f32x4 mfma16x16x32(const u32x4& a, const u32x4& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

RGD_DEV float silu(float g) { return g / (1.0f + __expf(-g)); }

constexpr int kStep = 64;  // k values per pipeline step

// X stage layouts.  Swizzled (the projections and SwiGLU): unpadded rows of
// XS * 64 k values whose 16-byte chunks are XOR-swizzled, chunk c of row r at
// chunk c ^ xswz<XS>(r); the A fragment reads (16 consecutive rows at one chunk
// per 16 lanes, the next lane group two chunks on) and the stage stores
// (consecutive lanes along a row) are then free of LDS bank conflicts, which
// the conflict counter put at 37-44% of the LDS cycles with padded rows (the
// functions were chosen by measuring each access pattern under that counter;
// 128-row tiles 3-15% faster).  Padded (the LM head, whose A fragment feeds
// four MFMAs): rows padded by 16 bytes, unswizzled; the swizzled layout made
// it 2-7% slower.
template <int XS>
RGD_DEV int xswz(int r) { return XS == 1 ? ((r & 7) ^ ((r >> 3) & 1)) : (r & 15); }

// panels of N rows, rounded up to whole groups
__host__ __device__ inline long long packed_panels(int N, int group) {
  return (long long)((N + 15) / 16 + group - 1) / group * group;
}

// W [N][K] row-major -> 2 KiB blocks [panel groups][K/64][group][2 halves]
// [64 lanes][8]; rows past N are zero.  One thread per 16-byte output chunk.
__global__ void pack_panels_kernel(const bf16_t* __restrict__ w, int N, int K, int group,
                                   bf16_t* __restrict__ out) {
  const long long nst = K / kStep;
  const long long total = packed_panels(N, group) * nst * 128;  // 16-byte chunks
  for (long long c = blockIdx.x * 256ll + threadIdx.x; c < total; c += 256ll * gridDim.x) {
    const int lane = int(c & 63), h = int((c >> 6) & 1);
    const long long blk = c >> 7;
    const long long gsz = nst * group, rem = blk % gsz;
    const long long st = rem / group, p = blk / gsz * group + rem % group;
    const int r = lane & 15, q = lane >> 4;
    const long long row = p * 16 + r;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (row < N) v = *(const u32x4*)(w + row * K + st * kStep + q * 16 + h * 8);
    *(u32x4*)(out + c * 8) = v;
  }
}

// XS: 64-k steps of X staged per LDS slot (one barrier per XS steps).
template <int MT, int NT, int NW, int SW, int MODE, int XS>
__global__ __launch_bounds__(NW * 64) void gemm_bf16_kernel(GemmArgs a) {
  constexpr int NTH = NW * 64, XSEG = MT * 16 * 8 * XS, XPT = (XSEG + NTH - 1) / NTH;
  static_assert(XS % SW == 0 || SW % XS == 0, "ring slots must stay static within an X stage");
  static_assert(XS == 1 || XS == 2 || XS == 4, "the X-stage swizzle covers stages of 1, 2 or 4 steps");
  // wave index as a scalar: the panel and weight segment it selects are then
  // scalar too (a per-lane index into the arguments becomes a vector load of
  // the argument segment and a full memory round trip before the first weight
  // request)
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), col16 = lane & 15;
  // Workgroups are handed out in linear order (x fastest), round-robin over
  // the chip's 8 XCDs, each with its own L2.  With several row blocks, the
  // work is reordered so that the row blocks of one column group are 8 apart
  // in that order: on one XCD at nearly the same time, so the later blocks'
  // weight reads can hit the lines the first one brought into that L2.
  int gx = blockIdx.x, gy = blockIdx.y;
  if (MT > 4 && gridDim.y > 1) {  // 64-row tiles are launched as one row block
    const int G = gridDim.x, Y = gridDim.y;
    const int lin = blockIdx.x + blockIdx.y * G;
    const int full = (G / 8) * 8;  // column groups in whole octets
    if (lin < full * Y) {
      gy = (lin / 8) % Y;
      gx = (lin / 8 / Y) * 8 + lin % 8;
    } else {
      const int rem = lin - full * Y, gr = G - full;
      gx = full + rem % gr;
      gy = rem / gr;
    }
  }
  const int m0 = gy * (MT * 16);
  const int split = blockIdx.z;
  const int K = a.K, nst = K / kStep;
  const int st0 = int((long long)split * nst / a.splits), st1 = int((long long)(split + 1) * nst / a.splits);

  // panels of this wave
  constexpr int HALF = (MODE == GEMM_SILU) ? NW / 2 : NW;
  const int wslot = (MODE == GEMM_SILU) ? (wave % HALF) : wave;
  const int p0 = (gx * HALF + wslot) * NT;  // first panel (in units of 16 columns)
  // panels interleaved per step in the weight layout: the LM head's wave groups
  constexpr int PG = (MODE == GEMM_LOGITS) ? NT : 1;
  static_assert(MODE != GEMM_LOGITS || NT == kHeadGroup, "LM head waves own one packed panel group");
  const bf16_t* wp[NT];
  int ncol[NT];
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    int p = p0 + j;
    int si = 0;
    if (MODE == GEMM_SILU) {
      si = wave / HALF;
    } else {
      if (a.nseg > 1 && p * 16 >= a.seg[1].n0) si = 1;
      if (a.nseg > 2 && p * 16 >= a.seg[2].n0) si = 2;
    }
    const int lp = min(p - a.seg[si].n0 / 16, (a.seg[si].n + 15) / 16 - 1);  // panel within the segment
    wp[j] = (const bf16_t*)a.seg[si].w + (((long long)(lp / PG) * nst) * PG + lp % PG) * 1024 + lane * 8;
    ncol[j] = p * 16 + col16;
  }

  // LDS: the two X stage slots; the SwiGLU hand-over of the up sums (after
  // the main loop, behind a barrier) reuses the same bytes
  constexpr bool XSW = MODE != GEMM_LOGITS;  // swizzled X stage (else padded)
  using XStage = bf16_t[2][MT * 16][XS * kStep + (XSW ? 0 : 8)];
  constexpr int kUpWaves = (MODE == GEMM_SILU) ? HALF : 1;  // sized for SwiGLU only
  using UpSums = float[kUpWaves][MT * NT * 4][64];
  constexpr int kLdsBytes = sizeof(XStage) > sizeof(UpSums) ? (int)sizeof(XStage) : (int)sizeof(UpSums);
  __shared__ __attribute__((aligned(16))) unsigned char lds[kLdsBytes];
  XStage& xs = *reinterpret_cast<XStage*>(lds);
  f32x4 acc[MT][NT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[mt][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // One 16-row tile (M <= 16, the probe's one-row steps): the A fragments come
  // straight from X in global memory (a few KiB, cache-resident) through a
  // register ring beside the weights' ring, with no LDS staging and no
  // barrier per stage.  Each lane reads the same row and k values it would
  // read from LDS, so the arithmetic is that of the staged path.
  constexpr bool XG = (MT == 1);
  const int kq = (lane >> 4) * 16;
  u32x4 wb[SW][NT][2], xr[XPT], xa[SW][2];
  const bf16_t* xrow = (const bf16_t*)a.x + (long long)min(m0 + col16, a.M - 1) * a.ldx + kq;
  auto loadxa = [&](int st, int slot) {
    xa[slot][0] = *(const u32x4*)(xrow + (long long)st * kStep);
    xa[slot][1] = *(const u32x4*)(xrow + (long long)st * kStep + 8);
  };
  auto loadw = [&](int st, int slot) {
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      const bf16_t* p = wp[j] + (long long)st * (PG * 1024);
      wb[slot][j][0] = __builtin_nontemporal_load((const u32x4*)p);
      wb[slot][j][1] = __builtin_nontemporal_load((const u32x4*)(p + 512));
    }
  };
  const bf16_t* X = (const bf16_t*)a.x;
  // X rows of the stage starting at step c0: XS * 8 16-byte segments per row
  auto loadx = [&](int c0) {
#pragma unroll
    for (int i = 0; i < XPT; ++i) {
      const int seg = threadIdx.x + i * NTH;
      const int r = seg / (8 * XS), c = (seg % (8 * XS)) * 8;
      const int m = m0 + r;
      const int k = c0 * kStep + c;
      xr[i] = (seg < XSEG && m < a.M && k < st1 * kStep) ? *(const u32x4*)(X + (long long)m * a.ldx + k)
                                                          : u32x4{0u, 0u, 0u, 0u};
    }
  };
  auto storex = [&](int slot) {
#pragma unroll
    for (int i = 0; i < XPT; ++i) {
      const int seg = threadIdx.x + i * NTH;
      const int row = seg / (8 * XS), c = seg % (8 * XS);
      if (seg < XSEG) *(u32x4*)&xs[slot][row][(XSW ? c ^ xswz<XS>(row) : c) * 8] = xr[i];
    }
  };

#pragma unroll
  for (int j = 0; j < SW; ++j)
    if (st0 + j < st1) {
      loadw(st0 + j, j);
      if (XG) loadxa(st0 + j, j);
    }
  if (!XG && st0 < st1) loadx(st0);
  // W ring: step st lives in slot (st - st0) % SW; X stage g covers steps
  // [st0 + g*XS, st0 + (g+1)*XS)
  constexpr int UN = XS > SW ? XS : SW;  // steps per unrolled block
  for (int sb = st0; sb < st1; sb += UN) {
#pragma unroll
    for (int j = 0; j < UN; ++j) {
      const int st = sb + j;
      if (st < st1) {
        const int g = (st - st0) / XS, kk = ((st - st0) % XS) * kStep;
        const int xsl = g & 1;
        if (!XG && kk == 0) {  // first step of a stage: publish it, fetch the next
          storex(xsl);
          if (st + XS < st1) loadx(st + XS);
          __syncthreads();
        }
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            const int xc = (kk + kq + h * 8) >> 3;  // 16-byte chunk of the fragment
            const u32x4 av = XG ? xa[j % SW][h]
                                : *(const u32x4*)&xs[xsl][mt * 16 + col16]
                                                   [(XSW ? xc ^ xswz<XS>(mt * 16 + col16) : xc) * 8];
#pragma unroll
            for (int jj = 0; jj < NT; ++jj) acc[mt][jj] = mfma16x16x32(av, wb[j % SW][jj][h], acc[mt][jj]);
          }
        if (st + SW < st1) {
          loadw(st + SW, j % SW);
          if (XG) loadxa(st + SW, j % SW);
        }
      }
    }
  }

  // D layout of the 16x16 MFMA: lane holds rows 4*(lane/16)+i of column lane%16
  const int rq = (lane >> 4) * 4;
  if (MODE == GEMM_STORE) {
    float* Y = (float*)a.y + (long long)split * a.split_stride;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int j = 0; j < NT; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = m0 + mt * 16 + rq + i;
          if (m < a.M && ncol[j] < a.N) Y[(long long)m * a.ldy + ncol[j]] = acc[mt][j][i];
        }
  } else if (MODE == GEMM_SILU) {
    // up-projection waves hand their sums to the gate waves through LDS
    UpSums& up = *reinterpret_cast<UpSums*>(lds);
    __syncthreads();  // every wave is past its last X read
    if (wave >= HALF) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int j = 0; j < NT; ++j)
#pragma unroll
          for (int i = 0; i < 4; ++i) up[wslot][(mt * NT + j) * 4 + i][lane] = acc[mt][j][i];
    }
    __syncthreads();
    if (wave < HALF) {
      bf16_t* Y = (bf16_t*)a.y;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int j = 0; j < NT; ++j)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int m = m0 + mt * 16 + rq + i;
            const float u = up[wslot][(mt * NT + j) * 4 + i][lane];
            if (m < a.M && ncol[j] < a.N)
              Y[(long long)m * a.ldy + ncol[j]] = f32_to_bf16(silu(acc[mt][j][i]) * u);
          }
    }
  } else {  // GEMM_LOGITS: logits plus one maximum (and argmax key) per (row, workgroup)
    float* Y = (float*)a.y;
    __shared__ float red[NW][MT * 16];
    __shared__ unsigned long long redk[NW][MT * 16];
    const bool keys = a.tilekey != nullptr;  // uniform
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = m0 + mt * 16 + rq + i;
        float v = -INFINITY;
        unsigned long long kb = 0ull;
#pragma unroll
        for (int j = 0; j < NT; ++j) {
          const bool ok = m < a.M && ncol[j] < a.N;
          if (ok) Y[(long long)m * a.ldy + ncol[j]] = acc[mt][j][i];
          v = fmaxf(v, ok ? acc[mt][j][i] : -INFINITY);
          if (ok) {
            const unsigned long long kj = ((unsigned long long)ordered_u32(acc[mt][j][i]) << 32) |
                                          (unsigned long long)(0xFFFFFFFFu - uint32_t(ncol[j]));
            kb = kj > kb ? kj : kb;
          }
        }
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) {
          v = fmaxf(v, __shfl_xor(v, o, 64));
          if (keys) {
            const unsigned long long ko = __shfl_xor(kb, o, 64);
            kb = ko > kb ? ko : kb;
          }
        }
        if (col16 == 0) {
          red[wave][mt * 16 + rq + i] = v;
          redk[wave][mt * 16 + rq + i] = kb;
        }
      }
    __syncthreads();
    for (int t = threadIdx.x; t < MT * 16; t += NTH) {
      float v = red[0][t];
      unsigned long long kb = redk[0][t];
      for (int w = 1; w < NW; ++w) {
        v = fmaxf(v, red[w][t]);
        kb = redk[w][t] > kb ? redk[w][t] : kb;
      }
      const int m = m0 + t;
      if (m < a.M) {
        a.tilemax[(long long)m * a.ntiles + gx] = v;
        if (keys) a.tilekey[(long long)m * a.ntiles + gx] = kb;
      }
    }
  }
}

// Row tiles per workgroup follow M (16, 32, 64 or 128 rows; larger M takes
// several 128-row blocks, whose weight reads then largely hit in L2); the
// 128-row tile stages X two 64-k steps at a time (LDS; one step per barrier
// measured 13-18% slower for the LM head and the projections at 128 rows).
// The tile height never changes a row's arithmetic.
template <int NT, int NW, int SW, int MODE, int XS>
hipError_t launch_bf16(const GemmArgs& a, int ngroups, hipStream_t s) {
  const int splits = a.splits;
  const dim3 blk(NW * 64);
  if (a.M <= 16) {
    hipLaunchKernelGGL((gemm_bf16_kernel<1, NT, NW, SW, MODE, XS>), dim3(ngroups, 1, splits), blk, 0, s, a);
  } else if (a.M <= 32) {
    hipLaunchKernelGGL((gemm_bf16_kernel<2, NT, NW, SW, MODE, XS>), dim3(ngroups, 1, splits), blk, 0, s, a);
  } else if (a.M <= 64) {
    hipLaunchKernelGGL((gemm_bf16_kernel<4, NT, NW, SW, MODE, XS>), dim3(ngroups, 1, splits), blk, 0, s, a);
  } else {
    hipLaunchKernelGGL((gemm_bf16_kernel<8, NT, NW, SW, MODE, 2>), dim3(ngroups, (a.M + 127) / 128, splits), blk,
                       0, s, a);
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
    for (int k = 0; k < K; ++k) {
      acc += x[k] * wg[k];
      acc2 += x[k] * wu[k];
    }
    if (ok) ((float*)a.y)[(long long)m * a.ldy + n] = silu(acc) * acc2;
    return;
  }
  int si = 0;
  if (a.nseg > 1 && nc >= a.seg[1].n0) si = 1;
  if (a.nseg > 2 && nc >= a.seg[2].n0) si = 2;
  const float* w = (const float*)a.seg[si].w + (long long)(nc - a.seg[si].n0) * K;
  for (int k = 0; k < K; ++k) acc += x[k] * w[k];
  float* Y = (float*)a.y;
  if (MODE == GEMM_STORE) {
    if (ok) Y[(long long)m * a.ldy + n] = acc;
  } else {
    if (ok) Y[(long long)m * a.ldy + n] = acc;
    // 64 consecutive columns form one wave: its max is that tile's max
    const float v = wave_max(ok ? acc : -INFINITY);
    if ((threadIdx.x & 63) == 0 && ok) a.tilemax[(long long)m * a.ntiles + n / 64] = v;
  }
}

}  // namespace

hipError_t pack_panels(const void* w, int N, int K, int group, void* out, hipStream_t s) {
  if (K % kStep || group < 1) return hipErrorInvalidValue;
  const long long chunks = packed_panels(N, group) * (K / kStep) * 128;
  const int blocks = int(std::min<long long>(8192, (chunks + 255) / 256));
  hipLaunchKernelGGL(pack_panels_kernel, dim3(blocks), dim3(256), 0, s, (const bf16_t*)w, N, K, group, (bf16_t*)out);
  return hipGetLastError();
}

size_t packed_elems(int N, int K, int group) { return (size_t)packed_panels(N, group) * 16 * K; }

int gemm_groups(int mode, int N) {
  switch (mode) {
    case GEMM_SILU: return (N + 31) / 32;     // 2 gate + 2 up panels of 16 features
    case GEMM_LOGITS: return (N + 511) / 512;  // 8 waves x 4 panels
    default: return (N + 127) / 128;          // 8 waves x 1 panel
  }
}

// Launch shapes (panels per wave, waves, weight steps in flight, X steps per
// LDS stage), chosen by measurement at the shapes of an 8B-class layer (the
// split-K factor comes with the call and depends on the shape only):
// * up to 64 rows: split-K projections <1, 8, 4, 2>, SwiGLU <1, 4, 4, 4>;
// * 65-128 rows (one 128-row tile): both <1, 8, 4> (128 columns per
//   workgroup for split-K, 64 output features for SwiGLU);
// * more rows: both <2, 8, 4> (256 columns / 128 features per workgroup: the
//   two 128-row blocks of a column group then stream twice the weights per
//   X stage they load), except split-K projections whose splits cover at most
//   8 steps (the O projection), which keep one panel per wave with two steps
//   in flight <1, 8, 2>;
// * the LM head <4, 8, 2> at every height (512 columns per workgroup: the X
//   rows every workgroup streams through LDS cost half as much per weight
//   byte).
// A row's arithmetic is the same under every shape (same k order, same
// split-K).
namespace {

// a workgroup of `cols` columns never straddles segments
bool segments_aligned(const GemmArgs& a, int cols) {
  for (int i = 1; i < a.nseg; ++i)
    if (a.seg[i].n0 % cols) return false;
  return true;
}
template <int NT, int NW, int SW, int XS>
hipError_t launch_store(const GemmArgs& a, hipStream_t s) {
  constexpr int cols = 16 * NT * NW;
  if (!segments_aligned(a, cols)) return hipErrorInvalidValue;
  return launch_bf16<NT, NW, SW, GEMM_STORE, XS>(a, (a.N + cols - 1) / cols, s);
}
template <int NT, int NW, int SW, int XS>
hipError_t launch_silu(const GemmArgs& a, hipStream_t s) {
  constexpr int feats = 16 * NT * (NW / 2);
  return launch_bf16<NT, NW, SW, GEMM_SILU, XS>(a, (a.N + feats - 1) / feats, s);
}

}  // namespace

hipError_t gemm_bf16(const GemmArgs& a, hipStream_t s) {
  if (a.K % kStep != 0 || a.M < 1 || a.splits < 1 || a.splits > a.K / kStep) return hipErrorInvalidValue;
  const int g = gemm_groups(a.mode, a.N);
  switch (a.mode) {
    case GEMM_STORE:
      // (segments that are not 256-column aligned keep 128-column workgroups)
      // (20.5 against 22.8 us for the O projection at 256 rows)
      if (a.M > 128 && a.K / a.splits <= 8 * kStep) return launch_store<1, 8, 2, 2>(a, s);
      if (a.M > 128 && segments_aligned(a, 256)) return launch_store<2, 8, 4, 2>(a, s);
      return launch_store<1, 8, 4, 2>(a, s);
    case GEMM_SILU:
      if (a.splits != 1) return hipErrorInvalidValue;
      if (a.M > 128) return launch_silu<2, 8, 4, 4>(a, s);
      if (a.M > 64) return launch_silu<1, 8, 4, 4>(a, s);
      return launch_silu<1, 4, 4, 4>(a, s);
    case GEMM_LOGITS:
      if (a.splits != 1 || a.ntiles != g) return hipErrorInvalidValue;
      return launch_bf16<4, 8, 2, GEMM_LOGITS, 1>(a, g, s);
    default:
      return hipErrorInvalidValue;
  }
}

hipError_t gemm_f32(const GemmArgs& a, hipStream_t s) {
  dim3 grid((a.N + 255) / 256, a.M);
  switch (a.mode) {
    case GEMM_STORE:
      hipLaunchKernelGGL(gemm_f32_kernel<GEMM_STORE>, grid, dim3(256), 0, s, a); break;
    case GEMM_SILU:
      hipLaunchKernelGGL(gemm_f32_kernel<GEMM_SILU>, grid, dim3(256), 0, s, a); break;
    default:
      hipLaunchKernelGGL(gemm_f32_kernel<GEMM_LOGITS>, grid, dim3(256), 0, s, a); break;
  }
  return hipGetLastError();
}

}  // namespace rgd
