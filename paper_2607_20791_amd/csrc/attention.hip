// Decode attention over a shared prompt KV plus per-row tails.
//
// The prompt KV of one prompt is read by every row (probe or branch) of that
// prompt.  bf16 path: the shared part is split over (prefix split, KV head,
// row block); a workgroup streams 64-position K/V tiles of its split through
// LDS once and all query vectors of the row block (rows x the G query heads of
// the KV head, up to RGD_ATTN_QV) consume them with MFMA.  Scores are computed
// transposed, S^T = K Q^T, with the K rows gathered so that each lane ends up
// holding eight consecutive positions of one query vector; those feed
// O^T += V^T P^T directly as the B operand, and the V cache is kept
// head-dim-major (transposed per KV head) so that V^T fragments are plain
// 16-byte reads.  Online softmax runs in the exp2 domain with a lazily moved
// exponent reference.  A second kernel attends each row's own paged tail (also
// on MFMA) and merges it with the prefix-split (o, log-sum-exp) partials in a
// fixed order.
//
// fp32 path: vector kernels of the same structure (prefix splits, then tail
// plus merge).
#include <algorithm>
#include <type_traits>

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

// 2^x on the hardware unit, without the denormal range fix-up of exp2f:
// results below 2^-126 flush to zero, far below what a softmax weight in
// bf16 or an fp32 sum of them can resolve.
RGD_DEV float exp2_raw(float x) { return __builtin_amdgcn_exp2f(x); }

// Exponent headroom of the lazy softmax rescale (log2 units).
constexpr float kLazy = 8.f;
// Exponent reference of a query vector with no visible position yet: finite,
// so that s*scale - kNoRef is huge for a visible score and -inf (never NaN)
// for a masked one.
constexpr float kNoRef = -3.0e38f;

#ifndef RGD_ATTN_NW
#define RGD_ATTN_NW 8
#endif
// Fragment reads in flight + 1 in the tile loop's register ring (measured at
// 64 rows: 5 and 7 alike, 3 slower by 0.3 us, 9 and 16 slower still).
#ifndef RGD_ATTN_RING
#define RGD_ATTN_RING 5
#endif

// K tiles sit in LDS as unpadded 256-byte rows whose 16-byte chunks are
// XOR-swizzled: chunk c of row r is stored at chunk c ^ kswz(r).  A fragment
// read touches rows {0..3, 8..11, 16..19, 24..27} (+ a multiple of 4) of a
// 32-row half, and kswz maps those to distinct chunk positions, so the reads
// are free of bank conflicts.
RGD_DEV int kswz(int r) { return (r & 3) | ((r >> 1) & 12); }

// V^T tiles sit in LDS as unpadded 128-byte rows (64 positions of one head
// dimension) whose 16-byte chunks are XOR-swizzled: chunk c of row r is stored
// at chunk c ^ vswz(r).  A fragment read (16 consecutive rows, one chunk each)
// and a tile store (8 lanes per row) are then free of bank conflicts by the
// LDS conflict counter; a padded 144-byte pitch, conflict-free on paper, was
// measured 2-way conflicted on the fragment reads.
RGD_DEV int vswz(int r) { return (r >> 1) & 7; }

// Row of a 64-position tile that lane l16 supplies as the A operand of score
// block (h, e).  With this order the score MFMA leaves lane (q, grp) holding
// positions h*32 + grp*8 + e*4 + {0..3}, i.e. eight consecutive positions per
// 32-position half: exactly the B operand layout of the P V product, and the
// matching V^T fragment is one contiguous 16-byte read.
RGD_DEV int k_gather_row(int h, int e, int l16) { return h * 32 + (l16 >> 2) * 8 + e * 4 + (l16 & 3); }

// Shared-prefix attention: one workgroup per (prefix split, KV head, block of
// up to RGD_ATTN_QV query vectors of one prompt).  The row blocks of one
// (split, KV head) are Hkv * splits workgroups apart in dispatch order, a
// multiple of the 8 XCDs the dispatcher deals workgroups to in turn, so they
// share one XCD's L2 for their common tiles.  NW waves each own NQ MFMA column
// tiles of 16 query vectors, so each K / V^T fragment read from LDS feeds NQ
// MFMAs and each 64-position tile is fetched from HBM once for all rows of the
// prompt.  The tile loop is software-pipelined: tiles are fetched into
// registers one tile ahead and stored into a ring of three LDS buffers, and
// the scores of tile t+1 are computed (MFMA) while the softmax of tile t runs
// on the vector units.  One barrier per tile.
template <int NW, int NQ>
__global__ __launch_bounds__(NW * 64) void attn_prefix_kernel(AttnArgs a) {
  constexpr int D = 128, TP = 64, NT = NW * 64, NB = 3;
  static_assert(NW * NQ * 16 == RGD_ATTN_QV, "a workgroup covers RGD_ATTN_QV query vectors");
  const int s = blockIdx.x, g = blockIdx.y;
  // the row block comes with the arguments
  const int4 rb = a.rblk[blockIdx.z];
  const int r0 = rb.x, nr = rb.y, b = rb.z, maxplen = rb.w;
  const int lo = s * a.split_len;
  const int hi = min(lo + a.split_len, maxplen);
  const int G = a.Hq / a.Hkv;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l16 = lane & 15, grp = lane >> 4;
  const int nq = nr * G;

  // B operand of the score MFMA: lane (q, grp) holds dims ks*32 + grp*8 + {0..7}
  u32x4 qf[NQ][4];
  bool vok[NQ];
  int vrow[NQ], vhead[NQ], vend[NQ];
  // Q fragments first (unconditional loads: a query vector past the block
  // reads row r0 and is zeroed), then the visible ends, whose loads then do
  // not hold up the Q loads
  int pl[NQ];
#pragma unroll
  for (int nt = 0; nt < NQ; ++nt) {
    const int v = wave * NQ * 16 + nt * 16 + l16;
    vok[nt] = v < nq;
    vrow[nt] = r0 + (vok[nt] ? v / G : 0);
    vhead[nt] = g * G + (vok[nt] ? v % G : 0);
    const bf16_t* qp = (const bf16_t*)a.q + ((long long)vrow[nt] * a.Hq + vhead[nt]) * D + grp * 8;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) qf[nt][ks] = *(const u32x4*)(qp + ks * 32);
    pl[nt] = a.rows.plen[vrow[nt]];
  }
  // the visible ends are formed after the prologue's barrier (their loads are
  // long back by then; waiting for them here would hold up the first tile)
  auto set_vend = [&]() {
#pragma unroll
    for (int nt = 0; nt < NQ; ++nt) {
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
        if (!vok[nt]) qf[nt][ks] = u32x4{0u, 0u, 0u, 0u};
      vend[nt] = vok[nt] ? min(prefix_part_end(pl[nt], a.split_len), hi) : lo;
    }
  };
  const bool wave_active = (wave * NQ * 16) < nq;

  __shared__ __attribute__((aligned(16))) bf16_t k_lds[NB][TP * D];
  __shared__ __attribute__((aligned(16))) bf16_t v_lds[NB][D][TP];

  // this (prompt, KV head): K rows [P][D]; V in 64-position blocks [VP/64][D][64]
  const long long bg = (long long)b * a.Hkv + g;
  const bf16_t* kbase = (const bf16_t*)a.kv.prefix_k + bg * a.kv.P * D;
  const bf16_t* vbase = (const bf16_t*)a.kv.prefix_v + bg * a.kv.VP * D;
  const float scale = rsqrtf(float(D)) * kLog2e;

  // m: exponent reference (log2 units) of a query vector; kNoRef until some
  // position of it is visible.  lacc: running sum of its weights, produced by
  // the P V MFMA against an all-ones A operand (every element holds the sum,
  // taken over the same bf16 weights as the output).
  float m[NQ];
  f32x4 o[8][NQ], lacc[NQ];
#pragma unroll
  for (int nt = 0; nt < NQ; ++nt) {
    m[nt] = kNoRef;
    lacc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) o[dt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const u32x4 ones = {0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u};  // bf16 1.0 x 8

  // Register staging of the next tile.  Nothing reads these registers before
  // store_tile, so the loads stay in flight through a whole tile of compute;
  // zeroing of V past the range (whose cache contents are arbitrary) is done
  // at the store.
  constexpr int KSEG = TP * 16 / NT, VSEG = D * (TP / 8) / NT;  // 16-byte segments per thread
  u32x4 kreg[KSEG], vreg[VSEG];
  int vt0 = 0;
  // The loads are unconditional (a predicated load makes the compiler wait
  // for it where the branches join): K rows past the range read row hi - 1
  // (their scores are masked), V of the tile's 64-position block is in the
  // padded cache and is zeroed past the range at the store.
  auto load_tile = [&](int t0) {
    vt0 = t0;
    const bf16_t* vblk = vbase + (long long)(t0 / TP) * D * TP;
#pragma unroll
    for (int i = 0; i < KSEG; ++i) {
      const int seg = threadIdx.x + i * NT;
      const int pos = min(t0 + (seg >> 4), hi - 1);
      kreg[i] = *(const u32x4*)(kbase + (long long)pos * D + (seg & 15) * 8);
    }
#pragma unroll
    for (int i = 0; i < VSEG; ++i) {
      const int seg = threadIdx.x + i * NT;
      vreg[i] = *(const u32x4*)(vblk + (seg >> 3) * TP + (seg & 7) * 8);
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int i = 0; i < KSEG; ++i) {
      const int seg = threadIdx.x + i * NT;
      const int row = seg >> 4;
      *(u32x4*)&k_lds[buf][row * D + (((seg & 15) ^ kswz(row)) * 8)] = kreg[i];
    }
    if (vt0 + TP <= hi) {
#pragma unroll
      for (int i = 0; i < VSEG; ++i) {
        const int seg = threadIdx.x + i * NT, row = seg >> 3;
        *(u32x4*)&v_lds[buf][row][((seg & 7) ^ vswz(row)) * 8] = vreg[i];
      }
    } else {
#pragma unroll
      for (int i = 0; i < VSEG; ++i) {
        const int seg = threadIdx.x + i * NT, row = seg >> 3;
        const int nv = hi - (vt0 + (seg & 7) * 8);  // valid positions of this segment
        u32x4 vv = vreg[i];
#pragma unroll
        for (int w = 0; w < 4; ++w) vv[w] &= nv >= 2 * w + 2 ? 0xFFFFFFFFu : (nv == 2 * w + 1 ? 0xFFFFu : 0u);
        *(u32x4*)&v_lds[buf][row][((seg & 7) ^ vswz(row)) * 8] = vv;
      }
    }
  };

  // The tile loop works on 32-position halves.  Scores of half hh of the tile
  // in buffer buf: sc[e][nt][i] is position hh*32 + grp*8 + e*4 + i.
  auto k_frag = [&](int buf, int hh, int e, int ks) -> u32x4 {
    const int row = k_gather_row(hh, e, l16);
    return *(const u32x4*)&k_lds[buf][row * D + (((ks * 4 + grp) ^ kswz(row)) * 8)];
  };
  // V^T fragment: lane (l16, grp) reads row dt*16 + l16 at positions hh*32 + grp*8 + {0..7}
  auto v_frag = [&](int buf, int dt, int hh) -> u32x4 {
    const int row = dt * 16 + l16;
    return *(const u32x4*)&v_lds[buf][row][((hh * 4 + grp) ^ vswz(row)) * 8];
  };
  auto scores = [&](int buf, int hh, f32x4 (&sc)[2][NQ]) {
#pragma unroll
    for (int e = 0; e < 2; ++e) {
#pragma unroll
      for (int nt = 0; nt < NQ; ++nt) sc[e][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const u32x4 ka = k_frag(buf, hh, e, ks);
#pragma unroll
        for (int nt = 0; nt < NQ; ++nt) sc[e][nt] = mfma16x16x32(ka, qf[nt][ks], sc[e][nt]);
      }
    }
  };

  // Masking, exponent arguments and the exponent reference of a half starting
  // at position p0; on return sc holds the base-2 exponents s*scale - m.
  // Positions past a query vector's end are masked (skipped when the half is
  // visible to every query vector of the wave).  Lazy rescaling: the
  // reference m of a query vector only moves when some score exceeds it by
  // more than kLazy, so weights stay below 2^kLazy and the accumulators are
  // rescaled on few halves.  The common path needs no cross-lane reduction:
  // each lane tests its own exponents (results of arithmetic, so their
  // maximum needs no NaN quieting), and only when some lane of the wave fails
  // are the raw maxima reduced over the four lane groups that share a query
  // vector.  A vector with no visible position yet has m = kNoRef: its
  // exponents are huge (a move) for visible scores and -inf for masked ones.
  auto prepare = [&](int p0, f32x4 (&sc)[2][NQ]) {
    bool full = true;
#pragma unroll
    for (int nt = 0; nt < NQ; ++nt) full &= p0 + 32 <= vend[nt];
    if (!__all(full)) {
#pragma unroll
      for (int nt = 0; nt < NQ; ++nt)
#pragma unroll
        for (int e = 0; e < 2; ++e)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (p0 + grp * 8 + e * 4 + i >= vend[nt]) sc[e][nt][i] = -INFINITY;
    }
    f32x4 t[2][NQ];
    bool grow = false;
#pragma unroll
    for (int nt = 0; nt < NQ; ++nt) {
#pragma unroll
      for (int e = 0; e < 2; ++e)
#pragma unroll
        for (int i = 0; i < 4; ++i) t[e][nt][i] = fmaf(sc[e][nt][i], scale, -m[nt]);
      const float x = fmaxf(fmaxf(fmaxf(t[0][nt][0], t[0][nt][1]), fmaxf(t[0][nt][2], t[0][nt][3])),
                            fmaxf(fmaxf(t[1][nt][0], t[1][nt][1]), fmaxf(t[1][nt][2], t[1][nt][3])));
      grow |= x > kLazy;
    }
    if (__any(grow)) {
#pragma unroll
      for (int nt = 0; nt < NQ; ++nt) {
        float x = fmaxf(fmaxf(fmaxf(sc[0][nt][0], sc[0][nt][1]), fmaxf(sc[0][nt][2], sc[0][nt][3])),
                        fmaxf(fmaxf(sc[1][nt][0], sc[1][nt][1]), fmaxf(sc[1][nt][2], sc[1][nt][3]))) * scale;
        x = fmaxf(x, __shfl_xor(x, 16, 64));
        x = fmaxf(x, __shfl_xor(x, 32, 64));
        // only a query vector whose own maximum passed its reference by more
        // than kLazy moves: its arithmetic never depends on the other query
        // vectors of the wave (rows batched together give the same results)
        if (x > m[nt] + kLazy) {
          const float alpha = exp2_raw(m[nt] - x);  // 0 when moving from kNoRef
          lacc[nt] *= alpha;
#pragma unroll
          for (int dt = 0; dt < 8; ++dt) o[dt][nt] *= alpha;
          m[nt] = x;
#pragma unroll
          for (int e = 0; e < 2; ++e)
#pragma unroll
            for (int i = 0; i < 4; ++i) t[e][nt][i] = fmaf(sc[e][nt][i], scale, -x);
        }
      }
    }
#pragma unroll
    for (int nt = 0; nt < NQ; ++nt) {
      sc[0][nt] = t[0][nt];
      sc[1][nt] = t[1][nt];
    }
  };

  // One straight-line stream per half: the scores of the following half
  // (buffer kb, half kh, into nxt), the exponentials of this half (cur)
  // interleaved with them, then this half's P V product (buffer vb, half vh).
  // The 16 fragment reads go through a register ring of RD slots, NQ MFMAs
  // each; the caller primes the ring before the half's softmax preparation so
  // that those reads overlap it, and every step ends in a scheduling barrier,
  // so that the reads stay RD - 1 steps ahead of their MFMAs as written (left
  // alone, the scheduler moves each read next to its use and the MFMAs wait
  // for LDS).  The two score blocks alternate, so consecutive score MFMAs are
  // independent.  After the last half kb holds stale data and nxt is simply
  // not used.
  constexpr int RD = RGD_ATTN_RING;  // fragment reads in flight + 1
  auto frag = [&](int kb, int kh, int vb, int vh, int f) -> u32x4 {
    return f < 8 ? k_frag(kb, kh, f & 1, f >> 1) : v_frag(vb, f - 8, vh);
  };
  auto prime = [&](int kb, int kh, int vb, int vh, u32x4 (&ring)[RD]) {
#pragma unroll
    for (int f = 0; f + 1 < RD; ++f) ring[f] = frag(kb, kh, vb, vh, f);
  };
  auto stream = [&](int kb, int kh, int vb, int vh, f32x4 (&cur)[2][NQ], f32x4 (&nxt)[2][NQ], u32x4 (&ring)[RD]) {
    float plo[NQ];
    uint32_t pw[NQ][4];  // packed weights, word 2e + (i >> 1)
#pragma unroll
    for (int f = 0; f < 16; ++f) {
      if (f + RD - 1 < 16) ring[(f + RD - 1) % RD] = frag(kb, kh, vb, vh, f + RD - 1);
      if (f < 8) {
        const int e = f & 1, ks = f >> 1;
        if (ks == 0) {
#pragma unroll
          for (int nt = 0; nt < NQ; ++nt) nxt[e][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int nt = 0; nt < NQ; ++nt) nxt[e][nt] = mfma16x16x32(ring[f % RD], qf[nt][ks], nxt[e][nt]);
        // step f exponentiates value i = f & 3 of block ce = f >> 2 of this
        // half; pairs are packed to bf16 as soon as both halves exist
        const int ce = f >> 2, i = f & 3;
#pragma unroll
        for (int nt = 0; nt < NQ; ++nt) {
          const float x = exp2_raw(cur[ce][nt][i]);
          if (i & 1) pw[nt][ce * 2 + (i >> 1)] = pack2(plo[nt], x);
          else plo[nt] = x;
        }
      } else {
        const int dt = f - 8;
#pragma unroll
        for (int nt = 0; nt < NQ; ++nt)
          o[dt][nt] = mfma16x16x32(ring[f % RD], u32x4{pw[nt][0], pw[nt][1], pw[nt][2], pw[nt][3]}, o[dt][nt]);
        if (dt == 7) {
#pragma unroll
          for (int n2 = 0; n2 < NQ; ++n2)
            lacc[n2] = mfma16x16x32(ones, u32x4{pw[n2][0], pw[n2][1], pw[n2][2], pw[n2][3]}, lacc[n2]);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  const int ntile = hi > lo ? (hi - lo + TP - 1) / TP : 0;
  // The loop is reached only through the prologue, whose first store waits for
  // every earlier load (the Q fragments included), so no wait for them is
  // needed inside the loop.
  if (ntile > 0) {
    load_tile(lo);
    store_tile(0);
    if (ntile > 1) load_tile(lo + TP);
    __syncthreads();
    set_vend();
    f32x4 sa[2][NQ], sb[2][NQ];
    if (wave_active) scores(0, 0, sa);
    // tile t uses ring buffer t % NB; the loop is unrolled by NB so that every
    // buffer index is a constant (LDS offsets fold into the instructions)
    auto tile = [&](int t, auto cbc) {
      constexpr int cb = decltype(cbc)::value, nb = (cb + 1) % NB;
      const int t0 = lo + t * TP;
      if (t + 1 < ntile) {  // publish tile t+1
        store_tile(nb);
        if (t + 2 < ntile) load_tile(t0 + 2 * TP);
      }
      __syncthreads();
      if (wave_active) {
        u32x4 ring[RD];
        prime(cb, 1, cb, 0, ring);
        prepare(t0, sa);
        stream(cb, 1, cb, 0, sa, sb, ring);
        prime(nb, 0, cb, 1, ring);
        prepare(t0 + 32, sb);
        stream(nb, 0, cb, 1, sb, sa, ring);
      }
    };
    static_assert(NB == 3, "the tile loop is unrolled by the number of LDS tile buffers");
    for (int t = 0; t < ntile; t += NB) {
      tile(t, std::integral_constant<int, 0>{});
      if (t + 1 < ntile) tile(t + 1, std::integral_constant<int, 1>{});
      if (t + 2 < ntile) tile(t + 2, std::integral_constant<int, 2>{});
    }
  }

#pragma unroll
  for (int nt = 0; nt < NQ; ++nt) {
    const float lt = lacc[nt][0];
    if (vok[nt]) {
      const long long idx = ((long long)s * a.rows.R + vrow[nt]) * a.Hq + vhead[nt];
      // normalised partial output, stored in bf16 (bounded by max|V|; the
      // merged output is bf16 as well)
      bf16_t* po = (bf16_t*)a.part_o + idx * D;
      const float inv = lt > 0.f ? 1.0f / lt : 0.f;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt)
        *(u32x2*)(po + dt * 16 + grp * 4) = u32x2{pack2(o[dt][nt][0] * inv, o[dt][nt][1] * inv),
                                                  pack2(o[dt][nt][2] * inv, o[dt][nt][3] * inv)};
      if (grp == 0) a.part_lse[idx] = lt > 0.f ? (m[nt] + __log2f(lt)) * kLn2 : -INFINITY;
    }
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

  const long long bg = (long long)a.rows.prompt[r] * a.Hkv + g;
  auto k_row = [&](int pos) -> const T* {
    if (PREFIX) return (const T*)a.kv.prefix_k + (bg * a.kv.P + pos) * D;
    const int ps = a.kv.page_size;
    const int page = a.rows.pages[(long long)r * a.rows.max_pages + pos / ps];
    return (const T*)a.kv.pool_k + (((long long)page * a.Hkv + g) * ps + pos % ps) * D;
  };
  auto v_at = [&](int pos, int d) -> float {
    if (PREFIX)
      return load_f((const T*)a.kv.prefix_v + ((bg * (a.kv.VP / 64) + pos / 64) * D + d) * 64 + pos % 64);
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
      const T* kr = (const T*)a.kv.pool_k + (((long long)pages[pos / ps] * a.Hkv + g) * ps + pos % ps) * D;
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

// Tail attention fused with the merge, bf16 caches: one workgroup of four
// waves per (row, KV head).  Each wave attends 32-position tiles of the row's
// paged tail (tiles wave, wave+4, ...) with MFMA: the G query heads of the KV
// head form one 16-column tile, K and V^T fragments are loaded straight from
// the pages (K rows in the gathered order of the prefix kernel, so every lane
// ends up with eight consecutive positions).  The four waves' tail states are
// merged through LDS, and wave h writes query head h's output.  The merge is
// in log-sum-exp form with a fixed split order; for the wave's first head the
// prefix-split partials are combined into one while the wave's first tile is
// loading, which leaves a two-term merge with the tail after the exchange.
constexpr int kMergeMaxSplits = 64;

__global__ __launch_bounds__(256) void attn_tail_merge_kernel(AttnArgs a, bf16_t* out) {
  constexpr int D = 128, TT = 32;
  const int r = blockIdx.x, g = blockIdx.y;
  const int G = a.Hq / a.Hkv;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l16 = lane & 15, grp = lane >> 4;
  const long long R = a.rows.R;
  const int ps = a.kv.page_size;
  const float scale = rsqrtf(float(D)) * kLog2e;

  __shared__ float w_m[4][16], w_l[4][16];
  __shared__ __attribute__((aligned(16))) float w_o[4][16][D + 4];  // [wave][query][dim]

  // First requests: the row's visible prefix length and its first 64 tail
  // page numbers (lane i holds page i), so that tile addresses need no
  // further dependent load.  Without tail pages a valid int array stands in.
  const int n = a.tail_len;
  const int* prow = n > 0 ? a.rows.pages + (long long)r * a.rows.max_pages : a.rows.plen;
  const int plen = a.rows.plen[r];
  const int pg_reg = prow[n > 0 ? min(lane, a.rows.max_pages - 1) : 0];
  const int ps_ = a.kv.page_size;
  const bool pg_in_regs = (n + ps_ - 1) / ps_ <= 64;  // uniform
  auto page_at = [&](int pi) -> int {
    return pg_in_regs ? __shfl(pg_reg, pi, 64) : prow[min(pi, a.rows.max_pages - 1)];
  };
  const int prompt = a.rows.prompt[r];

  // The prefix-split partials and log-sum-exps do not depend on the tail:
  // request those of this wave's first head now so their latency overlaps the
  // tail attention (splits beyond kPrefetch are loaded by the combine).
  const int S = a.splits;
  constexpr int kPrefetch = 16;
  const long long pstep = R * a.Hq * D;
  // (Loads in this kernel are unconditional, from clamped addresses, and
  // masked afterwards: a predicated load makes the compiler wait for it where
  // the branches join, one memory round trip each.)
  // (a wave past the G heads loads head G-1's and does not use them)
  uint32_t pre[kPrefetch];  // bf16 pairs
  float pre_lse;
  {
    const int head = g * G + min(wave, G - 1);
    const bf16_t* po = (const bf16_t*)a.part_o + ((long long)r * a.Hq + head) * D + 2 * lane;
#pragma unroll
    for (int k = 0; k < kPrefetch; ++k) pre[k] = *(const uint32_t*)(po + min(k, S - 1) * pstep);
    const float ls = a.part_lse[((long long)min(lane, S - 1) * R + r) * a.Hq + head];
    pre_lse = lane < S ? ls : -INFINITY;
  }

  u32x4 qf[4];
  {
    const bool ok = l16 < G;
    const bf16_t* qp = (const bf16_t*)a.q + ((long long)r * a.Hq + g * G + (ok ? l16 : 0)) * D + grp * 8;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const u32x4 x = *(const u32x4*)(qp + ks * 32);
      qf[ks] = ok ? x : u32x4{0u, 0u, 0u, 0u};
    }
  }
  float m = -INFINITY, lsum = 0.f;
  f32x4 o[8];
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  // The prefix splits of this wave's first head combined into one partial
  // (natural-log log-sum-exp s_lse, normalised output s_o0 / s_o1 for dims
  // 2*lane, 2*lane+1), in fixed split order.  It needs no tail data, so it is
  // formed while the first tile's loads are in flight.
  float s_lse = -INFINITY, s_o0 = 0.f, s_o1 = 0.f;
  auto combine_splits = [&]() {
    const int head = g * G + min(wave, G - 1);
    float mx = pre_lse;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
    const float w = pre_lse == -INFINITY ? 0.f : __expf(pre_lse - mx);
    float den = w;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) den += __shfl_xor(den, off, 64);
    const float inv = den > 0.f ? 1.f / den : 0.f;
    const bf16_t* po = (const bf16_t*)a.part_o + ((long long)r * a.Hq + head) * D + 2 * lane;
    float o0 = 0.f, o1 = 0.f;
    // weight of split sp sits in lane sp
#pragma unroll
    for (int k = 0; k < kPrefetch; ++k) {
      if (k < S) {
        const float wk = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w), k)) * inv;
        o0 += wk * __uint_as_float(pre[k] << 16);
        o1 += wk * __uint_as_float(pre[k] & 0xFFFF0000u);
      }
    }
#pragma unroll 1
    for (int k = kPrefetch; k < S; ++k) {  // splits past the prefetched ones (long prompts)
      const uint32_t v = *(const uint32_t*)(po + k * pstep);
      const float wk = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w), k)) * inv;
      o0 += wk * __uint_as_float(v << 16);
      o1 += wk * __uint_as_float(v & 0xFFFF0000u);
    }
    s_lse = den > 0.f ? mx + __logf(den) : -INFINITY;
    s_o0 = o0;
    s_o1 = o1;
  };
  bool combined = false;
  // the row's own positions: first its prefix positions the split kernel left
  // (fewer than 64 past a split boundary, read in place from the shared
  // prefix), then its paged tail; 32-position tiles of either, dealt to the
  // four waves in turn
  const int pe = prefix_part_end(plen, a.split_len);
  const int n_ovt = (plen - pe + TT - 1) / TT, n_all = n_ovt + (n + TT - 1) / TT;
  const long long bg = (long long)prompt * a.Hkv + g;
  const bf16_t* pk = (const bf16_t*)a.kv.prefix_k + bg * a.kv.P * D;
  const bf16_t* pv = (const bf16_t*)a.kv.prefix_v + bg * a.kv.VP * D;
  for (int vt = wave; vt < n_all; vt += 4) {
    const bool ov = vt < n_ovt;
    const int tb = ov ? pe + vt * TT : (vt - n_ovt) * TT;  // first position of the tile
    const int lim = ov ? plen : n;                          // positions < lim exist
    // every address of the tile first (page numbers come from registers),
    // then all its loads back to back
    int kp[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int pos = tb + k_gather_row(0, e, l16);
      kp[e] = pos < lim ? pos : tb;
    }
    // this lane's eight positions p0 .. p0+7 lie in one page (ps % 8 == 0) or
    // one 64-position block of the prefix V layout (p0 % 8 == 0)
    const int p0 = tb + grp * 8;
    const int nv = lim - p0;
    const int vp = nv > 0 ? p0 : tb;
    const int kpg0 = page_at(ov ? 0 : kp[0] / ps), kpg1 = page_at(ov ? 0 : kp[1] / ps);
    const int vpg = page_at(ov ? 0 : vp / ps);
    const bf16_t* kr[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int pg = e ? kpg1 : kpg0;
      kr[e] = ov ? pk + (long long)kp[e] * D + grp * 8
                 : (const bf16_t*)a.kv.pool_k + (((long long)pg * a.Hkv + g) * ps + kp[e] % ps) * D + grp * 8;
    }
    const bf16_t* vr = ov ? pv + ((long long)(vp / 64) * D + l16) * 64 + vp % 64
                          : (const bf16_t*)a.kv.pool_v + (((long long)vpg * a.Hkv + g) * D + l16) * ps + vp % ps;
    const long long vstep = ov ? 16LL * 64 : 16LL * ps;  // 16 head-dim rows
    u32x4 ka[2][4], va[8];
#pragma unroll
    for (int e = 0; e < 2; ++e)
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) ka[e][ks] = *(const u32x4*)(kr[e] + ks * 32);  // past the end: masked scores
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) va[dt] = *(const u32x4*)(vr + dt * vstep);  // past the end: zeroed below
    if (!combined) {  // uniform: the first tile of the wave
      combine_splits();
      combined = true;
    }
    f32x4 sc[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      sc[e] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) sc[e] = mfma16x16x32(ka[e][ks], qf[ks], sc[e]);
    }
    float x = -INFINITY;
#pragma unroll
    for (int e = 0; e < 2; ++e)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (p0 + e * 4 + i >= lim) sc[e][i] = -INFINITY;
        x = fmaxf(x, sc[e][i]);
      }
    x = fmaxf(x, __shfl_xor(x, 16, 64));
    x = fmaxf(x, __shfl_xor(x, 32, 64));
    x *= scale;
    if (x > m) {
      const float alpha = exp2_raw(m - x);
      lsum *= alpha;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) o[dt] *= alpha;
      m = x;
    }
    const float msub = m == -INFINITY ? INFINITY : m;
    float p[8];
#pragma unroll
    for (int e = 0; e < 2; ++e)
#pragma unroll
      for (int i = 0; i < 4; ++i) p[e * 4 + i] = exp2_raw(fmaf(sc[e][i], scale, -msub));
#pragma unroll
    for (int i = 0; i < 8; ++i) lsum += p[i];
    const u32x4 pb = {pack2(p[0], p[1]), pack2(p[2], p[3]), pack2(p[4], p[5]), pack2(p[6], p[7])};
    if (nv < 8) {  // V past the row's end is arbitrary (unwritten slots): zero it
#pragma unroll
      for (int dt = 0; dt < 8; ++dt)
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          if (2 * w >= nv) va[dt][w] = 0u;
          else if (2 * w + 1 >= nv) va[dt][w] &= 0xFFFFu;
        }
    }
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) o[dt] = mfma16x16x32(va[dt], pb, o[dt]);
  }
  if (!combined) combine_splits();
  // per-wave tail states -> LDS (query q = l16, dims dt*16 + grp*4 + i)
  lsum += __shfl_xor(lsum, 16, 64);
  lsum += __shfl_xor(lsum, 32, 64);
  if (grp == 0) {
    w_m[wave][l16] = m;
    w_l[wave][l16] = lsum;
  }
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) *(f32x4*)&w_o[wave][l16][dt * 16 + grp * 4] = o[dt];
  __syncthreads();

  // merge: wave h handles query heads h, h+4, ...; lane holds dims 2*lane, 2*lane+1
  auto finish = [&](int h, bool first) {
    const int head = g * G + h;
    // tail state of this head (exp2 domain) from the four waves
    float tm = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) tm = fmaxf(tm, w_m[w][h]);
    float tl = 0.f, to0 = 0.f, to1 = 0.f;
    if (tm != -INFINITY) {
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const float f = exp2_raw(w_m[w][h] - tm);
        tl += f * w_l[w][h];
        to0 += f * w_o[w][h][2 * lane];
        to1 += f * w_o[w][h][2 * lane + 1];
      }
    }
    const float tail_lse = tl > 0.f ? (tm + __log2f(tl)) * kLn2 : -INFINITY;
    if (first) {  // the prefix splits are combined already: two partials left
      const float mx = fmaxf(s_lse, tail_lse);
      const float ws = s_lse == -INFINITY ? 0.f : __expf(s_lse - mx);
      const float wt = tail_lse == -INFINITY ? 0.f : __expf(tail_lse - mx);
      const float den = ws + wt;
      const float inv = den > 0.f ? 1.f / den : 0.f;
      const float ft = tl > 0.f ? wt * inv / tl : 0.f;  // applied to the unnormalised tail sum
      const float fs = ws * inv;
      *(uint32_t*)(out + ((long long)r * a.Hq + head) * D + 2 * lane) =
          pack_bf16x2(fs * s_o0 + ft * to0, fs * s_o1 + ft * to1);
      return;
    }
    // further heads (G > 4): split log-sum-exps, lane sp holds split sp's
    const float ls = lane < S ? a.part_lse[((long long)lane * R + r) * a.Hq + head] : -INFINITY;
    float mx = fmaxf(ls, tail_lse);
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
    const float w = ls == -INFINITY ? 0.f : __expf(ls - mx);
    const float wt = tail_lse == -INFINITY ? 0.f : __expf(tail_lse - mx);
    float den = w;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) den += __shfl_xor(den, off, 64);
    den += wt;
    const float inv = den > 0.f ? 1.f / den : 0.f;
    const float ft = tl > 0.f ? wt * inv / tl : 0.f;  // applied to the unnormalised tail sum
    float o0 = ft * to0, o1 = ft * to1;
    const bf16_t* po = (const bf16_t*)a.part_o + ((long long)r * a.Hq + head) * D + 2 * lane;
    // weight of split sp sits in lane sp; fixed split order
#pragma unroll
    for (int k = 0; k < kMergeMaxSplits; ++k) {
      if (k < S) {
        const uint32_t v = *(const uint32_t*)(po + k * pstep);
        const float wk = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w), k)) * inv;
        o0 += wk * __uint_as_float(v << 16);
        o1 += wk * __uint_as_float(v & 0xFFFF0000u);
      }
    }
    *(uint32_t*)(out + ((long long)r * a.Hq + head) * D + 2 * lane) = pack_bf16x2(o0, o1);
  };
  // the first head of the wave uses the combined prefix partial
  if (wave < G) finish(wave, true);
  for (int h = wave + 4; h < G; h += 4) finish(h, false);
}

}  // namespace

hipError_t attn_prefix_bf16(const AttnArgs& a, hipStream_t s) {
  if (a.D != 128 || a.Hq / a.Hkv > RGD_ATTN_QV || a.split_len % 64 || a.kv.VP % 64) return hipErrorInvalidValue;
  if (a.splits <= 0 || a.nrblocks <= 0) return hipSuccess;
  if (!a.rblocks) return hipErrorInvalidValue;
  // one launch per kAttnInlineBlocks row blocks
  for (int c0 = 0; c0 < a.nrblocks; c0 += kAttnInlineBlocks) {
    AttnArgs b = a;
    const int n = std::min(kAttnInlineBlocks, a.nrblocks - c0);
    for (int i = 0; i < n; ++i) b.rblk[i] = a.rblocks[c0 + i];
    hipLaunchKernelGGL((attn_prefix_kernel<RGD_ATTN_NW, RGD_ATTN_QV / 16 / RGD_ATTN_NW>), dim3(a.splits, a.Hkv, n),
                       dim3(RGD_ATTN_NW * 64), 0, s, b);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

template <typename T>
hipError_t attn_prefix_vec(const AttnArgs& a, hipStream_t s) {
  if (a.D > 256 || a.Hq / a.Hkv > 8 || a.split_len > kChunk) return hipErrorInvalidValue;
  if (a.splits <= 0) return hipSuccess;
  hipLaunchKernelGGL((attn_vec_kernel<T, true>), dim3(a.splits, a.Hkv, a.rows.R), dim3(256), 0, s, a);
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

hipError_t attn_tail_merge_bf16(const AttnArgs& a, bf16_t* out, hipStream_t s) {
  if (a.D != 128 || a.Hq / a.Hkv > 16 || a.splits > kMergeMaxSplits || a.splits < 1 ||
      (a.tail_len > 0 && (!a.rows.pages || a.kv.page_size % 8)))
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(attn_tail_merge_kernel, dim3(a.rows.R, a.Hkv), dim3(256), 0, s, a, out);
  return hipGetLastError();
}

template hipError_t attn_prefix_vec<float>(const AttnArgs&, hipStream_t);
template hipError_t attn_prefix_vec<bf16_t>(const AttnArgs&, hipStream_t);
template hipError_t attn_tail_combine<float>(const AttnArgs&, float*, hipStream_t);

}  // namespace rgd
