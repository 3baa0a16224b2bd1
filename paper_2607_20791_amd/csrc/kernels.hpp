// Launch interface of the HIP kernels (internal; not part of the C ABI).
#pragma once
#include "common.hpp"

namespace rgd {

// ---------------------------------------------------------------- GEMM ----
// Y = X W^T with X [M][K] (row stride ldx) and W [N][K] row-major, possibly
// given as up to three row segments (for the fused Q/K/V projection).
struct GemmSeg {
  const void* w;   // [n][K]
  int n0, n;       // output columns [n0, n0 + n)
};

enum GemmMode {
  GEMM_STORE = 0,   // fp32 Y[split][M][N] = X W^T over the split's K range
  GEMM_SILU = 2,    // dual weights (gate = seg 0, up = seg 1): out_T[M][N] = silu(g) * u
  GEMM_LOGITS = 3,  // fp32 Y[M][N] plus one maximum per (row, column group)
};

struct GemmArgs {
  const void* x; int ldx; int M;
  GemmSeg seg[3]; int nseg;
  int N, K;
  int splits;             // split-K factor (GEMM_STORE); 1 otherwise
  void* y; int ldy;       // output (fp32, or T for GEMM_SILU)
  long long split_stride; // elements between split partials
  float* tilemax; int ntiles;  // GEMM_LOGITS: [M][ntiles]
  // GEMM_LOGITS, optional [M][ntiles]: per workgroup tile the packed argmax
  // key (ordered value << 32 | ~index: larger value, then lower index, wins)
  unsigned long long* tilekey;
  int mode;
};

// bf16 weights are used in the packed panel layout (see gemm.hip); the LM
// head's panels are interleaved step by step in groups of kHeadGroup (the
// panels one wave of its GEMM owns), the other matrices' are not (group 1).
constexpr int kHeadGroup = 4;
hipError_t pack_panels(const void* w, int N, int K, int group, void* out, hipStream_t s);
size_t packed_elems(int N, int K, int group);
int gemm_groups(int mode, int N);   // workgroups along N for a mode
hipError_t gemm_bf16(const GemmArgs& a, hipStream_t s);
hipError_t gemm_f32(const GemmArgs& a, hipStream_t s);

// ------------------------------------------------------- row bookkeeping ----
// Rows of one decode step (or one prefill segment).
struct Rows {
  int R;
  const int* prompt;    // [R] prompt index (selects the shared prefix)
  const int* base_pos;  // [R] position of tail slot 0 (decode) or of the token (prefill)
  const int* plen;      // [R] prefix positions this row attends to
  const int* pages;     // [R][max_pages] tail pages (decode) or null
  int max_pages;
  int t;                // tail slot written this step (decode)
  int prefill;          // 1: K/V go to the prefix at base_pos; no tail
};

// Caches are KV-head-major so that a tile of consecutive positions of one head
// is one contiguous run; V is stored transposed (head dim before position) in
// blocks of 64 positions so that attention's V^T operand tile is a plain copy.
struct KVLayout {
  void* prefix_k;  // this layer: [B][Hkv][P][D]
  void* prefix_v;  // this layer: [B][Hkv][VP/64][D][64]
  void* pool_k;    // this layer: [pages][Hkv][page_size][D]
  void* pool_v;    // this layer: [pages][Hkv][D][page_size]
  int P;           // prefix capacity per prompt
  int VP;          // P rounded up to a multiple of 64
  int page_size;
  int split_len;   // positions per prefix split of the bf16 attention (fixed per KV state)
};

inline int v_stride(int P) { return (P + 63) / 64 * 64; }

// bf16 attention: the prefix positions of a row attended by the prefix-split
// kernel are [0, end); when a row's prefix passes a split boundary by fewer
// than 64 positions, those last positions [end, plen) are attended by the
// tail kernel instead (read in place from the prefix), so that no split holds
// a nearly empty 64-position tile.  A function of the row's own length and the
// KV state's split length only.
__host__ __device__ inline int prefix_part_end(int plen, int split_len) {
  const int rem = plen % split_len;
  return (plen >= split_len && rem < 64) ? plen - rem : plen;
}

// ------------------------------------------------------------ elementwise ----
// x[r] = E[tok[i * tok_stride]] with i = tok_map[r] (tok_map null: i = r), ids
// clamped to [0, V); xn[r] = rmsnorm(x[r]) * g
template <typename T>
hipError_t embed_rmsnorm(const int* tok, int tok_stride, const int* tok_map, int R, const T* E, int d, int V,
                         float* x, const float* g, float eps, T* xn, hipStream_t s);
// split-K partial outputs a consumer kernel sums (at most)
constexpr int kMaxSplitK = 16;
// x[r] += sum_p parts[p][r] (nparts <= kMaxSplitK); xn[r] = rmsnorm(x[r]) * g
template <typename T>
hipError_t residual_rmsnorm(float* x, const float* parts, int nparts, long long part_stride, const float* g,
                            float eps, int R, int d, T* xn, hipStream_t s);
// q/k/v = sum of nparts split partials [R][(Hq+2Hkv)D] fp32 -> RoPE -> q (T),
// k/v appended to the cache.  rope_cs: [max_pos + 1][D/2] (cos, sin) pairs.
template <typename T>
hipError_t qkv_rope_store(const float* parts, int nparts, long long part_stride, const Rows& rows, int Hq,
                          int Hkv, int D, const float* rope_cs, int max_pos, T* q, const KVLayout& kv,
                          hipStream_t s);

// Residual-stream readout (Appendix A): out[r] = 1 / (1 + exp(-(w . x_r + b)))
// for rows x_r = x + (row0 + r * stride) * d of the fp32 residual stream.
hipError_t residual_readout(const float* x, long long row0, long long stride, int nrows, int d, const float* w,
                            float b, float* out, hipStream_t s);

// -------------------------------------------------------------- attention ----
// Query vectors (rows x the G query heads of one KV head) per workgroup of the
// bf16 shared-prefix attention, and the number of (prefix split, KV head)
// pairs its split length is sized for.  128 query vectors (32 rows of a GQA
// group of 4) and 128 pairs: a 64-row decode step runs 256 workgroups, two
// row blocks per 512-position split of an 8193-position prefix, which halves
// the split partials that 256-vector blocks over 256-position splits write and
// merge.
#ifndef RGD_ATTN_QV
#define RGD_ATTN_QV 128
#endif
#ifndef RGD_ATTN_WGS
#define RGD_ATTN_WGS 128
#endif
constexpr int kAttnInlineBlocks = 64;
struct AttnArgs {
  const void* q;            // [R][Hq][D]
  Rows rows;
  KVLayout kv;
  int Hq, Hkv, D;
  float* part_o;            // [nparts][R][Hq][D], fp32; the bf16 prefix path stores bf16 here
  float* part_lse;          // [nparts][R][Hq]
  int nparts;
  // prefix (shared) part
  // (r0, nr, prompt, maxplen) row blocks of the MFMA path: a host array; the
  // launcher passes them by value, kAttnInlineBlocks per launch (scalar loads
  // of the arguments, no memory round trip before the first Q load)
  const int4* rblocks; int nrblocks;
  int4 rblk[kAttnInlineBlocks];
  int splits; int split_len;          // prefix splits (part index 0..splits-1)
  // tail part
  int tail_len;             // visible tail positions (decode), 0 for prefill
  int tail_chunk; int tail_chunks;    // part index splits .. splits+tail_chunks-1
};
// bf16, head_dim 128: prefix-split partials 0 .. splits-1 on MFMA, row blocks
// of up to RGD_ATTN_QV query vectors of one prompt
hipError_t attn_prefix_bf16(const AttnArgs& a, hipStream_t s);
// bf16, head_dim 128, G <= 16: each row's paged tail on MFMA, merged with the
// prefix-split partials into the final output
hipError_t attn_tail_merge_bf16(const AttnArgs& a, bf16_t* out, hipStream_t s);
template <typename T> hipError_t attn_prefix_vec(const AttnArgs& a, hipStream_t s);
// fp32: attends each row's tail (vector units) and merges it with the
// prefix-split partials 0 .. splits-1 into the final output
template <typename T> hipError_t attn_tail_combine(const AttnArgs& a, T* out, hipStream_t s);

// ---------------------------------------------------------------- sampler ----
hipError_t fill_u32(uint32_t* p, uint32_t v, long long n, hipStream_t s);
// per-chunk maxima of fp32 rows (standalone sampler)
hipError_t chunk_max(const float* z, long long ldz, int R, int V, int chunk, float* cmax, hipStream_t s);
// argmax: packed (value, -index) keys, max over chunks via 64-bit atomics
hipError_t argmax_rows(const float* z, long long ldz, int R, int V, unsigned long long* best, hipStream_t s);
struct SampleArgs {
  const float* z; long long ldz; int R; int V;
  const float* pmax; int npmax;   // [R][npmax] partial maxima; row max = their max
  float T; float p_min;
  int chunk; int nchunks;
  float* chunk_sums;              // [R][nchunks]
  const unsigned long long* seeds;  // [R]
  unsigned int ctr; unsigned int stream;
  int* out; long long out_stride; int out_col;   // token of row r -> out[r*out_stride + out_col]
  int* cur_tok;                   // optional [R] copy of the token (next step's input)
  int* status;                    // device flag: set to 1 on a non-finite row maximum
  // optional: the next decode step's input row of each drawn token, x = E[tok]
  // (fp32 [R][d]) and xn = RMSNorm(x) * gain (model dtype), written by the
  // selecting workgroup (null embed: not fused; needs d % 4 == 0, d <= 4096)
  const void* embed; int embed_bf16; int d; int vocab;
  const float* gain; float eps; float* x; void* xn;
  // optional [R] per-row threshold on w (p-less); null: p_min for every row
  const float* row_thr;
  // optional [R][nchunks * 16] kept sums of the 256-logit sub-chunks (decode
  // path, nchunks * 16 <= 1024): written by the sum pass, located by one wave
  // of the draw, which then rescans one sub-chunk instead of a whole chunk
  float* sub_sums;
};
hipError_t minp_sample(const SampleArgs& a, hipStream_t s);
// rows without producer maxima: chunk maxima into cmax [R][nchunks] and the
// chunk sums in one read of the logits (plus rereads of chunks whose maximum
// is within the min-p window of the row maximum), then the draw
hipError_t minp_sample_standalone(const SampleArgs& a, float* cmax, hipStream_t s);
// p-less truncation: chunk statistics into stats [3][R][nchunks] (maxima, sum
// of w, sum of w^2 relative to the chunk maximum), the per-row threshold into
// thr [R], the chunk kept sums, then the draw (chunk == 4096, V % 4 == 0)
hipError_t pless_sample(const SampleArgs& a, float* stats, float* thr, hipStream_t s);
// many draws per row from precomputed chunk sums (counter (ctr, stream0 + d))
hipError_t minp_multi_draw(const SampleArgs& a, int draws, unsigned int stream0, int* out,
                           hipStream_t s);

// ------------------------------------------------------------------- gate ----
struct GateArgs {
  const unsigned long long* best;  // [R] argmax keys
  const int* row_prompt; int R;
  int* cur_tok;
  int* probe_tokens; int k;        // [B][k]
  int* probe_len; int* event;      // [B]
  const int* offsets; const int* tokens; const int* owner; int n_entries; int min_match;
  int eos;
  unsigned long long* best_reset;  // same as best (cleared after use)
  int all_compatible;              // no refusal table (fixed-length probe): every probe passes
  // no early exit (fixed probe): a probe runs to k tokens or to eos whatever
  // its tokens are; failed[b] remembers an incompatible token and the event is
  // set only when the probe ends (INCOMPAT if it failed, else STOP / MAXLEN)
  int no_early_exit;
  int* failed;                     // [B], cleared by the probe's initialisation
  // optional: the argmax keys come as [R][ntiles] tile keys from the LM-head
  // epilogue (best unused); the row's key is their maximum
  const unsigned long long* tilekeys; int ntiles;
  // optional: the next step's input row of each row, x = E[t] (fp32 [R][d])
  // and xn = RMSNorm(x) * gain, for t = probe_tokens[prompt][feed_col] read
  // after this step's update (what the next step feeds); d % 4 == 0, d <= 4096
  const void* embed; int embed_bf16; int d; int vocab; int feed_col;
  const float* gain; float eps; float* x; void* xn;
};
hipError_t probe_update(const GateArgs& a, hipStream_t s);

// Soft compatibility gate (Appendix C): a probe step whose greedy token would
// make the probe incompatible may instead append the most probable
// compatible token among the K most probable ones, when their probability
// mass (softmax at temperature 1 over the whole vocabulary) reaches rho.
constexpr int kMaxTopK = 32;
struct SoftArgs {
  GateArgs g;                   // best/best_reset unused
  const float* z; long long ldz; int V;   // logits of the step, row r at z + r * ldz
  int chunk, nchunks, K;
  unsigned long long* keys;     // workspace [R][nchunks][K]
  float* cmax; float* csum;     // workspace [R][nchunks]
  float rho; int soft_steps;    // tokens 1..soft_steps are soft steps, later ones hard
};
// one probe step for rows 0..R-1 (a.g.R): chunk pass + decision
hipError_t probe_update_soft(const SoftArgs& a, hipStream_t s);
hipError_t gate_decide(const int* event, int B, int* decision, int* n_miss, int* miss_idx,
                       hipStream_t s);

}  // namespace rgd
