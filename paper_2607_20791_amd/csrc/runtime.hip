// Host runtime behind the C ABI: model / KV / table handles, the page pool of
// per-row tails, the decode step, and the probe, gate and sampling loops of
// refusal-gated decoding (Algorithm 1).
#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "entry.hpp"
#include "kernels.hpp"
#include "rgd.h"

using namespace rgd;

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

#define HIP_OK(expr)                                                                   \
  do {                                                                                 \
    hipError_t e_ = (expr);                                                            \
    if (e_ != hipSuccess)                                                              \
      return fail(RGD_E_HIP, "%s failed: %s", #expr, hipGetErrorString(e_));           \
  } while (0)

#define RGD_TRY(expr)            \
  do {                           \
    int rc_ = (expr);            \
    if (rc_ != RGD_OK) return rc_; \
  } while (0)

inline long long cdiv(long long a, long long b) { return (a + b - 1) / b; }

constexpr int kMaxParts = 40;      // attention partials per row (prefix splits + tail chunks)
constexpr int kVecSplit = 256;     // prefix positions per split of the fp32 attention

// Positions per prefix split of the bf16 attention: a function of the KV
// state's shape only (prompt capacity, prompts, KV heads), never of the rows
// of a step, so the split boundaries a row sees do not depend on the other
// rows.  About RGD_ATTN_WGS (split, KV head) pairs over the prompts (each with
// one workgroup per row block), at most kMaxParts splits: S* splits share the whole 64-position tiles
// of the capacity evenly, and a row's positions past a split boundary by fewer
// than 64 go to the tail kernel (prefix_part_end), so a row never needs more
// than S* splits (an 8193-position prefix: 16 splits of 512, the last position
// with the tail).
int prefix_split_len(int P, int prompts, int Hkv) {
  const long long S = std::min<long long>(kMaxParts, std::max<long long>(1, cdiv(RGD_ATTN_WGS, (long long)std::max(prompts, 1) * Hkv)));
  return (int)(64 * cdiv(std::max(P / 64, 1), S));
}
constexpr int kSampleChunk = 4096; // logits per sampler workgroup
constexpr int kTailChunk = 256;

struct DevBuf {
  void* p = nullptr;
  ~DevBuf() {
    if (p) (void)hipFree(p);
  }
};

}  // namespace

// ------------------------------------------------------------------ handles --
struct rgd_table {
  int n_entries = 0, min_match = 2;
  int* d_offsets = nullptr;
  int* d_tokens = nullptr;
  int* d_owner = nullptr;
  ~rgd_table() {
    if (d_offsets) (void)hipFree(d_offsets);
    if (d_tokens) (void)hipFree(d_tokens);
    if (d_owner) (void)hipFree(d_owner);
  }
};

struct rgd_model {
  rgd_model_config cfg{};
  bool bf16 = false;
  const void* embed = nullptr;
  const float* final_norm = nullptr;
  const void* lm_head = nullptr;
  std::vector<rgd_layer_weights> layers;
  // bf16 matrices repacked into the GEMM panel layout (owned); fp32 models use
  // the caller's matrices directly
  struct Packed {
    void *wq, *wk, *wv, *wo, *w_gate, *w_up, *w_down;
  };
  std::vector<Packed> packed;
  void* lm_head_packed = nullptr;
  int max_rows = 0;
  int part_rows = 0;  // row capacity of the split-K partial buffers
  int nqkv = 0, ntiles = 0, nchunks = 0;
  size_t esz = 4;
  // workspace
  std::vector<void*> allocs;
  float* x = nullptr;
  void* xn = nullptr;
  float* qkv_part = nullptr;
  void* q = nullptr;
  float* part_o = nullptr;
  float* part_lse = nullptr;
  float* rope_cs = nullptr;  // [max_pos + 1][head_dim / 2] (cos, sin)
  void* attn_out = nullptr;
  float* o_part = nullptr;
  void* act = nullptr;
  float* down_part = nullptr;
  float* logits = nullptr;
  float* tilemax = nullptr;
  unsigned long long* tilekey = nullptr;  // [R][ntiles] LM-head argmax keys (bf16 models)
  float* chunk_sums = nullptr;
  float* sub_sums = nullptr;  // [R][nchunks * 16] kept sums of 256-logit sub-chunks
  float* pl_stats = nullptr;  // p-less: chunk maxima, sums of w and w^2 [3][R][nchunks]
  float* pl_thr = nullptr;    // p-less: per-row threshold on w [R]
  unsigned long long* best = nullptr;
  int* cur_tok = nullptr;
  int* status = nullptr;
  int* row_map = nullptr;
  int* probe_fail = nullptr;  // fixed probe: incompatible token seen, per prompt [R]
  unsigned long long* soft_keys = nullptr;  // soft gate: per-chunk top-K keys [R][nchunks][kMaxTopK]
  float* soft_cm = nullptr;                 // soft gate: chunk maxima and sums [2][R][nchunks]
  // per-call row arrays
  int* d_prompt = nullptr;
  int* d_base = nullptr;
  int* d_plen = nullptr;
  int* h_stage = nullptr;  // pinned staging for uploads
  size_t stage_ints = 0;
  hipEvent_t stage_done = nullptr;
  hipEvent_t poll_done = nullptr;  // a probe poll's copy of the events reached host memory
  hipEvent_t sync_done = nullptr;  // marks the end of the queued work for spin_sync
  int* h_events = nullptr;  // pinned host copies: probe events, gate results [2 * max_rows + 1]
  int* d_gate = nullptr;    // gate results on the device: decision [R], n_miss, miss list [R]
  // in-situ timing: event pairs per timed unit
  bool timing = false;
  std::vector<hipEvent_t> tev[RGD_TIMER_COUNT];
  int tused[RGD_TIMER_COUNT] = {0};
  // steps of a sampling call are timed when tstep % tperiod == 0 (tstep = the
  // decode step - 1; the draw from the prompt logits is never timed); outside
  // the sampling loop tstep is 0 and every launch is timed
  int tstep = 0;
  int tperiod = 1;
  // inside the sampling loop one unit is timed per timed step, in turn (unit
  // (tstep / tperiod) % RGD_TIMER_COUNT), so no unit's events sit inside
  // another's timed region
  bool tloop = false;
  ~rgd_model() {
    for (auto& v : tev)
      for (hipEvent_t e : v) (void)hipEventDestroy(e);
    for (void* p : allocs) (void)hipFree(p);
    if (h_stage) (void)hipHostFree(h_stage);
    if (h_events) (void)hipHostFree(h_events);
    if (stage_done) (void)hipEventDestroy(stage_done);
    if (poll_done) (void)hipEventDestroy(poll_done);
    if (sync_done) (void)hipEventDestroy(sync_done);
  }
  template <typename P>
  int alloc(P** out, size_t bytes) {
    void* p = nullptr;
    hipError_t e = hipMalloc(&p, std::max<size_t>(bytes, 256));
    if (e != hipSuccess)
      return fail(e == hipErrorOutOfMemory ? RGD_E_OOM : RGD_E_HIP, "workspace allocation of %zu bytes failed: %s",
                  bytes, hipGetErrorString(e));
    allocs.push_back(p);
    *out = (P*)p;
    return RGD_OK;
  }
};

struct rgd_kv {
  const rgd_model* m = nullptr;
  int max_prompts = 0, max_prefix = 0, n_pages = 0, page_size = 16;
  void *prefix_k = nullptr, *prefix_v = nullptr, *pool_k = nullptr, *pool_v = nullptr;
  std::vector<int> plen;
  std::vector<int> free_pages;
  std::vector<std::vector<int>> probe_pages;  // pages held by each prompt's probe
  bool probe_held = false;
  int max_pages = 0;   // page-table width per row
  int* d_pages = nullptr;
  ~rgd_kv() {
    if (d_pages) (void)hipFree(d_pages);
  }
  KVLayout layer(int l) const {
    const rgd_model_config& c = m->cfg;
    const long long per_pos = (long long)c.n_kv_heads * c.head_dim;
    const long long pre_k = (long long)max_prompts * max_prefix * per_pos * m->esz;
    const long long pre_v = (long long)max_prompts * v_stride(max_prefix) * per_pos * m->esz;
    const long long pool = (long long)n_pages * page_size * per_pos * m->esz;
    KVLayout k;
    k.prefix_k = (char*)prefix_k + l * pre_k;
    k.prefix_v = (char*)prefix_v + l * pre_v;
    k.pool_k = (char*)pool_k + l * pool;
    k.pool_v = (char*)pool_v + l * pool;
    k.P = max_prefix;
    k.VP = v_stride(max_prefix);
    k.split_len = prefix_split_len(max_prefix, max_prompts, m->cfg.n_kv_heads);
    k.page_size = page_size;
    return k;
  }
};

namespace {

// ------------------------------------------------------------- host waits --
// Waits for an event by polling it from this thread.  A blocking wait wakes
// the host some tens of microseconds after the GPU is done, and on the probe's
// polls (the host reads the events, then launches the next step) that time is
// GPU idle time.  Falls back to a blocking wait after a second.
hipError_t spin_wait(hipEvent_t ev) {
  const auto t0 = std::chrono::steady_clock::now();
  for (;;) {
    const hipError_t e = hipEventQuery(ev);
    if (e != hipErrorNotReady) return e;
    if (std::chrono::steady_clock::now() - t0 > std::chrono::seconds(1)) return hipEventSynchronize(ev);
  }
}

// everything queued on s so far is done
hipError_t spin_sync(rgd_model* m, hipStream_t s) {
  const hipError_t e = hipEventRecord(m->sync_done, s);
  return e != hipSuccess ? e : spin_wait(m->sync_done);
}

// ------------------------------------------------------------ timing hooks --
constexpr int kTimerPairs = 8192;  // timed launches kept per unit between reads

struct TimeScope {
  rgd_model* m;
  int unit;
  hipStream_t s;
  bool on;
  TimeScope(rgd_model* m_, int unit_, hipStream_t s_) : m(m_), unit(unit_), s(s_) {
    on = m->timing && m->tstep % m->tperiod == 0 &&
         (!m->tloop || (m->tstep / m->tperiod) % RGD_TIMER_COUNT == unit) &&
         m->tused[unit] < (int)m->tev[unit].size() / 2;
    if (on) (void)hipEventRecord(m->tev[unit][2 * m->tused[unit]], s);
  }
  ~TimeScope() {
    if (on) {
      (void)hipEventRecord(m->tev[unit][2 * m->tused[unit] + 1], s);
      ++m->tused[unit];
    }
  }
};

// ----------------------------------------------------------- upload helper --
// Copies host ints to device through the model's pinned staging buffer.  The
// previous upload is waited for before the buffer is rewritten.
struct Upload {
  int* dst;
  const int* src;
  size_t n;
};

int upload(rgd_model* m, const std::vector<Upload>& ups, hipStream_t s) {
  size_t total = 0;
  for (auto& u : ups) total += u.n;
  if (total > m->stage_ints) return fail(RGD_E_OOM, "upload of %zu ints exceeds staging", total);
  HIP_OK(hipEventSynchronize(m->stage_done));
  size_t off = 0;
  for (auto& u : ups) {
    if (!u.n) continue;
    memcpy(m->h_stage + off, u.src, u.n * sizeof(int));
    HIP_OK(hipMemcpyAsync(u.dst, m->h_stage + off, u.n * sizeof(int), hipMemcpyHostToDevice, s));
    off += u.n;
  }
  HIP_OK(hipEventRecord(m->stage_done, s));
  return RGD_OK;
}


// Host description of the rows of one step.
struct HostRows {
  std::vector<int> prompt, base, plen;
  std::vector<int4> blocks;  // row blocks of one prompt for the MFMA attention path
  int maxplen = 0;
};

// Row blocks of one prompt for the shared-prefix attention kernel: up to
// RGD_ATTN_QV query vectors (rows x G query heads) per block.
void build_blocks(const rgd_model* m, HostRows& h) {
  const int G = m->cfg.n_heads / m->cfg.n_kv_heads;
  const int per = std::max(1, (m->bf16 ? RGD_ATTN_QV : 64) / G);
  h.blocks.clear();
  h.maxplen = 0;
  const int R = (int)h.prompt.size();
  int r = 0;
  while (r < R) {
    const int b = h.prompt[r];
    int e = r;
    int mp = 0;
    while (e < R && h.prompt[e] == b && e - r < per) mp = std::max(mp, h.plen[e++]);
    h.blocks.push_back(make_int4(r, e - r, b, mp));
    h.maxplen = std::max(h.maxplen, mp);
    r = e;
  }
}

int upload_rows(rgd_model* m, const HostRows& h, hipStream_t s) {
  const size_t R = h.prompt.size();
  return upload(m,
                {{m->d_prompt, h.prompt.data(), R},
                 {m->d_base, h.base.data(), R},
                 {m->d_plen, h.plen.data(), R}},
                s);
}

Rows device_rows(const rgd_model* m, const rgd_kv* kv, int R, int t, bool prefill) {
  Rows r;
  r.R = R;
  r.prompt = m->d_prompt;
  r.base_pos = m->d_base;
  r.plen = m->d_plen;
  r.pages = prefill ? nullptr : kv->d_pages;
  r.max_pages = kv ? kv->max_pages : 0;
  r.t = t;
  r.prefill = prefill ? 1 : 0;
  return r;
}

// split-K factor of a bf16 GEMM: a function of its shape only (never of the
// number of rows), so that a row's arithmetic does not depend on which other
// rows share the launch.  The smallest power of two that gives at least 192
// workgroups (three quarters of the CUs) for one 64-row block, at most
// kMaxSplitK, with at least 4 steps of 64 k per split.  Measured with a cold
// cache at 64 rows: the QKV projection (48 column groups) takes 17.0 us with 4
// splits against 18.2 us with 8, and its partial outputs halve; O and down
// (32 groups) stay at 8 splits.
int pick_splits(int groups, int K) {
  int ks = 1;
  while (ks < kMaxSplitK && (long long)groups * ks < 192) ks *= 2;
  while (ks > 1 && K / 64 / ks < 4) ks /= 2;
  return ks;
}


// -------------------------------------------------------------- attention --
int run_attention(rgd_model* m, const KVLayout& kvl, const Rows& rows, const HostRows& h,
                  int tail_len, int force_splits, void* out, hipStream_t s) {
  const rgd_model_config& c = m->cfg;
  AttnArgs a{};
  a.q = m->q;
  a.rows = rows;
  a.kv = kvl;
  a.Hq = c.n_heads;
  a.Hkv = c.n_kv_heads;
  a.D = c.head_dim;
  a.part_o = m->part_o;
  a.part_lse = m->part_lse;
  a.rblocks = h.blocks.data();
  a.nrblocks = (int)h.blocks.size();
  a.tail_len = tail_len;
  a.tail_chunk = kTailChunk;
  a.tail_chunks = 0;  // tails are attended inside the merge kernel
  const int R = rows.R;
  const int cap = kMaxParts;  // the partial buffers hold kMaxParts x max_rows rows
  if (m->bf16) {
    if (force_splits > 0) {  // kernel-level entry point: an explicit split count
      const int S = (int)std::max<long long>(1, std::min<long long>(force_splits, cdiv(std::max(h.maxplen, 1), 64)));
      a.split_len = (int)cdiv(cdiv(std::max(h.maxplen, 1), S), 64) * 64;
    } else {
      a.split_len = kvl.split_len;
    }
    // splits up to the longest row's prefix-kernel part (the rest of a row's
    // prefix, fewer than 64 positions past a split boundary, is attended with
    // its tail)
    int pe = 1;
    for (int p : h.plen) pe = std::max(pe, prefix_part_end(p, a.split_len));
    a.splits = (int)cdiv(pe, a.split_len);
  } else {
    a.split_len = kVecSplit;
    a.splits = (int)cdiv(std::max(h.maxplen, 1), kVecSplit);
  }
  a.nparts = a.splits + a.tail_chunks;
  if (a.nparts > cap || a.splits < 1)
    return fail(RGD_E_UNSUPPORTED, "attention needs %d partials for %d rows (capacity %d)", a.nparts, R, cap);
  TimeScope ts(m, RGD_TIMER_ATTENTION, s);
  if (m->bf16) {
    {
      TimeScope tp(m, RGD_TIMER_ATTN_PREFIX, s);
      HIP_OK(attn_prefix_bf16(a, s));
    }
    HIP_OK(attn_tail_merge_bf16(a, (bf16_t*)out, s));
  } else {
    HIP_OK(attn_prefix_vec<float>(a, s));
    HIP_OK(attn_tail_combine<float>(a, (float*)out, s));
  }
  return RGD_OK;
}

// -------------------------------------------------------------- GEMM glue --
int gemm(rgd_model* m, GemmArgs& g, hipStream_t s) {
  hipError_t e = m->bf16 ? gemm_bf16(g, s) : gemm_f32(g, s);
  if (e != hipSuccess) return fail(RGD_E_HIP, "gemm launch failed: %s", hipGetErrorString(e));
  return RGD_OK;
}

int lm_head(rgd_model* m, const void* x, int ldx, int R, float* logits, hipStream_t s) {
  GemmArgs g{};
  g.x = x;
  g.ldx = ldx;
  g.M = R;
  g.seg[0] = {m->bf16 ? m->lm_head_packed : m->lm_head, 0, m->cfg.vocab};
  g.nseg = 1;
  g.N = m->cfg.vocab;
  g.K = m->cfg.d_model;
  g.splits = 1;
  g.y = logits;
  g.ldy = m->cfg.vocab;
  g.tilemax = m->tilemax;
  g.tilekey = m->bf16 ? m->tilekey : nullptr;
  g.ntiles = m->ntiles;
  g.mode = GEMM_LOGITS;
  TimeScope ts(m, RGD_TIMER_LM_HEAD, s);
  return gemm(m, g, s);
}

// Residual-stream readout taken inside a forward pass: after block `layer`
// (1-based; 0 = the embedding), rows row0 + r * stride (r < nrows) of the
// residual stream are scored into out[r].
struct Readout {
  int layer;
  const float* w;
  float b;
  long long row0, stride;
  int nrows;
  float* out;
};

// One forward pass of R rows through every layer.  feed: token of row r at
// feed[r * feed_stride]; embedded: the input rows (m->x, m->xn) were already
// written by the sampler for these tokens.  Leaves the final normalised hidden
// state in m->xn.
// feed: input token of row r at feed[i * feed_stride], i = feed_map[r] (null map: i = r)
int forward_rows(rgd_model* m, rgd_kv* kv, const Rows& rows, const HostRows& h, const int* feed,
                 int feed_stride, hipStream_t s, bool embedded = false, const Readout* ro = nullptr,
                 const int* feed_map = nullptr) {
  const rgd_model_config& c = m->cfg;
  const int R = rows.R, d = c.d_model, Hq = c.n_heads, Hkv = c.n_kv_heads, D = c.head_dim;
  const int F = c.ffn_dim;
  const bool bf = m->bf16;
  const int mblocks = (int)cdiv(R, 64);
  const float* g0 = (const float*)m->layers[0].attn_norm;
  if (!embedded && bf)
    HIP_OK(embed_rmsnorm<bf16_t>(feed, feed_stride, feed_map, R, (const bf16_t*)m->embed, d, c.vocab, m->x, g0,
                                 c.rms_eps, (bf16_t*)m->xn, s));
  else if (!embedded)
    HIP_OK(embed_rmsnorm<float>(feed, feed_stride, feed_map, R, (const float*)m->embed, d, c.vocab, m->x, g0,
                                c.rms_eps, (float*)m->xn, s));
  auto readout = [&](int layer) -> hipError_t {
    if (!ro || ro->layer != layer) return hipSuccess;
    return residual_readout(m->x, ro->row0, ro->stride, ro->nrows, d, ro->w, ro->b, ro->out, s);
  };
  HIP_OK(readout(0));
  auto norm = [&](const float* parts, int np, const void* gain) -> hipError_t {
    const long long stride = (long long)R * d;
    return bf ? residual_rmsnorm<bf16_t>(m->x, parts, np, stride, (const float*)gain, c.rms_eps, R, d,
                                         (bf16_t*)m->xn, s)
              : residual_rmsnorm<float>(m->x, parts, np, stride, (const float*)gain, c.rms_eps, R, d,
                                        (float*)m->xn, s);
  };
  auto splits = [&](int mode, int N, int K) { return bf ? pick_splits(gemm_groups(mode, N), K) : 1; };
  for (int l = 0; l < c.n_layers; ++l) {
    const rgd_layer_weights& L = m->layers[l];
    const KVLayout kvl = kv->layer(l);
    const void* wq = bf ? m->packed[l].wq : L.wq;
    const void* wk = bf ? m->packed[l].wk : L.wk;
    const void* wv = bf ? m->packed[l].wv : L.wv;
    // fused Q/K/V projection (split-K partials, summed by the RoPE epilogue)
    GemmArgs g{};
    g.x = m->xn;
    g.ldx = d;
    g.M = R;
    g.seg[0] = {wq, 0, Hq * D};
    g.seg[1] = {wk, Hq * D, Hkv * D};
    g.seg[2] = {wv, (Hq + Hkv) * D, Hkv * D};
    g.nseg = 3;
    g.N = m->nqkv;
    g.K = d;
    g.splits = splits(GEMM_STORE, g.N, d);
    g.y = m->qkv_part;
    g.ldy = g.N;
    g.split_stride = (long long)R * g.N;
    g.mode = GEMM_STORE;
    RGD_TRY(gemm(m, g, s));
    if (bf)
      HIP_OK(qkv_rope_store<bf16_t>(m->qkv_part, g.splits, g.split_stride, rows, Hq, Hkv, D, m->rope_cs, c.max_pos,
                                    (bf16_t*)m->q, kvl, s));
    else
      HIP_OK(qkv_rope_store<float>(m->qkv_part, g.splits, g.split_stride, rows, Hq, Hkv, D, m->rope_cs, c.max_pos,
                                   (float*)m->q, kvl, s));
    RGD_TRY(run_attention(m, kvl, rows, h, rows.prefill ? 0 : rows.t + 1, 0, m->attn_out, s));
    // output projection: partials added to the residual stream by the FFN norm
    GemmArgs o{};
    o.x = m->attn_out;
    o.ldx = Hq * D;
    o.M = R;
    o.seg[0] = {bf ? m->packed[l].wo : L.wo, 0, d};
    o.nseg = 1;
    o.N = d;
    o.K = Hq * D;
    o.splits = splits(GEMM_STORE, d, o.K);
    o.y = m->o_part;
    o.ldy = d;
    o.split_stride = (long long)R * d;
    o.mode = GEMM_STORE;
    RGD_TRY(gemm(m, o, s));
    HIP_OK(norm(m->o_part, o.splits, L.ffn_norm));
    // SwiGLU: act = silu(W_gate xn) * (W_up xn)
    GemmArgs f{};
    f.x = m->xn;
    f.ldx = d;
    f.M = R;
    f.seg[0] = {bf ? m->packed[l].w_gate : L.w_gate, 0, F};
    f.seg[1] = {bf ? m->packed[l].w_up : L.w_up, 0, F};
    f.nseg = 2;
    f.N = F;
    f.K = d;
    f.splits = 1;
    f.y = m->act;
    f.ldy = F;
    f.mode = GEMM_SILU;
    RGD_TRY(gemm(m, f, s));
    GemmArgs dn{};
    dn.x = m->act;
    dn.ldx = F;
    dn.M = R;
    dn.seg[0] = {bf ? m->packed[l].w_down : L.w_down, 0, d};
    dn.nseg = 1;
    dn.N = d;
    dn.K = F;
    dn.splits = splits(GEMM_STORE, d, F);
    dn.y = m->down_part;
    dn.ldy = d;
    dn.split_stride = (long long)R * d;
    dn.mode = GEMM_STORE;
    RGD_TRY(gemm(m, dn, s));
    const void* next_gain = l + 1 < c.n_layers ? m->layers[l + 1].attn_norm : (const void*)m->final_norm;
    HIP_OK(norm(m->down_part, dn.splits, next_gain));
    HIP_OK(readout(l + 1));
  }
  return RGD_OK;
}

SampleArgs sample_args(rgd_model* m, const float* z, long long ldz, int R, int V, float T, float p_min,
                       const float* pmax, int npmax, const unsigned long long* seeds, unsigned ctr, int* out,
                       long long out_stride, int out_col, int* cur) {
  SampleArgs a{};
  a.z = z;
  a.ldz = ldz;
  a.R = R;
  a.V = V;
  a.pmax = pmax;
  a.npmax = npmax;
  a.T = T;
  a.p_min = p_min;
  a.chunk = kSampleChunk;
  a.nchunks = (int)cdiv(V, kSampleChunk);
  a.chunk_sums = m->chunk_sums;
  if (a.nchunks * 16 <= 1024) a.sub_sums = m->sub_sums;
  a.seeds = seeds;
  a.ctr = ctr;
  a.stream = 0;
  a.out = out;
  a.out_stride = out_stride;
  a.out_col = out_col;
  a.cur_tok = cur;
  a.status = m->status;
  return a;
}

__global__ void gather_rows_kernel(const float* src, long long lds, const int* map, int V, float* dst) {
  const int r = blockIdx.y;
  const float* s = src + (long long)map[r] * lds;
  for (int i = blockIdx.x * 256 + threadIdx.x; i < V; i += 256 * gridDim.x) dst[(long long)r * V + i] = s[i];
}

__global__ void argmax_finish_kernel(unsigned long long* best, int R, int* out, long long stride, int col,
                                     int* cur) {
  const int r = blockIdx.x * 256 + threadIdx.x;
  if (r >= R) return;
  const int tok = int(0xFFFFFFFFu - uint32_t(best[r] & 0xFFFFFFFFull));
  out[r * stride + col] = tok;
  if (cur) cur[r] = tok;
  best[r] = 0ull;
}

// Probe state before token 1; with pre-check scores, a prompt scored <= theta
// is decided at once (SKIPPED: sampled without any check token).
__global__ void probe_init_kernel(int B, int k, int* tokens, int* len, int* event, const float* scores,
                                  float theta, int* failed) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < B * k) tokens[i] = 0;
  if (i < B) {
    len[i] = 0;
    event[i] = (scores && scores[i] <= theta) ? 3 : -1;
    failed[i] = 0;
  }
}

// Selects one token per row from logits z (ldz).  T == 0: argmax; otherwise
// min-p with p_min, or p-less when pless is set (p_min unused).  With
// fuse_embed the sampling workgroups also write the next step's input rows
// (embedding + first RMSNorm into m->x, m->xn) where the shapes allow it;
// *embedded tells the caller whether they did.
int select_tokens(rgd_model* m, const float* z, long long ldz, int R, const float* pmax, int npmax, float T,
                  float p_min, const unsigned long long* seeds, unsigned ctr, int* out, long long out_stride,
                  int out_col, int* cur, hipStream_t s, bool fuse_embed = false, bool* embedded = nullptr,
                  bool pless = false) {
  const int V = m->cfg.vocab;
  if (embedded) *embedded = false;
  if (T == 0.f) {
    HIP_OK(argmax_rows(z, ldz, R, V, m->best, s));
    hipLaunchKernelGGL(argmax_finish_kernel, dim3((R + 255) / 256), dim3(256), 0, s, m->best, R, out,
                       out_stride, out_col, cur);
    HIP_OK(hipGetLastError());
    return RGD_OK;
  }
  SampleArgs a = sample_args(m, z, ldz, R, V, T, p_min, pmax, npmax, seeds, ctr, out, out_stride, out_col, cur);
  const int d = m->cfg.d_model;
  if (fuse_embed && d % 4 == 0 && d <= 4096) {
    a.embed = m->embed;
    a.embed_bf16 = m->bf16;
    a.d = d;
    a.vocab = V;
    a.gain = (const float*)m->layers[0].attn_norm;
    a.eps = m->cfg.rms_eps;
    a.x = m->x;
    a.xn = m->xn;
    if (embedded) *embedded = true;
  }
  TimeScope ts(m, RGD_TIMER_SAMPLER, s);
  if (pless)
    HIP_OK(pless_sample(a, m->pl_stats, m->pl_thr, s));
  else
    HIP_OK(minp_sample(a, s));
  return RGD_OK;
}

bool valid_dtype_shapes(const rgd_model_config& c, std::string& why) {
  if (c.n_layers < 1 || c.d_model < 1 || c.n_heads < 1 || c.n_kv_heads < 1 || c.head_dim < 2 ||
      c.ffn_dim < 1 || c.vocab < 2 || c.max_pos < 1) {
    why = "all sizes must be positive";
    return false;
  }
  if (c.n_heads % c.n_kv_heads) {
    why = "n_heads must be a multiple of n_kv_heads";
    return false;
  }
  if (c.head_dim < 8 || c.head_dim > 128 || 256 % c.head_dim) {
    why = "head_dim must be 8, 16, 32, 64 or 128";
    return false;
  }
  if (c.vocab % 4) {
    why = "vocab must be a multiple of 4";
    return false;
  }
  if ((long long)c.vocab > 256LL * kSampleChunk) {
    why = "vocab too large";
    return false;
  }
  if (c.dtype == RGD_DTYPE_BF16) {
    if (c.head_dim != 128 || c.d_model % 128 || (c.n_heads * c.head_dim) % 128 || c.ffn_dim % 128) {
      why = "bf16 models need head_dim 128 and d_model, Hq*D, ffn multiples of 128";
      return false;
    }
    if ((c.n_heads * c.head_dim) % 64 || (c.n_kv_heads * c.head_dim) % 64 || c.ffn_dim % 32) {
      why = "projection widths must be multiples of 64";
      return false;
    }
    if (c.n_heads / c.n_kv_heads > 16) {
      why = "bf16 models support at most 16 query heads per KV head";
      return false;
    }
  } else if (c.dtype == RGD_DTYPE_F32) {
    if (c.n_heads / c.n_kv_heads > 8) {
      why = "fp32 models support at most 8 query heads per KV head";
      return false;
    }
  } else {
    why = "unknown dtype";
    return false;
  }
  return true;
}

}  // namespace

// ===================================================================== ABI ===
extern "C" {

const char* rgd_version(void) { return "rgd-mi355x 0.1 (gfx950)"; }

const char* rgd_last_error(void) { return g_err.c_str(); }

int32_t rgd_model_create(const rgd_model_config* cfg, const rgd_weights* w, int32_t max_rows, rgd_model** out) {
  g_err.clear();
  if (!cfg || !w || !out) return fail(RGD_E_INVALID_ARG, "null argument");
  *out = nullptr;
  std::string why;
  if (!valid_dtype_shapes(*cfg, why)) {
    const bool bad_arg = cfg->dtype != RGD_DTYPE_F32 && cfg->dtype != RGD_DTYPE_BF16;
    return fail(bad_arg ? RGD_E_INVALID_ARG : RGD_E_UNSUPPORTED, "model config: %s", why.c_str());
  }
  if (max_rows < 1 || max_rows > 65536) return fail(RGD_E_INVALID_ARG, "max_rows must be in [1, 65536]");
  if (!w->embed || !w->final_norm || !w->lm_head || !w->layers)
    return fail(RGD_E_INVALID_ARG, "null weight pointer");
  for (int l = 0; l < cfg->n_layers; ++l) {
    const rgd_layer_weights& L = w->layers[l];
    if (!L.attn_norm || !L.wq || !L.wk || !L.wv || !L.wo || !L.ffn_norm || !L.w_gate || !L.w_up || !L.w_down)
      return fail(RGD_E_INVALID_ARG, "null weight pointer in layer %d", l);
  }
  rgd_model* m = new rgd_model();
  m->cfg = *cfg;
  m->bf16 = cfg->dtype == RGD_DTYPE_BF16;
  m->esz = m->bf16 ? 2 : 4;
  m->embed = w->embed;
  m->final_norm = (const float*)w->final_norm;
  m->lm_head = w->lm_head;
  m->layers.assign(w->layers, w->layers + cfg->n_layers);
  m->max_rows = max_rows;
  // split-K partials: every row of a step times the largest split factor of
  // the model's projections
  const int ksmax = cfg->dtype == RGD_DTYPE_BF16
                        ? std::max({pick_splits(gemm_groups(GEMM_STORE, (cfg->n_heads + 2 * cfg->n_kv_heads) * cfg->head_dim),
                                                cfg->d_model),
                                    pick_splits(gemm_groups(GEMM_STORE, cfg->d_model), cfg->n_heads * cfg->head_dim),
                                    pick_splits(gemm_groups(GEMM_STORE, cfg->d_model), cfg->ffn_dim)})
                        : 1;
  m->part_rows = max_rows * ksmax;
  const int R = max_rows, d = cfg->d_model, Hq = cfg->n_heads, Hkv = cfg->n_kv_heads, D = cfg->head_dim;
  m->nqkv = (Hq + 2 * Hkv) * D;
  m->ntiles = m->bf16 ? gemm_groups(GEMM_LOGITS, cfg->vocab) : (int)cdiv(cfg->vocab, 64);
  m->nchunks = (int)cdiv(cfg->vocab, kSampleChunk);
  const size_t e = m->esz;
  const size_t PR = m->part_rows;
  int rc = RGD_OK;
  auto A = [&](auto** p, size_t bytes) {
    if (rc == RGD_OK) rc = m->alloc(p, bytes);
  };
  A(&m->x, (size_t)R * d * 4);
  A(&m->xn, (size_t)R * d * e);
  A(&m->qkv_part, PR * m->nqkv * 4);
  A(&m->q, (size_t)R * Hq * D * e);
  A(&m->part_o, (size_t)kMaxParts * R * Hq * D * 4);
  A(&m->part_lse, (size_t)kMaxParts * R * Hq * 4);
  A(&m->attn_out, (size_t)R * Hq * D * e);
  A(&m->o_part, PR * d * 4);
  A(&m->act, (size_t)R * cfg->ffn_dim * e);
  A(&m->down_part, PR * d * 4);
  A(&m->logits, (size_t)R * cfg->vocab * 4);
  A(&m->tilemax, (size_t)R * m->ntiles * 4);
  A(&m->tilekey, (size_t)R * m->ntiles * 8);
  A(&m->chunk_sums, (size_t)R * m->nchunks * 4);
  A(&m->sub_sums, (size_t)R * m->nchunks * 16 * 4);
  A(&m->pl_stats, (size_t)3 * R * m->nchunks * 4);
  A(&m->pl_thr, (size_t)R * 4);
  A(&m->best, (size_t)R * 8);
  A(&m->cur_tok, (size_t)R * 4);
  A(&m->status, 4);
  A(&m->row_map, (size_t)R * 4);
  A(&m->probe_fail, (size_t)R * 4);
  A(&m->d_gate, (size_t)(2 * R + 1) * 4);
  A(&m->soft_keys, (size_t)R * m->nchunks * kMaxTopK * 8);
  A(&m->soft_cm, (size_t)2 * R * m->nchunks * 4);
  A(&m->d_prompt, (size_t)R * 4);
  A(&m->d_base, (size_t)R * 4);
  A(&m->d_plen, (size_t)R * 4);
  // RoPE rotations: angle pos * theta^(-2j/D) in fp64, rounded to fp32 once
  const int half = D / 2;
  const size_t ncs = ((size_t)cfg->max_pos + 1) * half;
  A(&m->rope_cs, ncs * 2 * sizeof(float));
  if (rc == RGD_OK) {
    std::vector<float> cs(ncs * 2);
    for (int j = 0; j < half; ++j) {
      const double f = std::pow((double)cfg->rope_theta, -2.0 * j / D);
      for (int pos = 0; pos <= cfg->max_pos; ++pos) {
        const double a = pos * f;
        cs[((size_t)pos * half + j) * 2] = (float)std::cos(a);
        cs[((size_t)pos * half + j) * 2 + 1] = (float)std::sin(a);
      }
    }
    if (hipMemcpy(m->rope_cs, cs.data(), cs.size() * sizeof(float), hipMemcpyHostToDevice) != hipSuccess)
      rc = fail(RGD_E_HIP, "RoPE table upload failed");
  }
  // bf16: repack every matrix into the GEMM panel layout
  if (rc == RGD_OK && m->bf16) {
    auto pack = [&](const void* src, int N, int K, void** dst, int group = 1) {
      if (rc != RGD_OK) return;
      rc = m->alloc(dst, packed_elems(N, K, group) * 2);
      if (rc == RGD_OK && pack_panels(src, N, K, group, *dst, nullptr) != hipSuccess)
        rc = fail(RGD_E_HIP, "weight packing failed");
    };
    m->packed.resize(cfg->n_layers);
    for (int l = 0; l < cfg->n_layers; ++l) {
      const rgd_layer_weights& L = m->layers[l];
      rgd_model::Packed& P = m->packed[l];
      pack(L.wq, Hq * D, d, &P.wq);
      pack(L.wk, Hkv * D, d, &P.wk);
      pack(L.wv, Hkv * D, d, &P.wv);
      pack(L.wo, d, Hq * D, &P.wo);
      pack(L.w_gate, cfg->ffn_dim, d, &P.w_gate);
      pack(L.w_up, cfg->ffn_dim, d, &P.w_up);
      pack(L.w_down, d, cfg->ffn_dim, &P.w_down);
    }
    pack(m->lm_head, cfg->vocab, d, &m->lm_head_packed, kHeadGroup);
  }
  if (rc != RGD_OK) {
    delete m;
    return rc;
  }
  m->stage_ints = (size_t)R * 8 + 64;
  if (hipHostMalloc((void**)&m->h_stage, m->stage_ints * sizeof(int), hipHostMallocDefault) != hipSuccess ||
      hipHostMalloc((void**)&m->h_events, (size_t)(2 * R + 1) * sizeof(int), hipHostMallocDefault) != hipSuccess ||
      hipEventCreateWithFlags(&m->stage_done, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&m->poll_done, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&m->sync_done, hipEventDisableTiming) != hipSuccess ||
      hipEventRecord(m->stage_done, nullptr) != hipSuccess) {
    delete m;
    return fail(RGD_E_HIP, "pinned staging allocation failed");
  }
  // argmax keys start cleared
  if (hipMemset(m->best, 0, (size_t)R * 8) != hipSuccess ||
      hipMemset(m->status, 0, 4) != hipSuccess || hipDeviceSynchronize() != hipSuccess) {
    delete m;
    return fail(RGD_E_HIP, "workspace initialisation failed");
  }
  *out = m;
  return RGD_OK;
}

void rgd_model_destroy(rgd_model* m) { delete m; }

int32_t rgd_kv_create(const rgd_model* m, int32_t max_prompts, int32_t max_prefix, int32_t n_pages, int32_t page_size,
                      void* prefix_k, void* prefix_v, void* pool_k, void* pool_v, rgd_kv** out) {
  g_err.clear();
  if (!m || !out || !prefix_k || !prefix_v || !pool_k || !pool_v) return fail(RGD_E_INVALID_ARG, "null argument");
  *out = nullptr;
  if (max_prompts < 1 || max_prefix < 1 || n_pages < 0 || page_size < 1 || page_size > 4096)
    return fail(RGD_E_INVALID_ARG, "kv sizes out of range");
  if (max_prefix > m->cfg.max_pos) return fail(RGD_E_INVALID_ARG, "max_prefix exceeds the model's max_pos");
  if (m->bf16 && page_size % 16) return fail(RGD_E_UNSUPPORTED, "bf16 models need page_size % 16 == 0");
  if (!m->bf16 && max_prefix > kMaxParts * kVecSplit)
    return fail(RGD_E_UNSUPPORTED, "fp32 models hold at most %d prefix positions", kMaxParts * kVecSplit);
  rgd_kv* kv = new rgd_kv();
  kv->m = m;
  kv->max_prompts = max_prompts;
  kv->max_prefix = max_prefix;
  kv->n_pages = n_pages;
  kv->page_size = page_size;
  kv->prefix_k = prefix_k;
  kv->prefix_v = prefix_v;
  kv->pool_k = pool_k;
  kv->pool_v = pool_v;
  kv->plen.assign(max_prompts, 0);
  kv->probe_pages.assign(max_prompts, {});
  for (int p = n_pages - 1; p >= 0; --p) kv->free_pages.push_back(p);
  kv->max_pages = (int)std::max<long long>(1, cdiv(m->cfg.max_pos, page_size));
  if (hipMalloc((void**)&kv->d_pages, (size_t)m->max_rows * kv->max_pages * 4) != hipSuccess) {
    delete kv;
    return fail(RGD_E_OOM, "page-table allocation failed");
  }
  // the model's pinned staging must hold one page table plus the row arrays
  rgd_model* mm = const_cast<rgd_model*>(m);
  const size_t need = (size_t)m->max_rows * (kv->max_pages + 8) + 64;
  if (mm->stage_ints < need) {
    int* p = nullptr;
    if (hipEventSynchronize(mm->stage_done) != hipSuccess ||
        hipHostMalloc((void**)&p, need * sizeof(int), hipHostMallocDefault) != hipSuccess) {
      delete kv;
      return fail(RGD_E_OOM, "pinned staging allocation failed");
    }
    (void)hipHostFree(mm->h_stage);
    mm->h_stage = p;
    mm->stage_ints = need;
  }
  *out = kv;
  return RGD_OK;
}

void rgd_kv_destroy(rgd_kv* kv) { delete kv; }

int32_t rgd_kv_set_prefix_len(rgd_kv* kv, int32_t prompt, int32_t len) {
  g_err.clear();
  if (!kv) return fail(RGD_E_INVALID_ARG, "null kv");
  if (prompt < 0 || prompt >= kv->max_prompts) return fail(RGD_E_INVALID_ARG, "prompt out of range");
  if (len < 0 || len > kv->max_prefix) return fail(RGD_E_INVALID_ARG, "len out of range");
  kv->plen[prompt] = len;
  return RGD_OK;
}

int32_t rgd_table_create(const int32_t* offsets, const int32_t* tokens, int32_t n_entries, const int32_t* owner,
                         int32_t min_match, rgd_table** out) {
  g_err.clear();
  if (!out) return fail(RGD_E_INVALID_ARG, "null out");
  *out = nullptr;
  if (n_entries < 0 || n_entries > (1 << 20)) return fail(RGD_E_INVALID_ARG, "n_entries out of range");
  if (n_entries > 0 && (!offsets || !tokens)) return fail(RGD_E_INVALID_ARG, "null table arrays");
  if (min_match < 1) return fail(RGD_E_INVALID_ARG, "min_match must be >= 1");
  if (n_entries > 0) {
    if (offsets[0] != 0) return fail(RGD_E_INVALID_ARG, "offsets[0] must be 0");
    for (int e = 0; e < n_entries; ++e)
      if (offsets[e + 1] < offsets[e]) return fail(RGD_E_INVALID_ARG, "offsets must be non-decreasing");
    for (int e = 0; e < n_entries; ++e)
      if (owner && owner[e] < -1) return fail(RGD_E_INVALID_ARG, "owner must be -1 or a prompt index");
  }
  rgd_table* t = new rgd_table();
  t->n_entries = n_entries;
  t->min_match = min_match;
  const int ntok = n_entries ? offsets[n_entries] : 0;
  std::vector<int> own(std::max(n_entries, 1), -1);
  if (owner) std::copy(owner, owner + n_entries, own.begin());
  std::vector<int> offs(n_entries + 1, 0);
  if (n_entries) std::copy(offsets, offsets + n_entries + 1, offs.begin());
  if (hipMalloc((void**)&t->d_offsets, offs.size() * 4) != hipSuccess ||
      hipMalloc((void**)&t->d_tokens, std::max(ntok, 1) * 4) != hipSuccess ||
      hipMalloc((void**)&t->d_owner, own.size() * 4) != hipSuccess) {
    delete t;
    return fail(RGD_E_OOM, "table allocation failed");
  }
  if (hipMemcpy(t->d_offsets, offs.data(), offs.size() * 4, hipMemcpyHostToDevice) != hipSuccess ||
      (ntok && hipMemcpy(t->d_tokens, tokens, ntok * 4, hipMemcpyHostToDevice) != hipSuccess) ||
      hipMemcpy(t->d_owner, own.data(), own.size() * 4, hipMemcpyHostToDevice) != hipSuccess) {
    delete t;
    return fail(RGD_E_HIP, "table upload failed");
  }
  *out = t;
  return RGD_OK;
}

void rgd_table_destroy(rgd_table* t) { delete t; }

namespace {

// Prefill shared by rgd_prefill_kv and rgd_prefill_kv_scored (cls_w non-null:
// score each prompt's last position after block cls_layer into scores[b]).
int prefill_impl(rgd_model* m, rgd_kv* kv, const int32_t* tokens, int32_t B, int32_t n, int32_t start_pos,
                 float* last_logits, int cls_layer, const float* cls_w, float cls_b, float* scores,
                 rgd_stream stream) {
  if (!m || !kv || !tokens || !last_logits) return fail(RGD_E_INVALID_ARG, "null argument");
  if (kv->m != m) return fail(RGD_E_INVALID_ARG, "kv belongs to another model");
  if (B < 1 || B > kv->max_prompts || n < 1 || start_pos < 0) return fail(RGD_E_INVALID_ARG, "bad B/n/start_pos");
  if ((long long)start_pos + n > kv->max_prefix) return fail(RGD_E_INVALID_ARG, "prompt exceeds max_prefix");
  for (int b = 0; b < B; ++b)
    if (kv->plen[b] != start_pos)
      return fail(RGD_E_STATE, "prompt %d holds %d positions, prefill starts at %d", b, kv->plen[b], start_pos);
  if (kv->probe_held) return fail(RGD_E_STATE, "probe tails not released (call rgd_gate)");
  hipStream_t s = (hipStream_t)stream;
  const int V = m->cfg.vocab, d = m->cfg.d_model;
  // chunks: whole prompts when n fits in max_rows, else segments of one prompt
  const int per_chunk = n <= m->max_rows ? m->max_rows / n : 0;
  const int seg = n <= m->max_rows ? n : m->max_rows;
  for (int b0 = 0; b0 < B;) {
    const int nb = per_chunk ? std::min(per_chunk, B - b0) : 1;
    for (int i0 = 0; i0 < n; i0 += seg) {
      const int len = std::min(seg, n - i0);
      HostRows h;
      for (int bb = 0; bb < nb; ++bb)
        for (int i = 0; i < len; ++i) {
          const int pos = start_pos + i0 + i;
          h.prompt.push_back(b0 + bb);
          h.base.push_back(pos);
          h.plen.push_back(pos + 1);
        }
      build_blocks(m, h);
      const int R = (int)h.prompt.size();
      RGD_TRY(upload_rows(m, h, s));
      Rows rows = device_rows(m, kv, R, 0, true);
      const int* feed = tokens + (long long)b0 * n + i0;
      // the prompts' last positions: rows bb * n + n - 1 (whole prompts), or
      // row len - 1 of a prompt's last segment
      Readout ro{cls_layer, cls_w, cls_b, per_chunk ? n - 1 : len - 1, per_chunk ? n : 1, per_chunk ? nb : 1,
                 scores + b0};
      const Readout* rop = (cls_w && (per_chunk || i0 + len == n)) ? &ro : nullptr;
      if (per_chunk) {
        RGD_TRY(forward_rows(m, kv, rows, h, feed, 1, s, false, rop));
        // logits of each prompt's last token: rows (bb * n + n - 1)
        RGD_TRY(lm_head(m, (const char*)m->xn + (size_t)(n - 1) * d * m->esz, n * d, nb,
                        last_logits + (long long)b0 * V, s));
      } else {
        RGD_TRY(forward_rows(m, kv, rows, h, feed, 1, s, false, rop));
        if (i0 + len == n)
          RGD_TRY(lm_head(m, (const char*)m->xn + (size_t)(len - 1) * d * m->esz, d, 1,
                          last_logits + (long long)b0 * V, s));
      }
    }
    b0 += nb;
  }
  for (int b = 0; b < B; ++b) kv->plen[b] = start_pos + n;
  return RGD_OK;
}

}  // namespace

int32_t rgd_prefill_kv(rgd_model* m, rgd_kv* kv, const int32_t* tokens, int32_t B, int32_t n, int32_t start_pos,
                       float* last_logits, rgd_stream stream) {
  g_err.clear();
  return prefill_impl(m, kv, tokens, B, n, start_pos, last_logits, 0, nullptr, 0.f, nullptr, stream);
}

int32_t rgd_prefill_kv_scored(rgd_model* m, rgd_kv* kv, const int32_t* tokens, int32_t B, int32_t n,
                              int32_t start_pos, float* last_logits, int32_t cls_layer, const float* cls_w,
                              float cls_b, float* scores, rgd_stream stream) {
  g_err.clear();
  if (!m || !cls_w || !scores) return fail(RGD_E_INVALID_ARG, "null argument");
  if (cls_layer < 0 || cls_layer > m->cfg.n_layers) return fail(RGD_E_INVALID_ARG, "cls_layer out of range");
  if (!(cls_b == cls_b)) return fail(RGD_E_INVALID_ARG, "cls_b is NaN");
  return prefill_impl(m, kv, tokens, B, n, start_pos, last_logits, cls_layer, cls_w, cls_b, scores, stream);
}

namespace {

// The probe loop shared by the hard and the soft gate (topk > 0: tokens 1..c
// are soft steps) and the fixed probe (fixed: no early exit, the table judges
// the finished probe).
int probe_impl(rgd_model* m, rgd_kv* kv, const float* last_logits, const rgd_table* tbl, int B, int k, int c,
               int eos_id, int topk, float rho, const float* scores, float theta, int* probe_tokens, int* probe_len,
               int* event, rgd_stream stream, bool fixed = false) {
  if (!m || !kv || !last_logits || !probe_tokens || !probe_len || !event)
    return fail(RGD_E_INVALID_ARG, "null argument");
  if (kv->m != m) return fail(RGD_E_INVALID_ARG, "kv belongs to another model");
  if (B < 1 || B > kv->max_prompts || B > m->max_rows) return fail(RGD_E_INVALID_ARG, "B out of range");
  if (k < 1 || c < 1) return fail(RGD_E_INVALID_ARG, "k and c must be >= 1");
  if (eos_id >= m->cfg.vocab) return fail(RGD_E_INVALID_ARG, "eos_id out of range");
  if (kv->probe_held) return fail(RGD_E_STATE, "previous probe tails not released (call rgd_gate)");
  for (int b = 0; b < B; ++b) {
    if (kv->plen[b] < 1) return fail(RGD_E_STATE, "prompt %d has no prefix (prefill first)", b);
    if ((long long)kv->plen[b] + k - 1 > m->cfg.max_pos) return fail(RGD_E_INVALID_ARG, "probe exceeds max_pos");
  }
  const int pages_per = (int)cdiv(std::max(k - 1, 0), kv->page_size);
  if (pages_per > kv->max_pages) return fail(RGD_E_INVALID_ARG, "probe longer than the page table");
  if ((long long)pages_per * B > (long long)kv->free_pages.size())
    return fail(RGD_E_OOM, "page pool too small for %d probes of %d tokens", B, k);
  hipStream_t s = (hipStream_t)stream;
  const int V = m->cfg.vocab;
  // hold pages for every probe tail
  for (int b = 0; b < B; ++b) {
    kv->probe_pages[b].clear();
    for (int i = 0; i < pages_per; ++i) {
      kv->probe_pages[b].push_back(kv->free_pages.back());
      kv->free_pages.pop_back();
    }
  }
  kv->probe_held = true;
  // a probe that fails part way (a HIP error) waits for its stream and returns
  // the tail pages, so the KV state is not left holding them
  struct ReleaseOnError {
    rgd_kv* kv;
    hipStream_t s;
    bool ok = false;
    ~ReleaseOnError() {
      if (ok) return;
      (void)hipStreamSynchronize(s);
      for (auto& pp : kv->probe_pages) {
        for (int p : pp) kv->free_pages.push_back(p);
        pp.clear();
      }
      kv->probe_held = false;
    }
  } release{kv, s};
  hipLaunchKernelGGL(probe_init_kernel, dim3((int)cdiv((long long)B * k, 256)), dim3(256), 0, s, B, k, probe_tokens,
                     probe_len, event, scores, theta, m->probe_fail);
  HIP_OK(hipGetLastError());

  GateArgs ga{};
  ga.best = m->best;
  ga.best_reset = m->best;
  ga.row_prompt = m->d_prompt;
  ga.cur_tok = m->cur_tok;
  ga.probe_tokens = probe_tokens;
  ga.k = k;
  ga.probe_len = probe_len;
  ga.event = event;
  if (tbl) {
    ga.offsets = tbl->d_offsets;
    ga.tokens = tbl->d_tokens;
    ga.owner = tbl->d_owner;
    ga.n_entries = tbl->n_entries;
    ga.min_match = tbl->min_match;
  } else {
    ga.all_compatible = 1;  // fixed-length probe
  }
  ga.eos = eos_id;
  ga.no_early_exit = fixed ? 1 : 0;
  ga.failed = m->probe_fail;
  SoftArgs sa{};
  sa.V = V;
  sa.chunk = kSampleChunk;
  sa.nchunks = m->nchunks;
  sa.K = topk;
  sa.keys = m->soft_keys;
  sa.cmax = m->soft_cm;
  sa.csum = m->soft_cm + (size_t)m->max_rows * m->nchunks;
  sa.rho = rho;
  sa.soft_steps = c;
  // one probe step on logits z (row r of the alive set at z + r * V): soft
  // for tokens 1..c when a soft gate is asked for, hard otherwise
  // The hard steps of a bf16 model take the argmax from the LM head's tile
  // keys (no pass over the logits; token 1 comes from the prompt logits) and
  // write the next step's input rows (embedding + first RMSNorm) for the
  // current row set: `embedded` tells the next forward pass whether they are
  // there (a soft step, or a change of the row set, leaves them out).
  const int dm = m->cfg.d_model;
  const bool fuse = m->bf16 && dm % 4 == 0 && dm <= 4096;
  bool embedded = false;
  auto step = [&](const float* z, int R, int token, bool lm_keys) -> int {
    ga.R = R;
    embedded = false;
    if (topk > 0 && token <= c) {
      sa.g = ga;
      sa.z = z;
      sa.ldz = V;
      HIP_OK(probe_update_soft(sa, s));
    } else {
      GateArgs g2 = ga;
      if (lm_keys && fuse) {
        g2.tilekeys = m->tilekey;
        g2.ntiles = m->ntiles;
      } else {
        HIP_OK(argmax_rows(z, V, R, V, m->best, s));
      }
      if (fuse && token < k) {
        g2.embed = m->embed;
        g2.embed_bf16 = 1;
        g2.d = dm;
        g2.vocab = V;
        g2.feed_col = token - 1;
        g2.gain = (const float*)m->layers[0].attn_norm;
        g2.eps = m->cfg.rms_eps;
        g2.x = m->x;
        g2.xn = m->xn;
        embedded = true;
      }
      HIP_OK(probe_update(g2, s));
    }
    return RGD_OK;
  };

  std::vector<int> alive(B);
  for (int b = 0; b < B; ++b) alive[b] = b;
  int* pinned_ev = m->h_events;  // B <= max_rows

  auto set_rows = [&](HostRows& h, std::vector<int>& pages) -> int {
    h.prompt.clear();
    h.base.clear();
    h.plen.clear();
    pages.assign((size_t)alive.size() * kv->max_pages, 0);
    for (size_t r = 0; r < alive.size(); ++r) {
      const int b = alive[r];
      h.prompt.push_back(b);
      h.base.push_back(kv->plen[b]);
      h.plen.push_back(kv->plen[b]);
      for (int i = 0; i < pages_per; ++i) pages[r * kv->max_pages + i] = kv->probe_pages[b][i];
    }
    build_blocks(m, h);
    return upload(m,
                  {{m->d_prompt, h.prompt.data(), h.prompt.size()},
                   {m->d_base, h.base.data(), h.base.size()},
                   {m->d_plen, h.plen.data(), h.plen.size()},
                   {kv->d_pages, pages.data(), pages.size()}},
                  s);
  };
  HostRows h;
  std::vector<int> pages;
  RGD_TRY(set_rows(h, pages));
  // token 1 from the prompt logits (rows are prompts 0..B-1 here)
  RGD_TRY(step(last_logits, B, 1, false));
  // Polls: after each of the first c tokens and every c tokens after that
  // (the checks of Algorithm 1), and after token k.  After token 1 (which
  // needs no decode step) and after token k the host waits for the events;
  // the other checks are pipelined: the copy of the events is enqueued after
  // token j-1 and read once the next step has been launched, so the GPU never
  // waits for the host; a probe that ended there has decoded one more token,
  // which leaves its events and tokens as they were (decided rows are not
  // updated) and only costs that step's time.
  bool done = false;
  auto apply_poll = [&]() -> int {
    std::vector<int> still;
    for (int b : alive)
      if (pinned_ev[b] == -1) still.push_back(b);
    if (still.empty()) {
      done = true;
      return RGD_OK;
    }
    if (still.size() != alive.size()) {
      alive.swap(still);
      RGD_TRY(set_rows(h, pages));
      embedded = false;  // the rows were renumbered
    }
    return RGD_OK;
  };
  for (int j = 2;; ++j) {
    const int done_tokens = j - 1;
    const bool first = done_tokens <= c, last = done_tokens >= k;
    const bool check = first || done_tokens % c == 0 || last;
    const bool pipelined = check && done_tokens > 1 && !last;
    if (check && !pipelined) {
      HIP_OK(hipMemcpyAsync(pinned_ev, event, (size_t)B * 4, hipMemcpyDeviceToHost, s));
      HIP_OK(spin_sync(m, s));
      RGD_TRY(apply_poll());
      if (done) break;
    }
    if (pipelined) {
      HIP_OK(hipMemcpyAsync(pinned_ev, event, (size_t)B * 4, hipMemcpyDeviceToHost, s));
      HIP_OK(hipEventRecord(m->poll_done, s));
    }
    if (j > k) break;  // cannot happen: every prompt is decided after k tokens
    const int R = (int)alive.size();
    // row r feeds token j-1 of its prompt's probe (probe_tokens[prompt[r]][j-2])
    Rows rows = device_rows(m, kv, R, j - 2, false);
    RGD_TRY(forward_rows(m, kv, rows, h, probe_tokens + (j - 2), k, s, embedded, nullptr, m->d_prompt));
    RGD_TRY(lm_head(m, m->xn, m->cfg.d_model, R, m->logits, s));
    RGD_TRY(step(m->logits, R, j, true));
    if (pipelined) {
      HIP_OK(spin_wait(m->poll_done));
      RGD_TRY(apply_poll());
      if (done) break;
    }
  }
  HIP_OK(spin_sync(m, s));
  release.ok = true;
  return RGD_OK;
}

}  // namespace

int32_t rgd_probe(rgd_model* m, rgd_kv* kv, const float* last_logits, const rgd_table* tbl, int32_t B, int32_t k,
                  int32_t c, int32_t eos_id, int32_t* probe_tokens, int32_t* probe_len, int32_t* event,
                  rgd_stream stream) {
  g_err.clear();
  return probe_impl(m, kv, last_logits, tbl, B, k, c, eos_id, 0, 0.f, nullptr, 0.f, probe_tokens, probe_len, event,
                    stream);
}

int32_t rgd_probe_fixed(rgd_model* m, rgd_kv* kv, const float* last_logits, const rgd_table* tbl, int32_t B,
                        int32_t k, int32_t c, int32_t eos_id, int32_t* probe_tokens, int32_t* probe_len,
                        int32_t* event, rgd_stream stream) {
  g_err.clear();
  return probe_impl(m, kv, last_logits, tbl, B, k, c, eos_id, 0, 0.f, nullptr, 0.f, probe_tokens, probe_len, event,
                    stream, true);
}

int32_t rgd_probe_soft(rgd_model* m, rgd_kv* kv, const float* last_logits, const rgd_table* tbl, int32_t B,
                       int32_t k, int32_t c, int32_t eos_id, int32_t topk, float rho, int32_t* probe_tokens,
                       int32_t* probe_len, int32_t* event, rgd_stream stream) {
  g_err.clear();
  if (!m) return fail(RGD_E_INVALID_ARG, "null model");
  if (topk < 1 || topk > kMaxTopK || topk > m->cfg.vocab)
    return fail(RGD_E_INVALID_ARG, "topk must be in [1, %d] and at most the vocabulary", kMaxTopK);
  if (!(rho == rho)) return fail(RGD_E_INVALID_ARG, "rho is NaN");
  return probe_impl(m, kv, last_logits, tbl, B, k, c, eos_id, topk, rho, nullptr, 0.f, probe_tokens, probe_len,
                    event, stream);
}

int32_t rgd_probe_adaptive(rgd_model* m, rgd_kv* kv, const float* last_logits, const rgd_table* tbl, int32_t B,
                           int32_t k, int32_t c, int32_t eos_id, int32_t topk, float rho, const float* scores,
                           float theta, int32_t* probe_tokens, int32_t* probe_len, int32_t* event,
                           rgd_stream stream) {
  g_err.clear();
  if (!m || !scores) return fail(RGD_E_INVALID_ARG, "null argument");
  if (topk < 0 || topk > kMaxTopK || topk > m->cfg.vocab)
    return fail(RGD_E_INVALID_ARG, "topk must be in [0, %d] and at most the vocabulary", kMaxTopK);
  if (!(rho == rho) || !(theta == theta)) return fail(RGD_E_INVALID_ARG, "rho or theta is NaN");
  return probe_impl(m, kv, last_logits, tbl, B, k, c, eos_id, topk, rho, scores, theta, probe_tokens, probe_len,
                    event, stream);
}

int32_t rgd_gate(rgd_kv* kv, const int32_t* event, int32_t B, int32_t* decision_host, int32_t* n_miss_host,
                 int32_t* miss_idx_host, rgd_stream stream) {
  g_err.clear();
  if (!kv || !event || !decision_host || !n_miss_host || !miss_idx_host) return fail(RGD_E_INVALID_ARG, "null argument");
  if (B < 1 || B > kv->max_prompts) return fail(RGD_E_INVALID_ARG, "B out of range");
  if (!kv->probe_held) return fail(RGD_E_STATE, "no probe to gate (call rgd_probe)");
  hipStream_t s = (hipStream_t)stream;
  rgd_model* m = const_cast<rgd_model*>(kv->m);
  if (B > m->max_rows) return fail(RGD_E_INVALID_ARG, "B exceeds max_rows");
  // device decision + ordered miss list in one run [decision B | n_miss | miss B],
  // brought back with one copy into pinned memory
  int* d_dec = m->d_gate;
  int* d_nmiss = d_dec + B;
  int* d_miss = d_nmiss + 1;
  HIP_OK(gate_decide(event, B, d_dec, d_nmiss, d_miss, s));
  HIP_OK(hipMemcpyAsync(m->h_events, d_dec, (2 * (size_t)B + 1) * 4, hipMemcpyDeviceToHost, s));
  HIP_OK(spin_sync(m, s));
  const int nm = m->h_events[B];
  std::memcpy(decision_host, m->h_events, (size_t)B * 4);
  *n_miss_host = nm;
  std::memcpy(miss_idx_host, m->h_events + B + 1, (size_t)nm * 4);
  // drop every probe tail: pages go back to the pool, nothing is copied
  for (auto& pp : kv->probe_pages) {
    for (int p : pp) kv->free_pages.push_back(p);
    pp.clear();
  }
  kv->probe_held = false;
  return RGD_OK;
}

}  // extern "C"

namespace {

int32_t sample_continuations(rgd_model* m, rgd_kv* kv, const float* last_logits, const int32_t* prompt_idx,
                             int32_t n, int32_t N, int32_t steps, float T, float min_p, bool pless,
                             const uint64_t* seeds, const int32_t* forced, float* logits_tap, int32_t* out,
                             rgd_stream stream) {
  if (!m || !kv || !last_logits || !prompt_idx || !seeds || !out) return fail(RGD_E_INVALID_ARG, "null argument");
  if (kv->m != m) return fail(RGD_E_INVALID_ARG, "kv belongs to another model");
  if (n < 1 || N < 1 || steps < 1) return fail(RGD_E_INVALID_ARG, "n, N and steps must be >= 1");
  if ((long long)n * N > m->max_rows) return fail(RGD_E_INVALID_ARG, "n*N exceeds max_rows");
  if (!(T >= 0.f)) return fail(RGD_E_INVALID_ARG, "T must be >= 0");
  if (!pless && !(min_p >= 0.f && min_p <= 1.f)) return fail(RGD_E_INVALID_ARG, "min_p must be in [0,1]");
  if (pless && T > 0.f && (m->cfg.vocab % 4 || m->nchunks > 256))
    return fail(RGD_E_UNSUPPORTED, "p-less sampling needs a vocabulary that is a multiple of 4");
  if (kv->probe_held) return fail(RGD_E_STATE, "probe tails not released (call rgd_gate)");
  for (int i = 0; i < n; ++i) {
    const int b = prompt_idx[i];
    if (b < 0 || b >= kv->max_prompts) return fail(RGD_E_INVALID_ARG, "prompt_idx out of range");
    if (kv->plen[b] < 1) return fail(RGD_E_STATE, "prompt %d has no prefix", b);
    if ((long long)kv->plen[b] + steps - 1 > m->cfg.max_pos) return fail(RGD_E_INVALID_ARG, "steps exceed max_pos");
  }
  const int R = n * N;
  const int pages_per = (int)cdiv(steps - 1, kv->page_size);
  if (pages_per > kv->max_pages) return fail(RGD_E_INVALID_ARG, "steps exceed the page table");
  if ((long long)pages_per * R > (long long)kv->free_pages.size())
    return fail(RGD_E_OOM, "page pool too small for %d rows of %d tokens", R, steps);
  hipStream_t s = (hipStream_t)stream;
  const int V = m->cfg.vocab;
  // rows (prompt-major), page tables, row -> prompt logits map
  HostRows h;
  std::vector<int> pages((size_t)R * kv->max_pages, 0), map(R);
  std::vector<int> taken;
  for (int i = 0; i < n; ++i)
    for (int j = 0; j < N; ++j) {
      const int r = i * N + j, b = prompt_idx[i];
      h.prompt.push_back(b);
      h.base.push_back(kv->plen[b]);
      h.plen.push_back(kv->plen[b]);
      map[r] = b;
      for (int p = 0; p < pages_per; ++p) {
        const int pg = kv->free_pages.back();
        kv->free_pages.pop_back();
        taken.push_back(pg);
        pages[(size_t)r * kv->max_pages + p] = pg;
      }
    }
  build_blocks(m, h);
  struct GiveBack {
    rgd_kv* kv;
    std::vector<int>& t;
    ~GiveBack() {
      for (auto it = t.rbegin(); it != t.rend(); ++it) kv->free_pages.push_back(*it);
    }
  } give{kv, taken};
  RGD_TRY(upload(m,
                 {{m->d_prompt, h.prompt.data(), (size_t)R},
                  {m->d_base, h.base.data(), (size_t)R},
                  {m->d_plen, h.plen.data(), (size_t)R},
                  {kv->d_pages, pages.data(), pages.size()},
                  {m->row_map, map.data(), (size_t)R}},
                 s));
  const unsigned long long* sd = (const unsigned long long*)seeds;
  // step 0: every branch draws from its prompt's last-position logits
  float* z0 = logits_tap ? logits_tap : m->logits;
  hipLaunchKernelGGL(gather_rows_kernel, dim3((int)cdiv(V, 256 * 8), R), dim3(256), 0, s, last_logits, (long long)V,
                     m->row_map, V, z0);
  HIP_OK(hipGetLastError());
  if (T > 0.f && !pless) HIP_OK(chunk_max(z0, V, R, V, kSampleChunk, m->tilemax, s));
  struct StepIndex {  // restores the timing step index on every exit
    rgd_model* m;
    ~StepIndex() {
      m->tstep = 0;
      m->tloop = false;
    }
  } step_index{m};
  m->tstep = -1;  // the first draw (prompt logits) is not timed
  m->tloop = true;
  // the sampler writes the next step's input rows itself unless tokens are
  // forced (teacher forcing feeds other tokens) or no step follows
  bool embedded = false;
  RGD_TRY(select_tokens(m, z0, V, R, m->tilemax, m->nchunks, T, min_p, sd, 0u, out, steps, 0, m->cur_tok, s,
                        !forced && steps > 1, &embedded, pless));
  for (int st = 1; st < steps; ++st) {
    m->tstep = st - 1;
    TimeScope tstep(m, RGD_TIMER_STEP, s);
    Rows rows = device_rows(m, kv, R, st - 1, false);
    const int* feed = forced ? forced + (st - 1) : m->cur_tok;
    const int fstride = forced ? steps : 1;
    RGD_TRY(forward_rows(m, kv, rows, h, feed, fstride, s, embedded));
    float* z = logits_tap ? logits_tap + (size_t)st * R * V : m->logits;
    RGD_TRY(lm_head(m, m->xn, m->cfg.d_model, R, z, s));
    RGD_TRY(select_tokens(m, z, V, R, m->tilemax, m->ntiles, T, min_p, sd, (unsigned)st, out, steps, st,
                          m->cur_tok, s, !forced && st + 1 < steps, &embedded, pless));
  }
  // pages are returned to the pool by `give` (work on them stays ordered on `s`)
  return RGD_OK;
}

}  // namespace

extern "C" {

int32_t rgd_sample_continuations(rgd_model* m, rgd_kv* kv, const float* last_logits, const int32_t* prompt_idx,
                                 int32_t n, int32_t N, int32_t steps, float T, float min_p, const uint64_t* seeds,
                                 const int32_t* forced, float* logits_tap, int32_t* out, rgd_stream stream) {
  g_err.clear();
  return sample_continuations(m, kv, last_logits, prompt_idx, n, N, steps, T, min_p, false, seeds, forced,
                              logits_tap, out, stream);
}

int32_t rgd_sample_continuations_pless(rgd_model* m, rgd_kv* kv, const float* last_logits,
                                       const int32_t* prompt_idx, int32_t n, int32_t N, int32_t steps, float T,
                                       const uint64_t* seeds, const int32_t* forced, float* logits_tap,
                                       int32_t* out, rgd_stream stream) {
  g_err.clear();
  return sample_continuations(m, kv, last_logits, prompt_idx, n, N, steps, T, 0.f, true, seeds, forced,
                              logits_tap, out, stream);
}

int32_t rgd_check_status(rgd_model* m, rgd_stream stream) {
  g_err.clear();
  if (!m) return fail(RGD_E_INVALID_ARG, "null model");
  int st = 0;
  hipStream_t s = (hipStream_t)stream;
  HIP_OK(hipMemcpyAsync(&st, m->status, 4, hipMemcpyDeviceToHost, s));
  HIP_OK(hipStreamSynchronize(s));
  if (st) {
    HIP_OK(hipMemsetAsync(m->status, 0, 4, s));
    HIP_OK(hipStreamSynchronize(s));
    return fail(RGD_E_NONFINITE, "a logit row had a non-finite maximum");
  }
  return RGD_OK;
}

int32_t rgd_timing_enable(rgd_model* m, int32_t period) {
  g_err.clear();
  if (!m) return fail(RGD_E_INVALID_ARG, "null model");
  if (period < 0) return fail(RGD_E_INVALID_ARG, "timing period must be >= 0");
  if (period && m->tev[0].empty()) {
    for (int u = 0; u < RGD_TIMER_COUNT; ++u) {
      m->tev[u].resize(2 * kTimerPairs);
      // timing-only events: no system-scope fence (no cache writeback and invalidate
      // between the timed kernels)
      for (auto& e : m->tev[u]) HIP_OK(hipEventCreateWithFlags(&e, hipEventDisableSystemFence));
    }
  }
  m->timing = period != 0;
  m->tperiod = std::max(period, 1);
  return RGD_OK;
}

int32_t rgd_timing_read(rgd_model* m, double* ms, int64_t* launches) {
  g_err.clear();
  if (!m || !ms || !launches) return fail(RGD_E_INVALID_ARG, "null argument");
  for (int u = 0; u < RGD_TIMER_COUNT; ++u) {
    double tot = 0.0;
    for (int i = 0; i < m->tused[u]; ++i) {
      HIP_OK(hipEventSynchronize(m->tev[u][2 * i + 1]));
      float t = 0.f;
      HIP_OK(hipEventElapsedTime(&t, m->tev[u][2 * i], m->tev[u][2 * i + 1]));
      tot += t;
    }
    ms[u] = tot;
    launches[u] = m->tused[u];
    m->tused[u] = 0;
  }
  return RGD_OK;
}

// --------------------------------------------------------- kernel-level ----
int32_t rgd_kernel_attention(rgd_model* m, const void* q, int32_t R, const int32_t* row_prompt, const int32_t* plen,
                             const void* prefix_k, const void* prefix_v, int32_t max_prompts, int32_t max_prefix,
                             const void* pool_k, const void* pool_v, int32_t page_size, const int32_t* pages,
                             int32_t max_pages, int32_t tail_len, int32_t splits, void* out, rgd_stream stream) {
  g_err.clear();
  if (!m || !q || !row_prompt || !plen || !prefix_k || !prefix_v || !out) return fail(RGD_E_INVALID_ARG, "null argument");
  if (R < 1 || R > m->max_rows) return fail(RGD_E_INVALID_ARG, "R out of range");
  if (max_prompts < 1 || max_prefix < 1 || tail_len < 0 || splits < 0) return fail(RGD_E_INVALID_ARG, "bad sizes");
  if (tail_len > 0 && (!pool_k || !pool_v || !pages || page_size < 1 || max_pages < cdiv(tail_len, page_size)))
    return fail(RGD_E_INVALID_ARG, "tail arguments inconsistent");
  if (m->bf16 && tail_len > 0 && page_size % 16) return fail(RGD_E_UNSUPPORTED, "bf16 needs page_size % 16 == 0");
  HostRows h;
  for (int r = 0; r < R; ++r) {
    if (row_prompt[r] < 0 || row_prompt[r] >= max_prompts) return fail(RGD_E_INVALID_ARG, "row_prompt out of range");
    if (plen[r] < 0 || plen[r] > max_prefix) return fail(RGD_E_INVALID_ARG, "plen out of range");
    if (r && row_prompt[r] != row_prompt[r - 1])
      for (int p = 0; p < r; ++p)
        if (row_prompt[p] == row_prompt[r]) return fail(RGD_E_INVALID_ARG, "rows of one prompt must be contiguous");
    h.prompt.push_back(row_prompt[r]);
    h.base.push_back(plen[r]);
    h.plen.push_back(plen[r]);
  }
  build_blocks(m, h);
  hipStream_t s = (hipStream_t)stream;
  RGD_TRY(upload_rows(m, h, s));
  Rows rows;
  rows.R = R;
  rows.prompt = m->d_prompt;
  rows.base_pos = m->d_base;
  rows.plen = m->d_plen;
  rows.pages = pages;
  rows.max_pages = max_pages;
  rows.t = tail_len - 1;
  rows.prefill = 0;
  KVLayout kvl;
  kvl.prefix_k = const_cast<void*>(prefix_k);
  kvl.prefix_v = const_cast<void*>(prefix_v);
  kvl.pool_k = const_cast<void*>(pool_k);
  kvl.pool_v = const_cast<void*>(pool_v);
  kvl.P = max_prefix;
  kvl.VP = v_stride(max_prefix);
  kvl.page_size = page_size;
  kvl.split_len = prefix_split_len(max_prefix, max_prompts, m->cfg.n_kv_heads);
  // q is read from the model's q buffer: copy the caller's q there first
  const size_t qbytes = (size_t)R * m->cfg.n_heads * m->cfg.head_dim * m->esz;
  HIP_OK(hipMemcpyAsync(m->q, q, qbytes, hipMemcpyDeviceToDevice, s));
  return run_attention(m, kvl, rows, h, tail_len, splits, out, s);
}

int32_t rgd_kernel_lm_head(rgd_model* m, const void* hvec, int32_t R, float* logits, rgd_stream stream) {
  g_err.clear();
  if (!m || !hvec || !logits) return fail(RGD_E_INVALID_ARG, "null argument");
  if (R < 1 || R > m->max_rows) return fail(RGD_E_INVALID_ARG, "R out of range");
  return lm_head(m, hvec, m->cfg.d_model, R, logits, (hipStream_t)stream);
}

uint64_t rgd_sampler_workspace_bytes(int32_t R, int32_t V) {
  if (R < 1 || V < 1) return 0;
  const long long nch = cdiv(V, kSampleChunk);
  // best u64 [R], chunk sums f32 [R][nch], chunk maxima, sums of w and of w^2
  // f32 [3][R][nch] (the last two for p-less), p-less thresholds f32 [R]
  return (uint64_t)(8LL * R + 16LL * R * nch + 4LL * R + 256);
}

int32_t rgd_kernel_probe_step(rgd_model* m, const float* logits, int32_t R, const rgd_table* tbl, int32_t k,
                              int32_t c, int32_t eos_id, int32_t topk, float rho, int32_t* probe_tokens,
                              int32_t* probe_len, int32_t* event, rgd_stream stream) {
  g_err.clear();
  if (!m || !logits || !probe_tokens || !probe_len || !event) return fail(RGD_E_INVALID_ARG, "null argument");
  if (R < 1 || R > m->max_rows) return fail(RGD_E_INVALID_ARG, "R out of range");
  if (k < 1 || c < 0) return fail(RGD_E_INVALID_ARG, "k must be >= 1 and c >= 0");
  if (topk < 0 || topk > kMaxTopK || topk > m->cfg.vocab) return fail(RGD_E_INVALID_ARG, "topk out of range");
  if (!(rho == rho)) return fail(RGD_E_INVALID_ARG, "rho is NaN");
  hipStream_t s = (hipStream_t)stream;
  const int V = m->cfg.vocab;
  std::vector<int> ident(R);
  for (int r = 0; r < R; ++r) ident[r] = r;
  RGD_TRY(upload(m, {{m->d_prompt, ident.data(), (size_t)R}}, s));
  GateArgs ga{};
  ga.best = m->best;
  ga.best_reset = m->best;
  ga.row_prompt = m->d_prompt;
  ga.R = R;
  ga.probe_tokens = probe_tokens;
  ga.k = k;
  ga.probe_len = probe_len;
  ga.event = event;
  if (tbl) {
    ga.offsets = tbl->d_offsets;
    ga.tokens = tbl->d_tokens;
    ga.owner = tbl->d_owner;
    ga.n_entries = tbl->n_entries;
    ga.min_match = tbl->min_match;
  } else {
    ga.all_compatible = 1;
  }
  ga.eos = eos_id;
  if (topk > 0) {
    SoftArgs sa{};
    sa.g = ga;
    sa.z = logits;
    sa.ldz = V;
    sa.V = V;
    sa.chunk = kSampleChunk;
    sa.nchunks = m->nchunks;
    sa.K = topk;
    sa.keys = m->soft_keys;
    sa.cmax = m->soft_cm;
    sa.csum = m->soft_cm + (size_t)m->max_rows * m->nchunks;
    sa.rho = rho;
    sa.soft_steps = c;
    HIP_OK(probe_update_soft(sa, s));
  } else {
    HIP_OK(argmax_rows(logits, V, R, V, m->best, s));
    HIP_OK(probe_update(ga, s));
  }
  return RGD_OK;
}

int32_t rgd_kernel_argmax(const float* z, int32_t R, int32_t V, void* workspace, int32_t* out, rgd_stream stream) {
  g_err.clear();
  if (!z || !workspace || !out) return fail(RGD_E_INVALID_ARG, "null argument");
  if (R < 1 || V < 1) return fail(RGD_E_INVALID_ARG, "R and V must be >= 1");
  if ((uintptr_t)workspace % 256) return fail(RGD_E_INVALID_ARG, "workspace must be 256-byte aligned");
  hipStream_t s = (hipStream_t)stream;
  unsigned long long* best = (unsigned long long*)workspace;
  HIP_OK(fill_u32((uint32_t*)best, 0u, 2LL * R, s));
  HIP_OK(argmax_rows(z, V, R, V, best, s));
  hipLaunchKernelGGL(argmax_finish_kernel, dim3((R + 255) / 256), dim3(256), 0, s, best, R, out, 1LL, 0,
                     (int*)nullptr);
  HIP_OK(hipGetLastError());
  return RGD_OK;
}

}  // extern "C"

namespace rgd {

int32_t set_error(int32_t code, const char* msg) { return fail(code, "%s", msg); }

int32_t kernel_sample(const float* z, int32_t R, int32_t V, float T, float min_p, bool pless,
                      const uint64_t* seeds, uint32_t ctr, uint32_t stream0, int32_t draws, void* workspace,
                      int32_t* out, rgd_stream stream) {
  if (!z || !seeds || !workspace || !out) return fail(RGD_E_INVALID_ARG, "null argument");
  if (R < 1 || V < 4 || V % 4 || (long long)V > 256LL * kSampleChunk || draws < 1)
    return fail(RGD_E_INVALID_ARG, "bad R/V/draws");
  if (!(T > 0.f)) return fail(RGD_E_INVALID_ARG, "T must be > 0");
  if (!pless && !(min_p >= 0.f && min_p <= 1.f)) return fail(RGD_E_INVALID_ARG, "min_p must be in [0,1]");
  if ((uintptr_t)workspace % 256) return fail(RGD_E_INVALID_ARG, "workspace must be 256-byte aligned");
  hipStream_t s = (hipStream_t)stream;
  const int nch = (int)cdiv(V, kSampleChunk);
  char* w = (char*)workspace;
  float* csum = (float*)(w + 8LL * R);
  float* cmax = csum + (long long)R * nch;  // start of the [3][R][nch] statistics
  float* thr = cmax + 3LL * R * nch;
  SampleArgs a{};
  a.z = z;
  a.ldz = V;
  a.R = R;
  a.V = V;
  a.pmax = cmax;
  a.npmax = nch;
  a.T = T;
  a.p_min = min_p;
  a.chunk = kSampleChunk;
  a.nchunks = nch;
  a.chunk_sums = csum;
  a.seeds = (const unsigned long long*)seeds;
  a.ctr = ctr;
  a.stream = stream0;
  a.out = out;
  a.out_stride = draws;
  a.out_col = 0;
  a.cur_tok = nullptr;
  a.status = nullptr;
  if (pless) {
    HIP_OK(pless_sample(a, cmax, thr, s));
    a.row_thr = thr;
  } else {
    HIP_OK(minp_sample_standalone(a, cmax, s));
  }
  if (draws > 1) HIP_OK(minp_multi_draw(a, draws, stream0, out, s));
  return RGD_OK;
}

}  // namespace rgd

extern "C" {

int32_t rgd_kernel_sample(const float* z, int32_t R, int32_t V, float T, float min_p, const uint64_t* seeds,
                          uint32_t ctr, uint32_t stream0, int32_t draws, void* workspace, int32_t* out,
                          rgd_stream stream) {
  g_err.clear();
  return kernel_sample(z, R, V, T, min_p, false, seeds, ctr, stream0, draws, workspace, out, stream);
}

int32_t rgd_kernel_sample_pless(const float* z, int32_t R, int32_t V, float T, const uint64_t* seeds,
                                uint32_t ctr, uint32_t stream0, int32_t draws, void* workspace, int32_t* out,
                                rgd_stream stream) {
  g_err.clear();
  return kernel_sample(z, R, V, T, 0.f, true, seeds, ctr, stream0, draws, workspace, out, stream);
}

}  // extern "C"
