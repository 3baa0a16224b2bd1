/*
 * rgd.h - C ABI of the MI355X (gfx950) refusal-gated decoding library.
 *
 * Refusal-gated decoding (Section 3, Algorithm 1): a prompt's KV cache is
 * computed once and shared; a short greedy probe decodes against it and is
 * checked after every token for compatibility with a table of refusal
 * prefixes; a probe that stays compatible to a stop token or the length cap is
 * returned as the greedy response, otherwise the probe's own positions are
 * dropped and N high-temperature continuations are sampled from the prompt.
 *
 * Conventions (all entry points):
 *  - Every function returns an rgd_status (int32).  On failure the reason is
 *    available from rgd_last_error() (thread-local, valid until the next call
 *    on the same thread).  Arguments are validated before any HIP call; an
 *    invalid argument leaves all state untouched.
 *  - "dev" pointers are device memory (e.g. PyTorch tensors on the GPU) and
 *    "host" pointers ordinary host memory.  The caller owns every buffer it
 *    passes; the library never frees them.  The library owns its handles and
 *    the workspace it allocates in the *_create calls; no entry point on the
 *    decode path allocates device memory.
 *  - stream is a hipStream_t (NULL = the null stream).  Work is enqueued on it;
 *    calls documented as synchronous wait for that stream.
 *  - Layouts are row-major with the last index fastest.  bf16 values are IEEE
 *    bfloat16 bit patterns, fp32 values IEEE binary32.
 *  - Results are deterministic: reductions use a fixed order and no floating
 *    point atomics, so equal inputs and seeds give bit-identical outputs.
 *  - A model and its KV state hold the workspace, staging buffers and page
 *    pool every call on them uses: calls on one model (or its KV states) must
 *    not overlap, from several threads or on several streams.  Different
 *    models are independent.
 */
#ifndef RGD_H
#define RGD_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct rgd_model rgd_model;
typedef struct rgd_kv rgd_kv;
typedef struct rgd_table rgd_table;
typedef void* rgd_stream; /* hipStream_t */

enum rgd_status {
  RGD_OK = 0,
  RGD_E_INVALID_ARG = 1, /* null pointer, size out of range, bad enum */
  RGD_E_OOM = 2,         /* page pool or workspace exhausted */
  RGD_E_HIP = 3,         /* a HIP runtime call failed */
  RGD_E_UNSUPPORTED = 4, /* dtype or shape the library does not handle */
  RGD_E_NONFINITE = 5,   /* a logit row had a non-finite maximum */
  RGD_E_STATE = 6        /* entry points called out of order */
};

enum rgd_dtype { RGD_DTYPE_F32 = 0, RGD_DTYPE_BF16 = 1 };

/* Decisive probe events (Algorithm 1: incompatibility, stop, length cap). */
enum rgd_event { RGD_EVENT_INCOMPAT = 0, RGD_EVENT_STOP = 1, RGD_EVENT_MAXLEN = 2,
                 RGD_EVENT_SKIPPED = 3 /* pre-check score <= theta: sampled without a check */ };

/* Target model M: a pre-norm decoder (RMSNorm, grouped-query attention with
 * rotate-half RoPE, SwiGLU feed-forward, untied LM head).  The paper runs
 * pretrained models of this family (Section 4).  d_model = n_heads * head_dim
 * is not required; n_heads must be a multiple of n_kv_heads. */
typedef struct rgd_model_config {
  int32_t n_layers;
  int32_t d_model;
  int32_t n_heads;    /* query heads Hq */
  int32_t n_kv_heads; /* key/value heads Hkv */
  int32_t head_dim;   /* D */
  int32_t ffn_dim;
  int32_t vocab;
  int32_t dtype;      /* rgd_dtype of weights, KV cache and activations */
  float rms_eps;
  float rope_theta;
  int32_t max_pos;    /* largest position any call may use, exclusive */
} rgd_model_config;

/* Per-layer weights, device pointers in the model dtype, W[out][in] row-major
 * (y = W x).  wq [Hq*D][d_model], wk/wv [Hkv*D][d_model], wo [d_model][Hq*D],
 * w_gate/w_up [ffn][d_model], w_down [d_model][ffn].  Norm gains are fp32
 * [d_model]. */
typedef struct rgd_layer_weights {
  const void* attn_norm;
  const void* wq;
  const void* wk;
  const void* wv;
  const void* wo;
  const void* ffn_norm;
  const void* w_gate;
  const void* w_up;
  const void* w_down;
} rgd_layer_weights;

/* embed [vocab][d_model] and lm_head [vocab][d_model] in the model dtype,
 * final_norm fp32 [d_model]; layers is a host array of n_layers entries. */
typedef struct rgd_weights {
  const void* embed;
  const void* final_norm;
  const void* lm_head;
  const rgd_layer_weights* layers;
} rgd_weights;

/* Library version string (static storage). */
const char* rgd_version(void);

/* Message for the last failing call on this thread ("" if none). */
const char* rgd_last_error(void);

/* Creates a model.  bf16 weight matrices are repacked here, once, into
 * library-owned buffers in the layout the GEMM kernels stream (16-row panels
 * of 64-wide k blocks); the caller's matrices are not read afterwards.  The
 * embedding table, the norm gains and fp32 matrices are used in place and
 * must outlive the handle.  max_rows bounds the rows of any decode step
 * (probe prompts, or prompts x branches) and the tokens processed per prefill
 * chunk; the workspace for that many rows is allocated here.  bf16 models
 * require head_dim == 128 and d_model, Hq*D, ffn multiples of 128. */
int32_t rgd_model_create(const rgd_model_config* cfg, const rgd_weights* w, int32_t max_rows,
                         rgd_model** out);
void rgd_model_destroy(rgd_model* m);

/* KV state for up to max_prompts prompts of up to max_prefix positions each.
 * All caches are KV-head-major, so the positions of one head form contiguous
 * runs; values are stored transposed (head dim before position) in blocks of
 * 64 positions.  VP = max_prefix rounded up to a multiple of 64:
 *  prefix_k: dev [n_layers][max_prompts][Hkv][max_prefix][D]
 *  prefix_v: dev [n_layers][max_prompts][Hkv][VP/64][D][64]
 *    - the shared prompt KV (rotated keys), written only by rgd_prefill_kv
 *    or by the caller, read in place by every probe and branch, never copied.
 *  pool_k: dev [n_layers][n_pages][Hkv][page_size][D]
 *  pool_v: dev [n_layers][n_pages][Hkv][D][page_size]
 *    - pages of the per-row tails (probe positions, branch positions).
 * bf16 models need page_size % 16 == 0.  The handle keeps per-prompt prefix
 * lengths, page tables and the page free list.  All four buffers are caller
 * owned. */
int32_t rgd_kv_create(const rgd_model* m, int32_t max_prompts, int32_t max_prefix, int32_t n_pages,
                      int32_t page_size, void* prefix_k, void* prefix_v, void* pool_k, void* pool_v,
                      rgd_kv** out);
void rgd_kv_destroy(rgd_kv* kv);

/* Declares that positions [0, len) of prompt `prompt` hold valid KV written by
 * the caller (e.g. a synthetic prefix).  Host-side bookkeeping only. */
int32_t rgd_kv_set_prefix_len(rgd_kv* kv, int32_t prompt, int32_t len);

/* Refusal-prefix table P (Section 3; token-level matching with a minimum match
 * length, Appendix D), copied to the device.  CSR on the host: entry e is
 * tokens[offsets[e] .. offsets[e+1]).  owner (host [n_entries] or NULL):
 * owner[e] = -1 makes the entry apply to every prompt, p >= 0 to prompt p only.
 * Entries shorter than min_match tokens never match.  n_entries may be 0 (every
 * probe is then incompatible at its first token). */
int32_t rgd_table_create(const int32_t* offsets, const int32_t* tokens, int32_t n_entries,
                         const int32_t* owner, int32_t min_match, rgd_table** out);
void rgd_table_destroy(rgd_table* t);

/* Prefill (Algorithm 1, first line; the prompt KV reused by both stages):
 * tokens dev int32 [B][n] for prompts 0..B-1 at positions
 * [start_pos, start_pos + n); each prompt must already hold start_pos valid
 * positions.  Writes their K/V into the prefix, sets each prefix length to
 * start_pos + n and writes the logits of each prompt's last position to
 * last_logits dev fp32 [B][vocab].  Asynchronous. */
int32_t rgd_prefill_kv(rgd_model* m, rgd_kv* kv, const int32_t* tokens, int32_t B, int32_t n,
                       int32_t start_pos, float* last_logits, rgd_stream stream);

/* rgd_prefill_kv plus the residual-stream classifier pre-check (Appendix A):
 * for each prompt b, scores[b] = 1 / (1 + exp(-(cls_w . h_b + cls_b))) where
 * h_b is the fp32 residual stream of the prompt's last position after block
 * cls_layer (1..n_layers; 0 = the embedding).  cls_w dev fp32 [d_model]
 * (caller-owned), scores dev fp32 [B].  The logits and the KV written are those
 * of rgd_prefill_kv.  Asynchronous. */
int32_t rgd_prefill_kv_scored(rgd_model* m, rgd_kv* kv, const int32_t* tokens, int32_t B, int32_t n,
                              int32_t start_pos, float* last_logits, int32_t cls_layer, const float* cls_w,
                              float cls_b, float* scores, rgd_stream stream);

/* Greedy probe (Algorithm 1: the c-token gate G_M and the post-cap probe B_M)
 * for prompts 0..B-1.  Token 1 is the argmax of last_logits (dev fp32
 * [B][vocab]); each further token is the argmax after feeding the probe, whose
 * K/V goes to pages of the prompt's probe tail.  After every token the probe
 * is checked against tbl: incompatible -> INCOMPAT, token == eos_id (eos_id <
 * 0: none) -> STOP, k tokens -> MAXLEN.  The host polls the device state after
 * each of the first c tokens and then every c tokens, and stops launching
 * steps once no prompt is undecided (early exit); the decision does not depend
 * on c.  Outputs (dev): probe_tokens int32 [B][k], probe_len int32 [B],
 * event int32 [B] (rgd_event).  Synchronous.  tbl NULL: no refusal set, every
 * probe stays compatible, so the probe runs to k tokens (or eos): the
 * fixed-length probe of the paper's ablations.  On success the probe tails are
 * held until rgd_gate; a probe that fails after validation (a HIP error) waits
 * for its stream and releases them itself. */
int32_t rgd_probe(rgd_model* m, rgd_kv* kv, const float* last_logits, const rgd_table* tbl,
                  int32_t B, int32_t k, int32_t c, int32_t eos_id, int32_t* probe_tokens,
                  int32_t* probe_len, int32_t* event, rgd_stream stream);

/* Probe without the compatibility gate (Appendix B's fixed-probe ablation;
 * with k = L, the naive greedy-then-high-temperature approach of Section 3):
 * greedy decoding always runs to k tokens, or to eos_id when it is set, and
 * the refusal detector (the table's compatibility predicate, tbl NULL = no
 * refusal set, every probe passes) is applied to the finished probe: event
 * INCOMPAT when the probe is incompatible with every entry (a miss), else
 * STOP or MAXLEN (a hit).  By prefix closure the decision equals rgd_probe's;
 * only the decoded tokens differ (k instead of stopping at the first
 * incompatible one).  Arguments, outputs, page use and the c cadence (host
 * polls after tokens 1..c and every c tokens, which only ends prompts that
 * reached eos) as rgd_probe.  Synchronous. */
int32_t rgd_probe_fixed(rgd_model* m, rgd_kv* kv, const float* last_logits, const rgd_table* tbl,
                        int32_t B, int32_t k, int32_t c, int32_t eos_id, int32_t* probe_tokens,
                        int32_t* probe_len, int32_t* event, rgd_stream stream);

/* Probe with the soft compatibility gate (Appendix C, the soft-gate
 * algorithm); arguments and outputs as rgd_probe.  Tokens 1..c are soft steps:
 * when the greedy token would make the probe incompatible, the topk most
 * probable next tokens (softmax of the logits at temperature 1 over the whole
 * vocabulary; equal logits: lower id first) are examined, and if those that
 * keep the probe compatible carry a probability mass >= rho, the most probable
 * of them is appended instead and the probe goes on.  Otherwise the failing
 * greedy token is recorded with event INCOMPAT.  Tokens after c follow the
 * hard rule of rgd_probe (there c only sets the polling cadence; here it is
 * also the number of soft steps).  1 <= topk <= 32 and topk <= vocab; rho is
 * any non-NaN value (rho > 1 never accepts: the hard gate).  The probe tokens
 * then hold the substituted tokens, which is what a hit returns.
 * Synchronous. */
int32_t rgd_probe_soft(rgd_model* m, rgd_kv* kv, const float* last_logits, const rgd_table* tbl,
                       int32_t B, int32_t k, int32_t c, int32_t eos_id, int32_t topk, float rho,
                       int32_t* probe_tokens, int32_t* probe_len, int32_t* event, rgd_stream stream);

/* The adaptive gate (Appendix A): prompts whose pre-check score (scores dev
 * fp32 [B], from rgd_prefill_kv_scored) is <= theta skip the greedy check: they
 * get event RGD_EVENT_SKIPPED and probe_len 0 (a miss for rgd_gate, sampled
 * without any check token); the others are probed as by rgd_probe (topk 0) or
 * rgd_probe_soft (topk >= 1, with rho).  Synchronous. */
int32_t rgd_probe_adaptive(rgd_model* m, rgd_kv* kv, const float* last_logits, const rgd_table* tbl,
                           int32_t B, int32_t k, int32_t c, int32_t eos_id, int32_t topk, float rho,
                           const float* scores, float theta, int32_t* probe_tokens, int32_t* probe_len,
                           int32_t* event, rgd_stream stream);

/* Gate (Algorithm 1, the return branches): prompt b is a hit (return the
 * greedy probe) iff event[b] is STOP or MAXLEN, otherwise (INCOMPAT, SKIPPED)
 * a miss (sample from the prompt).  Releases every probe-tail page (the probe's K/V is dropped,
 * never copied; the shared prefix is untouched).  event dev int32 [B].
 * decision_host int32 [B] (1 = hit, 0 = miss), *n_miss_host, miss_idx_host
 * int32 [B] (first *n_miss_host entries: missed prompts in increasing order).
 * Synchronous. */
int32_t rgd_gate(rgd_kv* kv, const int32_t* event, int32_t B, int32_t* decision_host,
                 int32_t* n_miss_host, int32_t* miss_idx_host, rgd_stream stream);

/* S_{T,theta}(M, p) (Section 3) with temperature-scaled min-p truncation for
 * the n prompts listed in prompt_idx (host int32 [n]), N branches each, `steps`
 * tokens per branch.  Branch j of listed prompt i is row r = i*N + j; it uses
 * Philox key seeds[r] (dev uint64 [n*N]) and counter (s, 0) for token s.
 * Token 0 is drawn from last_logits (dev fp32 [B][vocab], row prompt_idx[i]);
 * token s >= 1 from the logits after feeding token s-1 at position
 * prefix_len + s - 1 (the branch restarts from the prompt; probe positions are
 * not visible).  T == 0 is greedy argmax.  A token i is kept iff
 * exp((z_i - max z)/T) >= min_p; the draw is the smallest kept id whose running
 * kept weight exceeds u * (total kept weight).
 *  forced (dev int32 [n*N][steps] or NULL): if given, token forced[r][s-1] is
 *    fed at step s instead of the drawn one (teacher forcing for tests).
 *  logits_tap (dev fp32 [steps][n*N][vocab] or NULL): receives every step's
 *    logits (tests).
 *  out: dev int32 [n][N][steps].
 * Asynchronous.  Requires every probe tail to have been released (rgd_gate). */
int32_t rgd_sample_continuations(rgd_model* m, rgd_kv* kv, const float* last_logits,
                                 const int32_t* prompt_idx, int32_t n, int32_t N, int32_t steps,
                                 float T, float min_p, const uint64_t* seeds, const int32_t* forced,
                                 float* logits_tap, int32_t* out, rgd_stream stream);

/* As rgd_sample_continuations, with p-less truncation in place of min-p (the
 * truncation Section 4 samples with; its rule, from the cited p-less paper:
 * with p = softmax(z/T), keep token i iff p_i >= sum_j p_j^2, which is
 * exp((z_i - max z)/T) >= S2/S1 for S1, S2 the sums of those weights and of
 * their squares).  No parameter besides T; T == 0 is greedy argmax.  The
 * vocabulary must be a multiple of 4 (RGD_E_UNSUPPORTED otherwise). */
int32_t rgd_sample_continuations_pless(rgd_model* m, rgd_kv* kv, const float* last_logits,
                                       const int32_t* prompt_idx, int32_t n, int32_t N, int32_t steps,
                                       float T, const uint64_t* seeds, const int32_t* forced,
                                       float* logits_tap, int32_t* out, rgd_stream stream);

/* Checks the device status flag raised by the sampler (non-finite row
 * maximum) and clears it.  Synchronous. */
int32_t rgd_check_status(rgd_model* m, rgd_stream stream);

/* ---- in-situ kernel timing (measurement hooks for the benchmark) ---- */

/* Timed units: the LM-head GEMM; the whole attention stage (shared-prefix
 * kernel, tail kernel and combine); the shared-prefix attention kernel alone;
 * the min-p sampler kernel of a decode step; one whole decode step (all layers,
 * LM head and token selection). */
enum rgd_timer {
  RGD_TIMER_LM_HEAD = 0,
  RGD_TIMER_ATTENTION = 1,
  RGD_TIMER_ATTN_PREFIX = 2,
  RGD_TIMER_SAMPLER = 3,
  RGD_TIMER_STEP = 4,
  RGD_TIMER_COUNT = 5
};

/* period >= 1: from now on the model records HIP events on the work stream
 * around timed units.  Inside rgd_sample_continuations, decode step s (s >= 1)
 * is timed when (s - 1) % period == 0, and only one unit is timed in such a
 * step: unit ((s - 1) / period) % RGD_TIMER_COUNT (LM head, attention stage,
 * shared-prefix attention kernel, sampler, whole step, in turn), so that no
 * unit's measurement holds another unit's event records; the draw from the
 * prompt's logits is never timed.  Elsewhere every launch of every unit is
 * timed (the prefix kernel's events then sit inside the attention stage's).
 * At most 8192 timed launches per unit between reads; later launches are not
 * timed.  Each event record leaves a small idle gap on the stream.  period == 0
 * stops recording; negative is RGD_E_INVALID_ARG.  Events are created on the
 * first enable, not on the decode path. */
int32_t rgd_timing_enable(rgd_model* m, int32_t period);

/* Waits for the recorded events and returns, per timed unit, the summed
 * duration in milliseconds (ms[RGD_TIMER_COUNT]) and the number of launches
 * (launches[RGD_TIMER_COUNT]); then clears the records.  Synchronous. */
int32_t rgd_timing_read(rgd_model* m, double* ms, int64_t* launches);

/* ---- kernel-level entry points (used by the tests and the benchmark) ---- */

/* Decode attention for R rows of one layer: q dev [R][Hq][D] (model dtype)
 * over prompt row_prompt[r]'s first plen[r] prefix positions followed by
 * tail_len positions of the row's own tail.  row_prompt and plen are HOST int32
 * [R]; rows of one prompt must be contiguous.  prefix_k, prefix_v, pool_k,
 * pool_v are one layer of the layouts of rgd_kv_create; pages dev int32
 * [R][max_pages] (may be NULL when tail_len == 0).  out dev
 * [R][Hq*D] (model dtype).  splits = 0 picks the prefix split count.
 * Asynchronous. */
int32_t rgd_kernel_attention(rgd_model* m, const void* q, int32_t R, const int32_t* row_prompt,
                             const int32_t* plen, const void* prefix_k, const void* prefix_v,
                             int32_t max_prompts, int32_t max_prefix, const void* pool_k,
                             const void* pool_v, int32_t page_size, const int32_t* pages,
                             int32_t max_pages, int32_t tail_len, int32_t splits, void* out,
                             rgd_stream stream);

/* LM head: logits dev fp32 [R][vocab] = h W_lm^T with h dev [R][d_model]
 * (model dtype, the already normalised final hidden state).  Asynchronous. */
int32_t rgd_kernel_lm_head(rgd_model* m, const void* h, int32_t R, float* logits, rgd_stream stream);

/* Bytes of caller-provided device workspace the sampler entry points below
 * need for R rows of V logits. */
uint64_t rgd_sampler_workspace_bytes(int32_t R, int32_t V);

/* Greedy token of each row of z dev fp32 [R][V] (first index of the maximum)
 * -> out dev int32 [R].  workspace: dev, rgd_sampler_workspace_bytes(R, V)
 * bytes, 256-byte aligned.  Asynchronous. */
int32_t rgd_kernel_argmax(const float* z, int32_t R, int32_t V, void* workspace, int32_t* out,
                          rgd_stream stream);

/* min-p draws on z dev fp32 [R][V] (V a multiple of 4, V <= 1048576, T > 0,
 * 0 <= min_p <= 1): draw d of row r uses Philox key seeds[r] (dev uint64 [R])
 * and counter (ctr, stream0 + d); out dev int32 [R][draws].  workspace as for
 * rgd_kernel_argmax.  Asynchronous. */
int32_t rgd_kernel_sample(const float* z, int32_t R, int32_t V, float T, float min_p,
                          const uint64_t* seeds, uint32_t ctr, uint32_t stream0, int32_t draws,
                          void* workspace, int32_t* out, rgd_stream stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the draws of
 * rgd_kernel_sample, same arguments without the workspace, which is taken from
 * a fixed array of RGD_NOALLOC_SCRATCH_BYTES the library holds on each device
 * it runs on until the process ends.  Allocates nothing.  Calls with
 * rgd_sampler_workspace_bytes(R, V) > RGD_NOALLOC_SCRATCH_BYTES are rejected
 * (RGD_E_INVALID_ARG) before any HIP call.  Every call on one device shares
 * that array: calls that overlap on one device (several streams or threads)
 * race and must be serialised by the caller.  The first call on a device
 * looks up the array's device address (hipGetSymbolAddress) with that device
 * current.  Asynchronous. */
#define RGD_NOALLOC_SCRATCH_BYTES 1048576
int32_t rgd_kernel_sample_noalloc(const float* z, int32_t R, int32_t V, float T, float min_p,
                                  const uint64_t* seeds, uint32_t ctr, uint32_t stream0, int32_t draws,
                                  int32_t* out, rgd_stream stream);

/* p-less draws on z dev fp32 [R][V] (keep p_i >= sum_j p_j^2 of softmax(z/T),
 * see rgd_sample_continuations_pless; V a multiple of 4, V <= 1048576,
 * T > 0); seeds, counters, workspace and out as for rgd_kernel_sample.
 * Asynchronous. */
int32_t rgd_kernel_sample_pless(const float* z, int32_t R, int32_t V, float T, const uint64_t* seeds,
                                uint32_t ctr, uint32_t stream0, int32_t draws, void* workspace,
                                int32_t* out, rgd_stream stream);

/* One probe step (Algorithm 1, or the soft gate of Appendix C when topk > 0)
 * for prompts 0..R-1 of the table, given their next-token logits dev fp32
 * [R][vocab of m] and their probe state probe_tokens dev int32 [R][k],
 * probe_len, event dev int32 [R] (updated in place; prompts whose event is
 * not -1 are left alone): appends one token and sets the event as rgd_probe
 * and rgd_probe_soft do for their step (c: soft steps when topk > 0; tbl NULL:
 * no table).  Uses m's workspace, so calls on one model must not overlap.
 * Asynchronous. */
int32_t rgd_kernel_probe_step(rgd_model* m, const float* logits, int32_t R, const rgd_table* tbl,
                              int32_t k, int32_t c, int32_t eos_id, int32_t topk, float rho,
                              int32_t* probe_tokens, int32_t* probe_len, int32_t* event,
                              rgd_stream stream);

#ifdef __cplusplus
}
#endif

#endif /* RGD_H */
