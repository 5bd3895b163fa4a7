/*
 * gm.h -- C ABI of libgm: a transformer decoder/encoder forward for MI355X
 * (gfx950) in which every graph-breaking pattern is resolved on the device.
 *
 * The operation.  GraphMend ("Code Transformations for Fixing Graph Breaks in
 * PyTorch 2") rewrites three source patterns so that a model forward stays in
 * one captured graph: a validation guard `if not C: raise` becomes an
 * asynchronous device assertion (rule [Trap]); a tensor-predicated if/else
 * becomes both branches plus a select (rule [Where]); print/logger calls are
 * recorded with their arguments and replayed after the graph (rule [Defer])
 * (Table "GraphMend transformation rules"; Semantics Preservation section).
 * This library is the forward those rewrites produce, written directly for
 * the GPU: the guards on the inputs, the `mask.any()` padding branch, the
 * rotary-cache regrow on sequence length and the fp16 `abs().max()` overflow
 * clamp are device reductions that feed flags read by later kernels, so the
 * host never reads a value back during a forward.  Each forward is one
 * hipGraphLaunch on the caller's stream.
 *
 * Conventions.
 *  - Every pointer marked "device" is a HIP device pointer on the device that
 *    was current when the model was created.  Every pointer marked "host" is
 *    ordinary host memory.
 *  - Every function returns GM_OK (0) or a negative GM_E_* code.  Errors that
 *    depend on input *values* (token range, mask values, rotary capacity) are
 *    never returned by gm_forward (that would need a host sync): they set the
 *    model's sticky device trap word, read with gm_check_error (rule [Trap]:
 *    the failure surfaces at the next synchronisation point).
 *  - A model is used from one host thread and one stream at a time.
 */
#ifndef GM_H_
#define GM_H_

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GM_ABI_VERSION 2
#define GM_MAX_LAYERS 64

/* ------------------------------------------------------------ return codes */
#define GM_OK          0
#define GM_E_INVAL    -1  /* null pointer, bad shape, unsupported combination */
#define GM_E_NOMEM    -2  /* device allocation failed (gm_model_create only)  */
#define GM_E_HIP      -3  /* a HIP runtime call failed; see gm_last_error     */
#define GM_E_CAPTURE  -4  /* graph capture or instantiation failed            */
#define GM_E_TRAP     -5  /* fragmented execution only: an input guard failed */

/* ------------------------------------------------------------ enums */
enum { GM_DTYPE_F32 = 0, GM_DTYPE_BF16 = 1, GM_DTYPE_F16 = 2 };
enum { GM_NORM_LAYER = 0, GM_NORM_RMS = 1 };
enum { GM_NORM_PRE = 0, GM_NORM_POST = 1 };
enum { GM_FFN_GELU = 0, GM_FFN_GEGLU = 1, GM_FFN_SWIGLU = 2 };
enum { GM_POS_NONE = 0, GM_POS_LEARNED = 1, GM_POS_ROTARY = 2 };

/* Trap codes, in the order the guards run (smaller code = earlier guard). */
enum { GM_TRAP_NONE = 0, GM_TRAP_TOKEN_RANGE = 1, GM_TRAP_MASK_VALUE = 2,
       GM_TRAP_ROPE_CAPACITY = 3, GM_TRAP_KV_CAPACITY = 4, GM_TRAP_MASK_GUARD = 5 };

/* Execution modes (gm_set_exec_mode). */
enum { GM_EXEC_GRAPH = 0, GM_EXEC_EAGER = 1, GM_EXEC_FRAGMENTED = 2 };

/* Kinds of deferred effect records (rule [Defer]). */
enum { GM_EFFECT_PAD = 1, GM_EFFECT_REGROW = 2, GM_EFFECT_CLAMP = 3, GM_EFFECT_LOG = 4 };

/* Rotary frequency scaling (gm_config.rope_scaling). */
enum { GM_ROPE_PLAIN = 0, GM_ROPE_LONG_SHORT = 1 };

/* ------------------------------------------------------------ config
 * Model hyper-parameters.  Read only during gm_model_create.
 *  d_model % n_heads == 0; head_dim = d_model / n_heads must be 32, 64 or
 *  128; for bf16/f16 d_model and d_ff must be multiples of 64.
 *  act_dtype is the storage dtype of weights, activations and logits; all
 *  accumulation is fp32.
 *  norm_place POST applies the norm after each residual add (no final norm);
 *  PRE applies it before each block and once before the head.
 *  emb_norm applies a norm (emb_ln_g/emb_ln_b) to the embedding output.
 *  Rotary: cos/sin table of rope_capacity rows, the first rope_init_len rows
 *  built at create; a forward that needs more rows (max position + 1 >
 *  cached length) grows it on the device to exactly that length.
 *  fp16_clamp (f16 + PRE only): after each residual add, if no element is
 *  NaN and max |h| > 65504 - clamp_margin, h is clamped to that bound.
 *  kv_cache (causal models without fp16_clamp or rope_scaling): keep every
 *  layer's k and v for max_batch x max_seq positions so that gm_decode_step
 *  can extend the sequences of the last forward one token at a time.
 *  log_hidden: after every layer, record max |h| of each sequence (a [B]
 *  tensor) as a deferred log effect (GM_EFFECT_LOG) replayed after the
 *  forward (rule [Defer] with a tensor argument).
 *  rope_scaling GM_ROPE_LONG_SHORT (rotary only): two frequency sets,
 *  theta_i = 1 / (factor_i * base^(2i/hd)) with the short or the long
 *  factors (gm_weights.rope_short_factor / rope_long_factor, fp32 [hd/2]);
 *  a forward uses the long set when max(position) + 1 > rope_orig_max
 *  (rule [Where]: both tables are built at create, a device flag selects);
 *  cos and sin are scaled by rope_attn_factor.  The regrow predicate does
 *  not apply: both tables hold rope_capacity rows from the start.
 *  n_dec_layers > 0 makes an encoder-decoder model (gm_forward_seq2seq):
 *  n_layers bidirectional pre-norm encoder layers over max_seq source
 *  positions (learned positions enc_pos_emb, final norm enc_lnf), then
 *  n_dec_layers pre-norm decoder layers over max_tgt target positions, each
 *  with causal self-attention, cross-attention to the encoder output and the
 *  FFN; the token embedding is shared by both stacks.  Needs norm_place PRE,
 *  pos LEARNED, causal, and none of fp16_clamp, kv_cache, log_hidden,
 *  rope_scaling, emb_norm.
 */
typedef struct gm_config {
  int32_t abi_version;      /* must be GM_ABI_VERSION */
  int32_t n_layers, d_model, n_heads, d_ff, vocab;
  int32_t max_batch, max_seq;
  int32_t norm, norm_place, emb_norm, ffn, pos, causal, has_bias, tied_head;
  float   norm_eps;
  float   rope_base;
  int32_t rope_init_len, rope_capacity;
  int32_t act_dtype;
  int32_t fp16_clamp;
  float   clamp_margin;
  int32_t kv_cache;
  int32_t log_hidden;
  int32_t rope_scaling;
  int32_t rope_orig_max;
  float   rope_attn_factor;
  int32_t n_dec_layers, max_tgt;
} gm_config;

/* ------------------------------------------------------------ weights
 * Device pointers in PyTorch nn.Linear layout (weight [out, in], row-major),
 * dtype act_dtype.  Pointers that the config does not use must be NULL.
 *  wqkv [3d, d]  rows: q (d), k (d), v (d); bqkv [3d]
 *  wo   [d, d];  bo [d]
 *  w1   [ff, d] (GELU) or [2ff, d] (gated: gate rows first, then up rows); b1
 *  w2   [d, ff]; b2 [d]
 *  ln*_g / ln*_b [d] (b only for LayerNorm)
 *  tok_emb [vocab, d]; pos_emb [max_seq, d] (learned positions)
 *  lm_head [vocab, d] (NULL when tied_head: the head is tok_emb)
 * The library copies (and repacks) everything during gm_model_create; the
 * caller may free its buffers when that call returns.
 */
typedef struct gm_layer_weights {
  const void *ln1_g, *ln1_b, *wqkv, *bqkv, *wo, *bo;
  const void *ln2_g, *ln2_b, *w1, *b1, *w2, *b2;
} gm_layer_weights;

/* Cross-attention of one decoder layer (encoder-decoder models):
 *  lnc_g / lnc_b [d]      pre-norm of the cross-attention block
 *  wq [d, d], bq [d]      query projection of the decoder stream
 *  wkv [2d, d], bkv [2d]  key and value projection of the encoder output
 *                         (rows: k (d), then v (d))
 *  wo [d, d], bo [d]      output projection (added to the decoder residual) */
typedef struct gm_cross_weights {
  const void *lnc_g, *lnc_b, *wq, *bq, *wkv, *bkv, *wo, *bo;
} gm_cross_weights;

typedef struct gm_weights {
  const void *tok_emb, *pos_emb, *emb_ln_g, *emb_ln_b, *lnf_g, *lnf_b, *lm_head;
  const gm_layer_weights *layers;   /* host array of n_layers entries */
  const float *rope_short_factor, *rope_long_factor;   /* device fp32 [hd/2], rope_scaling only */
  /* encoder-decoder models: layers are the encoder's n_layers layers;
   * pos_emb [max_tgt, d] and lnf_* are the decoder's; tok_emb (and lm_head)
   * are shared */
  const void *enc_pos_emb, *enc_lnf_g, *enc_lnf_b;  /* [max_seq, d], [d], [d] */
  const gm_layer_weights *dec_layers;               /* host array, n_dec_layers */
  const gm_cross_weights *dec_cross;                /* host array, n_dec_layers */
} gm_weights;

typedef struct gm_model gm_model;

/* Decisions of the last completed forward (the device predicates). */
typedef struct gm_decisions {
  int32_t pad_any;        /* mask had a 0 -> key-padding mask applied        */
  int32_t regrow;         /* rotary table grown in this forward              */
  int32_t need;           /* max(position) + 1                               */
  int32_t cached_len;     /* rotary rows valid after this forward (state)    */
  int32_t n_clamp_sites;  /* 2 * n_layers with fp16_clamp, else 0            */
  int32_t clamp[2 * GM_MAX_LAYERS];        /* site 2l: after attention, 2l+1: after FFN */
  float   clamp_absmax[2 * GM_MAX_LAYERS]; /* max |h| over non-NaN elements */
  int32_t clamp_nan[2 * GM_MAX_LAYERS];    /* some element of h was NaN     */
  int32_t forward_index;  /* 0-based count of forwards enqueued before it     */
  int32_t rope_long;      /* rope_scaling: the long frequency set was used    */
  int32_t pad_any_tgt;    /* encoder-decoder: the target mask had a 0 (pad_any
                             is then the source's)                          */
} gm_decisions;

/* One deferred effect: what the original program would have printed. */
typedef struct gm_effect {
  int32_t forward;   /* forward_index of the forward that recorded it          */
  int32_t kind;      /* GM_EFFECT_*                                            */
  int32_t layer;     /* clamp, log: layer; otherwise -1                        */
  int32_t site;      /* clamp: 0 attention, 1 FFN; log: 0; otherwise -1        */
  float   value;     /* pad: #pad positions; regrow: need; clamp: max |h|;
                        log: number of values                                  */
  int32_t n_values;  /* log: B (max |h| of each sequence); otherwise 0        */
  const float *values; /* host memory valid during the callback, or NULL      */
} gm_effect;

typedef void (*gm_effect_cb)(const gm_effect *effect, void *user);

/* Kernel kinds reported by gm_profile_forward. */
enum { GM_K_PROLOGUE = 0, GM_K_ROPE = 1, GM_K_EMBED = 2, GM_K_NORM = 3,
       GM_K_GEMM_QKV = 4, GM_K_ATTENTION = 5, GM_K_GEMM_O = 6, GM_K_GEMM_UP = 7,
       GM_K_GEMM_DOWN = 8, GM_K_GEMM_HEAD = 9, GM_K_EFFECTS = 10, GM_K_KV_STORE = 11,
       GM_K_ARGMAX = 12, GM_K_LOG = 13, GM_K_GEMM_XQ = 14, GM_K_GEMM_XKV = 15,
       GM_K_GEMM_XO = 16, GM_K_XATTN = 17 };

/* One kernel launch of a profiled forward.  flops/bytes are the launch's
 * algorithmic work (2*M*N*K for a GEMM; 4*hd*visible (query,key) pairs per
 * head for attention; bytes read + written once for the others). */
typedef struct gm_kernel_time {
  int32_t kind;      /* GM_K_*                                  */
  int32_t layer;     /* layer index, -1 outside the layer stack */
  float   ms;        /* duration between the events around it   */
  double  flops;
  double  bytes;
} gm_kernel_time;

typedef struct gm_stats {
  uint64_t forwards;         /* gm_forward / gm_forward_ex calls              */
  uint64_t captures;         /* graphs captured (cold calls)                  */
  uint64_t graph_launches;   /* hipGraphLaunch calls                          */
  uint64_t eager_forwards;   /* forwards enqueued without a graph             */
  uint64_t host_syncs_in_forward; /* sync-class HIP calls made inside a forward */
  uint64_t kernels_per_forward;   /* kernel nodes in the last captured graph  */
  uint64_t decode_steps;     /* gm_decode_step calls                          */
} gm_stats;

/* ------------------------------------------------------------ entry points */

/* Paper: the Predicated Trap Lowering Transformation (host checks of tensor
 * metadata stay on the host, value checks move to the device) and the
 * hoisted, memoised initialisation of the Semantics Preservation section.
 * Create a model on the current device: validate cfg (host checks of shapes
 * and dtypes, the static half of [Trap]), allocate weights, workspace for
 * max_batch x max_seq tokens and device state, copy and repack the weights,
 * build rotary rows [0, rope_init_len).  Synchronous.  On success *out owns
 * all of it; free with gm_model_destroy.  Returns GM_E_INVAL, GM_E_NOMEM or
 * GM_E_HIP on failure (*out is then NULL). */
int gm_model_create(const gm_config *cfg, const gm_weights *w, gm_model **out);

/* Release everything the model owns.  Synchronises the device first.  NULL
 * is ignored. */
void gm_model_destroy(gm_model *m);

/* Paper: Table "GraphMend transformation rules" ([Trap], [Where], [Defer]
 * applied to the forward) and Evaluation, "Overhead Analysis of Graph
 * Breaks" (the mended forward runs as one continuous graph with no CPU-GPU
 * synchronisation) and "Full-Graph Capture for Serving Frameworks".
 * Enqueue one forward over [max_batch, max_seq] tokens on `stream`.
 *  token_ids  device int32 [B, S] row-major, each in [0, vocab)
 *  attn_mask  device int32 [B, S] row-major, 1 = token, 0 = padding
 *  out_logits device [B, S, vocab] in act_dtype, row-major
 * All three pointers must be 16-byte aligned (GM_E_INVAL otherwise; every
 * allocator in use returns at least that).
 * Asynchronous: no host synchronisation, no device-to-host copy and no
 * allocation once the (B, S, pointers) combination has been seen; the first
 * call with a new combination captures and instantiates a graph (cold
 * start).  The buffers must stay valid until the stream reaches the end of
 * the forward.  Value errors go to the trap word (gm_check_error); the
 * logits of a trapped forward are unspecified but every access stays in
 * bounds.  Part of the work (the second half of the batch, or of a decode
 * step's sequences) runs on a stream the library owns, forked from `stream`
 * with an event after the prologue and joined back with an event before the
 * forward's closing kernels (a decode step: before its LM head, which runs
 * once over all rows): everything is complete once `stream` is.  Calls
 * that overlap on one model race (they share its workspace). */
int gm_forward(gm_model *m, const int32_t *token_ids, const int32_t *attn_mask,
               void *out_logits, hipStream_t stream);

/* Paper: as gm_forward (the transformation rules table; Evaluation,
 * "Overhead Analysis of Graph Breaks"), for any batch and sequence length.
 * As gm_forward over B <= max_batch sequences of S <= max_seq tokens.  With
 * kv_cache it also stores every position's k and v (with its mask value) and
 * sets the length of sequence b to 1 + its last unmasked position: the
 * prefill that gm_decode_step continues. */
int gm_forward_ex(gm_model *m, int32_t B, int32_t S, const int32_t *token_ids,
                  const int32_t *attn_mask, void *out_logits, hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops, harnesses that forbid hipMalloc): the forward of
 * gm_forward_ex enqueued directly on `stream`, kernel by kernel (so a
 * caller's stream capture records it), as one branch, with its activation
 * workspace (h, a, qkv, ctx, f, and tmp for post-norm models) taken from a
 * static device array of the library instead of the model's buffers.  It
 * calls no allocating routine.  Same arguments, results, decisions, effects
 * and trap behaviour as gm_forward_ex.
 *  Limit: B * S * (6 * d_model + d_ff) elements of act_dtype (each buffer
 *  rounded up to 256 bytes; 7 * d_model for post-norm models) must fit in
 *  the 64 MiB array, else GM_E_INVAL with the sizes in gm_last_error.
 *  The current device must be the model's device.
 *  The array is one per device, shared by every call on that device (of
 *  any model) and it keeps the last call's contents (the forward writes
 *  every workspace element before reading it): calls that overlap on one
 *  device race.  Not for encoder-decoder models. */
int gm_forward_noalloc(gm_model *m, int32_t B, int32_t S, const int32_t *token_ids,
                       const int32_t *attn_mask, void *out_logits, hipStream_t stream);

/* Paper: Evaluation, "Experimental Setup" (text models generate greedily
 * token by token) and "Throughput Improvement"; the rotary-cache regrow of
 * the Motivation's Phi-4 example fires mid-generation (rule [Where]).
 * One decode step (kv_cache models): append token_ids[b] to sequence b at
 * position p_b = its current length, run the layer stack on those B rows
 * with attention over the cached keys 0..p_b (keys the prefill masked stay
 * masked), and write the logits of the new positions.  The result equals the
 * last row of a full forward over the extended sequences (causal models:
 * earlier positions do not depend on later ones).
 *  B          must equal the batch of the last gm_forward_ex
 *  token_ids  device int32 [B], each in [0, vocab)
 *  out_logits device [B, vocab] in act_dtype
 *  next_ids   device int32 [B] or NULL: greedy choice argmax_v logits[b, v]
 *             (lowest index among equal values, the first NaN if any); may
 *             equal token_ids, so that repeated steps generate greedily
 *             without the host reading anything back
 * All pointers 16-byte aligned.  Same asynchronous, one-graph-per-pointer-set
 * behaviour as gm_forward.  Guards (trap word, smallest code first): token
 * range (index b), rotary capacity, a sequence already at max_seq
 * (GM_TRAP_KV_CAPACITY, index b); a trapped step stores nothing and leaves
 * every length as it was.  The rotary regrow runs exactly as in a forward (need = max p_b + 1)
 * and is recorded as a deferred effect.  Not available in fragmented mode. */
int gm_decode_step(gm_model *m, int32_t B, const int32_t *token_ids, void *out_logits,
                   int32_t *next_ids, hipStream_t stream);

/* Paper: Evaluation, "Benchmark Suite" (encoder-decoder text models) with
 * the rules [Trap], [Where] and [Defer] applied to each of the two inputs.
 * Encoder-decoder forward (n_dec_layers > 0): the encoder over
 * src_ids/src_mask [B, S_src] (S_src <= max_seq), then the decoder over
 * tgt_ids/tgt_mask [B, S_tgt] (S_tgt <= max_tgt) attending to the encoder
 * output; out_logits [B, S_tgt, vocab].  Device int32 inputs, 16-byte
 * aligned pointers, one graph launch per call as gm_forward.  Each mask has
 * its own `mask.any()` branch (source: encoder self-attention and the
 * decoder's cross-attention; target: decoder self-attention), recorded as PAD
 * effects with site 0 (source) and 1 (target).  Guards: token ids, then
 * mask values, each over the source followed by the target (the position
 * of a target element is B * S_src + its row-major index).  Graph and eager
 * execution; not in fragmented mode. */
int gm_forward_seq2seq(gm_model *m, int32_t B, int32_t S_src, const int32_t *src_ids,
                       const int32_t *src_mask, int32_t S_tgt, const int32_t *tgt_ids,
                       const int32_t *tgt_mask, void *out_logits, hipStream_t stream);

/* Paper: Evaluation, "Profiling Methodology" (per-kernel attribution of
 * forward time).
 * Run one forward without a graph, recording a HIP event on `stream` after
 * every kernel, wait for it, and write one gm_kernel_time per launch (in
 * launch order) to out[0 .. min(cap, *n_out)).  Same kernels and results as
 * gm_forward_ex; synchronises `stream`, so it is a profiling call, not a
 * hot-path one. */
int gm_profile_forward(gm_model *m, int32_t B, int32_t S, const int32_t *token_ids,
                       const int32_t *attn_mask, void *out_logits, hipStream_t stream,
                       gm_kernel_time *out, int32_t cap, int32_t *n_out);

/* Paper: Evaluation, "Experimental Setup" (one CUDA graph per fused region
 * between breaks) and "Overhead Analysis of Graph Breaks" (a break costs a
 * stream synchronisation, a device-to-host copy and host evaluation).
 * How gm_forward runs the same kernels (same results in every mode):
 *  GM_EXEC_GRAPH (default)  one captured hipGraph per forward, no host sync;
 *  GM_EXEC_EAGER            kernels enqueued one by one, no host sync;
 *  GM_EXEC_FRAGMENTED       the unmended program the paper starts from: one
 *    captured graph per region between graph breaks, and at every break a
 *    hipStreamSynchronize, a device-to-host copy of the predicate's inputs
 *    and the branch evaluated on the host (after the input guards / padding
 *    / rotary predicates, and after every fp16 clamp site).  A failed guard
 *    ends the forward there and returns GM_E_TRAP (the original `raise`).
 *    Synchronous; for comparisons only (Evaluation, "Overhead Analysis of
 *    Graph Breaks": sync + D2H copy + host evaluation per break). */
int gm_set_exec_mode(gm_model *m, int32_t mode);

/* gm_set_exec_mode(m, enabled ? GM_EXEC_GRAPH : GM_EXEC_EAGER). */
int gm_set_graph_mode(gm_model *m, int32_t enabled);

/* Paper: rule [Where] (Predicated Data-dependent Control Flow
 * Transformation): the predicate values the original program's host `if`
 * would have read, computed on the device.
 * Copy the decisions of the last forward enqueued on `stream` into *out.
 * Synchronises `stream`; not for use inside a timed loop. */
int gm_read_decisions(gm_model *m, gm_decisions *out, hipStream_t stream);

/* Paper: rule [Where]; the predicate tensors stay on the device.
 * Device address of the model's int32 decision slots, for zero-sync reads by
 * later kernels: [0] pad_any, [1] regrow, [2] need, [3] cached_len. */
const int32_t *gm_decisions_device_ptr(const gm_model *m);

/* Paper: Predicated Validation Guards paragraph, Figure "guard_example",
 * Predicated Trap Lowering Transformation.
 * Validation guard `if not torch.equal(attn_mask, expected): raise
 * ValueError("unsupported attention mask")` on every later forward, lowered
 * as in rule [Trap]: the host checks the metadata (expected is int32 [B, S];
 * a forward of another shape fails the guard), the device checks
 * (attn_mask == expected).all() and sets trap GM_TRAP_MASK_GUARD at the
 * first differing element.  expected: device, 16-byte aligned, valid while
 * the guard is set; NULL removes the guard.  Synchronises the device and
 * drops the cached graphs (they hold the previous guard). */
int gm_set_mask_guard(gm_model *m, const int32_t *expected, int32_t B, int32_t S);

/* Paper: Predicated Trap Lowering Transformation (the uid that maps a
 * device trap back to the original exception).
 * The original exception of a trap code ("uid" of rule [Trap]): its Python
 * type name and message, for the caller to raise when gm_check_error
 * reports the code.  Static strings. */
int gm_trap_info(int32_t code, const char **exception_type, const char **message);

/* Paper: rule [Trap]: a failed guard is reported at the next
 * synchronisation point (Predicated Trap Lowering Transformation).
 * Return and clear the sticky trap word: *code = GM_TRAP_* of the first
 * failing guard of the first trapped forward since the last call, *index =
 * row-major position of the first offending element (0 for the rotary
 * capacity).  Synchronises the device. */
int gm_check_error(gm_model *m, int32_t *code, int32_t *index);

/* Paper: rule [Defer] (Deferred Side Effect Transformation): effects are
 * recorded with their arguments during the graph and replayed in FIFO order
 * after it.
 * Replay the deferred effect records in FIFO order through cb (which may be
 * NULL to discard them) and empty the buffer.  *n_dropped (may be NULL)
 * receives the number of records lost to overflow since the last flush.
 * Synchronises the device. */
int gm_flush_effects(gm_model *m, gm_effect_cb cb, void *user, int32_t *n_dropped);

/* No passage: test instrumentation for per-layer parity.
 * The forward of gm_forward_ex (pre-norm models), enqueued on `stream`
 * without a graph and as one branch, copying every layer's storage points
 * into `dump` (device, 16-byte aligned, at least
 * n_layers * T * (8 * d_model + d_ff) elements of act_dtype, T = B * S):
 * layer l's block starts at element l * T * (8d + ff) and holds, row-major,
 *   a1 [T, d]     the first norm's output (with the preceding clamp site's
 *                 select applied to the stream it reads),
 *   qkv [T, 3d]   q | k | v after the projection epilogue (rotary applied),
 *   ctx [T, d]    the attention context,
 *   h_mid [T, d]  the stream after the attention residual (before the clamp
 *                 site's select, which the next norm applies),
 *   a2 [T, d]     the second norm's output,
 *   f [T, ff]     the FFN hidden after the activation or gate product,
 *   h_out [T, d]  the stream after the FFN residual (before its select).
 * Asynchronous (no host sync); the logits, decisions and effects are those
 * of an ordinary forward.  Not for the hot path. */
int gm_debug_forward_layers(gm_model *m, int32_t B, int32_t S, const int32_t *token_ids,
                            const int32_t *attn_mask, void *out_logits, hipStream_t stream,
                            void *dump, uint64_t dump_bytes);

/* No passage: inspection plumbing for tests.
 * Device address and size in bytes of an internal activation buffer, for
 * inspection after the stream has completed a forward (debugging and
 * tests).  which: 0 residual stream h [T, d], 1 norm output [T, d],
 * 2 fused q|k|v [T, 3d], 3 attention context [T, d], 4 FFN hidden [T, d_ff]
 * (T = max_batch * max_seq rows, act_dtype).  Contents are those left by the
 * last kernel that wrote the buffer. */
int gm_debug_buffer(const gm_model *m, int32_t which, void **ptr, uint64_t *bytes);

/* Paper: Evaluation, "Overhead Analysis of Graph Breaks" and "Steady-State
 * Forward Pass Speedup": the counters show what a forward costs on the host
 * (graph launches; sync-class HIP calls, which must stay 0 in a forward).
 * Host counters (no device access). */
int gm_get_stats(const gm_model *m, gm_stats *out);

/* Static description of a return code, and the last HIP error message of
 * the calling thread. */
const char *gm_strerror(int code);
const char *gm_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* GM_H_ */
