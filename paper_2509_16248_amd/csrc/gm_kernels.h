// gm_kernels.h -- host-side launch functions of the libgm kernels.
// Every function only enqueues on `stream`; none synchronises.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gm {

enum DType : int { kF32 = 0, kBF16 = 1, kF16 = 2 };

// GEMM epilogues.  The GEMM computes acc[m][n] = sum_k A[m][k] * W[n][k] over
// packed weight rows n; the epilogue turns it into the stored output.
enum Epi : int {
  kEpiStore = 0,      // out[m][n] = R(acc + bias)
  kEpiGelu = 1,       // out[m][n] = R(gelu(acc + bias))
  kEpiGatedGelu = 2,  // rows interleaved in 16-row groups (gate, up):
  kEpiGatedSilu = 3,  //   out[m][j] = R(act(gate_j) * up_j)
  kEpiResid = 4,      // out[m][n] = R(resid[m][n] + acc + bias), clamp-site max
  kEpiRope = 5,       // q,k rows interleaved per head in 16-row groups (i, i+hd/2);
                      //   rotate-half rotary on q and k, plain store of v
};

struct GemmArgs {
  int dtype;
  int M, N, K;              // N counts packed weight rows
  const void* A; int lda;   // [M, K]
  const void* W; int ldw;   // [N, K]
  int epi;
  const void* bias;         // [N] packed order, or null
  void* out; int ldo;
  const void* resid; int ldr;
  int32_t* state; int site; // clamp-site reduction target (site < 0: none)
  const float* rope_cos; const float* rope_sin; int rope_rows;
  int rope_set_stride;      // long/short select: the long set starts this many
                            // floats later, used when state[kRopeLong]
  int seq;                  // positions are m % seq, or pos[m] when pos is set
  const int32_t* pos;       // per-row positions (decode step), or null
  int head_dim; int d_model;
  // decode step, QKV projection only (kc != null): the k and v columns of
  // row b are also stored at position pos[b] of the KV cache
  // ([B][H][kv_max_seq][head_dim]) and the position marked valid, unless the
  // step trapped
  void* kc; void* vc; uint8_t* kv_valid; int kv_max_seq; int heads;
};
// M <= 16 rows (a decode step, or a tiny forward) runs on a weight-streaming
// kernel; larger M on the tiled MFMA kernel.
void launch_gemm(const GemmArgs& a, hipStream_t s);

struct AttnArgs {
  int dtype;
  int B, Sq, Sk, H, hd, d;
  const void* q; int ldq;   // query (b, i) at row b*Sq + i, head h at columns h*hd
  const void* k; const void* v; int ldkv;   // key/value (b, j) at row b*Sk + j
  void* ctx;                // [B*Sq, d]
  const int32_t* mask;      // [B, Sk] key mask
  const int32_t* state;     // the padding flag state[pad_slot] and the key
  int pad_slot, kvlen_base; // lengths state[kvlen_base + b]
  int causal;               // self-attention only (Sq == Sk): keys j <= i
  float scale;              // 1/sqrt(hd)
};
void launch_attention(const AttnArgs& a, hipStream_t s);

// The forward's guards and predicates (see k_prologue).  expected != null
// adds the mask-equality guard (trap 5): guard_meta_ok is the host's shape
// check of expected against [B, S].  log_vals > 0 zeroes that many floats of
// log_stage (per-forward tensor log values).  rope_orig > 0: long/short
// rotary frequency select, long when max(position) + 1 > rope_orig.
// second != 0: the second input of an encoder-decoder forward (the target):
// its guards join the trap word already set by the first, with positions
// offset by index_offset; its padding predicate goes to the target slots and
// its key lengths to state[kvlen_base + b]; nothing else is touched.
void launch_prologue(const int32_t* ids, const int32_t* mask, int B, int S,
                     int vocab, int rotary, int capacity, int n_sites,
                     const int32_t* expected, int guard_meta_ok,
                     float* log_stage, int log_vals, int rope_orig,
                     int32_t* state, hipStream_t s, int second = 0, int index_offset = 0,
                     int kvlen_base = 0);

// Tensor-valued log at layer `layer`: stage[layer*B + b] = max |x| over the
// rows of sequence b of x [B*S, d] (NaN if any element is NaN), as float bits
// reduced with integer max.  stage must be zero before the first call.
// clamp_site >= 0: that site's clamp select, if it tripped, applies to x.
void launch_log_seqmax(const void* x, int dtype, int B, int S, int d, float* stage, int layer,
                       const int32_t* state, int clamp_site, float clamp_thr, hipStream_t s);

void launch_rope_fill(float* cos, float* sin, int head_dim, double base,
                      const int32_t* state, hipStream_t s);

// Rows [0, rows) of a frequency set scaled by factor[hd/2] (device fp32),
// cos/sin multiplied by attn.
void launch_rope_fill_scaled(float* cos, float* sin, int head_dim, double base,
                             const float* factor, float attn, int rows, hipStream_t s);

struct RowArgs {
  int dtype;
  int rows, d;
  // source: embedding gather (ids != null) or a [rows, d] tensor x
  const int32_t* ids; const void* tok_emb; const void* pos_emb; int seq; int vocab;
  const int32_t* pos;       // embedding positions per row (decode step), or null: row % seq
  void* x;                  // embedding: written with R(emb); else read (and clamped in place)
  int norm;                 // -1 none, 0 LayerNorm, 1 RMSNorm
  const void* g; const void* b; float eps;
  void* out;                // normalised output (may equal x)
  int32_t* state; int clamp_site; float clamp_thr;
};
void launch_rownorm(const RowArgs& a, hipStream_t s);

// Effects of a forward in program order: pad, regrow, then per layer the two
// clamp sites and (n_log_layers > 0) the layer's tensor log of B values,
// copied from log_stage into the arena (the value at the call site).
// seq2seq: an encoder-decoder forward, whose source and target padding
// branches give PAD records with site 0 and 1.
void launch_emit_effects(int32_t* state, void* fifo, int fifo_cap, int n_sites,
                         const float* log_stage, float* arena, int arena_cap, int n_log_layers,
                         int B, int seq2seq, hipStream_t s);

// ------------------------------------------------------------ decode step
// KV cache: per layer, K and V as [max_batch][H][max_seq][hd] (act dtype) and
// one byte per (sequence, position) saying whether that key may be attended.

// Guards and positions of one decode step (one workgroup): ids in [0, vocab)
// (trap 1, index b), seqlen[b] < max_seq (trap 4, index b), rotary need =
// max_b seqlen[b] + 1 <= capacity (trap 3); pos[b] = seqlen[b] (clamped);
// rotary regrow as in the prologue; per-forward slots reset.
void launch_decode_prologue(const int32_t* ids, int B, int vocab, int max_seq, int rotary,
                            int capacity, int n_sites, const int32_t* seqlen, int32_t* pos,
                            int32_t* state, hipStream_t s);

struct KvArgs {
  int dtype;
  int rows;                 // token rows of qkv
  int S;                    // prefill: row = b*S + s; 0 for a decode step (row b at pos[b])
  const int32_t* pos;       // decode: [rows]
  const int32_t* mask;      // prefill: [B, S] key validity
  const int32_t* state;     // decode: nothing is stored when the step trapped
  const void* qkv; int d, H, hd;
  void* kc; void* vc;       // this layer's cache
  uint8_t* valid;           // [max_batch][max_seq]
  int max_seq;
};
void launch_kv_store(const KvArgs& a, hipStream_t s);

struct DecAttnArgs {
  int dtype;
  int B, H, hd, d;
  const void* qkv;          // [B, 3d]: q of sequence b at row b, head h at columns h*hd
  const void* kc; const void* vc; const uint8_t* valid; int max_seq;
  const int32_t* pos;       // keys 0 .. pos[b] of sequence b
  void* ctx;                // [B, d]
  float* part;              // [B*H*nsplit*(hd+2)] partial softmax state per key chunk
  int nsplit, chunk;        // key chunks per head (1: no merge pass) and their size
  float scale;
};
void launch_decode_attention(const DecAttnArgs& a, hipStream_t s);

// next[b] = index of the largest logit of row b (first NaN if any; lowest
// index among equal values).
void launch_argmax(const void* logits, int dtype, int B, int V, int32_t* next, hipStream_t s);

// Sequence lengths after a forward: prefill seqlen[b] = 1 + last unmasked
// key; decode seqlen[b] = pos[b] + 1 unless the step trapped.
void launch_seqlen_update(int32_t* seqlen, const int32_t* pos, const int32_t* state, int B,
                          int decode, hipStream_t s);

void launch_gather_rows(void* dst, const void* src, const int32_t* row_map,
                        int rows, int row_bytes, hipStream_t s);

}  // namespace gm
