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
  int seq;                  // positions are m % seq
  int head_dim; int d_model;
};
void launch_gemm(const GemmArgs& a, hipStream_t s);

struct AttnArgs {
  int dtype;
  int B, S, H, hd, d;
  const void* qkv;          // [B*S, 3d]: q | k | v, head h at columns h*hd
  void* ctx;                // [B*S, d]
  const int32_t* mask;      // [B, S]
  const int32_t* state;     // pad_any flag and kv_len
  int causal;
  float scale;              // 1/sqrt(hd)
};
void launch_attention(const AttnArgs& a, hipStream_t s);

void launch_prologue(const int32_t* ids, const int32_t* mask, int B, int S,
                     int vocab, int rotary, int capacity, int n_sites,
                     int32_t* state, hipStream_t s);

void launch_rope_fill(float* cos, float* sin, int head_dim, double base,
                      const int32_t* state, hipStream_t s);

struct RowArgs {
  int dtype;
  int rows, d;
  // source: embedding gather (ids != null) or a [rows, d] tensor x
  const int32_t* ids; const void* tok_emb; const void* pos_emb; int seq; int vocab;
  void* x;                  // embedding: written with R(emb); else read (and clamped in place)
  int norm;                 // -1 none, 0 LayerNorm, 1 RMSNorm
  const void* g; const void* b; float eps;
  void* out;                // normalised output (may equal x)
  int32_t* state; int clamp_site; float clamp_thr;
};
void launch_rownorm(const RowArgs& a, hipStream_t s);

void launch_emit_effects(int32_t* state, void* fifo, int fifo_cap, int n_sites,
                         hipStream_t s);

void launch_gather_rows(void* dst, const void* src, const int32_t* row_map,
                        int rows, int row_bytes, hipStream_t s);

}  // namespace gm
