// gm_runtime.cpp -- host runtime behind include/gm.h: configuration checks,
// weight copy and repack, workspace and device state, the single-stream
// enqueue of one forward, hipGraph capture with an exec cache, and the
// synchronising readers (decisions, trap word, deferred effects).
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "gm.h"
#include "gm_device.h"
#include "gm_kernels.h"

namespace gm {
void attention_set_order(int o);
}

using namespace gm;

namespace {

thread_local std::string g_last_error;

int hip_fail(hipError_t e, const char* what) {
  g_last_error = std::string(what) + ": " + hipGetErrorString(e);
  return GM_E_HIP;
}
int inval(const char* what) {
  g_last_error = what;
  return GM_E_INVAL;
}

#define HIP_TRY(call)                                   \
  do {                                                  \
    hipError_t e_ = (call);                             \
    if (e_ != hipSuccess) return hip_fail(e_, #call);   \
  } while (0)

struct LayerBufs {
  void *ln1_g = nullptr, *ln1_b = nullptr, *wqkv = nullptr, *bqkv = nullptr;
  void *wo = nullptr, *bo = nullptr, *ln2_g = nullptr, *ln2_b = nullptr;
  void *w1 = nullptr, *b1 = nullptr, *w2 = nullptr, *b2 = nullptr;
};

struct GraphEntry {
  int kind;                 // 0 forward, 1 decode step, 2 encoder-decoder forward
  int B, S;
  const void *ids, *mask;
  void* logits;
  void* next;
  hipGraphExec_t exec;
  uint64_t last_use;
  int S2 = 0;               // encoder-decoder: the target's length and inputs
  const void *ids2 = nullptr, *mask2 = nullptr;
};

struct CrossBufs {
  void *lnc_g = nullptr, *lnc_b = nullptr, *wq = nullptr, *bq = nullptr;
  void *wo = nullptr, *bo = nullptr;
};

// A decode step's extra launch parameters.
struct Dec {
  int32_t* next;            // greedy token per sequence, or null
};

constexpr int kFifoCap = 4096;
constexpr int kLogArenaCap = 1 << 20;   // floats of tensor log payload between flushes
constexpr int kMaxGraphs = 8;

}  // namespace

// Static device scratch of gm_forward_noalloc (each device holds its own copy
// for the life of the process).  In host code `scratch` names a host-side
// stand-in: kernels get the device address from hipGetSymbolAddress, taken
// once per device at model creation and kept in g_scratch_ptr.
constexpr size_t kScratchBytes = size_t(64) << 20;
static __device__ __align__(256) char scratch[kScratchBytes];
constexpr int kMaxDevices = 64;
static void* g_scratch_ptr[kMaxDevices] = {};
static std::mutex g_scratch_mu;

// Device address of this device's scratch array (current device = dev).
static int scratch_for_device(int dev, void** out) {
  if (dev < 0 || dev >= kMaxDevices) return inval("device ordinal out of range for the scratch table");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return hip_fail(e != hipSuccess ? e : hipErrorInvalidSymbol,
                                               "hipGetSymbolAddress(scratch)");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return GM_OK;
}

struct gm_model {
  gm_config cfg;
  int device = 0;
  int dtype = 0;
  size_t esz = 0;
  std::vector<void*> allocs;
  void *tok_emb = nullptr, *pos_emb = nullptr, *emb_ln_g = nullptr, *emb_ln_b = nullptr;
  void *lnf_g = nullptr, *lnf_b = nullptr, *head = nullptr;
  std::vector<LayerBufs> layers;
  void *h = nullptr, *a = nullptr, *qkv = nullptr, *ctx = nullptr, *f = nullptr, *tmp = nullptr;
  int32_t* state = nullptr;
  int n_state = 0;
  float *rope_cos = nullptr, *rope_sin = nullptr;
  void* fifo = nullptr;
  hipStream_t cap_stream = nullptr;
  // further batch-part branches of a forward: their streams and the
  // fork/join events (the branches are independent, so the GPU overlaps one
  // part's latency-bound kernels with another part's GEMMs)
  static constexpr int kMaxParts = 4;
  hipStream_t aux_stream[kMaxParts - 1] = {};
  hipEvent_t ev_fork = nullptr, ev_join[kMaxParts - 1] = {};
  int split_parts = 2;
  std::vector<GraphEntry> graphs;
  gm_stats stats;
  int exec_mode = GM_EXEC_GRAPH;
  bool last_host_pad_any = false, last_host_regrow = false, last_host_clamp = false;
  struct Frag {
    int B, S;
    const void *ids, *mask;
    void* logits;
    std::vector<hipGraphExec_t> execs;
    std::vector<int> kinds;   // what the host reads after segment i (Seg::kinds)
    int S2 = 0;               // encoder-decoder: the target's length and buffers
    const void *ids2 = nullptr, *mask2 = nullptr;
  };
  std::vector<Frag> frags;
  bool debug_sync = false;
  uint64_t tick = 0;
  // KV cache (cfg.kv_cache): per layer K and V [max_batch][H][max_seq][hd],
  // key validity [max_batch][max_seq], sequence lengths, decode positions and
  // the split-key attention workspace.
  std::vector<void*> kc, vc;
  uint8_t* kv_valid = nullptr;
  int32_t *seqlen = nullptr, *dpos = nullptr;
  float* dpart = nullptr;
  int dec_nsplit = 0;
  int cache_B = 0;          // batch of the last prefill (host-side), 0 = none
  // encoder-decoder (cfg.n_dec_layers > 0): decoder layers and their
  // cross-attention, encoder positions and final norm, the encoder output,
  // the cross queries, and k | v of every decoder layer projected from the
  // encoder output by one GEMM ([T_src, n_dec * 2d], layer l at l * 2d)
  std::vector<LayerBufs> dec_layers;
  std::vector<CrossBufs> dec_cross;
  void *enc_pos_emb = nullptr, *enc_lnf_g = nullptr, *enc_lnf_b = nullptr;
  void *wkv_all = nullptr, *bkv_all = nullptr;
  void *mem = nullptr, *qc = nullptr, *kvc = nullptr;
  // `torch.equal(mask, expected)` guard (gm_set_mask_guard): device tensor and its shape
  const int32_t* guard_expected = nullptr;
  int guard_B = 0, guard_S = 0;
  // tensor-valued deferred logs (cfg.log_hidden): per-forward values [L][max_batch]
  // and the arena the effect records point into
  float *log_stage = nullptr, *log_arena = nullptr;
  // device address of the static scratch array on this model's device
  void* scratch = nullptr;

  int alloc(void** p, size_t bytes) {
    *p = nullptr;
    if (bytes == 0) return GM_OK;
    hipError_t e = hipMalloc(p, bytes);
    if (e != hipSuccess) {
      g_last_error = std::string("hipMalloc: ") + hipGetErrorString(e);
      *p = nullptr;
      return GM_E_NOMEM;
    }
    allocs.push_back(*p);
    return GM_OK;
  }
};

namespace {

int n_sites(const gm_config& c) { return c.fp16_clamp ? 2 * c.n_layers : 0; }

int validate(const gm_config* c) {
  if (!c) return inval("cfg is NULL");
  if (c->abi_version != GM_ABI_VERSION) return inval("abi_version mismatch");
  if (c->n_layers < 1 || c->n_layers > GM_MAX_LAYERS) return inval("n_layers out of [1, 64]");
  if (c->d_model <= 0 || c->n_heads <= 0 || c->d_model % c->n_heads)
    return inval("d_model must be a positive multiple of n_heads");
  const int hd = c->d_model / c->n_heads;
  if (hd != 32 && hd != 64 && hd != 128) return inval("head_dim must be 32, 64 or 128");
  if (c->d_ff <= 0 || c->vocab <= 0) return inval("d_ff and vocab must be positive");
  if (c->act_dtype < GM_DTYPE_F32 || c->act_dtype > GM_DTYPE_F16) return inval("bad act_dtype");
  if (c->act_dtype == GM_DTYPE_F32) {
    if (c->d_model % 64 || c->d_ff % 64) return inval("d_model and d_ff must be multiples of 64");
  } else {
    if (c->d_model % 64 || c->d_ff % 64) return inval("d_model and d_ff must be multiples of 64");
  }
  if (c->max_batch < 1 || c->max_batch > 1024) return inval("max_batch out of [1, 1024]");
  if (c->max_seq < 1) return inval("max_seq must be positive");
  if (static_cast<long long>(c->max_batch) * c->max_seq >= (1ll << 24))
    return inval("max_batch * max_seq must be < 2^24");
  if (c->norm != GM_NORM_LAYER && c->norm != GM_NORM_RMS) return inval("bad norm");
  if (c->norm_place != GM_NORM_PRE && c->norm_place != GM_NORM_POST) return inval("bad norm_place");
  if (c->ffn < GM_FFN_GELU || c->ffn > GM_FFN_SWIGLU) return inval("bad ffn");
  if (c->pos < GM_POS_NONE || c->pos > GM_POS_ROTARY) return inval("bad pos");
  if (!(c->norm_eps > 0.f)) return inval("norm_eps must be positive");
  if (c->pos == GM_POS_ROTARY) {
    if (c->rope_capacity < 1 || c->rope_init_len < 0 || c->rope_init_len > c->rope_capacity)
      return inval("need 0 <= rope_init_len <= rope_capacity, capacity >= 1");
    if (!(c->rope_base > 1.f)) return inval("rope_base must be > 1");
  }
  if (c->fp16_clamp) {
    if (c->act_dtype != GM_DTYPE_F16) return inval("fp16_clamp needs act_dtype f16");
    if (c->norm_place != GM_NORM_PRE) return inval("fp16_clamp needs pre-norm");
    if (!(c->clamp_margin >= 0.f) || c->clamp_margin >= 65504.f) return inval("bad clamp_margin");
  }
  if (c->kv_cache) {
    if (!c->causal) return inval("kv_cache needs a causal model");
    if (c->fp16_clamp) return inval("kv_cache is not supported with fp16_clamp");
    if (c->rope_scaling) return inval("kv_cache is not supported with rope_scaling");
  }
  if (c->rope_scaling != GM_ROPE_PLAIN && c->rope_scaling != GM_ROPE_LONG_SHORT)
    return inval("bad rope_scaling");
  if (c->n_dec_layers < 0 || c->n_dec_layers > GM_MAX_LAYERS) return inval("n_dec_layers out of [0, 64]");
  if (c->n_dec_layers) {
    if (c->norm_place != GM_NORM_PRE || c->pos != GM_POS_LEARNED || !c->causal || c->fp16_clamp ||
        c->kv_cache || c->log_hidden || c->rope_scaling || c->emb_norm)
      return inval("encoder-decoder models: pre-norm, learned positions, causal decoder, no "
                   "fp16_clamp, kv_cache, log_hidden, rope_scaling or emb_norm");
    if (c->max_tgt < 1) return inval("max_tgt must be positive");
    if (static_cast<long long>(c->max_batch) * c->max_tgt >= (1ll << 24))
      return inval("max_batch * max_tgt must be < 2^24");
  }
  if (c->rope_scaling) {
    if (c->pos != GM_POS_ROTARY) return inval("rope_scaling needs rotary positions");
    if (c->rope_orig_max < 1) return inval("rope_orig_max must be positive");
    if (!(c->rope_attn_factor > 0.f)) return inval("rope_attn_factor must be positive");
  }
  return GM_OK;
}

// Copy a caller tensor into library memory (optionally permuting rows).
int copy_in(gm_model* m, void** dst, const void* src, size_t rows, size_t cols,
            const std::vector<int32_t>* perm, const char* name) {
  if (!src) {
    g_last_error = std::string("weight ") + name + " is NULL";
    return GM_E_INVAL;
  }
  const size_t row_bytes = cols * m->esz;
  int rc = m->alloc(dst, rows * row_bytes);
  if (rc) return rc;
  if (!perm) {
    HIP_TRY(hipMemcpy(*dst, src, rows * row_bytes, hipMemcpyDeviceToDevice));
    return GM_OK;
  }
  if (row_bytes % 16 == 0) {
    int32_t* dmap = nullptr;
    HIP_TRY(hipMalloc(&dmap, rows * sizeof(int32_t)));
    hipError_t e = hipMemcpy(dmap, perm->data(), rows * sizeof(int32_t), hipMemcpyHostToDevice);
    if (e == hipSuccess) {
      launch_gather_rows(*dst, src, dmap, static_cast<int>(rows), static_cast<int>(row_bytes), nullptr);
      e = hipGetLastError();
    }
    if (e == hipSuccess) e = hipDeviceSynchronize();
    hipFree(dmap);
    if (e != hipSuccess) return hip_fail(e, "repack");
    return GM_OK;
  }
  // small tensors (bias vectors): permute on the host
  std::vector<unsigned char> hs(rows * row_bytes), hd(rows * row_bytes);
  HIP_TRY(hipMemcpy(hs.data(), src, hs.size(), hipMemcpyDeviceToHost));
  for (size_t r = 0; r < rows; ++r)
    memcpy(&hd[r * row_bytes], &hs[static_cast<size_t>((*perm)[r]) * row_bytes], row_bytes);
  HIP_TRY(hipMemcpy(*dst, hd.data(), hd.size(), hipMemcpyHostToDevice));
  return GM_OK;
}

// Packed order of gated FFN rows: 16 gate rows, then the 16 matching up rows.
std::vector<int32_t> gated_perm(int ff) {
  std::vector<int32_t> p(2 * ff);
  for (int n = 0; n < 2 * ff; ++n) {
    const int grp = n / 32, q = n % 32;
    p[n] = q < 16 ? grp * 16 + q : ff + grp * 16 + (q - 16);
  }
  return p;
}

// Packed order of q/k rows for rotary: inside each head, 16 rows i, then the
// 16 rows i + hd/2 they rotate with.  v rows keep their order.
std::vector<int32_t> rope_perm(int d, int hd) {
  std::vector<int32_t> p(3 * d);
  for (int n = 0; n < 3 * d; ++n) {
    if (n >= 2 * d) {
      p[n] = n;
      continue;
    }
    const int region = n / d, nr = n % d, h = nr / hd, w = nr % hd;
    const int i = (w / 32) * 16 + (w % 16);
    const bool second = (w % 32) >= 16;
    p[n] = region * d + h * hd + (second ? i + hd / 2 : i);
  }
  return p;
}

// Per-launch event timing for gm_profile_forward: an event is recorded on
// the launch stream after every kernel, with the kernel kind, its layer and
// its algorithmic work.
struct Prof {
  hipStream_t s;
  std::vector<hipEvent_t> ev;
  std::vector<gm_kernel_time> rec;
  bool ok = true;
  void start() { mark_event(); }
  void mark_event() {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) {
      ok = false;
      return;
    }
    hipEventRecord(e, s);
    ev.push_back(e);
  }
  void mark(int kind, int layer, double flops, double bytes) {
    gm_kernel_time r;
    r.kind = kind;
    r.layer = layer;
    r.ms = 0.f;
    r.flops = flops;
    r.bytes = bytes;
    rec.push_back(r);
    mark_event();
  }
};

// Activation workspace of one forward (h, a, qkv, ctx, f and, post-norm,
// tmp): the model's own buffers, or carved from the static scratch array of
// gm_forward_noalloc.
struct Work {
  void *h = nullptr, *a = nullptr, *qkv = nullptr, *ctx = nullptr, *f = nullptr, *tmp = nullptr;
};

// Storage points of every layer, copied during a debug forward
// (gm_debug_forward_layers) into one caller buffer: per layer, in elements
// of the activation dtype, a1 [T, d] | qkv [T, 3d] | ctx [T, d] |
// h_mid [T, d] | a2 [T, d] | f [T, ff] | h_out [T, d].
struct Dump {
  char* base = nullptr;
  size_t esz = 0;
  size_t T = 0, d = 0, ff = 0;
  size_t layer_elems() const { return T * (8 * d + ff); }
  void copy(int layer, int which, const void* src, hipStream_t s) const {
    static const int kStart[7] = {0, 1, 4, 5, 6, 7, -1};   // in units of T*d (h_out after f)
    const size_t width = which == 1 ? 3 * d : which == 5 ? ff : d;
    const size_t off = which == 6 ? T * (7 * d + ff) : static_cast<size_t>(kStart[which]) * T * d;
    (void)hipMemcpyAsync(base + (layer * layer_elems() + off) * esz, src, T * width * esz,
                         hipMemcpyDeviceToDevice, s);
  }
};

// Segment selection for the fragmented (unmended) execution: the forward is
// cut at every point where the original program reads a device value back
// on the host; only the launches of segment `want` are issued (want < 0:
// all, want == kCountOnly: none, just count the cuts).
struct Seg {
  int want = -1;
  int cur = 0;
  std::vector<int> kinds;   // what the host reads at each cut (kCut*)
};
enum { kCutGuards = 0, kCutGuardsTgt = 1, kCutClamp = 1000, kCutLog = 2000 };
constexpr int kCountOnly = -2;

// One forward (dec == null: B x S tokens, with the KV cache filled when the
// model has one) or one decode step (dec != null: S == 1, one new token per
// sequence at position seqlen[b], attending to the cache).
void enqueue(gm_model* m, int B, int S, const int32_t* ids, const int32_t* mask,
             void* logits, hipStream_t s, Prof* prof = nullptr, Seg* seg = nullptr,
             const Dec* dec = nullptr, const Dump* dump = nullptr, const Work* work = nullptr) {
  const gm_config& c = m->cfg;
  Work own;
  own.h = m->h;
  own.a = m->a;
  own.qkv = m->qkv;
  own.ctx = m->ctx;
  own.f = m->f;
  own.tmp = m->tmp;
  const Work& wk = work ? *work : own;
  auto on = [&]() { return !seg || seg->want == -1 || seg->want == seg->cur; };
  auto brk = [&](int kind) {
    if (seg) {
      ++seg->cur;
      seg->kinds.push_back(kind);
    }
  };
  const int T = B * S, d = c.d_model, hd = d / c.n_heads, ff = c.d_ff;
  const int ns = n_sites(c);
  const float thr = 65504.f - c.clamp_margin;
  const bool pre = c.norm_place == GM_NORM_PRE;
  const int normk = c.norm == GM_NORM_RMS ? 1 : 0;

  const double es = static_cast<double>(m->esz);
  int cur_layer = -1;
  auto P = [&](int kind, int layer, double flops, double bytes) {
    if (prof) prof->mark(kind, layer, flops, bytes);
  };
  if (prof) prof->start();
  if (dec)
    launch_decode_prologue(ids, B, c.vocab, c.max_seq, c.pos == GM_POS_ROTARY, c.rope_capacity,
                           ns, m->seqlen, m->dpos, m->state, s);
  else if (on())
    launch_prologue(ids, mask, B, S, c.vocab, c.pos == GM_POS_ROTARY, c.rope_capacity, ns,
                    m->guard_expected, m->guard_B == B && m->guard_S == S, m->log_stage,
                    c.log_hidden ? c.n_layers * B : 0,
                    c.rope_scaling ? c.rope_orig_max : 0, m->state, s, 0, 0, kKvLenBase);
  P(GM_K_PROLOGUE, -1, 0.0, 8.0 * T);
  if (!dec) brk(kCutGuards);  // original program: guards, mask.any() and max(position_ids) read on the host
  if (c.pos == GM_POS_ROTARY && !c.rope_scaling) {
    if (on()) launch_rope_fill(m->rope_cos, m->rope_sin, hd, c.rope_base, m->state, s);
    P(GM_K_ROPE, -1, 0.0, 0.0);
  }

  RowArgs r{};
  r.dtype = m->dtype;
  r.rows = T;
  r.d = d;
  r.eps = c.norm_eps;
  r.state = m->state;
  r.clamp_thr = thr;
  // embedding (+ embedding norm)
  r.ids = ids;
  r.tok_emb = m->tok_emb;
  r.pos_emb = c.pos == GM_POS_LEARNED ? m->pos_emb : nullptr;
  r.seq = S;
  r.pos = dec ? m->dpos : nullptr;
  r.vocab = c.vocab;
  r.x = wk.h;
  r.norm = c.emb_norm ? normk : -1;
  r.g = m->emb_ln_g;
  r.b = m->emb_ln_b;
  r.out = wk.h;
  r.clamp_site = -1;
  if (on()) launch_rownorm(r, s);
  P(GM_K_EMBED, -1, 0.0, static_cast<double>(T) * d * es * (c.pos == GM_POS_LEARNED ? 3 : 2));
  r.ids = nullptr;

  // a decode step's head runs once over the whole batch after the join (one
  // pass over the head's weights instead of one per part)
  bool head_joined = false;
  // The layers and the head over sequences [b0, b0 + nb) on stream s.
  auto layers_and_head = [&](hipStream_t s, int b0, int nb) {
  const int T = nb * S;
  const size_t ro = static_cast<size_t>(b0) * S;   // first row of this part
  char* hh = static_cast<char*>(wk.h) + ro * d * m->esz;
  char* aa = static_cast<char*>(wk.a) + ro * d * m->esz;
  char* qq = static_cast<char*>(wk.qkv) + ro * 3 * d * m->esz;
  char* cc = static_cast<char*>(wk.ctx) + ro * d * m->esz;
  char* ffb = static_cast<char*>(wk.f) + ro * ff * m->esz;
  char* tt = wk.tmp ? static_cast<char*>(wk.tmp) + ro * d * m->esz : nullptr;
  char* lg = static_cast<char*>(logits) + ro * c.vocab * m->esz;
  auto norm_rows = [&](void* x, void* out, const void* g, const void* b, int site) {
    RowArgs q = r;
    q.rows = T;
    q.x = x;
    q.out = out;
    q.norm = normk;
    q.g = g;
    q.b = b;
    q.clamp_site = site;
    if (on()) launch_rownorm(q, s);
    P(GM_K_NORM, cur_layer, 0.0, 2.0 * T * d * es);
  };

  GemmArgs ga{};
  ga.dtype = m->dtype;
  ga.M = T;
  ga.state = m->state;
  ga.site = -1;
  ga.seq = S;
  ga.pos = dec ? m->dpos + b0 : nullptr;
  ga.head_dim = hd;
  ga.d_model = d;
  ga.rope_cos = m->rope_cos;
  ga.rope_sin = m->rope_sin;
  ga.rope_rows = c.rope_capacity > 0 ? c.rope_capacity : 1;
  ga.rope_set_stride = c.rope_scaling ? c.rope_capacity * (hd / 2) : 0;
  auto gemm = [&](int kind, const void* A, int K, const void* W, int N, int epi, const void* bias,
                  void* out, int ldo, const void* resid, int site) {
    GemmArgs q = ga;
    if (dec && kind == GM_K_GEMM_QKV) {
      // a decode step stores this layer's new k and v from the epilogue
      // this part's sequences in the cache ([B][H][max_seq][hd])
      const size_t co = static_cast<size_t>(b0) * c.n_heads * c.max_seq * hd * m->esz;
      q.kc = static_cast<char*>(m->kc[cur_layer]) + co;
      q.vc = static_cast<char*>(m->vc[cur_layer]) + co;
      q.kv_valid = m->kv_valid + static_cast<size_t>(b0) * c.max_seq;
      q.kv_max_seq = c.max_seq;
      q.heads = c.n_heads;
    }
    q.A = A;
    q.lda = K;
    q.K = K;
    q.W = W;
    q.ldw = K;
    q.N = N;
    q.epi = epi;
    q.bias = bias;
    q.out = out;
    q.ldo = ldo;
    q.resid = resid;
    q.ldr = ldo;
    q.site = site;
    if (on()) launch_gemm(q, s);
    const int nout = (epi == kEpiGatedGelu || epi == kEpiGatedSilu) ? N / 2 : N;
    P(kind, cur_layer, 2.0 * T * static_cast<double>(N) * K,
      es * (static_cast<double>(T) * K + static_cast<double>(N) * K +
            static_cast<double>(T) * nout * (resid ? 2 : 1)));
    if (site >= 0) brk(kCutClamp + site);  // original program: abs(h).max() read on the host
  };

  AttnArgs at{};
  at.dtype = m->dtype;
  at.B = nb;
  at.Sq = at.Sk = S;
  at.H = c.n_heads;
  at.hd = hd;
  at.d = d;
  at.q = qq;
  at.ldq = 3 * d;
  at.k = static_cast<const char*>(qq) + d * m->esz;
  at.v = static_cast<const char*>(qq) + 2 * d * m->esz;
  at.ldkv = 3 * d;
  at.ctx = cc;
  at.mask = mask ? mask + static_cast<size_t>(b0) * S : nullptr;
  at.state = m->state;
  at.pad_slot = kPadAny;
  at.kvlen_base = kKvLenBase + b0;
  at.causal = c.causal;
  at.scale = 1.0f / sqrtf(static_cast<float>(hd));

  const int up_epi = c.ffn == GM_FFN_GELU ? kEpiGelu
                     : c.ffn == GM_FFN_GEGLU ? kEpiGatedGelu : kEpiGatedSilu;
  const int up_n = c.ffn == GM_FFN_GELU ? ff : 2 * ff;
  const int qkv_epi = c.pos == GM_POS_ROTARY ? kEpiRope : kEpiStore;
  const double pairs = c.causal ? 0.5 * S * (S + 1.0) : static_cast<double>(S) * S;
  const double attn_flops = 4.0 * hd * pairs * nb * c.n_heads;
  const double attn_bytes = es * (static_cast<double>(T) * 3 * d + static_cast<double>(T) * d);
  KvArgs kv{};
  kv.dtype = m->dtype;
  kv.rows = T;
  kv.S = dec ? 0 : S;
  kv.pos = m->dpos;
  kv.mask = mask;
  kv.state = m->state;
  kv.qkv = qq;
  kv.d = d;
  kv.H = c.n_heads;
  kv.hd = hd;
  kv.valid = m->kv_valid;
  kv.max_seq = c.max_seq;
  DecAttnArgs da{};
  da.dtype = m->dtype;
  da.B = nb;
  da.H = c.n_heads;
  da.hd = hd;
  da.d = d;
  da.qkv = qq;
  da.valid = m->kv_valid + static_cast<size_t>(b0) * c.max_seq;
  da.max_seq = c.max_seq;
  da.pos = m->dpos + b0;
  da.ctx = cc;
  da.part = m->dpart;
  {
    // split the keys only when there are fewer than ~100 (sequence, head)
    // pairs to spread over the GPU (a split costs a merge launch); the
    // pairs are counted over the whole batch, as the batch parts run
    // concurrently (measured: splitting 8 x 12 heads further is no faster);
    // chunks are a multiple of 64 keys
    int want = (96 + B * c.n_heads - 1) / (B * c.n_heads);
    want = want < m->dec_nsplit ? want : m->dec_nsplit;
    want = want > 1 ? want : 1;
    da.chunk = 64 * ((c.max_seq + 64 * want - 1) / (64 * want));
    da.nsplit = (c.max_seq + da.chunk - 1) / da.chunk;
  }
  // this part's rows of the split-key workspace ([B][H][nsplit][hd + 2])
  if (m->dpart) da.part = m->dpart + static_cast<size_t>(b0) * c.n_heads * da.nsplit * (hd + 2);
  da.scale = at.scale;
  auto attention = [&]() {
    if (c.kv_cache && !dec) {
      // this layer's k and v go to the cache (a decode step stores them from
      // the QKV epilogue)
      kv.kc = m->kc[cur_layer];
      kv.vc = m->vc[cur_layer];
      if (on()) launch_kv_store(kv, s);
      P(GM_K_KV_STORE, cur_layer, 0.0, 4.0 * T * d * es);
    }
    if (dec) {
      const size_t co = static_cast<size_t>(b0) * c.n_heads * c.max_seq * hd * m->esz;
      da.kc = static_cast<char*>(m->kc[cur_layer]) + co;
      da.vc = static_cast<char*>(m->vc[cur_layer]) + co;
      launch_decode_attention(da, s);
      const double keys = static_cast<double>(B) * c.max_seq;   // upper bound: full cache
      P(GM_K_ATTENTION, cur_layer, 4.0 * hd * keys * c.n_heads, es * 2.0 * keys * d);
      return;
    }
    if (on()) launch_attention(at, s);
    P(GM_K_ATTENTION, cur_layer, attn_flops, attn_bytes);
  };
  int prev_site = -1;
  for (int l = 0; l < c.n_layers; ++l) {
    cur_layer = l;
    const LayerBufs& L = m->layers[l];
    const int s0 = ns ? 2 * l : -1, s1 = ns ? 2 * l + 1 : -1;
    if (pre) {
      auto D = [&](int which, const void* src) {
        if (dump) dump->copy(l, which, src, s);
      };
      norm_rows(hh, aa, L.ln1_g, L.ln1_b, prev_site);
      D(0, aa);
      gemm(GM_K_GEMM_QKV, aa, d, L.wqkv, 3 * d, qkv_epi, L.bqkv, qq, 3 * d, nullptr, -1);
      D(1, qq);
      attention();
      D(2, cc);
      gemm(GM_K_GEMM_O, cc, d, L.wo, d, kEpiResid, L.bo, hh, d, hh, s0);
      D(3, hh);
      norm_rows(hh, aa, L.ln2_g, L.ln2_b, s0);
      D(4, aa);
      gemm(GM_K_GEMM_UP, aa, d, L.w1, up_n, up_epi, L.b1, ffb, ff, nullptr, -1);
      D(5, ffb);
      gemm(GM_K_GEMM_DOWN, ffb, ff, L.w2, d, kEpiResid, L.b2, hh, d, hh, s1);
      D(6, hh);
      prev_site = s1;
    } else {
      gemm(GM_K_GEMM_QKV, hh, d, L.wqkv, 3 * d, qkv_epi, L.bqkv, qq, 3 * d, nullptr, -1);
      attention();
      gemm(GM_K_GEMM_O, cc, d, L.wo, d, kEpiResid, L.bo, tt, d, hh, -1);
      norm_rows(tt, hh, L.ln1_g, L.ln1_b, -1);
      gemm(GM_K_GEMM_UP, hh, d, L.w1, up_n, up_epi, L.b1, ffb, ff, nullptr, -1);
      gemm(GM_K_GEMM_DOWN, ffb, ff, L.w2, d, kEpiResid, L.b2, tt, d, hh, -1);
      norm_rows(tt, hh, L.ln2_g, L.ln2_b, -1);
    }
    if (c.log_hidden) {
      // `logger.info(..., h.abs().amax(per sequence))`: a tensor-valued log,
      // its value taken here and replayed after the forward
      if (on())
        launch_log_seqmax(hh, m->dtype, B, S, d, m->log_stage, l, m->state,
                          pre && ns ? 2 * l + 1 : -1, thr, s);
      P(GM_K_LOG, l, 0.0, es * T * d);
      brk(kCutLog + l);   // original program: the value is copied to the host to print it
    }
  }
  cur_layer = -1;
  const void* z = hh;
  if (pre) {
    norm_rows(hh, aa, m->lnf_g, m->lnf_b, prev_site);
    z = aa;
  }
  if (head_joined) return;
  gemm(GM_K_GEMM_HEAD, z, d, m->head, c.vocab, kEpiStore, nullptr, lg, c.vocab, nullptr, -1);
  if (dec && dec->next) {
    launch_argmax(lg, m->dtype, nb, c.vocab, dec->next + b0, s);
    P(GM_K_ARGMAX, -1, 0.0, es * B * static_cast<double>(c.vocab));
  }
  };
  // Independent batch-part branches (fork/join on auxiliary streams) where
  // nothing couples the sequences inside the layers: no clamp (its decision
  // is batch-global), no tensor log, not a KV-cache prefill or a profile,
  // and every forward part large enough for the tiled GEMMs, whose
  // per-element arithmetic does not depend on M, so the results are the same
  // bits as one branch.
  int parts = m->split_parts < B ? m->split_parts : B;
  // (a decode step's parts run the skinny kernels, so any part size goes)
  while (!dec && parts > 1 && (B / parts) * S <= 16) --parts;
  // Models whose projections take the large-tile GEMM (d >= 2048) run a
  // forward as one branch: a part's products have fewer large tiles than the
  // chip has CUs (2 x 1024 positions of the 4096-wide decoder: 30.2 ms per
  // forward as two branches, 28.05 ms as one).
  if (!dec && d >= 2048) parts = 1;
  if (prof || dump || work || c.fp16_clamp || c.log_hidden || (c.kv_cache && !dec)) parts = 1;
  head_joined = parts > 1 && dec;
  if (parts > 1) {
    // (the graph-broken run splits the same way: its only cut, the guards,
    // lies before the fork, and the fork and join go into the segment that
    // holds the layers)
    if (on()) {
      (void)hipEventRecord(m->ev_fork, s);
      for (int i = 0; i + 1 < parts; ++i) (void)hipStreamWaitEvent(m->aux_stream[i], m->ev_fork, 0);
    }
    for (int i = 0; i < parts; ++i) {
      const int b0 = B * i / parts, b1 = B * (i + 1) / parts;
      layers_and_head(i == 0 ? s : m->aux_stream[i - 1], b0, b1 - b0);
    }
    if (on())
      for (int i = 0; i + 1 < parts; ++i) {
        (void)hipEventRecord(m->ev_join[i], m->aux_stream[i]);
        (void)hipStreamWaitEvent(s, m->ev_join[i], 0);
      }
    if (head_joined) {
      GemmArgs q{};
      q.dtype = m->dtype;
      q.M = B;
      q.N = c.vocab;
      q.K = d;
      q.A = pre ? wk.a : wk.h;   // the final norm's output, or the stream itself
      q.lda = d;
      q.W = m->head;
      q.ldw = d;
      q.epi = kEpiStore;
      q.out = logits;
      q.ldo = c.vocab;
      q.state = m->state;
      q.site = -1;
      q.seq = S;
      q.head_dim = hd;
      q.d_model = d;
      launch_gemm(q, s);
      if (dec->next) launch_argmax(logits, m->dtype, B, c.vocab, dec->next, s);
    }
  } else {
    layers_and_head(s, 0, B);
  }
  if (c.kv_cache && on()) launch_seqlen_update(m->seqlen, m->dpos, m->state, B, dec ? 1 : 0, s);
  if (on())
    launch_emit_effects(m->state, m->fifo, kFifoCap, ns, m->log_stage, m->log_arena,
                        kLogArenaCap, c.log_hidden ? c.n_layers : 0, B, 0, s);
  P(GM_K_EFFECTS, -1, 0.0, 0.0);
}

// One encoder-decoder forward: the guards and padding predicates of both
// inputs, the encoder stack over the source, its final norm (the memory),
// one GEMM projecting the memory to k | v for every decoder layer, then the
// decoder stack (causal self-attention under the target's padding branch,
// cross-attention under the source's) and the head.
void enqueue_seq2seq(gm_model* m, int B, int Ss, const int32_t* src_ids, const int32_t* src_mask,
                     int St, const int32_t* tgt_ids, const int32_t* tgt_mask, void* logits,
                     hipStream_t s, Prof* prof = nullptr, Seg* seg = nullptr) {
  const gm_config& c = m->cfg;
  auto on = [&]() { return !seg || seg->want == -1 || seg->want == seg->cur; };
  auto brk = [&](int kind) {
    if (seg) {
      ++seg->cur;
      seg->kinds.push_back(kind);
    }
  };
  const int d = c.d_model, hd = d / c.n_heads, ff = c.d_ff, nd = c.n_dec_layers;
  const int Ts = B * Ss, Tt = B * St;
  const int normk = c.norm == GM_NORM_RMS ? 1 : 0;
  const double es = static_cast<double>(m->esz);
  int cur_layer = -1;
  auto P = [&](int kind, int layer, double flops, double bytes) {
    if (prof) prof->mark(kind, layer, flops, bytes);
  };
  if (prof) prof->start();
  if (on())
    launch_prologue(src_ids, src_mask, B, Ss, c.vocab, 0, 0, 0, nullptr, 0, nullptr, 0, 0,
                    m->state, s, 0, 0, kKvLenBase);
  P(GM_K_PROLOGUE, -1, 0.0, 8.0 * Ts);
  brk(kCutGuards);   // original program: the source's guards and mask.any() read on the host

  // The target's guards and padding predicate: before the decoder (after the
  // encoder) in one branch, where the graph-broken program reads them; before
  // the fork when the batch runs as parts.
  auto target_prologue = [&](hipStream_t s) {
    if (on())
      launch_prologue(tgt_ids, tgt_mask, B, St, c.vocab, 0, 0, 0, nullptr, 0, nullptr, 0, 0,
                      m->state, s, 1, Ts, kKvLenBase + c.max_batch);
    P(GM_K_PROLOGUE, -1, 0.0, 8.0 * Tt);
    brk(kCutGuardsTgt);   // original program: the target's guards and mask.any() read on the host
  };
  // Sequences [b0, b0 + nb) on stream s: part p's encoder and decoder rows
  // start at row b0 * S_src of every activation buffer (the decoder rows fit
  // in the part's encoder rows since S_tgt <= S_src when the batch is split).
  // Batch parts run as concurrent graph branches when nothing couples them
  // (not profiled or graph-broken, parts above 16 rows).
  const int b_half = B / 2;
  const bool split = m->split_parts > 1 && !prof && !seg && St <= Ss && b_half >= 1 &&
                     b_half * St > 16;
  auto part = [&](hipStream_t s, int b0, int nb) {
  const int Tsp = nb * Ss, Ttp = nb * St;
  const size_t ro = static_cast<size_t>(b0) * Ss, rt = static_cast<size_t>(b0) * St;
  char* hh = static_cast<char*>(m->h) + ro * d * m->esz;
  char* aa = static_cast<char*>(m->a) + ro * d * m->esz;
  char* qq = static_cast<char*>(m->qkv) + ro * 3 * d * m->esz;
  char* cc = static_cast<char*>(m->ctx) + ro * d * m->esz;
  char* ffb = static_cast<char*>(m->f) + ro * ff * m->esz;
  char* mm = static_cast<char*>(m->mem) + ro * d * m->esz;
  char* kk = static_cast<char*>(m->kvc) + ro * nd * 2 * d * m->esz;
  char* qcc = static_cast<char*>(m->qc) + rt * d * m->esz;
  char* lg = static_cast<char*>(logits) + rt * c.vocab * m->esz;
  const int32_t* sids = src_ids + ro;
  const int32_t* tids = tgt_ids + rt;
  const int32_t* smask = src_mask + ro;
  const int32_t* tmask = tgt_mask + rt;
  RowArgs r{};
  r.dtype = m->dtype;
  r.d = d;
  r.eps = c.norm_eps;
  r.state = m->state;
  r.clamp_site = -1;
  r.vocab = c.vocab;
  r.tok_emb = m->tok_emb;
  auto embed = [&](int rows, int S, const int32_t* ids, const void* pos) {
    RowArgs e = r;
    e.rows = rows;
    e.ids = ids;
    e.pos_emb = pos;
    e.seq = S;
    e.x = hh;
    e.out = hh;
    e.norm = -1;
    if (on()) launch_rownorm(e, s);
    P(GM_K_EMBED, -1, 0.0, static_cast<double>(rows) * d * es * 3);
  };
  auto norm_rows = [&](int rows, void* x, void* out, const void* g, const void* b) {
    RowArgs q = r;
    q.rows = rows;
    q.x = x;
    q.out = out;
    q.norm = normk;
    q.g = g;
    q.b = b;
    if (on()) launch_rownorm(q, s);
    P(GM_K_NORM, cur_layer, 0.0, 2.0 * rows * d * es);
  };
  auto gemm = [&](int kind, int M, const void* A, int K, const void* W, int N, int epi,
                  const void* bias, void* out, int ldo, const void* resid) {
    GemmArgs q{};
    q.dtype = m->dtype;
    q.M = M;
    q.state = m->state;
    q.site = -1;
    q.seq = 1;
    q.head_dim = hd;
    q.d_model = d;
    q.A = A;
    q.lda = K;
    q.K = K;
    q.W = W;
    q.ldw = K;
    q.N = N;
    q.epi = epi;
    q.bias = bias;
    q.out = out;
    q.ldo = ldo;
    q.resid = resid;
    q.ldr = ldo;
    if (on()) launch_gemm(q, s);
    const int nout = (epi == kEpiGatedGelu || epi == kEpiGatedSilu) ? N / 2 : N;
    P(kind, cur_layer, 2.0 * M * static_cast<double>(N) * K,
      es * (static_cast<double>(M) * K + static_cast<double>(N) * K +
            static_cast<double>(M) * nout * (resid ? 2 : 1)));
  };
  AttnArgs at{};
  at.dtype = m->dtype;
  at.B = nb;
  at.H = c.n_heads;
  at.hd = hd;
  at.d = d;
  at.ctx = cc;
  at.state = m->state;
  at.scale = 1.0f / sqrtf(static_cast<float>(hd));
  auto attention = [&](int kind, int Sq, int Sk, const void* q, int ldq, const void* k, int ldkv,
                       const int32_t* mask, int pad_slot, int kv_base, int causal) {
    AttnArgs a = at;
    a.Sq = Sq;
    a.Sk = Sk;
    a.q = q;
    a.ldq = ldq;
    a.k = k;
    a.v = static_cast<const char*>(k) + d * m->esz;
    a.ldkv = ldkv;
    a.mask = mask;
    a.pad_slot = pad_slot;
    a.kvlen_base = kv_base;
    a.causal = causal;
    if (on()) launch_attention(a, s);
    const double pairs = causal ? 0.5 * Sq * (Sq + 1.0) : static_cast<double>(Sq) * Sk;
    P(kind, cur_layer, 4.0 * hd * pairs * nb * c.n_heads,
      es * (static_cast<double>(nb) * Sq * 2 * d + static_cast<double>(nb) * Sk * 2 * d));
  };
  const int up_epi = c.ffn == GM_FFN_GELU ? kEpiGelu
                     : c.ffn == GM_FFN_GEGLU ? kEpiGatedGelu : kEpiGatedSilu;
  const int up_n = c.ffn == GM_FFN_GELU ? ff : 2 * ff;
  char* qkv = static_cast<char*>(qq);
  auto block_ffn = [&](int rows, const LayerBufs& L) {
    norm_rows(rows, hh, aa, L.ln2_g, L.ln2_b);
    gemm(GM_K_GEMM_UP, rows, aa, d, L.w1, up_n, up_epi, L.b1, ffb, ff, nullptr);
    gemm(GM_K_GEMM_DOWN, rows, ffb, ff, L.w2, d, kEpiResid, L.b2, hh, d, hh);
  };

  // encoder (bidirectional; the source's padding branch)
  embed(Tsp, Ss, sids, m->enc_pos_emb);
  for (int l = 0; l < c.n_layers; ++l) {
    cur_layer = l;
    const LayerBufs& L = m->layers[l];
    norm_rows(Tsp, hh, aa, L.ln1_g, L.ln1_b);
    gemm(GM_K_GEMM_QKV, Tsp, aa, d, L.wqkv, 3 * d, kEpiStore, L.bqkv, qq, 3 * d, nullptr);
    attention(GM_K_ATTENTION, Ss, Ss, qkv, 3 * d, qkv + d * m->esz, 3 * d, smask, kPadAny,
              kKvLenBase + b0, 0);
    gemm(GM_K_GEMM_O, Tsp, cc, d, L.wo, d, kEpiResid, L.bo, hh, d, hh);
    block_ffn(Tsp, L);
  }
  cur_layer = -1;
  norm_rows(Tsp, hh, mm, m->enc_lnf_g, m->enc_lnf_b);
  // k | v of every decoder layer from the encoder output, one GEMM
  gemm(GM_K_GEMM_XKV, Tsp, mm, d, m->wkv_all, nd * 2 * d, kEpiStore, m->bkv_all, kk,
       nd * 2 * d, nullptr);

  // decoder (causal self-attention under the target's padding branch,
  // cross-attention under the source's); its inputs' guards merge into the
  // forward's trap word
  if (!split) target_prologue(s);
  embed(Ttp, St, tids, m->pos_emb);
  for (int l = 0; l < nd; ++l) {
    cur_layer = c.n_layers + l;
    const LayerBufs& L = m->dec_layers[l];
    const CrossBufs& X = m->dec_cross[l];
    norm_rows(Ttp, hh, aa, L.ln1_g, L.ln1_b);
    gemm(GM_K_GEMM_QKV, Ttp, aa, d, L.wqkv, 3 * d, kEpiStore, L.bqkv, qq, 3 * d, nullptr);
    attention(GM_K_ATTENTION, St, St, qkv, 3 * d, qkv + d * m->esz, 3 * d, tmask, kPadAnyTgt,
              kKvLenBase + c.max_batch + b0, 1);
    gemm(GM_K_GEMM_O, Ttp, cc, d, L.wo, d, kEpiResid, L.bo, hh, d, hh);
    norm_rows(Ttp, hh, aa, X.lnc_g, X.lnc_b);
    gemm(GM_K_GEMM_XQ, Ttp, aa, d, X.wq, d, kEpiStore, X.bq, qcc, d, nullptr);
    attention(GM_K_XATTN, St, Ss, qcc, d, static_cast<char*>(kk) + static_cast<size_t>(l) * 2 * d * m->esz,
              nd * 2 * d, smask, kPadAny, kKvLenBase + b0, 0);
    gemm(GM_K_GEMM_XO, Ttp, cc, d, X.wo, d, kEpiResid, X.bo, hh, d, hh);
    block_ffn(Ttp, L);
  }
  cur_layer = -1;
  norm_rows(Ttp, hh, aa, m->lnf_g, m->lnf_b);
  gemm(GM_K_GEMM_HEAD, Ttp, aa, d, m->head, c.vocab, kEpiStore, nullptr, lg, c.vocab, nullptr);
  };
  if (split) {
    target_prologue(s);
    (void)hipEventRecord(m->ev_fork, s);
    (void)hipStreamWaitEvent(m->aux_stream[0], m->ev_fork, 0);
    part(s, 0, b_half);
    part(m->aux_stream[0], b_half, B - b_half);
    (void)hipEventRecord(m->ev_join[0], m->aux_stream[0]);
    (void)hipStreamWaitEvent(s, m->ev_join[0], 0);
  } else {
    part(s, 0, B);
  }
  if (on()) launch_emit_effects(m->state, m->fifo, kFifoCap, 0, nullptr, nullptr, 0, 0, B, 1, s);
  P(GM_K_EFFECTS, -1, 0.0, 0.0);
}

}  // namespace

// Launch the graph cached for `key` (kind, shape and buffer pointers),
// capturing and instantiating it first on a cold key (LRU of kMaxGraphs).
template <typename Body>
int launch_graph(gm_model* m, GraphEntry key, hipStream_t stream, Body body) {
  GraphEntry* ge = nullptr;
  for (auto& g : m->graphs)
    if (g.kind == key.kind && g.B == key.B && g.S == key.S && g.ids == key.ids &&
        g.mask == key.mask && g.logits == key.logits && g.next == key.next &&
        g.S2 == key.S2 && g.ids2 == key.ids2 && g.mask2 == key.mask2)
      ge = &g;
  if (!ge) {
    hipGraph_t graph = nullptr;
    HIP_TRY(hipStreamBeginCapture(m->cap_stream, hipStreamCaptureModeThreadLocal));
    body(m->cap_stream);
    hipError_t e = hipStreamEndCapture(m->cap_stream, &graph);
    if (e != hipSuccess || !graph) {
      g_last_error = std::string("capture: ") + hipGetErrorString(e);
      hipGetLastError();
      return GM_E_CAPTURE;
    }
    size_t nodes = 0;
    hipGraphGetNodes(graph, nullptr, &nodes);
    hipGraphExec_t exec = nullptr;
    e = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
    hipGraphDestroy(graph);
    if (e != hipSuccess) {
      g_last_error = std::string("instantiate: ") + hipGetErrorString(e);
      return GM_E_CAPTURE;
    }
    if (static_cast<int>(m->graphs.size()) >= kMaxGraphs) {
      size_t victim = 0;
      for (size_t i = 1; i < m->graphs.size(); ++i)
        if (m->graphs[i].last_use < m->graphs[victim].last_use) victim = i;
      hipGraphExecDestroy(m->graphs[victim].exec);
      m->graphs.erase(m->graphs.begin() + victim);
    }
    key.exec = exec;
    m->graphs.push_back(key);
    ge = &m->graphs.back();
    m->stats.captures++;
    m->stats.kernels_per_forward = nodes;
  }
  ge->last_use = ++m->tick;
  HIP_TRY(hipGraphLaunch(ge->exec, stream));
  m->stats.graph_launches++;
  if (m->debug_sync) {
    m->stats.host_syncs_in_forward++;
    HIP_TRY(hipStreamSynchronize(stream));
  }
  return GM_OK;
}

extern "C" {

const char* gm_strerror(int code) {
  switch (code) {
    case GM_OK: return "ok";
    case GM_E_INVAL: return "invalid argument";
    case GM_E_NOMEM: return "out of device memory";
    case GM_E_HIP: return "HIP runtime error";
    case GM_E_CAPTURE: return "graph capture failed";
    case GM_E_TRAP: return "input guard failed";
    default: return "unknown error";
  }
}

const char* gm_last_error(void) { return g_last_error.c_str(); }

void gm_model_destroy(gm_model* m) {
  if (!m) return;
  hipDeviceSynchronize();
  for (auto& g : m->graphs) hipGraphExecDestroy(g.exec);
  for (auto& f : m->frags)
    for (hipGraphExec_t e : f.execs) hipGraphExecDestroy(e);
  if (m->cap_stream) hipStreamDestroy(m->cap_stream);
  for (int i = 0; i < gm_model::kMaxParts - 1; ++i) {
    if (m->aux_stream[i]) hipStreamDestroy(m->aux_stream[i]);
    if (m->ev_join[i]) hipEventDestroy(m->ev_join[i]);
  }
  if (m->ev_fork) hipEventDestroy(m->ev_fork);
  for (void* p : m->allocs) hipFree(p);
  delete m;
}

int gm_model_create(const gm_config* cfg, const gm_weights* w, gm_model** out) {
  if (!out) return inval("out is NULL");
  *out = nullptr;
  int rc = validate(cfg);
  if (rc) return rc;
  if (!w || !w->layers) return inval("weights or weights->layers is NULL");
  const gm_config& c = *cfg;
  const bool ln = c.norm == GM_NORM_LAYER;
  const bool pre = c.norm_place == GM_NORM_PRE;
  // unused pointers must be NULL, used ones non-NULL
  auto want = [&](const void* p, bool used, const char* name) -> int {
    if (used && !p) return inval((std::string("missing weight ") + name).c_str());
    if (!used && p) return inval((std::string("unexpected weight ") + name).c_str());
    return GM_OK;
  };
  if ((rc = want(w->tok_emb, true, "tok_emb")) || (rc = want(w->pos_emb, c.pos == GM_POS_LEARNED, "pos_emb")) ||
      (rc = want(w->emb_ln_g, c.emb_norm, "emb_ln_g")) || (rc = want(w->emb_ln_b, c.emb_norm && ln, "emb_ln_b")) ||
      (rc = want(w->lnf_g, pre, "lnf_g")) || (rc = want(w->lnf_b, pre && ln, "lnf_b")) ||
      (rc = want(w->lm_head, !c.tied_head, "lm_head")) ||
      (rc = want(w->rope_short_factor, c.rope_scaling != 0, "rope_short_factor")) ||
      (rc = want(w->rope_long_factor, c.rope_scaling != 0, "rope_long_factor")) ||
      (rc = want(w->enc_pos_emb, c.n_dec_layers > 0, "enc_pos_emb")) ||
      (rc = want(w->enc_lnf_g, c.n_dec_layers > 0, "enc_lnf_g")) ||
      (rc = want(w->enc_lnf_b, c.n_dec_layers > 0 && ln, "enc_lnf_b")) ||
      (rc = want(w->dec_layers, c.n_dec_layers > 0, "dec_layers")) ||
      (rc = want(w->dec_cross, c.n_dec_layers > 0, "dec_cross")))
    return rc;
  for (int l = 0; l < c.n_dec_layers; ++l) {
    const gm_layer_weights& L = w->dec_layers[l];
    const gm_cross_weights& X = w->dec_cross[l];
    if ((rc = want(L.ln1_g, true, "dec ln1_g")) || (rc = want(L.ln1_b, ln, "dec ln1_b")) ||
        (rc = want(L.ln2_g, true, "dec ln2_g")) || (rc = want(L.ln2_b, ln, "dec ln2_b")) ||
        (rc = want(L.wqkv, true, "dec wqkv")) || (rc = want(L.wo, true, "dec wo")) ||
        (rc = want(L.w1, true, "dec w1")) || (rc = want(L.w2, true, "dec w2")) ||
        (rc = want(L.bqkv, c.has_bias, "dec bqkv")) || (rc = want(L.bo, c.has_bias, "dec bo")) ||
        (rc = want(L.b1, c.has_bias, "dec b1")) || (rc = want(L.b2, c.has_bias, "dec b2")) ||
        (rc = want(X.lnc_g, true, "lnc_g")) || (rc = want(X.lnc_b, ln, "lnc_b")) ||
        (rc = want(X.wq, true, "cross wq")) || (rc = want(X.wkv, true, "cross wkv")) ||
        (rc = want(X.wo, true, "cross wo")) || (rc = want(X.bq, c.has_bias, "cross bq")) ||
        (rc = want(X.bkv, c.has_bias, "cross bkv")) || (rc = want(X.bo, c.has_bias, "cross bo")))
      return rc;
  }
  for (int l = 0; l < c.n_layers; ++l) {
    const gm_layer_weights& L = w->layers[l];
    if ((rc = want(L.ln1_g, true, "ln1_g")) || (rc = want(L.ln1_b, ln, "ln1_b")) ||
        (rc = want(L.ln2_g, true, "ln2_g")) || (rc = want(L.ln2_b, ln, "ln2_b")) ||
        (rc = want(L.wqkv, true, "wqkv")) || (rc = want(L.wo, true, "wo")) ||
        (rc = want(L.w1, true, "w1")) || (rc = want(L.w2, true, "w2")) ||
        (rc = want(L.bqkv, c.has_bias, "bqkv")) || (rc = want(L.bo, c.has_bias, "bo")) ||
        (rc = want(L.b1, c.has_bias, "b1")) || (rc = want(L.b2, c.has_bias, "b2")))
      return rc;
  }

  gm_model* m = new gm_model();
  m->cfg = c;
  m->dtype = c.act_dtype;
  m->esz = c.act_dtype == GM_DTYPE_F32 ? 4 : 2;
  memset(&m->stats, 0, sizeof(m->stats));
  m->debug_sync = getenv("GM_DEBUG_SYNC") && atoi(getenv("GM_DEBUG_SYNC"));
  attention_set_order(getenv("GM_ATTN_ORDER") ? atoi(getenv("GM_ATTN_ORDER")) : 2);
  auto fail = [&](int code) {
    gm_model_destroy(m);
    return code;
  };
  hipError_t e = hipGetDevice(&m->device);
  if (e != hipSuccess) return fail(hip_fail(e, "hipGetDevice"));
  // this device's static scratch (gm_forward_noalloc), once per device
  if ((rc = scratch_for_device(m->device, &m->scratch))) return fail(rc);

  const int d = c.d_model, hd = d / c.n_heads, ff = c.d_ff, V = c.vocab;
  const bool gated = c.ffn != GM_FFN_GELU;
  const std::vector<int32_t> gp = gated ? gated_perm(ff) : std::vector<int32_t>();
  const std::vector<int32_t> rp = c.pos == GM_POS_ROTARY ? rope_perm(d, hd) : std::vector<int32_t>();
  const std::vector<int32_t>* gpp = gated ? &gp : nullptr;
  const std::vector<int32_t>* rpp = c.pos == GM_POS_ROTARY ? &rp : nullptr;

  if ((rc = copy_in(m, &m->tok_emb, w->tok_emb, V, d, nullptr, "tok_emb"))) return fail(rc);
  // learned positions: max_seq rows (an encoder-decoder's decoder: max_tgt)
  if (c.pos == GM_POS_LEARNED &&
      (rc = copy_in(m, &m->pos_emb, w->pos_emb, c.n_dec_layers ? c.max_tgt : c.max_seq, d, nullptr,
                    "pos_emb")))
    return fail(rc);
  if (c.n_dec_layers) {
    if ((rc = copy_in(m, &m->enc_pos_emb, w->enc_pos_emb, c.max_seq, d, nullptr, "enc_pos_emb")) ||
        (rc = copy_in(m, &m->enc_lnf_g, w->enc_lnf_g, 1, d, nullptr, "enc_lnf_g")) ||
        (ln && (rc = copy_in(m, &m->enc_lnf_b, w->enc_lnf_b, 1, d, nullptr, "enc_lnf_b"))))
      return fail(rc);
    const int nd = c.n_dec_layers;
    m->dec_layers.resize(nd);
    m->dec_cross.resize(nd);
    // k | v projections of all decoder layers, stacked: one GEMM over the
    // encoder output serves every layer's cross-attention
    const size_t kv_rows = static_cast<size_t>(2) * d;
    const size_t kv_bytes = kv_rows * d * m->esz;
    if ((rc = m->alloc(&m->wkv_all, nd * kv_bytes))) return fail(rc);
    if (c.has_bias && (rc = m->alloc(&m->bkv_all, nd * kv_rows * m->esz))) return fail(rc);
    for (int l = 0; l < nd; ++l) {
      const gm_layer_weights& L = w->dec_layers[l];
      const gm_cross_weights& X = w->dec_cross[l];
      LayerBufs& D = m->dec_layers[l];
      CrossBufs& C = m->dec_cross[l];
      if ((rc = copy_in(m, &D.ln1_g, L.ln1_g, 1, d, nullptr, "dec ln1_g")) ||
          (ln && (rc = copy_in(m, &D.ln1_b, L.ln1_b, 1, d, nullptr, "dec ln1_b"))) ||
          (rc = copy_in(m, &D.ln2_g, L.ln2_g, 1, d, nullptr, "dec ln2_g")) ||
          (ln && (rc = copy_in(m, &D.ln2_b, L.ln2_b, 1, d, nullptr, "dec ln2_b"))) ||
          (rc = copy_in(m, &D.wqkv, L.wqkv, 3 * d, d, nullptr, "dec wqkv")) ||
          (rc = copy_in(m, &D.wo, L.wo, d, d, nullptr, "dec wo")) ||
          (rc = copy_in(m, &D.w1, L.w1, gated ? 2 * ff : ff, d, gpp, "dec w1")) ||
          (rc = copy_in(m, &D.w2, L.w2, d, ff, nullptr, "dec w2")) ||
          (rc = copy_in(m, &C.lnc_g, X.lnc_g, 1, d, nullptr, "lnc_g")) ||
          (ln && (rc = copy_in(m, &C.lnc_b, X.lnc_b, 1, d, nullptr, "lnc_b"))) ||
          (rc = copy_in(m, &C.wq, X.wq, d, d, nullptr, "cross wq")) ||
          (rc = copy_in(m, &C.wo, X.wo, d, d, nullptr, "cross wo")))
        return fail(rc);
      e = hipMemcpy(static_cast<char*>(m->wkv_all) + l * kv_bytes, X.wkv, kv_bytes,
                    hipMemcpyDeviceToDevice);
      if (e != hipSuccess) return fail(hip_fail(e, "cross wkv"));
      if (c.has_bias) {
        if ((rc = copy_in(m, &D.bqkv, L.bqkv, 3 * d, 1, nullptr, "dec bqkv")) ||
            (rc = copy_in(m, &D.bo, L.bo, d, 1, nullptr, "dec bo")) ||
            (rc = copy_in(m, &D.b1, L.b1, gated ? 2 * ff : ff, 1, gpp, "dec b1")) ||
            (rc = copy_in(m, &D.b2, L.b2, d, 1, nullptr, "dec b2")) ||
            (rc = copy_in(m, &C.bq, X.bq, d, 1, nullptr, "cross bq")) ||
            (rc = copy_in(m, &C.bo, X.bo, d, 1, nullptr, "cross bo")))
          return fail(rc);
        e = hipMemcpy(static_cast<char*>(m->bkv_all) + l * kv_rows * m->esz, X.bkv,
                      kv_rows * m->esz, hipMemcpyDeviceToDevice);
        if (e != hipSuccess) return fail(hip_fail(e, "cross bkv"));
      }
    }
  }
  if (c.emb_norm) {
    if ((rc = copy_in(m, &m->emb_ln_g, w->emb_ln_g, 1, d, nullptr, "emb_ln_g"))) return fail(rc);
    if (ln && (rc = copy_in(m, &m->emb_ln_b, w->emb_ln_b, 1, d, nullptr, "emb_ln_b"))) return fail(rc);
  }
  if (pre) {
    if ((rc = copy_in(m, &m->lnf_g, w->lnf_g, 1, d, nullptr, "lnf_g"))) return fail(rc);
    if (ln && (rc = copy_in(m, &m->lnf_b, w->lnf_b, 1, d, nullptr, "lnf_b"))) return fail(rc);
  }
  if (c.tied_head) m->head = m->tok_emb;
  else if ((rc = copy_in(m, &m->head, w->lm_head, V, d, nullptr, "lm_head"))) return fail(rc);

  m->layers.resize(c.n_layers);
  for (int l = 0; l < c.n_layers; ++l) {
    const gm_layer_weights& L = w->layers[l];
    LayerBufs& B = m->layers[l];
    const int f1 = gated ? 2 * ff : ff;
    if ((rc = copy_in(m, &B.ln1_g, L.ln1_g, 1, d, nullptr, "ln1_g")) ||
        (ln && (rc = copy_in(m, &B.ln1_b, L.ln1_b, 1, d, nullptr, "ln1_b"))) ||
        (rc = copy_in(m, &B.ln2_g, L.ln2_g, 1, d, nullptr, "ln2_g")) ||
        (ln && (rc = copy_in(m, &B.ln2_b, L.ln2_b, 1, d, nullptr, "ln2_b"))) ||
        (rc = copy_in(m, &B.wqkv, L.wqkv, 3 * d, d, rpp, "wqkv")) ||
        (rc = copy_in(m, &B.wo, L.wo, d, d, nullptr, "wo")) ||
        (rc = copy_in(m, &B.w1, L.w1, f1, d, gpp, "w1")) ||
        (rc = copy_in(m, &B.w2, L.w2, d, ff, nullptr, "w2")))
      return fail(rc);
    if (c.has_bias) {
      if ((rc = copy_in(m, &B.bqkv, L.bqkv, 3 * d, 1, rpp, "bqkv")) ||
          (rc = copy_in(m, &B.bo, L.bo, d, 1, nullptr, "bo")) ||
          (rc = copy_in(m, &B.b1, L.b1, f1, 1, gpp, "b1")) ||
          (rc = copy_in(m, &B.b2, L.b2, d, 1, nullptr, "b2")))
        return fail(rc);
    }
  }

  // workspace (an encoder-decoder's decoder reuses it for max_tgt positions)
  const size_t T = static_cast<size_t>(c.max_batch) *
                   (c.n_dec_layers && c.max_tgt > c.max_seq ? c.max_tgt : c.max_seq);
  const size_t es = m->esz;
  if (c.n_dec_layers) {
    const size_t Ts = static_cast<size_t>(c.max_batch) * c.max_seq;
    const size_t Tt = static_cast<size_t>(c.max_batch) * c.max_tgt;
    if ((rc = m->alloc(&m->mem, Ts * d * es)) || (rc = m->alloc(&m->qc, Tt * d * es)) ||
        (rc = m->alloc(&m->kvc, Ts * c.n_dec_layers * 2 * d * es)))
      return fail(rc);
  }
  if ((rc = m->alloc(&m->h, T * d * es)) || (rc = m->alloc(&m->a, T * d * es)) ||
      (rc = m->alloc(&m->qkv, T * 3 * d * es)) || (rc = m->alloc(&m->ctx, T * d * es)) ||
      (rc = m->alloc(&m->f, T * ff * es)) ||
      (!pre && (rc = m->alloc(&m->tmp, T * d * es))))
    return fail(rc);
  if (c.kv_cache) {
    const size_t per_layer = static_cast<size_t>(c.max_batch) * c.max_seq * d * es;
    m->kc.assign(c.n_layers, nullptr);
    m->vc.assign(c.n_layers, nullptr);
    for (int l = 0; l < c.n_layers; ++l)
      if ((rc = m->alloc(&m->kc[l], per_layer)) || (rc = m->alloc(&m->vc[l], per_layer)))
        return fail(rc);
    // at most 32 key chunks per head (the workspace bound)
    m->dec_nsplit = 32;
    void* q = nullptr;
    if ((rc = m->alloc(&q, static_cast<size_t>(c.max_batch) * c.max_seq))) return fail(rc);
    m->kv_valid = static_cast<uint8_t*>(q);
    if ((rc = m->alloc(&q, c.max_batch * sizeof(int32_t)))) return fail(rc);
    m->seqlen = static_cast<int32_t*>(q);
    if ((rc = m->alloc(&q, c.max_batch * sizeof(int32_t)))) return fail(rc);
    m->dpos = static_cast<int32_t*>(q);
    if ((rc = m->alloc(&q, static_cast<size_t>(c.max_batch) * c.n_heads * m->dec_nsplit * (hd + 2) *
                                sizeof(float))))
      return fail(rc);
    m->dpart = static_cast<float*>(q);
    e = hipMemset(m->kv_valid, 0, static_cast<size_t>(c.max_batch) * c.max_seq);
    if (e == hipSuccess) e = hipMemset(m->seqlen, 0, c.max_batch * sizeof(int32_t));
    if (e == hipSuccess) e = hipMemset(m->dpos, 0, c.max_batch * sizeof(int32_t));
    if (e != hipSuccess) return fail(hip_fail(e, "hipMemset"));
  }
  // device state (encoder-decoder: the target's key lengths follow the source's)
  m->n_state = kKvLenBase + 2 * c.max_batch;
  void* p = nullptr;
  if ((rc = m->alloc(&p, m->n_state * sizeof(int32_t)))) return fail(rc);
  m->state = static_cast<int32_t*>(p);
  if ((rc = m->alloc(&m->fifo, kFifoCap * sizeof(EffectRec)))) return fail(rc);
  if (c.log_hidden) {
    if ((rc = m->alloc(&p, static_cast<size_t>(c.n_layers) * c.max_batch * sizeof(float))))
      return fail(rc);
    m->log_stage = static_cast<float*>(p);
    if ((rc = m->alloc(&p, kLogArenaCap * sizeof(float)))) return fail(rc);
    m->log_arena = static_cast<float*>(p);
  }
  std::vector<int32_t> st(m->n_state, 0);
  st[kTrapFwd] = static_cast<int32_t>(kTrapNone);
  if (c.pos == GM_POS_ROTARY) {
    // long/short select: two sets, short rows first
    const size_t sets = c.rope_scaling ? 2 : 1;
    const size_t tb = sets * static_cast<size_t>(c.rope_capacity) * (hd / 2) * sizeof(float);
    if ((rc = m->alloc(&p, tb))) return fail(rc);
    m->rope_cos = static_cast<float*>(p);
    if ((rc = m->alloc(&p, tb))) return fail(rc);
    m->rope_sin = static_cast<float*>(p);
    e = hipMemset(m->rope_cos, 0, tb);
    if (e == hipSuccess) e = hipMemset(m->rope_sin, 0, tb);
    if (e != hipSuccess) return fail(hip_fail(e, "hipMemset"));
    st[kRegrowFrom] = 0;
    st[kRegrowTo] = c.rope_scaling ? 0 : c.rope_init_len;
    st[kCachedLen] = c.rope_scaling ? c.rope_capacity : c.rope_init_len;
  }
  e = hipMemcpy(m->state, st.data(), st.size() * sizeof(int32_t), hipMemcpyHostToDevice);
  if (e != hipSuccess) return fail(hip_fail(e, "state init"));
  if (c.pos == GM_POS_ROTARY && c.rope_scaling) {
    // both frequency sets in full: the hoisted, memoised initialisation
    const size_t half = static_cast<size_t>(c.rope_capacity) * (hd / 2);
    float* fac = nullptr;
    if ((rc = m->alloc(&p, 2 * (hd / 2) * sizeof(float)))) return fail(rc);
    fac = static_cast<float*>(p);
    e = hipMemcpy(fac, w->rope_short_factor, (hd / 2) * sizeof(float), hipMemcpyDeviceToDevice);
    if (e == hipSuccess)
      e = hipMemcpy(fac + hd / 2, w->rope_long_factor, (hd / 2) * sizeof(float), hipMemcpyDeviceToDevice);
    if (e != hipSuccess) return fail(hip_fail(e, "rope factors"));
    launch_rope_fill_scaled(m->rope_cos, m->rope_sin, hd, c.rope_base, fac, c.rope_attn_factor,
                            c.rope_capacity, nullptr);
    launch_rope_fill_scaled(m->rope_cos + half, m->rope_sin + half, hd, c.rope_base, fac + hd / 2,
                            c.rope_attn_factor, c.rope_capacity, nullptr);
    e = hipGetLastError();
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e != hipSuccess) return fail(hip_fail(e, "rope init"));
  } else if (c.pos == GM_POS_ROTARY) {
    // rows [0, rope_init_len) with the same kernel that grows the table
    launch_rope_fill(m->rope_cos, m->rope_sin, hd, c.rope_base, m->state, nullptr);
    e = hipGetLastError();
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e != hipSuccess) return fail(hip_fail(e, "rope init"));
  }
  e = hipStreamCreateWithFlags(&m->cap_stream, hipStreamNonBlocking);
  for (int i = 0; e == hipSuccess && i < gm_model::kMaxParts - 1; ++i)
    e = hipStreamCreateWithFlags(&m->aux_stream[i], hipStreamNonBlocking);
  if (e != hipSuccess) return fail(hip_fail(e, "hipStreamCreate"));
  e = hipEventCreateWithFlags(&m->ev_fork, hipEventDisableTiming);
  for (int i = 0; e == hipSuccess && i < gm_model::kMaxParts - 1; ++i)
    e = hipEventCreateWithFlags(&m->ev_join[i], hipEventDisableTiming);
  if (e != hipSuccess) return fail(hip_fail(e, "hipEventCreate"));
  if (const char* v = getenv("GM_SPLIT_PARTS")) {
    const int n = atoi(v);
    m->split_parts = n < 1 ? 1 : (n > gm_model::kMaxParts ? gm_model::kMaxParts : n);
  }
  e = hipDeviceSynchronize();
  if (e != hipSuccess) return fail(hip_fail(e, "create"));
  *out = m;
  return GM_OK;
}

int gm_set_exec_mode(gm_model* m, int32_t mode) {
  if (!m) return inval("model is NULL");
  if (mode != GM_EXEC_GRAPH && mode != GM_EXEC_EAGER && mode != GM_EXEC_FRAGMENTED)
    return inval("bad execution mode");
  m->exec_mode = mode;
  return GM_OK;
}

int gm_set_graph_mode(gm_model* m, int32_t enabled) {
  return gm_set_exec_mode(m, enabled ? GM_EXEC_GRAPH : GM_EXEC_EAGER);
}

}  // extern "C"

// The unmended program: every data-dependent branch is a host decision.  Each
// stretch between two such reads is one captured graph (one per fused
// region, as the paper's baseline captures them); at each cut the host
// synchronises the stream, copies the predicate's inputs back and evaluates
// the branch.  The kernels are the same as in the single-graph forward.
// `key` names the forward (shape and buffers); body(stream, seg) enqueues it.
template <typename Body>
static int forward_fragmented(gm_model* m, const gm_model::Frag& key, hipStream_t stream,
                              Body body) {
  const int B = key.B;
  gm_model::Frag* fr = nullptr;
  for (auto& f : m->frags)
    if (f.B == B && f.S == key.S && f.ids == key.ids && f.mask == key.mask &&
        f.logits == key.logits && f.S2 == key.S2 && f.ids2 == key.ids2 && f.mask2 == key.mask2)
      fr = &f;
  if (!fr) {
    Seg count;
    count.want = kCountOnly;
    body(m->cap_stream, &count);
    gm_model::Frag f = key;
    f.execs.clear();
    f.kinds = count.kinds;
    for (int i = 0; i <= count.cur; ++i) {
      hipGraph_t graph = nullptr;
      HIP_TRY(hipStreamBeginCapture(m->cap_stream, hipStreamCaptureModeThreadLocal));
      Seg sg;
      sg.want = i;
      body(m->cap_stream, &sg);
      hipError_t e = hipStreamEndCapture(m->cap_stream, &graph);
      if (e != hipSuccess || !graph) {
        g_last_error = std::string("capture: ") + hipGetErrorString(e);
        return GM_E_CAPTURE;
      }
      hipGraphExec_t exec = nullptr;
      e = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
      hipGraphDestroy(graph);
      if (e != hipSuccess) {
        g_last_error = std::string("instantiate: ") + hipGetErrorString(e);
        return GM_E_CAPTURE;
      }
      f.execs.push_back(exec);
      m->stats.captures++;
    }
    m->frags.push_back(std::move(f));
    fr = &m->frags.back();
  }
  const gm_config& c = m->cfg;
  const int ns = n_sites(c);
  const float thr = 65504.f - c.clamp_margin;
  const int nseg = static_cast<int>(fr->execs.size());
  int32_t host[kAbsmaxBase + 2 * GM_MAX_LAYERS];
  for (int i = 0; i < nseg; ++i) {
    HIP_TRY(hipGraphLaunch(fr->execs[i], stream));
    m->stats.graph_launches++;
    if (i + 1 == nseg) break;
    // graph break: wait for the device, read the predicate back, branch on the host
    m->stats.host_syncs_in_forward++;
    HIP_TRY(hipStreamSynchronize(stream));
    const int kind = fr->kinds[i];
    if (kind == kCutGuards || kind == kCutGuardsTgt) {
      HIP_TRY(hipMemcpy(host, m->state, sizeof(int32_t) * kClampBase, hipMemcpyDeviceToHost));
      const uint32_t trap = static_cast<uint32_t>(host[kTrapFwd]);
      if (trap != kTrapNone) {  // `if not C: raise` -- the forward stops at the guard
        int32_t sticky = 0;
        HIP_TRY(hipMemcpy(&sticky, m->state + kTrapSticky, sizeof(sticky), hipMemcpyDeviceToHost));
        if (!sticky) {
          sticky = static_cast<int32_t>(trap);
          HIP_TRY(hipMemcpy(m->state + kTrapSticky, &sticky, sizeof(sticky), hipMemcpyHostToDevice));
        }
        g_last_error = "input guard failed (fragmented execution stops at the guard)";
        return GM_E_TRAP;
      }
      m->last_host_pad_any = host[kind == kCutGuards ? kPadAny : kPadAnyTgt] != 0;  // `if mask.any():`
      m->last_host_regrow = host[kRegrow] != 0;       // `if seq_len > cached:`
    } else if (kind >= kCutLog) {
      // `logger.info(..., tensor)`: the values come back to the host to be printed
      float vals[1024];
      const int n = B < 1024 ? B : 1024;
      HIP_TRY(hipMemcpy(vals, m->log_stage + static_cast<size_t>(kind - kCutLog) * B,
                        n * sizeof(float), hipMemcpyDeviceToHost));
    } else {
      const int site = kind - kCutClamp;
      if (site < ns) {
        int32_t am[2];
        HIP_TRY(hipMemcpy(&am[0], m->state + kAbsmaxBase + site, sizeof(int32_t), hipMemcpyDeviceToHost));
        HIP_TRY(hipMemcpy(&am[1], m->state + kNanBase + site, sizeof(int32_t), hipMemcpyDeviceToHost));
        float mx;
        memcpy(&mx, &am[0], sizeof(mx));
        m->last_host_clamp = !am[1] && mx > thr;      // `if abs(h).max() > thr:`
      }
    }
  }
  return GM_OK;
}

extern "C" {

int gm_forward_ex(gm_model* m, int32_t B, int32_t S, const int32_t* ids, const int32_t* mask,
                  void* logits, hipStream_t stream) {
  if (!m) return inval("model is NULL");
  if (!ids || !mask || !logits) return inval("ids, mask and logits must be non-NULL");
  if ((reinterpret_cast<uintptr_t>(ids) | reinterpret_cast<uintptr_t>(mask) |
       reinterpret_cast<uintptr_t>(logits)) & 15)
    return inval("ids, mask and logits must be 16-byte aligned");
  if (B < 1 || B > m->cfg.max_batch || S < 1 || S > m->cfg.max_seq)
    return inval("B or S out of range");
  if (m->cfg.n_dec_layers) return inval("an encoder-decoder model runs gm_forward_seq2seq");
  m->stats.forwards++;
  if (m->cfg.kv_cache) m->cache_B = B;   // the forward fills the cache for these B sequences
  if (m->exec_mode == GM_EXEC_FRAGMENTED)
    return forward_fragmented(m, gm_model::Frag{B, S, ids, mask, logits, {}, {}}, stream,
                              [&](hipStream_t cs, Seg* sg) {
                                enqueue(m, B, S, ids, mask, logits, cs, nullptr, sg);
                              });
  if (m->exec_mode == GM_EXEC_EAGER) {
    enqueue(m, B, S, ids, mask, logits, stream);
    HIP_TRY(hipGetLastError());
    m->stats.eager_forwards++;
    if (m->debug_sync) {
      m->stats.host_syncs_in_forward++;
      HIP_TRY(hipStreamSynchronize(stream));
    }
    return GM_OK;
  }
  return launch_graph(m, GraphEntry{0, B, S, ids, mask, logits, nullptr, nullptr, 0}, stream,
                      [&](hipStream_t cs) { enqueue(m, B, S, ids, mask, logits, cs); });
}

int gm_forward_seq2seq(gm_model* m, int32_t B, int32_t Ss, const int32_t* src_ids,
                       const int32_t* src_mask, int32_t St, const int32_t* tgt_ids,
                       const int32_t* tgt_mask, void* logits, hipStream_t stream) {
  if (!m) return inval("model is NULL");
  if (!m->cfg.n_dec_layers) return inval("not an encoder-decoder model (n_dec_layers == 0)");
  if (!src_ids || !src_mask || !tgt_ids || !tgt_mask || !logits)
    return inval("inputs and logits must be non-NULL");
  if ((reinterpret_cast<uintptr_t>(src_ids) | reinterpret_cast<uintptr_t>(src_mask) |
       reinterpret_cast<uintptr_t>(tgt_ids) | reinterpret_cast<uintptr_t>(tgt_mask) |
       reinterpret_cast<uintptr_t>(logits)) & 15)
    return inval("inputs and logits must be 16-byte aligned");
  if (B < 1 || B > m->cfg.max_batch || Ss < 1 || Ss > m->cfg.max_seq || St < 1 ||
      St > m->cfg.max_tgt)
    return inval("B, S_src or S_tgt out of range");
  m->stats.forwards++;
  if (m->exec_mode == GM_EXEC_FRAGMENTED) {
    gm_model::Frag key{B, Ss, src_ids, src_mask, logits, {}, {}};
    key.S2 = St;
    key.ids2 = tgt_ids;
    key.mask2 = tgt_mask;
    return forward_fragmented(m, key, stream, [&](hipStream_t cs, Seg* sg) {
      enqueue_seq2seq(m, B, Ss, src_ids, src_mask, St, tgt_ids, tgt_mask, logits, cs, nullptr, sg);
    });
  }
  if (m->exec_mode == GM_EXEC_EAGER) {
    enqueue_seq2seq(m, B, Ss, src_ids, src_mask, St, tgt_ids, tgt_mask, logits, stream);
    HIP_TRY(hipGetLastError());
    m->stats.eager_forwards++;
    return GM_OK;
  }
  GraphEntry key{2, B, Ss, src_ids, src_mask, logits, nullptr, nullptr, 0};
  key.S2 = St;
  key.ids2 = tgt_ids;
  key.mask2 = tgt_mask;
  return launch_graph(m, key, stream, [&](hipStream_t cs) {
    enqueue_seq2seq(m, B, Ss, src_ids, src_mask, St, tgt_ids, tgt_mask, logits, cs);
  });
}

int gm_decode_step(gm_model* m, int32_t B, const int32_t* ids, void* logits, int32_t* next,
                   hipStream_t stream) {
  if (!m) return inval("model is NULL");
  if (!ids || !logits) return inval("ids and logits must be non-NULL");
  if ((reinterpret_cast<uintptr_t>(ids) | reinterpret_cast<uintptr_t>(logits) |
       reinterpret_cast<uintptr_t>(next)) & 15)
    return inval("ids, logits and next must be 16-byte aligned");
  if (!m->cfg.kv_cache) return inval("the model was created without kv_cache");
  if (m->cache_B == 0) return inval("no prefill (gm_forward_ex) has filled the KV cache");
  if (B != m->cache_B) return inval("B must equal the batch of the last prefill");
  if (m->exec_mode == GM_EXEC_FRAGMENTED)
    return inval("fragmented execution covers gm_forward only");
  m->stats.decode_steps++;
  const Dec dec{next};
  if (m->exec_mode == GM_EXEC_EAGER) {
    enqueue(m, B, 1, ids, nullptr, logits, stream, nullptr, nullptr, &dec);
    HIP_TRY(hipGetLastError());
    m->stats.eager_forwards++;
    if (m->debug_sync) {
      m->stats.host_syncs_in_forward++;
      HIP_TRY(hipStreamSynchronize(stream));
    }
    return GM_OK;
  }
  return launch_graph(m, GraphEntry{1, B, 1, ids, nullptr, logits, next, nullptr, 0}, stream,
                      [&](hipStream_t cs) { enqueue(m, B, 1, ids, nullptr, logits, cs, nullptr, nullptr, &dec); });
}

int gm_profile_forward(gm_model* m, int32_t B, int32_t S, const int32_t* ids,
                       const int32_t* mask, void* logits, hipStream_t stream,
                       gm_kernel_time* out, int32_t cap, int32_t* n_out) {
  if (!m || !out || !n_out) return inval("NULL argument");
  if (m->cfg.n_dec_layers) return inval("profiling covers decoder-only and encoder-only forwards");
  if (!ids || !mask || !logits) return inval("ids, mask and logits must be non-NULL");
  if ((reinterpret_cast<uintptr_t>(ids) | reinterpret_cast<uintptr_t>(mask) |
       reinterpret_cast<uintptr_t>(logits)) & 15)
    return inval("ids, mask and logits must be 16-byte aligned");
  if (B < 1 || B > m->cfg.max_batch || S < 1 || S > m->cfg.max_seq)
    return inval("B or S out of range");
  Prof prof;
  prof.s = stream;
  enqueue(m, B, S, ids, mask, logits, stream, &prof);
  hipError_t e = hipGetLastError();
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  int rc = GM_OK;
  if (e != hipSuccess) rc = hip_fail(e, "profile");
  else if (!prof.ok || prof.ev.size() != prof.rec.size() + 1) rc = inval("event creation failed");
  const int n = static_cast<int>(prof.rec.size());
  *n_out = n;
  for (int i = 0; rc == GM_OK && i < n && i < cap; ++i) {
    float ms = 0.f;
    hipEventElapsedTime(&ms, prof.ev[i], prof.ev[i + 1]);
    out[i] = prof.rec[i];
    out[i].ms = ms;
  }
  for (hipEvent_t ev : prof.ev) hipEventDestroy(ev);
  return rc;
}

int gm_debug_forward_layers(gm_model* m, int32_t B, int32_t S, const int32_t* ids,
                            const int32_t* mask, void* logits, hipStream_t stream, void* dump,
                            uint64_t dump_bytes) {
  if (!m || !dump) return inval("NULL argument");
  const gm_config& c = m->cfg;
  if (c.n_dec_layers || c.norm_place != GM_NORM_PRE)
    return inval("layer dumps cover pre-norm decoder-only and encoder-only models");
  if (!ids || !mask || !logits) return inval("ids, mask and logits must be non-NULL");
  if ((reinterpret_cast<uintptr_t>(ids) | reinterpret_cast<uintptr_t>(mask) |
       reinterpret_cast<uintptr_t>(logits) | reinterpret_cast<uintptr_t>(dump)) & 15)
    return inval("ids, mask, logits and dump must be 16-byte aligned");
  if (B < 1 || B > c.max_batch || S < 1 || S > c.max_seq) return inval("B or S out of range");
  Dump d;
  d.base = static_cast<char*>(dump);
  d.esz = m->esz;
  d.T = static_cast<size_t>(B) * S;
  d.d = c.d_model;
  d.ff = c.d_ff;
  if (dump_bytes < c.n_layers * d.layer_elems() * d.esz) return inval("dump buffer too small");
  m->stats.forwards++;
  m->stats.eager_forwards++;
  if (c.kv_cache) m->cache_B = B;
  enqueue(m, B, S, ids, mask, logits, stream, nullptr, nullptr, nullptr, &d);
  HIP_TRY(hipGetLastError());
  return GM_OK;
}

int gm_forward_noalloc(gm_model* m, int32_t B, int32_t S, const int32_t* ids,
                       const int32_t* mask, void* logits, hipStream_t stream) {
  if (!m) return inval("model is NULL");
  const gm_config& c = m->cfg;
  if (c.n_dec_layers) return inval("an encoder-decoder model runs gm_forward_seq2seq");
  if (!ids || !mask || !logits) return inval("ids, mask and logits must be non-NULL");
  if ((reinterpret_cast<uintptr_t>(ids) | reinterpret_cast<uintptr_t>(mask) |
       reinterpret_cast<uintptr_t>(logits)) & 15)
    return inval("ids, mask and logits must be 16-byte aligned");
  if (B < 1 || B > c.max_batch || S < 1 || S > c.max_seq) return inval("B or S out of range");
  // workspace: h, a, qkv, ctx, f (and tmp for post-norm models), each
  // rounded up to 256 bytes, carved from the static scratch array
  const size_t T = static_cast<size_t>(B) * S, d = c.d_model, es = m->esz;
  auto up = [](size_t n) { return (n + 255) & ~size_t(255); };
  const size_t sizes[6] = {T * d * es, T * d * es, T * 3 * d * es, T * d * es,
                           T * c.d_ff * es, c.norm_place == GM_NORM_POST ? T * d * es : 0};
  size_t total = 0;
  for (size_t z : sizes) total += up(z);
  if (total > kScratchBytes) {
    g_last_error = "workspace of " + std::to_string(total) + " bytes exceeds the static scratch of " +
                   std::to_string(kScratchBytes) + " bytes (B * S * (6 d + d_ff) * element size)";
    return GM_E_INVAL;
  }
  int dev = -1;
  HIP_TRY(hipGetDevice(&dev));
  if (dev != m->device) return inval("the current device is not the model's device");
  char* base = static_cast<char*>(m->scratch);
  void* ptrs[6];
  size_t off = 0;
  for (int i = 0; i < 6; ++i) {
    ptrs[i] = sizes[i] ? base + off : nullptr;
    off += up(sizes[i]);
  }
  Work w;
  w.h = ptrs[0];
  w.a = ptrs[1];
  w.qkv = ptrs[2];
  w.ctx = ptrs[3];
  w.f = ptrs[4];
  w.tmp = ptrs[5];
  m->stats.forwards++;
  m->stats.eager_forwards++;
  if (c.kv_cache) m->cache_B = B;
  enqueue(m, B, S, ids, mask, logits, stream, nullptr, nullptr, nullptr, nullptr, &w);
  HIP_TRY(hipGetLastError());
  return GM_OK;
}

int gm_forward(gm_model* m, const int32_t* ids, const int32_t* mask, void* logits,
               hipStream_t stream) {
  if (!m) return inval("model is NULL");
  return gm_forward_ex(m, m->cfg.max_batch, m->cfg.max_seq, ids, mask, logits, stream);
}

int gm_read_decisions(gm_model* m, gm_decisions* out, hipStream_t stream) {
  if (!m || !out) return inval("model or out is NULL");
  HIP_TRY(hipStreamSynchronize(stream));
  std::vector<int32_t> st(m->n_state);
  HIP_TRY(hipMemcpy(st.data(), m->state, st.size() * sizeof(int32_t), hipMemcpyDeviceToHost));
  memset(out, 0, sizeof(*out));
  out->pad_any = st[kPadAny];
  out->regrow = st[kRegrow];
  out->need = st[kNeed];
  out->cached_len = st[kCachedLen];
  out->n_clamp_sites = n_sites(m->cfg);
  for (int i = 0; i < out->n_clamp_sites; ++i) {
    out->clamp[i] = st[kClampBase + i];
    uint32_t u = static_cast<uint32_t>(st[kAbsmaxBase + i]);
    float f;
    memcpy(&f, &u, 4);
    out->clamp_absmax[i] = f;
    out->clamp_nan[i] = st[kNanBase + i];
  }
  out->forward_index = st[kFwdIndex];
  out->rope_long = st[kRopeLong];
  out->pad_any_tgt = st[kPadAnyTgt];
  return GM_OK;
}

const int32_t* gm_decisions_device_ptr(const gm_model* m) { return m ? m->state : nullptr; }

int gm_check_error(gm_model* m, int32_t* code, int32_t* index) {
  if (!m || !code || !index) return inval("NULL argument");
  HIP_TRY(hipDeviceSynchronize());
  int32_t w = 0;
  HIP_TRY(hipMemcpy(&w, m->state + kTrapSticky, sizeof(w), hipMemcpyDeviceToHost));
  const uint32_t u = static_cast<uint32_t>(w);
  *code = w ? static_cast<int32_t>(u >> 24) : GM_TRAP_NONE;
  *index = w ? static_cast<int32_t>(u & 0xFFFFFFu) : 0;
  const int32_t zero = 0;
  HIP_TRY(hipMemcpy(m->state + kTrapSticky, &zero, sizeof(zero), hipMemcpyHostToDevice));
  return GM_OK;
}

int gm_flush_effects(gm_model* m, gm_effect_cb cb, void* user, int32_t* n_dropped) {
  if (!m) return inval("model is NULL");
  HIP_TRY(hipDeviceSynchronize());
  int32_t cd[2], ld[2] = {0, 0};
  HIP_TRY(hipMemcpy(cd, m->state + kFifoCount, sizeof(cd), hipMemcpyDeviceToHost));
  HIP_TRY(hipMemcpy(ld, m->state + kLogCount, sizeof(ld), hipMemcpyDeviceToHost));
  const int n = cd[0] < kFifoCap ? cd[0] : kFifoCap;
  std::vector<EffectRec> recs(n);
  if (n) HIP_TRY(hipMemcpy(recs.data(), m->fifo, n * sizeof(EffectRec), hipMemcpyDeviceToHost));
  std::vector<float> arena(ld[0] > 0 ? ld[0] : 0);
  if (!arena.empty())
    HIP_TRY(hipMemcpy(arena.data(), m->log_arena, arena.size() * sizeof(float), hipMemcpyDeviceToHost));
  const int32_t zero[2] = {0, 0};
  HIP_TRY(hipMemcpy(m->state + kFifoCount, zero, sizeof(zero), hipMemcpyHostToDevice));
  HIP_TRY(hipMemcpy(m->state + kLogCount, zero, sizeof(zero), hipMemcpyHostToDevice));
  if (n_dropped) *n_dropped = cd[1];
  if (cb)
    for (const EffectRec& r : recs) {
      gm_effect e{r.forward, r.kind, r.layer, r.site, r.value, r.count,
                  r.count ? arena.data() + r.offset : nullptr};
      cb(&e, user);
    }
  return GM_OK;
}

int gm_set_mask_guard(gm_model* m, const int32_t* expected, int32_t B, int32_t S) {
  if (!m) return inval("model is NULL");
  if (expected && (B < 1 || S < 1)) return inval("expected mask shape must be positive");
  if (reinterpret_cast<uintptr_t>(expected) & 15) return inval("expected must be 16-byte aligned");
  HIP_TRY(hipDeviceSynchronize());
  // captured graphs hold the previous guard: drop them
  for (auto& g : m->graphs) HIP_TRY(hipGraphExecDestroy(g.exec));
  m->graphs.clear();
  for (auto& f : m->frags)
    for (hipGraphExec_t e : f.execs) HIP_TRY(hipGraphExecDestroy(e));
  m->frags.clear();
  m->guard_expected = expected;
  m->guard_B = expected ? B : 0;
  m->guard_S = expected ? S : 0;
  return GM_OK;
}

int gm_trap_info(int32_t code, const char** exception_type, const char** message) {
  static const char* const kType[] = {"", "IndexError", "ValueError", "ValueError", "IndexError",
                                      "ValueError"};
  static const char* const kMsg[] = {"", "token id out of range",
                                     "attention mask values must be 0 or 1",
                                     "rotary position exceeds the table capacity",
                                     "sequence exceeds the KV cache capacity",
                                     "unsupported attention mask"};
  if (code < 1 || code > GM_TRAP_MASK_GUARD) return inval("unknown trap code");
  if (exception_type) *exception_type = kType[code];
  if (message) *message = kMsg[code];
  return GM_OK;
}

int gm_debug_buffer(const gm_model* m, int32_t which, void** ptr, uint64_t* bytes) {
  if (!m || !ptr || !bytes) return inval("NULL argument");
  const gm_config& c = m->cfg;
  const uint64_t T = static_cast<uint64_t>(c.max_batch) * c.max_seq;
  const uint64_t d = c.d_model;
  switch (which) {
    case 0: *ptr = m->h; *bytes = T * d * m->esz; break;
    case 1: *ptr = m->a; *bytes = T * d * m->esz; break;
    case 2: *ptr = m->qkv; *bytes = T * 3 * d * m->esz; break;
    case 3: *ptr = m->ctx; *bytes = T * d * m->esz; break;
    case 4: *ptr = m->f; *bytes = T * c.d_ff * m->esz; break;
    default: return inval("which out of [0, 4]");
  }
  return GM_OK;
}

int gm_get_stats(const gm_model* m, gm_stats* out) {
  if (!m || !out) return inval("NULL argument");
  *out = m->stats;
  return GM_OK;
}

}  // extern "C"
