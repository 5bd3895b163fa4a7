// gm_rows.hip -- the small kernels of the forward: the prologue that
// evaluates every device predicate, the rotary-table fill, the row kernel
// (embedding gather, LayerNorm/RMSNorm, fp16 clamp select) and the effect
// emitter that runs last.
#include <math.h>

#include "gm_device.h"
#include "gm_kernels.h"

namespace gm {

// ------------------------------------------------------------ prologue
// One workgroup.  Evaluates, without any host read-back:
//  * the input guards of rule [Trap]: ids in [0, vocab), mask in {0, 1},
//    and for rotary models max(position)+1 <= capacity; the failing guard
//    that runs first (smallest code), at its first offending position,
//    becomes this forward's trap word;
//  * the padding predicate of the `mask.any()` branch (pad_any) and, per
//    sequence, 1 + the position of its last unmasked key;
//  * the rotary-cache predicate need > cached_len; when it holds (and no
//    guard failed) the new rows [cached_len, need) are scheduled for the
//    fill kernel and cached_len becomes need (a memoised initialisation,
//    which is what makes the hoisted branch body safe to run every time);
//  * resets the per-forward clamp-site slots.
constexpr int kPrologueThreads = 1024;

__global__ __launch_bounds__(kPrologueThreads) void k_prologue(
    const int32_t* __restrict__ ids, const int32_t* __restrict__ mask, int B,
    int S, int vocab, int rotary, int capacity, int n_sites,
    const int32_t* __restrict__ expected, int guard_meta_ok,
    float* __restrict__ log_stage, int log_vals, int rope_orig,
    int32_t* __restrict__ state, int pad_slot, int padcount_slot, int kvlen_base,
    int index_offset, int merge) {
  __shared__ int kv[1024];
  __shared__ uint32_t red_trap[kPrologueThreads / 64];
  __shared__ int red_pad[kPrologueThreads / 64];
  __shared__ int red_need[kPrologueThreads / 64];
  const int tid = threadIdx.x;
  for (int b = tid; b < B; b += blockDim.x) kv[b] = 0;
  for (int i = tid; i < (merge ? 0 : n_sites); i += blockDim.x) {
    state[kClampBase + i] = 0;
    state[kAbsmaxBase + i] = 0;
    state[kNanBase + i] = 0;
  }
  for (int i = tid; i < (merge ? 0 : log_vals); i += blockDim.x) log_stage[i] = 0.f;
  __syncthreads();
  uint32_t trap = kTrapNone;
  int pads = 0, need = 0;
  const int n = B * S;
  for (int i = tid; i < n; i += blockDim.x) {
    const int id = ids[i];
    const int mk = mask[i];
    const int s = i % S;
    const uint32_t pos_i = static_cast<uint32_t>(index_offset + i);
    if (id < 0 || id >= vocab) trap = min(trap, (1u << 24) | pos_i);
    if (mk != 0 && mk != 1) trap = min(trap, (2u << 24) | pos_i);
    // `if not torch.equal(mask, expected): raise` as (mask == expected).all()
    if (expected && guard_meta_ok && mk != expected[i])
      trap = min(trap, (5u << 24) | static_cast<uint32_t>(i));
    if (mk == 0) ++pads;
    else atomicMax(&kv[i / S], s + 1);
    need = max(need, s + 1);           // positions are 0..S-1
  }
  // wave reductions, then across waves
  for (int o = 32; o > 0; o >>= 1) {
    uint32_t t2 = __shfl_xor(trap, o, 64);
    trap = min(trap, t2);
    pads += __shfl_xor(pads, o, 64);
    need = max(need, __shfl_xor(need, o, 64));
  }
  const int w = tid >> 6;
  if ((tid & 63) == 0) {
    red_trap[w] = trap;
    red_pad[w] = pads;
    red_need[w] = need;
  }
  __syncthreads();
  for (int b = tid; b < B; b += blockDim.x) state[kvlen_base + b] = kv[b];
  if (tid == 0 && merge) {
    // second input of an encoder-decoder forward: its guards join the
    // forward's trap word, its padding predicate gets its own slots
    for (int i = 1; i < static_cast<int>(blockDim.x >> 6); ++i) {
      trap = min(trap, red_trap[i]);
      pads += red_pad[i];
    }
    state[kTrapFwd] = static_cast<int32_t>(min(trap, static_cast<uint32_t>(state[kTrapFwd])));
    state[padcount_slot] = pads;
    state[pad_slot] = pads > 0;
  } else if (tid == 0) {
    for (int i = 1; i < static_cast<int>(blockDim.x >> 6); ++i) {
      trap = min(trap, red_trap[i]);
      pads += red_pad[i];
      need = max(need, red_need[i]);
    }
    if (rotary && need > capacity) trap = min(trap, 3u << 24);
    if (expected && !guard_meta_ok) trap = min(trap, 5u << 24);   // shapes differ: never equal
    int regrow = 0;
    const int cached = state[kCachedLen];
    int from = 0, to = 0;
    state[kRopeLong] = rope_orig > 0 && need > rope_orig;
    if (rotary && rope_orig <= 0 && trap == kTrapNone && need > cached) {
      regrow = 1;
      from = cached;
      to = need;
      state[kCachedLen] = need;
    }
    state[kTrapFwd] = static_cast<int32_t>(trap);
    state[padcount_slot] = pads;
    state[pad_slot] = pads > 0;
    state[kPadAnyTgt] = 0;
    state[kPadCountTgt] = 0;
    state[kNeed] = need;
    state[kRegrow] = regrow;
    state[kRegrowFrom] = from;
    state[kRegrowTo] = to;
    const int f = state[kFwdCount];
    state[kFwdIndex] = f;
    state[kFwdCount] = f + 1;
  }
}

void launch_prologue(const int32_t* ids, const int32_t* mask, int B, int S,
                     int vocab, int rotary, int capacity, int n_sites,
                     const int32_t* expected, int guard_meta_ok,
                     float* log_stage, int log_vals, int rope_orig,
                     int32_t* state, hipStream_t s, int second, int index_offset,
                     int kvlen_base) {
  // the second input (an encoder-decoder's target) has its own padding
  // slots and key lengths; its positions follow the first input's in the
  // trap index
  hipLaunchKernelGGL(k_prologue, dim3(1), dim3(kPrologueThreads), 0, s, ids,
                     mask, B, S, vocab, rotary, capacity, n_sites, expected, guard_meta_ok,
                     log_stage, log_vals, rope_orig, state, second ? kPadAnyTgt : kPadAny,
                     second ? kPadCountTgt : kPadCount, kvlen_base, index_offset, second);
}

// ------------------------------------------------------------ tensor log
// max |x| per sequence for the deferred log of a layer ([Defer] with a tensor
// argument: the value is taken here, at the call site, and replayed after
// the forward).  Absolute values as float bits compare like integers, and a
// NaN's bits exceed every number's, so an integer max propagates NaN.
// A clamp site whose select is still pending (applied by the next reader of
// h) is applied here too: the log sees h as the program holds it.
template <typename T>
__global__ __launch_bounds__(256) void k_log_seqmax(const T* __restrict__ x, int S, int d,
                                                     float* __restrict__ stage,
                                                     const int32_t* __restrict__ state,
                                                     int site, float thr) {
  const int b = blockIdx.y;
  const long long n = static_cast<long long>(S) * d;
  const T* xs = x + static_cast<long long>(b) * n;
  const bool trip = site >= 0 && clamp_trip(state, site, thr);
  uint32_t mx = 0;
  for (long long i = blockIdx.x * 256ll + threadIdx.x; i < n; i += 256ll * gridDim.x) {
    float v = to_f32(xs[i]);
    if (trip) v = round_as<T>(fminf(fmaxf(v, -thr), thr));
    mx = max(mx, __float_as_uint(v) & 0x7FFFFFFFu);
  }
  mx = wave_max_u32(mx);
  __shared__ uint32_t red[4];
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = mx;
  __syncthreads();
  if (threadIdx.x == 0) {
    mx = max(max(red[0], red[1]), max(red[2], red[3]));
    atomicMax(reinterpret_cast<unsigned int*>(stage) + b, mx);
  }
}

void launch_log_seqmax(const void* x, int dtype, int B, int S, int d, float* stage, int layer,
                       const int32_t* state, int clamp_site, float clamp_thr, hipStream_t s) {
  const dim3 grid(32, B), block(256);
  float* st = stage + static_cast<long long>(layer) * B;
  if (dtype == kF32)
    hipLaunchKernelGGL(k_log_seqmax<float>, grid, block, 0, s, static_cast<const float*>(x), S, d,
                       st, state, clamp_site, clamp_thr);
  else if (dtype == kBF16)
    hipLaunchKernelGGL(k_log_seqmax<bf16_t>, grid, block, 0, s, static_cast<const bf16_t*>(x), S,
                       d, st, state, clamp_site, clamp_thr);
  else
    hipLaunchKernelGGL(k_log_seqmax<f16_t>, grid, block, 0, s, static_cast<const f16_t*>(x), S, d,
                       st, state, clamp_site, clamp_thr);
}

// ------------------------------------------------------------ rotary fill
// Fills rows [from, to) of the cos/sin tables (both [capacity, hd/2] fp32)
// with cos/sin(p * theta_i), theta_i = base^(-2i/hd).  theta_i is rounded to
// fp32 (the frequency buffer is fp32); angle, cos and sin are evaluated in
// fp64 and rounded once to fp32.  A row depends only on p, so a grown table
// equals a freshly built one.
__global__ __launch_bounds__(256) void k_rope_fill(float* __restrict__ cs,
                                                    float* __restrict__ sn,
                                                    int hd, double base,
                                                    const int32_t* __restrict__ state) {
  const int from = state[kRegrowFrom];
  const int to = state[kRegrowTo];
  const int half = hd / 2;
  const long long total = static_cast<long long>(to - from) * half;
  for (long long e = blockIdx.x * 256ll + threadIdx.x; e < total;
       e += static_cast<long long>(gridDim.x) * 256) {
    const int p = from + static_cast<int>(e / half);
    const int i = static_cast<int>(e % half);
    const double theta = static_cast<double>(
        static_cast<float>(pow(base, -2.0 * static_cast<double>(i) / hd)));
    const double ang = static_cast<double>(p) * theta;
    cs[static_cast<long long>(p) * half + i] = static_cast<float>(cos(ang));
    sn[static_cast<long long>(p) * half + i] = static_cast<float>(sin(ang));
  }
}

void launch_rope_fill(float* cs, float* sn, int hd, double base,
                      const int32_t* state, hipStream_t s) {
  hipLaunchKernelGGL(k_rope_fill, dim3(256), dim3(256), 0, s, cs, sn, hd, base, state);
}

// Rows [0, rows) of one scaled frequency set (the long/short select of a
// Phi-4-style rotary embedding): theta_i = 1 / (f_i * base^(2i/hd)) with the
// base power rounded to fp32 and the product and quotient as fp32
// operations; cos and sin of p * theta_i in fp64, rounded to fp32, times the
// attention factor as an fp32 product.
__global__ __launch_bounds__(256) void k_rope_fill_scaled(float* __restrict__ cs,
                                                           float* __restrict__ sn, int hd,
                                                           double base,
                                                           const float* __restrict__ factor,
                                                           float attn, int rows) {
  const int half = hd / 2;
  const long long total = static_cast<long long>(rows) * half;
  for (long long e = blockIdx.x * 256ll + threadIdx.x; e < total;
       e += static_cast<long long>(gridDim.x) * 256) {
    const int p = static_cast<int>(e / half);
    const int i = static_cast<int>(e % half);
    const float ib = static_cast<float>(pow(base, 2.0 * static_cast<double>(i) / hd));
    const float denom = static_cast<float>(static_cast<double>(factor[i]) * ib);
    const double theta = static_cast<double>(static_cast<float>(1.0 / static_cast<double>(denom)));
    const double ang = static_cast<double>(p) * theta;
    const float c = static_cast<float>(cos(ang)), sv = static_cast<float>(sin(ang));
    cs[e] = static_cast<float>(static_cast<double>(c) * attn);
    sn[e] = static_cast<float>(static_cast<double>(sv) * attn);
  }
}

void launch_rope_fill_scaled(float* cs, float* sn, int hd, double base, const float* factor,
                             float attn, int rows, hipStream_t s) {
  hipLaunchKernelGGL(k_rope_fill_scaled, dim3(256), dim3(256), 0, s, cs, sn, hd, base, factor,
                     attn, rows);
}

// ------------------------------------------------------------ row kernel
// One wavefront per row of d elements, 16-byte vector accesses.
//  1. source: embedding gather R(tok_emb[id] + pos_emb[s]) written to x, or
//     the stored row x;
//  2. fp16 overflow guard of a clamp site (rule [Where] as a select): if the
//     site's reduction says NaN-free and max |h| > thr, the row is replaced by
//     R(clamp(h, -thr, thr)) and written back; otherwise it is untouched;
//  3. optional LayerNorm / RMSNorm with fp32 statistics, stored to out.
template <typename T> struct Vec;
template <> struct Vec<float> { typedef f32x4v type; static constexpr int n = 4; };
template <> struct Vec<bf16_t> { typedef u32x4 type; static constexpr int n = 8; };
template <> struct Vec<f16_t> { typedef u32x4 type; static constexpr int n = 8; };

template <typename T>
__device__ __forceinline__ void vload(const T* p, float* v) {
  typedef typename Vec<T>::type V;
  V raw = *reinterpret_cast<const V*>(p);
  const T* e = reinterpret_cast<const T*>(&raw);
#pragma unroll
  for (int i = 0; i < Vec<T>::n; ++i) v[i] = to_f32(e[i]);
}
template <typename T>
__device__ __forceinline__ void vstore(T* p, const float* v) {
  typedef typename Vec<T>::type V;
  V raw;
  T* e = reinterpret_cast<T*>(&raw);
#pragma unroll
  for (int i = 0; i < Vec<T>::n; ++i) e[i] = from_f32<T>(v[i]);
  *reinterpret_cast<V*>(p) = raw;
}

template <typename T, int MAXV>
__global__ __launch_bounds__(256) void k_rownorm(RowArgs a) {
  constexpr int VN = Vec<T>::n;
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int d = a.d;
  const int nvec = d / VN;
  bool trip = false;
  if (a.clamp_site >= 0) {
    trip = clamp_trip(a.state, a.clamp_site, a.clamp_thr);
    if (blockIdx.x == 0 && threadIdx.x == 0) a.state[kClampBase + a.clamp_site] = trip;
  }
  if (row >= a.rows) return;
  // the norm's gain and bias vectors of this lane, fetched before the row
  // so that they are in flight with it (not one round trip per vector after
  // the statistics)
  typedef typename Vec<T>::type RV;
  RV graw[MAXV], braw[MAXV];
  const T* g = static_cast<const T*>(a.g);
  const T* bb = static_cast<const T*>(a.b);
  if (a.norm >= 0) {
#pragma unroll
    for (int j = 0; j < MAXV; ++j) {
      const int c = (lane + 64 * j);
      if (c < nvec) {
        graw[j] = *reinterpret_cast<const RV*>(g + c * VN);
        if (bb) braw[j] = *reinterpret_cast<const RV*>(bb + c * VN);
      }
    }
  }
  float v[MAXV][VN];
  T* x = static_cast<T*>(a.x) + static_cast<long long>(row) * d;
  if (a.ids) {
    int id = a.ids[row];
    id = id < 0 ? 0 : (id >= a.vocab ? a.vocab - 1 : id);   // in bounds even when trapped
    const T* e = static_cast<const T*>(a.tok_emb) + static_cast<long long>(id) * d;
    const int position = a.pos ? a.pos[row] : row % a.seq;
    const T* p = a.pos_emb ? static_cast<const T*>(a.pos_emb) + static_cast<long long>(position) * d
                           : nullptr;
    // every load of the row first, then the stores (a store between two
    // loads would make the second wait for it)
    RV praw[MAXV];
#pragma unroll
    for (int j = 0; j < MAXV; ++j) {
      const int c = (lane + 64 * j);
      if (c < nvec) {
        vload(e + c * VN, v[j]);
        if (p) praw[j] = *reinterpret_cast<const RV*>(p + c * VN);
      }
    }
#pragma unroll
    for (int j = 0; j < MAXV; ++j) {
      const int c = (lane + 64 * j);
      if (c < nvec) {
        if (p) {
          const T* pe = reinterpret_cast<const T*>(&praw[j]);
#pragma unroll
          for (int i = 0; i < VN; ++i) v[j][i] += to_f32(pe[i]);
        }
#pragma unroll
        for (int i = 0; i < VN; ++i) v[j][i] = round_as<T>(v[j][i]);
        vstore(x + c * VN, v[j]);
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < MAXV; ++j) {
      const int c = (lane + 64 * j);
      if (c < nvec) vload(x + c * VN, v[j]);
    }
    if (trip) {
      const float t = a.clamp_thr;
#pragma unroll
      for (int j = 0; j < MAXV; ++j) {
        const int c = (lane + 64 * j);
        if (c < nvec) {
#pragma unroll
          for (int i = 0; i < VN; ++i) v[j][i] = round_as<T>(fminf(fmaxf(v[j][i], -t), t));
          vstore(x + c * VN, v[j]);
        }
      }
    }
  }
  if (a.norm < 0) return;
  // statistics in fp32: mean and centred second moment (LayerNorm) or mean square (RMSNorm)
  float s1 = 0.f;
  if (a.norm == 0) {
#pragma unroll
    for (int j = 0; j < MAXV; ++j)
      if (lane + 64 * j < nvec)
#pragma unroll
        for (int i = 0; i < VN; ++i) s1 += v[j][i];
    s1 = wave_sum(s1);
  }
  const float mean = a.norm == 0 ? s1 / d : 0.f;
  float s2 = 0.f;
#pragma unroll
  for (int j = 0; j < MAXV; ++j)
    if (lane + 64 * j < nvec)
#pragma unroll
      for (int i = 0; i < VN; ++i) {
        const float c = v[j][i] - mean;
        s2 += c * c;
      }
  s2 = wave_sum(s2);
  const float rstd = 1.0f / sqrtf(s2 / d + a.eps);
  T* out = static_cast<T*>(a.out) + static_cast<long long>(row) * d;
#pragma unroll
  for (int j = 0; j < MAXV; ++j) {
    const int c = (lane + 64 * j);
    if (c < nvec) {
      float gv[VN], bv[VN];
      const T* ge = reinterpret_cast<const T*>(&graw[j]);
#pragma unroll
      for (int i = 0; i < VN; ++i) gv[i] = to_f32(ge[i]);
      if (bb) {
        const T* be = reinterpret_cast<const T*>(&braw[j]);
#pragma unroll
        for (int i = 0; i < VN; ++i) bv[i] = to_f32(be[i]);
      } else {
#pragma unroll
        for (int i = 0; i < VN; ++i) bv[i] = 0.f;
      }
#pragma unroll
      for (int i = 0; i < VN; ++i) v[j][i] = (v[j][i] - mean) * rstd * gv[i] + bv[i];
      vstore(out + c * VN, v[j]);
    }
  }
}

template <typename T>
static void rownorm_t(const RowArgs& a, hipStream_t s) {
  const int nvec = a.d / Vec<T>::n;
  const dim3 grid((a.rows + 3) / 4), block(256);
  if (nvec <= 64) hipLaunchKernelGGL((k_rownorm<T, 1>), grid, block, 0, s, a);
  else if (nvec <= 128) hipLaunchKernelGGL((k_rownorm<T, 2>), grid, block, 0, s, a);
  else if (nvec <= 256) hipLaunchKernelGGL((k_rownorm<T, 4>), grid, block, 0, s, a);
  else if (nvec <= 512) hipLaunchKernelGGL((k_rownorm<T, 8>), grid, block, 0, s, a);
  else hipLaunchKernelGGL((k_rownorm<T, 16>), grid, block, 0, s, a);
}

void launch_rownorm(const RowArgs& a, hipStream_t s) {
  if (a.dtype == kF32) rownorm_t<float>(a, s);
  else if (a.dtype == kBF16) rownorm_t<bf16_t>(a, s);
  else rownorm_t<f16_t>(a, s);
}

// ------------------------------------------------------------ effects
// Last kernel of a forward (rule [Defer]): commits a failed guard to the
// sticky trap word and records nothing else for that forward; otherwise
// appends one record per taken branch, in program order (padding branch,
// rotary regrow, then the clamp sites in layer order), to the FIFO that the
// host replays after the stream completes.  One thread: the order is fixed.
__global__ void k_emit_effects(int32_t* __restrict__ state, EffectRec* __restrict__ fifo,
                               int cap, int n_sites, const float* __restrict__ log_stage,
                               float* __restrict__ arena, int arena_cap, int n_log_layers,
                               int B, int seq2seq) {
  if (threadIdx.x != 0) return;
  const int fwd = state[kFwdIndex];
  const uint32_t trap = static_cast<uint32_t>(state[kTrapFwd]);
  if (trap != kTrapNone) {
    if (state[kTrapSticky] == 0) state[kTrapSticky] = static_cast<int32_t>(trap);
    return;
  }
  int count = state[kFifoCount];
  int dropped = state[kFifoDropped];
  int lcount = state[kLogCount];
  int ldropped = state[kLogDropped];
  auto push = [&](int kind, int layer, int site, float value, int offset, int n) {
    if (count < cap) {
      EffectRec r;
      r.forward = fwd;
      r.kind = kind;
      r.layer = layer;
      r.site = site;
      r.value = value;
      r.offset = offset;
      r.count = n;
      fifo[count] = r;
      ++count;
    } else {
      ++dropped;
    }
  };
  if (state[kPadAny]) push(1, -1, seq2seq ? 0 : -1, static_cast<float>(state[kPadCount]), 0, 0);
  if (seq2seq && state[kPadAnyTgt]) push(1, -1, 1, static_cast<float>(state[kPadCountTgt]), 0, 0);
  if (state[kRegrow]) push(2, -1, -1, static_cast<float>(state[kNeed]), 0, 0);
  const int layers = max(n_sites / 2, n_log_layers);
  for (int l = 0; l < layers; ++l) {
    for (int s2 = 0; s2 < 2; ++s2) {
      const int i = 2 * l + s2;
      if (i < n_sites && state[kClampBase + i])
        push(3, l, s2, __uint_as_float(static_cast<uint32_t>(state[kAbsmaxBase + i])), 0, 0);
    }
    if (l < n_log_layers) {
      // the tensor argument is cloned into the arena; the record points at it
      if (lcount + B <= arena_cap) {
        for (int b = 0; b < B; ++b) arena[lcount + b] = log_stage[l * B + b];
        push(4, l, 0, static_cast<float>(B), lcount, B);
        lcount += B;
      } else {
        ldropped += B;
        ++dropped;
      }
    }
  }
  state[kFifoCount] = count;
  state[kFifoDropped] = dropped;
  state[kLogCount] = lcount;
  state[kLogDropped] = ldropped;
}

void launch_emit_effects(int32_t* state, void* fifo, int cap, int n_sites, const float* log_stage,
                         float* arena, int arena_cap, int n_log_layers, int B, int seq2seq,
                         hipStream_t s) {
  hipLaunchKernelGGL(k_emit_effects, dim3(1), dim3(64), 0, s, state,
                     static_cast<EffectRec*>(fifo), cap, n_sites, log_stage, arena, arena_cap,
                     n_log_layers, B, seq2seq);
}

// ------------------------------------------------------------ row gather
// dst row r = src row row_map[r]; used once at model creation to repack
// weight rows.  row_bytes must be a multiple of 16.
__global__ __launch_bounds__(256) void k_gather_rows(u32x4* __restrict__ dst,
                                                      const u32x4* __restrict__ src,
                                                      const int32_t* __restrict__ map,
                                                      int rows, int row_vecs) {
  const long long total = static_cast<long long>(rows) * row_vecs;
  for (long long e = blockIdx.x * 256ll + threadIdx.x; e < total;
       e += static_cast<long long>(gridDim.x) * 256) {
    const int r = static_cast<int>(e / row_vecs);
    const int c = static_cast<int>(e % row_vecs);
    dst[e] = src[static_cast<long long>(map[r]) * row_vecs + c];
  }
}

void launch_gather_rows(void* dst, const void* src, const int32_t* map, int rows,
                        int row_bytes, hipStream_t s) {
  hipLaunchKernelGGL(k_gather_rows, dim3(1024), dim3(256), 0, s,
                     static_cast<u32x4*>(dst), static_cast<const u32x4*>(src), map,
                     rows, row_bytes / 16);
}

}  // namespace gm
