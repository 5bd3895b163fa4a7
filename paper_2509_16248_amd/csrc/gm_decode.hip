// gm_decode.hip -- the kernels that only a decode step (one new token per
// sequence against a KV cache) needs: its guard/position prologue, the
// append of k and v to the cache, split-key attention over the cache, the
// greedy argmax and the sequence-length update.  The projections, norms and
// effects are the forward's own kernels run on B rows.
#include <math.h>

#include <type_traits>

#include "gm_device.h"
#include "gm_kernels.h"

namespace gm {

// ------------------------------------------------------------ prologue
// The [Trap] guards of a step and the rotary predicate (same memoised regrow
// as the forward's prologue: rows [cached_len, need) are scheduled and
// cached_len becomes need when need > cached_len and no guard failed).  The
// padding branch does not exist in a decode step: pad_any is 0.
constexpr int kDecPrologueThreads = 256;

__global__ __launch_bounds__(kDecPrologueThreads) void k_decode_prologue(
    const int32_t* __restrict__ ids, int B, int vocab, int max_seq, int rotary, int capacity,
    int n_sites, const int32_t* __restrict__ seqlen, int32_t* __restrict__ pos,
    int32_t* __restrict__ state) {
  __shared__ uint32_t red_trap[kDecPrologueThreads / 64];
  __shared__ int red_need[kDecPrologueThreads / 64];
  const int tid = threadIdx.x;
  for (int i = tid; i < n_sites; i += blockDim.x) {
    state[kClampBase + i] = 0;
    state[kAbsmaxBase + i] = 0;
    state[kNanBase + i] = 0;
  }
  uint32_t trap = kTrapNone;
  int need = 0;
  for (int b = tid; b < B; b += blockDim.x) {
    const int id = ids[b];
    const int p = seqlen[b];
    if (id < 0 || id >= vocab) trap = min(trap, (1u << 24) | static_cast<uint32_t>(b));
    if (p >= max_seq) trap = min(trap, (4u << 24) | static_cast<uint32_t>(b));
    need = max(need, p + 1);
    pos[b] = p < max_seq ? p : max_seq - 1;   // in bounds even when trapped
  }
  for (int o = 32; o > 0; o >>= 1) {
    trap = min(trap, static_cast<uint32_t>(__shfl_xor(static_cast<int>(trap), o, 64)));
    need = max(need, __shfl_xor(need, o, 64));
  }
  if ((tid & 63) == 0) {
    red_trap[tid >> 6] = trap;
    red_need[tid >> 6] = need;
  }
  __syncthreads();
  if (tid == 0) {
    for (int i = 1; i < kDecPrologueThreads / 64; ++i) {
      trap = min(trap, red_trap[i]);
      need = max(need, red_need[i]);
    }
    if (rotary && need > capacity) trap = min(trap, 3u << 24);
    int regrow = 0, from = 0, to = 0;
    const int cached = state[kCachedLen];
    if (rotary && trap == kTrapNone && need > cached) {
      regrow = 1;
      from = cached;
      to = need;
      state[kCachedLen] = need;
    }
    state[kTrapFwd] = static_cast<int32_t>(trap);
    state[kPadCount] = 0;
    state[kPadAny] = 0;
    state[kNeed] = need;
    state[kRegrow] = regrow;
    state[kRegrowFrom] = from;
    state[kRegrowTo] = to;
    const int f = state[kFwdCount];
    state[kFwdIndex] = f;
    state[kFwdCount] = f + 1;
  }
}

void launch_decode_prologue(const int32_t* ids, int B, int vocab, int max_seq, int rotary,
                            int capacity, int n_sites, const int32_t* seqlen, int32_t* pos,
                            int32_t* state, hipStream_t s) {
  hipLaunchKernelGGL(k_decode_prologue, dim3(1), dim3(kDecPrologueThreads), 0, s, ids, B, vocab,
                     max_seq, rotary, capacity, n_sites, seqlen, pos, state);
}

// ------------------------------------------------------------ KV append
// One thread per 16-byte vector of k or v: row r of the fused q|k|v output
// goes to (sequence b, position p) of this layer's cache, head-major.
__global__ __launch_bounds__(256) void k_kv_store(KvArgs a, int vn) {
  if (!a.S && static_cast<uint32_t>(a.state[kTrapFwd]) != kTrapNone) return;
  const int esz = a.dtype == kF32 ? 4 : 2;
  const int nv = a.d / vn;                      // vectors per k (or v) row
  const long long total = static_cast<long long>(a.rows) * 2 * nv;
  const char* qkv = static_cast<const char*>(a.qkv);
  for (long long e = blockIdx.x * 256ll + threadIdx.x; e < total;
       e += static_cast<long long>(gridDim.x) * 256) {
    const int row = static_cast<int>(e / (2 * nv));
    const int rem = static_cast<int>(e % (2 * nv));
    const int which = rem / nv, c = (rem % nv) * vn;
    const int h = c / a.hd, i = c % a.hd;
    int b, p;
    if (a.S) {
      b = row / a.S;
      p = row % a.S;
    } else {
      b = row;
      p = a.pos[row];
    }
    const long long src = (static_cast<long long>(row) * 3 * a.d + (1 + which) * a.d + c) * esz;
    const long long dst =
        ((((static_cast<long long>(b) * a.H + h) * a.max_seq) + p) * a.hd + i) * esz;
    char* cache = static_cast<char*>(which ? a.vc : a.kc);
    *reinterpret_cast<u32x4*>(cache + dst) = *reinterpret_cast<const u32x4*>(qkv + src);
    if (which == 0 && c == 0)
      a.valid[static_cast<long long>(b) * a.max_seq + p] = a.S ? (a.mask[row] != 0) : 1;
  }
}

void launch_kv_store(const KvArgs& a, hipStream_t s) {
  const int vn = a.dtype == kF32 ? 4 : 8;
  const long long total = static_cast<long long>(a.rows) * 2 * (a.d / vn);
  long long blocks = (total + 255) / 256;
  blocks = blocks < 4096 ? blocks : 4096;
  hipLaunchKernelGGL(k_kv_store, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s, a, vn);
}

// ------------------------------------------------------------ attention
// Split-key decode attention.  Workgroup (b*H + h, split) covers keys
// [split*chunk, (split+1)*chunk) of sequence b up to its position pos[b]:
// G = hd/VN lanes hold one key row (16 bytes each), so a wavefront handles
// 64/G keys per step; each lane group keeps an online softmax (max m, sum l,
// unnormalised output o over its VN dimensions).  16 wavefronts, so that a
// cache of up to 512 keys (16-bit, head size 64) is one round trip of
// loads.  The groups of a wavefront are merged by shuffles, the wavefronts
// in LDS; with one chunk per head the workgroup normalises and writes the
// context, otherwise the chunk's (m, l, o) goes to the workspace and
// k_decode_combine merges the chunks.  (A last-workgroup-merges ticket would
// save that launch but needs a device-scope fence per workgroup, which on
// this GPU writes back the XCD's whole L2: far slower than the launch.)
// Keys marked invalid get weight 0; a sequence without a valid key gets a
// zero context.
template <typename T, int HD>
__global__ __launch_bounds__(1024) void k_decode_attn(DecAttnArgs a) {
  constexpr int NWV = 16;                      // wavefronts
  constexpr int VN = 16 / static_cast<int>(sizeof(T));
  constexpr int G = HD / VN;
  constexpr int KPW = 64 / G;
  constexpr int NG = NWV * KPW;                // lane groups in the workgroup
  typedef typename std::conditional<sizeof(T) == 4, f32x4v, u32x4>::type V;
  __shared__ float s_m[NWV], s_l[NWV];
  __shared__ float s_o[NWV][HD + 1];
  const int bh = blockIdx.x, split = blockIdx.y;
  const int b = bh / a.H, h = bh % a.H;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int grp = lane / G, gl = lane % G;
  const int k0 = split * a.chunk;
  const int last = a.pos[b];

  float q[VN];
  {
    const V raw = *reinterpret_cast<const V*>(static_cast<const T*>(a.qkv) +
                                              static_cast<long long>(b) * 3 * a.d + h * HD + gl * VN);
    const T* e = reinterpret_cast<const T*>(&raw);
#pragma unroll
    for (int i = 0; i < VN; ++i) q[i] = to_f32(e[i]);
  }
  const long long head = (static_cast<long long>(b) * a.H + h) * a.max_seq;
  const T* kc = static_cast<const T*>(a.kc) + head * HD + gl * VN;
  const T* vc = static_cast<const T*>(a.vc) + head * HD + gl * VN;
  const uint8_t* valid = a.valid + static_cast<long long>(b) * a.max_seq;
  float m = -INFINITY, l = 0.f, o[VN];
#pragma unroll
  for (int i = 0; i < VN; ++i) o[i] = 0.f;
  constexpr int U = 4;
  // U keys per lane group per trip, their K and V rows loaded up front so
  // that the loads of U keys are in flight together (16 wavefronts: 512
  // keys per trip at head size 64 in 16-bit).  The first trip's rows
  // are fetched before pos[b] (the end of the keys) is known: their
  // addresses do not depend on it (rows past the chunk read its first row,
  // inside the cache either way).
  const int cap = min(k0 + a.chunk, a.max_seq);
  const int jb = k0 + wave * KPW + grp;
  V kr[U], vr[U];
  uint8_t vl[U];
  auto fetch = [&](int j0) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + u * NG;
      const int jj = j < cap ? j : k0;
      kr[u] = *reinterpret_cast<const V*>(kc + static_cast<long long>(jj) * HD);
      vr[u] = *reinterpret_cast<const V*>(vc + static_cast<long long>(jj) * HD);
      vl[u] = valid[jj];
    }
  };
  fetch(jb);
  const int k1 = min(k0 + a.chunk, last + 1);
  for (int j0 = jb; j0 < k1; j0 += U * NG) {
    if (j0 != jb) fetch(j0);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const T* ke = reinterpret_cast<const T*>(&kr[u]);
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < VN; ++i) s += q[i] * to_f32(ke[i]);
#pragma unroll
      for (int off = G / 2; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
      if (!(j0 + u * NG < k1 && vl[u])) continue;   // the same for the whole lane group
      s *= a.scale;
      const float mn = fmaxf(m, s);
      const float corr = expf(m - mn), p = expf(s - mn);
      const T* ve = reinterpret_cast<const T*>(&vr[u]);
      l = l * corr + p;
#pragma unroll
      for (int i = 0; i < VN; ++i) o[i] = o[i] * corr + p * to_f32(ve[i]);
      m = mn;
    }
  }
  // merge the wavefront's lane groups (lanes G, 2G, .. apart hold the same
  // dimensions of other keys), then the wavefronts in LDS
#pragma unroll
  for (int off = G; off < 64; off <<= 1) {
    const float mo = __shfl_xor(m, off, 64), lo = __shfl_xor(l, off, 64);
    const float mm = fmaxf(m, mo);
    const float w0 = m == -INFINITY ? 0.f : expf(m - mm);
    const float w1 = mo == -INFINITY ? 0.f : expf(mo - mm);
    l = l * w0 + lo * w1;
#pragma unroll
    for (int i = 0; i < VN; ++i) o[i] = o[i] * w0 + __shfl_xor(o[i], off, 64) * w1;
    m = mm;
  }
  if (lane < G) {
    if (lane == 0) {
      s_m[wave] = m;
      s_l[wave] = l;
    }
#pragma unroll
    for (int i = 0; i < VN; ++i) s_o[wave][gl * VN + i] = o[i];
  }
  __syncthreads();
  float* part = a.part + ((static_cast<long long>(bh) * a.nsplit) + split) * (HD + 2);
  T* ctx = static_cast<T*>(a.ctx) + static_cast<long long>(b) * a.d + h * HD;
  for (int i = threadIdx.x; i < HD; i += blockDim.x) {
    float M = -INFINITY;
    for (int g2 = 0; g2 < NWV; ++g2) M = fmaxf(M, s_m[g2]);
    float L = 0.f, O = 0.f;
    if (M != -INFINITY)
      for (int g2 = 0; g2 < NWV; ++g2) {
        if (s_m[g2] == -INFINITY) continue;
        const float w = expf(s_m[g2] - M);
        L += s_l[g2] * w;
        O += s_o[g2][i] * w;
      }
    if (a.nsplit == 1) {                 // one chunk: normalise here
      ctx[i] = from_f32<T>(L > 0.f ? O / L : 0.f);
      continue;
    }
    part[2 + i] = O;
    if (i == 0) {
      part[0] = M;
      part[1] = L;
    }
  }
}

template <typename T, int HD>
__global__ __launch_bounds__(HD) void k_decode_combine(DecAttnArgs a) {
  const int bh = blockIdx.x, i = threadIdx.x;
  const float* part = a.part + static_cast<long long>(bh) * a.nsplit * (HD + 2);
  float M = -INFINITY;
  for (int sp = 0; sp < a.nsplit; ++sp) M = fmaxf(M, part[sp * (HD + 2)]);
  float L = 0.f, O = 0.f;
  if (M != -INFINITY)
    for (int sp = 0; sp < a.nsplit; ++sp) {
      const float ms = part[sp * (HD + 2)];
      if (ms == -INFINITY) continue;
      const float w = expf(ms - M);
      L += part[sp * (HD + 2) + 1] * w;
      O += part[sp * (HD + 2) + 2 + i] * w;
    }
  const int b = bh / a.H, h = bh % a.H;
  T* ctx = static_cast<T*>(a.ctx) + static_cast<long long>(b) * a.d + h * HD + i;
  *ctx = from_f32<T>(L > 0.f ? O / L : 0.f);
}

template <typename T, int HD>
static void decode_attn_t(const DecAttnArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((k_decode_attn<T, HD>), dim3(a.B * a.H, a.nsplit), dim3(1024), 0, s, a);
  if (a.nsplit > 1)
    hipLaunchKernelGGL((k_decode_combine<T, HD>), dim3(a.B * a.H), dim3(HD), 0, s, a);
}

template <typename T>
static void decode_attn_d(const DecAttnArgs& a, hipStream_t s) {
  if (a.hd == 32) decode_attn_t<T, 32>(a, s);
  else if (a.hd == 64) decode_attn_t<T, 64>(a, s);
  else decode_attn_t<T, 128>(a, s);
}

void launch_decode_attention(const DecAttnArgs& a, hipStream_t s) {
  if (a.dtype == kF32) decode_attn_d<float>(a, s);
  else if (a.dtype == kBF16) decode_attn_d<bf16_t>(a, s);
  else decode_attn_d<f16_t>(a, s);
}

// ------------------------------------------------------------ greedy argmax
template <typename T>
__global__ __launch_bounds__(1024) void k_argmax(const T* __restrict__ logits, int V,
                                                  int32_t* __restrict__ next) {
  __shared__ float s_v[16];
  __shared__ int s_i[16], s_n[16];
  const T* row = logits + static_cast<long long>(blockIdx.x) * V;
  float best = -INFINITY;
  int bi = 0x7FFFFFFF, ni = 0x7FFFFFFF;
  auto visit = [&](float v, int i) {
    if (v != v) ni = min(ni, i);
    else if (v > best || (v == best && i < bi)) {
      best = v;
      bi = i;
    }
  };
  // Rows of odd length start anywhere: scalar loads up to the first 16-byte
  // boundary, then 16-byte vectors (several in flight per thread), then the
  // scalar tail.  The visiting order does not matter: ties go to the
  // smaller index either way.
  constexpr int VN = 16 / static_cast<int>(sizeof(T));
  int head = static_cast<int>(((16 - (reinterpret_cast<uintptr_t>(row) & 15)) & 15) / sizeof(T));
  head = head < V ? head : V;
  for (int i = threadIdx.x; i < head; i += blockDim.x) visit(to_f32(row[i]), i);
  const int nvec = (V - head) / VN;
  const u32x4* vrow = reinterpret_cast<const u32x4*>(row + head);
#pragma unroll 4
  for (int j = threadIdx.x; j < nvec; j += blockDim.x) {
    const u32x4 raw = vrow[j];
    const T* e = reinterpret_cast<const T*>(&raw);
#pragma unroll
    for (int k = 0; k < VN; ++k) visit(to_f32(e[k]), head + j * VN + k);
  }
  for (int i = head + nvec * VN + threadIdx.x; i < V; i += blockDim.x) visit(to_f32(row[i]), i);
  for (int o = 32; o > 0; o >>= 1) {
    const float v2 = __shfl_xor(best, o, 64);
    const int i2 = __shfl_xor(bi, o, 64);
    if (v2 > best || (v2 == best && i2 < bi)) {
      best = v2;
      bi = i2;
    }
    ni = min(ni, __shfl_xor(ni, o, 64));
  }
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    s_v[w] = best;
    s_i[w] = bi;
    s_n[w] = ni;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int k = 1; k < static_cast<int>(blockDim.x >> 6); ++k) {
      if (s_v[k] > best || (s_v[k] == best && s_i[k] < bi)) {
        best = s_v[k];
        bi = s_i[k];
      }
      ni = min(ni, s_n[k]);
    }
    next[blockIdx.x] = ni != 0x7FFFFFFF ? ni : bi;
  }
}

void launch_argmax(const void* logits, int dtype, int B, int V, int32_t* next, hipStream_t s) {
  if (dtype == kF32)
    hipLaunchKernelGGL(k_argmax<float>, dim3(B), dim3(1024), 0, s, static_cast<const float*>(logits), V, next);
  else if (dtype == kBF16)
    hipLaunchKernelGGL(k_argmax<bf16_t>, dim3(B), dim3(1024), 0, s, static_cast<const bf16_t*>(logits), V, next);
  else
    hipLaunchKernelGGL(k_argmax<f16_t>, dim3(B), dim3(1024), 0, s, static_cast<const f16_t*>(logits), V, next);
}

// ------------------------------------------------------------ lengths
__global__ void k_seqlen(int32_t* __restrict__ seqlen, const int32_t* __restrict__ pos,
                         const int32_t* __restrict__ state, int B, int decode) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  if (!decode) seqlen[b] = state[kKvLenBase + b];
  else if (static_cast<uint32_t>(state[kTrapFwd]) == kTrapNone) seqlen[b] = pos[b] + 1;
}

void launch_seqlen_update(int32_t* seqlen, const int32_t* pos, const int32_t* state, int B,
                          int decode, hipStream_t s) {
  hipLaunchKernelGGL(k_seqlen, dim3((B + 255) / 256), dim3(256), 0, s, seqlen, pos, state, B, decode);
}

}  // namespace gm
