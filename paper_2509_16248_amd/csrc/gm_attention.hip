// gm_attention.hip -- softmax(q k^T / sqrt(hd) + mask) v per (sequence, head).
//
// The key-padding mask is applied only when the device padding predicate
// (state[kPadAny], the `mask.any()` branch) is set: the branch becomes a
// flag read inside the kernel instead of a host decision.  Masked keys get
// weight exactly 0; a query with no visible key produces zeros.  With the
// flag set, key tiles at or past 1 + the last unmasked key of the sequence
// are skipped.  Causal models see keys j <= i.
//
// q, k and v are read in place from row-major activations with given row
// strides: for self-attention all three from the fused projection output
// [B*S, 3d] (q | k | v, head h at columns h*hd); for cross-attention q from
// the decoder's [B*Sq, d] projection and k | v from [B*Sk, 2d] projected from
// the encoder output.  The context is written as [B*Sq, d] with head h at
// columns h*hd, the layout the output projection reads.
#include <math.h>

#include "gm_device.h"
#include "gm_kernels.h"

namespace gm {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------ reference kernel
// One wavefront per (query, head, sequence): scores in LDS, two passes for
// max and sum, then one output channel per lane.  Used for fp32 and for
// head dims the MFMA kernel does not cover.
template <typename T>
__global__ __launch_bounds__(64) void k_attn_rows(AttnArgs a) {
  extern __shared__ float sm[];
  const int i = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int lane = threadIdx.x;
  const int Sk = a.Sk, hd = a.hd;
  float* sq = sm;           // [hd]
  float* sp = sm + hd;      // [Sk]
  const T* q = static_cast<const T*>(a.q) + (static_cast<long long>(b) * a.Sq + i) * a.ldq + h * hd;
  const T* kb = static_cast<const T*>(a.k) + static_cast<long long>(b) * Sk * a.ldkv + h * hd;
  const T* vb = static_cast<const T*>(a.v) + static_cast<long long>(b) * Sk * a.ldkv + h * hd;
  for (int c = lane; c < hd; c += 64) sq[c] = to_f32(q[c]);
  const int pad = a.state[a.pad_slot];
  int kend = pad ? a.state[a.kvlen_base + b] : Sk;
  if (a.causal) kend = kend < i + 1 ? kend : i + 1;
  const int32_t* mk = a.mask + static_cast<long long>(b) * Sk;
  __syncthreads();
  float lmax = -INFINITY;
  for (int j = lane; j < kend; j += 64) {
    const bool ok = !pad || mk[j] != 0;
    float s = -INFINITY;
    if (ok) {
      const T* k = kb + static_cast<long long>(j) * a.ldkv;
      float acc = 0.f;
      for (int c = 0; c < hd; ++c) acc = fmaf(sq[c], to_f32(k[c]), acc);
      s = acc * a.scale;
      lmax = fmaxf(lmax, s);
    }
    sp[j] = s;
  }
  const float m = wave_max(lmax);
  float lsum = 0.f;
  for (int j = lane; j < kend; j += 64) {
    const float s = sp[j];
    const float p = s == -INFINITY ? 0.f : expf(s - m);
    sp[j] = p;
    lsum += p;
  }
  const float l = wave_sum(lsum);
  __syncthreads();
  T* out = static_cast<T*>(a.ctx) + (static_cast<long long>(b) * a.Sq + i) * a.d + h * hd;
  for (int c = lane; c < hd; c += 64) {
    float o = 0.f;
    for (int j = 0; j < kend; ++j) {
      const float p = sp[j];
      if (p != 0.f) o = fmaf(p, to_f32(vb[static_cast<long long>(j) * a.ldkv + c]), o);
    }
    out[c] = from_f32<T>(l > 0.f ? o / l : 0.f);
  }
}

// ------------------------------------------------------------ MFMA flash kernel
// Workgroup = 128 queries of one (sequence, head), 4 wavefronts x 32
// queries; key/value tiles of 64 keys staged in LDS (V transposed).
// Per tile each wavefront computes S^T = K Q^T with v_mfma_f32_16x16x32
// (K from LDS as the A operand, Q kept in registers as the B operand), so
// every lane holds 4 consecutive keys of one query; online softmax in fp32
// with exp2; then O^T += V^T P^T where the lane's probabilities are
// directly the B operand (the 8 keys of a lane group are
// {4g..4g+3, 16+4g..16+4g+3} of a 32-key chunk, and V^T is read from LDS
// in that same key order).  O^T tiles leave each lane with 4 consecutive
// channels of the same query whose softmax statistics it holds.
template <typename T> struct MfmaA;
template <> struct MfmaA<bf16_t> {
  typedef bf16x8 vec;
  static __device__ __forceinline__ f32x4 run(vec a, vec b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct MfmaA<f16_t> {
  typedef f16x8 vec;
  static __device__ __forceinline__ f32x4 run(vec a, vec b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
  }
};

constexpr int kKB = 64;

// K and V tiles move global -> registers -> LDS.  The tile after the current
// one is fetched into registers while the current one is multiplied, and the
// LDS tiles are double-buffered, so there is one barrier per key tile.  V is
// transposed on the way into LDS, two keys at a time (4-byte LDS writes).
// With a causal mask, query blocks run heaviest (last) first.  A wavefront
// holds 16 U queries (U = 1: 64 queries per workgroup).
template <typename T, int HD, int U, int ORD>
__global__ __launch_bounds__(256) void k_attn_mfma(AttnArgs a) {
  constexpr int QB = 64 * U;       // queries per workgroup: 4 wavefronts x 16U
  typedef typename MfmaA<T>::vec vec;
  constexpr int LDK = HD + 8;      // K tile row pitch (elements)
  constexpr int LDV = kKB + 4;     // V^T tile row pitch (transposing writes spread over banks)
  constexpr int NC = HD / 32;      // 32-wide chunks of the head dim
  constexpr int NCT = HD / 16;     // 16-wide channel tiles
  constexpr int VPR = HD / 8;      // 16-byte vectors per key row
  constexpr int KL = kKB * VPR / 256;          // K vectors per thread
  constexpr int VL = (kKB / 2) * VPR / 256;    // V key pairs per thread
  static_assert(KL >= 1 && VL >= 1, "tile too small for the workgroup");
  __shared__ __attribute__((aligned(16))) T sK[2][kKB * LDK];
  __shared__ __attribute__((aligned(16))) T sVt[2][HD * LDV];
  __shared__ int sMask[2][kKB];
  __shared__ int sFull[2];         // every key of the tile visible (no padding inside it)
  const int nqb = (a.Sq + QB - 1) / QB;
  int qb, h, b;
  if constexpr (ORD == 0) {
    qb = a.causal ? nqb - 1 - static_cast<int>(blockIdx.x) : static_cast<int>(blockIdx.x);
    h = blockIdx.y;
    b = blockIdx.z;
  } else {
    const int P = a.B * a.H;
    int p = blockIdx.x;
    if constexpr (ORD == 2) {
      constexpr int kSlot = 256;
      const int sl = p / kSlot;
      if ((sl & 1) && (sl + 1) * kSlot <= nqb * P) p = sl * kSlot + (kSlot - 1 - (p - sl * kSlot));
    }
    const int qi = p / P, pair = p - qi * P;
    qb = a.causal ? nqb - 1 - qi : qi;
    b = pair / a.H;
    h = pair - b * a.H;
  }
  const int Sq = a.Sq, S = a.Sk, d = a.d, ld = a.ldkv;
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  const int l16 = lane & 15, g = lane >> 4;
  const T* kbase = static_cast<const T*>(a.k) + static_cast<long long>(b) * S * ld + h * HD;
  const T* vbase = static_cast<const T*>(a.v) + static_cast<long long>(b) * S * ld + h * HD;
  const int32_t* mk = a.mask + static_cast<long long>(b) * S;
  const int q0 = qb * QB + wave * 16 * U;

  vec qf[U][NC];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    int qi = q0 + 16 * u + l16;
    qi = qi < Sq ? qi : Sq - 1;
    const T* qp = static_cast<const T*>(a.q) + (static_cast<long long>(b) * Sq + qi) * a.ldq + h * HD;
#pragma unroll
    for (int c = 0; c < NC; ++c) qf[u][c] = *reinterpret_cast<const vec*>(qp + 32 * c + 8 * g);
  }
  const int pad = a.state[a.pad_slot];
  int kend = S;
  if (a.causal) kend = kend < (qb + 1) * QB ? kend : (qb + 1) * QB;
  if (pad) {
    const int kv = a.state[a.kvlen_base + b];
    kend = kend < kv ? kend : kv;
  }
  const float sl2 = a.scale * 1.4426950408889634f;

  float mrow[U], lrow[U];
  f32x4 oacc[U][NCT];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    mrow[u] = -INFINITY;
    lrow[u] = 0.f;
  }
#pragma unroll
  for (int u = 0; u < U; ++u)
#pragma unroll
    for (int c = 0; c < NCT; ++c) oacc[u][c] = f32x4{0.f, 0.f, 0.f, 0.f};

  u32x4 rk[KL], rv[VL][2];
  int rm = 0;
  auto gload = [&](int kb) {
#pragma unroll
    for (int v = 0; v < KL; ++v) {
      const int idx = t + 256 * v;
      int key = kb + idx / VPR;
      key = key < S ? key : S - 1;
      rk[v] = *reinterpret_cast<const u32x4*>(kbase + static_cast<long long>(key) * ld + (idx % VPR) * 8);
    }
#pragma unroll
    for (int v = 0; v < VL; ++v) {
      const int idx = t + 256 * v;
      const int c = (idx % VPR) * 8;
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        int key = kb + 2 * (idx / VPR) + e;
        key = key < S ? key : S - 1;
        rv[v][e] = *reinterpret_cast<const u32x4*>(vbase + static_cast<long long>(key) * ld + c);
      }
    }
    if (t < kKB) {
      const int key = kb + t;
      rm = key < S ? (pad ? mk[key] != 0 : 1) : 0;
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int v = 0; v < KL; ++v) {
      const int idx = t + 256 * v;
      *reinterpret_cast<u32x4*>(&sK[buf][(idx / VPR) * LDK + (idx % VPR) * 8]) = rk[v];
    }
#pragma unroll
    for (int v = 0; v < VL; ++v) {
      const int idx = t + 256 * v;
      const int pr = idx / VPR, c = (idx % VPR) * 8;
      const T* v0 = reinterpret_cast<const T*>(&rv[v][0]);
      const T* v1 = reinterpret_cast<const T*>(&rv[v][1]);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        T pair[2] = {v0[e], v1[e]};
        *reinterpret_cast<uint32_t*>(&sVt[buf][(c + e) * LDV + 2 * pr]) =
            *reinterpret_cast<const uint32_t*>(pair);
      }
    }
    if (t < kKB) {                 // wavefront 0, all lanes
      sMask[buf][t] = rm;
      const unsigned long long all = __ballot(rm != 0);
      if (t == 0) sFull[buf] = all == ~0ull;
    }
  };

  if (kend > 0) gload(0);
  int it = 0;
  for (int kb = 0; kb < kend; kb += kKB, ++it) {
    const int buf = it & 1;
    sstore(buf);
    __syncthreads();
    if (kb + kKB < kend) gload(kb + kKB);

    // ---- S^T = K Q^T
    f32x4 sacc[4][U];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int u = 0; u < U; ++u) sacc[kt][u] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NC; ++c) {
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        const vec kf = *reinterpret_cast<const vec*>(&sK[buf][(16 * kt + l16) * LDK + 32 * c + 8 * g]);
#pragma unroll
        for (int u = 0; u < U; ++u) sacc[kt][u] = MfmaA<T>::run(kf, qf[u][c], sacc[kt][u]);
      }
    }
    // ---- masks and online softmax (per query = per (u, l16)).  A tile with
    // no padded key that lies wholly at or below this wavefront's first
    // query needs no mask (the same scores, without the per-key tests).
    const bool open = sFull[buf] && (!a.causal || kb + kKB - 1 <= q0);
    float p[4][U][4];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int qi = q0 + 16 * u + l16;
      float tmax = -INFINITY;
      if (open) {
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float s = sacc[kt][u][r] * sl2;
            p[kt][u][r] = s;
            tmax = fmaxf(tmax, s);
          }
      } else {
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int kl = 16 * kt + 4 * g + r;
            const bool ok = sMask[buf][kl] && (!a.causal || kb + kl <= qi);
            const float s = ok ? sacc[kt][u][r] * sl2 : -INFINITY;
            p[kt][u][r] = s;
            tmax = fmaxf(tmax, s);
          }
      }
      tmax = fmaxf(tmax, __shfl_xor(tmax, 16, 64));
      tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
      const float mnew = fmaxf(mrow[u], tmax);
      // while every key so far is masked, mnew is -inf: subtract 0 instead
      // (masked scores are -inf and give exp2 = 0 either way)
      const float msub = mnew == -INFINITY ? 0.f : mnew;
      const float alpha = __builtin_amdgcn_exp2f(mrow[u] - msub);
      float tsum = 0.f;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float e = round_as<T>(__builtin_amdgcn_exp2f(p[kt][u][r] - msub));
          p[kt][u][r] = e;
          tsum += e;
        }
      tsum += __shfl_xor(tsum, 16, 64);
      tsum += __shfl_xor(tsum, 32, 64);
      lrow[u] = lrow[u] * alpha + tsum;
      mrow[u] = mnew;
#pragma unroll
      for (int c = 0; c < NCT; ++c) oacc[u][c] *= alpha;
    }
    // ---- O^T += V^T P^T
#pragma unroll
    for (int kc = 0; kc < 2; ++kc) {
      vec pb[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        T tmp[8];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          tmp[r] = from_f32<T>(p[2 * kc][u][r]);
          tmp[4 + r] = from_f32<T>(p[2 * kc + 1][u][r]);
        }
        pb[u] = *reinterpret_cast<const vec*>(tmp);
      }
#pragma unroll
      for (int c = 0; c < NCT; ++c) {
        const T* vr = &sVt[buf][(16 * c + l16) * LDV + 32 * kc + 4 * g];
        T tmp[8];
        *reinterpret_cast<u32x2*>(&tmp[0]) = *reinterpret_cast<const u32x2*>(vr);
        *reinterpret_cast<u32x2*>(&tmp[4]) = *reinterpret_cast<const u32x2*>(vr + 16);
        const vec vf = *reinterpret_cast<const vec*>(tmp);
#pragma unroll
        for (int u = 0; u < U; ++u) oacc[u][c] = MfmaA<T>::run(vf, pb[u], oacc[u][c]);
      }
    }
  }
  // ---- normalise and store: lane holds channels 16c + 4g + r of query (u, l16)
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int qi = q0 + 16 * u + l16;
    if (qi >= Sq) continue;
    const float inv = lrow[u] > 0.f ? 1.f / lrow[u] : 0.f;
    T* out = static_cast<T*>(a.ctx) + (static_cast<long long>(b) * Sq + qi) * d + h * HD;
#pragma unroll
    for (int c = 0; c < NCT; ++c) {
      u32x2 r2;
      T* e = reinterpret_cast<T*>(&r2);
#pragma unroll
      for (int r = 0; r < 4; ++r) e[r] = from_f32<T>(oacc[u][c][r] * inv);
      *reinterpret_cast<u32x2*>(out + 16 * c + 4 * g) = r2;
    }
  }
}

static int g_attn_order = 2;
void attention_set_order(int o) { g_attn_order = o; }

template <int U, int ORD>
static void launch_attn_ord(const AttnArgs& a, dim3 grid, hipStream_t s) {
  if (a.dtype == kBF16) {
    if (a.hd == 64) hipLaunchKernelGGL((k_attn_mfma<bf16_t, 64, U, ORD>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((k_attn_mfma<bf16_t, 128, U, ORD>), grid, dim3(256), 0, s, a);
  } else {
    if (a.hd == 64) hipLaunchKernelGGL((k_attn_mfma<f16_t, 64, U, ORD>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((k_attn_mfma<f16_t, 128, U, ORD>), grid, dim3(256), 0, s, a);
  }
}

void launch_attention(const AttnArgs& a, hipStream_t s) {
  const bool mfma_ok = a.dtype != kF32 && (a.hd == 64 || a.hd == 128);
  if (!mfma_ok) {
    const dim3 grid(a.Sq, a.H, a.B);
    const size_t lds = (a.hd + a.Sk) * sizeof(float);
    if (a.dtype == kF32) hipLaunchKernelGGL(k_attn_rows<float>, grid, dim3(64), lds, s, a);
    else if (a.dtype == kBF16) hipLaunchKernelGGL(k_attn_rows<bf16_t>, grid, dim3(64), lds, s, a);
    else hipLaunchKernelGGL(k_attn_rows<f16_t>, grid, dim3(64), lds, s, a);
    return;
  }
  // 16 queries per wavefront: twice the workgroups and wavefronts of 32
  // (measured 9% faster at 8 x 12 heads x 512 causal), since each key tile
  // is a dependent chain (scores, masked online softmax, P.V) that needs
  // other wavefronts to hide its latency
  constexpr int U = 1;
  const int nqb = (a.Sq + 64 * U - 1) / (64 * U);
  if (g_attn_order == 0) {
    const dim3 grid(nqb, a.H, a.B);
    launch_attn_ord<U, 0>(a, grid, s);
  } else {
    const dim3 grid(nqb * a.H * a.B);
    if (g_attn_order == 1) launch_attn_ord<U, 1>(a, grid, s);
    else launch_attn_ord<U, 2>(a, grid, s);
  }
}

}  // namespace gm
