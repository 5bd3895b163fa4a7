// gm_attention.hip -- softmax(q k^T / sqrt(hd) + mask) v per (sequence, head).
//
// The key-padding mask is applied only when the device padding predicate
// (state[kPadAny], the `mask.any()` branch) is set: the branch becomes a
// flag read inside the kernel instead of a host decision.  Masked keys get
// weight exactly 0; a query with no visible key produces zeros.  With the
// flag set, key tiles at or past 1 + the last unmasked key of the sequence
// are skipped.  Causal models see keys j <= i.
//
// q, k and v are read in place from the fused projection output
// [B*S, 3d] (q | k | v, head h at columns h*hd); the context is written as
// [B*S, d] with head h at columns h*hd, the layout the output projection
// reads.
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
  const int S = a.S, hd = a.hd, ld = 3 * a.d;
  float* sq = sm;           // [hd]
  float* sp = sm + hd;      // [S]
  const T* base = static_cast<const T*>(a.qkv) + static_cast<long long>(b) * S * ld;
  const T* q = base + static_cast<long long>(i) * ld + h * hd;
  for (int c = lane; c < hd; c += 64) sq[c] = to_f32(q[c]);
  const int pad = a.state[kPadAny];
  int kend = pad ? a.state[kKvLenBase + b] : S;
  if (a.causal) kend = kend < i + 1 ? kend : i + 1;
  const int32_t* mk = a.mask + static_cast<long long>(b) * S;
  __syncthreads();
  float lmax = -INFINITY;
  for (int j = lane; j < kend; j += 64) {
    const bool ok = !pad || mk[j] != 0;
    float s = -INFINITY;
    if (ok) {
      const T* k = base + static_cast<long long>(j) * ld + a.d + h * hd;
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
  T* out = static_cast<T*>(a.ctx) + (static_cast<long long>(b) * S + i) * a.d + h * hd;
  for (int c = lane; c < hd; c += 64) {
    float o = 0.f;
    for (int j = 0; j < kend; ++j) {
      const float p = sp[j];
      if (p != 0.f) o = fmaf(p, to_f32(base[static_cast<long long>(j) * ld + 2 * a.d + h * hd + c]), o);
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

constexpr int kQB = 128, kKB = 64;

template <typename T, int HD>
__global__ __launch_bounds__(256) void k_attn_mfma(AttnArgs a) {
  typedef typename MfmaA<T>::vec vec;
  constexpr int LDK = HD + 8;      // K tile row pitch (elements)
  constexpr int LDV = kKB + 8;     // V^T tile row pitch
  constexpr int NC = HD / 32;      // 32-wide chunks of the head dim
  constexpr int NCT = HD / 16;     // 16-wide channel tiles
  __shared__ __attribute__((aligned(16))) T sK[kKB * LDK];
  __shared__ __attribute__((aligned(16))) T sVt[HD * LDV];
  __shared__ int sMask[kKB];
  const int qb = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int S = a.S, d = a.d, ld = 3 * d;
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  const int l16 = lane & 15, g = lane >> 4;
  const T* base = static_cast<const T*>(a.qkv) + static_cast<long long>(b) * S * ld;
  const int32_t* mk = a.mask + static_cast<long long>(b) * S;
  const int q0 = qb * kQB + wave * 32;

  vec qf[2][NC];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    int qi = q0 + 16 * u + l16;
    qi = qi < S ? qi : S - 1;
    const T* qp = base + static_cast<long long>(qi) * ld + h * HD;
#pragma unroll
    for (int c = 0; c < NC; ++c) qf[u][c] = *reinterpret_cast<const vec*>(qp + 32 * c + 8 * g);
  }
  const int pad = a.state[kPadAny];
  int kend = S;
  if (a.causal) kend = kend < (qb + 1) * kQB ? kend : (qb + 1) * kQB;
  if (pad) {
    const int kv = a.state[kKvLenBase + b];
    kend = kend < kv ? kend : kv;
  }
  const float sl2 = a.scale * 1.4426950408889634f;

  float mrow[2] = {-INFINITY, -INFINITY}, lrow[2] = {0.f, 0.f};
  f32x4 oacc[2][NCT];
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int c = 0; c < NCT; ++c) oacc[u][c] = f32x4{0.f, 0.f, 0.f, 0.f};

  constexpr int VPR = HD / 8;                 // 16-byte vectors per key row
  constexpr int LOADS = kKB * VPR / 256;      // per thread
  for (int kb = 0; kb < kend; kb += kKB) {
    // ---- stage K (row-major) and V (transposed) for keys kb..kb+63
#pragma unroll
    for (int v = 0; v < LOADS; ++v) {
      const int idx = t + 256 * v;
      const int r = idx / VPR, c = (idx % VPR) * 8;
      int key = kb + r;
      key = key < S ? key : S - 1;
      const T* kp = base + static_cast<long long>(key) * ld + d + h * HD + c;
      *reinterpret_cast<u32x4*>(&sK[r * LDK + c]) = *reinterpret_cast<const u32x4*>(kp);
      const u32x4 vv = *reinterpret_cast<const u32x4*>(kp + d);
      const T* ve = reinterpret_cast<const T*>(&vv);
#pragma unroll
      for (int e = 0; e < 8; ++e) sVt[(c + e) * LDV + r] = ve[e];
    }
    if (t < kKB) {
      const int key = kb + t;
      sMask[t] = key < S ? (pad ? mk[key] != 0 : 1) : 0;
    }
    __syncthreads();

    // ---- S^T = K Q^T
    f32x4 sacc[4][2];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int u = 0; u < 2; ++u) sacc[kt][u] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NC; ++c) {
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        const vec kf = *reinterpret_cast<const vec*>(&sK[(16 * kt + l16) * LDK + 32 * c + 8 * g]);
#pragma unroll
        for (int u = 0; u < 2; ++u) sacc[kt][u] = MfmaA<T>::run(kf, qf[u][c], sacc[kt][u]);
      }
    }
    // ---- masks and online softmax (per query = per (u, l16))
    float p[4][2][4];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int qi = q0 + 16 * u + l16;
      float tmax = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int kl = 16 * kt + 4 * g + r;
          const bool ok = sMask[kl] && (!a.causal || kb + kl <= qi);
          const float s = ok ? sacc[kt][u][r] * sl2 : -INFINITY;
          p[kt][u][r] = s;
          tmax = fmaxf(tmax, s);
        }
      tmax = fmaxf(tmax, __shfl_xor(tmax, 16, 64));
      tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
      const float mnew = fmaxf(mrow[u], tmax);
      const float alpha = mnew == -INFINITY ? 1.f : exp2f(mrow[u] - mnew);
      float tsum = 0.f;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float s = p[kt][u][r];
          const float e = s == -INFINITY ? 0.f : round_as<T>(exp2f(s - mnew));
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
      vec pb[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
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
        const T* vr = &sVt[(16 * c + l16) * LDV + 32 * kc + 4 * g];
        T tmp[8];
        *reinterpret_cast<u32x2*>(&tmp[0]) = *reinterpret_cast<const u32x2*>(vr);
        *reinterpret_cast<u32x2*>(&tmp[4]) = *reinterpret_cast<const u32x2*>(vr + 16);
        const vec vf = *reinterpret_cast<const vec*>(tmp);
#pragma unroll
        for (int u = 0; u < 2; ++u) oacc[u][c] = MfmaA<T>::run(vf, pb[u], oacc[u][c]);
      }
    }
    __syncthreads();
  }
  // ---- normalise and store: lane holds channels 16c + 4g + r of query (u, l16)
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int qi = q0 + 16 * u + l16;
    if (qi >= S) continue;
    const float inv = lrow[u] > 0.f ? 1.f / lrow[u] : 0.f;
    T* out = static_cast<T*>(a.ctx) + (static_cast<long long>(b) * S + qi) * d + h * HD;
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

static bool g_attn_rows = false;
void attention_force_rows(bool on) { g_attn_rows = on; }

void launch_attention(const AttnArgs& a, hipStream_t s) {
  const bool mfma_ok = a.dtype != kF32 && (a.hd == 64 || a.hd == 128) && !g_attn_rows;
  if (!mfma_ok) {
    const dim3 grid(a.S, a.H, a.B);
    const size_t lds = (a.hd + a.S) * sizeof(float);
    if (a.dtype == kF32) hipLaunchKernelGGL(k_attn_rows<float>, grid, dim3(64), lds, s, a);
    else if (a.dtype == kBF16) hipLaunchKernelGGL(k_attn_rows<bf16_t>, grid, dim3(64), lds, s, a);
    else hipLaunchKernelGGL(k_attn_rows<f16_t>, grid, dim3(64), lds, s, a);
    return;
  }
  const dim3 grid((a.S + kQB - 1) / kQB, a.H, a.B);
  if (a.dtype == kBF16) {
    if (a.hd == 64) hipLaunchKernelGGL((k_attn_mfma<bf16_t, 64>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((k_attn_mfma<bf16_t, 128>), grid, dim3(256), 0, s, a);
  } else {
    if (a.hd == 64) hipLaunchKernelGGL((k_attn_mfma<f16_t, 64>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((k_attn_mfma<f16_t, 128>), grid, dim3(256), 0, s, a);
  }
}

}  // namespace gm
