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

#include <type_traits>

#include "gm_device.h"
#include "gm_kernels.h"

namespace gm {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

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

// ------------------------------------------------------------ MFMA 32x32 flash kernel
// Workgroup = 128 queries of one (sequence, head): 4 wavefronts x 32
// queries, key/value tiles of 64 keys double-buffered in LDS (both
// row-major), one barrier per tile; with a causal mask the heaviest query
// blocks run first, and a wavefront skips the tiles wholly after its queries.  Per tile a wavefront computes
// S^T = K Q^T on v_mfma_f32_32x32x16 (K from LDS as the A operand, Q^T in
// registers as the B operand), so a lane holds 32 scores of ONE query (keys
// 8i + 4(lane/32) + r of each 32-key block); the row statistics are per
// lane plus one exchange with lane ^ 32.  O^T += V^T P^T takes the lane's own
// probabilities as the B operand (MFMA k slot 8(lane/32) + j stands for key
// 8(j/4) + 4(lane/32) + j%4 of a 16-key step, and the V^T operand is read in
// that key order by transposing LDS reads), and leaves each lane 4
// consecutive channels of its query.
//
// Online softmax with a lazily moved maximum: a tile whose scores exceed the
// running maximum by more than kTau (log2 units) for some query of the
// wavefront moves the maximum of every query of the wavefront and rescales
// the accumulators; otherwise the running maximum stays, and the
// probabilities of that tile are at most 2^kTau.  The result is the same
// quotient of sums (only the common factor differs); the rescale, 64
// multiplications per lane, is then skipped on most tiles.
template <typename T> struct Mfma32A;
template <> struct Mfma32A<bf16_t> {
  typedef bf16x8 vec;
  static __device__ __forceinline__ f32x16 run(vec a, vec b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct Mfma32A<f16_t> {
  typedef f16x8 vec;
  static __device__ __forceinline__ f32x16 run(vec a, vec b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
  }
};

constexpr float kTau = 8.0f;

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2v __attribute__((ext_vector_type(2)));

// Two floats rounded to T (nearest even) in one 32-bit word, lo first: one
// v_cvt_pk_bf16_f32 for bf16.
template <typename T> __device__ __forceinline__ uint32_t pack2(float lo, float hi);
template <> __device__ __forceinline__ uint32_t pack2<bf16_t>(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2v));
}
template <> __device__ __forceinline__ uint32_t pack2<f16_t>(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, f16x2v));
}

typedef __attribute__((address_space(3))) void* lds_vptr;
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// 16 bytes from global memory straight into LDS (global_load_lds_dwordx4):
// lane i of the wavefront writes bytes [16i, 16i + 16) from `lds`, which
// must be the same for every lane.
__device__ __forceinline__ void dma16(const void* g, void* lds) {
  __builtin_amdgcn_global_load_lds(g, (lds_vptr)lds, 16, 0, 0);
}

// ds_read_b64_tr_b16: in each group of 16 lanes, lane i receives element
// (i % 4) of the 4-element rows read by lanes i/4, 4 + i/4, 8 + i/4 and
// 12 + i/4 of its group, in that order.  Issued as inline assembly: the
// compiler would otherwise make this read wait for every LDS copy in
// flight (it cannot tell that they fill the other stage).  Its result is
// therefore invisible to the compiler's wait counting; lgkm_wait() below
// must precede any use.
template <int OFF>
__device__ __forceinline__ u32x2 lds_read_tr16(uint32_t addr) {
  u32x2 v;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "i"(OFF) : "memory");
  return v;
}

// Wait until at most N LDS reads are outstanding (LDS reads complete in
// issue order; no scalar memory read is in flight here), then tie the
// values to the wait so that no use moves above it.
template <int N>
__device__ __forceinline__ void lgkm_wait(u32x2* v, int n) {
  static_assert(N >= 0 && N < 16, "lgkmcnt range");
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"i"(N) : "memory");
  for (int i = 0; i < n; ++i) asm volatile("" : "+v"(v[i]));
}

__device__ __forceinline__ void wait_vmcnt0() {
  __builtin_amdgcn_s_waitcnt((0x7 << 4) | (0xF << 8));   // vmcnt(0), others untouched
}

// K and V tiles are copied global -> LDS without passing through registers,
// both row-major with 16-byte chunks XOR-swizzled per row: K so that the 16
// rows one phase of a 16-byte read touches fall in distinct banks, V so that
// the 4 rows x 4 chunks of a transposing read phase do.  V^T operands come
// from the transposing LDS read: lane 4e + q of a 16-lane group points at
// key e (of 4 consecutive keys) and channels 4q..4q+3 of the group's 16, so
// that every lane receives its own channel for the 4 keys.
template <typename T, int HD, int ORD>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2)))
void k_flash(AttnArgs a) {
  constexpr int QB = 128, KB = 64, NW = 4;
  typedef typename Mfma32A<T>::vec vec;
  constexpr int KS = HD / 16;                 // k steps of S^T (head dim)
  constexpr int CB = HD / 32;                 // 32-channel blocks of O^T
  constexpr int CPR = HD / 8;                 // 16-byte chunks per key row
  constexpr int RPL = 16 / CPR;               // key rows per 256 bytes
  constexpr int RPI = 64 / CPR;               // key rows per 1 KB copy instruction
  constexpr int LPW = KB / RPI / NW;          // copy instructions per wavefront, tile and operand
  constexpr int TILE = KB * HD;
  static_assert(LPW >= 1 && CPR >= 8, "tile shape");
  // one array per stage and operand: the copies into one stage and the
  // reads of the other are then known not to overlap, and the reads need
  // not wait for the copies in flight
  __shared__ __attribute__((aligned(1024))) T sK0[TILE];
  __shared__ __attribute__((aligned(1024))) T sK1[TILE];
  __shared__ __attribute__((aligned(1024))) T sV0[TILE];
  __shared__ __attribute__((aligned(1024))) T sV1[TILE];
  __shared__ unsigned long long sBits[2];     // key visible by the mask (bit per key)

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
  const int Sq = a.Sq, S = a.Sk, ld = a.ldkv;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int l32 = lane & 31, h2 = lane >> 5;
  const T* kbase = static_cast<const T*>(a.k) + static_cast<long long>(b) * S * ld + h * HD;
  const T* vbase = static_cast<const T*>(a.v) + static_cast<long long>(b) * S * ld + h * HD;
  const int32_t* mk = a.mask + static_cast<long long>(b) * S;
  const int qw0 = qb * QB + wave * 32;        // first query of this wavefront
  const int qi = qw0 + l32;                   // this lane's query

  vec qf[KS];
  {
    const int qc = qi < Sq ? qi : Sq - 1;
    const T* qp = static_cast<const T*>(a.q) + (static_cast<long long>(b) * Sq + qc) * a.ldq + h * HD;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[ks] = *reinterpret_cast<const vec*>(qp + 16 * ks + 8 * h2);
  }
  const int pad = a.state[a.pad_slot];
  int kend = S;
  if (a.causal) kend = kend < (qb + 1) * QB ? kend : (qb + 1) * QB;
  if (pad) {
    const int kv = a.state[a.kvlen_base + b];
    kend = kend < kv ? kend : kv;
  }
  const float c2 = a.scale * 1.4426950408889634f;   // scores to log2 units

  float mrun = -INFINITY, lrun = 0.f;
  f32x16 oacc[CB];
#pragma unroll
  for (int c = 0; c < CB; ++c)
#pragma unroll
    for (int i = 0; i < 16; ++i) oacc[c][i] = 0.f;

  // swizzles: chunk c of key row r sits at chunk position c ^ f(r)
  // copies: lane -> row (wave * LPW + j) * RPI + lane / CPR, position lane % CPR
  const int cr = lane / CPR, cpos = lane % CPR;
  int mraw = 1;                               // wavefront 0: mask word of key kb + lane of the tile in flight
  auto issue = [&](int kb, T* dk, T* dv) {
#pragma unroll
    for (int j = 0; j < LPW; ++j) {
      const int r = (wave * LPW + j) * RPI + cr;
      int key = kb + r;
      key = key < S ? key : S - 1;
      const long long go = static_cast<long long>(key) * ld;
      const int fk = (r / RPL) % CPR, fv = 4 * ((r / RPL) % (CPR / 4));
      dma16(kbase + go + 8 * (cpos ^ fk), dk + (wave * LPW + j) * RPI * HD);
      dma16(vbase + go + 8 * (cpos ^ fv), dv + (wave * LPW + j) * RPI * HD);
    }
    if (wave == 0 && pad) {
      const int key = kb + lane;
      mraw = mk[key < S ? key : S - 1];
    }
  };
  // K operand reads: row 32kk + l32, chunk 2ks + h2
  const int kswz = (l32 / RPL) % CPR;
  // V^T operand reads: lane 4e + q of group g reads key 16k2 + 8rr + 4(g/2) + e,
  // channels 32cb + 16(g%2) + 4q .. +3
  const int g = lane >> 4, e4 = (lane & 15) >> 2, q4 = lane & 3;
  const int vrow = 4 * (g >> 1) + e4;
  const int vswz4 = (vrow / RPL) % (CPR / 4);          // f(r) / 4, the same for every k2, rr
  const int vsub = 2 * (g & 1) + (q4 >> 1);            // chunk within the 4-chunk block
  const int vin = 4 * (q4 & 1);                        // element within the chunk
  uint32_t vaddr[CB];                                  // byte offsets within a stage, key step 0
#pragma unroll
  for (int c = 0; c < CB; ++c) vaddr[c] = 2 * (vrow * HD + 8 * (4 * (c ^ vswz4) + vsub) + vin);

  // one key tile from stage BUF (the other stage receives the next tile)
  auto tile = [&](auto BUF, int kb) {
    constexpr int buf = decltype(BUF)::value;
    T* sk = buf ? sK1 : sK0;
    T* sv = buf ? sV1 : sV0;
    if (wave == 0) {
      const int key = kb + lane;
      const unsigned long long bits = __ballot(key < S && mraw != 0);
      if (lane == 0) sBits[buf] = bits;
    }
    wait_vmcnt0();                              // this wavefront's copies of the tile landed
    __syncthreads();
    if (kb + KB < kend) issue(kb + KB, buf ? sK0 : sK1, buf ? sV0 : sV1);
    if (a.causal && kb > qw0 + 31) return;     // every key of the tile after this wavefront's queries
    // ---- S^T = K Q^T: two 32-key blocks
    f32x16 sacc[2];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int i = 0; i < 16; ++i) sacc[kk][i] = 0.f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        const vec kf = *reinterpret_cast<const vec*>(sk + (32 * kk + l32) * HD + 8 * ((2 * ks + h2) ^ kswz));
        sacc[kk] = Mfma32A<T>::run(kf, qf[ks], sacc[kk]);
      }
    }
    // ---- mask (padding bits; causal keys past the query) unless the tile
    // is wholly visible to every query of the wavefront
    const unsigned long long bits = sBits[buf];
    const bool open = bits == ~0ull && (!a.causal || kb + KB - 1 <= qw0);
    if (!open) {
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int kl = 32 * kk + 8 * (i >> 2) + 4 * h2 + (i & 3);
          const bool ok = ((bits >> kl) & 1ull) && (!a.causal || kb + kl <= qi);
          sacc[kk][i] = ok ? sacc[kk][i] : -INFINITY;
        }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sacc[kk][i]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float mt = mx * c2;
    if (__ballot(mt > mrun + kTau)) {          // move the maximum (wavefront-uniform)
      const float mnew = fmaxf(mrun, mt);
      const float alpha = mnew == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(mrun - mnew);
      lrun *= alpha;
#pragma unroll
      for (int c = 0; c < CB; ++c) oacc[c] *= alpha;
      mrun = mnew;
    }
    const float msub = mrun == -INFINITY ? 0.f : mrun;
    // ---- probabilities, their sum, and P^T as 16-bit B operands
    vec pb[4];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        u32x4 w;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float p0 = __builtin_amdgcn_exp2f(fmaf(sacc[kk][8 * hf + 2 * j], c2, -msub));
          const float p1 = __builtin_amdgcn_exp2f(fmaf(sacc[kk][8 * hf + 2 * j + 1], c2, -msub));
          lrun += p0 + p1;
          w[j] = pack2<T>(p0, p1);
        }
        pb[2 * kk + hf] = __builtin_bit_cast(vec, w);
      }
    }
    // ---- O^T += V^T P^T: four 16-key steps; the V^T operands of step
    // k2 + 1 are read while step k2 multiplies
    const uint32_t vb = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_vptr)sv));
    u32x2 vf[2][CB][2];
    auto vread = [&](auto K2, u32x2 (&dst)[CB][2]) {
      constexpr int k2 = decltype(K2)::value;
#pragma unroll
      for (int c = 0; c < CB; ++c) {
        dst[c][0] = lds_read_tr16<(16 * k2) * HD * 2>(vb + vaddr[c]);
        dst[c][1] = lds_read_tr16<(16 * k2 + 8) * HD * 2>(vb + vaddr[c]);
      }
    };
    auto vmul = [&](int k2, u32x2 (&src)[CB][2]) {
#pragma unroll
      for (int c = 0; c < CB; ++c) {
        u32x4 w;
        w[0] = src[c][0][0]; w[1] = src[c][0][1]; w[2] = src[c][1][0]; w[3] = src[c][1][1];
        oacc[c] = Mfma32A<T>::run(__builtin_bit_cast(vec, w), pb[k2], oacc[c]);
      }
    };
    vread(std::integral_constant<int, 0>(), vf[0]);
    vread(std::integral_constant<int, 1>(), vf[1]);
    lgkm_wait<2 * CB>(&vf[0][0][0], 2 * CB);
    vmul(0, vf[0]);
    vread(std::integral_constant<int, 2>(), vf[0]);
    lgkm_wait<2 * CB>(&vf[1][0][0], 2 * CB);
    vmul(1, vf[1]);
    vread(std::integral_constant<int, 3>(), vf[1]);
    lgkm_wait<2 * CB>(&vf[0][0][0], 2 * CB);
    vmul(2, vf[0]);
    lgkm_wait<0>(&vf[1][0][0], 2 * CB);
    vmul(3, vf[1]);
  };
  if (kend > 0) issue(0, sK0, sV0);
  for (int kb = 0; kb < kend; kb += 2 * KB) {
    tile(std::integral_constant<int, 0>(), kb);
    if (kb + KB < kend) tile(std::integral_constant<int, 1>(), kb + KB);
  }
  // ---- normalise and store: lane holds channels 32c + 8i + 4(lane/32) + r of its query
  const float L = lrun + __shfl_xor(lrun, 32, 64);
  if (qi >= Sq) return;
  const float inv = L > 0.f ? 1.f / L : 0.f;
  T* out = static_cast<T*>(a.ctx) + (static_cast<long long>(b) * Sq + qi) * a.d + h * HD;
#pragma unroll
  for (int c = 0; c < CB; ++c)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      u32x2 r2;
      r2[0] = pack2<T>(oacc[c][4 * i] * inv, oacc[c][4 * i + 1] * inv);
      r2[1] = pack2<T>(oacc[c][4 * i + 2] * inv, oacc[c][4 * i + 3] * inv);
      *reinterpret_cast<u32x2*>(out + 32 * c + 8 * i + 4 * h2) = r2;
    }
}

static int g_attn_order = 2;
void attention_set_order(int o) { g_attn_order = o; }

template <int ORD>
static void launch_flash_ord(const AttnArgs& a, dim3 grid, hipStream_t s) {
  if (a.dtype == kBF16) {
    if (a.hd == 64) hipLaunchKernelGGL((k_flash<bf16_t, 64, ORD>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((k_flash<bf16_t, 128, ORD>), grid, dim3(256), 0, s, a);
  } else {
    if (a.hd == 64) hipLaunchKernelGGL((k_flash<f16_t, 64, ORD>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((k_flash<f16_t, 128, ORD>), grid, dim3(256), 0, s, a);
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
  // 128 queries (4 wavefronts x 32) per workgroup
  const int nqb = (a.Sq + 127) / 128;
  if (g_attn_order == 0) {
    launch_flash_ord<0>(a, dim3(nqb, a.H, a.B), s);
  } else {
    const dim3 grid(nqb * a.H * a.B);
    if (g_attn_order == 1) launch_flash_ord<1>(a, grid, s);
    else launch_flash_ord<2>(a, grid, s);
  }
}

}  // namespace gm
