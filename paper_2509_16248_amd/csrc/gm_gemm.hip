// gm_gemm.hip -- out = epilogue(A . W^T) for the projections and the head.
//
// A is [M, K] (activations, row-major), W is [N, K] (nn.Linear weight
// layout, row-major): both operands are contiguous along K, which is the
// operand layout the matrix cores read.  bf16/fp16 run on gfx950 MFMA
// (v_mfma_f32_32x32x16_{bf16,f16}) with fp32 accumulation; fp32 runs on a
// plain LDS-tiled FMA kernel.  All epilogues work on fp32 accumulators and
// round once to the storage dtype.
#include <math.h>

#include <type_traits>

#include "gm_device.h"
#include "gm_kernels.h"

namespace gm {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// ------------------------------------------------------------ epilogue
template <typename T>
__device__ __forceinline__ void load4(const T* p, float* v, int nvalid, bool vec) {
  if (vec) {
    if constexpr (sizeof(T) == 4) {
      const f32x4v r = *reinterpret_cast<const f32x4v*>(p);
      v[0] = r[0]; v[1] = r[1]; v[2] = r[2]; v[3] = r[3];
    } else {
      const u32x2 r = *reinterpret_cast<const u32x2*>(p);
      const T* e = reinterpret_cast<const T*>(&r);
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = to_f32(e[i]);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = i < nvalid ? to_f32(p[i]) : 0.f;
  }
}

template <typename T>
__device__ __forceinline__ void store4(T* p, const float* v, int nvalid, bool vec) {
  if (vec) {
    if constexpr (sizeof(T) == 4) {
      *reinterpret_cast<f32x4v*>(p) = f32x4v{v[0], v[1], v[2], v[3]};
    } else {
      u32x2 r;
      T* e = reinterpret_cast<T*>(&r);
#pragma unroll
      for (int i = 0; i < 4; ++i) e[i] = from_f32<T>(v[i]);
      *reinterpret_cast<u32x2*>(p) = r;
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (i < nvalid) p[i] = from_f32<T>(v[i]);
  }
}

__device__ __forceinline__ float gelu_f(float x) {
  return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f));
}
// x * sigmoid(x) from the hardware exponential and reciprocal (v_exp_f32,
// v_rcp_f32, about 1 ulp each): x -> -inf gives 1/inf = 0, x -> +inf gives x
__device__ __forceinline__ float silu_f(float x) {
  return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(x * -1.4426950408889634f));
}

struct SiteMax {
  uint32_t amax = 0;
  int nan = 0;
  __device__ __forceinline__ void add(float y) {
    if (y != y) nan = 1;
    else {
      const uint32_t u = __float_as_uint(y) & 0x7FFFFFFFu;
      amax = u > amax ? u : amax;
    }
  }
};

// Decode step: four consecutive output columns n..n+3 of row b in the k
// (region 1) or v (region 2) block of q|k|v also go to the KV cache.
template <typename T>
__device__ __forceinline__ void cache4(const GemmArgs& a, int b, int n, const float* v) {
  const int d = a.d_model, region = n / d;
  if (region < 1 || region > 2) return;
  if (static_cast<uint32_t>(a.state[kTrapFwd]) != kTrapNone) return;
  const int c = n - region * d, h = c / a.head_dim, i = c - h * a.head_dim;
  const int p = a.pos[b];
  T* dst = static_cast<T*>(region == 1 ? a.kc : a.vc) +
           ((static_cast<long long>(b) * a.heads + h) * a.kv_max_seq + p) * a.head_dim + i;
  store4(dst, v, 4, true);
  if (region == 1 && c == 0) a.kv_valid[static_cast<long long>(b) * a.kv_max_seq + p] = 1;
}

// Four consecutive packed columns nA..nA+3 (first tile of a pair, values
// va) and nA+16..nA+19 (second tile, values vb) of output row m.
template <typename T>
__device__ __forceinline__ void epi_pair(const GemmArgs& a, int m, int nA,
                                         const float* va, const float* vb,
                                         SiteMax& sm) {
  if (m >= a.M) return;
  const T* bias = static_cast<const T*>(a.bias);
  T* out = static_cast<T*>(a.out);
  const long long orow = static_cast<long long>(m) * a.ldo;
  if (a.epi == kEpiGatedGelu || a.epi == kEpiGatedSilu) {
    const int jo = (nA >> 5) * 16 + (nA & 15);
    float y[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float g = va[r], u = vb[r];
      if (bias) {
        g += to_f32(bias[nA + r]);
        u += to_f32(bias[nA + 16 + r]);
      }
      const float act = a.epi == kEpiGatedGelu ? gelu_f(g) : silu_f(g);
      y[r] = act * u;
    }
    store4(out + orow + jo, y, 4, (a.ldo & 3) == 0);
    return;
  }
  if (a.epi == kEpiRope && nA < 2 * a.d_model) {
    const int d = a.d_model, hd = a.head_dim, P = hd >> 1;
    const int region = nA >= d;
    const int nr = nA - region * d;
    const int h = nr / hd, within = nr - h * hd;
    const int i = (within >> 5) * 16 + (within & 15);
    int pos = a.pos ? a.pos[m] : m % a.seq;
    pos = pos < a.rope_rows ? pos : a.rope_rows - 1;
    // [Where]: both frequency sets exist; the forward's flag selects one
    const long long set = a.rope_set_stride && a.state[kRopeLong] ? a.rope_set_stride : 0;
    const float* cs = a.rope_cos + set + static_cast<long long>(pos) * P + i;
    const float* sn = a.rope_sin + set + static_cast<long long>(pos) * P + i;
    float o1[4], o2[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float x1 = va[r], x2 = vb[r];
      if (bias) {
        x1 += to_f32(bias[nA + r]);
        x2 += to_f32(bias[nA + 16 + r]);
      }
      o1[r] = x1 * cs[r] - x2 * sn[r];
      o2[r] = x2 * cs[r] + x1 * sn[r];
    }
    const long long base = orow + region * d + h * hd + i;
    const bool vec = (a.ldo & 3) == 0;
    store4(out + base, o1, 4, vec);
    store4(out + base + P, o2, 4, vec);
    if (a.kc && region == 1) {
      cache4<T>(a, m, d + h * hd + i, o1);
      cache4<T>(a, m, d + h * hd + i + P, o2);
    }
    return;
  }
  // independent columns: store / gelu / residual (and v of kEpiRope)
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int n0 = nA + 16 * t;
    if (n0 >= a.N) continue;
    const float* v = t ? vb : va;
    const int nvalid = a.N - n0 < 4 ? a.N - n0 : 4;
    const bool vec = nvalid == 4 && (a.ldo & 3) == 0;
    float y[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) y[r] = v[r];
    if (bias)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (r < nvalid) y[r] += to_f32(bias[n0 + r]);
    if (a.epi == kEpiGelu)
#pragma unroll
      for (int r = 0; r < 4; ++r) y[r] = gelu_f(y[r]);
    if (a.epi == kEpiResid) {
      float rv[4];
      load4(static_cast<const T*>(a.resid) + static_cast<long long>(m) * a.ldr + n0, rv,
            nvalid, nvalid == 4 && (a.ldr & 3) == 0);
#pragma unroll
      for (int r = 0; r < 4; ++r) y[r] += rv[r];
      if (a.site >= 0)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (r < nvalid) sm.add(round_as<T>(y[r]));
    }
    store4(out + orow + n0, y, nvalid, vec);
    if (a.kc) cache4<T>(a, m, n0, y);
  }
}

__device__ __forceinline__ void site_flush(const GemmArgs& a, SiteMax& sm) {
  if (a.site < 0) return;
  const uint32_t m = wave_max_u32(sm.amax);
  const int n = wave_or(sm.nan);
  if ((threadIdx.x & 63) == 0) {
    if (m) atomicMax(reinterpret_cast<unsigned int*>(a.state + kAbsmaxBase + a.site), m);
    if (n) atomicOr(a.state + kNanBase + a.site, 1);
  }
}

// ------------------------------------------------------------ MFMA 32x32 kernel
constexpr int kBK = 64, kLDK = kBK + 8;   // K step; padded LDS row (elements)

// Workgroup tile BM x BN, K step 64, WGM x WGN wavefronts; each wavefront
// owns (BM/WGM) x (BN/WGN) as TM x TN tiles of v_mfma_f32_32x32x16 (bf16/f16
// in, fp32 accumulate).  W is the MFMA A
// operand and the activations the B operand: a lane ends up with the output
// columns n = 32j + 8q + 4(lane/32) + r (q, r = 0..3) of row
// m = 32i + lane%32, so the columns of a 16-row weight group (q = 0, 1) and
// of its partner group (q + 2) sit in the same lane, which is what the
// gated and rotary epilogues pair.
// Both operand tiles are staged in LDS (row pitch padded by 16 bytes so the
// 32 rows a wavefront reads at once fall in distinct banks), two stages;
// the next K step's tiles are fetched into registers while the current one
// is multiplied.  Tiles are visited XCD by XCD and, within an XCD, in
// groups of GM tile-rows, so that concurrently running workgroups share
// operand tiles in the same L2.
template <int I, int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<I + 1, N>(f);
  }
}

template <typename T> struct Mfma32;
template <> struct Mfma32<bf16_t> {
  typedef bf16x8 vec;
  static __device__ __forceinline__ f32x16 run(vec a, vec b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct Mfma32<f16_t> {
  typedef f16x8 vec;
  static __device__ __forceinline__ f32x16 run(vec a, vec b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
  }
};

__device__ __forceinline__ void tile_of(int bid, int tiles_m, int tiles_n, int& tm, int& tn) {
  // XCD-major renumbering: hardware deals workgroups round-robin to the 8
  // XCDs, so workgroup b runs on XCD b % 8.  Give each XCD a contiguous
  // range of tile ids.
  const int total = tiles_m * tiles_n;
  int t = bid;
  if (total % 8 == 0) t = (bid % 8) * (total / 8) + bid / 8;
  // grouped order: GM tile-rows sweep the columns together
  constexpr int GM = 8;
  const int group = t / (GM * tiles_n);
  const int first = group * GM;
  const int rows = tiles_m - first < GM ? tiles_m - first : GM;
  const int in = t - group * GM * tiles_n;
  tm = first + in % rows;
  tn = in / rows;
}

// Epilogue of one BM x BN output tile held as 32x32 MFMA accumulators:
// wavefront (wm, wn) owns rows wm*WTM.. and columns wn*WTN.. as TM x TN
// tiles; lane l holds columns 32j + 8q + 4(l/32) + r of row 32i + l%32.
// Column-independent epilogues (store, GELU, residual) finish in registers
// (bias, then GELU or the residual, one rounding to the output type, the
// site statistics of the rounded values) and, when STAGE (the tile fits in
// smem in the output type), leave through LDS with consecutive lanes on
// consecutive columns: 16-byte chunks when output rows are 16-byte aligned,
// single elements otherwise (the odd vocabulary of the head).  The gated and
// rotary epilogues combine column groups 16 apart in registers (epi_pair).
template <typename T, int BM, int BN, int WGM, int WGN, bool STAGE>
__device__ __forceinline__ void tile_epilogue(const GemmArgs& a,
                                              f32x16 (&acc)[BM / WGM / 32][BN / WGN / 32],
                                              char* smem, int bm, int bn) {
  constexpr int NT = 64 * WGM * WGN;
  constexpr int WTM = BM / WGM, WTN = BN / WGN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  const int wm = wave / WGN, wn = wave % WGN;
  const int l32 = lane & 31, g = lane >> 5;
  __syncthreads();   // every wavefront is done reading operand tiles from smem
  SiteMax sm;
  const bool gated = a.epi == kEpiGatedGelu || a.epi == kEpiGatedSilu;
  // rotary pairs stay inside the tile when whole heads do
  const bool rope = a.epi == kEpiRope && BN % a.head_dim == 0;
  const bool plain = a.epi == kEpiStore || a.epi == kEpiGelu || a.epi == kEpiResid;
  if (STAGE && !a.kc && (plain || gated || rope)) {
    // The tile finishes in registers (bias, then GELU, the residual, the
    // gate product or the rotation; one rounding to the output type; the
    // site statistics of the rounded values), is staged in LDS in the
    // output type at its output columns (a gated tile is BN/2 wide; rotated
    // q/k columns go back to their head positions, which stay inside the
    // tile), and rows leave with consecutive lanes on consecutive columns:
    // 16-byte chunks when output rows are 16-byte aligned, single elements
    // otherwise (the odd vocabulary of the head).
    constexpr int LDB = BN + 8;
    T* stb = reinterpret_cast<T*>(smem);
    const T* bias = static_cast<const T*>(a.bias);
    const bool bias8 = (reinterpret_cast<uintptr_t>(bias) & 7) == 0;
    T* out = static_cast<T*>(a.out);
    const bool resid = a.epi == kEpiResid;
    const T* res = static_cast<const T*>(a.resid);
    const bool res8 = resid && (a.ldr & 3) == 0 && (reinterpret_cast<uintptr_t>(res) & 7) == 0;
    auto stage4 = [&](int ml, int col, const float* v) {
      u32x2 w;
      T* we = reinterpret_cast<T*>(&w);
#pragma unroll
      for (int r = 0; r < 4; ++r) we[r] = from_f32<T>(v[r]);
      *reinterpret_cast<u32x2*>(&stb[ml * LDB + col]) = w;
    };
    if (gated) {
      static_for<0, TM>([&](auto i) {
        const int ml = wm * WTM + 32 * i + l32;
        static_for<0, TN>([&](auto j) {
          static_for<0, 2>([&](auto q) {
            const int nl = wn * WTN + 32 * j + 8 * q + 4 * g;
            const int nA = bn + nl;
            float y[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              float gv = acc[i][j][4 * q + r], u = acc[i][j][4 * (q + 2) + r];
              if (bias && nA + 16 + r < a.N) {
                gv += to_f32(bias[nA + r]);
                u += to_f32(bias[nA + 16 + r]);
              }
              const float act = a.epi == kEpiGatedGelu ? gelu_f(gv) : silu_f(gv);
              y[r] = act * u;
            }
            stage4(ml, (nl >> 5) * 16 + (nl & 15), y);
          });
        });
      });
    } else if (rope) {
      const int d = a.d_model, hd = a.head_dim, P = hd >> 1;
      const long long set = a.rope_set_stride && a.state[kRopeLong] ? a.rope_set_stride : 0;
      static_for<0, TM>([&](auto i) {
        const int ml = wm * WTM + 32 * i + l32;
        const int m = bm + ml;
        int pos = m < a.M ? (a.pos ? a.pos[m] : m % a.seq) : 0;
        pos = pos < a.rope_rows ? pos : a.rope_rows - 1;
        static_for<0, TN>([&](auto j) {
          static_for<0, 2>([&](auto q) {
            const int nl = wn * WTN + 32 * j + 8 * q + 4 * g;
            const int nA = bn + nl;
            float x1[4], x2[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              x1[r] = acc[i][j][4 * q + r];
              x2[r] = acc[i][j][4 * (q + 2) + r];
              if (bias && nA + 16 + r < a.N) {
                x1[r] += to_f32(bias[nA + r]);
                x2[r] += to_f32(bias[nA + 16 + r]);
              }
            }
            if (nA < 2 * d) {
              const int region = nA >= d;
              const int nr = nA - region * d;
              const int h = nr / hd, within = nr - h * hd;
              const int ii = (within >> 5) * 16 + (within & 15);
              const float* cs = a.rope_cos + set + static_cast<long long>(pos) * P + ii;
              const float* sn = a.rope_sin + set + static_cast<long long>(pos) * P + ii;
              float o1[4], o2[4];
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                o1[r] = x1[r] * cs[r] - x2[r] * sn[r];
                o2[r] = x2[r] * cs[r] + x1[r] * sn[r];
              }
              const int col = region * d + h * hd + ii - bn;
              stage4(ml, col, o1);
              stage4(ml, col + P, o2);
            } else {
              stage4(ml, nl, x1);
              stage4(ml, nl + 16, x2);
            }
          });
        });
      });
    } else {
      static_for<0, TM>([&](auto i) {
        const int ml = wm * WTM + 32 * i + l32;
        const int m = bm + ml;
        static_for<0, TN>([&](auto j) {
          static_for<0, 4>([&](auto q) {
            const int nl = wn * WTN + 32 * j + 8 * q + 4 * g;
            const int n0 = bn + nl;
            float v[4];
  #pragma unroll
            for (int r = 0; r < 4; ++r) v[r] = acc[i][j][4 * q + r];
            if (bias) {
              if (bias8 && n0 + 4 <= a.N) {
                const u32x2 bb = *reinterpret_cast<const u32x2*>(bias + n0);
                const T* be = reinterpret_cast<const T*>(&bb);
  #pragma unroll
                for (int r = 0; r < 4; ++r) v[r] += to_f32(be[r]);
              } else {
  #pragma unroll
                for (int r = 0; r < 4; ++r)
                  if (n0 + r < a.N) v[r] += to_f32(bias[n0 + r]);
              }
            }
            if (a.epi == kEpiGelu)
  #pragma unroll
              for (int r = 0; r < 4; ++r) v[r] = gelu_f(v[r]);
            if (resid && m < a.M) {
              const T* rrow = res + static_cast<long long>(m) * a.ldr + n0;
              if (res8 && n0 + 4 <= a.N) {
                const u32x2 rr = *reinterpret_cast<const u32x2*>(rrow);
                const T* re = reinterpret_cast<const T*>(&rr);
  #pragma unroll
                for (int r = 0; r < 4; ++r) v[r] += to_f32(re[r]);
              } else {
  #pragma unroll
                for (int r = 0; r < 4; ++r)
                  if (n0 + r < a.N) v[r] += to_f32(rrow[r]);
              }
            }
            u32x2 w;
            T* we = reinterpret_cast<T*>(&w);
  #pragma unroll
            for (int r = 0; r < 4; ++r) we[r] = from_f32<T>(v[r]);
            if (resid && a.site >= 0 && m < a.M)
  #pragma unroll
              for (int r = 0; r < 4; ++r)
                if (n0 + r < a.N) sm.add(to_f32(we[r]));
            *reinterpret_cast<u32x2*>(&stb[ml * LDB + nl]) = w;
          });
        });
      });
    }
    __syncthreads();
    // output tile: OW columns from column ob of rows of a.ldo elements
    const int OW = gated ? BN / 2 : BN;
    const int ob = gated ? bn / 2 : bn;
    const int nout = gated ? a.N / 2 : a.N;
    const int ncol = nout - ob < OW ? nout - ob : OW;
    if ((a.ldo & 7) == 0) {
      const int cpr = OW / 8;
      for (int e = t; e < BM * cpr; e += NT) {
        const int ml = e / cpr, j0 = 8 * (e % cpr);
        const int m = bm + ml;
        if (m >= a.M || j0 >= ncol) continue;
        const u32x4 w = *reinterpret_cast<const u32x4*>(&stb[ml * LDB + j0]);
        T* orow = out + static_cast<long long>(m) * a.ldo + ob;
        if (j0 + 8 <= ncol) {
          *reinterpret_cast<u32x4*>(orow + j0) = w;
        } else {
          const T* we = reinterpret_cast<const T*>(&w);
#pragma unroll
          for (int r = 0; r < 8; ++r)
            if (j0 + r < ncol) orow[j0 + r] = we[r];
        }
      }
    } else {
      for (int e = t; e < BM * OW; e += NT) {
        const int ml = e / OW, nl = e % OW;
        const int m = bm + ml;
        if (m >= a.M || nl >= ncol) continue;
        out[static_cast<long long>(m) * a.ldo + ob + nl] = stb[ml * LDB + nl];
      }
    }
  } else {
    static_for<0, TM>([&](auto i) {
      const int m = bm + wm * WTM + 32 * i + l32;
      static_for<0, TN>([&](auto j) {
        static_for<0, 2>([&](auto q) {
          const int nA = bn + wn * WTN + 32 * j + 8 * q + 4 * g;
          float va[4], vb[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            va[r] = acc[i][j][4 * q + r];
            vb[r] = acc[i][j][4 * (q + 2) + r];
          }
          epi_pair<T>(a, m, nA, va, vb, sm);
        });
      });
    });
  }
  site_flush(a, sm);
}

template <typename T, int BM, int BN, int WGM, int WGN, int PF>
__global__ __launch_bounds__(64 * WGM * WGN) void k_gemm_x(GemmArgs a) {
  typedef typename Mfma32<T>::vec vec;
  constexpr int NT = 64 * WGM * WGN;            // threads
  constexpr int WTM = BM / WGM, WTN = BN / WGN; // wavefront tile
  constexpr int TM = WTM / 32, TN = WTN / 32;   // 32x32 MFMA tiles per wavefront
  constexpr int RPP = NT / 8;                   // tile rows loaded per pass
  constexpr int VA = BM / RPP, VB = BN / RPP;   // 16-byte loads per thread per stage
  constexpr int KS = kBK / 16;                  // MFMA k-steps per stage
  static_assert(BM % RPP == 0 && BN % RPP == 0, "tile rows must split evenly");
  static_assert(TM >= 1 && TN >= 1, "wavefront tile below 32x32");
  constexpr int LDS_OPS = 2 * (BM + BN) * kLDK * static_cast<int>(sizeof(T));
  constexpr bool STAGE = BM * (BN + 8) * static_cast<int>(sizeof(T)) <= LDS_OPS;  // output-type staging tile
  __shared__ __attribute__((aligned(16))) char smem[LDS_OPS];
  T (*sA)[BM * kLDK] = reinterpret_cast<T (*)[BM * kLDK]>(smem);
  T (*sB)[BN * kLDK] = reinterpret_cast<T (*)[BN * kLDK]>(smem + 2 * BM * kLDK * sizeof(T));
  const int tiles_m = (a.M + BM - 1) / BM, tiles_n = (a.N + BN - 1) / BN;
  int tm, tn;
  tile_of(blockIdx.x, tiles_m, tiles_n, tm, tn);
  const int bm = tm * BM, bn = tn * BN;
  const int t = threadIdx.x;
  const int lrow = t >> 3, lcol = (t & 7) * 8;
  // element offsets of this thread's rows (rows past the end are clamped to
  // the last row: loaded, never stored)
  uint32_t oa[VA], ob[VB];
#pragma unroll
  for (int v = 0; v < VA; ++v) {
    int r = bm + lrow + RPP * v;
    r = r < a.M ? r : a.M - 1;
    oa[v] = static_cast<uint32_t>(r) * a.lda + lcol;
  }
#pragma unroll
  for (int v = 0; v < VB; ++v) {
    int c = bn + lrow + RPP * v;
    c = c < a.N ? c : a.N - 1;
    ob[v] = static_cast<uint32_t>(c) * a.ldw + lcol;
  }
  const T* __restrict__ A0 = static_cast<const T*>(a.A);
  const T* __restrict__ W0 = static_cast<const T*>(a.W);
  const int wave = t >> 6, lane = t & 63;
  const int wm = wave / WGN, wn = wave % WGN;
  const int l32 = lane & 31, g = lane >> 5;
  const int rdA = (wm * WTM + l32) * kLDK + 8 * g;
  const int rdB = (wn * WTN + l32) * kLDK + 8 * g;
  const int wr = lrow * kLDK + lcol;

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  u32x4 ra[PF][VA], rb[PF][VB];
  const int nk = a.K / kBK;
  auto gload = [&](auto set, int k0) {
#pragma unroll
    for (int v = 0; v < VA; ++v) ra[set][v] = *reinterpret_cast<const u32x4*>(A0 + oa[v] + k0);
#pragma unroll
    for (int v = 0; v < VB; ++v) rb[set][v] = *reinterpret_cast<const u32x4*>(W0 + ob[v] + k0);
  };
  auto sstore = [&](auto set, int buf) {
#pragma unroll
    for (int v = 0; v < VA; ++v)
      *reinterpret_cast<u32x4*>(&sA[buf][wr + RPP * v * kLDK]) = ra[set][v];
#pragma unroll
    for (int v = 0; v < VB; ++v)
      *reinterpret_cast<u32x4*>(&sB[buf][wr + RPP * v * kLDK]) = rb[set][v];
  };
  auto compute = [&](int buf) {
    const T* pa = &sA[buf][rdA];
    const T* pb = &sB[buf][rdB];
    vec af[2][TM], bfr[2][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i) af[0][i] = *reinterpret_cast<const vec*>(pa + 32 * i * kLDK);
#pragma unroll
    for (int j = 0; j < TN; ++j) bfr[0][j] = *reinterpret_cast<const vec*>(pb + 32 * j * kLDK);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const int cur = ks & 1;
      if (ks + 1 < KS) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
          af[cur ^ 1][i] = *reinterpret_cast<const vec*>(pa + 32 * i * kLDK + 16 * (ks + 1));
#pragma unroll
        for (int j = 0; j < TN; ++j)
          bfr[cur ^ 1][j] = *reinterpret_cast<const vec*>(pb + 32 * j * kLDK + 16 * (ks + 1));
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = Mfma32<T>::run(bfr[cur][j], af[cur][i], acc[i][j]);
    }
  };

  // Register ring of PF stages: while stage k is multiplied out of LDS
  // buffer k & 1, stages k+1 .. k+PF are in flight from global memory into
  // register set (stage % PF).  At the end of iteration k, set (k+1) % PF
  // (fetched PF-1 iterations earlier) goes to the other LDS buffer.  The loop
  // is unrolled by PF so every set index is a compile-time constant.
  // Every iteration issues its loads unconditionally (stages past the end
  // re-read the last one): the number of loads in flight is then the same on
  // every path, and the wait before an LDS store lets the younger PF - 1
  // stages stay in flight instead of draining all of them.
  auto stage = [&](int k) { return (k < nk ? k : nk - 1) * kBK; };
  static_for<0, PF>([&](auto st) { gload(st, stage(st)); });
  sstore(std::integral_constant<int, 0>{}, 0);
  __syncthreads();
  for (int kt = 0; kt < nk; kt += PF) {
    static_for<0, PF>([&](auto P) {
      constexpr int p = decltype(P)::value;        // k % PF
      constexpr int nxt = (p + 1) % PF;            // set holding stage k + 1
      const int k = kt + p;
      gload(P, stage(k + PF));                     // set p went to LDS last iteration
      if (k < nk) {
        compute(k & 1);
        if (k + 1 < nk) sstore(std::integral_constant<int, nxt>{}, (k + 1) & 1);
        __syncthreads();
      }
    });
  }

  tile_epilogue<T, BM, BN, WGM, WGN, STAGE>(a, acc, smem, bm, bn);
}

// ------------------------------------------------------------ large-tile kernel
// For products with enough tiles of 256 x 256 (or 128 x 384, 128 x 256): 8
// wavefronts (WGM x WGN = 2 x 4) of 128 x 64 (64 x 96, 64 x 64) on
// v_mfma_f32_32x32x16, the same operand
// roles, k order and epilogue as k_gemm_x, so the results are the same bits.
// A wavefront tile of 128 x 64 reads 6 KB of LDS per 8 MFMAs (the 64 x 32
// tile of k_gemm_x reads 3 KB per 2), and a 256 x 256 workgroup tile loads
// half the bytes per flop from L2 of a 128 x 128 one.
// Operand tiles travel from global memory straight into LDS
// (global_load_lds_dwordx4: lane i of a wavefront instruction writes bytes
// 16i..16i+15 of a 1 KB block), through a ring of NS stages of BK columns.
// A row of BK bf16 is CPR 16-byte chunks; chunk c of row r is stored in slot
// c ^ ((r / RPB) % CPR), RPB = rows per 256 bytes, so the 16 rows that 16
// consecutive lanes read at once (one MFMA operand fragment) fall into 16
// distinct 16-byte bank groups of the 64 four-byte banks.
// Loop schedule: the fragments of the next k-step are read while the MFMAs
// of the current one run, and across stages too: before the last k-step of
// stage k the wavefront waits for its loads of stage k+1, meets the others
// at the barrier (after it nobody reads stage k any more, and stage k+1 is
// in LDS), issues the loads of stage k+NS into stage k's slot and the
// fragment reads of stage k+1, then runs the MFMAs of stage k's last k-step.
typedef __attribute__((address_space(3))) void* lds_ptr_t;

__device__ __forceinline__ void dma16(const void* g, void* lds) {
  __builtin_amdgcn_global_load_lds(g, (lds_ptr_t)lds, 16, 0, 0);
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

__device__ __forceinline__ void wait_lgkmcnt0() {
  __builtin_amdgcn_s_waitcnt(0xF | (0x3 << 14) | (0x7 << 4));   // lgkmcnt(0), others untouched
}

template <typename T, int BM, int BN, int WGM, int WGN, int BK, int NS>
__global__ __launch_bounds__(64 * WGM * WGN)
__attribute__((amdgpu_waves_per_eu(WGM * WGN / 4, WGM * WGN / 4))) void k_gemm_big(GemmArgs a) {
  typedef typename Mfma32<T>::vec vec;
  constexpr int NW = WGM * WGN;
  constexpr int WTM = BM / WGM, WTN = BN / WGN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int KS = BK / 16;                           // k-steps per stage
  constexpr int CPR = BK * 2 / 16;                      // 16-byte chunks per row
  constexpr int RPB = 16 / CPR;                         // rows per 256 bytes
  constexpr int RPI = 1024 / (BK * 2);                  // rows per wavefront instruction
  constexpr int STAGE_ELEMS = (BM + BN) * BK;
  constexpr int LPW = (BM + BN) / RPI / NW;             // loads per wavefront per stage
  constexpr int RING = NS * STAGE_ELEMS * 2;
  constexpr int OUTB = BM * (BN + 8) * 2;
  constexpr int SMEM = RING > OUTB ? RING : OUTB;
  static_assert(sizeof(T) == 2, "16-bit operands");
  static_assert((BM + BN) % (RPI * NW) == 0, "stage rows must split over the wavefronts");
  static_assert(LPW * (NS - 1) < 64, "vmcnt range");
  static_assert(KS % 2 == 0, "fragment sets alternate per k-step across stages");
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];
  T* lds = reinterpret_cast<T*>(smem);
  const int tiles_m = (a.M + BM - 1) / BM, tiles_n = (a.N + BN - 1) / BN;
  int tm, tn;
  tile_of(blockIdx.x, tiles_m, tiles_n, tm, tn);
  const int bm = tm * BM, bn = tn * BN;
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  const T* __restrict__ A0 = static_cast<const T*>(a.A);
  const T* __restrict__ W0 = static_cast<const T*>(a.W);

  // this lane's source for each of its LPW loads: stage row
  // sr = (wave * LPW + j) * RPI + lane / CPR (rows < BM: activations, the
  // rest weight rows), chunk chosen so that it lands in its swizzled slot
  const T* src[LPW];
#pragma unroll
  for (int j = 0; j < LPW; ++j) {
    const int sr = (wave * LPW + j) * RPI + lane / CPR;
    const int chunk = (lane % CPR) ^ ((sr / RPB) % CPR);
    if (sr < BM) {
      int r = bm + sr;
      r = r < a.M ? r : a.M - 1;
      src[j] = A0 + static_cast<long long>(r) * a.lda + chunk * 8;
    } else {
      int c = bn + sr - BM;
      c = c < a.N ? c : a.N - 1;
      src[j] = W0 + static_cast<long long>(c) * a.ldw + chunk * 8;
    }
  }
  auto issue = [&](int buf, int k0) {
#pragma unroll
    for (int j = 0; j < LPW; ++j)
      dma16(src[j] + k0, lds + buf * STAGE_ELEMS + (wave * LPW + j) * RPI * BK);
  };

  const int wm = wave / WGN, wn = wave % WGN;
  const int l32 = lane & 31, g = lane >> 5;
  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  // fragment rows differ by multiples of 32 from l32, so the swizzle term
  // depends on the lane only
  const int swz = (l32 / RPB) % CPR;
  const int offA = (wm * WTM + l32) * BK, offB = (BM + wn * WTN + l32) * BK;
  vec fa[2][TM], fb[2][TN];
  auto read_frags = [&](auto set, int buf, int ks) {
    const T* st = lds + buf * STAGE_ELEMS;
    const int col = ((2 * ks + g) ^ swz) * 8;
#pragma unroll
    for (int j = 0; j < TN; ++j) fb[set][j] = *reinterpret_cast<const vec*>(st + offB + 32 * j * BK + col);
#pragma unroll
    for (int i = 0; i < TM; ++i) fa[set][i] = *reinterpret_cast<const vec*>(st + offA + 32 * i * BK + col);
  };
  auto mfmas = [&](auto set) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) acc[i][j] = Mfma32<T>::run(fb[set][j], fa[set][i], acc[i][j]);
  };

  const int nk = a.K / BK;
  // every slot of the ring starts loading
  static_for<0, NS>([&](auto st) {
    if (st < nk) issue(st, st * BK);
  });
  // stage 0 landed (the younger NS - 1 stages may stay in flight)
  if (nk >= NS) wait_vmcnt<LPW * (NS - 1)>();
  else wait_vmcnt<0>();
  __builtin_amdgcn_s_barrier();
  read_frags(std::integral_constant<int, 0>{}, 0, 0);
  // One stage.  STEADY: stage k + NS exists, so NS - 2 younger stages stay
  // in flight at the wait and the loads of stage k + NS are issued; the
  // steady loop has no branches, so the compiler's waits before the MFMAs
  // of the last k-step only cover fragments read before the barrier.
  auto stage = [&](auto steady, int k) {
    const int buf = k % NS;
    static_for<0, KS>([&](auto KSI) {
      constexpr int ks = decltype(KSI)::value;
      constexpr int cur = ks & 1;   // KS is even: the set of (k, ks) is ks & 1
      constexpr int NF = TM + TN, NM = TM * TN;   // fragment reads, MFMAs per k-step
      if constexpr (ks + 1 < KS) {
        read_frags(std::integral_constant<int, cur ^ 1>{}, buf, ks + 1);
        mfmas(std::integral_constant<int, cur>{});
        // one MFMA, then one fragment read, alternating
        static_for<0, NM>([&](auto q) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          if constexpr (decltype(q)::value < NF) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        });
      } else if constexpr (decltype(steady)::value) {
        wait_vmcnt<LPW * (NS - 2)>();   // stage k+1 landed
        wait_lgkmcnt0();                // this wavefront's reads of stage k are complete
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        issue(buf, (k + NS) * BK);
        read_frags(std::integral_constant<int, cur ^ 1>{}, (k + 1) % NS, 0);
        mfmas(std::integral_constant<int, cur>{});
        // the loads of stage k+NS, then the fragment reads of stage k+1,
        // each between two MFMAs
        static_for<0, NM>([&](auto q) {
          constexpr int i = decltype(q)::value;
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          if constexpr (i < LPW) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
          else if constexpr (i - LPW < NF) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        });
      } else {
        if (k + 1 < nk) {
          wait_vmcnt<0>();
          wait_lgkmcnt0();
          __builtin_amdgcn_s_barrier();
          asm volatile("" ::: "memory");
          read_frags(std::integral_constant<int, cur ^ 1>{}, (k + 1) % NS, 0);
        }
        mfmas(std::integral_constant<int, cur>{});
      }
    });
  };
  int k = 0;
  for (; k + NS < nk; ++k) stage(std::true_type{}, k);
  for (; k < nk; ++k) stage(std::false_type{}, k);
  tile_epilogue<T, BM, BN, WGM, WGN, (OUTB <= SMEM)>(a, acc, smem, bm, bn);
}

template <typename T, int BM, int BN, int WGM, int WGN, int BK, int NS>
static void run_big(const GemmArgs& a, hipStream_t s) {
  const dim3 grid(((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN));
  hipLaunchKernelGGL((k_gemm_big<T, BM, BN, WGM, WGN, BK, NS>), grid, dim3(64 * WGM * WGN), 0, s, a);
}

template <typename T, int BM, int BN, int WGM, int WGN, int PF>
static void run_x(const GemmArgs& a, hipStream_t s) {
  const dim3 grid(((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN));
  hipLaunchKernelGGL((k_gemm_x<T, BM, BN, WGM, WGN, PF>), grid, dim3(64 * WGM * WGN), 0, s, a);
}

template <typename T>
static void gemm_mfma(const GemmArgs& a, hipStream_t s) {
  // Long products (K >= 2048: the 4096-wide decoder's projections and head)
  // take the large-tile kernel, with the tile that fills the chip best:
  // 128 x 384 when it fills whole waves (QKV), 256 x 256 from 1.25 waves of
  // such tiles (256 CUs; gate/up, head), 128 x 256 from one wave on (O and
  // down at 2048 x 4096).  The 128 x 256 tile gives each wavefront 64 x 64
  // (4 fragment reads per 4 MFMAs; 256 x 128 gave it 128 x 32, 5 reads):
  // O 76.6 -> 73.8 us, down 184 -> 177 us.  The 256 x 256 tile takes a K
  // step of 64 in two stages: against a step of 32 in four, gate/up 357 ->
  // 340 us and the head 497 -> 465 us (one barrier per 32 MFMAs of a
  // wavefront instead of 16).  Measured on those shapes, same bits.
  // Shorter K (the 768- and 1024-wide models) stays on 128 x 128 tiles, 8
  // wavefronts of 64 x 32, operands fetched two K steps ahead; products too
  // small to give the chip ~160 such tiles (1024-row decoder GEMMs of an
  // encoder-decoder: N 768 gives 48) take 64 x 64 tiles on 4 wavefronts of
  // 32 x 32: four times the workgroups.
  auto tiles = [&](int bm, int bn) {
    return ((a.M + bm - 1) / bm) * static_cast<long long>((a.N + bn - 1) / bn);
  };
  if (a.K >= 2048) {
    // 128 x 384 when that fills whole waves exactly (QKV 2048 x 12288: 512
    // tiles, where 256 x 256 gives 1.5 waves): 233 -> 218 us
    if (tiles(128, 384) % 256 == 0 && a.N % 384 == 0 && a.M % 128 == 0)
      return run_big<T, 128, 384, 2, 4, 64, 2>(a, s);
    if (tiles(256, 256) >= 320) return run_big<T, 256, 256, 2, 4, 64, 2>(a, s);
    if (tiles(128, 256) >= 224) return run_big<T, 128, 256, 2, 4, 64, 3>(a, s);
  }
  if (tiles(128, 128) < 160) run_x<T, 64, 64, 2, 2, 2>(a, s);
  else run_x<T, 128, 128, 2, 4, 2>(a, s);
}

// ------------------------------------------------------------ fp32 kernel
// 64 x 64 tile, K step 16; thread t owns row t/4 and, in each of the four
// 16-column groups, the 4 consecutive columns 4*(t%4).. (same pairing of
// 16-column groups as the MFMA kernel, so the epilogue is shared).
template <typename T>
__global__ __launch_bounds__(256) void k_gemm_simple(GemmArgs a) {
  __shared__ float sA[64][17];
  __shared__ float sB[64][17];
  const int tiles_n = (a.N + 63) / 64;
  const int bm = (blockIdx.x / tiles_n) * 64, bn = (blockIdx.x % tiles_n) * 64;
  const int t = threadIdx.x;
  const int mr = t >> 2, c4 = (t & 3) * 4;
  float acc[4][4] = {};
  const T* A = static_cast<const T*>(a.A);
  const T* W = static_cast<const T*>(a.W);
  for (int k0 = 0; k0 < a.K; k0 += 16) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int idx = t + 256 * v, r = idx >> 4, c = idx & 15;
      int gm = bm + r;
      gm = gm < a.M ? gm : a.M - 1;
      int gn = bn + r;
      gn = gn < a.N ? gn : a.N - 1;
      const bool kin = k0 + c < a.K;
      sA[r][c] = kin ? to_f32(A[static_cast<long long>(gm) * a.lda + k0 + c]) : 0.f;
      sB[r][c] = kin ? to_f32(W[static_cast<long long>(gn) * a.ldw + k0 + c]) : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      const float x = sA[mr][kk];
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[j][r] = fmaf(x, sB[16 * j + c4 + r][kk], acc[j][r]);
    }
    __syncthreads();
  }
  SiteMax sm;
  const int m = bm + mr;
#pragma unroll
  for (int j = 0; j < 4; j += 2) epi_pair<T>(a, m, bn + 16 * j + c4, acc[j], acc[j + 1], sm);
  site_flush(a, sm);
}

// ------------------------------------------------------------ M <= 16 kernel
// A decode step multiplies B <= 16 rows by the whole weight: the work is the
// stream of weight bytes, so the kernel is laid out for HBM, not for MFMA.
// Workgroup = 8 wavefronts; wavefront w streams R consecutive packed weight
// rows with 16-byte coalesced loads, every lane covering a slice of K for
// all MP activation rows (read through L1/L2).  R = 4 (32 rows: a 16-row
// pair group) for the gated and rotary epilogues, R = 1 (8 rows, four times
// the workgroups) for the others.  The 64 lanes' partial sums are reduced by
// a transposing butterfly (each step halves the values a lane carries), the
// results meet in LDS, and wavefront 0 runs the same epilogue as the tiled
// kernel.
template <int NV>
__device__ __forceinline__ float lane_transpose_sum(float (&v)[NV], int lane, int& index) {
  index = 0;
  static_for<0, 6>([&](auto st) {
    constexpr int o = 32 >> decltype(st)::value;
    constexpr int n = NV >> decltype(st)::value;
    if constexpr (n >= 2) {
      constexpr int half = n / 2;
      const bool up = (lane & o) != 0;
#pragma unroll
      for (int j = 0; j < half; ++j) {
        const float send = up ? v[j] : v[j + half];
        const float keep = up ? v[j + half] : v[j];
        v[j] = keep + __shfl_xor(send, o, 64);
      }
      if (up) index += half;
    } else {
      v[0] += __shfl_xor(v[0], o, 64);
    }
  });
  return v[0];
}

template <typename T, int MP, int R>
__global__ __launch_bounds__(512) void k_gemm_skinny(GemmArgs a) {
  constexpr int VN = 16 / static_cast<int>(sizeof(T));
  constexpr int ROWS = 8 * R;               // weight rows per workgroup
  typedef typename std::conditional<sizeof(T) == 4, f32x4v, u32x4>::type V;
  __shared__ float res[ROWS][MP + 1];
  const int n0 = blockIdx.x * ROWS;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const T* W = static_cast<const T*>(a.W);
  const T* A = static_cast<const T*>(a.A);
  const T* wrow[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    int n = n0 + wave * R + r;
    n = n < a.N ? n : a.N - 1;
    wrow[r] = W + static_cast<long long>(n) * a.ldw;
  }
  const T* arow[MP];
#pragma unroll
  for (int m = 0; m < MP; ++m) arow[m] = A + static_cast<long long>(m < a.M ? m : a.M - 1) * a.lda;
  float acc[R * MP];
#pragma unroll
  for (int j = 0; j < R * MP; ++j) acc[j] = 0.f;
#pragma unroll 2
  for (int k = lane * VN; k < a.K; k += 64 * VN) {
    float w[R][VN];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const V raw = *reinterpret_cast<const V*>(wrow[r] + k);
      const T* e = reinterpret_cast<const T*>(&raw);
#pragma unroll
      for (int i = 0; i < VN; ++i) w[r][i] = to_f32(e[i]);
    }
#pragma unroll
    for (int m = 0; m < MP; ++m) {
      const V raw = *reinterpret_cast<const V*>(arow[m] + k);
      const T* e = reinterpret_cast<const T*>(&raw);
#pragma unroll
      for (int i = 0; i < VN; ++i) {
        const float x = to_f32(e[i]);
#pragma unroll
        for (int r = 0; r < R; ++r) acc[r * MP + m] = fmaf(w[r][i], x, acc[r * MP + m]);
      }
    }
  }
  int idx;
  const float sum = lane_transpose_sum<R * MP>(acc, lane, idx);
  // lanes that differ only in their low bits hold the same value
  if ((lane & (64 / (R * MP) - 1)) == 0) res[wave * R + idx / MP][idx % MP] = sum;
  __syncthreads();
  if (wave != 0) return;
  SiteMax sm;
  if (R == 4) {
    // a 16-row pair group: packed rows n0 + 4q + r and n0 + 16 + 4q + r
    const int m = lane >> 2, q = lane & 3;
    if (m < MP && m < a.M) {
      float va[4], vb[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        va[r] = res[4 * q + r][m];
        vb[r] = res[16 + 4 * q + r][m];
      }
      epi_pair<T>(a, m, n0 + 4 * q, va, vb, sm);
    }
  } else {
    // independent columns: 8 rows as two groups of 4; the partner columns
    // the pair epilogue would also write lie beyond this workgroup's N
    GemmArgs b = a;
    b.N = a.N - n0 < ROWS ? a.N : n0 + ROWS;
    const int m = lane >> 1, q = lane & 1;
    if (m < MP && m < a.M) {
      float va[4], vb[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int r = 0; r < 4; ++r) va[r] = res[4 * q + r][m];
      epi_pair<T>(b, m, n0 + 4 * q, va, vb, sm);
    }
  }
  site_flush(a, sm);
}

// Independent-column epilogues on a narrow output: workgroup = 8 weight
// rows, and the 8 wavefronts split K instead of the rows, each covering all
// 8 rows for its K slice, so every lane's loads (8 weight and MP activation
// vectors per step) leave together and a short K needs a single round trip
// to memory.  Lane partials are reduced by the transposing butterfly, the 8
// wavefronts' sums are added in LDS.
template <typename T, int MP>
__global__ __launch_bounds__(512) void k_gemm_skinny_ks(GemmArgs a) {
  constexpr int VN = 16 / static_cast<int>(sizeof(T));
  constexpr int R = 8;
  typedef typename std::conditional<sizeof(T) == 4, f32x4v, u32x4>::type V;
  __shared__ float part[8][R * MP];
  __shared__ float res[R][MP + 1];
  const int n0 = blockIdx.x * R;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const T* W = static_cast<const T*>(a.W);
  const T* A = static_cast<const T*>(a.A);
  // this wavefront's K slice, a multiple of VN
  const int per = ((a.K + 8 * VN - 1) / (8 * VN)) * VN;
  const int kb = wave * per, ke = min(a.K, kb + per);
  const T* wrow[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    int n = n0 + r;
    n = n < a.N ? n : a.N - 1;
    wrow[r] = W + static_cast<long long>(n) * a.ldw;
  }
  const T* arow[MP];
#pragma unroll
  for (int m = 0; m < MP; ++m) arow[m] = A + static_cast<long long>(m < a.M ? m : a.M - 1) * a.lda;
  float acc[R * MP];
#pragma unroll
  for (int j = 0; j < R * MP; ++j) acc[j] = 0.f;
  for (int k = kb + lane * VN; k < ke; k += 64 * VN) {
    V wv[R], av[MP];
#pragma unroll
    for (int r = 0; r < R; ++r) wv[r] = *reinterpret_cast<const V*>(wrow[r] + k);
#pragma unroll
    for (int m = 0; m < MP; ++m) av[m] = *reinterpret_cast<const V*>(arow[m] + k);
#pragma unroll
    for (int m = 0; m < MP; ++m) {
      const T* ae = reinterpret_cast<const T*>(&av[m]);
#pragma unroll
      for (int i = 0; i < VN; ++i) {
        const float x = to_f32(ae[i]);
#pragma unroll
        for (int r = 0; r < R; ++r)
          acc[r * MP + m] = fmaf(to_f32(reinterpret_cast<const T*>(&wv[r])[i]), x, acc[r * MP + m]);
      }
    }
  }
  int idx;
  const float sum = lane_transpose_sum<R * MP>(acc, lane, idx);
  if ((lane & (64 / (R * MP) - 1)) == 0) part[wave][idx] = sum;
  __syncthreads();
  if (threadIdx.x < R * MP) {
    float t = 0.f;
#pragma unroll
    for (int w2 = 0; w2 < 8; ++w2) t += part[w2][threadIdx.x];
    res[threadIdx.x / MP][threadIdx.x % MP] = t;
  }
  __syncthreads();
  if (wave != 0) return;
  SiteMax sm;
  GemmArgs b = a;
  b.N = a.N - n0 < R ? a.N : n0 + R;
  const int m = lane >> 1, q = lane & 1;
  if (m < MP && m < a.M) {
    float va[4], vb[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int r = 0; r < 4; ++r) va[r] = res[4 * q + r][m];
    epi_pair<T>(b, m, n0 + 4 * q, va, vb, sm);
  }
  site_flush(a, sm);
}

// A few rows (M <= 16) against a wide plain output (the LM head of a
// decode step): the 2 M N K multiply-adds on the matrix cores instead of
// the VALU.  Each wavefront computes 16 output columns for every row with
// v_mfma_f32_16x16x32 (16 weight rows as the A operand, the activation rows
// padded to 16 as the B operand; lane l supplies row l % 16 and k
// 8 (l / 16) .. + 7 of each 32-wide k step), 8 k steps of loads in flight,
// and ends with columns 4 (l / 16) .. + 3 of activation row l % 16.
template <typename T> struct Mfma16;
template <> struct Mfma16<bf16_t> {
  typedef bf16x8 vec;
  static __device__ __forceinline__ f32x4 run(vec a, vec b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct Mfma16<f16_t> {
  typedef f16x8 vec;
  static __device__ __forceinline__ f32x4 run(vec a, vec b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
  }
};

template <typename T>
__global__ __launch_bounds__(256) void k_gemm_skinny_mfma(GemmArgs a) {
  typedef typename Mfma16<T>::vec vec;
  constexpr int U = 8;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int n0 = (blockIdx.x * 4 + wave) * 16;
  if (n0 >= a.N) return;                     // no barrier in this kernel
  const int l16 = lane & 15, kg = lane >> 4;
  const int n = n0 + l16 < a.N ? n0 + l16 : a.N - 1;
  const int m = l16 < a.M ? l16 : a.M - 1;
  const T* wp = static_cast<const T*>(a.W) + static_cast<long long>(n) * a.ldw + 8 * kg;
  const T* xp = static_cast<const T*>(a.A) + static_cast<long long>(m) * a.lda + 8 * kg;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  int k = 0;
  for (; k + 32 * U <= a.K; k += 32 * U) {
    vec wf[U], xf[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      wf[u] = *reinterpret_cast<const vec*>(wp + k + 32 * u);
      xf[u] = *reinterpret_cast<const vec*>(xp + k + 32 * u);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) acc = Mfma16<T>::run(wf[u], xf[u], acc);
  }
  for (; k < a.K; k += 32)
    acc = Mfma16<T>::run(*reinterpret_cast<const vec*>(wp + k), *reinterpret_cast<const vec*>(xp + k),
                         acc);
  SiteMax sm;
  GemmArgs b = a;
  b.N = a.N - n0 < 16 ? a.N : n0 + 16;       // the pair columns (+16) lie beyond this wavefront's
  const float va[4] = {acc[0], acc[1], acc[2], acc[3]};
  const float vb[4] = {0.f, 0.f, 0.f, 0.f};
  epi_pair<T>(b, l16, n0 + 4 * kg, va, vb, sm);
  site_flush(a, sm);
}

template <typename T>
static void skinny_ks(const GemmArgs& a, hipStream_t s) {
  const dim3 grid((a.N + 7) / 8), block(512);
  if (a.M <= 1) hipLaunchKernelGGL((k_gemm_skinny_ks<T, 1>), grid, block, 0, s, a);
  else if (a.M <= 2) hipLaunchKernelGGL((k_gemm_skinny_ks<T, 2>), grid, block, 0, s, a);
  else if (a.M <= 4) hipLaunchKernelGGL((k_gemm_skinny_ks<T, 4>), grid, block, 0, s, a);
  else hipLaunchKernelGGL((k_gemm_skinny_ks<T, 8>), grid, block, 0, s, a);
}

template <typename T, int R>
static void skinny_r(const GemmArgs& a, hipStream_t s) {
  const dim3 grid((a.N + 8 * R - 1) / (8 * R)), block(512);
  if (a.M <= 1) hipLaunchKernelGGL((k_gemm_skinny<T, 1, R>), grid, block, 0, s, a);
  else if (a.M <= 2) hipLaunchKernelGGL((k_gemm_skinny<T, 2, R>), grid, block, 0, s, a);
  else if (a.M <= 4) hipLaunchKernelGGL((k_gemm_skinny<T, 4, R>), grid, block, 0, s, a);
  else if (a.M <= 8) hipLaunchKernelGGL((k_gemm_skinny<T, 8, R>), grid, block, 0, s, a);
  else hipLaunchKernelGGL((k_gemm_skinny<T, 16, R>), grid, block, 0, s, a);
}

template <typename T>
static void skinny_t(const GemmArgs& a, hipStream_t s) {
  // the gated and rotary epilogues combine packed rows 16 apart; a wide
  // output (the head) has workgroups enough with 32 rows each, and four rows
  // per wavefront reuse every activation load four times
  // a wide plain output (the head) in 16-bit on the matrix cores
  if constexpr (sizeof(T) == 2) {
    if (a.epi == kEpiStore && !a.bias && a.site < 0 && !a.kc && a.N >= 8192 && a.K % 32 == 0) {
      hipLaunchKernelGGL((k_gemm_skinny_mfma<T>), dim3((a.N + 63) / 64), dim3(256), 0, s, a);
      return;
    }
  }
  if (a.epi == kEpiGatedGelu || a.epi == kEpiGatedSilu || a.epi == kEpiRope || a.N >= 8192)
    skinny_r<T, 4>(a, s);
  else if (a.M <= 8 && a.N < 2048)     // few row groups: split K across the wavefronts
    skinny_ks<T>(a, s);
  else
    skinny_r<T, 1>(a, s);
}

void launch_gemm(const GemmArgs& a, hipStream_t s) {
  if (a.M <= 16) {
    if (a.dtype == kF32) skinny_t<float>(a, s);
    else if (a.dtype == kBF16) skinny_t<bf16_t>(a, s);
    else skinny_t<f16_t>(a, s);
    return;
  }
  if (a.dtype == kF32) {
    const dim3 grid(((a.M + 63) / 64) * ((a.N + 63) / 64));
    hipLaunchKernelGGL(k_gemm_simple<float>, grid, dim3(256), 0, s, a);
    return;
  }
  if (a.dtype == kBF16) gemm_mfma<bf16_t>(a, s);
  else gemm_mfma<f16_t>(a, s);
}

}  // namespace gm
