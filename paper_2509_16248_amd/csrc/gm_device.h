// gm_device.h -- device-side helpers shared by the libgm kernels:
// storage-dtype conversion, wavefront reductions, and the layout of the
// model's int32 state slots.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gm {

// ------------------------------------------------------------ state slots
// One int32 array per model.  "per-forward" slots are rewritten by the
// prologue kernel of every forward; "persistent" slots survive forwards.
enum Slot : int {
  kPadAny = 0,       // per-forward: 1 if the mask has a 0 (padding branch taken)
  kRegrow = 1,       // per-forward: 1 if the rotary table grew in this forward
  kNeed = 2,         // per-forward: max(position) + 1
  kCachedLen = 3,    // persistent: rotary rows valid
  kTrapFwd = 4,      // per-forward: (code << 24 | index), 0xFFFFFFFF = none
  kTrapSticky = 5,   // persistent: first trap word since the last check, 0 = none
  kFwdCount = 6,     // persistent: forwards run so far
  kRegrowFrom = 7,   // per-forward: rotary rows [from, to) to fill
  kRegrowTo = 8,
  kFifoCount = 9,    // persistent until flush: records written
  kFifoDropped = 10, // persistent until flush: records lost to overflow
  kPadCount = 11,    // per-forward: number of mask zeros
  kFwdIndex = 12,    // per-forward: index of this forward
  kLogCount = 13,    // persistent until flush: log values written to the arena
  kLogDropped = 14,  // persistent until flush: log values lost to overflow
  kRopeLong = 15,    // per-forward: long rotary frequencies selected
  kPadAnyTgt = 16,   // per-forward, encoder-decoder: the target mask has a 0
  kPadCountTgt = 17, // per-forward, encoder-decoder: number of target mask zeros
  kClampBase = 32,                    // per-forward: 2*kMaxLayers trip decisions
  kAbsmaxBase = kClampBase + 128,     // per-forward: bits of max |h| per site
  kNanBase = kAbsmaxBase + 128,       // per-forward: NaN seen per site
  kKvLenBase = kNanBase + 128,        // per-forward: 1 + last unmasked key, per sequence
                                      // (encoder-decoder: the target's follow at + max_batch)
};
constexpr int kMaxLayers = 64;
constexpr uint32_t kTrapNone = 0xFFFFFFFFu;

struct EffectRec {   // gm_effect, with its tensor payload as a range of the log arena
  int32_t forward, kind, layer, site;
  float value;
  int32_t offset, count;
};

// ------------------------------------------------------------ vector types
// Native clang vector types for 8/16-byte memory accesses.  (HIP's uint4 /
// float4 are structs with unions; arrays of them are not promoted to
// registers and end up in scratch memory.)
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4v __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------ storage dtypes
typedef uint16_t bf16_t;   // bfloat16 bit pattern
typedef _Float16 f16_t;

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16_t x) {
  return __uint_as_float(static_cast<uint32_t>(x) << 16);
}
__device__ __forceinline__ float to_f32(f16_t x) { return static_cast<float>(x); }

template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
// float32 -> bfloat16, round to nearest even, NaN kept quiet (gfx950's
// v_cvt_pk_bf16_f32).
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float x) {
  return __builtin_bit_cast(bf16_t, static_cast<__bf16>(x));
}
template <> __device__ __forceinline__ f16_t from_f32<f16_t>(float x) {
  return static_cast<f16_t>(x);
}

// Value after storage in T, as float.
template <typename T> __device__ __forceinline__ float round_as(float x) {
  return to_f32(from_f32<T>(x));
}

// ------------------------------------------------------------ reductions
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    uint32_t w = __shfl_xor(v, o, 64);
    v = v > w ? v : w;
  }
  return v;
}
__device__ __forceinline__ int wave_or(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v |= __shfl_xor(v, o, 64);
  return v;
}

// fp16 overflow guard: clamp bound and trip test on a site's reduction.
__device__ __forceinline__ bool clamp_trip(const int32_t* state, int site, float thr) {
  if (state[kNanBase + site]) return false;  // max() propagates NaN; NaN > thr is false
  return __uint_as_float(static_cast<uint32_t>(state[kAbsmaxBase + site])) > thr;
}

}  // namespace gm
