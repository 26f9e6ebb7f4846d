// Internal definitions shared by the GLIDE HIP kernels and the C-ABI layer.
// Device code for gfx950 only (64-wide wavefronts, MFMA 16x16 tiles).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "glide.h"

namespace glide {

constexpr int kMaxLayersPerLaunch = 64;
constexpr int kMaxG = 16;  // query heads per KV head: one MFMA row tile

__host__ __device__ inline int64_t align256(int64_t x) { return (x + 255) & ~int64_t(255); }

// Ring slots of a layer with softmax window W: R > W keeps the slot of the
// token leaving the window distinct from the slot the new token is written
// to, so both can be touched in one decode pass.  Multiple of 8 so that an
// 8-token block of the transposed value ring never wraps.
__host__ __device__ inline int32_t ring_slots(int32_t W) { return W > 0 ? ((W + 1 + 7) & ~7) : 0; }

// Byte offsets of the sections of one layer, relative to the layer's start.
struct LayerSections {
  int64_t pos, S, z, K, V, bytes;
};

__host__ __device__ inline LayerSections layer_sections(int B, int Hkv, int d, int Df, int R, int esize) {
  LayerSections s;
  const int64_t units = int64_t(B) * Hkv;
  s.pos = 0;
  s.S = align256(units * 8);
  s.z = s.S + align256(units * Df * d * 4);
  s.K = s.z + align256(units * Df * 4);
  s.V = s.K + align256(units * int64_t(R) * d * esize);
  s.bytes = s.V + align256(units * int64_t(R) * d * esize);
  return s;
}

// Per-layer description handed to kernels by value.
struct LayerArg {
  int64_t base;    // byte offset of the layer inside the state blob
  int32_t W;       // softmax window
  int32_t R;       // ring slots
  int32_t slot;    // index of the layer inside the call's q/k/v/out/phi_w arrays
  int32_t pad;
};

// ---------------------------------------------------------------------------
// Element types.  bf16 is carried as raw 16-bit patterns.
typedef uint16_t bf16_t;

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16_t x) { return __uint_as_float(uint32_t(x) << 16); }

template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
// Round to nearest even (NaN kept quiet).
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float x) {
  uint32_t u = __float_as_uint(x);
  if ((u & 0x7fffffffu) > 0x7f800000u) return bf16_t((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return bf16_t(u >> 16);
}

// ---------------------------------------------------------------------------
// MFMA fragments.  Every contraction is issued as 16x16 output tiles with a
// 32-wide slab of the reduction index k.  For both element types, lane l
// holds 8 values of row (l % 16) at k = 8*(l/16) .. 8*(l/16)+7 of the slab
// (A operand: row = m; B operand: row = n).  The accumulator holds rows
// 4*(l/16) + i (i = 0..3) of column l % 16.
//   bf16: one v_mfma_f32_16x16x32_bf16 per slab.
//   fp32: eight v_mfma_f32_16x16x4_f32, step s taking element s of every
//         lane (k = 8*(l/16) + s), which covers the same 32 k values.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

template <typename T> struct Frag;
template <> struct Frag<bf16_t> {
  uint4 v;  // 8 packed bf16
  __device__ __forceinline__ void zero() { v = make_uint4(0, 0, 0, 0); }
  __device__ __forceinline__ void load(const bf16_t* p) { v = *reinterpret_cast<const uint4*>(p); }
  __device__ __forceinline__ float get(int i) const {
    const uint32_t w = (&v.x)[i >> 1];
    return __uint_as_float((i & 1) ? (w & 0xffff0000u) : (w << 16));
  }
  __device__ __forceinline__ void set(int i, float x) {
    uint32_t& w = (&v.x)[i >> 1];
    const uint32_t b = from_f32<bf16_t>(x);
    w = (i & 1) ? ((w & 0xffffu) | (b << 16)) : ((w & 0xffff0000u) | b);
  }
  __device__ __forceinline__ void set_raw(int i, bf16_t b) {
    uint32_t& w = (&v.x)[i >> 1];
    w = (i & 1) ? ((w & 0xffffu) | (uint32_t(b) << 16)) : ((w & 0xffff0000u) | b);
  }
};
template <> struct Frag<float> {
  float v[8];
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = 0.f;
  }
  __device__ __forceinline__ void load(const float* p) {
    const float4 a = reinterpret_cast<const float4*>(p)[0];
    const float4 b = reinterpret_cast<const float4*>(p)[1];
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  }
  __device__ __forceinline__ float get(int i) const { return v[i]; }
  __device__ __forceinline__ void set(int i, float x) { v[i] = x; }
  __device__ __forceinline__ void set_raw(int i, float x) { v[i] = x; }
};

__device__ __forceinline__ f32x4_t mma(const Frag<bf16_t>& a, const Frag<bf16_t>& b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a.v),
                                                 __builtin_bit_cast(bf16x8_t, b.v), c, 0, 0, 0);
}
__device__ __forceinline__ f32x4_t mma(const Frag<float>& a, const Frag<float>& b, f32x4_t c) {
#pragma unroll
  for (int s = 0; s < 8; ++s) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[s], b.v[s], c, 0, 0, 0);
  return c;
}

__device__ __forceinline__ f32x4_t zero4() { return f32x4_t{0.f, 0.f, 0.f, 0.f}; }

// ---------------------------------------------------------------------------
// Launch descriptors.

struct DecodeArgs {
  char* state;
  const void* phi_w;
  const void* q;
  const void* k;
  const void* v;
  void* out;
  int32_t B, Hq, Hkv, G;
  int32_t linear;
  float tau;
  int32_t n_layers;  // layers in this launch (<= kMaxLayersPerLaunch)
  int32_t pad;
  LayerArg layers[kMaxLayersPerLaunch];  // sorted by decreasing W
};

// Host-side launchers (one translation unit per kernel family).
hipError_t launch_decode(const DecodeArgs& a, int d, int Df, int dtype, hipStream_t stream);

}  // namespace glide
