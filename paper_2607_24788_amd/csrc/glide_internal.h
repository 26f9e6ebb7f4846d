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

// Deferred folding.  Decode folds the tokens that have left the window into
// S and z in batches: a unit keeps up to kFoldPeriod of them "pending" in its
// ring (their contribution to the read-out is added from the ring), and folds
// them all at once on one step out of kFoldPeriod.  The step is staggered over
// units, so on every step about 1/kFoldPeriod of the state is written back
// instead of all of it.  W = 0 layers (no ring) fold every step.
constexpr int kFoldPeriod = 8;
static_assert((kFoldPeriod & (kFoldPeriod - 1)) == 0, "the fold turn is a bit mask");

// Ring slots of a layer with softmax window W: R >= W + kFoldPeriod holds the
// window, the pending tokens and keeps the new token's slot distinct from
// both.  A multiple of 32 so that a 32-token tile (token j0 = 0 mod 32) is one
// contiguous 32-slot ring block.
__host__ __device__ inline int32_t ring_slots(int32_t W) { return W > 0 ? ((W + kFoldPeriod + 31) & ~31) : 0; }

// (x mod R) for 0 <= x < 2R.
__device__ __forceinline__ uint32_t wrap_once(uint32_t x, uint32_t R) { return x >= R ? x - R : x; }

// Ring layouts, per (sequence, KV head), in 32-slot blocks of 32*D elements.
// Both are the MFMA fragment order of the decode kernel, so every fragment
// load of a wave reads 1 KB (bf16) of consecutive memory.
//  key   : block [t][D/32][4][16][8] -- slot offset o = 8*(m/4) + 4*t + m%4
//          (row m of 16-key sub-tile t), element c = 32*kk + 8*g + e
//  value : block [D/16][4][16][8]    -- slot offset o = 8*g + e, element
//          c = 16*ct + n
__host__ __device__ inline int64_t kring_elem(int32_t slot, int c, int D) {
  const int blk = slot >> 5, o = slot & 31;
  const int t = (o >> 2) & 1, m = ((o >> 3) << 2) | (o & 3);
  const int kk = c >> 5, g = (c >> 3) & 3, e = c & 7;
  return int64_t(blk) * 32 * D + ((((t * (D / 32) + kk) * 4 + g) * 16 + m) * 8 + e);
}
__host__ __device__ inline int64_t vring_elem(int32_t slot, int c, int D) {
  const int blk = slot >> 5, o = slot & 31;
  const int ct = c >> 4, n = c & 15, g = o >> 3, e = o & 7;
  return int64_t(blk) * 32 * D + (((ct * 4 + g) * 16 + n) * 8 + e);
}
// First element of the 8-element key chunk (k-slab kk, lane group g) of slot s.
__host__ __device__ inline int64_t kring_chunk(int32_t slot, int kk, int g, int D) {
  return kring_elem(slot, 32 * kk + 8 * g, D);
}

// Byte offsets of the sections of one layer, relative to the layer's start.
// A gated layer (GLIDE_GATED) appends, per unit, G_cur and G_fold (fp64) and
// a ring of the cumulative log-gates G_j of its ring tokens (fp64, slot j mod
// R); the other offsets do not depend on it.
struct LayerSections {
  int64_t pos, nf, cnt, S, z, K, V, G, GR, bytes;
};

__host__ __device__ inline LayerSections layer_sections(int B, int Hkv, int d, int Df, int R, int esize,
                                                        bool gated = false) {
  LayerSections s;
  const int64_t units = int64_t(B) * Hkv;
  s.pos = 0;
  s.nf = align256(units * 8);
  s.cnt = s.nf + align256(units * 8);
  s.S = s.cnt + align256(units * 4);
  s.z = s.S + align256(units * Df * d * 4);
  s.K = s.z + align256(units * Df * 4);
  s.V = s.K + align256(units * int64_t(R) * d * esize);
  s.G = s.V + align256(units * int64_t(R) * d * esize);
  s.GR = s.G + (gated ? align256(units * 16) : 0);
  s.bytes = s.GR + (gated ? align256(units * int64_t(R) * 8) : 0);
  return s;
}

// exp(x) of a log-decay x <= 0 (fp32, base-2 hardware exponential).
__device__ __forceinline__ float decay_exp(float x) { return __builtin_amdgcn_exp2f(x * 1.4426950408889634f); }

// Per-layer description handed to kernels by value.
struct LayerArg {
  int64_t base;    // byte offset of the layer inside the state blob
  int32_t W;       // softmax window
  int32_t R;       // ring slots
  int32_t slot;    // index of the layer inside the call's q/k/v/out/phi_w arrays
  int32_t npiece;  // decode: workgroups per unit (window split), >= 1
  int32_t prow0;   // decode: piece row (workgroup / (B*Hkv)) of the layer's piece 0
  int32_t prow1;   // decode: piece row of its piece 1 (pieces 1.. are consecutive)
};

// Decode window split.  When a call has few units the longest windows would
// leave most CUs idle, so a unit's window tiles are spread over npiece
// workgroups ("pieces"); piece 0 also does the ring write and the state.
// Pieces write partial records (running max, sum and weighted values of the
// window part per head; piece 0 adds the linear part); the piece that
// finishes last (a per-unit counter in the state) merges them.  The split
// depends on the layers of the launch and on the device: the pieces are made
// as small as possible while every workgroup of the launch still fits in one
// round of resident workgroups (kDecodeWgPerCu per CU, from the device's CU
// count), since a second round would be latency-bound; launches with that
// many units or more are not split.  kMaxDecodeSlots bounds the round on any
// device (and with it the partial records the workspace must hold).
constexpr int kDecodeWgPerCu = 2;
constexpr int kMaxDecodeSlots = 1024;
constexpr int kMaxPieces = 16;
// The state pass of piece 0 counted in 32-token window tiles, for the shares
// of a split window: in a latency-bound launch (small pieces) it is a chain
// of dependent loads and LDS steps that lasts as long as about 16 tiles; in
// a bandwidth-bound one (pieces of kStreamPieceTiles tiles or more) it costs
// its bytes, about 4 tiles.
constexpr int kStateTilesLatency = 16;
constexpr int kStateTilesStream = 4;
constexpr int kStreamPieceTiles = 32;
// A unit whose window has fewer tiles than this is not split: the merge of
// the pieces (records written through to memory, a counter, the records read
// back) lasts longer than a whole workgroup's pass over such a window.
constexpr int kSplitMinTiles = 10;
__host__ __device__ inline int decode_tiles_max(int32_t W) { return W > 0 ? (W + 31) / 32 + 1 : 0; }
// floats of one partial record: per head m, l, dn, acc[d], nm[d]
__host__ __device__ inline int64_t part_floats(int G, int d) { return int64_t(G) * (2 * d + 3); }

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

// Two floats to a packed bf16 pair (round to nearest even, v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  const bf16x2_t h = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, h);
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
  // Elements k, k+stride, ..., k+7*stride of a strided row (e.g. a column
  // of a row-major matrix).
  __device__ __forceinline__ void load_strided(const bf16_t* p, int stride) {
    v.x = uint32_t(p[0]) | (uint32_t(p[stride]) << 16);
    v.y = uint32_t(p[2 * stride]) | (uint32_t(p[3 * stride]) << 16);
    v.z = uint32_t(p[4 * stride]) | (uint32_t(p[5 * stride]) << 16);
    v.w = uint32_t(p[6 * stride]) | (uint32_t(p[7 * stride]) << 16);
  }
  __device__ __forceinline__ void to_floats(float* x) const {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[2 * i] = __uint_as_float(w[i] << 16);
      x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
  // Sum of the 8 elements as fp32.
  __device__ __forceinline__ float sum() const {
    float s = 0.f;
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) s += __uint_as_float(w[i] << 16) + __uint_as_float(w[i] & 0xffff0000u);
    return s;
  }
  // 8 floats -> 8 bf16 (compile-time positions only)
  __device__ __forceinline__ void set8(const float* x) {
    v.x = pack_bf16x2(x[0], x[1]);
    v.y = pack_bf16x2(x[2], x[3]);
    v.z = pack_bf16x2(x[4], x[5]);
    v.w = pack_bf16x2(x[6], x[7]);
  }
  // Every element's sign flipped (exact).
  __device__ __forceinline__ void negate() {
    v.x ^= 0x80008000u;
    v.y ^= 0x80008000u;
    v.z ^= 0x80008000u;
    v.w ^= 0x80008000u;
  }
  // Replace element i (runtime, 0..7) by b without indexing registers
  // dynamically (a dynamic index would force the fragment to scratch).
  __device__ __forceinline__ void patch(int i, bf16_t b) {
    const uint32_t sh = (i & 1) * 16;
    const uint32_t keep = ~(0xffffu << sh), put = uint32_t(b) << sh;
    const int wi = i >> 1;
    v.x = wi == 0 ? ((v.x & keep) | put) : v.x;
    v.y = wi == 1 ? ((v.y & keep) | put) : v.y;
    v.z = wi == 2 ? ((v.z & keep) | put) : v.z;
    v.w = wi == 3 ? ((v.w & keep) | put) : v.w;
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
  __device__ __forceinline__ void to_floats(float* x) const {
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = v[i];
  }
  __device__ __forceinline__ void load_strided(const float* p, int stride) {
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = p[i * stride];
  }
  __device__ __forceinline__ float sum() const {
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) s += v[i];
    return s;
  }
  __device__ __forceinline__ void set8(const float* x) {
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = x[i];
  }
  __device__ __forceinline__ void negate() {
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = -v[i];
  }
  __device__ __forceinline__ void patch(int i, float b) {
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = (e == i) ? b : v[e];
  }
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

// The feature map's activation on y = x . Wf: ReLU (phi = 0), ELU + 1
// (phi = 1: y + 1 for y > 0, e^y otherwise; never zero), or, for the softmax
// map (phi = 2), y itself: the row is normalised afterwards by a pass over all
// its features (softmax_rows_lds, or in registers where one wave holds them).
__device__ __forceinline__ float feat_act(float y, int phi) {
  return phi == GLIDE_PHI_ELU1   ? (y > 0.f ? y + 1.f : __builtin_amdgcn_exp2f(y * 1.4426950408889634f))
         : phi == GLIDE_PHI_RELU ? fmaxf(y, 0.f)
                                 : y;
}

// Cross-lane reductions with DPP moves inside 16-lane rows.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_mv(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, ROW_MASK, 0xf, false));
}
// Sum over lanes 0 .. N-1 of each 32-lane half (N = 16 or 32; other lanes may
// hold anything): every lane of a row holds its row's sum (N = 16), or lanes
// 16 .. 31 hold the 32-lane sum (N = 32).
template <int N>
__device__ __forceinline__ float dpp_sum_rows(float v) {
  static_assert(N == 16 || N == 32, "16 or 32 lanes");
  v += dpp_mv<0xb1, 0xf>(v);   // quad_perm [1,0,3,2]
  v += dpp_mv<0x4e, 0xf>(v);   // quad_perm [2,3,0,1]
  v += dpp_mv<0x141, 0xf>(v);  // row_half_mirror
  v += dpp_mv<0x140, 0xf>(v);  // row_mirror: every lane holds its row's sum
  if constexpr (N == 32) v += dpp_mv<0x142, 0xa>(v);  // row_bcast:15 into rows 1 and 3
  return v;
}
// Maximum over the 16 lanes of each row, in every lane of the row.
__device__ __forceinline__ float dpp_max_row16(float v) {
  v = fmaxf(v, dpp_mv<0xb1, 0xf>(v));
  v = fmaxf(v, dpp_mv<0x4e, 0xf>(v));
  v = fmaxf(v, dpp_mv<0x141, 0xf>(v));
  v = fmaxf(v, dpp_mv<0x140, 0xf>(v));
  return v;
}

// The softmax feature map's normalisation, in place, on rows [0, nrows) of an
// fp32 LDS matrix (row r at base + r * stride, DF features): x <- e^(x - max)
// / sum e^(x - max).  16 lanes (one DPP row) per row, DF / 16 features each;
// every thread of the workgroup (NTH threads) calls it, between barriers.
template <int DF, int NTH>
__device__ __forceinline__ void softmax_rows_lds(float* base, int stride, int nrows) {
  constexpr int FPL = DF / 16;
  const int sub = int(threadIdx.x) & 15;
  for (int r0 = 0; r0 < nrows; r0 += NTH / 16) {
    const int r = r0 + int(threadIdx.x >> 4);
    const bool ok = r < nrows;
    float* row = base + (ok ? r : 0) * stride + sub * FPL;
    float x[FPL];
    float m = -INFINITY;
#pragma unroll
    for (int j = 0; j < FPL; ++j) {
      x[j] = ok ? row[j] : 0.f;
      m = fmaxf(m, x[j]);
    }
    m = dpp_max_row16(m);
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < FPL; ++j) {
      x[j] = __builtin_amdgcn_exp2f((x[j] - m) * 1.4426950408889634f);
      s += x[j];
    }
    s = dpp_sum_rows<16>(s);
    const float inv = 1.f / s;
    if (ok) {
#pragma unroll
      for (int j = 0; j < FPL; ++j) row[j] = x[j] * inv;
    }
  }
}

// Fragment of 8 consecutive ROWS of one column from a row-major LDS tile M
// (row stride rs elements): lane (n = lane%16, g = lane/16) receives
// M[row0 + e][col0 + n], e = 0..7, where row0 must be equal across each group
// of 16 lanes (here row0 = 8*g + const).  This is the operand layout of a
// contraction over rows (keys) with the tile stored naturally.
//   bf16: two ds_read_b64_tr_b16.  Within a 16-lane group, source lane i
//   supplies 4 consecutive 16-bit values and output lane j receives, in slot
//   s, element j%4 of source lane 4s + j/4; pointing source lane i at
//   M[row0 + i/4][col0 + 4*(i%4)] therefore hands lane j the column
//   M[row0 .. row0+3][col0 + j].
//   fp32: eight scalar LDS reads.
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4_t lds_i16x4_t;

__device__ __forceinline__ void load_colfrag(Frag<bf16_t>& f, const bf16_t* M, int rs, int row0, int col0) {
  const int n = threadIdx.x & 15;
  const bf16_t* p = M + (row0 + (n >> 2)) * rs + col0 + 4 * (n & 3);
  const auto* p1 = (lds_i16x4_t*)(__attribute__((address_space(3))) bf16_t*)(p);
  const auto* p2 = (lds_i16x4_t*)(__attribute__((address_space(3))) bf16_t*)(p + 4 * rs);
  const i16x4_t a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t*)p1);
  const i16x4_t b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t*)p2);
  f.v.x = uint32_t(uint16_t(a[0])) | (uint32_t(uint16_t(a[1])) << 16);
  f.v.y = uint32_t(uint16_t(a[2])) | (uint32_t(uint16_t(a[3])) << 16);
  f.v.z = uint32_t(uint16_t(b[0])) | (uint32_t(uint16_t(b[1])) << 16);
  f.v.w = uint32_t(uint16_t(b[2])) | (uint32_t(uint16_t(b[3])) << 16);
}
__device__ __forceinline__ void load_colfrag(Frag<float>& f, const float* M, int rs, int row0, int col0) {
  const int n = threadIdx.x & 15;
#pragma unroll
  for (int e = 0; e < 8; ++e) f.v[e] = M[(row0 + e) * rs + col0 + n];
}
// As load_colfrag, with the 8 rows taken as rows r0 .. r0+3, then r1 .. r1+3
// (a permuted order of the reduction index, shared with the other operand).
__device__ __forceinline__ void load_colfrag2(Frag<bf16_t>& f, const bf16_t* M, int rs, int r0, int r1, int col0) {
  const int n = threadIdx.x & 15;
  const bf16_t* p = M + (r0 + (n >> 2)) * rs + col0 + 4 * (n & 3);
  const bf16_t* q = M + (r1 + (n >> 2)) * rs + col0 + 4 * (n & 3);
  const i16x4_t a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t*)(__attribute__((address_space(3))) bf16_t*)(p));
  const i16x4_t b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t*)(__attribute__((address_space(3))) bf16_t*)(q));
  f.v.x = uint32_t(uint16_t(a[0])) | (uint32_t(uint16_t(a[1])) << 16);
  f.v.y = uint32_t(uint16_t(a[2])) | (uint32_t(uint16_t(a[3])) << 16);
  f.v.z = uint32_t(uint16_t(b[0])) | (uint32_t(uint16_t(b[1])) << 16);
  f.v.w = uint32_t(uint16_t(b[2])) | (uint32_t(uint16_t(b[3])) << 16);
}
__device__ __forceinline__ void load_colfrag2(Frag<float>& f, const float* M, int rs, int r0, int r1, int col0) {
  const int n = threadIdx.x & 15;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    f.v[e] = M[(r0 + e) * rs + col0 + n];
    f.v[4 + e] = M[(r1 + e) * rs + col0 + n];
  }
}
// From an fp32 LDS tile, converted to the fragment's element type.
__device__ __forceinline__ void load_colfrag2_f32(Frag<bf16_t>& f, const float* M, int rs, int r0, int r1,
                                                  int col0) {
  const int n = threadIdx.x & 15;
  float x[8];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    x[e] = M[(r0 + e) * rs + col0 + n];
    x[4 + e] = M[(r1 + e) * rs + col0 + n];
  }
  f.set8(x);
}
__device__ __forceinline__ void load_colfrag2_f32(Frag<float>& f, const float* M, int rs, int r0, int r1, int col0) {
  load_colfrag2(f, M, rs, r0, r1, col0);
}
// 8 elements of one row: 4 at column c0, 4 at column c1 (the same permuted
// reduction order, for an operand stored row-major).
__device__ __forceinline__ void load_row2(Frag<bf16_t>& f, const bf16_t* row, int c0, int c1) {
  const uint2 a = *reinterpret_cast<const uint2*>(row + c0);
  const uint2 b = *reinterpret_cast<const uint2*>(row + c1);
  f.v = make_uint4(a.x, a.y, b.x, b.y);
}
__device__ __forceinline__ void load_row2(Frag<float>& f, const float* row, int c0, int c1) {
  const float4 a = *reinterpret_cast<const float4*>(row + c0);
  const float4 b = *reinterpret_cast<const float4*>(row + c1);
  f.v[0] = a.x; f.v[1] = a.y; f.v[2] = a.z; f.v[3] = a.w;
  f.v[4] = b.x; f.v[5] = b.y; f.v[6] = b.z; f.v[7] = b.w;
}
// The same from an fp32 row, converted to the fragment's element type.
__device__ __forceinline__ void load_row2_f32(Frag<bf16_t>& f, const float* row, int c0, int c1) {
  const float4 a = *reinterpret_cast<const float4*>(row + c0);
  const float4 b = *reinterpret_cast<const float4*>(row + c1);
  const float x[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
  f.set8(x);
}
__device__ __forceinline__ void load_row2_f32(Frag<float>& f, const float* row, int c0, int c1) {
  load_row2(f, row, c0, c1);
}

// Raw buffer loads: a descriptor (base, size in bytes) in scalar registers
// and a 32-bit byte offset per lane.  A read at or beyond the size returns 0
// without a memory access, so a load that may not be needed is issued
// unconditionally with offset kOOB: no branch around it, and the compiler's
// memory-counter waits stay exact.
typedef __amdgpu_buffer_rsrc_t brsrc_t;
constexpr uint32_t kOOB = 0x80000000u;
__device__ __forceinline__ brsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, int(bytes), 0x00020000);
}
__device__ __forceinline__ uint4 bload16(brsrc_t r, uint32_t off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
__device__ __forceinline__ float4 bload_f4(brsrc_t r, uint32_t off) {
  return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
__device__ __forceinline__ float bload_f(brsrc_t r, uint32_t off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}
// Non-temporal loads (cache policy nt): for data that will not be read
// again while it could still be cached, such as a decode unit's window tiles
// and state rows when the whole state blob is far larger than the 256 MB
// Infinity Cache; they would otherwise displace reused lines (Wf, the pending
// tokens).  Measured on the batch-32 32K-context stack (5.3 GB of state):
// 907 -> 840 us per decode step.  A blob that fits the cache is re-read from
// it on the next step, and plain loads keep it there (the batch-1 8K stack,
// 77 MB: 22.4 us per step with plain loads, 23.0 with non-temporal ones).
constexpr int kNonTemporal = 2;
constexpr int64_t kStreamingStateBytes = int64_t(128) << 20;
__device__ __forceinline__ void bload_frag_nt(Frag<bf16_t>& f, brsrc_t r, uint32_t off) {
  f.v = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kNonTemporal));
}
__device__ __forceinline__ void bload_frag_nt(Frag<float>& f, brsrc_t r, uint32_t off) {
  const float4 a = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kNonTemporal));
  const float4 b = __builtin_bit_cast(
      float4, __builtin_amdgcn_raw_buffer_load_b128(r, off == kOOB ? kOOB : off + 16, 0, kNonTemporal));
  f.v[0] = a.x; f.v[1] = a.y; f.v[2] = a.z; f.v[3] = a.w;
  f.v[4] = b.x; f.v[5] = b.y; f.v[6] = b.z; f.v[7] = b.w;
}
__device__ __forceinline__ float4 bload_f4_nt(brsrc_t r, uint32_t off) {
  return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kNonTemporal));
}
// Non-temporal when NT, plain otherwise (the cache policy is an immediate).
template <bool NT, typename T>
__device__ __forceinline__ void bload_frag_s(Frag<T>& f, brsrc_t r, uint32_t off) {
  if constexpr (NT) bload_frag_nt(f, r, off);
  else bload_frag(f, r, off);
}
template <bool NT>
__device__ __forceinline__ float4 bload_f4_s(brsrc_t r, uint32_t off) {
  if constexpr (NT) return bload_f4_nt(r, off);
  else return bload_f4(r, off);
}

// System-coherent access (cache policy sc0 sc1): stores are written through
// to memory and loads are served from memory, not from a cache that may hold
// an older copy.  For data one workgroup writes and another, possibly on
// another XCD (each XCD has its own L2), reads within the same kernel.
constexpr int kSysCoherent = 1 | 16;
__device__ __forceinline__ float bload_f_sys(brsrc_t r, uint32_t off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kSysCoherent));
}
__device__ __forceinline__ void bstore_f_sys(brsrc_t r, uint32_t off, float x) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, x), r, off, 0, kSysCoherent);
}
__device__ __forceinline__ bf16_t bload_elem(brsrc_t r, uint32_t off, bf16_t) {
  return bf16_t(__builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0));
}
__device__ __forceinline__ float bload_elem(brsrc_t r, uint32_t off, float) { return bload_f(r, off); }
// One element, raw, zero-extended into its own 32-bit register (bf16 bits
// or fp32 bits), converted with raw_to_f32 where it is used.
__device__ __forceinline__ uint32_t bload_raw(brsrc_t r, uint32_t off, bf16_t) {
  return uint32_t(__builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0));
}
__device__ __forceinline__ uint32_t bload_raw(brsrc_t r, uint32_t off, float) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
}
__device__ __forceinline__ float raw_to_f32(uint32_t x, bf16_t) { return __uint_as_float(x << 16); }
__device__ __forceinline__ float raw_to_f32(uint32_t x, float) { return __uint_as_float(x); }
// Fragment loads through a descriptor: 8 consecutive elements at byte offset off.
__device__ __forceinline__ void bload_frag(Frag<bf16_t>& f, brsrc_t r, uint32_t off) { f.v = bload16(r, off); }
__device__ __forceinline__ void bload_frag(Frag<float>& f, brsrc_t r, uint32_t off) {
  const float4 a = bload_f4(r, off), b = bload_f4(r, off == kOOB ? kOOB : off + 16);
  f.v[0] = a.x; f.v[1] = a.y; f.v[2] = a.z; f.v[3] = a.w;
  f.v[4] = b.x; f.v[5] = b.y; f.v[6] = b.z; f.v[7] = b.w;
}
// 8 elements at byte offsets off, off + stride, ...  (kOOB: zeros)
__device__ __forceinline__ void bload_frag_strided(Frag<bf16_t>& f, brsrc_t r, uint32_t off, uint32_t stride) {
  uint16_t e[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) e[i] = uint16_t(__builtin_amdgcn_raw_buffer_load_b16(r, off + i * stride, 0, 0));
  f.v.x = uint32_t(e[0]) | (uint32_t(e[1]) << 16);
  f.v.y = uint32_t(e[2]) | (uint32_t(e[3]) << 16);
  f.v.z = uint32_t(e[4]) | (uint32_t(e[5]) << 16);
  f.v.w = uint32_t(e[6]) | (uint32_t(e[7]) << 16);
}
__device__ __forceinline__ void bload_frag_strided(Frag<float>& f, brsrc_t r, uint32_t off, uint32_t stride) {
#pragma unroll
  for (int i = 0; i < 8; ++i) f.v[i] = bload_f(r, off + i * stride);
}
__device__ __forceinline__ Frag<bf16_t> frag_or(const Frag<bf16_t>& a, const Frag<bf16_t>& b) {
  Frag<bf16_t> r;
  r.v = make_uint4(a.v.x | b.v.x, a.v.y | b.v.y, a.v.z | b.v.z, a.v.w | b.v.w);
  return r;
}
__device__ __forceinline__ Frag<float> frag_or(const Frag<float>& a, const Frag<float>& b) {
  Frag<float> r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r.v[i] = __uint_as_float(__float_as_uint(a.v[i]) | __float_as_uint(b.v[i]));
  return r;
}
// The same LDS address, opaque to the compiler.  Taken at the start of a
// phase, it keeps that phase's accesses to one base register per array plus
// constants carried in the instructions' 16-bit offset field.  (Constants
// counted from the start of an LDS allocation over 64 KiB do not fit that
// field: each then takes a register of its own, computed once and kept live,
// or spilled, across the whole kernel.)
template <typename P>
__device__ __forceinline__ P* lds_fresh(P* p) {
  uint32_t a = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) P*)p));
  asm volatile("" : "+s"(a));
  return (P*)((__attribute__((address_space(3))) P*)(uintptr_t)a);
}

// The same wave-uniform pointer, opaque to the compiler: per-lane addresses
// derived from it after this point are computed there, not hoisted from a
// loop and kept live (or spilled) across it.
template <typename P>
__device__ __forceinline__ P* sfresh(P* p) {
  // through the global address space, so that accesses stay global (not flat)
  auto q = (__attribute__((address_space(1))) P*)p;
  asm volatile("" : "+s"(q));
  return (P*)q;
}

// Max / sum over the 4 lanes that share lane % 16 (the lane groups of an
// MFMA fragment), with the gfx950 row-swap permutes (no LDS round trip):
// permlane16_swap pairs rows (0,1), (2,3); permlane32_swap pairs the halves.
// Wave-uniform control flow only (every lane active).
__device__ __forceinline__ float lg_max(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float lg_sum(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// a if keep, else zeros: a select on registers (taken where the value is
// used), not a branch around the load that produced a.
__device__ __forceinline__ Frag<bf16_t> frag_keep(const Frag<bf16_t>& a, bool keep) {
  Frag<bf16_t> r;
  r.v = make_uint4(keep ? a.v.x : 0u, keep ? a.v.y : 0u, keep ? a.v.z : 0u, keep ? a.v.w : 0u);
  return r;
}
__device__ __forceinline__ Frag<float> frag_keep(const Frag<float>& a, bool keep) {
  Frag<float> r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r.v[i] = keep ? a.v[i] : 0.f;
  return r;
}

// Streaming 16-byte store (non-temporal: the line is not kept in the caches).
__device__ __forceinline__ void store_nt(float* p, float4 v) {
  __builtin_nontemporal_store(f32x4_t{v.x, v.y, v.z, v.w}, reinterpret_cast<f32x4_t*>(p));
}

// ---------------------------------------------------------------------------
// Launch descriptors.

struct DecodeArgs {
  char* state;
  float* part;       // partial records [workgroup][G][2d+3] (split layers only)
  const void* phi_w;
  const void* q;
  const void* k;
  const void* v;
  void* out;
  int32_t B, Hq, Hkv, G;
  int32_t linear;
  float tau;
  int32_t n_layers;  // layers in this launch (<= kMaxLayersPerLaunch)
  int32_t form;      // 0: shared denominator; 1, 2: the Appendix's hybrid forms (2: state over every token)
  int32_t phi;       // feature map: 0 ReLU, 1 ELU + 1
  int32_t row_stride;  // workgroups per piece row: B * Hkv
  int32_t gated;       // GLIDE_GATED: log_gates [layer][B][Hkv] fp32, gate sections in the state
  const float* gates;
  int32_t wf_heads;  // 1: phi_w holds one Wf per KV head ([layer][Hkv][d][Df])
  int32_t state_tiles;  // the state pass's weight in window tiles for the shares of split windows
  LayerArg layers[kMaxLayersPerLaunch];  // sorted by decreasing W
  // layer (index into layers) of every piece row: workgroup w of the main
  // pass belongs to layer piece_layer[w / row_stride].  The rows of every
  // layer's piece 0 (the state pass, the longest chain) come first, so their
  // loads are issued, and served, first.
  uint8_t piece_layer[kMaxLayersPerLaunch * kMaxPieces];
};

// Host-side launchers (one translation unit per kernel family).
// total_wg: workgroups of the main pass; merge: some layer is split.
// streaming: the state blob is far larger than the Infinity Cache (window
// tiles and state rows read with non-temporal loads)
hipError_t launch_decode(const DecodeArgs& a, int total_wg, int d, int Df, int dtype, bool streaming,
                         hipStream_t stream);
hipError_t launch_flush(const DecodeArgs& a, int d, int Df, int dtype, hipStream_t stream);
hipError_t launch_phi_rows(const void* Wf, const void* x, int64_t rows, void* out, int d, int Df, int dtype,
                           bool out_f32, int phi, hipStream_t stream);

// ---------------------------------------------------------------------------
// Prefill.  Sequences are processed in groups of at most kMaxSeqPerLaunch so
// the per-sequence tables travel in the kernel arguments.
constexpr int kMaxSeqPerLaunch = 128;

// Layers are batched: every prefill kernel takes up to kMaxLayersPerLaunch
// layers in one launch (the grid's last dimension), each with a workspace
// slot of its own, within kPrefillWsBudget bytes of workspace.
constexpr size_t kPrefillWsBudget = size_t(1) << 30;

struct PrefillLayer {
  int64_t layer_base;  // byte offset of the layer in the state blob
  int32_t W, R;
  int32_t li;          // position of the layer in the call (inputs, outputs and Wf at li strides)
  int32_t pad;
};

struct PrefillArgs {
  char* state;
  const char* q;        // [n][T][Hq][d]   the call's inputs (layer li at li * q_stride bytes)
  const char* k;        // [n][T][Hkv][d]  (kv_stride)
  const char* v;        // [n][T][Hkv][d]  (kv_stride)
  char* out;            // [n][T][Hq][d]   (q_stride)
  const char* wf;       // [n][d][Df], or [n][Hkv][d][Df] (wf_stride; head stride wf_hs)
  int64_t q_stride, kv_stride, wf_stride;
  char* ws;             // workspace: slot ls at ls * ws_slot bytes; per slot
  int64_t ws_slot;      //   history keys [B][Hkv][Wcap][d] at 0, history values at ws_hv,
  int64_t ws_hv, ws_seg;  // per (segment, KV head) S [Df][d] then z [Df] at ws_seg
  int32_t B, Hq, Hkv, G;
  int32_t linear;
  float tau;
  int32_t C;            // chunk tokens (multiple of 32)
  int32_t seg_len;      // segment tokens (multiple of C)
  int32_t Wcap;         // history capacity per (sequence, KV head)
  int32_t nseq;         // sequences in this group
  int32_t seq0;         // first sequence of the group
  int32_t seg0;         // first segment record of the group
  int32_t nseg;         // segments in this group
  int32_t nlayer;       // layers in this launch
  int32_t form;         // 0: shared denominator; 1, 2: the Appendix's hybrid forms (2: state over every token)
  int32_t wf_hs;        // bytes between the KV heads' Wf (0: one Wf per layer)
  int32_t pad1;
  int32_t phi;          // feature map: 0 ReLU, 1 ELU + 1
  int32_t gated;        // GLIDE_GATED: log_gates [n][T][Hkv] fp32 (layer li at li * g_stride floats)
  int32_t pad2;
  const float* gates;
  int64_t g_stride;
  int64_t ws_hg, ws_gc;  // per slot: history G [B][Hkv][Wcap] fp64, new tokens' G [T][Hkv] fp64
  PrefillLayer layers[kMaxLayersPerLaunch];  // the launch's layers, by decreasing window
  int32_t seq_start[kMaxSeqPerLaunch];     // packed row of the sequence's first new token
  int32_t seq_len[kMaxSeqPerLaunch];       // new tokens of the sequence
  int32_t seg_base[kMaxSeqPerLaunch + 1];  // first segment (within the group) of the sequence
};
static_assert(sizeof(PrefillArgs) <= 4096, "kernel argument block");

// Segments hold at least kMinSegTokens tokens, which bounds the records.
constexpr int kMinSegTokens = 128;

// Chunks per prefill segment, for a launch of nl layers: at least
// kMinSegTokens tokens, and about kSegRounds workgroups per CU over the
// launch's (segment, KV head, layer) grid when the call is large enough
// (longer segments amortise each workgroup's start, the state load, over
// more chunks; several rounds keep the CUs evenly loaded across layers of
// different windows); at most 16 chunks walked in order by one workgroup.
// More layers per launch never give shorter segments, so the workspace's
// record bound, taken at nl = 1, holds for every launch.
constexpr int kSegRounds = 8;
inline int32_t segment_chunks(int64_t T, int Hkv, int32_t chunk, int32_t nl) {
  const int32_t lo = (kMinSegTokens + chunk - 1) / chunk;
  const int64_t fill = T * Hkv * nl / (int64_t(chunk) * 256 * kSegRounds);
  return int32_t(fill > lo ? (fill < 16 ? fill : 16) : lo);
}

struct PrefillWorkspace {
  size_t hk, hv, seg, hg, gc, slot;  // offsets within a slot, and the slot's bytes
};

// One layer's slot for calls of T tokens in launches of nl layers: the
// records bound takes the shortest segment any legal chunk gives for T.
// Gated: the history tokens' and the new tokens' cumulative log-gates (fp64).
inline PrefillWorkspace prefill_workspace(int64_t T, int B, int Hkv, int d, int Df, int esize, int Wcap,
                                          bool linear, int32_t nl, bool gated = false) {
  PrefillWorkspace w;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += size_t(align256(int64_t(bytes)));
    return o;
  };
  int64_t seg_min = INT64_MAX;
  for (int32_t c = 32; c <= 256; c += 32) {
    const int64_t sl = int64_t(c) * segment_chunks(T, Hkv, c, nl);
    seg_min = sl < seg_min ? sl : seg_min;
  }
  w.hk = take(size_t(B) * Hkv * Wcap * d * esize);
  w.hv = take(size_t(B) * Hkv * Wcap * d * esize);
  w.seg = take(linear ? (size_t(T / seg_min) + B) * Hkv * (size_t(Df) * d + Df) * 4 : 0);
  w.hg = take(gated ? size_t(B) * Hkv * Wcap * 8 : 0);
  w.gc = take(gated ? size_t(T) * Hkv * 8 : 0);
  w.slot = off;
  return w;
}

// Layers per launch for a workspace of `bytes`: the most layers nl (up to
// kMaxLayersPerLaunch and n_layers) whose nl slots, sized for launches of nl
// layers, fit; 0 if not even one layer's slot fits.
template <typename SlotFn>
inline int32_t prefill_layers_per_launch(int32_t n_layers, size_t bytes, SlotFn slot_of) {
  int32_t n = n_layers < kMaxLayersPerLaunch ? n_layers : kMaxLayersPerLaunch;
  for (; n >= 1; --n)
    if (size_t(n) * slot_of(n) <= bytes) return n;
  return 0;
}

hipError_t launch_prefill_layer(const PrefillArgs& a, int d, int Df, int dtype, hipStream_t stream);
hipError_t launch_prefill_gather(const PrefillArgs& a, int d, int Df, int dtype, hipStream_t stream);
hipError_t launch_prefill_ringfill(const PrefillArgs& a, int d, int Df, int dtype, hipStream_t stream);

}  // namespace glide
