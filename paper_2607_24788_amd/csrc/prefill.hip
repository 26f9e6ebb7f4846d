// GLIDE chunked prefill (kernel c), one layer at a time.
//
// For query t (0-indexed position) with window W the layer needs
//   softmax over keys [t-W+1, t]  and  the linear part over keys [0, t-W],
// merged over one denominator (GLIDE Sec. III-B).  In chunked form the linear
// part is causal linear attention on keys delayed by W: a chunk of queries
// [t0, t0+C) sees the state S_c = sum_{j < t0-W} phi(k_j)^T v_j plus, for its
// query t0+i, the delayed keys t0-W .. t0-W+i (an inclusive lower-triangular
// block), and S_{c+1} = S_c + the sum over the chunk's C delayed keys.
//
// Kernels (per layer):
//   gather   ring tokens [max(0,p0-W), p0) of a continuing prefill into a
//            natural-layout side buffer (the "history");
//   segsum   per (sequence, KV head, segment of chunks): the segment's state
//            increment from its delayed keys (MFMA, keys as the reduction);
//   scan     exclusive prefix over segments on top of the incoming state;
//            its end is the new S, z;
//   main     per (segment, KV head): the segment's chunks in order, S_c kept
//            in LDS in fp32.  Per pass of 256 query rows: first the banded
//            window attention over LDS-staged key tiles on MFMA (online
//            softmax, running max m per row); then the linear part, phi(q) on
//            MFMA, the read-out phi(Q)S_c, phi(q).z_c and the masked block of
//            the chunk's delayed keys (whose phi(k) is computed once and also
//            feeds S_{c+1}), all scaled by 2^-m so that they add straight
//            onto the band's numerator and denominator (the shared-denominator
//            merge, in the band's frame);
//   ringfill the last W tokens into the ring;   advance: pos += T_b.
// Tokens a decode step left pending are folded (glide_state_flush) before the
// first of these kernels runs, so the incoming state is S = sum_{j < p0-W}.
//
// The feature map phi(x) = max(0, x Wf) is evaluated where it is needed, on
// MFMA against Wf.  phi(q) is produced transposed (features as MFMA rows),
// which hands every lane features {32s+4g .. 32s+4g+3, 32s+16+4g .. +3} of its
// query row for lane group g and feature slab s: that permuted order of the
// reduction index is used, identically, by every operand it meets (S_c, z_c
// and the delayed keys' phi(k)).
#include <math.h>

#include "glide_internal.h"

namespace glide {

namespace {

constexpr int kThreads = 256;  // helper kernels
constexpr int kWaves = 4;
constexpr int kRB = 256;       // main kernel: query rows per pass of a chunk
constexpr float kLog2e = 1.4426950408889634f;

// Rows of one (sequence, KV head) of a layer: new tokens come from the
// packed inputs, older tokens from the history side buffer (stride Wcap).
template <typename T, int D>
struct SeqRows {
  const T *kin, *vin, *kh, *vh;  // inputs of the layer, then this unit's history
  int Hq, Hkv, G, start;
  int b, g;
  int64_t p0, h0;

  __device__ const T* k(int64_t j) const {
    if (j >= p0) return kin + ((int64_t(start) + (j - p0)) * Hkv + g) * D;
    if (j >= h0) return kh + (j - h0) * D;
    return nullptr;
  }
  __device__ const T* v(int64_t j) const {
    if (j >= p0) return vin + ((int64_t(start) + (j - p0)) * Hkv + g) * D;
    if (j >= h0) return vh + (j - h0) * D;
    return nullptr;
  }
  // packed query row of new token i (0-based within the call) and head hh of the group
  __device__ int64_t qrow(int i, int hh) const { return (int64_t(start) + i) * Hq + int64_t(g) * G + hh; }
};

// Layer slot ls of the launch: its window, ring, state section, inputs,
// outputs and workspace slot.
struct LayerView {
  char* base;  // the layer's sections in the state blob
  int32_t W, R;
  int32_t Wd;  // the linear part's delay: W, or 0 when the state holds every token
  const void *q, *k, *v, *wf;
  void* out;
  void *hk, *hv;
  float* seg;
  int ls;      // slot of the layer within the launch
  int li;      // position of the layer in the call
};
__device__ __forceinline__ LayerView layer_view(const PrefillArgs& a, int ls) {
  const PrefillLayer& L = a.layers[ls];
  LayerView v;
  v.base = a.state + L.layer_base;
  v.W = L.W;
  v.R = L.R;
  v.Wd = a.form == 2 ? 0 : L.W;
  v.q = a.q + int64_t(L.li) * a.q_stride;
  v.out = a.out + int64_t(L.li) * a.q_stride;
  v.k = a.k + int64_t(L.li) * a.kv_stride;
  v.v = a.v + int64_t(L.li) * a.kv_stride;
  v.wf = a.wf + int64_t(L.li) * a.wf_stride;
  char* slot = a.ws + int64_t(ls) * a.ws_slot;
  v.hk = slot;
  v.hv = slot + a.ws_hv;
  v.seg = reinterpret_cast<float*>(slot + a.ws_seg);
  v.ls = ls;
  v.li = L.li;
  return v;
}

template <typename T, int D, int DF>
__device__ __forceinline__ SeqRows<T, D> seq_rows(const PrefillArgs& a, const LayerView& L, int bl, int g) {
  SeqRows<T, D> r;
  r.b = a.seq0 + bl;
  r.g = g;
  r.start = a.seq_start[bl];
  r.Hq = a.Hq;
  r.Hkv = a.Hkv;
  r.G = a.G;
  const int64_t unit = int64_t(r.b) * a.Hkv + g;
  r.kin = static_cast<const T*>(L.k);
  r.vin = static_cast<const T*>(L.v);
  r.kh = static_cast<const T*>(L.hk) + unit * a.Wcap * D;
  r.vh = static_cast<const T*>(L.hv) + unit * a.Wcap * D;
  const LayerSections sec = layer_sections(a.B, a.Hkv, D, DF, L.R, sizeof(T));
  r.p0 = reinterpret_cast<const int64_t*>(L.base + sec.pos)[unit];
  r.h0 = r.p0 - L.W > 0 ? r.p0 - L.W : 0;
  return r;
}

// Cumulative log-gates G_j of a gated prefill (GLIDE_GATED): those of the new
// tokens from this call's scan (gc [T][Hkv], workspace), those of the history
// tokens from their copy of the gate ring (hg), and G_{p0-1}, the state's G at
// the call's start (the reference its incoming S, z are decayed to).
struct SeqGates {
  const double *gc, *hg;
  double g0;
  int64_t p0, h0;
  int start, Hkv, g;
  __device__ double at(int64_t j) const {
    if (j >= p0) return gc[(int64_t(start) + (j - p0)) * Hkv + g];
    if (j == p0 - 1 || j < h0) return g0;
    return hg[j - h0];
  }
};
template <typename T, int D, int DF>
__device__ __forceinline__ SeqGates seq_gates(const PrefillArgs& a, const LayerView& L, const SeqRows<T, D>& sr) {
  SeqGates q;
  char* slot = a.ws + int64_t(L.ls) * a.ws_slot;
  const int64_t unit = int64_t(sr.b) * a.Hkv + sr.g;
  q.gc = reinterpret_cast<const double*>(slot + a.ws_gc);
  q.hg = reinterpret_cast<const double*>(slot + a.ws_hg) + unit * a.Wcap;
  const LayerSections sec = layer_sections(a.B, a.Hkv, D, DF, L.R, sizeof(T), true);
  q.g0 = reinterpret_cast<const double*>(L.base + sec.G)[2 * unit];
  q.p0 = sr.p0;
  q.h0 = sr.h0;
  q.start = sr.start;
  q.Hkv = a.Hkv;
  q.g = sr.g;
  return q;
}

// Sequence (within the group) owning segment sg.
__device__ __forceinline__ int find_seq(const PrefillArgs& a, int sg) {
  int bl = 0;
  while (bl + 1 < a.nseq && a.seg_base[bl + 1] <= sg) ++bl;
  return bl;
}

__device__ __forceinline__ void store8(bf16_t* dst, const Frag<bf16_t>& f) { *reinterpret_cast<uint4*>(dst) = f.v; }
__device__ __forceinline__ void store8(float* dst, const Frag<float>& f) {
  reinterpret_cast<float4*>(dst)[0] = make_float4(f.v[0], f.v[1], f.v[2], f.v[3]);
  reinterpret_cast<float4*>(dst)[1] = make_float4(f.v[4], f.v[5], f.v[6], f.v[7]);
}


// LDS row strides (elements): tiles read with 16-byte fragment loads use a
// padding of 8; tiles read with load_colfrag use 16 so the four rows a
// 16-lane group touches fall on distinct banks.
template <int N> constexpr int row_a() { return N + 8; }
template <int N> constexpr int row_t() { return N + 16; }

// Columns of Wf [D][DF] as MFMA fragments (rows d = 32kk + 8g .. +7 of column
// col0 + lane%16): from a natural LDS copy, or (fp32, where the copy would not
// fit next to the rest) from global memory.
template <typename T, int D, int DF, bool kLds>
struct WfCols {
  const T* src;  // kLds: LDS [D][row_t<DF>]; else global [D][DF]
  __device__ __forceinline__ void col(Frag<T>& f, int kk, int col0) const {
    const int lane = threadIdx.x & 63, hq = lane & 15, lg = lane >> 4;
    if constexpr (kLds) load_colfrag(f, src, row_t<DF>(), 32 * kk + 8 * lg, col0);
    else f.load_strided(src + (32 * kk + 8 * lg) * DF + col0 + hq, DF);
  }
};

// 4 consecutive outputs (scaled) in one store: 8 bytes (bf16) or 16 (fp32).
__device__ __forceinline__ void store4(bf16_t* dst, f32x4_t x, float s) {
  *reinterpret_cast<uint2*>(dst) = make_uint2(pack_bf16x2(x[0] * s, x[1] * s), pack_bf16x2(x[2] * s, x[3] * s));
}
__device__ __forceinline__ void store4(float* dst, f32x4_t x, float s) {
  *reinterpret_cast<float4*>(dst) = make_float4(x[0] * s, x[1] * s, x[2] * s, x[3] * s);
}
// dst[0..3] += x * s (the second pass of a hybrid-form prefill)
__device__ __forceinline__ void add4(bf16_t* dst, f32x4_t x, float s) {
  const uint2 o = *reinterpret_cast<const uint2*>(dst);
  const float y0 = __uint_as_float(o.x << 16) + x[0] * s, y1 = __uint_as_float(o.x & 0xffff0000u) + x[1] * s;
  const float y2 = __uint_as_float(o.y << 16) + x[2] * s, y3 = __uint_as_float(o.y & 0xffff0000u) + x[3] * s;
  *reinterpret_cast<uint2*>(dst) = make_uint2(pack_bf16x2(y0, y1), pack_bf16x2(y2, y3));
}
__device__ __forceinline__ void add4(float* dst, f32x4_t x, float s) {
  float4 o = *reinterpret_cast<const float4*>(dst);
  o.x += x[0] * s; o.y += x[1] * s; o.z += x[2] * s; o.w += x[3] * s;
  *reinterpret_cast<float4*>(dst) = o;
}
__device__ __forceinline__ f32x4_t act4(f32x4_t x, int phi) {
  return f32x4_t{feat_act(x[0], phi), feat_act(x[1], phi), feat_act(x[2], phi), feat_act(x[3], phi)};
}

// Wf [D][DF] into LDS, natural layout (NTH threads cooperating; every load
// is issued before the first store).
template <typename T, int D, int DF, int NTH>
__device__ __forceinline__ void stage_wf(const T* Wf, T* Wn) {
  constexpr int WROW = row_t<DF>(), N = D * DF / 8 / NTH;
  static_assert(N * NTH == D * DF / 8, "even split");
  Frag<T> f[N];
#pragma unroll
  for (int u = 0; u < N; ++u) {
    const int i = threadIdx.x + u * NTH, r = i / (DF / 8), ch = i - r * (DF / 8);
    f[u].load(Wf + r * DF + 8 * ch);
  }
#pragma unroll
  for (int u = 0; u < N; ++u) {
    const int i = threadIdx.x + u * NTH, r = i / (DF / 8), ch = i - r * (DF / 8);
    store8(Wn + r * WROW + 8 * ch, f[u]);
  }
}

// phi of NK keys (16 per key tile) into LDS pk[NK][row_t<DF>] (element type,
// natural layout).  The NK/16 x DF/16 output tiles are spread over the NW
// waves of the workgroup so that every tile of a wave has the same key tile
// (slab_key_tile): phi_slab takes that tile's key rows as A fragments x
// (rows that do not exist are zeros).
template <int D, int DF, int NK>
__device__ __forceinline__ int slab_key_tile(int nw) {
  constexpr int FT = DF / 16;
  return (int(threadIdx.x >> 6) * ((NK / 16) * FT / nw)) / FT;
}
template <typename T, int D, int DF>
struct SlabKeys {
  Frag<T> x[D / 32];
  bool ok;  // the lane's key row exists (else it counts as zeros)
};
// kw: the weight of the lane's key row (16 kt + hq) multiplied into its
// features (a gated segment's decay; 1 otherwise).
template <typename T, int D, int DF, int NK, int PHI, int NW, bool kLds>
__device__ __forceinline__ void phi_slab(const WfCols<T, D, DF, kLds>& wf, const Frag<T> (&x)[D / 32], T* pk,
                                         int rlo, int rhi, float kw = 1.f) {
  constexpr int KS = D / 32, FT = DF / 16, PROW = row_t<DF>();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, hq = lane & 15, lg = lane >> 4;
  constexpr int per = (NK / 16) * FT / NW;
  static_assert(per >= 1 && per * NW == (NK / 16) * FT, "phi tiles must spread evenly over the waves");
  if constexpr (PHI == GLIDE_PHI_SOFTMAX) {
    // The softmax map needs each key row's max and sum over all DF features;
    // the row's feature tiles are spread over WPK = FT / per waves (per <= 4
    // tiles each, one key tile per wave).  Each wave reduces its part (its
    // lanes, then the row's 4 lane groups), the parts meet in the 16 spare
    // elements at the end of the row, two barriers apart.
    constexpr int kPerMax = per;
    static_assert(FT % per == 0 && FT / per <= 4, "a row's parts fit the row's spare elements");
    const int kt = (wave * per) / FT, ft0 = (wave * per) % FT, wk = ft0 / per, WPK = FT / per;
    const int key = 16 * kt + hq;
    f32x4_t acc[kPerMax];
    float m = -INFINITY;
#pragma unroll
    for (int u = 0; u < kPerMax; ++u) {
      acc[u] = zero4();
      if (u < per) {
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) {
          Frag<T> wb;
          wf.col(wb, kk, 16 * (ft0 + u));
          acc[u] = mma(wb, x[kk], acc[u]);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) m = fmaxf(m, acc[u][i]);
      }
    }
    m = fmaxf(m, __shfl_xor(m, 16));
    m = fmaxf(m, __shfl_xor(m, 32));
    char* pad = reinterpret_cast<char*>(pk + key * PROW + DF);  // [0, 4): maxima, [4, 8): sums (floats)
    if (lg == 0) __builtin_memcpy(pad + 4 * wk, &m, 4);
    __syncthreads();
    float M = -INFINITY;
    for (int w = 0; w < WPK; ++w) {
      float t;
      __builtin_memcpy(&t, pad + 4 * w, 4);
      M = fmaxf(M, t);
    }
    float sum = 0.f;
#pragma unroll
    for (int u = 0; u < kPerMax; ++u)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        acc[u][i] = u < per ? __builtin_amdgcn_exp2f((acc[u][i] - M) * 1.4426950408889634f) : 0.f;
        sum += acc[u][i];
      }
    sum += __shfl_xor(sum, 16);
    sum += __shfl_xor(sum, 32);
    if (lg == 0) __builtin_memcpy(pad + 16 + 4 * wk, &sum, 4);
    __syncthreads();
    float tot = 0.f;
    for (int w = 0; w < WPK; ++w) {
      float t;
      __builtin_memcpy(&t, pad + 16 + 4 * w, 4);
      tot += t;
    }
    const bool is_key = key >= rlo && key < rhi;
#pragma unroll
    for (int u = 0; u < kPerMax; ++u)
      if (u < per) store4(pk + key * PROW + 16 * (ft0 + u) + 4 * lg, is_key ? acc[u] : zero4(), kw / tot);
    return;
  }
  // transposed (Wf^T K^T): lane (hq, lg) gets features 16ft+4lg .. +3 of
  // key 16kt+hq, one 4-element store per tile.  The wave's tiles share the
  // key tile; their Wf fragments are read one reduction step at a time for
  // all tiles, so the tiles' MFMA chains interleave.
  f32x4_t acc[per];
#pragma unroll
  for (int u = 0; u < per; ++u) acc[u] = zero4();
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    Frag<T> wb[per];
#pragma unroll
    for (int u = 0; u < per; ++u) wf.col(wb[u], kk, 16 * ((wave * per + u) % FT));
#pragma unroll
    for (int u = 0; u < per; ++u) acc[u] = mma(wb[u], x[kk], acc[u]);
  }
#pragma unroll
  for (int u = 0; u < per; ++u) {
    const int tile = wave * per + u, kt = tile / FT, ft = tile - kt * FT;
    // rows outside [rlo, rhi) are no keys (zero rows): their features must
    // be 0, which ReLU gives by itself and ELU + 1 (phi(0) = 1) does not
    const int key = 16 * kt + hq;
    if constexpr (PHI == 0) {
      store4(pk + key * PROW + 16 * ft + 4 * lg, act4(acc[u], 0), kw);
    } else {
      store4(pk + key * PROW + 16 * ft + 4 * lg, key >= rlo && key < rhi ? act4(acc[u], PHI) : zero4(), kw);
    }
  }
}

// ---------------------------------------------------------------------------
// gather: history tokens [h0, p0) of a continuing prefill, ring -> [b][g][Wcap][d]
template <typename T, int D, int DF>
__global__ __launch_bounds__(kThreads) void prefill_gather(PrefillArgs a) {
  const int bl = blockIdx.y, g = int(blockIdx.z) % a.Hkv;
  const LayerView L = layer_view(a, int(blockIdx.z) / a.Hkv);
  if (L.W == 0) return;
  const SeqRows<T, D> sr = seq_rows<T, D, DF>(a, L, bl, g);
  const int n = int(sr.p0 - sr.h0);
  if (n <= 0) return;
  const LayerSections sec = layer_sections(a.B, a.Hkv, D, DF, L.R, sizeof(T));
  const int64_t unit = int64_t(sr.b) * a.Hkv + g;
  const T* Kr = reinterpret_cast<const T*>(L.base + sec.K) + unit * L.R * D;
  const T* Vr = reinterpret_cast<const T*>(L.base + sec.V) + unit * L.R * D;
  T* hk = static_cast<T*>(L.hk) + unit * a.Wcap * D;
  T* hv = static_cast<T*>(L.hv) + unit * a.Wcap * D;
  for (int idx = blockIdx.x * kThreads + threadIdx.x; idx < n * D; idx += gridDim.x * kThreads) {
    const int i = idx / D, c = idx - i * D;
    const int32_t s = int32_t((sr.h0 + i) % L.R);
    hk[int64_t(i) * D + c] = Kr[kring_elem(s, c, D)];
    hv[int64_t(i) * D + c] = Vr[vring_elem(s, c, D)];
  }
  if (a.gated) {  // the history tokens' G_j, from the gate ring
    const LayerSections sg = layer_sections(a.B, a.Hkv, D, DF, L.R, sizeof(T), true);
    const double* grg = reinterpret_cast<const double*>(L.base + sg.GR) + unit * L.R;
    double* hg = reinterpret_cast<double*>(a.ws + int64_t(L.ls) * a.ws_slot + a.ws_hg) + unit * a.Wcap;
    for (int i = blockIdx.x * kThreads + threadIdx.x; i < n; i += gridDim.x * kThreads) hg[i] = grg[(sr.h0 + i) % L.R];
  }
}

// ---------------------------------------------------------------------------
// gates (GLIDE_GATED): the cumulative log-gates of the new tokens of one
// (sequence, KV head), G_t = G_{p0-1} + g_{p0} + ... + g_t, in fp64 (an
// inclusive scan over blocks of consecutive tokens, one block per thread).
template <typename T, int D, int DF>
__global__ __launch_bounds__(kThreads) void prefill_gates(PrefillArgs a) {
  __shared__ double part[kThreads];
  const int bl = blockIdx.x, g = blockIdx.y, tid = threadIdx.x;
  const LayerView L = layer_view(a, blockIdx.z);
  const int Tb = a.seq_len[bl], start = a.seq_start[bl];
  const int64_t unit = int64_t(a.seq0 + bl) * a.Hkv + g;
  const LayerSections sec = layer_sections(a.B, a.Hkv, D, DF, L.R, sizeof(T), true);
  const double g0 = reinterpret_cast<const double*>(L.base + sec.G)[2 * unit];
  const float* gin = a.gates + int64_t(L.li) * a.g_stride;
  double* gc = reinterpret_cast<double*>(a.ws + int64_t(L.ls) * a.ws_slot + a.ws_gc);
  const int per = (Tb + kThreads - 1) / kThreads;
  const int i0 = tid * per, i1 = min(Tb, i0 + per);
  double sum = 0.0;
  for (int i = i0; i < i1; ++i) sum += double(gin[(int64_t(start) + i) * a.Hkv + g]);
  part[tid] = sum;
  __syncthreads();
  if (tid == 0) {
    double run = g0;
    for (int t = 0; t < kThreads; ++t) {
      const double x = part[t];
      part[t] = run;
      run += x;
    }
  }
  __syncthreads();
  double run = part[tid];
  for (int i = i0; i < i1; ++i) {
    run += double(gin[(int64_t(start) + i) * a.Hkv + g]);
    gc[(int64_t(start) + i) * a.Hkv + g] = run;
  }
}

// ---------------------------------------------------------------------------
// segsum: state increment of one segment from its delayed keys
//   dS[f][c] = sum_j phi(k_j)[f] v_j[c],  dz[f] = sum_j phi(k_j)[f],
//   j in [t_lo - W, t_hi - W) and j >= 0, where [t_lo, t_hi) are the segment's queries.
// 8 waves, slabs of 64 keys; each wave owns 1/8 of the dS tiles (registers),
// computed transposed so that a lane holds 4 consecutive columns of one
// feature row (16-byte stores of the record); dz comes from the same phi(k)
// fragments.
constexpr int kSegThreads = 512, kSegWaves = 8, kSegSlab = 64;

template <typename T, int D, int DF>
struct SegLds {
  static constexpr int WROW = row_t<DF>(), PROW = row_t<DF>(), VROW = row_t<D>();
  static constexpr size_t bytes = (size_t(D) * WROW + size_t(kSegSlab) * (PROW + VROW)) * sizeof(T);
};

template <typename T, int D, int DF, int PHI>
__global__ __launch_bounds__(kSegThreads) void prefill_segsum(PrefillArgs a) {
  using LD = SegLds<T, D, DF>;
  constexpr int CT = D / 16, FT = DF / 16, CPR = D / 8;
  constexpr int NT = FT * CT / kSegWaves;                  // dS tiles per wave
  constexpr int VPT = kSegSlab * CPR / kSegThreads;        // value chunks per thread
  constexpr int WROW = LD::WROW, PROW = LD::PROW, VROW = LD::VROW;
  static_assert(NT * kSegWaves == FT * CT && VPT * kSegThreads == kSegSlab * CPR, "even split");
  static_assert(NT <= CT, "at most one ct == 0 tile per wave (it carries dz)");
  __shared__ __align__(16) char smem[LD::bytes];
  T* Wn = reinterpret_cast<T*>(smem);  // [D][WROW]      Wf
  T* pk = Wn + D * WROW;                // [64][PROW]     phi(k) of a slab of delayed keys
  T* vs = pk + kSegSlab * PROW;         // [64][VROW]     their values
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hq = lane & 15, lg = lane >> 4;
  const int sg = blockIdx.x, g = blockIdx.y;
  const LayerView L = layer_view(a, blockIdx.z);
  const int bl = find_seq(a, sg);
  const SeqRows<T, D> sr = seq_rows<T, D, DF>(a, L, bl, g);
  const int sigma = sg - a.seg_base[bl];
  const int s_lo = sigma * a.seg_len, s_hi = min(a.seq_len[bl], s_lo + a.seg_len);
  int64_t jlo = sr.p0 + s_lo - L.Wd;
  const int64_t jhi = sr.p0 + s_hi - L.Wd;
  if (jlo < 0) jlo = 0;
  // gated: each delayed key decayed to the segment's last query (the scan
  // carries the records from one segment's end to the next)
  SeqGates gt{};
  double gend = 0.0;
  if (a.gated) {
    gt = seq_gates<T, D, DF>(a, L, sr);
    gend = gt.at(sr.p0 + s_hi - 1);
  }

  f32x4_t sacc[NT];
#pragma unroll
  for (int x = 0; x < NT; ++x) sacc[x] = zero4();
  float zp = 0.f;  // lanes of ct == 0 tiles: keys 8lg.. of feature 16ft+hq
  // the next slab's key rows and values are loaded while the current one is
  // computed
  SlabKeys<T, D, DF> kx;
  Frag<T> vx[VPT];
  bool vok[VPT];
  // Rows through buffer descriptors with 32-bit byte offsets per lane (the
  // host guarantees a sequence's rows span less than 2 GiB): a row past the
  // segment, or a history row of a slab that has none, reads zeros with no
  // memory access.  New tokens' rows are Hkv * D elements apart; history
  // rows (a continuing prefill) are consecutive.
  const uint32_t rowb = uint32_t(a.Hkv) * D * sizeof(T);
  const brsrc_t rkn = make_rsrc(sr.kin + (int64_t(sr.start) * a.Hkv + g) * D, uint32_t(a.seq_len[bl]) * rowb);
  const brsrc_t rvn = make_rsrc(sr.vin + (int64_t(sr.start) * a.Hkv + g) * D, uint32_t(a.seq_len[bl]) * rowb);
  const int nhist = int(sr.p0 - sr.h0);
  const brsrc_t rkh = make_rsrc(sr.kh, uint32_t(nhist) * D * sizeof(T));
  const brsrc_t rvh = make_rsrc(sr.vh, uint32_t(nhist) * D * sizeof(T));
  // row j (absolute), byte cb of the row: its offset among the new rows
  // and among the history rows (kOOB where it is not one, or not wanted)
  auto offs = [&](int64_t j, uint32_t cb, bool ok, uint32_t& on, uint32_t& oh) {
    const int jr = int(j - sr.p0);
    on = ok && jr >= 0 ? uint32_t(jr) * rowb + cb : kOOB;
    oh = ok && jr < 0 ? uint32_t(jr + nhist) * uint32_t(D * sizeof(T)) + cb : kOOB;
  };
  auto load_slab = [&](int64_t j0) {
    const bool hist = j0 < sr.p0;  // the slab reaches into the history rows (uniform)
    {  // the lane's key row of the slab's key tile (phi_slab's A fragments)
      const int64_t j = j0 + 16 * slab_key_tile<D, DF, kSegSlab>(kSegWaves) + hq;
      kx.ok = j < jhi;
#pragma unroll
      for (int kk = 0; kk < D / 32; ++kk) {
        uint32_t on, oh;
        offs(j, uint32_t((32 * kk + 8 * lg) * sizeof(T)), kx.ok, on, oh);
        bload_frag(kx.x[kk], rkn, on);
        if (hist) {
          Frag<T> h;
          bload_frag(h, rkh, oh);
          kx.x[kk] = frag_or(kx.x[kk], h);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < VPT; ++u) {
      const int id = tid + u * kSegThreads, r = id / CPR, ch = id - r * CPR;
      vok[u] = j0 + r < jhi;
      uint32_t on, oh;
      offs(j0 + r, uint32_t(8 * sizeof(T)) * ch, vok[u], on, oh);
      bload_frag(vx[u], rvn, on);
      if (hist) {
        Frag<T> h;
        bload_frag(h, rvh, oh);
        vx[u] = frag_or(vx[u], h);
      }
    }
  };
  if (jlo < jhi) load_slab(jlo);
  stage_wf<T, D, DF, kSegThreads>(reinterpret_cast<const T*>(static_cast<const char*>(L.wf) + int64_t(g) * a.wf_hs), Wn);
  for (int64_t j0 = jlo; j0 < jhi; j0 += kSegSlab) {
    __syncthreads();  // Wf staged; the previous slab's readers are done
    {
      Frag<T> x[D / 32];
#pragma unroll
      for (int kk = 0; kk < D / 32; ++kk) x[kk] = frag_keep(kx.x[kk], kx.ok);
      const int64_t nrow = jhi - j0;
      float kw = 1.f;
      if (a.gated) {
        const int64_t j = j0 + 16 * slab_key_tile<D, DF, kSegSlab>(kSegWaves) + hq;
        kw = j < jhi ? decay_exp(float(gend - gt.at(j))) : 0.f;
      }
      phi_slab<T, D, DF, kSegSlab, PHI, kSegWaves>(WfCols<T, D, DF, true>{lds_fresh(static_cast<const T*>(Wn))}, x,
                                                   lds_fresh(pk), 0, nrow < kSegSlab ? int(nrow) : kSegSlab, kw);
    }
    {
      T* vw = lds_fresh(vs);
#pragma unroll
      for (int u = 0; u < VPT; ++u) {
        const int id = tid + u * kSegThreads, r = id / CPR, ch = id - r * CPR;
        store8(vw + r * VROW + 8 * ch, frag_keep(vx[u], vok[u]));
      }
    }
    if (j0 + kSegSlab < jhi) load_slab(j0 + kSegSlab);
    __syncthreads();
    const T* pr = lds_fresh(static_cast<const T*>(pk));
    const T* vr = lds_fresh(static_cast<const T*>(vs));
#pragma unroll
    for (int x = 0; x < NT; ++x) {
      const int tile = wave * NT + x, ft = tile / CT, ct = tile - ft * CT;
#pragma unroll
      for (int kh = 0; kh < kSegSlab / 32; ++kh) {
        Frag<T> fv, fp;
        load_colfrag(fv, vr, VROW, 32 * kh + 8 * lg, 16 * ct);
        load_colfrag(fp, pr, PROW, 32 * kh + 8 * lg, 16 * ft);
        sacc[x] = mma(fv, fp, sacc[x]);  // rows c = 16ct+4lg+i, column f = 16ft+hq
        if (ct == 0) zp += fp.sum();
      }
    }
  }
  float* rec = L.seg + (int64_t(a.seg0 + sg) * a.Hkv + g) * (int64_t(DF) * D + DF);
#pragma unroll
  for (int x = 0; x < NT; ++x) {
    const int tile = wave * NT + x, ft = tile / CT, ct = tile - ft * CT;
    *reinterpret_cast<float4*>(rec + (16 * ft + hq) * D + 16 * ct + 4 * lg) =
        make_float4(sacc[x][0], sacc[x][1], sacc[x][2], sacc[x][3]);
  }
  // dz: the owner wave of each feature block's ct == 0 tile
  zp = lg_sum(zp);
#pragma unroll
  for (int x = 0; x < NT; ++x) {
    const int tile = wave * NT + x, ft = tile / CT, ct = tile - ft * CT;
    if (ct == 0 && lg == 0) rec[DF * D + 16 * ft + hq] = zp;
  }
}

// ---------------------------------------------------------------------------
// scan: rec[sigma] <- S_in + sum_{sigma' < sigma} dS_sigma'; state <- total
template <typename T, int D, int DF>
__global__ __launch_bounds__(kThreads) void prefill_scan(PrefillArgs a) {
  constexpr int E = DF * D + DF;
  const int bl = blockIdx.y, g = int(blockIdx.z) % a.Hkv, b = a.seq0 + bl;
  const LayerView L = layer_view(a, int(blockIdx.z) / a.Hkv);
  const int e = 4 * (blockIdx.x * kThreads + threadIdx.x);
  if (e >= E) return;
  const LayerSections sec = layer_sections(a.B, a.Hkv, D, DF, L.R, sizeof(T));
  const int64_t unit = int64_t(b) * a.Hkv + g;
  float* st = e < DF * D ? reinterpret_cast<float*>(L.base + sec.S) + unit * DF * D + e
                         : reinterpret_cast<float*>(L.base + sec.z) + unit * DF + (e - DF * D);
  float4 run = *reinterpret_cast<const float4*>(st);
  auto rec = [&](int sg) { return reinterpret_cast<float4*>(L.seg + (int64_t(a.seg0 + sg) * a.Hkv + g) * E + e); };
  const int s1 = a.seg_base[bl + 1];
  const int sb = a.seg_base[bl];
  int sg = sb;
  // gated: the running state is decayed across each segment, from G at the
  // token before it to G at its last token, before the segment's increment
  // (decayed to that last token) is added
  SeqGates gt{};
  if (a.gated) gt = seq_gates<T, D, DF>(a, L, seq_rows<T, D, DF>(a, L, bl, g));
  const int Tb = a.seq_len[bl];
  auto seg_decay = [&](int sgi) {
    if (!a.gated) return 1.f;
    const int lo = (sgi - sb) * a.seg_len, hi = min(Tb, lo + a.seg_len);
    return decay_exp(float(gt.at(gt.p0 + hi - 1) - gt.at(gt.p0 + lo - 1)));
  };
  // eight records' loads in flight at a time (the sum itself is serial)
  for (; sg + 8 <= s1; sg += 8) {
    float4 d[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) d[u] = *rec(sg + u);
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      *rec(sg + u) = run;
      const float f = seg_decay(sg + u);
      run.x = run.x * f + d[u].x; run.y = run.y * f + d[u].y; run.z = run.z * f + d[u].z; run.w = run.w * f + d[u].w;
    }
  }
  for (; sg < s1; ++sg) {
    const float4 d = *rec(sg);
    *rec(sg) = run;
    const float f = seg_decay(sg);
    run.x = run.x * f + d.x; run.y = run.y * f + d.y; run.z = run.z * f + d.z; run.w = run.w * f + d.w;
  }
  *reinterpret_cast<float4*>(st) = run;
}

// ---------------------------------------------------------------------------
// main: the outputs of one segment of one (sequence, KV head), chunk by chunk.
//
// Accumulators are kept transposed (O^T = V^T P^T): a lane holds 4
// consecutive output columns of one query row, so the online-softmax rescale
// and the final normalisation are lane-local and the output leaves in 8-byte
// (bf16) stores.
//
// The walk is software-pipelined over passes (256 query rows of a chunk):
// the next pass's query rows, first slab of delayed keys and first band tile
// are loaded before this pass's output stores.  Loads and stores retire in
// order, so a load issued after the stores could only be waited for together
// with them.
//
// A pass's 256 rows are spread over MW waves, 256 / MW rows (16-row q-tiles)
// each: every K and V fragment read from a band tile feeds 256 / (16 MW)
// q-tiles' MFMAs.  The workgroup's LDS (about 155 KB) admits one workgroup
// per CU, so MW waves run MW / 4 per SIMD with 512 / (MW / 4) registers
// each.
template <typename T, int D>
constexpr int main_waves() { return 8; }

template <typename T, int D, int DF>
struct MainLds {
  static constexpr int NBUF = 2;  // band stages
  static constexpr int SLAB = sizeof(T) == 4 && D == 128 ? 32 : 64;  // delayed keys per slab
  static constexpr int WROW = row_t<DF>(), PROW = row_t<DF>(), VROW = row_t<D>();
  static constexpr int SROW = DF + 4;                  // fp32 S^T rows: 16 rows of a 16-byte access on distinct banks
  static constexpr int KROW = row_a<D>();
  static constexpr int BAND = 32 * KROW + 32 * VROW;  // one band buffer (elements)
  // the slab (phi(k), values, raw keys) and the band buffers are never live
  // together
  static constexpr size_t slab_b = size_t(SLAB) * (PROW + VROW + KROW) * sizeof(T);
  static constexpr size_t band_b = size_t(NBUF) * BAND * sizeof(T);
  static constexpr size_t shared_b = slab_b > band_b ? slab_b : band_b;
  static constexpr size_t rest = size_t(D) * SROW * 4 + size_t(DF) * 4 + shared_b;
  // Wf in LDS when it fits beside the rest (fp32 with d = 128 reads it from
  // global memory)
  static constexpr bool kWfLds = size_t(D) * WROW * sizeof(T) + rest <= 160 * 1024;
  static constexpr size_t wn = 0;
  static constexpr size_t sn = wn + (kWfLds ? size_t(D) * WROW * sizeof(T) : 0);
  static constexpr size_t zs = sn + size_t(D) * SROW * 4;
  static constexpr size_t sh = zs + size_t(DF) * 4;
  static constexpr size_t bytes = sh + shared_b;
  static_assert(bytes <= 160 * 1024, "LDS budget");
};

// PHI: the feature map (0 ReLU, 1 ELU + 1).  PASS: 0 the band and the
// linear part over one shared denominator; for the hybrid forms, 1 the
// linear part alone (normalised on its own) and 2 the band alone, its
// normalised output added to what out holds.  One instantiation each.
// GATED (PASS 0 only): the gated linear state.  S_c is decayed to G_{t0-1}
// (the token before the chunk); row t reads it scaled by e^{G_t - G_{t0-1}},
// the masked block weighs pair (t, j) by e^{G_t - G_j} element by element
// (every factor <= 1, whatever the gates), and on the chunk's last pass
// S_{c+1} = e^{G_e - G_{t0-1}} S_c + sum_j e^{G_e - G_j} phi(k_j)^T v_j,
// G_e the chunk's last token, after the masked block has read phi(k).
template <typename T, int D, int DF, int PHI, int PASS, bool GATED, int MW>
__global__ __launch_bounds__(64 * MW) __attribute__((amdgpu_waves_per_eu(MW / 4, MW / 4)))
void prefill_main(PrefillArgs a) {
  using LD = MainLds<T, D, DF>;
  constexpr int NTH = 64 * MW, QT = kRB / (16 * MW);  // threads; 16-row q-tiles per wave
  static_assert(QT * 16 * MW == kRB, "a pass's rows must spread evenly over the waves");
  constexpr int KS = D / 32, KSF = DF / 32, CT = D / 16, FT = DF / 16;
  constexpr int NT = FT * CT / MW;            // S tiles per wave (state update)
  constexpr int SL = LD::SLAB;
  constexpr int SROW = LD::SROW, PROW = LD::PROW, VROW = LD::VROW, KROW = LD::KROW;
  constexpr int BAND = LD::BAND;
  constexpr int CPR = D / 8;                   // 8-element chunks per K/V row
  constexpr int VPT = SL * CPR / NTH;          // slab chunks per thread (keys; values alike)
  constexpr int SPT = (32 * CPR + NTH - 1) / NTH;  // band tile chunks per thread
  static_assert(NT * MW == FT * CT, "S tiles must spread evenly over the waves");
  static_assert(VPT >= 1 && VPT * NTH == SL * CPR && (SPT == 1 || SPT * NTH == 32 * CPR), "staging must divide evenly");
  // static LDS: the layout is fixed per instantiation
  __shared__ __align__(16) char smem[LD::bytes];
  T* Wn = reinterpret_cast<T*>(smem + LD::wn);          // [D][WROW]    Wf
  float* St = reinterpret_cast<float*>(smem + LD::sn);  // [D][SROW]    S_c^T, fp32
  float* zs = reinterpret_cast<float*>(smem + LD::zs);  // [DF]         z_c
  T* pk = reinterpret_cast<T*>(smem + LD::sh);          // [SL][PROW]   phi(k) of the delayed keys
  T* vs = pk + SL * PROW;                               // [SL][VROW]   their values
  T* kr = vs + SL * VROW;                               // [SL][KROW]   their keys
  T* bnd = reinterpret_cast<T*>(smem + LD::sh);         // band tiles: [2] x (K [32][KROW], V [32][VROW])

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hq = lane & 15, lg = lane >> 4;
  const int sg = blockIdx.x, g = blockIdx.y;
  const LayerView L = layer_view(a, blockIdx.z);
  const int bl = find_seq(a, sg);
  SeqRows<T, D> sr = seq_rows<T, D, DF>(a, L, bl, g);
  const int sigma = sg - a.seg_base[bl];
  const int s_lo = sigma * a.seg_len, s_hi = min(a.seq_len[bl], s_lo + a.seg_len);
  const int G = a.G, C = a.C;
  SeqGates gt{};
  if constexpr (GATED) gt = seq_gates<T, D, DF>(a, L, sr);
  __shared__ float gk_lds[LD::SLAB];  // gated: G_j - G_{t0-1} of the slab's delayed keys
  const int W = PASS == 1 ? 0 : L.W;  // the band's window (0: this pass has no band)
  const int Wd = L.Wd;                // the linear part's delay
  const bool linear = PASS != 2 && a.linear != 0;
  constexpr bool accum = PASS == 2;
  if (PASS == 2 && W == 0) return;    // a band-only pass: nothing to add for this layer
  // The band works on raw scores q.k scaled by sc2 >= 0 inside the exponent:
  // a negative tau is carried by the queries' sign (negated in registers for
  // the band, undone in the feature map), and a zero tau is raised to 1e-30,
  // whose products with any finite score are far below fp32 resolution
  // around the running max (every weight still comes out as exactly 1).
  const bool qneg = a.tau < 0.f;
  const float sc2 = fmaxf(fabsf(a.tau) * kLog2e, 1e-30f);
  const float inv_sc2 = 1.f / sc2;
  constexpr bool kOnesSum = sizeof(T) == 2;  // the band's row sums on the matrix cores
  const T* Q = static_cast<const T*>(L.q);
  T* O = static_cast<T*>(L.out);
  // the global bases, made opaque once per pass: row addresses are then
  // computed where they are used instead of being kept across the walk
  auto refresh = [&]() {
    sr.kin = sfresh(sr.kin);
    sr.vin = sfresh(sr.vin);
    sr.kh = sfresh(sr.kh);
    sr.vh = sfresh(sr.vh);
    Q = sfresh(Q);
    O = sfresh(O);
  };
  // Wf columns, with a fresh LDS base per phase
  auto wf_cols = [&]() {
    if constexpr (LD::kWfLds) return WfCols<T, D, DF, true>{lds_fresh(static_cast<const T*>(Wn))};
    else return WfCols<T, D, DF, false>{reinterpret_cast<const T*>(static_cast<const char*>(L.wf) + int64_t(g) * a.wf_hs)};
  };

  // ---- pass geometry: chunk c0 (nk tokens from absolute position t0), rows
  //      [rb, rb + kRB) of its nrow = nk * G query rows
  int c0 = s_lo, rb = 0, nk = 0, nrow = 0, ti_min = 0, ti_max = 0, wti_max = 0, ntile = 0;
  bool last_pass = true;
  int64_t t0 = 0, klo = 0, khi = 0, kb0 = 0;
  int ti[QT], hh[QT];  // this lane's query row (row hq) in each of its 16-row q-tiles
  bool rv[QT];
  auto geom = [&]() {
    nk = min(s_hi, c0 + C) - c0;
    t0 = sr.p0 + c0;
    nrow = nk * G;
    last_pass = rb + kRB >= nrow;
    const int r_end = min(nrow, rb + kRB);
    ti_min = rb / G;
    ti_max = (r_end - 1) / G;
    wti_max = min(r_end - 1, rb + 16 * QT * (wave + 1) - 1) / G;
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      const int r = rb + 16 * QT * wave + 16 * qt + hq;
      rv[qt] = r < nrow;
      const int rr = rv[qt] ? r : rb;
      ti[qt] = rr / G;
      hh[qt] = rr - ti[qt] * G;
    }
    // band keys [klo, khi]: the window of every row of the pass
    klo = t0 + ti_min - W + 1;
    if (klo < 0) klo = 0;
    khi = t0 + ti_max;
    kb0 = klo & ~int64_t(31);
    ntile = int((khi - kb0) / 32) + 1;
  };

  // ---- loads into registers (all unconditional; rows that do not exist are
  //      read from a row that does and replaced by zeros where stored)
  Frag<T> qf[QT][KS];
  auto load_q = [&]() {
#pragma unroll
    for (int qt = 0; qt < QT; ++qt)
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) qf[qt][kk].load(Q + sr.qrow(c0 + ti[qt], hh[qt]) * D + 32 * kk + 8 * lg);
  };
  // delayed keys i' of the chunk (key j = t0 - Wd + i'), a slab of SL at a time
  Frag<T> kst[VPT], vst[VPT];
  // Key and value rows are read through buffer descriptors with 32-bit
  // byte offsets per lane (the host guarantees a sequence's rows span less
  // than 2 GiB): a row that is not needed, or a history row of a slab that
  // has none, reads zeros with no memory access.  New tokens' rows are
  // Hkv * D elements apart; history rows (a continuing prefill) are
  // consecutive.
  const uint32_t rowb = uint32_t(a.Hkv) * D * sizeof(T);
  const uint32_t nbytes = uint32_t(a.seq_len[bl]) * rowb;  // the sequence's new rows
  const T* kn0 = sr.kin + (int64_t(sr.start) * a.Hkv + g) * D;  // this KV head's first new row
  const T* vn0 = sr.vin + (int64_t(sr.start) * a.Hkv + g) * D;
  const uint32_t hbytes = uint32_t(sr.p0 - sr.h0) * D * sizeof(T);  // the history rows
  auto load_slab = [&](int s0) {
    const int64_t jb = t0 - Wd + s0;  // the slab's first key (uniform)
#pragma unroll
    for (int u = 0; u < VPT; ++u) {
      const int id = tid + u * NTH, r = id / CPR, ch = id - r * CPR;
      const int64_t j = jb + r;
      const bool ok = s0 + r < nk && j >= 0;
      const int jr = int(j - sr.p0);  // key relative to the first new token
      const uint32_t cb = uint32_t(8 * sizeof(T)) * ch;
      const uint32_t on = ok && jr >= 0 ? uint32_t(jr) * rowb + cb : kOOB;
      bload_frag(kst[u], make_rsrc(kn0, nbytes), on);
      bload_frag(vst[u], make_rsrc(vn0, nbytes), on);
      if (jb < sr.p0) {  // the slab reaches into the history rows
        const uint32_t oh = ok && jr < 0 ? uint32_t(jr + int(sr.p0 - sr.h0)) * uint32_t(D * sizeof(T)) + cb : kOOB;
        Frag<T> hk, hv;
        bload_frag(hk, make_rsrc(sr.kh, hbytes), oh);
        bload_frag(hv, make_rsrc(sr.vh, hbytes), oh);
        kst[u] = frag_or(kst[u], hk);
        vst[u] = frag_or(vst[u], hv);
      }
    }
  };
  // (rows outside the slab were read as zeros: stored as they are)
  auto put_slab = [&]() {
    T* krw = lds_fresh(kr);
    T* vsw = lds_fresh(vs);
#pragma unroll
    for (int u = 0; u < VPT; ++u) {
      const int id = tid + u * NTH, r = id / CPR, ch = id - r * CPR;
      store8(krw + r * KROW + 8 * ch, kst[u]);
      store8(vsw + r * VROW + 8 * ch, vst[u]);
    }
  };
  // band tiles: this thread's chunk of tile n (K and V), for buffer n % 2
  // Band rows are read through buffer descriptors with 32-bit byte offsets
  // per lane (the host guarantees a sequence's rows span less than 2 GiB): a
  // row outside the band, or a history row of a tile that has none, reads
  // zeros with no memory access.  New tokens' rows are Hkv * D elements
  // apart; history rows (a continuing prefill) are consecutive.
  Frag<T> sk[SPT], sv[SPT];
  // wave-uniform; every thread when the tile's chunks cover the workgroup
  const bool stager = 32 * CPR >= NTH || tid < 32 * CPR;
  auto fetch = [&](int n) {
    if (stager) {
      const int64_t jt = kb0 + 32 * int64_t(n);   // the tile's first key (uniform)
      const int lo = int(klo - jt), hi = int(khi - jt);
      const T* kn = sr.kin + (int64_t(sr.start) * a.Hkv + g) * D;
      const T* vn = sr.vin + (int64_t(sr.start) * a.Hkv + g) * D;
#pragma unroll
      for (int u = 0; u < SPT; ++u) {
        const int id = tid + u * NTH, srr = id / CPR, sch = id - srr * CPR;
        const bool ok = srr >= lo && srr <= hi;
        const int jr = int(jt - sr.p0) + srr;      // key relative to the first new token
        const uint32_t cb = uint32_t(8 * sizeof(T)) * sch;  // the thread's 8-element chunk of the row
        const uint32_t on = ok && jr >= 0 ? uint32_t(jr) * rowb + cb : kOOB;
        bload_frag(sk[u], make_rsrc(kn, nbytes), on);
        bload_frag(sv[u], make_rsrc(vn, nbytes), on);
        if (jt < sr.p0) {  // the tile reaches into the history rows
          const uint32_t hb = uint32_t(sr.p0 - sr.h0) * D * sizeof(T);
          const uint32_t oh = ok && jr < 0 ? uint32_t(jr + int(sr.p0 - sr.h0)) * uint32_t(D * sizeof(T)) + cb : kOOB;
          Frag<T> hk, hv;
          bload_frag(hk, make_rsrc(sr.kh, hb), oh);
          bload_frag(hv, make_rsrc(sr.vh, hb), oh);
          sk[u] = frag_or(sk[u], hk);
          sv[u] = frag_or(sv[u], hv);
        }
      }
    }
  };
  auto store = [&](int n) {
    if (stager) {
      T* kt = lds_fresh(bnd + (n & 1) * BAND);
#pragma unroll
      for (int u = 0; u < SPT; ++u) {
        const int id = tid + u * NTH, srr = id / CPR, sch = id - srr * CPR;
        store8(kt + srr * KROW + 8 * sch, sk[u]);
        store8(kt + 32 * KROW + srr * VROW + 8 * sch, sv[u]);
      }
    }
  };
  // (the first slab of delayed keys is loaded after the band, with or
  // without one: its registers are not held through the band loop, and
  // every path issues its loads in the same order, so the compiler's
  // memory-counter waits for the queries do not also wait for the slab)
  auto prefetch = [&]() {
    load_q();  // the band's queries, then the feature map's input
    if (W > 0) fetch(0);
  };

  geom();
  prefetch();
  // ---- 0. (behind the first pass's loads) Wf into LDS; S, z at the
  //         segment start (the scan's record), fp32, into LDS (S transposed);
  //         they stay there for the whole walk
  if (linear) {
    if constexpr (LD::kWfLds) stage_wf<T, D, DF, NTH>(reinterpret_cast<const T*>(static_cast<const char*>(L.wf) + int64_t(g) * a.wf_hs), Wn);
    const float* S0 = L.seg + (int64_t(a.seg0 + sg) * a.Hkv + g) * (int64_t(DF) * D + DF);
    constexpr int NS = DF * D / 4 / NTH;
    static_assert(NS * NTH * 4 == DF * D, "even split");
    float4 x[NS];
#pragma unroll
    for (int u = 0; u < NS; ++u) {
      const int i = tid + u * NTH, f = i / (D / 4), c4 = 4 * (i - f * (D / 4));
      x[u] = *reinterpret_cast<const float4*>(S0 + f * D + c4);
    }
    const float zv = tid < DF ? S0[DF * D + tid] : 0.f;
#pragma unroll
    for (int u = 0; u < NS; ++u) {
      const int i = tid + u * NTH, f = i / (D / 4), c4 = 4 * (i - f * (D / 4));
      St[(c4 + 0) * SROW + f] = x[u].x;
      St[(c4 + 1) * SROW + f] = x[u].y;
      St[(c4 + 2) * SROW + f] = x[u].z;
      St[(c4 + 3) * SROW + f] = x[u].w;
    }
    if (tid < DF) zs[tid] = zv;
  }
  __syncthreads();  // Wf, S, z staged

  while (true) {
    f32x4_t acc[QT][CT];  // transposed: value columns 16ct+4lg+i of query row hq
    float m_run[QT], l_run[QT];
    float m_use[QT];  // m_run, or 0 while it is -inf
    float s_up[QT];   // raw score above which the band's running max moves
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) acc[qt][ct] = zero4();
      m_run[qt] = -INFINITY;
      l_run[qt] = 0.f;
      m_use[qt] = 0.f;
      s_up[qt] = -INFINITY;
    }

    // ---- 1. banded window attention, keys [klo, khi], 32-key tiles, two
    //         LDS stages (the previous pass ended at a barrier: the shared
    //         region is free)
    if (W > 0) {
      refresh();
      store(0);  // tile 0 was fetched with the pass's other prefetches
      if (qneg) {
#pragma unroll
        for (int qt = 0; qt < QT; ++qt)
#pragma unroll
          for (int kk = 0; kk < KS; ++kk) qf[qt][kk].negate();
      }
      __syncthreads();
      // bf16: each row's sum of the weights is a matrix product too, P^T
      // times a ones fragment, on the weights as rounded for P V (every
      // lane of the row's 16-lane column holds the full sum)
      f32x4_t lsum[QT];
      Frag<T> ones;
      if constexpr (kOnesSum) {
        ones.v = make_uint4(0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u);
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) lsum[qt] = zero4();
      }
      for (int n = 0; n < ntile; ++n) {
        if (n + 1 < ntile) fetch(n + 1);
        const T* kt = lds_fresh(static_cast<const T*>(bnd) + (n & 1) * BAND);
        const T* vt = kt + 32 * KROW;
        // scores: key row m of sub-tile t is key kb + 16t + m, so that a
        // 16-lane group's K reads cover 16 consecutive rows (distinct LDS
        // banks); lane (hq, lg) then holds the scores of keys 16t + 4lg + i,
        // the order its P^T fragment gives P V's reduction (V read at rows
        // 4lg .. 4lg+3 and 16+4lg .. 16+4lg+3 alike)
        f32x4_t sc[QT][2];
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) sc[qt][0] = sc[qt][1] = zero4();
        // the tile's K fragments, all issued before the first score MFMA
        Frag<T> kfr[2][KS];
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int kk = 0; kk < KS; ++kk) kfr[t][kk].load(kt + (16 * t + hq) * KROW + 32 * kk + 8 * lg);
#pragma unroll
        for (int kk = 0; kk < KS; ++kk)
#pragma unroll
          for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int qt = 0; qt < QT; ++qt) sc[qt][t] = mma(kfr[t][kk], qf[qt][kk], sc[qt][t]);
        // the V column fragments, in flight during the softmax
        Frag<T> fvr[CT];
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) load_colfrag2(fvr[ct], vt, VROW, 4 * lg, 16 + 4 * lg, 16 * ct);
        // the tile's first key, relative to the chunk's first token t0 (a
        // band spans less than 2^31 keys: 32-bit arithmetic)
        const int kb = int(kb0 - t0) + 32 * n;
        // keys [kb, kb+31] lie inside the band of every row of the pass
        // (tokens t0+ti_min .. t0+ti_max) for all but the edge tiles
        const bool interior = kb >= ti_max - W + 1 && kb + 31 <= ti_min;
        // raw scores, -inf outside the band (edge tiles; set in place)
        Frag<T> pf[QT];
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
          if (!interior) {
            // j - tq = base + off;  valid: j >= klo, tq - W < j <= tq, row
            // exists: one interval [olo, ohi] of offsets per row (empty for a
            // row that does not exist), tested without branches
            const int base = kb - ti[qt];
            const int offlo = int(klo - t0) - kb;  // first in-band offset of the tile (<= 31)
            const int lo = offlo < -1 ? -1 : offlo;
            const int olo = max(lo, 1 - W - base);
            const int ohi = rv[qt] ? -base : -1;
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                const int off = 16 * t + 4 * lg + i;
                const bool ok = (off >= olo) & (off <= ohi);
                sc[qt][t][i] = ok ? sc[qt][t][i] : -INFINITY;
              }
          }
        }
        // lazy rescale (one test for all the wave's rows): the running max
        // moves only when a score exceeds it by more than 2^8 (a raw score
        // above s_up = (m + 8) / sc2), so p = 2^(s - m) <= 256 and acc, l
        // stay in range; only then are the rows' tile maxima taken
        bool up = false;
#pragma unroll
        for (int qt = 0; qt < QT; ++qt)
#pragma unroll
          for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i) up = up | (sc[qt][t][i] > s_up[qt]);
        if (__any(up)) {
#pragma unroll
          for (int qt = 0; qt < QT; ++qt) {
            float x = fmaxf(sc[qt][0][0], sc[qt][1][0]);
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
              for (int i = 1; i < 4; ++i) x = fmaxf(x, sc[qt][t][i]);
            const float m_new = fmaxf(m_run[qt], lg_max(x) * sc2);
            const float alpha = m_new == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m_run[qt] - m_new);
            l_run[qt] *= alpha;
            if constexpr (kOnesSum) {
#pragma unroll
              for (int i = 0; i < 4; ++i) lsum[qt][i] *= alpha;
            }
            m_run[qt] = m_new;
            m_use[qt] = m_new == -INFINITY ? 0.f : m_new;
            s_up[qt] = (m_new + 8.f) * inv_sc2;
#pragma unroll
            for (int ct = 0; ct < CT; ++ct)
#pragma unroll
              for (int i = 0; i < 4; ++i) acc[qt][ct][i] *= alpha;
          }
        }
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
          float pv[8];
#pragma unroll
          for (int i = 0; i < 8; ++i) pv[i] = __builtin_amdgcn_exp2f(fmaf(sc[qt][i >> 2][i & 3], sc2, -m_use[qt]));
          pf[qt].set8(pv);
          if constexpr (!kOnesSum) {
            float ps = 0.f;
#pragma unroll
            for (int i = 0; i < 8; ++i) ps += pv[i];
            l_run[qt] += ps;
          }
        }
#pragma unroll
        for (int ct = 0; ct < CT; ++ct)
#pragma unroll
          for (int qt = 0; qt < QT; ++qt) acc[qt][ct] = mma(fvr[ct], pf[qt], acc[qt][ct]);
        if constexpr (kOnesSum) {
#pragma unroll
          for (int qt = 0; qt < QT; ++qt) lsum[qt] = mma(ones, pf[qt], lsum[qt]);
        }
        if (n + 1 < ntile) store(n + 1);
        __syncthreads();
      }
      if constexpr (kOnesSum) {
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) l_run[qt] += lg == 0 ? lsum[qt][0] : 0.f;
      }
    }


    // ---- 2. linear part.  The band's running max m (log2 domain) is the
    //         row's frame: the linear terms enter scaled by 2^-m, m raised to
    //         -60 first (the band's terms rescaled to match) so that 2^-m
    //         stays finite; without a band (W = 0) m = 0.
    if (linear) {
      load_slab(0);  // behind the feature map and the read-out
      float qscale[QT];
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
        const bool none = m_run[qt] == -INFINITY;
        const float m0 = none ? 0.f : fmaxf(m_run[qt], -60.f);
        const float alpha = none ? 1.f : __builtin_amdgcn_exp2f(m_run[qt] - m0);
        if (__any(alpha != 1.f)) {
          l_run[qt] *= alpha;
#pragma unroll
          for (int ct = 0; ct < CT; ++ct)
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[qt][ct][i] *= alpha;
        }
        m_run[qt] = m0;
        // (with the band's queries negated, phi takes them back: -(-q) Wf)
        qscale[qt] = (W > 0 && qneg) ? -__builtin_amdgcn_exp2f(-m0) : __builtin_amdgcn_exp2f(-m0);
      }
      // gated: G_t - G_{t0-1} of each row and its read-out factor
      float gqr[QT], fq[QT];
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
        gqr[qt] = 0.f;
        fq[qt] = 1.f;
      }
      double gref = 0.0;
      if constexpr (GATED) {
        gref = gt.at(t0 - 1);
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
          gqr[qt] = float(gt.at(t0 + ti[qt]) - gref);
          fq[qt] = decay_exp(gqr[qt]);
        }
      }
      // phi(q) 2^-m, transposed: lane (row hq, group lg) gets features
      // 32kf+4lg+i and 32kf+16+4lg+i of its query row in fragment kf
      Frag<T> pqf[QT][KSF];
      const auto wf = wf_cols();
      // the softmax map: each query row's max and 1 / sum over its DF
      // features, from a first pass (running max and rescaled sum per lane,
      // then over the row's 4 lane groups)
      float qmax[QT], qinv[QT];
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
        qmax[qt] = 0.f;
        qinv[qt] = 1.f;
      }
      if constexpr (PHI == GLIDE_PHI_SOFTMAX) {
        float m[QT], sm[QT];
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
          m[qt] = -INFINITY;
          sm[qt] = 0.f;
        }
#pragma unroll
        for (int kf = 0; kf < KSF; ++kf) {
#pragma unroll
          for (int half = 0; half < 2; ++half) {
            f32x4_t ph[QT];
#pragma unroll
            for (int qt = 0; qt < QT; ++qt) ph[qt] = zero4();
#pragma unroll
            for (int kk = 0; kk < KS; ++kk) {
              Frag<T> wa;
              wf.col(wa, kk, 32 * kf + 16 * half);
#pragma unroll
              for (int qt = 0; qt < QT; ++qt) ph[qt] = mma(wa, qf[qt][kk], ph[qt]);
            }
#pragma unroll
            for (int qt = 0; qt < QT; ++qt) {
              float y[4], mg = -INFINITY;
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                y[i] = qscale[qt] < 0.f ? -ph[qt][i] : ph[qt][i];
                mg = fmaxf(mg, y[i]);
              }
              const float mn = fmaxf(m[qt], mg);
              float add = 0.f;
#pragma unroll
              for (int i = 0; i < 4; ++i) add += __builtin_amdgcn_exp2f((y[i] - mn) * kLog2e);
              sm[qt] = sm[qt] * __builtin_amdgcn_exp2f((m[qt] - mn) * kLog2e) + add;
              m[qt] = mn;
            }
          }
        }
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
#pragma unroll
          for (int off = 16; off < 64; off <<= 1) {
            const float mo = __shfl_xor(m[qt], off), so = __shfl_xor(sm[qt], off);
            const float mn = fmaxf(m[qt], mo);
            sm[qt] = sm[qt] * __builtin_amdgcn_exp2f((m[qt] - mn) * kLog2e) +
                     so * __builtin_amdgcn_exp2f((mo - mn) * kLog2e);
            m[qt] = mn;
          }
          qmax[qt] = m[qt];
          qinv[qt] = 1.f / sm[qt];
        }
      }
#pragma unroll
      for (int kf = 0; kf < KSF; ++kf) {
        float pv[QT][8];
        // the 32 columns' Wf fragments, read in one batch
        Frag<T> wa[2][KS];
#pragma unroll
        for (int half = 0; half < 2; ++half)
#pragma unroll
          for (int kk = 0; kk < KS; ++kk) wf.col(wa[half][kk], kk, 32 * kf + 16 * half);
        f32x4_t ph[2][QT];
#pragma unroll
        for (int half = 0; half < 2; ++half)
#pragma unroll
          for (int qt = 0; qt < QT; ++qt) ph[half][qt] = zero4();
#pragma unroll
        for (int kk = 0; kk < KS; ++kk)
#pragma unroll
          for (int half = 0; half < 2; ++half)
#pragma unroll
            for (int qt = 0; qt < QT; ++qt) ph[half][qt] = mma(wa[half][kk], qf[qt][kk], ph[half][qt]);
#pragma unroll
        for (int half = 0; half < 2; ++half) {
#pragma unroll
          for (int qt = 0; qt < QT; ++qt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              if constexpr (PHI == 0)
                pv[qt][4 * half + i] = fmaxf(ph[half][qt][i] * qscale[qt], 0.f);
              else if constexpr (PHI == GLIDE_PHI_SOFTMAX)
                pv[qt][4 * half + i] =
                    __builtin_amdgcn_exp2f(((qscale[qt] < 0.f ? -ph[half][qt][i] : ph[half][qt][i]) - qmax[qt]) * kLog2e) *
                    qinv[qt] * fabsf(qscale[qt]);
              else  // (qscale's sign undoes the band's query negation)
                pv[qt][4 * half + i] =
                    feat_act(qscale[qt] < 0.f ? -ph[half][qt][i] : ph[half][qt][i], PHI) * fabsf(qscale[qt]);
            }
        }
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) pqf[qt][kf].set8(pv[qt]);
      }
      // read-out (phi(q).S_c)^T = S_c^T phi(q)^T, and phi(q).z_c
      const float* Sr = lds_fresh(static_cast<const float*>(St)) + hq * SROW;
#pragma unroll
      for (int kf = 0; kf < KSF; ++kf) {
        Frag<T> rq[QT];  // the read-out's phi(q): decayed when gated
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
          if constexpr (GATED) {
            float x[8];
            pqf[qt][kf].to_floats(x);
#pragma unroll
            for (int i = 0; i < 8; ++i) x[i] *= fq[qt];
            rq[qt].set8(x);
          } else {
            rq[qt] = pqf[qt][kf];
          }
        }
        // S^T rows read four column tiles at a time
        constexpr int CB = CT < 4 ? CT : 4;
#pragma unroll
        for (int c0 = 0; c0 < CT; c0 += CB) {
          Frag<T> fs[CB];
#pragma unroll
          for (int c = 0; c < CB; ++c)
            load_row2_f32(fs[c], Sr + 16 * (c0 + c) * SROW, 32 * kf + 4 * lg, 32 * kf + 16 + 4 * lg);
#pragma unroll
          for (int c = 0; c < CB; ++c)
#pragma unroll
            for (int qt = 0; qt < QT; ++qt) acc[qt][c0 + c] = mma(fs[c], rq[qt], acc[qt][c0 + c]);
        }
      }
      float den[QT];
      const float* zr = lds_fresh(static_cast<const float*>(zs));
      // bf16: the masked block's weight sums go to the matrix cores as in
      // the band (P^T times a ones fragment, full sums in every lane group)
      Frag<T> ones;
      f32x4_t dsum[QT];
      if constexpr (kOnesSum) {
        ones.v = make_uint4(0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u);
        // phi(q).z on the matrix cores too: z (fp32, as a bf16 hi + lo
        // pair, about 16 bits) is the A fragment of every row, in phi(q)'s
        // feature order
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) dsum[qt] = zero4();
#pragma unroll
        for (int kf = 0; kf < KSF; ++kf) {
          const float4 za = *reinterpret_cast<const float4*>(zr + 32 * kf + 4 * lg);
          const float4 zb = *reinterpret_cast<const float4*>(zr + 32 * kf + 16 + 4 * lg);
          float x[8] = {za.x, za.y, za.z, za.w, zb.x, zb.y, zb.z, zb.w}, h[8];
          Frag<T> zh, zl;
          zh.set8(x);
          zh.to_floats(h);
#pragma unroll
          for (int i = 0; i < 8; ++i) x[i] -= h[i];
          zl.set8(x);
#pragma unroll
          for (int qt = 0; qt < QT; ++qt) {
            dsum[qt] = mma(zh, pqf[qt][kf], dsum[qt]);
            dsum[qt] = mma(zl, pqf[qt][kf], dsum[qt]);
          }
        }
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
          den[qt] = lg == 0 ? dsum[qt][0] * fq[qt] : 0.f;
          dsum[qt] = zero4();
        }
      } else {
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
          float dz = 0.f;
#pragma unroll
          for (int kf = 0; kf < KSF; ++kf) {
            float qv[8];
            pqf[qt][kf].to_floats(qv);
            const float4 za = *reinterpret_cast<const float4*>(zr + 32 * kf + 4 * lg);
            const float4 zb = *reinterpret_cast<const float4*>(zr + 32 * kf + 16 + 4 * lg);
            dz = fmaf(qv[0], za.x, dz); dz = fmaf(qv[1], za.y, dz);
            dz = fmaf(qv[2], za.z, dz); dz = fmaf(qv[3], za.w, dz);
            dz = fmaf(qv[4], zb.x, dz); dz = fmaf(qv[5], zb.y, dz);
            dz = fmaf(qv[6], zb.z, dz); dz = fmaf(qv[7], zb.w, dz);
          }
          den[qt] = dz * fq[qt];
        }
      }
      // the chunk's delayed keys, SL at a time: phi(k) into LDS, the masked
      // block i' <= ti of every query row, and (last pass: every read-out of
      // S_c, z_c is done, and the loop covers all the chunk's keys)
      // S_{c+1} = S_c + phi(k)^T v, z_{c+1} = z_c + sum phi(k), in place
      put_slab();  // the first slab's keys and values (made visible by the slab loop's barrier)
      for (int s0 = 0; s0 < nk; s0 += SL) {
        if (s0 > ti_max) break;
        if (s0 > 0) {
          __syncthreads();  // the previous slab's readers are done
          load_slab(s0);
          put_slab();
        }
        if constexpr (GATED) {
          if (tid < SL) {
            const int64_t j = t0 - Wd + s0 + tid;
            gk_lds[tid] = (s0 + tid < nk && j >= 0) ? float(gt.at(j) - gref) : 0.f;
          }
        }
        __syncthreads();  // keys and values staged; the read-outs of S_c, z_c are done
        {
          const int kt = slab_key_tile<D, DF, SL>(MW);
          const T* krr = lds_fresh(static_cast<const T*>(kr));
          Frag<T> x[KS];
#pragma unroll
          for (int kk = 0; kk < KS; ++kk) x[kk].load(krr + (16 * kt + hq) * KROW + 32 * kk + 8 * lg);
          // the slab's keys: i' = s0 + r < nk, and key t0 - Wd + i' >= 0
          const int64_t rlo = int64_t(Wd) - t0 - s0;
          phi_slab<T, D, DF, SL, PHI, MW>(wf_cols(), x, lds_fresh(pk), rlo > 0 ? int(rlo < SL ? rlo : SL) : 0,
                                          nk - s0);
        }
        __syncthreads();
        const T* pkr = lds_fresh(static_cast<const T*>(pk));
        const T* vsr = lds_fresh(static_cast<const T*>(vs));
        // S_{c+1} = dch S_c + phi(k)^T v (dch: the chunk's decay, applied with
        // the first slab; 1 ungated).  Every S tile (and z slice) has one
        // owner wave: plain updates.  Lane (hq, lg) gets features 16ft+4lg..
        // of value column 16ct+hq, 4 consecutive floats of S^T
        auto state_update = [&](float dch) {
          float* Sw = lds_fresh(St);
          float* zw = lds_fresh(zs);
#pragma unroll
          for (int x = 0; x < NT; ++x) {
            const int tile = wave * NT + x, ft = tile / CT, ct = tile - ft * CT;
            f32x4_t d = zero4();
            float zp = 0.f;
#pragma unroll
            for (int kh = 0; kh < SL / 32; ++kh) {
              Frag<T> fa, fb;
              // keys 32kh + 4lg .. +3 and 32kh + 16 + 4lg .. +3 (distinct
              // LDS banks within each 32-lane half)
              load_colfrag2(fa, pkr, PROW, 32 * kh + 4 * lg, 32 * kh + 16 + 4 * lg, 16 * ft);
              load_colfrag2(fb, vsr, VROW, 32 * kh + 4 * lg, 32 * kh + 16 + 4 * lg, 16 * ct);
              d = mma(fa, fb, d);
              if (ct == 0) zp += fa.sum();  // those keys' feature 16ft+hq
            }
            float4* sp = reinterpret_cast<float4*>(Sw + (16 * ct + hq) * SROW + 16 * ft + 4 * lg);
            float4 s4 = *sp;
            if constexpr (GATED) {
              s4.x = fmaf(s4.x, dch, d[0]); s4.y = fmaf(s4.y, dch, d[1]);
              s4.z = fmaf(s4.z, dch, d[2]); s4.w = fmaf(s4.w, dch, d[3]);
            } else {
              s4.x += d[0]; s4.y += d[1]; s4.z += d[2]; s4.w += d[3];
            }
            *sp = s4;
            if (ct == 0) {
              zp = lg_sum(zp);
              if (lg == 0) zw[16 * ft + hq] = fmaf(zw[16 * ft + hq], GATED ? dch : 1.f, zp);
            }
          }
        };
        if (!GATED && last_pass) state_update(1.f);
        // scores: key row m of sub-tile t of 32-key block kb is
        // i' = s0 + 32kb + 16t + m (consecutive rows per lane group), so lane
        // (hq, lg) holds keys 32kb + 16t + 4lg + i
        // (a block of keys after every row of this wave is skipped: the
        // wave's rows are consecutive, its last token is wti_max)
#pragma unroll
        for (int kb = 0; kb < SL / 32; ++kb) {
          if (s0 + 32 * kb > wti_max) break;
          f32x4_t sc[QT][2];
#pragma unroll
          for (int qt = 0; qt < QT; ++qt) sc[qt][0] = sc[qt][1] = zero4();
          // the block's phi(k) fragments, then its V column fragments (in
          // flight during the mask), each read in one batch
          Frag<T> fa[2][KSF];
#pragma unroll
          for (int t = 0; t < 2; ++t) {
            const T* prow = pkr + (32 * kb + 16 * t + hq) * PROW;
#pragma unroll
            for (int kf = 0; kf < KSF; ++kf) load_row2(fa[t][kf], prow, 32 * kf + 4 * lg, 32 * kf + 16 + 4 * lg);
          }
#pragma unroll
          for (int kf = 0; kf < KSF; ++kf)
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
              for (int qt = 0; qt < QT; ++qt) sc[qt][t] = mma(fa[t][kf], pqf[qt][kf], sc[qt][t]);
          Frag<T> fv[CT];
#pragma unroll
          for (int ct = 0; ct < CT; ++ct) load_colfrag2(fv[ct], vsr, VROW, 32 * kb + 4 * lg, 32 * kb + 16 + 4 * lg, 16 * ct);
          Frag<T> pf[QT];
#pragma unroll
          for (int qt = 0; qt < QT; ++qt) {
            float pv[8];
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                const int kr_ = 32 * kb + 16 * t + 4 * lg + i;  // the key within the slab
                const float w = GATED ? decay_exp(gqr[qt] - gk_lds[kr_]) : 1.f;
                pv[4 * t + i] = (s0 + kr_ <= ti[qt]) ? sc[qt][t][i] * w : 0.f;
              }
            pf[qt].set8(pv);
            if constexpr (!kOnesSum) den[qt] += pf[qt].sum();
          }
#pragma unroll
          for (int ct = 0; ct < CT; ++ct)
#pragma unroll
            for (int qt = 0; qt < QT; ++qt) acc[qt][ct] = mma(fv[ct], pf[qt], acc[qt][ct]);
          if constexpr (kOnesSum) {
#pragma unroll
            for (int qt = 0; qt < QT; ++qt) dsum[qt] = mma(ones, pf[qt], dsum[qt]);
          }
        }
        if constexpr (GATED) {
          if (last_pass) {
            // the masked block has read phi(k): each key row is now decayed
            // to the chunk's last token, then S_{c+1}
            __syncthreads();
            const float gend_rel = float(gt.at(t0 + nk - 1) - gref);
            T* pkw = lds_fresh(pk);
            for (int e = tid; e < SL * DF; e += NTH) {
              const int r = e / DF, f = e - r * DF;
              pkw[r * PROW + f] = from_f32<T>(to_f32(pkw[r * PROW + f]) * decay_exp(gend_rel - gk_lds[r]));
            }
            __syncthreads();
            state_update(s0 == 0 ? decay_exp(gend_rel) : 1.f);
          }
        }
      }
      // the shared denominator: band sum + linear part (per-lane partials)
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
        if constexpr (kOnesSum) den[qt] += lg == 0 ? dsum[qt][0] : 0.f;
        l_run[qt] += den[qt];
      }
    }

    // ---- 3. the next pass's loads, then this pass's outputs: value columns
    //         16ct+4lg .. +3 of query row hq
    int64_t orow[QT];
    bool ov[QT];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      orow[qt] = sr.qrow(c0 + ti[qt], hh[qt]) * D + 4 * lg;
      ov[qt] = rv[qt];
    }
    const bool more = !(last_pass && c0 + C >= s_hi);
    if (more) {
      if (last_pass) {
        c0 += C;
        rb = 0;
      } else {
        rb += kRB;
      }
      geom();
    }
    // Unconditional, so that every path issues the same loads here (the
    // compiler's wait counts merge paths, and a path without these loads
    // would make the stores below wait for them).  After the last pass it
    // reloads that pass's rows: valid addresses, never waited for.
    refresh();
    prefetch();
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      const float ls = lg_sum(l_run[qt]);
      const float inv = ls > 0.f ? 1.f / ls : 0.f;
      if (ov[qt]) {
        if constexpr (accum) {
#pragma unroll
          for (int ct = 0; ct < CT; ++ct) add4(O + orow[qt] + 16 * ct, acc[qt][ct], inv);
        } else {
#pragma unroll
          for (int ct = 0; ct < CT; ++ct) store4(O + orow[qt] + 16 * ct, acc[qt][ct], inv);
        }
      }
    }
    if (!more) break;
    // pass boundary: the next pass writes the slab staging (and, at a chunk
    // boundary, reads S_{c+1}, z_{c+1})
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// ringfill: tokens [max(p0, p_end - W), p_end) into their ring slots.  A key
// slot takes 16-byte chunks (8 consecutive columns); the value layout keeps 8
// consecutive slots of one column together, so a thread gathers one column of
// 8 consecutive tokens (R is a multiple of 8, so such a group never wraps)
// and stores it at once, or element by element where the group is only partly
// in range (its other slots may hold live tokens).
template <typename T, int D, int DF>
__global__ __launch_bounds__(kThreads) void prefill_ringfill(PrefillArgs a) {
  const int bl = blockIdx.y, g = int(blockIdx.z) % a.Hkv;
  const LayerView L = layer_view(a, int(blockIdx.z) / a.Hkv);
  if (L.W == 0) return;
  const SeqRows<T, D> sr = seq_rows<T, D, DF>(a, L, bl, g);
  const int Tb = a.seq_len[bl];
  const int64_t pend = sr.p0 + Tb;
  int64_t jlo = pend - L.W;
  if (jlo < sr.p0) jlo = sr.p0;
  const int n = int(pend - jlo);
  if (n <= 0) return;
  const LayerSections sec = layer_sections(a.B, a.Hkv, D, DF, L.R, sizeof(T));
  const int64_t unit = int64_t(sr.b) * a.Hkv + g;
  T* Kr = reinterpret_cast<T*>(L.base + sec.K) + unit * L.R * D;
  T* Vr = reinterpret_cast<T*>(L.base + sec.V) + unit * L.R * D;
  constexpr int CPR = D / 8;
  const int stride = gridDim.x * kThreads;
  for (int idx = blockIdx.x * kThreads + threadIdx.x; idx < n * CPR; idx += stride) {
    const int i = idx / CPR, ch = idx - i * CPR;
    const int64_t j = jlo + i;
    Frag<T> f;
    f.load(sr.k(j) + 8 * ch);
    store8(Kr + kring_elem(int32_t(j % L.R), 8 * ch, D), f);
  }
  if (a.gated) {  // the ring tokens' G_j
    const LayerSections sg = layer_sections(a.B, a.Hkv, D, DF, L.R, sizeof(T), true);
    double* grg = reinterpret_cast<double*>(L.base + sg.GR) + unit * L.R;
    const SeqGates gt = seq_gates<T, D, DF>(a, L, sr);
    for (int idx = blockIdx.x * kThreads + threadIdx.x; idx < n; idx += stride)
      grg[(jlo + idx) % L.R] = gt.at(jlo + idx);
  }
  const int64_t m0 = jlo >> 3;
  const int ng = int(((pend - 1) >> 3) - m0 + 1);
  for (int idx = blockIdx.x * kThreads + threadIdx.x; idx < ng * D; idx += stride) {
    const int gi = idx / D, c = idx - gi * D;
    const int64_t j0 = (m0 + gi) * 8;
    T* dst = Vr + vring_elem(int32_t(j0 % L.R), c, D);  // slots s0 .. s0+7 of column c
    if (j0 >= jlo && j0 + 8 <= pend) {
      float x[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = to_f32(sr.v(j0 + e)[c]);
      Frag<T> f;
      f.set8(x);
      store8(dst, f);
    } else {
      for (int e = 0; e < 8; ++e)
        if (j0 + e >= jlo && j0 + e < pend) dst[e] = sr.v(j0 + e)[c];
    }
  }
}

// advance: pos += T_b (after every other kernel of the layer read pos); the
// scan left S, z = the sums over tokens [0, max(0, pos - Wd)), nothing
// pending.
template <typename T, int D, int DF>
__global__ void prefill_advance(PrefillArgs a) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.nseq * a.Hkv) return;
  const LayerView L = layer_view(a, blockIdx.y);
  const int bl = i / a.Hkv, g = i - bl * a.Hkv;
  const LayerSections sec = layer_sections(a.B, a.Hkv, D, DF, L.R, sizeof(T));
  const int64_t unit = int64_t(a.seq0 + bl) * a.Hkv + g;
  int64_t* pos = reinterpret_cast<int64_t*>(L.base + sec.pos) + unit;
  int64_t* nf = reinterpret_cast<int64_t*>(L.base + sec.nf) + unit;
  const int64_t p = *pos + a.seq_len[bl];
  *pos = p;
  *nf = p - L.Wd > 0 ? p - L.Wd : 0;
  if (a.gated && a.seq_len[bl] > 0) {  // G_{p-1}; the scan left S, z decayed to it
    const LayerSections sg = layer_sections(a.B, a.Hkv, D, DF, L.R, sizeof(T), true);
    double* gst = reinterpret_cast<double*>(L.base + sg.G) + 2 * unit;
    const double* gc = reinterpret_cast<const double*>(a.ws + int64_t(L.ls) * a.ws_slot + a.ws_gc);
    const double ge = gc[(int64_t(a.seq_start[bl]) + a.seq_len[bl] - 1) * a.Hkv + g];
    gst[0] = ge;
    gst[1] = ge;
  }
}

// The kernels of one prefill launch, for the a.nlayer layers of a.layers
// (the grid's last dimension runs over them, longest windows first).
template <typename T, int D, int DF>
hipError_t layer_t(const PrefillArgs& a, hipStream_t s) {
  constexpr int MW = main_waves<T, D>();
  hipError_t e;
  const unsigned nl = unsigned(a.nlayer);
  bool window = false;
  for (int i = 0; i < a.nlayer; ++i) window = window || a.layers[i].W > 0;
  auto main = [&](int pass) {
    const dim3 grid(a.nseg, a.Hkv, nl), block(64 * MW);
    if (a.gated) {  // the shared denominator only
      if (a.phi == GLIDE_PHI_SOFTMAX) hipLaunchKernelGGL((prefill_main<T, D, DF, 2, 0, true, MW>), grid, block, 0, s, a);
      else if (a.phi) hipLaunchKernelGGL((prefill_main<T, D, DF, 1, 0, true, MW>), grid, block, 0, s, a);
      else hipLaunchKernelGGL((prefill_main<T, D, DF, 0, 0, true, MW>), grid, block, 0, s, a);
      return;
    }
    if (a.phi == GLIDE_PHI_SOFTMAX) {
      if (pass == 0) hipLaunchKernelGGL((prefill_main<T, D, DF, 2, 0, false, MW>), grid, block, 0, s, a);
      if (pass == 1) hipLaunchKernelGGL((prefill_main<T, D, DF, 2, 1, false, MW>), grid, block, 0, s, a);
      if (pass == 2) hipLaunchKernelGGL((prefill_main<T, D, DF, 2, 2, false, MW>), grid, block, 0, s, a);
    } else if (a.phi) {
      if (pass == 0) hipLaunchKernelGGL((prefill_main<T, D, DF, 1, 0, false, MW>), grid, block, 0, s, a);
      if (pass == 1) hipLaunchKernelGGL((prefill_main<T, D, DF, 1, 1, false, MW>), grid, block, 0, s, a);
      if (pass == 2) hipLaunchKernelGGL((prefill_main<T, D, DF, 1, 2, false, MW>), grid, block, 0, s, a);
    } else {
      if (pass == 0) hipLaunchKernelGGL((prefill_main<T, D, DF, 0, 0, false, MW>), grid, block, 0, s, a);
      if (pass == 1) hipLaunchKernelGGL((prefill_main<T, D, DF, 0, 1, false, MW>), grid, block, 0, s, a);
      if (pass == 2) hipLaunchKernelGGL((prefill_main<T, D, DF, 0, 2, false, MW>), grid, block, 0, s, a);
    }
  };
  if (a.gated) {  // the new tokens' cumulative log-gates, before any kernel reads them
    hipLaunchKernelGGL((prefill_gates<T, D, DF>), dim3(a.nseq, a.Hkv, nl), dim3(kThreads), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (a.nseg > 0) {
    if (a.linear) {
      if (a.phi == GLIDE_PHI_SOFTMAX)
        hipLaunchKernelGGL((prefill_segsum<T, D, DF, 2>), dim3(a.nseg, a.Hkv, nl), dim3(kSegThreads), 0, s, a);
      else if (a.phi)
        hipLaunchKernelGGL((prefill_segsum<T, D, DF, 1>), dim3(a.nseg, a.Hkv, nl), dim3(kSegThreads), 0, s, a);
      else
        hipLaunchKernelGGL((prefill_segsum<T, D, DF, 0>), dim3(a.nseg, a.Hkv, nl), dim3(kSegThreads), 0, s, a);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      const int E = DF * D + DF;
      hipLaunchKernelGGL((prefill_scan<T, D, DF>), dim3((E / 4 + kThreads - 1) / kThreads, a.nseq, a.Hkv * nl),
                         dim3(kThreads), 0, s, a);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (a.form == 0) {
      main(0);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    } else {
      // hybrid forms: the linear part normalised on its own, then the band's
      // normalised output added to it
      main(1);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      if (window) {
        main(2);
        if ((e = hipGetLastError()) != hipSuccess) return e;
      }
    }
  }
  if (window) {
    hipLaunchKernelGGL((prefill_ringfill<T, D, DF>), dim3(32, a.nseq, a.Hkv * nl), dim3(kThreads), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  hipLaunchKernelGGL((prefill_advance<T, D, DF>), dim3((a.nseq * a.Hkv + 255) / 256, nl), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <typename T, int D, int DF>
hipError_t gather_t(const PrefillArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((prefill_gather<T, D, DF>), dim3(16, a.nseq, a.Hkv * unsigned(a.nlayer)), dim3(kThreads), 0,
                     s, a);
  return hipGetLastError();
}

}  // namespace

#define GLIDE_DISPATCH(FN, ...)                                                   \
  do {                                                                            \
    if (dtype == GLIDE_BF16) {                                                    \
      if (d == 128 && Df == 128) return FN<bf16_t, 128, 128>(__VA_ARGS__);        \
      if (d == 128 && Df == 64) return FN<bf16_t, 128, 64>(__VA_ARGS__);          \
      if (d == 64 && Df == 128) return FN<bf16_t, 64, 128>(__VA_ARGS__);         \
      if (d == 64 && Df == 64) return FN<bf16_t, 64, 64>(__VA_ARGS__);           \
    } else {                                                                      \
      if (d == 128 && Df == 128) return FN<float, 128, 128>(__VA_ARGS__);         \
      if (d == 128 && Df == 64) return FN<float, 128, 64>(__VA_ARGS__);           \
      if (d == 64 && Df == 128) return FN<float, 64, 128>(__VA_ARGS__);          \
      if (d == 64 && Df == 64) return FN<float, 64, 64>(__VA_ARGS__);            \
    }                                                                             \
    return hipErrorInvalidValue;                                                  \
  } while (0)

hipError_t launch_prefill_layer(const PrefillArgs& a, int d, int Df, int dtype, hipStream_t s) {
  GLIDE_DISPATCH(layer_t, a, s);
}
hipError_t launch_prefill_gather(const PrefillArgs& a, int d, int Df, int dtype, hipStream_t s) {
  GLIDE_DISPATCH(gather_t, a, s);
}

}  // namespace glide
