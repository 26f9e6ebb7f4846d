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
//   main     per segment, chunks in order with S carried in fp32 MFMA
//            accumulators: the linear read-out phi(Q)S_c plus the masked
//            intra-chunk block start every query row's online softmax as one
//            pseudo-key of weight a = phi(q).z_c + sum of the block's weights
//            and value A/a (exactly the shared-denominator merge); then the
//            banded window attention over LDS-staged key tiles on MFMA;
//   ringfill the last W tokens into the ring;   advance: pos += T_b.
#include <math.h>

#include "glide_internal.h"

namespace glide {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr int kPad = 8;  // LDS row padding (elements)
constexpr float kLog2e = 1.4426950408889634f;

// Rows of one (sequence, KV head) of a layer: new tokens come from the
// packed inputs, older tokens from the history side buffer (stride W).
template <typename T, int D, int DF>
struct SeqRows {
  const T *kin, *vin, *pkin, *kh, *vh, *pkh;  // inputs of the layer, then this unit's history
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
  __device__ const T* phk(int64_t j) const {
    if (j >= p0) return pkin + ((int64_t(start) + (j - p0)) * Hkv + g) * DF;
    if (j >= h0) return pkh + (j - h0) * DF;
    return nullptr;
  }
  // packed query row of new token i (0-based within the call) and head hh of the group
  __device__ int64_t qrow(int i, int hh) const { return (int64_t(start) + i) * Hq + int64_t(g) * G + hh; }
};

template <typename T, int D, int DF>
__device__ __forceinline__ SeqRows<T, D, DF> seq_rows(const PrefillArgs& a, int bl, int g) {
  SeqRows<T, D, DF> r;
  r.b = a.seq0 + bl;
  r.g = g;
  r.start = a.seq_start[bl];
  r.Hq = a.Hq;
  r.Hkv = a.Hkv;
  r.G = a.G;
  const int64_t unit = int64_t(r.b) * a.Hkv + g;
  r.kin = static_cast<const T*>(a.k);
  r.vin = static_cast<const T*>(a.v);
  r.pkin = static_cast<const T*>(a.phk);
  r.kh = static_cast<const T*>(a.hk) + unit * a.W * D;
  r.vh = static_cast<const T*>(a.hv) + unit * a.W * D;
  r.pkh = static_cast<const T*>(a.hphk) + unit * a.W * DF;
  const LayerSections sec = layer_sections(a.B, a.Hkv, D, DF, a.R, sizeof(T));
  r.p0 = reinterpret_cast<const int64_t*>(a.state + a.layer_base + sec.pos)[unit];
  r.h0 = r.p0 - a.W > 0 ? r.p0 - a.W : 0;
  return r;
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
__device__ __forceinline__ void store_t8(bf16_t* dst, int stride, const Frag<bf16_t>& f) {
  const uint32_t w[4] = {f.v.x, f.v.y, f.v.z, f.v.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    dst[(2 * e) * stride] = bf16_t(w[e] & 0xffffu);
    dst[(2 * e + 1) * stride] = bf16_t(w[e] >> 16);
  }
}
__device__ __forceinline__ void store_t8(float* dst, int stride, const Frag<float>& f) {
#pragma unroll
  for (int e = 0; e < 8; ++e) dst[e * stride] = f.v[e];
}

// Stage 32 token rows of NC elements into LDS: natural [32][NC + kPad] and/or
// transposed [NC][32 + kPad].  row(r) gives the row pointer, nullptr = zeros.
template <typename T, int NC, typename RowFn>
__device__ __forceinline__ void stage32(T* nat, T* trans, RowFn row) {
  constexpr int CPR = NC / 8;
  for (int id = threadIdx.x; id < 32 * CPR; id += kThreads) {
    const int r = id / CPR, ch = id - r * CPR;
    const T* src = row(r);
    Frag<T> f;
    if (src) f.load(src + 8 * ch);
    else f.zero();
    if (nat) store8(nat + r * (NC + kPad) + 8 * ch, f);
    if (trans) store_t8(trans + (8 * ch) * (32 + kPad) + r, 32 + kPad, f);
  }
}

// ---------------------------------------------------------------------------
// gather: history tokens [h0, p0) of a continuing prefill, ring -> [b][g][W][d]
template <typename T, int D, int DF>
__global__ __launch_bounds__(kThreads) void prefill_gather(PrefillArgs a) {
  const int bl = blockIdx.y, g = blockIdx.z;
  const SeqRows<T, D, DF> sr = seq_rows<T, D, DF>(a, bl, g);
  const int n = int(sr.p0 - sr.h0);
  if (n <= 0) return;
  const LayerSections sec = layer_sections(a.B, a.Hkv, D, DF, a.R, sizeof(T));
  const int64_t unit = int64_t(sr.b) * a.Hkv + g;
  const T* Kr = reinterpret_cast<const T*>(a.state + a.layer_base + sec.K) + unit * a.R * D;
  const T* Vr = reinterpret_cast<const T*>(a.state + a.layer_base + sec.V) + unit * a.R * D;
  T* hk = static_cast<T*>(a.hk) + unit * a.W * D;
  T* hv = static_cast<T*>(a.hv) + unit * a.W * D;
  for (int idx = blockIdx.x * kThreads + threadIdx.x; idx < n * D; idx += gridDim.x * kThreads) {
    const int i = idx / D, c = idx - i * D;
    const int32_t s = int32_t((sr.h0 + i) % a.R);
    hk[int64_t(i) * D + c] = Kr[kring_elem(s, c, D)];
    hv[int64_t(i) * D + c] = Vr[vring_elem(s, c, D)];
  }
}

// ---------------------------------------------------------------------------
// segsum: state increment of one segment from its delayed keys
//   dS[f][c] = sum_j phi(k_j)[f] v_j[c],  dz[f] = sum_j phi(k_j)[f],
//   j in [t_lo - W, t_hi - W) and j >= 0, where [t_lo, t_hi) are the segment's queries.
template <typename T, int D, int DF>
__global__ __launch_bounds__(kThreads) void prefill_segsum(PrefillArgs a) {
  constexpr int CT = D / 16;
  constexpr int FTW = DF / 16 / kWaves;  // feature tiles per wave
  extern __shared__ __align__(16) char smem[];
  T* pkT = reinterpret_cast<T*>(smem);      // [DF][32 + kPad]
  T* vT = pkT + DF * (32 + kPad);           // [D][32 + kPad]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hq = lane & 15, lg = lane >> 4;
  const int sg = blockIdx.x, g = blockIdx.y;
  const int bl = find_seq(a, sg);
  const SeqRows<T, D, DF> sr = seq_rows<T, D, DF>(a, bl, g);
  const int sigma = sg - a.seg_base[bl];
  const int s_lo = sigma * a.seg_len, s_hi = min(a.seq_len[bl], s_lo + a.seg_len);
  int64_t jlo = sr.p0 + s_lo - a.W, jhi = sr.p0 + s_hi - a.W;
  if (jlo < 0) jlo = 0;

  f32x4_t sacc[FTW][CT];
#pragma unroll
  for (int x = 0; x < FTW; ++x)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) sacc[x][ct] = zero4();
  float zinc = 0.f;
  for (int64_t j0 = jlo; j0 < jhi; j0 += 32) {
    __syncthreads();
    stage32<T, DF>(nullptr, pkT, [&](int r) { return j0 + r < jhi ? sr.phk(j0 + r) : nullptr; });
    stage32<T, D>(nullptr, vT, [&](int r) { return j0 + r < jhi ? sr.v(j0 + r) : nullptr; });
    __syncthreads();
#pragma unroll
    for (int x = 0; x < FTW; ++x) {
      Frag<T> fa;
      fa.load(pkT + (16 * (wave * FTW + x) + hq) * (32 + kPad) + 8 * lg);
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) {
        Frag<T> fb;
        fb.load(vT + (16 * ct + hq) * (32 + kPad) + 8 * lg);
        sacc[x][ct] = mma(fa, fb, sacc[x][ct]);
      }
    }
    if (tid < DF) {
#pragma unroll 8
      for (int r = 0; r < 32; ++r) zinc += to_f32(pkT[tid * (32 + kPad) + r]);
    }
  }
  float* rec = a.seg + (int64_t(a.seg0 + sg) * a.Hkv + g) * (int64_t(DF) * D + DF);
#pragma unroll
  for (int x = 0; x < FTW; ++x)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int i = 0; i < 4; ++i) rec[(16 * (wave * FTW + x) + 4 * lg + i) * D + 16 * ct + hq] = sacc[x][ct][i];
  if (tid < DF) rec[DF * D + tid] = zinc;
}

// ---------------------------------------------------------------------------
// scan: rec[sigma] <- S_in + sum_{sigma' < sigma} dS_sigma'; state <- total
template <typename T, int D, int DF>
__global__ __launch_bounds__(kThreads) void prefill_scan(PrefillArgs a) {
  constexpr int E = DF * D + DF;
  const int bl = blockIdx.y, g = blockIdx.z, b = a.seq0 + bl;
  const int e = 4 * (blockIdx.x * kThreads + threadIdx.x);
  if (e >= E) return;
  const LayerSections sec = layer_sections(a.B, a.Hkv, D, DF, a.R, sizeof(T));
  const int64_t unit = int64_t(b) * a.Hkv + g;
  float* st = e < DF * D ? reinterpret_cast<float*>(a.state + a.layer_base + sec.S) + unit * DF * D + e
                         : reinterpret_cast<float*>(a.state + a.layer_base + sec.z) + unit * DF + (e - DF * D);
  float4 run = *reinterpret_cast<const float4*>(st);
  for (int sg = a.seg_base[bl]; sg < a.seg_base[bl + 1]; ++sg) {
    float4* rec = reinterpret_cast<float4*>(a.seg + (int64_t(a.seg0 + sg) * a.Hkv + g) * E + e);
    const float4 d = *rec;
    *rec = run;
    run.x += d.x; run.y += d.y; run.z += d.z; run.w += d.w;
  }
  *reinterpret_cast<float4*>(st) = run;
}

// ---------------------------------------------------------------------------
// main: outputs of one segment
template <typename T, int D, int DF>
__global__ __launch_bounds__(kThreads) void prefill_main(PrefillArgs a) {
  constexpr int KS = D / 32, KSF = DF / 32, CT = D / 16;
  constexpr int FTW = DF / 16 / kWaves;
  constexpr int SROW = DF + kPad;  // sT row stride
  extern __shared__ __align__(16) char smem[];
  T* sT = reinterpret_cast<T*>(smem);                                        // [D][DF + kPad]: S^T
  float* zs = reinterpret_cast<float*>(smem + size_t(D) * SROW * sizeof(T));  // [DF]
  T* reg = reinterpret_cast<T*>(smem + size_t(D) * SROW * sizeof(T) + DF * 4);
  // band tiles
  T* kt = reg;                        // [32][D + kPad]
  T* vt = kt + 32 * (D + kPad);       // [D][32 + kPad]
  // chunk slab (aliases the band tiles)
  T* pk = reg;                        // [32][DF + kPad]
  T* pkT = pk + 32 * (DF + kPad);     // [DF][32 + kPad]
  T* vT = pkT + DF * (32 + kPad);     // [D][32 + kPad]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hq = lane & 15, lg = lane >> 4;
  const int sg = blockIdx.x, g = blockIdx.y;
  const int bl = find_seq(a, sg);
  const SeqRows<T, D, DF> sr = seq_rows<T, D, DF>(a, bl, g);
  const int sigma = sg - a.seg_base[bl];
  const int s_lo = sigma * a.seg_len, s_hi = min(a.seq_len[bl], s_lo + a.seg_len);
  const int G = a.G, W = a.W;
  const bool linear = a.linear != 0;
  const float sc2 = a.tau * kLog2e;
  const T* Q = static_cast<const T*>(a.q);
  const T* PQ = static_cast<const T*>(a.phq);
  T* O = static_cast<T*>(a.out);

  // S carried across the segment's chunks: wave w owns feature tiles
  // w*FTW .. w*FTW+FTW-1 (rows f), all column tiles (c).
  f32x4_t sacc[FTW][CT];
  if (linear) {
    const float* S0 = a.seg + (int64_t(a.seg0 + sg) * a.Hkv + g) * (int64_t(DF) * D + DF);
#pragma unroll
    for (int x = 0; x < FTW; ++x)
#pragma unroll
      for (int ct = 0; ct < CT; ++ct)
#pragma unroll
        for (int i = 0; i < 4; ++i) sacc[x][ct][i] = S0[(16 * (wave * FTW + x) + 4 * lg + i) * D + 16 * ct + hq];
    for (int f = tid; f < DF; f += kThreads) zs[f] = S0[DF * D + f];
#pragma unroll
    for (int x = 0; x < FTW; ++x)
#pragma unroll
      for (int ct = 0; ct < CT; ++ct)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          sT[(16 * ct + hq) * SROW + 16 * (wave * FTW + x) + 4 * lg + i] = from_f32<T>(sacc[x][ct][i]);
  }
  __syncthreads();

  for (int c0 = s_lo; c0 < s_hi; c0 += a.C) {
    const int c1 = min(s_hi, c0 + a.C);
    const int64_t t0 = sr.p0 + c0;  // absolute position of the chunk's first token
    const int rows = (c1 - c0) * G;
    const int npass = (rows + 127) / 128;
    float zinc = 0.f;
    for (int pass = 0; pass < npass; ++pass) {
      const bool last = pass == npass - 1;
      const int r_end = min(rows, 128 * (pass + 1));
      const int ti_min = (128 * pass) / G, ti_max = (r_end - 1) / G;  // chunk-relative tokens of the pass
      // this lane's query row in the score layout, per q-tile
      int ti[2], hh[2];
      bool rv[2];
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) {
        const int r = 128 * pass + 32 * wave + 16 * qt + hq;
        rv[qt] = r < rows;
        const int rr = rv[qt] ? r : 128 * pass;
        ti[qt] = rr / G;
        hh[qt] = rr - ti[qt] * G;
      }
      f32x4_t acc[2][CT];
#pragma unroll
      for (int qt = 0; qt < 2; ++qt)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) acc[qt][ct] = zero4();
      float m_run[2] = {-INFINITY, -INFINITY}, l_run[2] = {0.f, 0.f};

      if (linear) {
        Frag<T> pqf[2][KSF];
#pragma unroll
        for (int qt = 0; qt < 2; ++qt)
#pragma unroll
          for (int kk = 0; kk < KSF; ++kk) pqf[qt][kk].load(PQ + sr.qrow(c0 + ti[qt], hh[qt]) * DF + 32 * kk + 8 * lg);
        // read-out phi(q) . S_c
#pragma unroll
        for (int kk = 0; kk < KSF; ++kk) {
#pragma unroll
          for (int ct = 0; ct < CT; ++ct) {
            Frag<T> fb;
            fb.load(sT + (16 * ct + hq) * SROW + 32 * kk + 8 * lg);
#pragma unroll
            for (int qt = 0; qt < 2; ++qt) acc[qt][ct] = mma(pqf[qt][kk], fb, acc[qt][ct]);
          }
        }
        float den[2];
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) {
          float dz = 0.f;
#pragma unroll
          for (int kk = 0; kk < KSF; ++kk) {
            // phi(q)_f * z_f over this lane's 8 features of the slab
            float qv[8];
            pqf[qt][kk].to_floats(qv);
            const float* zz = zs + 32 * kk + 8 * lg;
#pragma unroll
            for (int e = 0; e < 8; ++e) dz = fmaf(qv[e], zz[e], dz);
          }
          den[qt] = dz;
        }
        // intra-chunk block: delayed keys i' in [0, ti], j = t0 - W + i'
        for (int s0 = 0; s0 <= ti_max; s0 += 32) {
          __syncthreads();
          const int nk = c1 - c0;
          auto key = [&](int r) -> int64_t { return t0 - W + s0 + r; };
          stage32<T, DF>(pk, last ? pkT : nullptr, [&](int r) {
            return (s0 + r < nk && key(r) >= 0) ? sr.phk(key(r)) : nullptr;
          });
          stage32<T, D>(nullptr, vT, [&](int r) { return (s0 + r < nk && key(r) >= 0) ? sr.v(key(r)) : nullptr; });
          __syncthreads();
          f32x4_t sc[2][2];
#pragma unroll
          for (int qt = 0; qt < 2; ++qt) sc[qt][0] = sc[qt][1] = zero4();
#pragma unroll
          for (int t = 0; t < 2; ++t) {
#pragma unroll
            for (int kk = 0; kk < KSF; ++kk) {
              Frag<T> fa;
              fa.load(pk + (8 * (hq >> 2) + 4 * t + (hq & 3)) * (DF + kPad) + 32 * kk + 8 * lg);
#pragma unroll
              for (int qt = 0; qt < 2; ++qt) sc[qt][t] = mma(fa, pqf[qt][kk], sc[qt][t]);
            }
          }
          Frag<T> pf[2];
#pragma unroll
          for (int qt = 0; qt < 2; ++qt) {
            float pv[8];
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
              for (int i = 0; i < 4; ++i) pv[4 * t + i] = (s0 + 8 * lg + 4 * t + i <= ti[qt]) ? sc[qt][t][i] : 0.f;
            pf[qt].set8(pv);
            den[qt] += pf[qt].sum();
          }
#pragma unroll
          for (int ct = 0; ct < CT; ++ct) {
            Frag<T> fb;
            fb.load(vT + (16 * ct + hq) * (32 + kPad) + 8 * lg);
#pragma unroll
            for (int qt = 0; qt < 2; ++qt) acc[qt][ct] = mma(pf[qt], fb, acc[qt][ct]);
          }
          if (last) {
            // the chunk's state increment (all delayed keys are covered by the last pass)
#pragma unroll
            for (int x = 0; x < FTW; ++x) {
              Frag<T> fa;
              fa.load(pkT + (16 * (wave * FTW + x) + hq) * (32 + kPad) + 8 * lg);
#pragma unroll
              for (int ct = 0; ct < CT; ++ct) {
                Frag<T> fb;
                fb.load(vT + (16 * ct + hq) * (32 + kPad) + 8 * lg);
                sacc[x][ct] = mma(fa, fb, sacc[x][ct]);
              }
            }
            if (tid < DF) {
#pragma unroll 8
              for (int r = 0; r < 32; ++r) zinc += to_f32(pkT[tid * (32 + kPad) + r]);
            }
          }
        }
        // the linear part as the starting state of the online softmax
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) {
          float dn = den[qt];
          dn += __shfl_xor(dn, 16);
          dn += __shfl_xor(dn, 32);
          m_run[qt] = dn > 0.f ? log2f(dn) : -INFINITY;
          l_run[qt] = (dn > 0.f && lg == 0) ? 1.f : 0.f;
          const float inv = dn > 0.f ? 1.f / dn : 0.f;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float ir = __shfl(inv, 4 * lg + i);
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) acc[qt][ct][i] *= ir;
          }
        }
      }

      // banded window attention, keys [t0 + ti_min - W + 1, t0 + ti_max]
      if (W > 0) {
        Frag<T> qf[2][KS];
#pragma unroll
        for (int qt = 0; qt < 2; ++qt)
#pragma unroll
          for (int kk = 0; kk < KS; ++kk) qf[qt][kk].load(Q + sr.qrow(c0 + ti[qt], hh[qt]) * D + 32 * kk + 8 * lg);
        int64_t klo = t0 + ti_min - W + 1;
        if (klo < 0) klo = 0;
        const int64_t khi = t0 + ti_max;
        for (int64_t kb = klo & ~int64_t(31); kb <= khi; kb += 32) {
          __syncthreads();
          stage32<T, D>(kt, nullptr, [&](int r) { return (kb + r >= klo && kb + r <= khi) ? sr.k(kb + r) : nullptr; });
          stage32<T, D>(nullptr, vt, [&](int r) { return (kb + r >= klo && kb + r <= khi) ? sr.v(kb + r) : nullptr; });
          __syncthreads();
          f32x4_t sc[2][2];
#pragma unroll
          for (int qt = 0; qt < 2; ++qt) sc[qt][0] = sc[qt][1] = zero4();
#pragma unroll
          for (int t = 0; t < 2; ++t) {
#pragma unroll
            for (int kk = 0; kk < KS; ++kk) {
              Frag<T> fa;
              fa.load(kt + (8 * (hq >> 2) + 4 * t + (hq & 3)) * (D + kPad) + 32 * kk + 8 * lg);
#pragma unroll
              for (int qt = 0; qt < 2; ++qt) sc[qt][t] = mma(fa, qf[qt][kk], sc[qt][t]);
            }
          }
          Frag<T> pf[2];
#pragma unroll
          for (int qt = 0; qt < 2; ++qt) {
            const int64_t tq = t0 + ti[qt];
            float s[8];
            float mx = -INFINITY;
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                const int64_t j = kb + 8 * lg + 4 * t + i;
                const bool ok = rv[qt] && j >= klo && j <= tq && j > tq - W;
                const float v = ok ? sc[qt][t][i] * sc2 : -INFINITY;
                s[4 * t + i] = v;
                mx = fmaxf(mx, v);
              }
            mx = fmaxf(mx, __shfl_xor(mx, 16));
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            const float m_new = fmaxf(m_run[qt], mx);
            const float m_use = m_new == -INFINITY ? 0.f : m_new;
            const float alpha = exp2f(m_run[qt] - m_use);
            float pv[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) pv[i] = exp2f(s[i] - m_use);
            pf[qt].set8(pv);
            l_run[qt] = l_run[qt] * alpha + pf[qt].sum();
            m_run[qt] = m_new;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const float al = __shfl(alpha, 4 * lg + i);
#pragma unroll
              for (int ct = 0; ct < CT; ++ct) acc[qt][ct][i] *= al;
            }
          }
#pragma unroll
          for (int ct = 0; ct < CT; ++ct) {
            Frag<T> fb;
            fb.load(vt + (16 * ct + hq) * (32 + kPad) + 8 * lg);
#pragma unroll
            for (int qt = 0; qt < 2; ++qt) acc[qt][ct] = mma(pf[qt], fb, acc[qt][ct]);
          }
        }
      }

      // outputs of this pass
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) {
        float ls = l_run[qt];
        ls += __shfl_xor(ls, 16);
        ls += __shfl_xor(ls, 32);
        const float inv = ls > 0.f ? 1.f / ls : 0.f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float ir = __shfl(inv, 4 * lg + i);
          const int r = 128 * pass + 32 * wave + 16 * qt + 4 * lg + i;
          if (r < rows) {
            const int tr = r / G, hr = r - tr * G;
            T* orow = O + sr.qrow(c0 + tr, hr) * D;
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) orow[16 * ct + hq] = from_f32<T>(acc[qt][ct][i] * ir);
          }
        }
      }
    }
    // next chunk's state: S^T copy and z
    if (linear) {
      __syncthreads();
      if (tid < DF) zs[tid] += zinc;
#pragma unroll
      for (int x = 0; x < FTW; ++x)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            sT[(16 * ct + hq) * SROW + 16 * (wave * FTW + x) + 4 * lg + i] = from_f32<T>(sacc[x][ct][i]);
      __syncthreads();
    }
  }
}

// ---------------------------------------------------------------------------
// ringfill: tokens [max(p0, p_end - W), p_end) into their ring slots
template <typename T, int D, int DF>
__global__ __launch_bounds__(kThreads) void prefill_ringfill(PrefillArgs a) {
  const int bl = blockIdx.y, g = blockIdx.z;
  const SeqRows<T, D, DF> sr = seq_rows<T, D, DF>(a, bl, g);
  const int Tb = a.seq_len[bl];
  const int64_t pend = sr.p0 + Tb;
  int64_t jlo = pend - a.W;
  if (jlo < sr.p0) jlo = sr.p0;
  const int n = int(pend - jlo);
  if (n <= 0 || a.W == 0) return;
  const LayerSections sec = layer_sections(a.B, a.Hkv, D, DF, a.R, sizeof(T));
  const int64_t unit = int64_t(sr.b) * a.Hkv + g;
  T* Kr = reinterpret_cast<T*>(a.state + a.layer_base + sec.K) + unit * a.R * D;
  T* Vr = reinterpret_cast<T*>(a.state + a.layer_base + sec.V) + unit * a.R * D;
  for (int idx = blockIdx.x * kThreads + threadIdx.x; idx < n * D; idx += gridDim.x * kThreads) {
    const int i = idx / D, c = idx - i * D;
    const int64_t j = jlo + i;
    const int32_t s = int32_t(j % a.R);
    Kr[kring_elem(s, c, D)] = sr.k(j)[c];
    Vr[vring_elem(s, c, D)] = sr.v(j)[c];
  }
}

// advance: pos += T_b (after every other kernel of the layer read pos)
template <typename T, int D, int DF>
__global__ void prefill_advance(PrefillArgs a) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.nseq * a.Hkv) return;
  const int bl = i / a.Hkv, g = i - bl * a.Hkv;
  const LayerSections sec = layer_sections(a.B, a.Hkv, D, DF, a.R, sizeof(T));
  int64_t* pos = reinterpret_cast<int64_t*>(a.state + a.layer_base + sec.pos) + int64_t(a.seq0 + bl) * a.Hkv + g;
  *pos += a.seq_len[bl];
}

template <typename T, int D, int DF>
size_t main_lds() {
  const size_t band = (size_t(32) * (D + kPad) + size_t(D) * (32 + kPad)) * sizeof(T);
  const size_t slab = (size_t(32) * (DF + kPad) + size_t(DF) * (32 + kPad) + size_t(D) * (32 + kPad)) * sizeof(T);
  return size_t(D) * (DF + kPad) * sizeof(T) + DF * 4 + (band > slab ? band : slab);
}

template <typename K>
hipError_t set_lds(K* kern, size_t bytes) {
  if (bytes <= 65536) return hipSuccess;
  return hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                             int(bytes));
}

template <typename T, int D, int DF>
hipError_t layer_t(const PrefillArgs& a, hipStream_t s) {
  hipError_t e;
  if (a.linear && a.nseg > 0) {
    const size_t lds_seg = (size_t(DF) * (32 + kPad) + size_t(D) * (32 + kPad)) * sizeof(T);
    hipLaunchKernelGGL((prefill_segsum<T, D, DF>), dim3(a.nseg, a.Hkv), dim3(kThreads), lds_seg, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const int E = DF * D + DF;
    hipLaunchKernelGGL((prefill_scan<T, D, DF>), dim3((E / 4 + kThreads - 1) / kThreads, a.nseq, a.Hkv),
                       dim3(kThreads), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (a.nseg > 0) {
    const size_t lds = main_lds<T, D, DF>();
    if ((e = set_lds(&prefill_main<T, D, DF>, lds)) != hipSuccess) return e;
    hipLaunchKernelGGL((prefill_main<T, D, DF>), dim3(a.nseg, a.Hkv), dim3(kThreads), lds, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (a.W > 0) {
    hipLaunchKernelGGL((prefill_ringfill<T, D, DF>), dim3(16, a.nseq, a.Hkv), dim3(kThreads), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  hipLaunchKernelGGL((prefill_advance<T, D, DF>), dim3((a.nseq * a.Hkv + 255) / 256), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <typename T, int D, int DF>
hipError_t gather_t(const PrefillArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((prefill_gather<T, D, DF>), dim3(16, a.nseq, a.Hkv), dim3(kThreads), 0, s, a);
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
