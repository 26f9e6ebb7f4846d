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
// Tokens a decode step left pending are folded (glide_state_flush) before the
// first of these kernels runs, so the incoming state is S = sum_{j < p0-W}.
#include <math.h>

#include "glide_internal.h"

namespace glide {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = 4;
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
// Stage 32 token rows of NC elements into LDS, natural layout [32][rs].
// row(r) gives the row pointer, nullptr = zeros.  Contractions over the rows
// read them back with load_colfrag (transposing reads), so no transposed copy
// is ever written.
template <typename T, int NC, typename RowFn>
__device__ __forceinline__ void stage32(T* nat, int rs, RowFn row) {
  constexpr int CPR = NC / 8;
  for (int id = threadIdx.x; id < 32 * CPR; id += kThreads) {
    const int r = id / CPR, ch = id - r * CPR;
    const T* src = row(r);
    Frag<T> f;
    if (src) f.load(src + 8 * ch);
    else f.zero();
    store8(nat + r * rs + 8 * ch, f);
  }
}

// LDS row strides (elements): tiles read with 16-byte fragment loads use a
// padding of 8; tiles read with load_colfrag use 16 so the four rows a
// 16-lane group touches fall on distinct banks.
template <int N> constexpr int row_a() { return N + 8; }
template <int N> constexpr int row_t() { return N + 16; }

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
  constexpr int PROW = row_t<DF>(), VROW = row_t<D>();
  extern __shared__ __align__(16) char smem[];
  T* pk = reinterpret_cast<T*>(smem);       // [32][PROW]  phi(k) of 32 delayed keys
  T* vs = pk + 32 * PROW;                   // [32][VROW]  their values
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
    stage32<T, DF>(pk, PROW, [&](int r) { return j0 + r < jhi ? sr.phk(j0 + r) : nullptr; });
    stage32<T, D>(vs, VROW, [&](int r) { return j0 + r < jhi ? sr.v(j0 + r) : nullptr; });
    __syncthreads();
#pragma unroll
    for (int x = 0; x < FTW; ++x) {
      Frag<T> fa;
      load_colfrag(fa, pk, PROW, 8 * lg, 16 * (wave * FTW + x));
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) {
        Frag<T> fb;
        load_colfrag(fb, vs, VROW, 8 * lg, 16 * ct);
        sacc[x][ct] = mma(fa, fb, sacc[x][ct]);
      }
    }
    if (tid < DF) {
#pragma unroll 8
      for (int r = 0; r < 32; ++r) zinc += to_f32(pk[r * PROW + tid]);
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
// main: the outputs of one (chunk, 128-row pass) of one (sequence, KV head)
//
//   1. S_c, z_c: the segment-start record plus the delayed keys of the
//      segment's earlier chunks (MFMA), kept in LDS in the element type as
//      S^T for the read-out;
//   2. linear part of each query row: phi(q).S_c plus the masked block of the
//      chunk's own delayed keys; it becomes the row's online-softmax start
//      (pseudo-key of weight a, value A/a);
//   3. banded window attention over 32-key tiles staged in LDS, the next
//      tile's global loads in flight while the current one computes;
//   4. O = acc / l.
template <typename T, int D, int DF>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void prefill_main(PrefillArgs a) {
  constexpr int KS = D / 32, KSF = DF / 32, CT = D / 16;
  constexpr int FTW = DF / 16 / kWaves;
  constexpr int SROW = row_a<DF>();           // sT row stride
  constexpr int KROW = row_a<D>(), VROW = row_t<D>(), PROW = row_t<DF>();
  constexpr int BAND = 32 * KROW + 32 * VROW;  // one band buffer (elements)
  constexpr int CPR = D / 8;                  // 8-element chunks per K/V row
  constexpr int NLD = 32 * CPR / kThreads;    // chunks per thread per tile (K and V each)
  static_assert(NLD * kThreads == 32 * CPR, "tile staging must divide evenly");
  extern __shared__ __align__(16) char smem[];
  T* sT = reinterpret_cast<T*>(smem);                                        // [D][SROW]
  float* zs = reinterpret_cast<float*>(smem + size_t(D) * SROW * sizeof(T));  // [DF]
  T* reg = reinterpret_cast<T*>(smem + size_t(D) * SROW * sizeof(T) + DF * 4);
  T* pk = reg;                        // slab: phi(k) of 32 delayed keys [32][PROW]
  T* vs = pk + 32 * PROW;             //       their values               [32][VROW]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hq = lane & 15, lg = lane >> 4;
  const int wgi = blockIdx.x, g = blockIdx.y;
  int bl = 0;
  while (bl + 1 < a.nseq && a.wg_base[bl + 1] <= wgi) ++bl;
  const int local = wgi - a.wg_base[bl];
  const int chunk = local / a.npass, pass = local - chunk * a.npass;
  const int Tb = a.seq_len[bl];
  const int c0 = chunk * a.C, c1 = min(Tb, c0 + a.C);
  const int G = a.G, W = a.W;
  const int rows = (c1 - c0) * G;
  if (128 * pass >= rows) return;
  const SeqRows<T, D, DF> sr = seq_rows<T, D, DF>(a, bl, g);
  const bool linear = a.linear != 0;
  const float sc2 = a.tau * kLog2e;
  const int64_t t0 = sr.p0 + c0;  // absolute position of the chunk's first token
  const int r_end = min(rows, 128 * (pass + 1));
  const int ti_min = (128 * pass) / G, ti_max = (r_end - 1) / G;  // chunk-relative tokens of the pass

  // ---- 1. S_c and z_c
  if (linear) {
    const int sigma = c0 / a.seg_len;
    const float* S0 = a.seg + (int64_t(a.seg0 + a.seg_base[bl] + sigma) * a.Hkv + g) * (int64_t(DF) * D + DF);
    f32x4_t sacc[FTW][CT];
#pragma unroll
    for (int x = 0; x < FTW; ++x)
#pragma unroll
      for (int ct = 0; ct < CT; ++ct)
#pragma unroll
        for (int i = 0; i < 4; ++i) sacc[x][ct][i] = S0[(16 * (wave * FTW + x) + 4 * lg + i) * D + 16 * ct + hq];
    float zacc = tid < DF ? S0[DF * D + tid] : 0.f;
    // delayed keys of the segment's earlier chunks: j in [p0 + sigma*seg_len - W, t0 - W)
    int64_t jlo = sr.p0 + int64_t(sigma) * a.seg_len - W;
    const int64_t jhi = t0 - W;
    if (jlo < 0) jlo = 0;
    for (int64_t j0 = jlo; j0 < jhi; j0 += 32) {
      __syncthreads();
      stage32<T, DF>(pk, PROW, [&](int r) { return j0 + r < jhi ? sr.phk(j0 + r) : nullptr; });
      stage32<T, D>(vs, VROW, [&](int r) { return j0 + r < jhi ? sr.v(j0 + r) : nullptr; });
      __syncthreads();
#pragma unroll
      for (int x = 0; x < FTW; ++x) {
        Frag<T> fa;
        load_colfrag(fa, pk, PROW, 8 * lg, 16 * (wave * FTW + x));
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
          Frag<T> fb;
          load_colfrag(fb, vs, VROW, 8 * lg, 16 * ct);
          sacc[x][ct] = mma(fa, fb, sacc[x][ct]);
        }
      }
      if (tid < DF) {
#pragma unroll 8
        for (int r = 0; r < 32; ++r) zacc += to_f32(pk[r * PROW + tid]);
      }
    }
#pragma unroll
    for (int x = 0; x < FTW; ++x)
#pragma unroll
      for (int ct = 0; ct < CT; ++ct)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          sT[(16 * ct + hq) * SROW + 16 * (wave * FTW + x) + 4 * lg + i] = from_f32<T>(sacc[x][ct][i]);
    if (tid < DF) zs[tid] = zacc;
  }
  __syncthreads();

  // this lane's query rows (score layout: row = hq of each 16-row q-tile)
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

  // ---- 2. linear part
  if (linear) {
    const T* PQ = static_cast<const T*>(a.phq);
    Frag<T> pqf[2][KSF];
#pragma unroll
    for (int qt = 0; qt < 2; ++qt)
#pragma unroll
      for (int kk = 0; kk < KSF; ++kk) pqf[qt][kk].load(PQ + sr.qrow(c0 + ti[qt], hh[qt]) * DF + 32 * kk + 8 * lg);
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
        float qv[8];
        pqf[qt][kk].to_floats(qv);
        const float* zz = zs + 32 * kk + 8 * lg;
#pragma unroll
        for (int e = 0; e < 8; ++e) dz = fmaf(qv[e], zz[e], dz);
      }
      den[qt] = dz;
    }
    // the chunk's own delayed keys i' in [0, ti], key j = t0 - W + i'
    const int nk = c1 - c0;
    for (int s0 = 0; s0 <= ti_max; s0 += 32) {
      __syncthreads();
      stage32<T, DF>(pk, PROW, [&](int r) {
        const int64_t j = t0 - W + s0 + r;
        return (s0 + r < nk && j >= 0) ? sr.phk(j) : nullptr;
      });
      stage32<T, D>(vs, VROW, [&](int r) {
        const int64_t j = t0 - W + s0 + r;
        return (s0 + r < nk && j >= 0) ? sr.v(j) : nullptr;
      });
      __syncthreads();
      f32x4_t sc[2][2];
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) sc[qt][0] = sc[qt][1] = zero4();
#pragma unroll
      for (int t = 0; t < 2; ++t) {
#pragma unroll
        for (int kk = 0; kk < KSF; ++kk) {
          Frag<T> fa;
          fa.load(pk + (8 * (hq >> 2) + 4 * t + (hq & 3)) * PROW + 32 * kk + 8 * lg);
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
        load_colfrag(fb, vs, VROW, 8 * lg, 16 * ct);
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) acc[qt][ct] = mma(pf[qt], fb, acc[qt][ct]);
      }
    }
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

  // ---- 3. banded window attention, keys [t0 + ti_min - W + 1, t0 + ti_max]
  if (W > 0) {
    const T* Q = static_cast<const T*>(a.q);
    Frag<T> qf[2][KS];
#pragma unroll
    for (int qt = 0; qt < 2; ++qt)
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) qf[qt][kk].load(Q + sr.qrow(c0 + ti[qt], hh[qt]) * D + 32 * kk + 8 * lg);
    int64_t klo = t0 + ti_min - W + 1;
    if (klo < 0) klo = 0;
    const int64_t khi = t0 + ti_max;
    const int64_t kb0 = klo & ~int64_t(31);
    const int ntile = int((khi - kb0) / 32) + 1;
    // staging registers: this thread's chunks of the next tile
    Frag<T> sk[NLD], sv[NLD];
    auto fetch = [&](int n) {
      const int64_t kb = kb0 + 32 * int64_t(n);
#pragma unroll
      for (int u = 0; u < NLD; ++u) {
        const int id = tid + u * kThreads, r = id / CPR, ch = id - r * CPR;
        const int64_t j = kb + r;
        const bool ok = j >= klo && j <= khi;
        if (ok) {
          sk[u].load(sr.k(j) + 8 * ch);
          sv[u].load(sr.v(j) + 8 * ch);
        } else {
          sk[u].zero();
          sv[u].zero();
        }
      }
    };
    auto store = [&](int buf) {
      T* kt = reg + buf * BAND;
      T* vt = kt + 32 * KROW;
#pragma unroll
      for (int u = 0; u < NLD; ++u) {
        const int id = tid + u * kThreads, r = id / CPR, ch = id - r * CPR;
        store8(kt + r * KROW + 8 * ch, sk[u]);
        store8(vt + r * VROW + 8 * ch, sv[u]);
      }
    };
    __syncthreads();  // the slab region is free again
    fetch(0);
    store(0);
    __syncthreads();
    for (int n = 0; n < ntile; ++n) {
      if (n + 1 < ntile) fetch(n + 1);
      const T* kt = reg + (n & 1) * BAND;
      const T* vt = kt + 32 * KROW;
      const int64_t kb = kb0 + 32 * int64_t(n);
      f32x4_t sc[2][2];
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) sc[qt][0] = sc[qt][1] = zero4();
#pragma unroll
      for (int t = 0; t < 2; ++t) {
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) {
          Frag<T> fa;
          fa.load(kt + (8 * (hq >> 2) + 4 * t + (hq & 3)) * KROW + 32 * kk + 8 * lg);
#pragma unroll
          for (int qt = 0; qt < 2; ++qt) sc[qt][t] = mma(fa, qf[qt][kk], sc[qt][t]);
        }
      }
      // keys [kb, kb+31] lie inside the band of every row of the pass
      // (tokens t0+ti_min .. t0+ti_max) for all but the edge tiles
      const bool interior = kb >= t0 + ti_max - W + 1 && kb + 31 <= t0 + ti_min;
      Frag<T> pf[2];
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) {
        float sv8[8];
        if (interior) {
#pragma unroll
          for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i) sv8[4 * t + i] = sc[qt][t][i] * sc2;
        } else {
          // j - tq = base + off;  valid: j >= klo, tq - W < j <= tq, row exists
          const int base = int(kb - (t0 + ti[qt]));
          const int64_t offlo = klo - kb;  // first in-band offset of the tile (<= 31)
          const int lo = offlo < -1 ? -1 : int(offlo);
#pragma unroll
          for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int off = 8 * lg + 4 * t + i;
              const bool ok = rv[qt] && off >= lo && base + off <= 0 && base + off > -W;
              sv8[4 * t + i] = ok ? sc[qt][t][i] * sc2 : -INFINITY;
            }
        }
        float mx = sv8[0];
#pragma unroll
        for (int i = 1; i < 8; ++i) mx = fmaxf(mx, sv8[i]);
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        // lazy rescale: the running max moves only when a score exceeds it by
        // more than 2^8, so p = 2^(s - m) <= 256 and acc, l stay in range
        if (__any(mx > m_run[qt] + 8.f)) {
          const float m_new = fmaxf(m_run[qt], mx);
          const float alpha = m_new == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m_run[qt] - m_new);
          l_run[qt] *= alpha;
          m_run[qt] = m_new;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float al = __shfl(alpha, 4 * lg + i);
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) acc[qt][ct][i] *= al;
          }
        }
        const float m_use = m_run[qt] == -INFINITY ? 0.f : m_run[qt];
        float pv[8], ps = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          pv[i] = __builtin_amdgcn_exp2f(sv8[i] - m_use);
          ps += pv[i];
        }
        pf[qt].set8(pv);
        l_run[qt] += ps;
      }
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) {
        Frag<T> fb;
        load_colfrag(fb, vt, VROW, 8 * lg, 16 * ct);
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) acc[qt][ct] = mma(pf[qt], fb, acc[qt][ct]);
      }
      if (n + 1 < ntile) store((n + 1) & 1);
      __syncthreads();
    }
  }

  // ---- 4. outputs
  T* O = static_cast<T*>(a.out);
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

// advance: pos += T_b (after every other kernel of the layer read pos); the
// scan left S, z = the sums over tokens [0, max(0, pos - W)), nothing pending.
template <typename T, int D, int DF>
__global__ void prefill_advance(PrefillArgs a) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.nseq * a.Hkv) return;
  const int bl = i / a.Hkv, g = i - bl * a.Hkv;
  const LayerSections sec = layer_sections(a.B, a.Hkv, D, DF, a.R, sizeof(T));
  const int64_t unit = int64_t(a.seq0 + bl) * a.Hkv + g;
  int64_t* pos = reinterpret_cast<int64_t*>(a.state + a.layer_base + sec.pos) + unit;
  int64_t* nf = reinterpret_cast<int64_t*>(a.state + a.layer_base + sec.nf) + unit;
  const int64_t p = *pos + a.seq_len[bl];
  *pos = p;
  *nf = p - a.W > 0 ? p - a.W : 0;
}

template <typename T, int D, int DF>
size_t main_lds() {
  const size_t band = 2 * (size_t(32) * row_a<D>() + size_t(32) * row_t<D>()) * sizeof(T);
  const size_t slab = (size_t(32) * row_t<DF>() + size_t(32) * row_t<D>()) * sizeof(T);
  return size_t(D) * row_a<DF>() * sizeof(T) + DF * 4 + (band > slab ? band : slab);
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
    const size_t lds_seg = (size_t(32) * row_t<DF>() + size_t(32) * row_t<D>()) * sizeof(T);
    hipLaunchKernelGGL((prefill_segsum<T, D, DF>), dim3(a.nseg, a.Hkv), dim3(kThreads), lds_seg, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const int E = DF * D + DF;
    hipLaunchKernelGGL((prefill_scan<T, D, DF>), dim3((E / 4 + kThreads - 1) / kThreads, a.nseq, a.Hkv),
                       dim3(kThreads), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (a.wg_base[a.nseq] > 0) {
    const size_t lds = main_lds<T, D, DF>();
    if ((e = set_lds(&prefill_main<T, D, DF>, lds)) != hipSuccess) return e;
    hipLaunchKernelGGL((prefill_main<T, D, DF>), dim3(a.wg_base[a.nseq], a.Hkv), dim3(kThreads), lds, s, a);
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
