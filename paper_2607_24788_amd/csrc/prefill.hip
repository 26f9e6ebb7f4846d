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
//   main     per (segment, KV head): the segment's chunks in order, S carried
//            in fp32 MFMA accumulators.  Per chunk: phi(q) on MFMA from the
//            query rows; the linear read-out phi(Q)S_c plus the masked block
//            of the chunk's delayed keys (whose phi(k) is computed once and
//            also feeds S_{c+1}) start every query row's online softmax as one
//            pseudo-key of weight a = phi(q).z_c + the block's weights and
//            value A/a (exactly the shared-denominator merge); then the banded
//            window attention over LDS-staged key tiles on MFMA;
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
constexpr int kMT = 512;       // main kernel: 8 waves, 32 query rows each
constexpr int kMW = 8;
constexpr int kRB = 32 * kMW;  // query rows per pass of a chunk
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

template <typename T, int D, int DF>
__device__ __forceinline__ SeqRows<T, D> seq_rows(const PrefillArgs& a, int bl, int g) {
  SeqRows<T, D> r;
  r.b = a.seq0 + bl;
  r.g = g;
  r.start = a.seq_start[bl];
  r.Hq = a.Hq;
  r.Hkv = a.Hkv;
  r.G = a.G;
  const int64_t unit = int64_t(r.b) * a.Hkv + g;
  r.kin = static_cast<const T*>(a.k);
  r.vin = static_cast<const T*>(a.v);
  r.kh = static_cast<const T*>(a.hk) + unit * a.Wcap * D;
  r.vh = static_cast<const T*>(a.hv) + unit * a.Wcap * D;
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

// Wf [D][DF] into LDS, natural layout (nthreads cooperating).
template <typename T, int D, int DF>
__device__ __forceinline__ void stage_wf(const T* Wf, T* Wn, int nthreads) {
  constexpr int WROW = row_t<DF>();
  for (int i = threadIdx.x; i < D * DF / 8; i += nthreads) {
    const int r = i / (DF / 8), ch = i - r * (DF / 8);
    Frag<T> f;
    f.load(Wf + r * DF + 8 * ch);
    store8(Wn + r * WROW + 8 * ch, f);
  }
}

// phi of 32 keys into LDS pk[32][row_t<DF>] (element type, natural layout).
// The 2 x DF/16 output tiles are spread over the nw waves of the workgroup;
// every tile of a wave has the same key tile (2*DF/16 is a multiple of nw), so
// a wave loads the key rows of its tile once (slab_keys), and the loads can be
// issued well before phi_slab consumes them.
template <typename T, int D, int DF>
struct SlabKeys {
  Frag<T> x[D / 32];
};
template <typename T, int D, int DF, typename RowFn>
__device__ __forceinline__ void slab_keys(SlabKeys<T, D, DF>& sk, int nw, RowFn krow) {
  constexpr int FT = DF / 16;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, hq = lane & 15, lg = lane >> 4;
  const int kt = (wave * (2 * FT / nw)) / FT;
  const T* src = krow(16 * kt + hq);
#pragma unroll
  for (int kk = 0; kk < D / 32; ++kk) {
    if (src) sk.x[kk].load(src + 32 * kk + 8 * lg);
    else sk.x[kk].zero();
  }
}
template <typename T, int D, int DF, bool kLds>
__device__ __forceinline__ void phi_slab(const WfCols<T, D, DF, kLds>& wf, const SlabKeys<T, D, DF>& sk, T* pk,
                                         int nw) {
  constexpr int KS = D / 32, FT = DF / 16, PROW = row_t<DF>();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, hq = lane & 15, lg = lane >> 4;
  const int per = 2 * FT / nw;  // tiles per wave
  for (int u = 0; u < per; ++u) {
    const int tile = wave * per + u, kt = tile / FT, ft = tile - kt * FT;
    f32x4_t acc = zero4();
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      Frag<T> wb;
      wf.col(wb, kk, 16 * ft);
      acc = mma(sk.x[kk], wb, acc);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) pk[(16 * kt + 4 * lg + i) * PROW + 16 * ft + hq] = from_f32<T>(fmaxf(acc[i], 0.f));
  }
}

// ---------------------------------------------------------------------------
// gather: history tokens [h0, p0) of a continuing prefill, ring -> [b][g][Wcap][d]
template <typename T, int D, int DF>
__global__ __launch_bounds__(kThreads) void prefill_gather(PrefillArgs a) {
  const int bl = blockIdx.y, g = blockIdx.z;
  const SeqRows<T, D> sr = seq_rows<T, D, DF>(a, bl, g);
  const int n = int(sr.p0 - sr.h0);
  if (n <= 0) return;
  const LayerSections sec = layer_sections(a.B, a.Hkv, D, DF, a.R, sizeof(T));
  const int64_t unit = int64_t(sr.b) * a.Hkv + g;
  const T* Kr = reinterpret_cast<const T*>(a.state + a.layer_base + sec.K) + unit * a.R * D;
  const T* Vr = reinterpret_cast<const T*>(a.state + a.layer_base + sec.V) + unit * a.R * D;
  T* hk = static_cast<T*>(a.hk) + unit * a.Wcap * D;
  T* hv = static_cast<T*>(a.hv) + unit * a.Wcap * D;
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
  constexpr int CT = D / 16, FT = DF / 16;
  constexpr int NT = FT * CT / kWaves;  // output tiles per wave
  constexpr int WROW = row_t<DF>(), PROW = row_t<DF>(), VROW = row_t<D>();
  extern __shared__ __align__(16) char smem[];
  T* Wn = reinterpret_cast<T*>(smem);  // [D][WROW]   Wf
  T* pk = Wn + D * WROW;                // [32][PROW]  phi(k) of 32 delayed keys
  T* vs = pk + 32 * PROW;               // [32][VROW]  their values
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hq = lane & 15, lg = lane >> 4;
  const int sg = blockIdx.x, g = blockIdx.y;
  const int bl = find_seq(a, sg);
  const SeqRows<T, D> sr = seq_rows<T, D, DF>(a, bl, g);
  const int sigma = sg - a.seg_base[bl];
  const int s_lo = sigma * a.seg_len, s_hi = min(a.seq_len[bl], s_lo + a.seg_len);
  int64_t jlo = sr.p0 + s_lo - a.W;
  const int64_t jhi = sr.p0 + s_hi - a.W;
  if (jlo < 0) jlo = 0;
  stage_wf<T, D, DF>(static_cast<const T*>(a.wf), Wn, kThreads);
  const WfCols<T, D, DF, true> wf{Wn};

  f32x4_t sacc[NT];
#pragma unroll
  for (int x = 0; x < NT; ++x) sacc[x] = zero4();
  float zinc = 0.f;
  // the next slab's key rows and values are loaded while the current one is
  // computed
  constexpr int VPT = 32 * D / 8 / kThreads;  // value chunks per thread
  SlabKeys<T, D, DF> kx;
  Frag<T> vx[VPT];
  auto load_slab = [&](int64_t j0) {
    slab_keys(kx, kWaves, [&](int r) { return j0 + r < jhi ? sr.k(j0 + r) : nullptr; });
#pragma unroll
    for (int u = 0; u < VPT; ++u) {
      const int id = tid + u * kThreads, r = id / (D / 8), ch = id - r * (D / 8);
      if (j0 + r < jhi) vx[u].load(sr.v(j0 + r) + 8 * ch);
      else vx[u].zero();
    }
  };
  if (jlo < jhi) load_slab(jlo);
  for (int64_t j0 = jlo; j0 < jhi; j0 += 32) {
    __syncthreads();
    phi_slab(wf, kx, pk, kWaves);
#pragma unroll
    for (int u = 0; u < VPT; ++u) {
      const int id = tid + u * kThreads, r = id / (D / 8), ch = id - r * (D / 8);
      store8(vs + r * VROW + 8 * ch, vx[u]);
    }
    if (j0 + 32 < jhi) load_slab(j0 + 32);
    __syncthreads();
#pragma unroll
    for (int x = 0; x < NT; ++x) {
      const int tile = wave * NT + x, ft = tile / CT, ct = tile - ft * CT;
      Frag<T> fa, fb;
      load_colfrag(fa, pk, PROW, 8 * lg, 16 * ft);
      load_colfrag(fb, vs, VROW, 8 * lg, 16 * ct);
      sacc[x] = mma(fa, fb, sacc[x]);
    }
    if (tid < DF) {
#pragma unroll 8
      for (int r = 0; r < 32; ++r) zinc += to_f32(pk[r * PROW + tid]);
    }
  }
  float* rec = a.seg + (int64_t(a.seg0 + sg) * a.Hkv + g) * (int64_t(DF) * D + DF);
#pragma unroll
  for (int x = 0; x < NT; ++x) {
    const int tile = wave * NT + x, ft = tile / CT, ct = tile - ft * CT;
#pragma unroll
    for (int i = 0; i < 4; ++i) rec[(16 * ft + 4 * lg + i) * D + 16 * ct + hq] = sacc[x][i];
  }
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
// main: the outputs of one segment of one (sequence, KV head), chunk by chunk.
template <typename T, int D, int DF>
struct MainLds {
  static constexpr int NBUF = sizeof(T) == 2 ? 2 : 1;  // band stages (fp32: one, to fit)
  static constexpr int WROW = row_t<DF>(), PROW = row_t<DF>(), VROW = row_t<D>();
  static constexpr int SROW = D + 4;                   // fp32 S: 4 rows of a 16-lane group on distinct banks
  static constexpr int KROW = row_a<D>();
  static constexpr int BAND = 32 * KROW + 32 * VROW;  // one band buffer (elements)
  static constexpr size_t rest = size_t(DF) * SROW * 4 + size_t(DF) * 4 + size_t(32) * PROW * sizeof(T) +
                                 size_t(32) * VROW * sizeof(T) + size_t(NBUF) * BAND * sizeof(T);
  // Wf in LDS when it fits beside the rest (all but fp32 with d = Df = 128,
  // which reads it from global memory)
  static constexpr bool kWfLds = size_t(D) * WROW * sizeof(T) + rest <= 160 * 1024;
  static constexpr size_t wn = 0;
  static constexpr size_t sn = wn + (kWfLds ? size_t(D) * WROW * sizeof(T) : 0);
  static constexpr size_t zs = sn + size_t(DF) * SROW * 4;
  static constexpr size_t pk = zs + size_t(DF) * 4;
  static constexpr size_t vs = pk + size_t(32) * PROW * sizeof(T);
  static constexpr size_t band = vs + size_t(32) * VROW * sizeof(T);
  static constexpr size_t bytes = band + size_t(NBUF) * BAND * sizeof(T);
};

template <typename T, int D, int DF>
__global__ __launch_bounds__(kMT) __attribute__((amdgpu_waves_per_eu(2, 2)))
void prefill_main(PrefillArgs a) {
  using LD = MainLds<T, D, DF>;
  constexpr int KS = D / 32, KSF = DF / 32, CT = D / 16, FT = DF / 16;
  constexpr int NT = FT * CT / kMW;            // S tiles per wave (state update)
  constexpr int SROW = LD::SROW, PROW = LD::PROW, VROW = LD::VROW, KROW = LD::KROW;
  constexpr int NBUF = LD::NBUF, BAND = LD::BAND;
  constexpr int CPR = D / 8;                   // 8-element chunks per K/V row
  static_assert(NT * kMW == FT * CT, "S tiles must spread evenly over the waves");
  static_assert(32 * CPR <= kMT, "one staging chunk per thread");
  extern __shared__ __align__(16) char smem[];
  T* Wn = reinterpret_cast<T*>(smem + LD::wn);    // [D][WROW]   Wf (bf16)
  float* Sn = reinterpret_cast<float*>(smem + LD::sn);  // [DF][SROW]  S_c, fp32
  float* zs = reinterpret_cast<float*>(smem + LD::zs);  // [DF] z_c
  T* pk = reinterpret_cast<T*>(smem + LD::pk);    // [32][PROW]  phi(k) of 32 delayed keys
  T* vs = reinterpret_cast<T*>(smem + LD::vs);    // [32][VROW]  their values
  T* bnd = reinterpret_cast<T*>(smem + LD::band); // band tiles: [NBUF] x (K [32][KROW], V [32][VROW])

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hq = lane & 15, lg = lane >> 4;
  const int sg = blockIdx.x, g = blockIdx.y;
  const int bl = find_seq(a, sg);
  const SeqRows<T, D> sr = seq_rows<T, D, DF>(a, bl, g);
  const int sigma = sg - a.seg_base[bl];
  const int s_lo = sigma * a.seg_len, s_hi = min(a.seq_len[bl], s_lo + a.seg_len);
  const int G = a.G, W = a.W, C = a.C;
  const bool linear = a.linear != 0;
  const float sc2 = a.tau * kLog2e;
  const T* Q = static_cast<const T*>(a.q);
  T* O = static_cast<T*>(a.out);
  const WfCols<T, D, DF, LD::kWfLds> wf{LD::kWfLds ? Wn : static_cast<const T*>(a.wf)};

  // ---- 0. Wf into LDS; S, z at the segment start (the scan's record), fp32,
  //         into LDS; they stay there for the whole walk
  if (linear) {
    if (LD::kWfLds) stage_wf<T, D, DF>(static_cast<const T*>(a.wf), Wn, kMT);
    const float* S0 = a.seg + (int64_t(a.seg0 + sg) * a.Hkv + g) * (int64_t(DF) * D + DF);
    for (int i = tid; i < DF * D / 4; i += kMT) {
      const int f = i / (D / 4), c4 = 4 * (i - f * (D / 4));
      *reinterpret_cast<float4*>(Sn + f * SROW + c4) = *reinterpret_cast<const float4*>(S0 + f * D + c4);
    }
    if (tid < DF) zs[tid] = S0[DF * D + tid];
  }
  __syncthreads();

  for (int c0 = s_lo; c0 < s_hi; c0 += C) {
    const int nk = min(s_hi, c0 + C) - c0;  // tokens of the chunk
    const int64_t t0 = sr.p0 + c0;          // absolute position of its first token
    const int nrow = nk * G;
    for (int rb = 0; rb < nrow; rb += kRB) {
      const bool first_pass = rb == 0, last_pass = rb + kRB >= nrow;
      const int r_end = min(nrow, rb + kRB);
      const int ti_min = rb / G, ti_max = (r_end - 1) / G;  // chunk-relative tokens of the pass

      // this lane's query rows (score layout: row = hq of each 16-row q-tile)
      int ti[2], hh[2];
      bool rv[2];
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) {
        const int r = rb + 32 * wave + 16 * qt + hq;
        rv[qt] = r < nrow;
        const int rr = rv[qt] ? r : rb;
        ti[qt] = rr / G;
        hh[qt] = rr - ti[qt] * G;
      }
      Frag<T> qf[2][KS];
#pragma unroll
      for (int qt = 0; qt < 2; ++qt)
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) qf[qt][kk].load(Q + sr.qrow(c0 + ti[qt], hh[qt]) * D + 32 * kk + 8 * lg);
      // loads issued now and consumed later: the first slab of delayed keys
      // (key rows and values) and the first band tile
      SlabKeys<T, D, DF> kx;
      Frag<T> vx;
      auto load_slab = [&](int s0) {
        slab_keys(kx, kMW, [&](int r) {
          const int64_t j = t0 - W + s0 + r;
          return (s0 + r < nk && j >= 0) ? sr.k(j) : nullptr;
        });
        const int r = tid / CPR, ch = tid - r * CPR;
        const int64_t j = t0 - W + s0 + r;
        if (tid < 32 * CPR && s0 + r < nk && j >= 0) vx.load(sr.v(j) + 8 * ch);
        else vx.zero();
      };
      if (linear) load_slab(0);
      int64_t klo = t0 + ti_min - W + 1;
      if (klo < 0) klo = 0;
      const int64_t khi = t0 + ti_max;
      const int64_t kb0 = klo & ~int64_t(31);
      const int ntile = int((khi - kb0) / 32) + 1;
      Frag<T> sk, sv;  // staging registers: this thread's chunk of the next band tile (K and V)
      const bool stager = tid < 32 * CPR;
      const int srr = tid / CPR, sch = tid - srr * CPR;
      auto fetch = [&](int n) {
        const int64_t j = kb0 + 32 * int64_t(n) + srr;
        if (stager && j >= klo && j <= khi) {
          sk.load(sr.k(j) + 8 * sch);
          sv.load(sr.v(j) + 8 * sch);
        } else {
          sk.zero();
          sv.zero();
        }
      };
      auto store = [&](int buf) {
        if (stager) {
          T* kt = bnd + buf * BAND;
          store8(kt + srr * KROW + 8 * sch, sk);
          store8(kt + 32 * KROW + srr * VROW + 8 * sch, sv);
        }
      };
      if (W > 0) fetch(0);
      f32x4_t acc[2][CT];
#pragma unroll
      for (int qt = 0; qt < 2; ++qt)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) acc[qt][ct] = zero4();
      float m_run[2] = {-INFINITY, -INFINITY}, l_run[2] = {0.f, 0.f};

      // ---- 1. linear part
      if (linear) {
        // phi(q), transposed: lane (row hq, group lg) gets features
        // 32kf+4lg+i and 32kf+16+4lg+i of its query row in fragment kf
        Frag<T> pqf[2][KSF];
#pragma unroll
        for (int kf = 0; kf < KSF; ++kf) {
          float pv[2][8];
#pragma unroll
          for (int half = 0; half < 2; ++half) {
            f32x4_t ph[2] = {zero4(), zero4()};
#pragma unroll
            for (int kk = 0; kk < KS; ++kk) {
              Frag<T> wa;
              wf.col(wa, kk, 32 * kf + 16 * half);
#pragma unroll
              for (int qt = 0; qt < 2; ++qt) ph[qt] = mma(wa, qf[qt][kk], ph[qt]);
            }
#pragma unroll
            for (int qt = 0; qt < 2; ++qt)
#pragma unroll
              for (int i = 0; i < 4; ++i) pv[qt][4 * half + i] = fmaxf(ph[qt][i], 0.f);
          }
#pragma unroll
          for (int qt = 0; qt < 2; ++qt) pqf[qt][kf].set8(pv[qt]);
        }
        // read-out phi(q).S_c and phi(q).z_c
#pragma unroll
        for (int kf = 0; kf < KSF; ++kf) {
#pragma unroll
          for (int ct = 0; ct < CT; ++ct) {
            Frag<T> fb;
            load_colfrag2_f32(fb, Sn, SROW, 32 * kf + 4 * lg, 32 * kf + 16 + 4 * lg, 16 * ct);
#pragma unroll
            for (int qt = 0; qt < 2; ++qt) acc[qt][ct] = mma(pqf[qt][kf], fb, acc[qt][ct]);
          }
        }
        float den[2];
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) {
          float dz = 0.f;
#pragma unroll
          for (int kf = 0; kf < KSF; ++kf) {
            float qv[8];
            pqf[qt][kf].to_floats(qv);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              dz = fmaf(qv[e], zs[32 * kf + 4 * lg + e], dz);
              dz = fmaf(qv[4 + e], zs[32 * kf + 16 + 4 * lg + e], dz);
            }
          }
          den[qt] = dz;
        }
        // the chunk's delayed keys i' (key j = t0 - W + i'), 32 at a time:
        // phi(k) and values into LDS, the masked block i' <= ti of every
        // query row, and (last pass: every read-out of S_c is done, the loop
        // covers all the chunk's keys) S_{c+1} = S_c + phi(k)^T v in place
        for (int s0 = 0; s0 < nk; s0 += 32) {
          if (s0 > ti_max) break;
          __syncthreads();
          phi_slab(wf, kx, pk, kMW);
          if (tid < 32 * CPR) {
            const int r = tid / CPR, ch = tid - r * CPR;
            store8(vs + r * VROW + 8 * ch, vx);
          }
          if (s0 + 32 < nk && s0 + 32 <= ti_max) load_slab(s0 + 32);
          __syncthreads();
          if (last_pass) {
#pragma unroll
            for (int x = 0; x < NT; ++x) {
              const int tile = wave * NT + x, ft = tile / CT, ct = tile - ft * CT;
              Frag<T> fa, fb;
              load_colfrag(fa, pk, PROW, 8 * lg, 16 * ft);
              load_colfrag(fb, vs, VROW, 8 * lg, 16 * ct);
              const f32x4_t d = mma(fa, fb, zero4());
#pragma unroll
              for (int i = 0; i < 4; ++i) Sn[(16 * ft + 4 * lg + i) * SROW + 16 * ct + hq] += d[i];
            }
            if (tid < DF) {
              float dz = 0.f;
#pragma unroll 8
              for (int r = 0; r < 32; ++r) dz += to_f32(pk[r * PROW + tid]);
              zs[tid] += dz;
            }
          }
          // scores: key row m of sub-tile t is i' = s0 + 8(m/4) + 4t + m%4
          f32x4_t sc[2][2];
#pragma unroll
          for (int qt = 0; qt < 2; ++qt) sc[qt][0] = sc[qt][1] = zero4();
#pragma unroll
          for (int t = 0; t < 2; ++t) {
            const T* prow = pk + (8 * (hq >> 2) + 4 * t + (hq & 3)) * PROW;
#pragma unroll
            for (int kf = 0; kf < KSF; ++kf) {
              Frag<T> fa;
              load_row2(fa, prow, 32 * kf + 4 * lg, 32 * kf + 16 + 4 * lg);
#pragma unroll
              for (int qt = 0; qt < 2; ++qt) sc[qt][t] = mma(fa, pqf[qt][kf], sc[qt][t]);
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
        // the linear part becomes the start of the online softmax: one
        // pseudo-key of weight den (log2 domain: max = log2 den, sum 1)
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

      // ---- 2. banded window attention, keys [t0 + ti_min - W + 1, t0 + ti_max]
      if (W > 0) {
        __syncthreads();  // the previous users of the band buffers are done
        store(0);         // tile 0 was fetched at the start of the pass
        __syncthreads();
        for (int n = 0; n < ntile; ++n) {
          const int buf = NBUF == 2 ? (n & 1) : 0;
          if (n + 1 < ntile) fetch(n + 1);
          const T* kt = bnd + buf * BAND;
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
            // lazy rescale: the running max moves only when a score exceeds it
            // by more than 2^8, so p = 2^(s - m) <= 256 and acc, l stay in range
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
          if (n + 1 < ntile) {
            if (NBUF == 1) __syncthreads();  // every wave is done with the single buffer
            store(NBUF == 2 ? ((n + 1) & 1) : 0);
          }
          __syncthreads();
        }
      }

      // ---- 3. outputs
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) {
        float ls = l_run[qt];
        ls += __shfl_xor(ls, 16);
        ls += __shfl_xor(ls, 32);
        const float inv = ls > 0.f ? 1.f / ls : 0.f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float ir = __shfl(inv, 4 * lg + i);
          const int r = rb + 32 * wave + 16 * qt + 4 * lg + i;
          if (r < nrow) {
            const int tr = r / G, hr = r - tr * G;
            T* orow = O + sr.qrow(c0 + tr, hr) * D;
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) orow[16 * ct + hq] = from_f32<T>(acc[qt][ct][i] * ir);
          }
        }
      }
    }

    // S_{c+1}, z_{c+1} are in LDS; the next chunk's first read of them comes
    // after a barrier (its band staging or its first delayed-key slab)
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// ringfill: tokens [max(p0, p_end - W), p_end) into their ring slots
template <typename T, int D, int DF>
__global__ __launch_bounds__(kThreads) void prefill_ringfill(PrefillArgs a) {
  const int bl = blockIdx.y, g = blockIdx.z;
  const SeqRows<T, D> sr = seq_rows<T, D, DF>(a, bl, g);
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

template <typename K>
hipError_t set_lds(K* kern, size_t bytes) {
  if (bytes <= 65536) return hipSuccess;
  return hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                             int(bytes));
}

template <typename T, int D, int DF>
hipError_t layer_t(const PrefillArgs& a, hipStream_t s) {
  hipError_t e;
  if (a.nseg > 0) {
    if (a.linear) {
      const size_t lds_seg = (size_t(D) * row_t<DF>() + size_t(32) * row_t<DF>() + size_t(32) * row_t<D>()) *
                             sizeof(T);
      if ((e = set_lds(&prefill_segsum<T, D, DF>, lds_seg)) != hipSuccess) return e;
      hipLaunchKernelGGL((prefill_segsum<T, D, DF>), dim3(a.nseg, a.Hkv), dim3(kThreads), lds_seg, s, a);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      const int E = DF * D + DF;
      hipLaunchKernelGGL((prefill_scan<T, D, DF>), dim3((E / 4 + kThreads - 1) / kThreads, a.nseq, a.Hkv),
                         dim3(kThreads), 0, s, a);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    const size_t lds = MainLds<T, D, DF>::bytes;
    if ((e = set_lds(&prefill_main<T, D, DF>, lds)) != hipSuccess) return e;
    hipLaunchKernelGGL((prefill_main<T, D, DF>), dim3(a.nseg, a.Hkv), dim3(kMT), lds, s, a);
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
