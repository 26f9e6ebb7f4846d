// GLIDE decode step: one fused pass per (layer, sequence, KV head).
//
// Per unit (GLIDE Sec. III-B; the state recurrence of Sec. II-B applied to
// the tokens that have left the window):
//   1. the new key/value is written to ring slot p mod R;
//   2. phi of the G query heads and of the pending keys (tokens that have
//      left the window but are not yet folded into S, z) on MFMA against Wf,
//      each wave producing the features of the state rows it owns;
//   3. state: S' = S + sum_pending phi(k_j)^T v_j (and z') in registers, the
//      read-out phi(q_h).S', phi(q_h).z' from the same pass over S; on the
//      unit's fold step S', z' are written back (deferred folding: at most
//      one write of the state per kFoldPeriod steps);
//   4. window: the W most recent tokens (ring tokens p-W+1 .. p-1 plus the new
//      token taken straight from the input) are streamed in 32-token tiles,
//      the next tile's loads in flight while the current one is computed;
//      QK^T and PV run on MFMA with the G query heads of the group as the
//      16-wide tile dimension; online softmax in the log2 domain;
//   5. merge of the two parts over one shared denominator, output, pos += 1.
//
// One workgroup of 4 waves handles one unit; units of the call are ordered by
// decreasing window so the longest streams start first.
#include <math.h>

#include "glide_internal.h"

namespace glide {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ float4 shfl_xor4(float4 v, int m) {
  return make_float4(__shfl_xor(v.x, m), __shfl_xor(v.y, m), __shfl_xor(v.z, m), __shfl_xor(v.w, m));
}

__device__ __forceinline__ int clamp_rel(int64_t x) { return int(x < -1 ? -1 : (x > 32 ? 32 : x)); }

template <typename T, int D>
struct WindowTile {
  Frag<T> k[2][D / 32];  // A operand rows of the two 16-key sub-tiles
  Frag<T> v[D / 16];     // B operand: 8 tokens x 1 column per lane, per column tile
};

#ifndef GLIDE_DECODE_STAGES
#define GLIDE_DECODE_STAGES 2   // register stages of the window stream (bf16)
#endif
#ifndef GLIDE_DECODE_STATE_LAST
#define GLIDE_DECODE_STATE_LAST 0  // 1: window stream first, state fold last
#endif
#ifndef GLIDE_DECODE_WAVES_PER_SIMD
#define GLIDE_DECODE_WAVES_PER_SIMD 2
#endif

template <typename T, int D, int DF>
__global__ __launch_bounds__(kThreads)
__attribute__((amdgpu_waves_per_eu(GLIDE_DECODE_WAVES_PER_SIMD, GLIDE_DECODE_WAVES_PER_SIMD)))
void decode_kernel(DecodeArgs a) {
  constexpr int KS = D / 32;       // 32-wide k slabs over the head dim
  constexpr int CT = D / 16;       // 16-wide column tiles of the output
  constexpr int RW = DF / kWaves;  // state rows (features) per wave
  constexpr int NTW = RW / 16;     // 16-feature tiles per wave
  constexpr int LPR = D / 4;       // lanes per state row (4 floats each)
  constexpr int RPS = 64 / LPR;    // state rows per wave step
  constexpr int STEPS = RW / RPS;
  constexpr bool kTwoStages = sizeof(T) == 2 && GLIDE_DECODE_STAGES == 2;
  static_assert(STEPS * RPS == RW && NTW * 16 == RW, "state rows must tile the wave");

  extern __shared__ __align__(16) char smem[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hq = lane & 15, lg = lane >> 4;
  const int G = a.G, B = a.B, Hkv = a.Hkv, Hq = a.Hq;
  const int per_layer = B * Hkv;
  const int li = blockIdx.x / per_layer;
  const int rem = blockIdx.x - li * per_layer;
  const int b = rem / Hkv, g = rem - b * Hkv;
  const LayerArg L = a.layers[li];
  const int W = L.W, R = L.R;
  const LayerSections sec = layer_sections(B, Hkv, D, DF, R, sizeof(T));
  char* lay = a.state + L.base;
  const int64_t unit = int64_t(b) * Hkv + g;
  int64_t* pos_ptr = reinterpret_cast<int64_t*>(lay + sec.pos) + unit;
  int64_t* nf_ptr = reinterpret_cast<int64_t*>(lay + sec.nf) + unit;
  float* S = reinterpret_cast<float*>(lay + sec.S) + unit * DF * D;
  float* z = reinterpret_cast<float*>(lay + sec.z) + unit * DF;
  T* Kr = reinterpret_cast<T*>(lay + sec.K) + unit * int64_t(R) * D;
  T* Vr = reinterpret_cast<T*>(lay + sec.V) + unit * int64_t(R) * D;
  const int64_t tok = int64_t(L.slot) * B + b;
  const T* qg = reinterpret_cast<const T*>(a.q) + (tok * Hq + int64_t(g) * G) * D;
  const T* kn = reinterpret_cast<const T*>(a.k) + (tok * Hkv + g) * D;
  const T* vn = reinterpret_cast<const T*>(a.v) + (tok * Hkv + g) * D;
  T* og = reinterpret_cast<T*>(a.out) + (tok * Hq + int64_t(g) * G) * D;
  const T* Wf = reinterpret_cast<const T*>(a.phi_w) + int64_t(L.slot) * D * DF;

  const int64_t p = *pos_ptr;

  float* ph = reinterpret_cast<float*>(smem);  // [G + kFoldPeriod][DF] phi(q_h), then phi(k_j) of pending j
  float* pv = ph + (G + kFoldPeriod) * DF;     // [kFoldPeriod][D]      values of the pending tokens
  float* lnum = pv + kFoldPeriod * D;          // [waves][G][D] linear numerator partials phi(q).S
  float* lden = lnum + kWaves * G * D;         // [waves][G]    linear denominator partials phi(q).z
  float* wacc = lden + kWaves * G;             // [waves][G][D] window partials sum e^s v
  float* wm = wacc + kWaves * G * D;           // [waves][G]    window running max (log2 units)
  float* wl = wm + kWaves * G;                 // [waves][G]    window sum e^s

  // Linear set after this step: tokens [0, beta).  S, z hold tokens [0, nf);
  // tokens [nf, beta) are pending (in the ring, or the new token when W = 0)
  // and enter the read-out through phi(k_j) v_j.  They are folded for good on
  // this step when the unit's turn comes (every step when W = 0).
  const int64_t beta = p + 1 - W > 0 ? p + 1 - W : 0;
  const bool lin = a.linear != 0 && beta > 0;
  const int fper = W > 0 ? kFoldPeriod : 1;
  // nf of a well-formed state lies in [beta - fper, beta]; the clamp keeps
  // every access in bounds whatever the blob holds.
  int64_t nf = *nf_ptr;
  nf = nf < beta ? nf : beta;
  nf = nf > beta - fper ? nf : beta - fper;
  nf = nf > 0 ? nf : 0;
  const int npend = lin ? int(beta - nf) : 0;  // 0 .. fper
  const bool fold = npend > 0 && (npend >= fper || (beta + int64_t(unit % fper)) % fper == 0);
  const bool s_nonzero = lin && nf > 0;  // S, z hold something

  // ---- loads issued up front: this wave's S rows, and its first window tile
  const int f0 = wave * RW;
  const int lr = lane / LPR, c4 = (lane % LPR) * 4;
  float4 sr[STEPS];
  auto load_state = [&]() {
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
      const int f = f0 + s * RPS + lr;
      sr[s] = s_nonzero ? *reinterpret_cast<const float4*>(S + f * D + c4) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
#if !GLIDE_DECODE_STATE_LAST
  load_state();
#endif
  // window: tokens [tlo, p] in 32-token tiles; wave w takes tiles w, w+4, ...
  const int64_t tlo = p - W + 1 > 0 ? p - W + 1 : 0;
  const int64_t tile0 = tlo >> 5;
  const int n_tiles = W > 0 ? int((p >> 5) - tile0 + 1) : 0;
  int it = wave;
  int64_t j0 = (tile0 + it) << 5;
  uint32_t s0 = (W > 0 && it < n_tiles) ? uint32_t(j0 % R) : 0u;
  const uint32_t step = W > 0 ? uint32_t((32 * kWaves) % R) : 0u;

  // Loads of one tile.  Key row m of sub-tile t is token j0 + 8(m/4) + 4t + m%4,
  // so that after QK^T lane group lg holds tokens j0 + 8lg .. j0 + 8lg + 7,
  // exactly the A-operand layout PV needs.  lo/pn: window bounds relative
  // to j0 (clamped to [-1, 32]); pn is also where the new token sits.
  // Tile loads.  s0t = (j0 mod R) is a multiple of 32, so the tile is ring
  // block s0t/32 and every fragment load is one contiguous 1 KB read.  Rows
  // outside the window (and the new token, whose key is still in the input)
  // read the new key instead; masked rows' scores and out-of-window values'
  // probabilities are exactly 0, so substitute data never matters and the
  // loads need no branches.
  auto load_tile = [&](WindowTile<T, D>& tl, uint32_t s0t, int lo, int pn) {
    const T* Kb = Kr + int64_t(s0t) * D;
    const T* Vb = Vr + int64_t(s0t) * D;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int off = 8 * (hq >> 2) + 4 * t + (hq & 3);
      const bool ring = off >= lo && off < pn;
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        const T* src = ring ? Kb + (((t * KS + kk) * 4 + lg) * 16 + hq) * 8 : kn + 32 * kk + 8 * lg;
        tl.k[t][kk].load(src);
      }
    }
    const int ob = 8 * lg;
    const bool bvalid = ob + 7 >= lo && ob <= pn;
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) tl.v[ct].load((bvalid ? Vb : Vr) + ((ct * 4 + lg) * 16 + hq) * 8);
    if (bvalid && pn - ob < 8) {
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) tl.v[ct].patch(pn - ob, vn[16 * ct + hq]);
    }
  };

  WindowTile<T, D> ta;
  if (it < n_tiles) load_tile(ta, s0, clamp_rel(tlo - j0), clamp_rel(p - j0));
  Frag<T> qf[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    if (W > 0 && hq < G) qf[kk].load(qg + hq * D + 32 * kk + 8 * lg);
    else qf[kk].zero();
  }

  // ---- 1. new token into its ring slot (no token this step reads that slot)
  if (W > 0) {
    const int32_t sn = int32_t(p % R);
    for (int c = tid; c < D; c += kThreads) {
      Kr[kring_elem(sn, c, D)] = kn[c];
      Vr[vring_elem(sn, c, D)] = vn[c];
    }
  }

  // ---- 2. feature map of the G query heads and the pending keys, on MFMA:
  //         rows [q_0 .. q_{G-1}, k_nf .. k_{beta-1}] x Wf, each wave computing
  //         its own RW features (the state rows it owns); fp32 into LDS.
  if (lin) {
    const int nrows = G + npend;
    for (int rt = 0; 16 * rt < nrows; ++rt) {
      const int r = 16 * rt + hq;
      f32x4_t acc[NTW];
#pragma unroll
      for (int nt = 0; nt < NTW; ++nt) acc[nt] = zero4();
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        Frag<T> xa;
        if (r < G) {
          xa.load(qg + r * D + 32 * kk + 8 * lg);
        } else if (r < nrows) {
          const int64_t j = nf + (r - G);
          if (W == 0) xa.load(kn + 32 * kk + 8 * lg);  // the pending token is the new one
          else xa.load(Kr + kring_chunk(int32_t(j % R), kk, lg, D));
        } else {
          xa.zero();
        }
#pragma unroll
        for (int nt = 0; nt < NTW; ++nt) {
          Frag<T> wb;
          wb.load_strided(Wf + int64_t(32 * kk + 8 * lg) * DF + f0 + 16 * nt + hq, DF);
          acc[nt] = mma(xa, wb, acc[nt]);
        }
      }
#pragma unroll
      for (int nt = 0; nt < NTW; ++nt) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = 16 * rt + 4 * lg + i;
          if (row < nrows) ph[row * DF + f0 + 16 * nt + hq] = fmaxf(acc[nt][i], 0.f);
        }
      }
    }
    for (int e = tid; e < npend * D; e += kThreads) {
      const int i = e / D, c = e - i * D;
      pv[e] = W == 0 ? to_f32(vn[c]) : to_f32(Vr[vring_elem(int32_t((nf + i) % R), c, D)]);
    }
  }
  __syncthreads();

  auto state_phase = [&]() {
  // ---- 3. state: the pending tokens are added to this wave's S rows in
  //         registers (S' = S + sum_j phi(k_j)^T v_j, z' likewise), the
  //         read-out phi(q_h).S', phi(q_h).z' is taken from them, and on a
  //         fold step S', z' are written back (rows no pending token touches
  //         are unchanged and skipped).  Per-wave partials are summed in the
  //         merge.
  if (lin) {
    const float* pk = ph + G * DF;
    uint32_t touched = 0;
    for (int i = 0; i < npend; ++i) {
      const float4 vv = *reinterpret_cast<const float4*>(pv + i * D + c4);
#pragma unroll
      for (int s = 0; s < STEPS; ++s) {
        const float w = pk[i * DF + f0 + s * RPS + lr];
        touched |= uint32_t(w != 0.f) << s;
        sr[s].x = fmaf(w, vv.x, sr[s].x);
        sr[s].y = fmaf(w, vv.y, sr[s].y);
        sr[s].z = fmaf(w, vv.z, sr[s].z);
        sr[s].w = fmaf(w, vv.w, sr[s].w);
      }
    }
    if (fold) {
      // On the first fold every row is written, whatever the memory held.
#pragma unroll
      for (int s = 0; s < STEPS; ++s)
        if (!s_nonzero || ((touched >> s) & 1u)) store_nt(S + (f0 + s * RPS + lr) * D + c4, sr[s]);
    }
    float zf = 0.f;
    if (lane < RW) {
      zf = s_nonzero ? z[f0 + lane] : 0.f;
      float dz = 0.f;
      for (int i = 0; i < npend; ++i) dz += pk[i * DF + f0 + lane];
      zf += dz;
      if (fold && (dz != 0.f || !s_nonzero)) z[f0 + lane] = zf;
    }
    for (int hh = 0; hh < G; ++hh) {
      const float* pq = ph + hh * DF;
      float4 n4 = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int s = 0; s < STEPS; ++s) {
        const float w = pq[f0 + s * RPS + lr];
        n4.x = fmaf(w, sr[s].x, n4.x);
        n4.y = fmaf(w, sr[s].y, n4.y);
        n4.z = fmaf(w, sr[s].z, n4.z);
        n4.w = fmaf(w, sr[s].w, n4.w);
      }
#pragma unroll
      for (int off = LPR; off < 64; off <<= 1) {
        const float4 o = shfl_xor4(n4, off);
        n4.x += o.x; n4.y += o.y; n4.z += o.z; n4.w += o.w;
      }
      if (lr == 0) *reinterpret_cast<float4*>(lnum + (wave * G + hh) * D + c4) = n4;
      float dp = lane < RW ? pq[f0 + lane] * zf : 0.f;
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) dp += __shfl_xor(dp, off);
      if (lane == 0) lden[wave * G + hh] = dp;
    }
  }

  };

  auto window_phase = [&]() {
  // ---- 3. window: softmax over tokens [tlo, p]
  if (W > 0) {
    const float sc2 = a.tau * kLog2e;
    f32x4_t acc[CT];
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) acc[ct] = zero4();
    float m_run = -INFINITY, l_run = 0.f;

    auto compute_tile = [&](const WindowTile<T, D>& tl, int lo, int pn) {
      f32x4_t sc[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        sc[t] = zero4();
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) sc[t] = mma(tl.k[t][kk], qf[kk], sc[t]);
      }
      float s[8];
      float mx = -INFINITY;
#pragma unroll
      for (int t = 0; t < 2; ++t) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int off = 8 * lg + 4 * t + i;
          const float v = (off >= lo && off <= pn) ? sc[t][i] * sc2 : -INFINITY;
          s[4 * t + i] = v;
          mx = fmaxf(mx, v);
        }
      }
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run, mx);
      const float alpha = exp2f(m_run - m_new);
      float pv[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) pv[i] = exp2f(s[i] - m_new);
      Frag<T> pf;
      pf.set8(pv);
      l_run = l_run * alpha + pf.sum();
      m_run = m_new;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float al = __shfl(alpha, 4 * lg + i);
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) acc[ct][i] *= al;
      }
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) acc[ct] = mma(pf, tl.v[ct], acc[ct]);
    };

    if constexpr (kTwoStages) {
      // two register stages: tile it+4 loads while tile it computes
      WindowTile<T, D> tb;
      while (it < n_tiles) {
        if (it + kWaves < n_tiles)
          load_tile(tb, wrap_once(s0 + step, R), clamp_rel(tlo - j0 - 32 * kWaves),
                    clamp_rel(p - j0 - 32 * kWaves));
        compute_tile(ta, clamp_rel(tlo - j0), clamp_rel(p - j0));
        it += kWaves;
        j0 += 32 * kWaves;
        s0 = wrap_once(s0 + step, R);
        if (it >= n_tiles) break;
        if (it + kWaves < n_tiles)
          load_tile(ta, wrap_once(s0 + step, R), clamp_rel(tlo - j0 - 32 * kWaves),
                    clamp_rel(p - j0 - 32 * kWaves));
        compute_tile(tb, clamp_rel(tlo - j0), clamp_rel(p - j0));
        it += kWaves;
        j0 += 32 * kWaves;
        s0 = wrap_once(s0 + step, R);
      }
    } else {
      while (it < n_tiles) {
        compute_tile(ta, clamp_rel(tlo - j0), clamp_rel(p - j0));
        it += kWaves;
        j0 += 32 * kWaves;
        s0 = wrap_once(s0 + step, R);
        if (it < n_tiles) load_tile(ta, s0, clamp_rel(tlo - j0), clamp_rel(p - j0));
      }
    }

    l_run += __shfl_xor(l_run, 16);
    l_run += __shfl_xor(l_run, 32);
    if (lane < G) {
      wm[wave * G + lane] = m_run;
      wl[wave * G + lane] = l_run;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int h = 4 * lg + i;
      if (h < G) {
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) wacc[(wave * G + h) * D + 16 * ct + hq] = acc[ct][i];
      }
    }
  }
  };

#if GLIDE_DECODE_STATE_LAST
  window_phase();
  load_state();
  state_phase();
#else
  state_phase();
  window_phase();
#endif
  __syncthreads();

  // ---- 4. shared-denominator merge and output
  for (int i = tid; i < G * D; i += kThreads) {
    const int hh = i / D, c = i - hh * D;
    float nm = 0.f, dn = 0.f;
    if (lin) {
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        nm += lnum[(w * G + hh) * D + c];
        dn += lden[w * G + hh];
      }
    }
    float o;
    if (W > 0) {
      float M = -INFINITY;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) M = fmaxf(M, wm[w * G + hh]);
      float Ls = 0.f, Ac = 0.f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const float mw = wm[w * G + hh];
        if (mw != -INFINITY) {
          const float e = exp2f(mw - M);
          Ls = fmaf(wl[w * G + hh], e, Ls);
          Ac = fmaf(wacc[(w * G + hh) * D + c], e, Ac);
        }
      }
      if (dn > 0.f) {
        const float c2 = fmaxf(M, log2f(dn));
        const float ws = exp2f(M - c2), wlin = exp2f(-c2);
        o = (Ac * ws + nm * wlin) / (Ls * ws + dn * wlin);
      } else {
        o = Ac / Ls;
      }
    } else {
      o = dn > 0.f ? nm / dn : 0.f;
    }
    og[i] = from_f32<T>(o);
  }
  if (tid == 0) {
    *pos_ptr = p + 1;
    if (fold) *nf_ptr = beta;
  }
}

// Fold every pending token of a unit into S and z (nf := beta = max(0, p-W)),
// leaving the state in its direct form S = sum_{j < beta} phi(k_j)^T v_j.
// Plain fp32 arithmetic: it runs once per prefill call, not per token.
template <typename T, int D, int DF>
__global__ __launch_bounds__(kThreads) void flush_kernel(DecodeArgs a) {
  __shared__ float kx[kFoldPeriod][D], vx[kFoldPeriod][D], pk[kFoldPeriod][DF];
  const int tid = threadIdx.x;
  const int per_layer = a.B * a.Hkv;
  const int li = blockIdx.x / per_layer;
  const int64_t unit = blockIdx.x - int64_t(li) * per_layer;
  const LayerArg L = a.layers[li];
  const int W = L.W, R = L.R;
  if (W == 0) return;  // W = 0 units fold on every step
  const LayerSections sec = layer_sections(a.B, a.Hkv, D, DF, R, sizeof(T));
  char* lay = a.state + L.base;
  const int64_t p = reinterpret_cast<const int64_t*>(lay + sec.pos)[unit];
  int64_t* nf_ptr = reinterpret_cast<int64_t*>(lay + sec.nf) + unit;
  const int64_t beta = p - W > 0 ? p - W : 0;
  int64_t nf = *nf_ptr;
  nf = nf < beta ? nf : beta;
  nf = nf > beta - kFoldPeriod ? nf : beta - kFoldPeriod;
  nf = nf > 0 ? nf : 0;
  const int n = int(beta - nf);
  if (n == 0) return;
  float* S = reinterpret_cast<float*>(lay + sec.S) + unit * DF * D;
  float* z = reinterpret_cast<float*>(lay + sec.z) + unit * DF;
  const T* Kr = reinterpret_cast<const T*>(lay + sec.K) + unit * int64_t(R) * D;
  const T* Vr = reinterpret_cast<const T*>(lay + sec.V) + unit * int64_t(R) * D;
  const T* Wf = reinterpret_cast<const T*>(a.phi_w) + int64_t(L.slot) * D * DF;
  for (int e = tid; e < n * D; e += kThreads) {
    const int i = e / D, c = e - i * D;
    const int32_t slot = int32_t((nf + i) % R);
    kx[i][c] = to_f32(Kr[kring_elem(slot, c, D)]);
    vx[i][c] = to_f32(Vr[vring_elem(slot, c, D)]);
  }
  __syncthreads();
  for (int e = tid; e < n * DF; e += kThreads) {
    const int i = e / DF, f = e - i * DF;
    float acc = 0.f;
    for (int c = 0; c < D; ++c) acc = fmaf(kx[i][c], to_f32(Wf[c * DF + f]), acc);
    pk[i][f] = fmaxf(acc, 0.f);
  }
  __syncthreads();
  const bool s_nonzero = nf > 0;
  for (int e = tid; e < DF * D / 4; e += kThreads) {
    const int f = e / (D / 4), c4 = (e - f * (D / 4)) * 4;
    float4 sv = s_nonzero ? *reinterpret_cast<const float4*>(S + f * D + c4) : make_float4(0.f, 0.f, 0.f, 0.f);
    for (int i = 0; i < n; ++i) {
      const float w = pk[i][f];
      sv.x = fmaf(w, vx[i][c4], sv.x);
      sv.y = fmaf(w, vx[i][c4 + 1], sv.y);
      sv.z = fmaf(w, vx[i][c4 + 2], sv.z);
      sv.w = fmaf(w, vx[i][c4 + 3], sv.w);
    }
    *reinterpret_cast<float4*>(S + f * D + c4) = sv;
  }
  for (int f = tid; f < DF; f += kThreads) {
    float zf = s_nonzero ? z[f] : 0.f;
    for (int i = 0; i < n; ++i) zf += pk[i][f];
    z[f] = zf;
  }
  if (tid == 0) *nf_ptr = beta;
}

template <typename T, int D, int DF>
hipError_t flush_t(const DecodeArgs& a, hipStream_t stream) {
  const dim3 grid(unsigned(a.n_layers) * unsigned(a.B) * unsigned(a.Hkv));
  hipLaunchKernelGGL((flush_kernel<T, D, DF>), grid, dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

template <typename T, int D, int DF>
hipError_t launch_t(const DecodeArgs& a, hipStream_t stream) {
  const int G = a.G;
  const size_t floats = size_t(G + kFoldPeriod) * DF + size_t(kFoldPeriod) * D +
                        2 * (size_t(kWaves) * G * D + kWaves * G) + kWaves * G;
  const dim3 grid(unsigned(a.n_layers) * unsigned(a.B) * unsigned(a.Hkv));
  hipLaunchKernelGGL((decode_kernel<T, D, DF>), grid, dim3(kThreads), floats * sizeof(float), stream, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_decode(const DecodeArgs& a, int d, int Df, int dtype, hipStream_t stream) {
  if (dtype == GLIDE_BF16) {
    if (d == 128 && Df == 128) return launch_t<bf16_t, 128, 128>(a, stream);
    if (d == 128 && Df == 64) return launch_t<bf16_t, 128, 64>(a, stream);
    if (d == 64 && Df == 128) return launch_t<bf16_t, 64, 128>(a, stream);
    if (d == 64 && Df == 64) return launch_t<bf16_t, 64, 64>(a, stream);
  } else {
    if (d == 128 && Df == 128) return launch_t<float, 128, 128>(a, stream);
    if (d == 128 && Df == 64) return launch_t<float, 128, 64>(a, stream);
    if (d == 64 && Df == 128) return launch_t<float, 64, 128>(a, stream);
    if (d == 64 && Df == 64) return launch_t<float, 64, 64>(a, stream);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_flush(const DecodeArgs& a, int d, int Df, int dtype, hipStream_t stream) {
  if (dtype == GLIDE_BF16) {
    if (d == 128 && Df == 128) return flush_t<bf16_t, 128, 128>(a, stream);
    if (d == 128 && Df == 64) return flush_t<bf16_t, 128, 64>(a, stream);
    if (d == 64 && Df == 128) return flush_t<bf16_t, 64, 128>(a, stream);
    if (d == 64 && Df == 64) return flush_t<bf16_t, 64, 64>(a, stream);
  } else {
    if (d == 128 && Df == 128) return flush_t<float, 128, 128>(a, stream);
    if (d == 128 && Df == 64) return flush_t<float, 128, 64>(a, stream);
    if (d == 64 && Df == 128) return flush_t<float, 64, 128>(a, stream);
    if (d == 64 && Df == 64) return flush_t<float, 64, 64>(a, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace glide
