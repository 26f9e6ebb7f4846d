// GLIDE decode step: one fused pass per (layer, sequence, KV head).
//
// Per unit, in the order of the layer definition (GLIDE Sec. III-B; state
// recurrence of Sec. II-B applied to the token leaving the window):
//   1. the new key/value is written to ring slot p mod R;
//   2. state: the token leaving the window (token p - W, or the new token when
//      W = 0) is folded, S += phi(k_e)^T v_e, z += phi(k_e), in place, and the
//      read-out phi(q_h).S, phi(q_h).z is taken from the updated rows in the
//      same pass over S.  phi of the G query heads and of k_e comes from the
//      feature-map kernel that runs just before (decode workspace);
//   3. window: the W most recent tokens (ring tokens p-W+1 .. p-1 plus the new
//      token taken straight from the input) are streamed in 32-token tiles,
//      the next tile's loads in flight while the current one is computed;
//      QK^T and PV run on MFMA with the G query heads of the group as the
//      16-wide tile dimension; online softmax in the log2 domain;
//   4. merge of the two parts over one shared denominator, output, pos += 1.
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
  constexpr int LPR = D / 4;       // lanes per state row (4 floats each)
  constexpr int RPS = 64 / LPR;    // state rows per wave step
  constexpr int STEPS = RW / RPS;
  constexpr bool kTwoStages = sizeof(T) == 2 && GLIDE_DECODE_STAGES == 2;
  static_assert(STEPS * RPS == RW, "state rows must tile the wave");

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
  float* S = reinterpret_cast<float*>(lay + sec.S) + unit * DF * D;
  float* z = reinterpret_cast<float*>(lay + sec.z) + unit * DF;
  T* Kr = reinterpret_cast<T*>(lay + sec.K) + unit * int64_t(R) * D;
  T* Vr = reinterpret_cast<T*>(lay + sec.V) + unit * int64_t(R) * D;
  const int64_t tok = int64_t(L.slot) * B + b;
  const T* qg = reinterpret_cast<const T*>(a.q) + (tok * Hq + int64_t(g) * G) * D;
  const T* kn = reinterpret_cast<const T*>(a.k) + (tok * Hkv + g) * D;
  const T* vn = reinterpret_cast<const T*>(a.v) + (tok * Hkv + g) * D;
  T* og = reinterpret_cast<T*>(a.out) + (tok * Hq + int64_t(g) * G) * D;
  const float* phw = a.phi_ws + ((int64_t(L.slot) * B * Hkv) + unit) * (G + 1) * DF;

  const int64_t p = *pos_ptr;

  float* ve = reinterpret_cast<float*>(smem);  // [D]           folded value
  float* ph = ve + D;                          // [G+1][DF]     phi(q_h), then phi(k_e)
  float* lnum = ph + (G + 1) * DF;             // [waves][G][D] linear numerator partials phi(q).S
  float* lden = lnum + kWaves * G * D;         // [waves][G]    linear denominator partials phi(q).z
  float* wacc = lden + kWaves * G;             // [waves][G][D] window partials sum e^s v
  float* wm = wacc + kWaves * G * D;           // [waves][G]    window running max (log2 units)
  float* wl = wm + kWaves * G;                 // [waves][G]    window sum e^s

  const bool linear = a.linear != 0;
  // Something is folded in this step exactly when the state is non-empty
  // after it, so the fold and the linear read-out go together.
  const bool fold = linear && (W == 0 || p >= W);
  const bool s_nonzero = linear && (p - W > 0);  // state non-empty before the fold

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

  // ---- 1. new token into its ring slot (no reader of that slot this step);
  //         stage phi rows and the folded value
  if (W > 0) {
    const int32_t sn = int32_t(p % R);
    for (int c = tid; c < D; c += kThreads) {
      Kr[kring_elem(sn, c, D)] = kn[c];
      Vr[vring_elem(sn, c, D)] = vn[c];
    }
  }
  if (fold) {
    for (int i = tid; i < (G + 1) * DF / 4; i += kThreads)
      reinterpret_cast<float4*>(ph)[i] = reinterpret_cast<const float4*>(phw)[i];
    if (W == 0) {
      for (int c = tid; c < D; c += kThreads) ve[c] = to_f32(vn[c]);
    } else {
      const int32_t se = int32_t((p - W) % R);
      for (int c = tid; c < D; c += kThreads) ve[c] = to_f32(Vr[vring_elem(se, c, D)]);
    }
  }
  __syncthreads();

  auto state_phase = [&]() {
  // ---- 2. state: fold + read-out, one read and one write of S; the
  //         per-wave read-out partials are summed in the merge
  if (fold) {
    const float* pk = ph + G * DF;
    const float4 vv = *reinterpret_cast<const float4*>(ve + c4);
    // Row f changes only where phi(k_e)_f != 0; with the ReLU feature map
    // about half of the rows are untouched and are not written back (on the
    // first fold every row is written, whatever the memory held).
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
      const int f = f0 + s * RPS + lr;
      const float w = pk[f];
      if (w != 0.f || !s_nonzero) {
        sr[s].x = fmaf(w, vv.x, sr[s].x);
        sr[s].y = fmaf(w, vv.y, sr[s].y);
        sr[s].z = fmaf(w, vv.z, sr[s].z);
        sr[s].w = fmaf(w, vv.w, sr[s].w);
        store_nt(S + f * D + c4, sr[s]);
      }
    }
    float zf = 0.f;
    if (lane < RW) {
      zf = s_nonzero ? z[f0 + lane] : 0.f;
      const float w = pk[f0 + lane];
      if (w != 0.f || !s_nonzero) {
        zf += w;
        z[f0 + lane] = zf;
      }
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
    if (fold) {
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
  if (tid == 0) *pos_ptr = p + 1;
}

template <typename T, int D, int DF>
hipError_t launch_t(const DecodeArgs& a, hipStream_t stream) {
  const int G = a.G;
  const size_t floats = D + size_t(G + 1) * DF + 2 * (size_t(kWaves) * G * D + kWaves * G) + kWaves * G;
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

}  // namespace glide
