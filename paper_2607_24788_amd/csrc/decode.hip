// GLIDE decode step: one fused pass per (layer, sequence, KV head).
//
// Per unit, in the order of the layer definition (GLIDE Sec. III-B; state
// recurrence of Sec. II-B applied to the token leaving the window):
//   1. the new key/value is written to ring slot p mod R;
//   2. state: the token leaving the window (token p - W, or the new token when
//      W = 0) is folded, S += phi(k_e)^T v_e, z += phi(k_e), in place, and the
//      read-out phi(q_h).S, phi(q_h).z is taken from the updated rows in the
//      same pass over S;
//   3. window: the W most recent tokens (ring tokens p-W+1 .. p-1 plus the new
//      token taken straight from the input) are streamed in 32-token tiles;
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

template <typename T, int D, int DF>
__global__ __launch_bounds__(kThreads) void decode_kernel(DecodeArgs a) {
  constexpr int KS = D / 32;       // 32-wide k slabs over the head dim
  constexpr int CT = D / 16;       // 16-wide column tiles of the output
  constexpr int RW = DF / kWaves;  // state rows per wave
  constexpr int LPR = D / 4;       // lanes per state row (4 floats each)
  constexpr int RPS = 64 / LPR;    // state rows per wave step
  constexpr int STEPS = RW / RPS;
  static_assert(STEPS * RPS == RW, "state rows must tile the wave");

  extern __shared__ float smem[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
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
  const T* Wf = reinterpret_cast<const T*>(a.phi_w) + int64_t(L.slot) * D * DF;

  const int64_t p = *pos_ptr;

  float* xs = smem;                     // [G+1][D]   q heads, then the folded key
  float* ve = xs + (G + 1) * D;         // [D]        folded value
  float* ph = ve + D;                   // [G+1][DF]  phi(q_h), then phi(k_e)
  float* red = ph + (G + 1) * DF;       // [waves][G][D] per-wave partials
  float* redm = red + kWaves * G * D;   // [waves][G]
  float* redl = redm + kWaves * G;      // [waves][G]
  float* lnum = redl + kWaves * G;      // [G][D]     linear numerator phi(q).S
  float* lden = lnum + G * D;           // [G]        linear denominator phi(q).z

  const bool linear = a.linear != 0;
  // Something is folded in this step exactly when the state is non-empty
  // after it, so the fold and the linear read-out go together.
  const bool fold = linear && (W == 0 || p >= W);
  const bool s_nonzero = linear && (p - W > 0);  // state non-empty before the fold

  // ---- 1. new token into its ring slot (no reader of that slot this step)
  if (W > 0) {
    const int64_t sn = p % R;
    for (int c = tid; c < D; c += kThreads) {
      Kr[sn * D + c] = kn[c];
      Vr[((sn >> 3) * D + c) * 8 + (sn & 7)] = vn[c];
    }
  }
  if (fold) {
    for (int i = tid; i < G * D; i += kThreads) xs[i] = to_f32(qg[i]);
    if (W == 0) {
      for (int c = tid; c < D; c += kThreads) {
        xs[G * D + c] = to_f32(kn[c]);
        ve[c] = to_f32(vn[c]);
      }
    } else {
      const int64_t se = (p - W) % R;
      for (int c = tid; c < D; c += kThreads) {
        xs[G * D + c] = to_f32(Kr[se * D + c]);
        ve[c] = to_f32(Vr[((se >> 3) * D + c) * 8 + (se & 7)]);
      }
    }
  }
  __syncthreads();

  // ---- 2. state: fold + read-out, one read and one write of S
  if (fold) {
    const int f0 = wave * RW;
    const int lr = lane / LPR, c4 = (lane % LPR) * 4;
    float4 sr[STEPS];
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
      const int f = f0 + s * RPS + lr;
      sr[s] = s_nonzero ? *reinterpret_cast<const float4*>(S + f * D + c4) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    // phi for this wave's rows, for the G query heads and the folded key
    for (int idx = lane; idx < (G + 1) * RW; idx += 64) {
      const int vec = idx / RW, f = f0 + idx % RW;
      const float* x = xs + vec * D;
      float acc = 0.f;
#pragma unroll 8
      for (int c = 0; c < D; ++c) acc = fmaf(x[c], to_f32(Wf[c * DF + f]), acc);
      ph[vec * DF + f] = fmaxf(acc, 0.f);
    }
    __syncthreads();
    const float* pk = ph + G * DF;
    const float4 vv = *reinterpret_cast<const float4*>(ve + c4);
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
      const int f = f0 + s * RPS + lr;
      const float w = pk[f];
      sr[s].x = fmaf(w, vv.x, sr[s].x);
      sr[s].y = fmaf(w, vv.y, sr[s].y);
      sr[s].z = fmaf(w, vv.z, sr[s].z);
      sr[s].w = fmaf(w, vv.w, sr[s].w);
      *reinterpret_cast<float4*>(S + f * D + c4) = sr[s];
    }
    float zf = 0.f;
    if (lane < RW) {
      zf = (s_nonzero ? z[f0 + lane] : 0.f) + pk[f0 + lane];
      z[f0 + lane] = zf;
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
      if (lr == 0) *reinterpret_cast<float4*>(red + (wave * G + hh) * D + c4) = n4;
      float dp = lane < RW ? pq[f0 + lane] * zf : 0.f;
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) dp += __shfl_xor(dp, off);
      if (lane == 0) redm[wave * G + hh] = dp;
    }
    __syncthreads();
    for (int i = tid; i < G * D; i += kThreads) {
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) s += red[w * G * D + i];
      lnum[i] = s;
    }
    for (int i = tid; i < G; i += kThreads) {
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) s += redm[w * G + i];
      lden[i] = s;
    }
    __syncthreads();
  }

  // ---- 3. window: softmax over tokens [max(0, p-W+1), p]
  if (W > 0) {
    const int64_t tlo = p - W + 1 > 0 ? p - W + 1 : 0;
    const int64_t tile0 = tlo >> 5;
    const int n_tiles = int((p >> 5) - tile0 + 1);
    const int hq = lane & 15, lg = lane >> 4;
    const float sc2 = a.tau * kLog2e;
    Frag<T> qf[KS];
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      if (hq < G) qf[kk].load(qg + hq * D + 32 * kk + 8 * lg);
      else qf[kk].zero();
    }
    f32x4_t acc[CT];
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) acc[ct] = zero4();
    float m_run = -INFINITY, l_run = 0.f;
    for (int it = wave; it < n_tiles; it += kWaves) {
      const int64_t j0 = (tile0 + it) << 5;
      const uint32_t s0 = uint32_t(j0 % R);
      // keys: A operand rows; row m of sub-tile t is token j0 + 8(m/4) + 4t + m%4
      Frag<T> kf[2][KS];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int off = 8 * (hq >> 2) + 4 * t + (hq & 3);
        const int64_t j = j0 + off;
        const bool valid = j >= tlo && j <= p;
        const T* src = (j == p) ? kn : Kr + int64_t((s0 + off) % uint32_t(R)) * D;
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) {
          if (valid) kf[t][kk].load(src + 32 * kk + 8 * lg);
          else kf[t][kk].zero();
        }
      }
      // values: B operand, 8 consecutive tokens of one column from the
      // transposed ring block; the new token is patched in from the input
      Frag<T> vf[CT];
      const int64_t jb = j0 + 8 * lg;
      const bool bvalid = (jb + 7 >= tlo) && (jb <= p);
      const int64_t sb = int64_t((s0 + 8 * lg) % uint32_t(R)) >> 3;
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) {
        if (bvalid) vf[ct].load(Vr + (sb * D + 16 * ct + hq) * 8);
        else vf[ct].zero();
      }
      if (bvalid && p - jb < 8) {
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) vf[ct].set_raw(int(p - jb), vn[16 * ct + hq]);
      }
      // scores (keys x heads), 8 per lane: tokens j0 + 8*lg + (4t + i), head hq
      f32x4_t sc[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        sc[t] = zero4();
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) sc[t] = mma(kf[t][kk], qf[kk], sc[t]);
      }
      float s[8];
      float mx = -INFINITY;
#pragma unroll
      for (int t = 0; t < 2; ++t) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int64_t j = jb + 4 * t + i;
          const float v = (j >= tlo && j <= p) ? sc[t][i] * sc2 : -INFINITY;
          s[4 * t + i] = v;
          mx = fmaxf(mx, v);
        }
      }
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run, mx);
      const float alpha = exp2f(m_run - m_new);
      Frag<T> pf;
      float ps = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        pf.set(i, exp2f(s[i] - m_new));
        ps += pf.get(i);
      }
      l_run = l_run * alpha + ps;
      m_run = m_new;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float al = __shfl(alpha, 4 * lg + i);
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) acc[ct][i] *= al;
      }
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) acc[ct] = mma(pf, vf[ct], acc[ct]);
    }
    l_run += __shfl_xor(l_run, 16);
    l_run += __shfl_xor(l_run, 32);
    if (lane < 16 && lane < G) {
      redm[wave * G + lane] = m_run;
      redl[wave * G + lane] = l_run;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int h = 4 * lg + i;
      if (h < G) {
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) red[(wave * G + h) * D + 16 * ct + hq] = acc[ct][i];
      }
    }
  }
  __syncthreads();

  // ---- 4. shared-denominator merge and output
  for (int i = tid; i < G * D; i += kThreads) {
    const int hh = i / D;
    const float nm = fold ? lnum[i] : 0.f;
    const float dn = fold ? lden[hh] : 0.f;
    float o;
    if (W > 0) {
      float M = -INFINITY;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) M = fmaxf(M, redm[w * G + hh]);
      float Ls = 0.f, Ac = 0.f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const float mw = redm[w * G + hh];
        if (mw != -INFINITY) {
          const float e = exp2f(mw - M);
          Ls = fmaf(redl[w * G + hh], e, Ls);
          Ac = fmaf(red[(w * G + hh) * D + (i - hh * D)], e, Ac);
        }
      }
      if (dn > 0.f) {
        const float c2 = fmaxf(M, log2f(dn));
        const float ws = exp2f(M - c2), wl = exp2f(-c2);
        o = (Ac * ws + nm * wl) / (Ls * ws + dn * wl);
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
  const size_t floats = size_t(G + 1) * D + D + size_t(G + 1) * DF + size_t(kWaves) * G * D +
                        2 * kWaves * G + size_t(G) * D + G;
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
