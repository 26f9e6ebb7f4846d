// Feature map phi(x) = max(0, x . Wf) (the ReLU kernel of the GLIDE
// Appendix's feature-map list; Wf non-learnable, d x Df, one per layer).
//
// A workgroup stages Wf transposed in LDS once (so every MFMA B fragment -- 8
// consecutive head-dim values of one feature -- is a single 16-byte LDS
// read) and runs 64-row tiles, 16 rows per wave: A = rows (k = head dim),
// B = Wf (k = head dim, n = features), fp32 accumulation, ReLU on store.
//
// Two row sources:
//   * dense rows x[rows][d]                (glide_feature_map, prefill)
//   * the decode gather: for every (sequence, KV head) unit of a layer, its G
//     query heads followed by the key that leaves the window this step
//     (ring slot (p - W) mod R, or the new key itself when W = 0); written as
//     fp32 [layer][unit][G+1][Df] for the decode kernel.
#include "glide_internal.h"

namespace glide {

namespace {

constexpr int kThreads = 256;

template <int D>
constexpr int wt_stride() { return D + 8; }  // padded LDS row of Wf^T

__device__ __forceinline__ void store_col8(bf16_t* dst, int stride, const bf16_t* src) {
  const uint4 r = *reinterpret_cast<const uint4*>(src);
  dst[0 * stride] = bf16_t(r.x & 0xffffu);
  dst[1 * stride] = bf16_t(r.x >> 16);
  dst[2 * stride] = bf16_t(r.y & 0xffffu);
  dst[3 * stride] = bf16_t(r.y >> 16);
  dst[4 * stride] = bf16_t(r.z & 0xffffu);
  dst[5 * stride] = bf16_t(r.z >> 16);
  dst[6 * stride] = bf16_t(r.w & 0xffffu);
  dst[7 * stride] = bf16_t(r.w >> 16);
}
__device__ __forceinline__ void store_col8(float* dst, int stride, const float* src) {
  const float4 a = reinterpret_cast<const float4*>(src)[0];
  const float4 b = reinterpret_cast<const float4*>(src)[1];
  dst[0 * stride] = a.x; dst[1 * stride] = a.y; dst[2 * stride] = a.z; dst[3 * stride] = a.w;
  dst[4 * stride] = b.x; dst[5 * stride] = b.y; dst[6 * stride] = b.z; dst[7 * stride] = b.w;
}

// wt[f][c] = Wf[c][f]
template <typename T, int D, int DF>
__device__ __forceinline__ void stage_wf_transposed(const T* Wf, T* wt) {
  constexpr int WTS = wt_stride<D>();
  constexpr int CH = D * DF / 8;
  for (int i = threadIdx.x; i < CH; i += kThreads) {
    const int c = i / (DF / 8), f0 = (i % (DF / 8)) * 8;
    store_col8(wt + f0 * WTS + c, WTS, Wf + c * DF + f0);
  }
}

// phi of 16 rows (this wave): row hq of the tile is read from `row` (nullptr:
// zero row); its 8-element chunk (k-slab kk, lane group g) sits at
// row + kk * skk + g * sg (32 and 8 for a plain row; the key ring's
// fragment-major block uses other strides).  acc[nt][i] = phi-input of tile
// row 4*(lane/16)+i, feature 16*nt + lane%16 (before ReLU).
template <typename T, int D, int DF>
__device__ __forceinline__ void phi_tile16(const T* wt, const T* row, int skk, int sg, f32x4_t (&acc)[DF / 16]) {
  constexpr int WTS = wt_stride<D>();
  const int lane = threadIdx.x & 63, hq = lane & 15, lg = lane >> 4;
#pragma unroll
  for (int nt = 0; nt < DF / 16; ++nt) acc[nt] = zero4();
#pragma unroll
  for (int kk = 0; kk < D / 32; ++kk) {
    Frag<T> a;
    if (row) a.load(row + kk * skk + lg * sg);
    else a.zero();
#pragma unroll
    for (int nt = 0; nt < DF / 16; ++nt) {
      Frag<T> w;
      w.load(wt + (16 * nt + hq) * WTS + 32 * kk + 8 * lg);
      acc[nt] = mma(a, w, acc[nt]);
    }
  }
}

// Dense rows: persistent workgroups.  Wave w owns features
// [w*DF/4, (w+1)*DF/4) and keeps their Wf fragments in registers for the
// whole launch; the workgroup walks 64-row tiles (every wave reads the same
// rows, so three of the four reads hit the L1).
template <typename T, int D, int DF, typename OutT>
__global__ __launch_bounds__(kThreads) void phi_rows_kernel(const T* __restrict__ Wf, const T* __restrict__ x,
                                                            int64_t rows, OutT* __restrict__ out) {
  constexpr int KS = D / 32, NTW = DF / 16 / 4;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, hq = lane & 15, lg = lane >> 4;
  const int f0 = wave * NTW * 16;
  Frag<T> wb[KS][NTW];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk)
#pragma unroll
    for (int nt = 0; nt < NTW; ++nt) wb[kk][nt].load_strided(Wf + int64_t(32 * kk + 8 * lg) * DF + f0 + 16 * nt + hq, DF);
  const int64_t ntile = (rows + 63) / 64;
  for (int64_t tile = blockIdx.x; tile < ntile; tile += gridDim.x) {
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) {
      const int64_t r0 = tile * 64 + 16 * rt;
      const int64_t r = r0 + hq;
      Frag<T> fa[KS];
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        if (r < rows) fa[kk].load(x + r * D + 32 * kk + 8 * lg);
        else fa[kk].zero();
      }
      f32x4_t acc[NTW];
#pragma unroll
      for (int nt = 0; nt < NTW; ++nt) {
        acc[nt] = zero4();
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) acc[nt] = mma(fa[kk], wb[kk][nt], acc[nt]);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int64_t ro = r0 + 4 * lg + i;
        if (ro < rows) {
#pragma unroll
          for (int nt = 0; nt < NTW; ++nt) out[ro * DF + f0 + 16 * nt + hq] = from_f32<OutT>(fmaxf(acc[nt][i], 0.f));
        }
      }
    }
  }
}

template <typename T, int D, int DF>
__global__ __launch_bounds__(kThreads) void phi_decode_kernel(DecodeArgs a) {
  extern __shared__ __align__(16) char smem[];
  T* wt = reinterpret_cast<T*>(smem);
  const LayerArg L = a.layers[blockIdx.y];
  const T* Wf = reinterpret_cast<const T*>(a.phi_w) + int64_t(L.slot) * D * DF;
  stage_wf_transposed<T, D, DF>(Wf, wt);
  __syncthreads();

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, hq = lane & 15, lg = lane >> 4;
  const int G = a.G, B = a.B, Hkv = a.Hkv, Hq = a.Hq;
  const int units = B * Hkv;
  const int64_t rows = int64_t(units) * (G + 1);
  const int W = L.W, R = L.R;
  const LayerSections sec = layer_sections(B, Hkv, D, DF, R, sizeof(T));
  const char* lay = a.state + L.base;
  const int64_t r0 = int64_t(blockIdx.x) * 64 + 16 * wave;
  const int64_t r = r0 + hq;
  const T* row = nullptr;
  int skk = 32, sg = 8;
  if (r < rows) {
    const int u = int(r / (G + 1)), vec = int(r - int64_t(u) * (G + 1));
    const int b = u / Hkv, g = u - b * Hkv;
    const int64_t tok = int64_t(L.slot) * B + b;
    if (vec < G) {
      row = reinterpret_cast<const T*>(a.q) + (tok * Hq + int64_t(g) * G + vec) * D;
    } else {
      const int64_t p = reinterpret_cast<const int64_t*>(lay + sec.pos)[u];
      if (W == 0) {
        row = reinterpret_cast<const T*>(a.k) + (tok * Hkv + g) * D;
      } else if (p >= W) {
        const int32_t se = int32_t((p - W) % R);
        row = reinterpret_cast<const T*>(lay + sec.K) + int64_t(u) * R * D + kring_chunk(se, 0, 0, D);
        skk = int(kring_chunk(se, 1, 0, D) - kring_chunk(se, 0, 0, D));
        sg = int(kring_chunk(se, 0, 1, D) - kring_chunk(se, 0, 0, D));
      }
    }
  }
  f32x4_t acc[DF / 16];
  phi_tile16<T, D, DF>(wt, row, skk, sg, acc);
  float* out = a.phi_ws + int64_t(L.slot) * rows * DF;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t ro = r0 + 4 * lg + i;
    if (ro < rows) {
#pragma unroll
      for (int nt = 0; nt < DF / 16; ++nt) out[ro * DF + 16 * nt + hq] = fmaxf(acc[nt][i], 0.f);
    }
  }
}

template <typename T, int D, int DF>
size_t wt_bytes() { return size_t(DF) * wt_stride<D>() * sizeof(T); }

template <typename T, int D, int DF, typename OutT>
hipError_t launch_rows_t(const void* Wf, const void* x, int64_t rows, void* out, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  const int64_t ntile = (rows + 63) / 64;
  const dim3 grid(unsigned(ntile < 1024 ? ntile : 1024));
  hipLaunchKernelGGL((phi_rows_kernel<T, D, DF, OutT>), grid, dim3(kThreads), 0, s, static_cast<const T*>(Wf),
                     static_cast<const T*>(x), rows, static_cast<OutT*>(out));
  return hipGetLastError();
}

template <typename T, int D, int DF>
hipError_t launch_dec_t(const DecodeArgs& a, hipStream_t s) {
  const int64_t rows = int64_t(a.B) * a.Hkv * (a.G + 1);
  const dim3 grid(unsigned((rows + 63) / 64), unsigned(a.n_layers));
  const size_t lds = wt_bytes<T, D, DF>();
  if (lds > 65536) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&phi_decode_kernel<T, D, DF>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((phi_decode_kernel<T, D, DF>), grid, dim3(kThreads), lds, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_phi_rows(const void* Wf, const void* x, int64_t rows, void* out, int d, int Df, int dtype,
                           bool out_f32, hipStream_t s) {
  if (dtype == GLIDE_BF16) {
    if (out_f32) {
      if (d == 128 && Df == 128) return launch_rows_t<bf16_t, 128, 128, float>(Wf, x, rows, out, s);
      if (d == 128 && Df == 64) return launch_rows_t<bf16_t, 128, 64, float>(Wf, x, rows, out, s);
      if (d == 64 && Df == 128) return launch_rows_t<bf16_t, 64, 128, float>(Wf, x, rows, out, s);
      if (d == 64 && Df == 64) return launch_rows_t<bf16_t, 64, 64, float>(Wf, x, rows, out, s);
    } else {
      if (d == 128 && Df == 128) return launch_rows_t<bf16_t, 128, 128, bf16_t>(Wf, x, rows, out, s);
      if (d == 128 && Df == 64) return launch_rows_t<bf16_t, 128, 64, bf16_t>(Wf, x, rows, out, s);
      if (d == 64 && Df == 128) return launch_rows_t<bf16_t, 64, 128, bf16_t>(Wf, x, rows, out, s);
      if (d == 64 && Df == 64) return launch_rows_t<bf16_t, 64, 64, bf16_t>(Wf, x, rows, out, s);
    }
  } else {
    if (d == 128 && Df == 128) return launch_rows_t<float, 128, 128, float>(Wf, x, rows, out, s);
    if (d == 128 && Df == 64) return launch_rows_t<float, 128, 64, float>(Wf, x, rows, out, s);
    if (d == 64 && Df == 128) return launch_rows_t<float, 64, 128, float>(Wf, x, rows, out, s);
    if (d == 64 && Df == 64) return launch_rows_t<float, 64, 64, float>(Wf, x, rows, out, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_phi_decode(const DecodeArgs& a, int d, int Df, int dtype, hipStream_t s) {
  if (dtype == GLIDE_BF16) {
    if (d == 128 && Df == 128) return launch_dec_t<bf16_t, 128, 128>(a, s);
    if (d == 128 && Df == 64) return launch_dec_t<bf16_t, 128, 64>(a, s);
    if (d == 64 && Df == 128) return launch_dec_t<bf16_t, 64, 128>(a, s);
    if (d == 64 && Df == 64) return launch_dec_t<bf16_t, 64, 64>(a, s);
  } else {
    if (d == 128 && Df == 128) return launch_dec_t<float, 128, 128>(a, s);
    if (d == 128 && Df == 64) return launch_dec_t<float, 128, 64>(a, s);
    if (d == 64 && Df == 128) return launch_dec_t<float, 64, 128>(a, s);
    if (d == 64 && Df == 64) return launch_dec_t<float, 64, 64>(a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace glide
