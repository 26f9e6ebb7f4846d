// Feature map phi(x) = act(x . Wf) (ReLU, ELU + 1 or the softmax over the
// features; Wf non-learnable, d x Df, one per layer), for dense rows
// x[rows][d] (glide_feature_map).  The decode step and the prefill compute
// their rows inside their own kernels.
//
// Persistent workgroups of 4 waves; wave w owns features [w*Df/4, (w+1)*Df/4)
// and keeps their Wf B fragments in registers for the whole launch; the
// workgroup walks 64-row tiles: A = 16 rows (k = head dim), B = Wf (k = head
// dim, n = features), fp32 accumulation, the activation on store.  The
// softmax map's rows are spread over the four waves: their raw values go to
// LDS (dynamic, only for that map), each row is normalised there, then stored.
#include "glide_internal.h"

namespace glide {

namespace {

constexpr int kThreads = 256;

// Every wave of a workgroup reads the same 64 rows; three of the four reads
// hit the L1.
template <typename T, int D, int DF, typename OutT>
__global__ __launch_bounds__(kThreads) void phi_rows_kernel(const T* __restrict__ Wf, const T* __restrict__ x,
                                                            int64_t rows, OutT* __restrict__ out, int phi) {
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
      if (phi == GLIDE_PHI_SOFTMAX) {  // uniform over the launch
        extern __shared__ float yt[];   // [16][DF]
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int nt = 0; nt < NTW; ++nt) yt[(4 * lg + i) * DF + f0 + 16 * nt + hq] = acc[nt][i];
        __syncthreads();
        softmax_rows_lds<DF, kThreads>(yt, DF, 16);
        __syncthreads();
        for (int e = threadIdx.x; e < 16 * DF; e += kThreads) {
          const int64_t ro = r0 + e / DF;
          if (ro < rows) out[ro * DF + e % DF] = from_f32<OutT>(yt[e]);
        }
        __syncthreads();
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int64_t ro = r0 + 4 * lg + i;
          if (ro < rows) {
#pragma unroll
            for (int nt = 0; nt < NTW; ++nt) out[ro * DF + f0 + 16 * nt + hq] = from_f32<OutT>(feat_act(acc[nt][i], phi));
          }
        }
      }
    }
  }
}

template <typename T, int D, int DF, typename OutT>
hipError_t launch_rows_t(const void* Wf, const void* x, int64_t rows, void* out, int phi, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  const int64_t ntile = (rows + 63) / 64;
  const dim3 grid(unsigned(ntile < 1024 ? ntile : 1024));
  const size_t lds = phi == GLIDE_PHI_SOFTMAX ? size_t(16) * DF * sizeof(float) : 0;
  hipLaunchKernelGGL((phi_rows_kernel<T, D, DF, OutT>), grid, dim3(kThreads), lds, s, static_cast<const T*>(Wf),
                     static_cast<const T*>(x), rows, static_cast<OutT*>(out), phi);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_phi_rows(const void* Wf, const void* x, int64_t rows, void* out, int d, int Df, int dtype,
                           bool out_f32, int phi, hipStream_t s) {
  if (dtype == GLIDE_BF16) {
    if (out_f32) {
      if (d == 128 && Df == 128) return launch_rows_t<bf16_t, 128, 128, float>(Wf, x, rows, out, phi, s);
      if (d == 128 && Df == 64) return launch_rows_t<bf16_t, 128, 64, float>(Wf, x, rows, out, phi, s);
      if (d == 64 && Df == 128) return launch_rows_t<bf16_t, 64, 128, float>(Wf, x, rows, out, phi, s);
      if (d == 64 && Df == 64) return launch_rows_t<bf16_t, 64, 64, float>(Wf, x, rows, out, phi, s);
    } else {
      if (d == 128 && Df == 128) return launch_rows_t<bf16_t, 128, 128, bf16_t>(Wf, x, rows, out, phi, s);
      if (d == 128 && Df == 64) return launch_rows_t<bf16_t, 128, 64, bf16_t>(Wf, x, rows, out, phi, s);
      if (d == 64 && Df == 128) return launch_rows_t<bf16_t, 64, 128, bf16_t>(Wf, x, rows, out, phi, s);
      if (d == 64 && Df == 64) return launch_rows_t<bf16_t, 64, 64, bf16_t>(Wf, x, rows, out, phi, s);
    }
  } else {
    if (d == 128 && Df == 128) return launch_rows_t<float, 128, 128, float>(Wf, x, rows, out, phi, s);
    if (d == 128 && Df == 64) return launch_rows_t<float, 128, 64, float>(Wf, x, rows, out, phi, s);
    if (d == 64 && Df == 128) return launch_rows_t<float, 64, 128, float>(Wf, x, rows, out, phi, s);
    if (d == 64 && Df == 64) return launch_rows_t<float, 64, 64, float>(Wf, x, rows, out, phi, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace glide
