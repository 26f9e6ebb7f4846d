// GLIDE decode step: one fused pass per (layer, sequence, KV head).
//
// Per unit (GLIDE Sec. III-B; the state recurrence of Sec. II-B applied to
// the tokens that have left the window):
//   1. the new key/value is written to ring slot p mod R;
//   2. phi of the G query heads and of the pending keys (tokens that have
//      left the window but are not yet folded into S, z) on MFMA against Wf,
//      each wave producing the features of the state rows it owns;
//   3. state: the read-out phi(q_h).S, phi(q_h).z from one pass over the S
//      rows, plus the pending tokens through a_hj = phi(q_h).phi(k_j)
//      (sum_j a_hj v_j, sum_j a_hj); on the unit's fold step the pending
//      tokens are first added to the rows in registers, S', z' written back
//      and read out (deferred folding: at most one write of the state per
//      kFoldPeriod steps);
//   4. window: the W most recent tokens (ring tokens p-W+1 .. p-1 plus the new
//      token taken straight from the input) are streamed in 32-token tiles,
//      the next tile's loads in flight while the current one is computed;
//      QK^T and PV run on MFMA with the G query heads of the group as the
//      16-wide tile dimension; online softmax in the log2 domain;
//   5. merge of the two parts over one shared denominator, output, pos += 1.
//
// One workgroup of 4 waves handles one unit, or one piece of a unit's window
// when a launch has few units (each piece writes a partial record to memory;
// the last to finish merges them); units of the call are ordered by
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

__device__ __forceinline__ uint2 bload8(brsrc_t r, uint32_t off) {
  return __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0));
}

// A wave-uniform 64-bit value from vector registers, in scalar registers.
__device__ __forceinline__ uint64_t uniform64(uint32_t lo, uint32_t hi) {
  return uint64_t(uint32_t(__builtin_amdgcn_readfirstlane(int(lo)))) |
         (uint64_t(uint32_t(__builtin_amdgcn_readfirstlane(int(hi)))) << 32);
}

// x mod R for a position x >= 0 (a 64-bit remainder only past 2^32).
__device__ __forceinline__ int32_t ring_slot(int64_t x, int32_t R) {
  return (uint64_t(x) >> 32) == 0 ? int32_t(uint32_t(x) % uint32_t(R)) : int32_t(x % R);
}

// (slot + off) mod R, for an offset of a few rings at most.
__device__ __forceinline__ int32_t ring_add(int32_t slot, int64_t off, int32_t R) {
  const int32_t m = (slot + int32_t(off)) % R;
  return m < 0 ? m + R : m;
}

__device__ __forceinline__ int clamp_rel(int64_t x) { return int(x < -1 ? -1 : (x > 32 ? 32 : x)); }

template <typename T, int D>
struct WindowTile {
  Frag<T> k[2][D / 32];  // A operand rows of the two 16-key sub-tiles
  Frag<T> v[D / 16];     // B operand: 8 tokens x 1 column per lane, per column tile
};

#ifndef GLIDE_DECODE_WAVES_PER_SIMD
#define GLIDE_DECODE_WAVES_PER_SIMD 2
#endif

// Merge of the pieces of a split unit, run by the last of its workgroups to
// finish (see the end of decode_kernel): the window parts (running max m, sum
// l, weighted values acc per piece) over one max, plus piece 0's linear part,
// over the shared denominator (hybrid forms: each part normalised on its
// own, then added); then pos = p + 1.  The pieces may run on different XCDs,
// whose L2s are not coherent with each other: the records were written
// through to memory and are read from there, every load of the workgroup
// issued before the first wait.
template <typename T, int D, int DF, int NP, int EPT>
__device__ __forceinline__ void merge_unit(const DecodeArgs& a, const LayerArg& L, int rem, int64_t p) {
  static_assert(kMaxPieces * kMaxG <= kThreads, "one (piece, head) scalar pair per thread");
  __shared__ float pw[kThreads];  // [piece][G]: m
  __shared__ float pe[kThreads];  // [piece][G]: the piece's weight e^(m - M)
  __shared__ float pl[kThreads];  // [piece][G]: l e^(m - M)
  __shared__ float pd[kMaxG];     // per head: the linear denominator
  __shared__ float pm[kMaxG];     // per head: M, the max over the pieces
  const int G = a.G, B = a.B, Hkv = a.Hkv, Hq = a.Hq;
  const int per_layer = B * Hkv;
  const int np = L.npiece;
  const int b = rem / Hkv, g = rem - b * Hkv;
  const int64_t unit = int64_t(b) * Hkv + g;
  const LayerSections sec = layer_sections(B, Hkv, D, DF, L.R, sizeof(T));
  int64_t* pos_ptr = reinterpret_cast<int64_t*>(a.state + L.base + sec.pos) + unit;
  const int64_t tok = int64_t(L.slot) * B + b;
  T* og = reinterpret_cast<T*>(a.out) + (tok * Hq + int64_t(g) * G) * D;
  constexpr int RH = 2 * D + 3;  // floats per head in a record
  const uint32_t rb = uint32_t(part_floats(G, D)) * 4;  // bytes per record
  // piece 0's record, and those of pieces 1 .. np-1 (consecutive rows)
  const brsrc_t r0 = make_rsrc(a.part + (int64_t(L.prow0) * per_layer + rem) * part_floats(G, D), rb);
  const brsrc_t r1 = make_rsrc(a.part + (int64_t(L.prow1) * per_layer + rem) * part_floats(G, D),
                               uint32_t(np - 1) * uint32_t(per_layer) * rb);
  const uint32_t rs = uint32_t(per_layer) * rb;  // bytes between pieces 1..
  const int tid = threadIdx.x;
  const int n = G * D;
  // per piece and head: m, l (threads tid < np * G), loaded first
  const int mpc = tid / G, mh = tid - mpc * G;
  const bool mok = tid < np * G;
  const uint32_t mo = uint32_t(mh * RH) * 4;
  const float m0 = bload_f_sys(r0, mok && mpc == 0 ? mo : kOOB);
  const float m1 = bload_f_sys(r1, mok && mpc > 0 ? (mpc - 1) * rs + mo : kOOB);
  const float l0 = bload_f_sys(r0, mok && mpc == 0 ? mo + 4 : kOOB);
  const float l1 = bload_f_sys(r1, mok && mpc > 0 ? (mpc - 1) * rs + mo + 4 : kOOB);
  const float dnv = bload_f_sys(r0, tid < G ? uint32_t(tid * RH + 2) * 4 : kOOB);  // linear denominator
  float v[EPT][NP], nmv[EPT];
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const int i = tid + e * kThreads;
    const int hh = i / D, c = i - hh * D;
    const uint32_t o = uint32_t(hh * RH + 3 + c) * 4;
    const bool ok = i < n;
    v[e][0] = bload_f_sys(r0, ok ? o : kOOB);
#pragma unroll
    for (int pc = 1; pc < NP; ++pc) v[e][pc] = bload_f_sys(r1, ok && pc < np ? (pc - 1) * rs + o : kOOB);
    nmv[e] = bload_f_sys(r0, ok ? o + D * 4 : kOOB);
  }
  // every thread writes its slot (kThreads slots; no branch, so the loads
  // above are not sunk behind the record loads)
  const float mm = m0 + m1, ll = l0 + l1;  // at most one of each pair is not an OOB zero
  pw[tid] = mm;
  if (tid < kMaxG) pd[tid] = dnv;
  __syncthreads();
  // the weight of each (piece, head), one thread each
  if (mok) {
    float M = -INFINITY;
#pragma unroll
    for (int pc = 0; pc < NP; ++pc)
      if (pc < np) M = fmaxf(M, pw[pc * G + mh]);
    const float w = mm == -INFINITY ? 0.f : exp2f(mm - M);
    pe[tid] = w;
    pl[tid] = ll * w;
    if (mpc == 0) pm[mh] = M;
  }
  __syncthreads();
  auto out_elem = [&](int i, const float (&vp)[NP], float nm) {
    const int hh = i / D;
    const float M = pm[hh];
    float Ls = 0.f, Ac = 0.f;
#pragma unroll
    for (int pc = 0; pc < NP; ++pc) {
      if (pc < np) {
        Ls += pl[pc * G + hh];
        Ac = fmaf(vp[pc], pe[pc * G + hh], Ac);
      }
    }
    const float dn = pd[hh];
    float o;
    if (a.form != 0) {  // hybrid forms: each part over its own denominator
      o = Ac / Ls + (dn > 0.f ? nm / dn : 0.f);
    } else {
      // (no branch: an empty linear part, dn = 0, weighs 0 and leaves Ac / Ls)
      const bool lin = dn > 0.f;
      const float c2 = fmaxf(M, lin ? log2f(dn) : -INFINITY);
      const float ws = exp2f(M - c2), wlin = lin ? exp2f(-c2) : 0.f;
      o = (Ac * ws + nm * wlin) / (Ls * ws + dn * wlin);
    }
    og[i] = from_f32<T>(o);
  };
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const int i = tid + e * kThreads;
    if (i < n) out_elem(i, v[e], nmv[e]);
  }
  for (int i = tid + EPT * kThreads; i < n; i += kThreads) {  // G * D > EPT * 256 (large G)
    const int hh = i / D, c = i - hh * D;
    const uint32_t o = uint32_t(hh * RH + 3 + c) * 4;
    float vp[NP];
    vp[0] = bload_f_sys(r0, o);
#pragma unroll
    for (int pc = 1; pc < NP; ++pc) vp[pc] = bload_f_sys(r1, pc < np ? (pc - 1) * rs + o : kOOB);
    out_elem(i, vp, bload_f_sys(r0, o + D * 4));
  }
  if (tid == 0) *pos_ptr = p + 1;
}

// NT: non-temporal state and window loads.  GATED: the gated state (its code
// in a separate instantiation, so that the ungated kernel stays smaller:
// 4% fewer instructions, 1-2% faster per step).
template <typename T, int D, int DF, bool NT, bool GATED>
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
  constexpr uint32_t ES = sizeof(T);
  constexpr int PVT = (kFoldPeriod * D + kThreads - 1) / kThreads;  // pending values per thread
  constexpr int WPR = RW * int(ES) / 16;   // 16-byte pieces per staged Wf row (bf16)
  constexpr int WCH = D * WPR / 64 > 0 ? D * WPR / 64 : 1;  // staged pieces per lane
  constexpr int WPITCH = RW + 4;           // staged row pitch in elements (8 bytes of padding: the
                                           // column reads are 8-byte transposing LDS reads)
  static_assert(STEPS * RPS == RW && NTW * 16 == RW, "state rows must tile the wave");
  static_assert(STEPS % 4 == 0, "a lane's state rows are read in fours");

  extern __shared__ __align__(16) float smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hq = lane & 15, lg = lane >> 4;
  const int G = a.G, B = a.B, Hkv = a.Hkv, Hq = a.Hq;
  const int per_layer = B * Hkv;
  const int prow = __builtin_amdgcn_readfirstlane(int(blockIdx.x) / a.row_stride);
  const int rem = int(blockIdx.x) - prow * a.row_stride;
  // (the table is read a dword at a time: a scalar load, no vector memory wait)
  const uint32_t lw = reinterpret_cast<const uint32_t*>(a.piece_layer)[prow >> 2];
  const LayerArg L = a.layers[(lw >> (8 * (prow & 3))) & 0xffu];
  const int piece = prow == L.prow0 ? 0 : prow - L.prow1 + 1;
  const bool split = L.npiece > 1;
  const int b = rem / Hkv, g = rem - b * Hkv;
  const int W = L.W, R = L.R;
  // Wd: the linear part's delay (its set is [0, p + 1 - Wd)): W, or 0 when
  // the state holds every token (the Appendix's second hybrid form)
  const int Wd = a.form == 2 ? 0 : W;
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
  const T* Wf = reinterpret_cast<const T*>(a.phi_w) +
                (a.wf_heads ? int64_t(L.slot) * Hkv + g : int64_t(L.slot)) * D * DF;

  // pos and nf (gated: also G_{p-1}, G_f and the new token's log-gate) are
  // the workgroup's first loads; every load that does not depend on them
  // (the state pass's Wf slice, S rows and z, the queries, the new
  // key/value) follows before the first wait.  They are vector loads read
  // back into scalar registers: scalar loads share one counter with the
  // kernel arguments, so a wait for an argument fetched after them would
  // also wait for them, and hold back the loads behind it.  The compiler
  // barrier keeps this issue order.
  const bool gated = GATED && piece == 0;
  const LayerSections secg = layer_sections(B, Hkv, D, DF, R, sizeof(T), gated);
  double* gst = reinterpret_cast<double*>(lay + secg.G) + 2 * unit;  // [G_{p-1}, G_f]
  double* grg = reinterpret_cast<double*>(lay + secg.GR) + unit * int64_t(R);
  const uint2 pw = bload8(make_rsrc(pos_ptr, 8), 0);
  const uint2 nw = bload8(make_rsrc(nf_ptr, 8), 0);
  const uint4 gw = bload16(make_rsrc(gst, gated ? 16 : 0), 0);
  const float gnw = bload_f(make_rsrc(gated ? a.gates + (tok * Hkv + g) : a.gates, gated ? 4 : 0), 0);
  __asm__ volatile("" ::: "memory");

  float* ph = smem;                        // [G + kFoldPeriod][DF] phi(q_h), then phi(k_j) of pending j
  float* pvl = ph + (G + kFoldPeriod) * DF;  // [kFoldPeriod][D]    values of the pending tokens
  float* kpl = pvl + kFoldPeriod * D;      // [D]           the new key
  float* vpl = kpl + D;                    // [D]           the new value
  float* spl = vpl + D;                    // [kMaxG]       the new token's score (log2 units)
  float* pa = spl + kMaxG;                 // [kMaxG][kFoldPeriod] phi(q_h).phi(k_j) of pending j
  float* lnum = pa + kMaxG * kFoldPeriod;               // [waves][RPS][G][D] linear numerator partials phi(q).S
  float* lden = lnum + kWaves * RPS * G * D;  // [waves][G]    linear denominator partials phi(q).z
  float* wacc = lden + kWaves * G;         // [waves][G][D] window partials sum e^s v
  float* wm = wacc + kWaves * G * D;       // [waves][G]    window running max (log2 units)
  float* wl = wm + kWaves * G;             // [waves][G]    window sum e^s
  // [waves][D][WPITCH] this wave's Wf columns (bf16), staged for the
  // column-gather of the feature map's B fragments.  It shares the memory of
  // lnum .. wl, which are first written after the barrier that follows the
  // feature map, when every wave has read its staged columns.
  T* wfs = reinterpret_cast<T*>(lnum) + wave * D * WPITCH;

  const brsrc_t rq = make_rsrc(qg, uint32_t(G * D) * ES);
  const brsrc_t rk = make_rsrc(kn, D * ES), rv = make_rsrc(vn, D * ES);
  const brsrc_t rS = make_rsrc(S, DF * D * 4), rz = make_rsrc(z, DF * 4);
  const brsrc_t rK = make_rsrc(Kr, uint32_t(R) * D * ES), rV = make_rsrc(Vr, uint32_t(R) * D * ES);
  const brsrc_t rW = make_rsrc(Wf, D * DF * ES);

  // ---- 1. prologue: every load up to the first window tile is issued before
  //         any of them is waited for.
  // The state pass belongs to piece 0 of a unit with a linear part; whether
  // the part is empty yet (beta = 0) or S holds anything (nf > 0) is known
  // only once pos and nf arrive, so the workgroup that may do it loads its
  // operands now and drops them then.
  const bool lin_call = a.linear != 0 && piece == 0;
  const int f0 = wave * RW;
  const int lr = lane / LPR, c4 = (lane % LPR) * 4;
  const int r0 = f0 + lr * STEPS;  // the lane's STEPS consecutive state rows r0 .. r0 + STEPS - 1
  uint4 wst[WCH];  // bf16: this wave's Wf columns, 16-byte row pieces
  Frag<T> wb[KS][NTW];
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int i = 0; i < WCH; ++i) {
      const int c = lane + 64 * i, r = c / WPR, x = c - r * WPR;
      wst[i] = bload16(rW, lin_call ? uint32_t((r * DF + f0 + 8 * x) * ES) : kOOB);
    }
  } else {
#pragma unroll
    for (int kk = 0; kk < KS; ++kk)
#pragma unroll
      for (int nt = 0; nt < NTW; ++nt)
        bload_frag_strided(wb[kk][nt], rW, lin_call ? uint32_t((32 * kk + 8 * lg) * DF + f0 + 16 * nt + hq) * ES : kOOB,
                           DF * ES);
  }
  float4 sr[STEPS];
#pragma unroll
  for (int s = 0; s < STEPS; ++s) sr[s] = bload_f4_s<NT>(rS, lin_call ? uint32_t(((r0 + s) * D + c4) * 4) : kOOB);
  float zf = bload_f(rz, lin_call && lane < RW ? uint32_t((f0 + lane) * 4) : kOOB);
  // the new token's element tid % D (its own score, and the ring write at the end)
  const T kraw = bload_elem(rk, uint32_t(tid % D) * ES, T());
  const T vraw = bload_elem(rv, uint32_t(tid % D) * ES, T());
  Frag<T> fq[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) bload_frag(fq[kk], rq, hq < G ? uint32_t(hq * D + 32 * kk + 8 * lg) * ES : kOOB);

  // (pos, nf and the gate values are read back into scalar registers here)
  const int64_t p = int64_t(uniform64(pw.x, pw.y));
  int64_t nf = int64_t(uniform64(nw.x, nw.y));
  const float gnew = gated ? __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, gnw))) : 0.f;
  const double gcur0 = gated ? __builtin_bit_cast(double, uniform64(gw.x, gw.y)) : 0.0;
  const double gfold = gated ? __builtin_bit_cast(double, uniform64(gw.z, gw.w)) : 0.0;
  const double gcur = gcur0 + double(gnew);  // G_p

  // Linear set after this step: tokens [0, beta).  S, z hold tokens [0, nf);
  // tokens [nf, beta) are pending (in the ring, or the new token when Wd = 0)
  // and enter the read-out through phi(k_j) v_j.  They are folded for good on
  // this step when the unit's turn comes (every step when Wd = 0).
  const int64_t beta = p + 1 - Wd > 0 ? p + 1 - Wd : 0;
  const bool lin_unit = a.linear != 0 && beta > 0;
  const bool lin = lin_unit && piece == 0;  // the state pass belongs to piece 0
  const int fper = Wd > 0 ? kFoldPeriod : 1;
  // nf of a well-formed state lies in [beta - fper, beta]; the clamp keeps
  // every access in bounds whatever the blob holds.
  nf = nf < beta ? nf : beta;
  nf = nf > beta - fper ? nf : beta - fper;
  nf = nf > 0 ? nf : 0;
  const int npend = lin ? int(beta - nf) : 0;  // 0 .. fper
  // (fper is a power of two: the unit's turn is (beta + unit) mod fper = 0)
  const bool fold = npend > 0 && (npend >= fper || ((beta + unit) & (fper - 1)) == 0);
  const bool s_nonzero = lin && nf > 0;  // S, z hold something
  // Ring slots in 32-bit arithmetic: the slot of p once, every other slot
  // from it by an offset of less than a few rings.
  const int32_t pr = R > 0 ? ring_slot(p, R) : 0;  // ring slot of token p
  const int32_t nf_slot = R > 0 ? ring_add(pr, nf - p, R) : 0;  // ring slot of token nf
  // gated: S, z are decayed to G_f; read at p they weigh e^{G_p - G_f}, and
  // pending token j weighs e^{G_p - G_j} (its G_j from the gate ring; the new
  // token itself, pending when Wd = 0, weighs 1)
  __shared__ float pend_decay[kFoldPeriod];
  const bool gate_pend = gated && lin && Wd > 0 && npend > 0;
  if (gate_pend && tid < npend)
    pend_decay[tid] = decay_exp(float(gcur - grg[wrap_once(uint32_t(nf_slot + tid), uint32_t(R))]));
  const float sdecay = gated && s_nonzero ? decay_exp(float(gcur - gfold)) : 1.f;

  // Window: tokens [tlo, p] in 32-token tiles.  Ring tiles cover [tlo, p-1];
  // the new token p (not in the ring yet) is a partial of its own.  The
  // piece takes tiles [t_first, n_tiles) (piece 0 fewer, as it also does the
  // state); wave w takes tiles t_first + w, t_first + w + 4, ...
  const int64_t tlo = p - W + 1 > 0 ? p - W + 1 : 0;
  const int64_t tile0 = tlo >> 5;
  const int n_all = W > 0 ? int((p >> 5) - tile0 + 1) : 0;
  int t_first = 0, n_tiles = n_all;
  if (split) {
    const int off = lin_unit ? a.state_tiles : 0;
    const int share = (n_all + off + L.npiece - 1) / L.npiece;
    t_first = piece * share - off;
    t_first = t_first > 0 ? t_first : 0;
    n_tiles = (piece + 1) * share - off;
    n_tiles = n_tiles < n_all ? n_tiles : n_all;
  }
  const bool own_p = W > 0 && t_first <= n_all - 1 && n_all - 1 < n_tiles;  // the new token's partial
  int it = t_first + wave;
  int64_t j0 = (tile0 + it) << 5;
  uint32_t s0 = W > 0 ? uint32_t(ring_add(pr, j0 - p, R)) : 0u;
  const uint32_t step = W > 0 ? uint32_t((32 * kWaves) % R) : 0u;
  const brsrc_t rpk = Wd > 0 ? rK : rk;  // where pending keys / values live
  const brsrc_t rpv = Wd > 0 ? rV : rv;

  // Tile loads: s0t = (j0 mod R) is a multiple of 32, so the tile is ring
  // block s0t/32 and every fragment load is one contiguous 1 KB read.  Key
  // row m of sub-tile t is token j0 + 8(m/4) + 4t + m%4, so that after QK^T
  // lane group lg holds tokens j0 + 8lg .. j0 + 8lg + 7, exactly the A-operand
  // layout PV needs.  A tile that is not needed reads zeros (no traffic).
  // Only the tile's tokens [lo, pn) (offsets from j0) are in the window: a
  // lane whose key row, or whose 8 value tokens, lie wholly outside it reads
  // zeros instead (no traffic; the edge tiles of a window would otherwise
  // fetch up to 31 tokens each beyond it).  NT: non-temporal loads (a state
  // blob far larger than the Infinity Cache).
  auto load_tile = [&](WindowTile<T, D>& tl, uint32_t s0t, bool valid, int lo, int pn) {
    const uint32_t base = valid ? s0t * D * ES : kOOB;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int tok = 8 * (hq >> 2) + 4 * t + (hq & 3);
      const bool kin = tok >= lo && tok < pn;
#pragma unroll
      for (int kk = 0; kk < KS; ++kk)
        bload_frag_s<NT>(tl.k[t][kk], rK, kin ? base + uint32_t((((t * KS + kk) * 4 + lg) * 16 + hq) * 8) * ES : kOOB);
    }
    const bool vin = 8 * lg + 8 > lo && 8 * lg < pn;
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
      bload_frag_s<NT>(tl.v[ct], rV, vin ? base + uint32_t(((ct * 4 + lg) * 16 + hq) * 8) * ES : kOOB);
  };

  // rows of the feature-map tile, which are also the queries of the window's
  // QK^T: row hq < G is query head hq, rows G .. G+npend-1 the pending keys
  // (second tile: rows 16 ..), other rows zero.  Columns of QK^T beyond G are
  // never read.
  Frag<T> xa[KS], xb[KS];
  {
    const int ia = hq - G, ib = 16 + hq - G;
    const bool pa = hq >= G && ia < npend, pb = ib >= 0 && ib < npend;
    // ring slots of pending tokens nf + i (i < 8 < R: one wrap at most)
    const int32_t sa = Wd > 0 ? int32_t(wrap_once(uint32_t(nf_slot + (pa ? ia : 0)), uint32_t(R))) : 0;
    const int32_t sb = Wd > 0 ? int32_t(wrap_once(uint32_t(nf_slot + (pb ? ib : 0)), uint32_t(R))) : 0;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      Frag<T> fp;
      const uint32_t oa = Wd > 0 ? uint32_t(kring_chunk(sa, kk, lg, D)) * ES : uint32_t(32 * kk + 8 * lg) * ES;
      bload_frag(fp, rpk, pa ? oa : kOOB);
      xa[kk] = frag_or(fq[kk], fp);
      const uint32_t ob = Wd > 0 ? uint32_t(kring_chunk(sb, kk, lg, D)) * ES : uint32_t(32 * kk + 8 * lg) * ES;
      bload_frag(xb[kk], rpk, pb ? ob : kOOB);
    }
  }
  // values of the pending tokens
  // (raw elements, one per register, issued unconditionally: converted only
  // where they are used, so no wait holds back the loads that follow)
  uint32_t pvr[PVT];
#pragma unroll
  for (int u = 0; u < PVT; ++u) {
    const int e = tid + u * kThreads, i = e / D, c = e - i * D;
    const bool ok = i < npend;
    const uint32_t off =
        Wd > 0 ? uint32_t(vring_elem(int32_t(wrap_once(uint32_t(nf_slot + (ok ? i : 0)), uint32_t(R))), c, D)) * ES
               : uint32_t(c) * ES;
    pvr[u] = bload_raw(rpv, ok ? off : kOOB, T());
  }
  // first window tile of this wave
  WindowTile<T, D> ta, tb;
  load_tile(ta, s0, W > 0 && it < n_tiles, clamp_rel(tlo - j0), clamp_rel(p - j0));

  // Wf B fragments of this wave's features: the staged rows are gathered by
  // column from LDS (the wave reads only what it wrote itself).
  if constexpr (sizeof(T) == 2) {
    if (lin) {
#pragma unroll
      for (int i = 0; i < WCH; ++i) {
        const int c = lane + 64 * i, r = c / WPR, x = c - r * WPR;
        T* d0 = wfs + r * WPITCH + 8 * x;
        const uint32_t w4[4] = {wst[i].x, wst[i].y, wst[i].z, wst[i].w};
        // (byte copies: the element reads below must not be ordered before
        // these writes, which a type-based alias assumption would allow)
#pragma unroll
        for (int j = 0; j < 4; ++j) __builtin_memcpy(d0 + 2 * j, &w4[j], 4);
      }
#pragma unroll
      for (int kk = 0; kk < KS; ++kk)
#pragma unroll
        for (int nt = 0; nt < NTW; ++nt) load_colfrag(wb[kk][nt], wfs, WPITCH, 32 * kk + 8 * lg, 16 * nt);
    }
  }

  // ---- 2. feature map on MFMA: rows x Wf, this wave's RW features, fp32
  if (lin) {
    const int nrows = G + npend;
    f32x4_t acc[NTW], acb[NTW];
#pragma unroll
    for (int nt = 0; nt < NTW; ++nt) {
      acc[nt] = zero4();
      acb[nt] = zero4();
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        acc[nt] = mma(xa[kk], wb[kk][nt], acc[nt]);
        acb[nt] = mma(xb[kk], wb[kk][nt], acb[nt]);
      }
    }
#pragma unroll
    for (int nt = 0; nt < NTW; ++nt) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = 4 * lg + i;
        if (row < nrows) ph[row * DF + f0 + 16 * nt + hq] = feat_act(acc[nt][i], a.phi);
        if (16 + row < nrows) ph[(16 + row) * DF + f0 + 16 * nt + hq] = feat_act(acb[nt][i], a.phi);
      }
    }
  }

  if (lin) {
#pragma unroll
    for (int u = 0; u < PVT; ++u) {
      const int e = tid + u * kThreads;
      if (e < kFoldPeriod * D) pvl[e] = raw_to_f32(pvr[u], T());
    }
  }
  if (own_p && tid < D) {
    kpl[tid] = to_f32(kraw);
    vpl[tid] = to_f32(vraw);
  }
  if (lin && a.phi == GLIDE_PHI_SOFTMAX) {  // the softmax map: normalise every row of ph
    __syncthreads();
    softmax_rows_lds<DF, kThreads>(ph, DF, G + npend);
  }
  if (tid < kMaxG) spl[tid] = -INFINITY;
  __syncthreads();
  if (gate_pend) {  // the pending keys' features carry their decay
    for (int e = tid; e < npend * DF; e += kThreads) ph[G * DF + e] *= pend_decay[e / DF];
    __syncthreads();
  }

  const float sc2 = a.tau * kLog2e;
  // ---- 3. the new token's score, one per query head (wave 0)
  if (own_p && wave == 0) {
    float d = 0.f;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      float x[8];
      xa[kk].to_floats(x);
#pragma unroll
      for (int e = 0; e < 8; ++e) d = fmaf(x[e], kpl[32 * kk + 8 * lg + e], d);
    }
    d += __shfl_xor(d, 16);
    d += __shfl_xor(d, 32);
    if (lane < G) spl[lane] = d * sc2;
  }

  // ---- 4. state.  The read-out of the pending tokens [nf, beta) needs no
  //         update of S: phi(q_h).S' = phi(q_h).S + sum_j a_hj v_j with
  //         a_hj = phi(q_h).phi(k_j) (z' likewise), so each wave reads out
  //         its S rows as loaded and the a_hj enter in the merge.  On a fold
  //         step the pending tokens are first added to the S rows, in
  //         registers, S', z' are written back (rows no pending token touches
  //         are unchanged and skipped), and the read-out is taken from S'.
  //         (Folding after this step's results are out, with the rows read
  //         again, made the B=1 step slower: the extra reads land at the end
  //         of the launch.)
  const bool early = fold;  // fold before the read-out
  const float* pk = ph + G * DF;
  // S' = S + sum_j phi(k_j)^T v_j on the wave's rows (and z'), written back.
  // The lane's rows are consecutive, so a token's weights for them come from
  // LDS in 16-byte reads; tokens go two at a time, their reads issued
  // together.  Every row is written on a fold: with up to kFoldPeriod tokens
  // a row none of them touches is rare.
  auto fold_rows = [&](float4 (&rows)[STEPS], float& zrow) {
    float dz = 0.f;
    for (int i = 0; i < npend; i += 2) {
      const int i1 = i + 1 < npend ? i + 1 : i;
      const float sc1 = i + 1 < npend ? 1.f : 0.f;  // an odd count: the last pair's second token weighs 0
      const float4 v0 = *reinterpret_cast<const float4*>(pvl + i * D + c4);
      float4 v1 = *reinterpret_cast<const float4*>(pvl + i1 * D + c4);
      v1 = make_float4(v1.x * sc1, v1.y * sc1, v1.z * sc1, v1.w * sc1);
      float w0[STEPS], w1[STEPS];
#pragma unroll
      for (int s = 0; s < STEPS; s += 4) {
        const float4 a = *reinterpret_cast<const float4*>(pk + i * DF + r0 + s);
        const float4 b = *reinterpret_cast<const float4*>(pk + i1 * DF + r0 + s);
        w0[s] = a.x; w0[s + 1] = a.y; w0[s + 2] = a.z; w0[s + 3] = a.w;
        w1[s] = b.x; w1[s + 1] = b.y; w1[s + 2] = b.z; w1[s + 3] = b.w;
      }
#pragma unroll
      for (int s = 0; s < STEPS; ++s) {
        rows[s].x = fmaf(w1[s], v1.x, fmaf(w0[s], v0.x, rows[s].x));
        rows[s].y = fmaf(w1[s], v1.y, fmaf(w0[s], v0.y, rows[s].y));
        rows[s].z = fmaf(w1[s], v1.z, fmaf(w0[s], v0.z, rows[s].z));
        rows[s].w = fmaf(w1[s], v1.w, fmaf(w0[s], v0.w, rows[s].w));
      }
      if (lane < RW) dz += pk[i * DF + f0 + lane] + sc1 * pk[i1 * DF + f0 + lane];
    }
    zrow += dz;
#pragma unroll
    for (int s = 0; s < STEPS; ++s) store_nt(S + (r0 + s) * D + c4, rows[s]);
    if (lane < RW) z[f0 + lane] = zrow;
  };
  if (lin) {
    // S, z are zero until the first fold (their memory is not read as such)
    if (!s_nonzero) {
#pragma unroll
      for (int s = 0; s < STEPS; ++s) sr[s] = make_float4(0.f, 0.f, 0.f, 0.f);
      zf = 0.f;
    } else if (gated) {  // S, z decayed from G_f to G_p
#pragma unroll
      for (int s = 0; s < STEPS; ++s)
        sr[s] = make_float4(sr[s].x * sdecay, sr[s].y * sdecay, sr[s].z * sdecay, sr[s].w * sdecay);
      zf *= sdecay;
    }
    if (early) fold_rows(sr, zf);
    for (int hh = 0; hh < G; ++hh) {
      const float* pq = ph + hh * DF;
      float4 n4 = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int s = 0; s < STEPS; s += 4) {
        const float4 w4 = *reinterpret_cast<const float4*>(pq + r0 + s);
        const float w[4] = {w4.x, w4.y, w4.z, w4.w};
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          n4.x = fmaf(w[u], sr[s + u].x, n4.x);
          n4.y = fmaf(w[u], sr[s + u].y, n4.y);
          n4.z = fmaf(w[u], sr[s + u].z, n4.z);
          n4.w = fmaf(w[u], sr[s + u].w, n4.w);
        }
      }
      // the RPS row groups of the wave are summed in the merge (no
      // cross-lane exchange here); the denominator partial over the wave's
      // RW features is reduced within DPP rows
      *reinterpret_cast<float4*>(lnum + ((wave * RPS + lr) * G + hh) * D + c4) = n4;
      const float dp = dpp_sum_rows<RW>(lane < RW ? pq[f0 + lane] * zf : 0.f);
      if (lane == (RW > 16 ? 16 : 0)) lden[wave * G + hh] = dp;
    }
    if (!early && npend > 0) {
      // a_hj = phi(q_h).phi(k_j): 16 lanes (one DPP row) per head, DF / 16
      // features each
      constexpr int FPL = DF / 16;
      const int hh = tid >> 4, sub = tid & 15;
      const bool hv = hh < G;
      float qf[FPL];
#pragma unroll
      for (int j = 0; j < FPL; ++j) qf[j] = hv ? ph[hh * DF + sub * FPL + j] : 0.f;
      for (int i = 0; i < npend; ++i) {
        float d = 0.f;
#pragma unroll
        for (int j = 0; j < FPL; ++j) d = fmaf(qf[j], pk[i * DF + sub * FPL + j], d);
        d = dpp_sum_rows<16>(d);
        if (hv && sub == 0) pa[hh * kFoldPeriod + i] = d;
      }
    }
  }

  // ---- 5. window: softmax over the ring tokens [tlo, p-1]
  if (W > 0) {
    f32x4_t acc[CT];
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) acc[ct] = zero4();
    // running max (log2 units) and per-lane sum; the accumulator is only
    // rescaled when the max grows by more than 8 (weights stay below 2^8)
    float m_run = -INFINITY, l_run = 0.f;

    auto compute_tile = [&](const WindowTile<T, D>& tl, int lo, int pn) {
      f32x4_t sc[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        sc[t] = zero4();
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) sc[t] = mma(tl.k[t][kk], xa[kk], sc[t]);
      }
      float s[8];
      if (lo <= 0 && pn >= 32) {
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int i = 0; i < 4; ++i) s[4 * t + i] = sc[t][i] * sc2;
      } else {
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int off = 8 * lg + 4 * t + i;
            s[4 * t + i] = (off >= lo && off < pn) ? sc[t][i] * sc2 : -INFINITY;
          }
      }
      float mx = s[0];
#pragma unroll
      for (int i = 1; i < 8; ++i) mx = fmaxf(mx, s[i]);
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      if (__any(mx > m_run + 8.f)) {
        const float m_new = fmaxf(m_run, mx);
        const float alpha = m_run == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m_run - m_new);
        l_run *= alpha;
        m_run = m_new;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float al = __shfl(alpha, 4 * lg + i);
#pragma unroll
          for (int ct = 0; ct < CT; ++ct) acc[ct][i] *= al;
        }
      }
      const float m_use = m_run == -INFINITY ? 0.f : m_run;
      float pv[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) pv[i] = __builtin_amdgcn_exp2f(s[i] - m_use);
      Frag<T> pf;
      pf.set8(pv);
      l_run += pf.sum();
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) acc[ct] = mma(pf, tl.v[ct], acc[ct]);
    };

    // two register stages: the next tile's loads are in flight while the
    // current one is computed (a tile past the range reads zeros)
    while (it < n_tiles) {
      load_tile(tb, wrap_once(s0 + step, R), it + kWaves < n_tiles, clamp_rel(tlo - j0 - 32 * kWaves),
                clamp_rel(p - j0 - 32 * kWaves));
      compute_tile(ta, clamp_rel(tlo - j0), clamp_rel(p - j0));
      it += kWaves;
      j0 += 32 * kWaves;
      s0 = wrap_once(s0 + step, R);
      if (it >= n_tiles) break;
      load_tile(ta, wrap_once(s0 + step, R), it + kWaves < n_tiles, clamp_rel(tlo - j0 - 32 * kWaves),
                clamp_rel(p - j0 - 32 * kWaves));
      compute_tile(tb, clamp_rel(tlo - j0), clamp_rel(p - j0));
      it += kWaves;
      j0 += 32 * kWaves;
      s0 = wrap_once(s0 + step, R);
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
  __syncthreads();

  // ---- 6. merge over the waves and the new token (and, for a split unit,
  //         over the pieces: each writes a record, the last to finish merges
  //         them): one shared denominator, or (hybrid forms) the window's and
  //         the linear part's normalised outputs added
  const brsrc_t rrec =
      make_rsrc(a.part + (int64_t(prow) * per_layer + rem) * part_floats(G, D), uint32_t(part_floats(G, D)) * 4);
  for (int i = tid; i < G * D; i += kThreads) {
    const int hh = i / D, c = i - hh * D;
    float nm = 0.f, dn = 0.f;
    if (lin) {
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
#pragma unroll
        for (int r = 0; r < RPS; ++r) nm += lnum[((w * RPS + r) * G + hh) * D + c];
        dn += lden[w * G + hh];
      }
      if (!early) {  // the pending tokens: sum_j a_hj v_j, sum_j a_hj
        for (int j = 0; j < npend; ++j) {
          const float aj = pa[hh * kFoldPeriod + j];
          nm = fmaf(aj, pvl[j * D + c], nm);
          dn += aj;
        }
      }
    }
    float M = -INFINITY, Ls = 0.f, Ac = 0.f;
    if (W > 0) {
      const float sp = spl[hh];
      M = sp;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) M = fmaxf(M, wm[w * G + hh]);
      // (no branches: a part with no scores has max -inf and weighs
      // exp2(-inf) = 0; the frame is 0 when every part is empty, and the
      // new token's value is selected only when it was scored)
      const float Mf = M == -INFINITY ? 0.f : M;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const float e = __builtin_amdgcn_exp2f(wm[w * G + hh] - Mf);
        Ls = fmaf(wl[w * G + hh], e, Ls);
        Ac = fmaf(wacc[(w * G + hh) * D + c], e, Ac);
      }
      const float ep = __builtin_amdgcn_exp2f(sp - Mf);
      Ls += ep;
      Ac = sp != -INFINITY ? fmaf(vpl[c], ep, Ac) : Ac;
    }
    if (split) {
      const uint32_t ro = uint32_t(hh * (2 * D + 3)) * 4;
      if (c == 0) {
        bstore_f_sys(rrec, ro, M);
        bstore_f_sys(rrec, ro + 4, Ls);
        bstore_f_sys(rrec, ro + 8, dn);
      }
      bstore_f_sys(rrec, ro + uint32_t(3 + c) * 4, Ac);
      if (piece == 0) bstore_f_sys(rrec, ro + uint32_t(3 + D + c) * 4, nm);
      continue;
    }
    float o;
    if (a.form != 0) {  // the Appendix's hybrid forms: two normalised outputs added
      o = (W > 0 ? Ac / Ls : 0.f) + (dn > 0.f ? nm / dn : 0.f);
    } else if (W > 0) {
      // (no branch: an empty linear part, dn = 0, weighs 0 and leaves Ac / Ls)
      const bool lin_part = dn > 0.f;
      const float c2 = fmaxf(M, lin_part ? log2f(dn) : -INFINITY);
      const float ws = exp2f(M - c2), wlin = lin_part ? exp2f(-c2) : 0.f;
      o = (Ac * ws + nm * wlin) / (Ls * ws + dn * wlin);
    } else {
      o = dn > 0.f ? nm / dn : 0.f;
    }
    og[i] = from_f32<T>(o);
  }
  if (split) {
    // Every record store of the workgroup has reached memory (written
    // through, and waited for) before the unit's count moves; the count is
    // a device-scope add, performed where every XCD sees it.  The workgroup
    // that brings it to npiece reads the records from memory, merges, and
    // resets the count.
    __shared__ int last;
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (tid == 0) {
      int* cnt = reinterpret_cast<int*>(lay + sec.cnt) + unit;
      last = __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == L.npiece - 1;
      if (last) __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    if (last) {
      // one instantiation per piece-count bound (record loads for 4, 8 or 16
      // pieces), four output elements per thread: more variants of this
      // rarely run merge grew the kernel's code enough to slow the window
      // loop of every workgroup (70B slice 748 -> 810 us per step)
      if (L.npiece <= 4) merge_unit<T, D, DF, 4, 4>(a, L, rem, p);
      else if (L.npiece <= 8) merge_unit<T, D, DF, 8, 4>(a, L, rem, p);
      else merge_unit<T, D, DF, kMaxPieces, 4>(a, L, rem, p);
    }
  }

  // ---- 7. the new token into its ring slot (no token of this step reads
  //         that slot), position and fold count
  if (W > 0 && piece == 0 && tid < D) {
    const int32_t sn = pr;
    Kr[kring_elem(sn, tid, D)] = kraw;
    Vr[vring_elem(sn, tid, D)] = vraw;
  }
  if (tid == 0 && piece == 0) {
    if (!split) *pos_ptr = p + 1;  // a split unit's position moves in merge_unit
    if (fold) *nf_ptr = beta;
    if (gated) {
      gst[0] = gcur;
      if (fold) gst[1] = gcur;
      if (W > 0) grg[pr] = gcur;
    }
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
  // units whose linear part is not delayed (W = 0, or the state over every
  // token) fold on every step
  if (W == 0 || a.form == 2) return;
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
  // gated: S, z (decayed to G_f) and the pending tokens are brought to
  // G_{p-1}, the last token consumed
  const bool gated = a.gated != 0;
  const LayerSections secg = layer_sections(a.B, a.Hkv, D, DF, R, sizeof(T), gated);
  double* gst = reinterpret_cast<double*>(lay + secg.G) + 2 * unit;
  const double* grg = reinterpret_cast<const double*>(lay + secg.GR) + unit * int64_t(R);
  const double gcur = gated ? gst[0] : 0.0;
  const bool regate = gated && nf > 0 && gst[1] != gcur;
  if (n == 0 && !regate) return;
  float* S = reinterpret_cast<float*>(lay + sec.S) + unit * DF * D;
  float* z = reinterpret_cast<float*>(lay + sec.z) + unit * DF;
  const T* Kr = reinterpret_cast<const T*>(lay + sec.K) + unit * int64_t(R) * D;
  const T* Vr = reinterpret_cast<const T*>(lay + sec.V) + unit * int64_t(R) * D;
  const T* Wf = reinterpret_cast<const T*>(a.phi_w) +
                (a.wf_heads ? int64_t(L.slot) * a.Hkv + int64_t(unit % a.Hkv) : int64_t(L.slot)) * D * DF;
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
    pk[i][f] = feat_act(acc, a.phi);
  }
  __syncthreads();
  if (a.phi == GLIDE_PHI_SOFTMAX) {
    softmax_rows_lds<DF, kThreads>(&pk[0][0], DF, n);
    __syncthreads();
  }
  if (gated && n > 0) {
    for (int e = tid; e < n * DF; e += kThreads) {
      const int i = e / DF, f = e - i * DF;
      pk[i][f] *= decay_exp(float(gcur - grg[(nf + i) % R]));
    }
    __syncthreads();
  }
  const bool s_nonzero = nf > 0;
  const float sd = gated && s_nonzero ? decay_exp(float(gcur - gst[1])) : 1.f;
  for (int e = tid; e < DF * D / 4; e += kThreads) {
    const int f = e / (D / 4), c4 = (e - f * (D / 4)) * 4;
    float4 sv = s_nonzero ? *reinterpret_cast<const float4*>(S + f * D + c4) : make_float4(0.f, 0.f, 0.f, 0.f);
    sv.x *= sd; sv.y *= sd; sv.z *= sd; sv.w *= sd;
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
    float zf = s_nonzero ? z[f] * sd : 0.f;
    for (int i = 0; i < n; ++i) zf += pk[i][f];
    z[f] = zf;
  }
  __syncthreads();  // every thread has read G_f
  if (tid == 0) {
    *nf_ptr = beta;
    if (gated) gst[1] = gcur;
  }
}

template <typename T, int D, int DF>
hipError_t flush_t(const DecodeArgs& a, hipStream_t stream) {
  const dim3 grid(unsigned(a.n_layers) * unsigned(a.B) * unsigned(a.Hkv));
  hipLaunchKernelGGL((flush_kernel<T, D, DF>), grid, dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

template <typename T, int D, int DF>
hipError_t launch_t(const DecodeArgs& a, int total_wg, bool streaming, hipStream_t stream) {
  const int G = a.G;
  // ph, pvl, kpl, vpl, spl, pa; then lnum .. wl, or the staged Wf columns that
  // share their memory (bf16: kWaves x D rows of RW + 2 elements)
  const size_t head = size_t(G + kFoldPeriod) * DF + size_t(kFoldPeriod) * D + 2 * D + kMaxG + kMaxG * kFoldPeriod;
  constexpr int RPS = 256 / D;  // state rows per wave step (lanes per row: D / 4)
  const size_t tail = size_t(kWaves) * RPS * G * D + kWaves * G + size_t(kWaves) * G * D + kWaves * G + kWaves * G;
  const size_t staged = sizeof(T) == 2 ? size_t(kWaves) * D * (DF / kWaves + 4) / 2 : 0;
  const size_t floats = head + (tail > staged ? tail : staged);
  const dim3 grid(static_cast<unsigned>(total_wg)), block(kThreads);
  const size_t lds = floats * sizeof(float);
  if (a.gated) {
    if (streaming) hipLaunchKernelGGL((decode_kernel<T, D, DF, true, true>), grid, block, lds, stream, a);
    else hipLaunchKernelGGL((decode_kernel<T, D, DF, false, true>), grid, block, lds, stream, a);
  } else {
    if (streaming) hipLaunchKernelGGL((decode_kernel<T, D, DF, true, false>), grid, block, lds, stream, a);
    else hipLaunchKernelGGL((decode_kernel<T, D, DF, false, false>), grid, block, lds, stream, a);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_decode(const DecodeArgs& a, int total_wg, int d, int Df, int dtype, bool streaming,
                         hipStream_t stream) {
  if (dtype == GLIDE_BF16) {
    if (d == 128 && Df == 128) return launch_t<bf16_t, 128, 128>(a, total_wg, streaming, stream);
    if (d == 128 && Df == 64) return launch_t<bf16_t, 128, 64>(a, total_wg, streaming, stream);
    if (d == 64 && Df == 128) return launch_t<bf16_t, 64, 128>(a, total_wg, streaming, stream);
    if (d == 64 && Df == 64) return launch_t<bf16_t, 64, 64>(a, total_wg, streaming, stream);
  } else {
    if (d == 128 && Df == 128) return launch_t<float, 128, 128>(a, total_wg, streaming, stream);
    if (d == 128 && Df == 64) return launch_t<float, 128, 64>(a, total_wg, streaming, stream);
    if (d == 64 && Df == 128) return launch_t<float, 64, 128>(a, total_wg, streaming, stream);
    if (d == 64 && Df == 64) return launch_t<float, 64, 64>(a, total_wg, streaming, stream);
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
