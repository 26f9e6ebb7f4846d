/*
 * GLIDE hybrid-attention layer: plain CPU oracle (test infrastructure only).
 *
 * This file is the reference the GPU kernels are judged against.  It is
 * deliberately slow and literal: scalar loops, double precision, no BLAS,
 * no blocking.  Only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg may load it; the product library never does, and the two
 * share no source, header or helper.
 *
 * What is computed (GLIDE paper, Sec. III-B, the first displayed equation of
 * the section and the two that expand it; Sec. II-B for linear attention;
 * Sec. II-C for the sliding window):
 *
 *   For layer window W >= 0, query position t (0-indexed) and query head h
 *   that reads KV head g = h / G (G = Hq / Hkv, contiguous groups):
 *
 *     beta(t)   = max(0, t + 1 - W)
 *     linear set   L = [0, beta)        (empty when the linear part is off)
 *     softmax set  X = [beta, t]        (min(W, t+1) tokens, current included)
 *     phi(x)_f  = max(0, sum_c x_c Wf[c][f])        (ReLU feature map; or, with
 *                 oracle_layer.phi = 1, ELU+1: y + 1 for y > 0, e^y otherwise,
 *                 y = sum_c x_c Wf[c][f]; both from the Appendix's list of
 *                 feature maps; or, with oracle_layer.phi = 2, the softmax
 *                 feature map Sec. III-B names as its default choice:
 *                 e^{y_f} / sum_f' e^{y_f'}, over the Df projected features)
 *                 (Wf: one per layer, or, with oracle_layer.wf_per_head, one per
 *                 KV head, used for that group's queries and keys)
 *     a_j       = phi(q_t) . phi(k_j)               for j in L
 *     A = sum_{j in L} a_j v_j ,  a = sum_{j in L} a_j
 *     s_j = tau * q_t . k_j                          for j in X
 *     O_t = (sum_{j in X} e^{s_j} v_j + A) / (sum_{j in X} e^{s_j} + a)
 *
 *   With a gated (GLA-style) linear state (oracle_attend_gated / oracle_state_gated,
 *   one log-gate lg[t][g] <= 0 per token and KV head; the paper names GLA-style
 *   gating among the linear forms it supports without fixing the gate), each
 *   a_j is weighted by e^{sum_{i=j+1..t} lg[i][g]}: the decay since j arrived.
 *
 *   i.e. the softmax window and the linear state share one denominator (the
 *   "merge weighted by the normalising denominators" of Sec. II-A / III-B).
 *   The expression is evaluated with a stabiliser c = max(m, ln a)
 *   (m = max_j s_j; c = m when a == 0); any c gives the same exact value.
 *   With W = 0 the softmax set is empty and O_t = A / a; 0/0 is defined as 0.
 *
 *   Recurrent state after p tokens (Sec. II-B recurrence, applied to the
 *   tokens that have left the window, Appendix hybrid form 1):
 *     S = sum_{j < p - W} phi(k_j)^T v_j   (Df x d),  z = sum_{j < p - W} phi(k_j)
 *
 *   A decode step at position p first folds the token leaving the window
 *   (token p - W when p >= W; the current token when W = 0), then appends the
 *   new token to the window, then reads out with the updated S and z.
 *
 * The Appendix's two hybrid-attention equations (retention-based sliding
 * window) add two separately normalised outputs instead, and the paper states
 * that GLIDE adapts both through its merge operator.  They are selected by
 * oracle_layer.form:
 *   form 0  GLIDE: the shared denominator above, linear set [0, beta);
 *   form 1  hybrid form 1: O_t = A / a + sum_X e^{s_j} v_j / sum_X e^{s_j},
 *           linear set [0, beta) (the tokens evicted from the window);
 *   form 2  hybrid form 2: the same sum, linear set [0, t] (the state holds
 *           every token, those still in the window included).
 * Each term of a sum is 0 when its set is empty (and A / a is 0 when a = 0).
 * The state after p tokens covers the linear set of the next position:
 * [0, p - W) in forms 0 and 1, [0, p) in form 2; a decode step in form 2
 * folds the new token itself (as W = 0 does in form 0).
 *
 * Two independent evaluations are provided: oracle_attend() evaluates the
 * definition directly (the quadratic form, Appendix eq. for O^Linear before
 * the rearrangement), oracle_decode_batch() runs the recurrence.  The tests
 * check that the two agree.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
  int32_t n_q_heads;   /* Hq */
  int32_t n_kv_heads;  /* Hkv, Hq % Hkv == 0 */
  int32_t head_dim;    /* d */
  int32_t feat_dim;    /* Df */
  int32_t window;      /* W >= 0 */
  int32_t linear;      /* 1: linear part on (GLIDE), 0: pure sliding window */
  int32_t form;        /* 0: shared denominator; 1, 2: the Appendix hybrid forms */
  int32_t phi;         /* 0: ReLU(x Wf); 1: ELU(x Wf) + 1; 2: softmax(x Wf) */
  int32_t wf_per_head; /* 0: one Wf [d][Df] per layer; 1: one per KV head, [Hkv][d][Df] */
  double  tau;         /* softmax scale */
} oracle_layer;

/* Planted-mistake switch, used only by the mutation tests that prove the
 * pins catch plausible errors.  0 = the correct oracle. */
#ifndef ORACLE_MUTANT
#define ORACLE_MUTANT 0
#endif

/* The feature map's Wf for KV head g: the layer's one matrix, or, per head,
 * the g-th (shared by the G query heads of the group and applied to the
 * group's keys, so that phi(q_h) and phi(k_j) meet in one feature space). */
static const double* wf_of(const oracle_layer* L, const double* Wf, int g) {
#if ORACLE_MUTANT == 13
  (void)g;
  return Wf;                                     /* mutant: every head takes head 0's Wf */
#else
  return L->wf_per_head ? Wf + (size_t)g * L->head_dim * L->feat_dim : Wf;
#endif
}

static int valid(const oracle_layer* L) {
  if (!L) return 0;
  if (L->n_q_heads <= 0 || L->n_kv_heads <= 0 || L->n_q_heads % L->n_kv_heads) return 0;
  if (L->head_dim <= 0 || L->feat_dim <= 0 || L->window < 0) return 0;
  if (L->window == 0 && !L->linear) return 0;   /* empty attention set */
  if (L->form < 0 || L->form > 2) return 0;
  if (L->form != 0 && !L->linear) return 0;     /* the forms differ only in the linear part */
  if (L->phi < 0 || L->phi > 2) return 0;
  return 1;
}

/* phi(x)_f = max(0, y_f) (kind 0), ELU(y_f) + 1 (kind 1), or e^{y_f} / sum_f' e^{y_f'}
 * (kind 2), y_f = sum_c x_c Wf[c][f]; Wf is d x Df, row-major. */
static void phi_row(int kind, int d, int Df, const double* Wf, const double* x, double* out) {
  if (kind == 2) {
    /* softmax over the projected features, with the row maximum subtracted
       (which leaves the value unchanged) */
    double ymax = -INFINITY;
    for (int f = 0; f < Df; ++f) {
      double acc = 0.0;
      for (int c = 0; c < d; ++c) acc += x[c] * Wf[(size_t)c * Df + f];
      out[f] = acc;
      if (acc > ymax) ymax = acc;
    }
    double sum = 0.0;
    for (int f = 0; f < Df; ++f) {
      out[f] = exp(out[f] - ymax);
      sum += out[f];
    }
#if ORACLE_MUTANT == 12
    sum = 1.0;                                    /* mutant: exponentials not normalised */
#endif
    for (int f = 0; f < Df; ++f) out[f] /= sum;
    return;
  }
  for (int f = 0; f < Df; ++f) {
    double acc = 0.0;
    for (int c = 0; c < d; ++c) {
#if ORACLE_MUTANT == 4
      acc += x[c] * Wf[(size_t)f * d + c];        /* mutant: Wf transposed */
#else
      acc += x[c] * Wf[(size_t)c * Df + f];
#endif
    }
#if ORACLE_MUTANT == 11
    if (kind == 1) { out[f] = acc > 0.0 ? acc : exp(acc) - 1.0; continue; }   /* mutant: ELU without the +1 */
#endif
    if (kind == 1) out[f] = acc > 0.0 ? acc + 1.0 : exp(acc);
    else out[f] = acc > 0.0 ? acc : 0.0;
  }
}

/* phi of dense rows with one Wf [d][Df] (per head: the caller passes that head's matrix). */
void oracle_phi(const oracle_layer* L, const double* Wf, int64_t rows, const double* x, double* out) {
  const int d = L->head_dim, Df = L->feat_dim;
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; ++r) phi_row(L->phi, d, Df, Wf, x + r * d, out + r * Df);
}

static double dot(int n, const double* a, const double* b) {
  double s = 0.0;
  for (int i = 0; i < n; ++i) s += a[i] * b[i];
  return s;
}

/*
 * Merge of the two parts for one query head (form 0: one shared denominator;
 * forms 1, 2: two separately normalised outputs added).
 *   sm_num[d], sm_den, m : softmax part as sum e^{s_j - m} v_j, sum e^{s_j - m}
 *                          (has_sm == 0 when the softmax set is empty)
 *   A[d], a              : linear part, unscaled
 */
static void merge(int form, int d, int has_sm, const double* sm_num, double sm_den, double m,
                  const double* A, double a, double* out) {
  if (form != 0) {
#if ORACLE_MUTANT == 10
    /* mutant: the linear term divided by both denominators */
    for (int c = 0; c < d; ++c)
      out[c] = (has_sm ? sm_num[c] / sm_den : 0.0) + (a > 0.0 ? A[c] / (a + (has_sm ? sm_den : 0.0)) : 0.0);
#else
    for (int c = 0; c < d; ++c)
      out[c] = (has_sm ? sm_num[c] / sm_den : 0.0) + (a > 0.0 ? A[c] / a : 0.0);
#endif
    return;
  }
  if (!has_sm) {
    for (int c = 0; c < d; ++c) out[c] = a > 0.0 ? A[c] / a : 0.0;
    return;
  }
#if ORACLE_MUTANT == 3
  /* mutant: two separately normalised outputs added ("+" form) */
  for (int c = 0; c < d; ++c) out[c] = sm_num[c] / sm_den + (a > 0.0 ? A[c] / a : 0.0);
  return;
#elif ORACLE_MUTANT == 6
  /* mutant: stabiliser applied to the softmax terms only */
  for (int c = 0; c < d; ++c) out[c] = (sm_num[c] + A[c]) / (sm_den + a);
  (void)m;
  return;
#else
  if (!(a > 0.0)) {   /* empty linear mass: A = 0 and a = 0 add nothing */
    for (int c = 0; c < d; ++c) out[c] = sm_num[c] / sm_den;
    return;
  }
  double cst = m;
  if (log(a) > cst) cst = log(a);
  const double ws = exp(m - cst), wl = exp(-cst);
  const double den = sm_den * ws + a * wl;
  for (int c = 0; c < d; ++c) out[c] = (sm_num[c] * ws + A[c] * wl) / den;
#endif
}

/*
 * Definition form for ONE sequence of n tokens (q [n][Hq][d], k,v [n][Hkv][d]).
 * Computes O_t for every position listed in pos[n_out], all Hq heads:
 * out [n_out][Hq][d].  phi(k_j) is evaluated once per key and reused.
 * Returns 0, or -1 on invalid arguments.
 */
/* Cumulative log-gates of the gated linear state: Gc[t][g] = sum_{i <= t} lg[i][g]
 * (NULL when ungated).  A linear-set token j read at time t weighs
 * e^{Gc[t] - Gc[j]}: it has decayed by the gates of the tokens after it. */
static double* cum_gates(const double* lg, int64_t n, int Hkv) {
  if (!lg || n <= 0) return NULL;
  double* Gc = (double*)malloc(sizeof(double) * (size_t)n * Hkv);
  if (!Gc) return NULL;
  for (int g = 0; g < Hkv; ++g) {
    double acc = 0.0;
    for (int64_t t = 0; t < n; ++t) {
      acc += lg[(size_t)t * Hkv + g];
      Gc[(size_t)t * Hkv + g] = acc;
    }
  }
  return Gc;
}
static double decay(const double* Gc, int Hkv, int g, int64_t t, int64_t j) {
  if (!Gc) return 1.0;
#if ORACLE_MUTANT == 14
  return exp(Gc[(size_t)t * Hkv + g] - (j > 0 ? Gc[(size_t)(j - 1) * Hkv + g] : 0.0));  /* mutant: j's own gate too */
#else
  return exp(Gc[(size_t)t * Hkv + g] - Gc[(size_t)j * Hkv + g]);
#endif
}

static int attend_impl(const oracle_layer* L, const double* Wf, int64_t n,
                       const double* q, const double* k, const double* v, const double* lg,
                       int64_t n_out, const int64_t* pos, double* out) {
  if (!valid(L) || n < 0 || n_out < 0) return -1;
  for (int64_t i = 0; i < n_out; ++i)
    if (pos[i] < 0 || pos[i] >= n) return -1;
  const int Hq = L->n_q_heads, Hkv = L->n_kv_heads, d = L->head_dim, Df = L->feat_dim;
  const int G = Hq / Hkv, W = L->window;
  int64_t tmax = -1;
  for (int64_t i = 0; i < n_out; ++i) if (pos[i] > tmax) tmax = pos[i];
  /* phi of every key that can be in a linear set */
  double* phik = NULL;
  if (L->linear && tmax >= 0) {
    phik = (double*)malloc(sizeof(double) * (size_t)(tmax + 1) * Hkv * Df);
    if (!phik) return -1;
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < (tmax + 1) * Hkv; ++r)
      phi_row(L->phi, d, Df, wf_of(L, Wf, (int)(r % Hkv)), k + r * d, phik + r * Df);
  }
  double* Gc = cum_gates(lg, tmax + 1, Hkv);
  if (lg && tmax >= 0 && !Gc) { free(phik); return -1; }
  int err = 0;
#pragma omp parallel
  {
    double* phq = (double*)malloc(sizeof(double) * Df);
    double* A = (double*)malloc(sizeof(double) * d);
    double* num = (double*)malloc(sizeof(double) * d);
    if (!phq || !A || !num) {
#pragma omp atomic write
      err = 1;
    } else {
#pragma omp for collapse(2) schedule(dynamic, 4)
      for (int64_t i = 0; i < n_out; ++i) {
        for (int h = 0; h < Hq; ++h) {
          const int64_t t = pos[i];
          const int g = h / G;
          const double* qt = q + ((size_t)t * Hq + h) * d;
#if ORACLE_MUTANT == 1
          int64_t beta = t - W;                    /* mutant: window one token too long */
#else
          int64_t beta = t + 1 - W;
#endif
          if (beta < 0) beta = 0;
          /* linear part over [0, lend): [0, beta), or [0, t] in form 2 */
#if ORACLE_MUTANT == 8
          const int64_t lend = L->form == 2 ? t : beta;        /* mutant: form 2 misses the current token */
#else
          const int64_t lend = L->form == 2 ? t + 1 : beta;
#endif
          double a = 0.0;
          for (int c = 0; c < d; ++c) A[c] = 0.0;
#if ORACLE_MUTANT != 2
          if (L->linear && lend > 0) {
            phi_row(L->phi, d, Df, wf_of(L, Wf, g), qt, phq);
            for (int64_t j = 0; j < lend; ++j) {
              const double aj = dot(Df, phq, phik + ((size_t)j * Hkv + g) * Df) * decay(Gc, Hkv, g, t, j);
              const double* vj = v + ((size_t)j * Hkv + g) * d;
              for (int c = 0; c < d; ++c) A[c] += aj * vj[c];
              a += aj;
            }
          }
#endif
          /* softmax part over [beta, t] */
          const int has_sm = (t >= beta);
          double m = -INFINITY, den = 0.0;
          for (int c = 0; c < d; ++c) num[c] = 0.0;
          if (has_sm) {
            for (int64_t j = beta; j <= t; ++j) {
#if ORACLE_MUTANT == 7
              const double s = dot(d, qt, k + ((size_t)j * Hkv + g) * d);   /* mutant: no tau */
#else
              const double s = L->tau * dot(d, qt, k + ((size_t)j * Hkv + g) * d);
#endif
              if (s > m) m = s;
            }
            for (int64_t j = beta; j <= t; ++j) {
              const double s = L->tau * dot(d, qt, k + ((size_t)j * Hkv + g) * d);
#if ORACLE_MUTANT == 7
              const double e = exp(dot(d, qt, k + ((size_t)j * Hkv + g) * d) - m);
#else
              const double e = exp(s - m);
#endif
              (void)s;
              const double* vj = v + ((size_t)j * Hkv + g) * d;
              for (int c = 0; c < d; ++c) num[c] += e * vj[c];
              den += e;
            }
          }
          merge(L->form, d, has_sm, num, den, m, A, a, out + ((size_t)i * Hq + h) * d);
        }
      }
    }
    free(phq); free(A); free(num);
  }
  free(phik);
  free(Gc);
  return err ? -1 : 0;
}

int oracle_attend(const oracle_layer* L, const double* Wf, int64_t n,
                  const double* q, const double* k, const double* v,
                  int64_t n_out, const int64_t* pos, double* out) {
  return attend_impl(L, Wf, n, q, k, v, NULL, n_out, pos, out);
}

/* The gated linear state (GLA-style decay, one log-gate lg[t][g] <= 0 per
 * token and KV head): the definition form with every linear-set token
 * weighted by the decay since it arrived. */
int oracle_attend_gated(const oracle_layer* L, const double* Wf, int64_t n,
                        const double* q, const double* k, const double* v, const double* lg,
                        int64_t n_out, const int64_t* pos, double* out) {
  if (!lg) return -1;
  return attend_impl(L, Wf, n, q, k, v, lg, n_out, pos, out);
}

/*
 * Recurrent state after consuming p tokens of one sequence, by direct sums:
 * S [Hkv][Df][d] = sum_{j < p-W} phi(k_j)^T v_j,  z [Hkv][Df] = sum phi(k_j)
 * (j < p in form 2).  Both zero when p <= W (forms 0, 1) or when the linear
 * part is off.
 */
static int state_impl(const oracle_layer* L, const double* Wf, int64_t p,
                      const double* k, const double* v, const double* lg, double* S, double* z) {
  if (!valid(L) || p < 0) return -1;
  const int Hkv = L->n_kv_heads, d = L->head_dim, Df = L->feat_dim, W = L->window;
  memset(S, 0, sizeof(double) * (size_t)Hkv * Df * d);
  memset(z, 0, sizeof(double) * (size_t)Hkv * Df);
  const int64_t nfold = !L->linear ? 0 : L->form == 2 ? p : (p - W > 0 ? p - W : 0);
  double* Gc = cum_gates(lg, p, Hkv);
  if (lg && p > 0 && !Gc) return -1;
  int err = 0;
#pragma omp parallel for schedule(static)
  for (int g = 0; g < Hkv; ++g) {
    double* pk = (double*)malloc(sizeof(double) * Df);
    if (!pk) { err = 1; continue; }
    for (int64_t j = 0; j < nfold; ++j) {
      phi_row(L->phi, d, Df, wf_of(L, Wf, g), k + ((size_t)j * Hkv + g) * d, pk);
      const double w = decay(Gc, Hkv, g, p - 1, j);   /* decayed through token p - 1 */
      const double* vj = v + ((size_t)j * Hkv + g) * d;
      for (int f = 0; f < Df; ++f) {
        double* Sr = S + ((size_t)g * Df + f) * d;
        for (int c = 0; c < d; ++c) Sr[c] += w * pk[f] * vj[c];
        z[(size_t)g * Df + f] += w * pk[f];
      }
    }
    free(pk);
  }
  free(Gc);
  return err ? -1 : 0;
}

int oracle_state(const oracle_layer* L, const double* Wf, int64_t p,
                 const double* k, const double* v, double* S, double* z) {
  return state_impl(L, Wf, p, k, v, NULL, S, z);
}

/* The gated state after p tokens: the same sums, each token decayed by the
 * gates of the tokens after it up to token p - 1. */
int oracle_state_gated(const oracle_layer* L, const double* Wf, int64_t p,
                       const double* k, const double* v, const double* lg, double* S, double* z) {
  if (!lg) return -1;
  return state_impl(L, Wf, p, k, v, lg, S, z);
}

/*
 * Recurrent form: one decode step for a batch of B sequences of one layer.
 *   S   [B][Hkv][Df][d], z [B][Hkv][Df]            (in/out)
 *   wk, wv [B][Hkv][W][d]: the window, oldest token first; sequence b holds
 *       min(W, pos[b]) tokens                       (in/out)
 *   pos [B]: tokens consumed so far                 (in/out, += 1)
 *   q [B][Hq][d], k, v [B][Hkv][d]: the new token;  out [B][Hq][d]
 * Order per (sequence, KV head): fold the token leaving the window into S, z
 * (the oldest window token when the window is full; the new token itself
 * when W = 0, and always in form 2), append the new token, then read out
 * every query head of the group from the updated state and window.
 */
int oracle_decode_batch(const oracle_layer* L, const double* Wf, int32_t B,
                        double* S, double* z, double* wk, double* wv, int64_t* pos,
                        const double* q, const double* k, const double* v, double* out) {
  if (!valid(L) || B < 0) return -1;
  const int Hq = L->n_q_heads, Hkv = L->n_kv_heads, d = L->head_dim, Df = L->feat_dim;
  const int G = Hq / Hkv, W = L->window;
  for (int b = 0; b < B; ++b) if (pos[b] < 0) return -1;
  int err = 0;
#pragma omp parallel for collapse(2) schedule(dynamic, 1)
  for (int b = 0; b < B; ++b) {
    for (int g = 0; g < Hkv; ++g) {
      const int64_t p = pos[b];
      double* Sg = S + ((size_t)b * Hkv + g) * Df * d;
      double* zg = z + ((size_t)b * Hkv + g) * Df;
      double* Wk = wk + ((size_t)b * Hkv + g) * (size_t)W * d;
      double* Wv = wv + ((size_t)b * Hkv + g) * (size_t)W * d;
      const double* kn = k + ((size_t)b * Hkv + g) * d;
      const double* vn = v + ((size_t)b * Hkv + g) * d;
      double* pk = (double*)malloc(sizeof(double) * Df);
      double* pq = (double*)malloc(sizeof(double) * Df);
      double* A = (double*)malloc(sizeof(double) * d);
      double* num = (double*)malloc(sizeof(double) * d);
      if (!pk || !pq || !A || !num) {
#pragma omp atomic write
        err = 1;
        free(pk); free(pq); free(A); free(num);
        continue;
      }
      /* 1. fold the token that leaves the softmax window */
      const double* fk = NULL;
      const double* fv = NULL;
      int64_t nwin = p < W ? p : W;            /* window tokens before this step */
#if ORACLE_MUTANT == 5
      if (L->linear && (W == 0 || nwin == W)) { fk = kn; fv = vn; }   /* mutant: folds the new token */
#else
      if (L->linear) {
#if ORACLE_MUTANT == 9
        if (W == 0) { fk = kn; fv = vn; }                               /* mutant: form 2 folds like form 1 */
#else
        if (W == 0 || L->form == 2) { fk = kn; fv = vn; }
#endif
        else if (nwin == W) { fk = Wk; fv = Wv; }                      /* oldest = token p - W */
      }
#endif
      if (fk) {
        phi_row(L->phi, d, Df, wf_of(L, Wf, g), fk, pk);
        for (int f = 0; f < Df; ++f) {
          for (int c = 0; c < d; ++c) Sg[(size_t)f * d + c] += pk[f] * fv[c];
          zg[f] += pk[f];
        }
      }
      /* 2. append the new token (drop the oldest when full) */
      if (W > 0) {
        if (nwin == W) {
          memmove(Wk, Wk + d, sizeof(double) * (size_t)(W - 1) * d);
          memmove(Wv, Wv + d, sizeof(double) * (size_t)(W - 1) * d);
          nwin = W - 1;
        }
        memcpy(Wk + (size_t)nwin * d, kn, sizeof(double) * d);
        memcpy(Wv + (size_t)nwin * d, vn, sizeof(double) * d);
        nwin += 1;
      }
      /* 3. read out every query head of the group */
      for (int hh = 0; hh < G; ++hh) {
        const int h = g * G + hh;
        const double* qt = q + ((size_t)b * Hq + h) * d;
        double a = 0.0;
        for (int c = 0; c < d; ++c) A[c] = 0.0;
        if (L->linear) {
          phi_row(L->phi, d, Df, wf_of(L, Wf, g), qt, pq);
          for (int f = 0; f < Df; ++f) {
            for (int c = 0; c < d; ++c) A[c] += pq[f] * Sg[(size_t)f * d + c];
            a += pq[f] * zg[f];
          }
        }
        double m = -INFINITY, den = 0.0;
        for (int c = 0; c < d; ++c) num[c] = 0.0;
        for (int64_t j = 0; j < nwin; ++j) {
          const double s = L->tau * dot(d, qt, Wk + (size_t)j * d);
          if (s > m) m = s;
        }
        for (int64_t j = 0; j < nwin; ++j) {
          const double e = exp(L->tau * dot(d, qt, Wk + (size_t)j * d) - m);
          for (int c = 0; c < d; ++c) num[c] += e * Wv[(size_t)j * d + c];
          den += e;
        }
        merge(L->form, d, nwin > 0, num, den, m, A, a, out + ((size_t)b * Hq + h) * d);
      }
      free(pk); free(pq); free(A); free(num);
    }
  }
  for (int b = 0; b < B; ++b) pos[b] += 1;
  return err ? -1 : 0;
}
