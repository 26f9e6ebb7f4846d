/*
 * glide.h -- C ABI of the GLIDE hybrid-attention step on AMD Instinct MI355X
 * (gfx950).
 *
 * One layer of GLIDE attention (GLIDE, Sec. III-B: the first displayed
 * equation of the section and the two that expand it, with the split point
 * read as the effective softmax window W = w - delta; the merge weighted by
 * the two normalising denominators described in Sec. II-A and III-B):
 *
 *   for query head h (KV head g = h / G, G = Hq / Hkv) at 0-indexed position t
 *     beta      = max(0, t + 1 - W)
 *     phi(x)    = max(0, x . Wf)                (Wf: d x Df, one per layer)
 *     A, a      = sum_{j < beta} (phi(q_t).phi(k_j)) v_j ,  sum_{j < beta} phi(q_t).phi(k_j)
 *               = phi(q_t) . S ,  phi(q_t) . z  with  S = sum phi(k_j)^T v_j,
 *                 z = sum phi(k_j)              (Sec. II-B recurrence)
 *     O_t       = (sum_{j=beta..t} e^{tau q_t.k_j} v_j + A) / (sum_{j=beta..t} e^{tau q_t.k_j} + a)
 *
 * W = 0 gives pure linear attention (the current token is folded before the
 * read-out); W >= context gives causal softmax attention (the two boundary
 * conditions stated in Sec. III-B).  0/0 (W = 0 and phi(q).z = 0) yields 0.
 *
 * Threading, memory and errors
 *   - Every device buffer is allocated and owned by the caller.  The library
 *     never allocates, frees or synchronises; all work is enqueued on the
 *     caller's stream (a hipStream_t passed as void*, NULL = default stream).
 *   - Host arrays (glide_config.windows, cu_seqlens_host) are read during the
 *     call only and never retained.  The library has no mutable global state.
 *   - Every argument is validated on the host before the first HIP call; on
 *     any error nothing is enqueued and the state is untouched.
 *   - A failed kernel launch returns GLIDE_ERR_HIP and leaves the state
 *     undefined (re-initialise it).  Asynchronous device faults surface at the
 *     caller's next synchronisation.  No C++ exception crosses this ABI.
 *   - Calls that mutate one state blob must not overlap; calls on different
 *     state blobs may run concurrently on different streams.
 */
#ifndef GLIDE_H_
#define GLIDE_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  GLIDE_OK = 0,
  GLIDE_ERR_NULL = -1,        /* a required pointer is NULL */
  GLIDE_ERR_INVALID = -2,     /* inconsistent or out-of-range argument */
  GLIDE_ERR_UNSUPPORTED = -3, /* valid per the definition, not built here (d, Df, G, dtype) */
  GLIDE_ERR_ALIGN = -4,       /* a device pointer is not 16-byte aligned (state: 256) */
  GLIDE_ERR_SIZE = -5,        /* state or workspace smaller than required */
  GLIDE_ERR_HIP = -6,         /* a HIP launch failed */
  GLIDE_ERR_SCRATCH = -7      /* glide_decode_step_noalloc: the call needs more than the library's
                                 fixed decode scratch (GLIDE_DECODE_SCRATCH_BYTES) */
} glide_status;

/* Element type of q, k, v, out, the window ring and phi_w.  S and z are fp32. */
enum { GLIDE_F32 = 0, GLIDE_BF16 = 1 };

/* Feature map on y = x . Wf (Wf is non-learnable, one d x Df matrix per
 * layer shared by every head, applied to queries and keys alike), from the
 * Appendix's feature-map list:
 *   GLIDE_PHI_RELU     phi = max(0, y)
 *   GLIDE_PHI_ELU1     phi = ELU(y) + 1 = y + 1 for y > 0, e^y otherwise (never 0)
 *   GLIDE_PHI_SOFTMAX  phi = softmax(y) over the Df features, e^{y_f} / sum e^{y_f'}
 *                      (the default kernel choice of Sec. III-B; positive, sums to 1) */
enum { GLIDE_PHI_RELU = 0, GLIDE_PHI_ELU1 = 1, GLIDE_PHI_SOFTMAX = 2 };

/* flags: GLIDE_NO_LINEAR turns the linear part off (plain sliding-window
 * softmax attention, the "Hybrid" preset with nothing kept beyond the
 * window); W = 0 is then rejected because the attention set is empty.
 *
 * GLIDE_HYBRID_SUM selects the Appendix's first hybrid-attention equation
 * (retention-based sliding window) instead of the shared denominator: the
 * window's softmax output and the linear part's own normalised output
 * phi(q).S / phi(q).z are added,
 *   O_t = sum_{j=beta..t} e^{s_j} v_j / sum_{j=beta..t} e^{s_j}  +  A / a,
 * each term 0 when its set is empty (A / a := 0 when a = 0).  Adding
 * GLIDE_HYBRID_STATE_ALL selects the Appendix's second equation: the same
 * sum with the state over every token up to the current one, window tokens
 * included (linear set [0, t]; S, z then hold tokens [0, p) after p tokens).
 * The paper states that GLIDE adapts both forms through its merge operator.
 * GLIDE_HYBRID_STATE_ALL requires GLIDE_HYBRID_SUM; neither combines with
 * GLIDE_NO_LINEAR.
 *
 * GLIDE_PER_HEAD_PHI gives every KV head its own feature-map matrix: phi_w is
 * then [n_layers][Hkv][d][Df], and head g's matrix maps the queries of its
 * group and its own keys (so that phi(q_h) . phi(k_j) pairs one feature
 * space; S and z are per KV head already).  It combines with every other
 * flag.  glide_feature_map takes one [d][Df] matrix either way.
 *
 * GLIDE_GATED gives the linear state a data-dependent decay, the GLA-style
 * gating Sec. III-B names among the linear forms GLIDE supports (the paper
 * does not fix the gate; here one scalar log-gate g_j <= 0 per token and KV
 * head, passed in by the caller): a linear-set token j read at position t
 * weighs e^{G_t - G_j}, G_t = g_0 + ... + g_t, i.e. it has decayed by the
 * gates of every token after it (window tokens included):
 *   A = sum_{j < beta} e^{G_t - G_j} (phi(q_t).phi(k_j)) v_j,  a likewise,
 * and after p tokens S = sum_{j < p - W} e^{G_{p-1} - G_j} phi(k_j)^T v_j,
 * z likewise (decayed through token p - 1).  The softmax window is not
 * gated.  Prefill and decode then take log_gates (fp32, every value <= 0 and
 * finite; the library does not check device data).  Only with the shared
 * denominator (no hybrid flag) and the linear part on. */
enum { GLIDE_NO_LINEAR = 1, GLIDE_HYBRID_SUM = 2, GLIDE_HYBRID_STATE_ALL = 4, GLIDE_PER_HEAD_PHI = 8,
       GLIDE_GATED = 16 };

typedef struct {
  int32_t n_layers;    /* layers held by one state blob (>= 1) */
  int32_t batch;       /* sequences B (>= 1) */
  int32_t n_q_heads;   /* Hq */
  int32_t n_kv_heads;  /* Hkv; Hq % Hkv == 0, G = Hq / Hkv in [1, 16] */
  int32_t head_dim;    /* d: 64 or 128 */
  int32_t feat_dim;    /* Df: 64 or 128 */
  int32_t dtype;       /* GLIDE_F32 or GLIDE_BF16 */
  int32_t phi;         /* GLIDE_PHI_RELU, GLIDE_PHI_ELU1 or GLIDE_PHI_SOFTMAX */
  int32_t flags;       /* 0, GLIDE_NO_LINEAR, GLIDE_HYBRID_SUM, GLIDE_HYBRID_SUM | GLIDE_HYBRID_STATE_ALL
                          or GLIDE_GATED, each optionally | GLIDE_PER_HEAD_PHI */
  float sm_scale;      /* tau, the softmax scale (1/sqrt(d) in the Appendix's attention) */
  const int32_t* windows; /* HOST array [n_layers]: W_l = w - delta_l, 0 <= W_l <= 2^20 */
} glide_config;

/* Position of the sections of one layer inside the state blob (bytes from the
 * blob's start).  Layout per layer l, every section 256-byte aligned:
 *   pos   int64 [B][Hkv]          p: tokens consumed by sequence b (equal over Hkv)
 *   nf    int64 [B][Hkv]          tokens folded into S and z (see below)
 *   cnt   int32 [B][Hkv]          decode bookkeeping: pieces of a split unit
 *                                 done in the current step; 0 between calls
 *   S     fp32  [B][Hkv][Df][d]   sum of phi(k_j)^T v_j over tokens j < nf
 *   z     fp32  [B][Hkv][Df]      sum of phi(k_j) over the same tokens
 *   kring dtype [B][Hkv][R*d]     keys, token j in slot s = j mod R
 *   vring dtype [B][Hkv][R*d]     values, token j in slot s = j mod R
 *   gate  fp64  [B][Hkv][2]       GLIDE_GATED only: G_{p-1} (the cumulative
 *                                 log-gate through the last token consumed)
 *                                 and G_f, the position S and z are decayed to
 *                                 (S = sum_{j < nf} e^{G_f - G_j} ...)
 *   gring fp64  [B][Hkv][R]       GLIDE_GATED only: G_j of ring token j, slot
 *                                 j mod R (empty sections have size 0)
 * Deferred folding: the linear part of the next read-out covers tokens
 * [0, beta), beta = max(0, p - W).  Decode steps fold the tokens leaving the
 * window in batches of up to 8 (staggered over units), so nf lies in
 * [beta - 8, beta] (W = 0: nf = beta); tokens [nf, beta) are "pending": kept
 * in the ring and added to the read-out from there.  glide_prefill and
 * glide_state_flush leave nf = beta.  With GLIDE_HYBRID_STATE_ALL, beta = p
 * and every step folds its own token (nf = p).  R = ring_slots =
 * round_up(W + 8, 32) for W > 0, 0 for W = 0.  After p tokens the ring holds
 * tokens [min(nf, p - W), p - 1] (W > 0); other slots are stale.
 * Both rings are stored in 32-slot blocks of 32*d elements, in the fragment
 * order of the decode kernel's matrix-core loads; with o = s % 32, block
 * s / 32, element c of the slot is at (within the block)
 *   kring: [(o/4)%2][c/32][(c/8)%4][4*(o/8) + o%4][c%8]
 *   vring: [c/16][o/8][c%16][o%8]                                          */
typedef struct {
  int64_t pos_offset, nf_offset, cnt_offset, s_offset, z_offset, kring_offset, vring_offset;
  int64_t gate_offset, gring_offset;
  int64_t layer_offset, layer_bytes;
  int32_t window;      /* W_l */
  int32_t ring_slots;  /* R_l */
} glide_layer_layout;

/* Bytes of the state blob for cfg (sum of all layers), 0 if cfg is invalid. */
size_t glide_state_bytes(const glide_config* cfg);

/* Fills *out with the layout of layer `layer` (0 <= layer < cfg->n_layers). */
glide_status glide_state_layout(const glide_config* cfg, int32_t layer, glide_layer_layout* out);

/* Workspace bytes needed by glide_prefill for calls of max_total_tokens
 * packed tokens (any chunk size) and by glide_decode_step (any layer range);
 * at least 256.  Prefill takes one slot per layer of a launch (history rows
 * and per-segment state records) and batches as many layers per launch as
 * the given workspace holds, up to 64; this size holds as many as fit in
 * 1 GiB (at least one).  Decode uses the workspace only when a launch has
 * fewer (sequence, KV head) units than the device holds resident decode
 * workgroups in one round (two per compute unit: 512 on MI355X): it then
 * splits long windows (more than 256 tokens) over several workgroups, whose
 * partial results it holds.  The size bounds that for every call on any device (at most 1024
 * records; a call over any subset of the layers).  0 if cfg is invalid. */
size_t glide_workspace_bytes(const glide_config* cfg, int64_t max_total_tokens);

/* Zeroes the whole state: S = 0, z = 0 (S_0, Z_0 of the Sec. II-B
 * recurrence), pos = nf = 0, ring contents 0.  state: device, 256-byte
 * aligned, state_bytes >= glide_state_bytes(cfg). */
glide_status glide_state_init(const glide_config* cfg, void* state, size_t state_bytes, void* stream);

/* Prefill (KV-cache population stage, Appendix "KV Cache"): appends
 * T_b = cu_seqlens[b+1] - cu_seqlens[b] >= 0 tokens to every sequence b,
 * starting at that sequence's current position (a continuing prefill is
 * legal), for layers [layer0, layer0 + n_layers), and writes one output per
 * appended token.  Within a layer the work is chunked: chunk C query tokens
 * share one softmax band pass and one state read-out (chunk = 0 -> 64; any
 * C in [32, 256] that is a multiple of 32 gives the same result up to
 * rounding).  Pending tokens are folded first (as glide_state_flush); on
 * return nf = max(0, p - W).
 *   phi_w  device [n_layers][d][Df]        (layer layer0 first; [n_layers][Hkv][d][Df]
 *          with GLIDE_PER_HEAD_PHI)
 *   q      device [n_layers][T][Hq][d]     T = total_tokens, packed by sequence
 *   k, v   device [n_layers][T][Hkv][d]
 *   log_gates  device fp32 [n_layers][T][Hkv] with GLIDE_GATED (the log-gate
 *          of every new token), else NULL
 *   cu_seqlens_host  HOST [B+1], cu[0] = 0, non-decreasing, cu[B] = T; one
 *          sequence's new q rows must span less than 2 GiB (T_b * Hq * d *
 *          element bytes < 2^31, else GLIDE_ERR_UNSUPPORTED)
 *   out    device [n_layers][T][Hq][d]
 *   workspace device, >= glide_workspace_bytes(cfg, T)
 * Element types follow cfg->dtype; device pointers 16-byte aligned. */
glide_status glide_prefill(const glide_config* cfg, void* state, size_t state_bytes,
                           int32_t layer0, int32_t n_layers, const void* phi_w,
                           const void* q, const void* k, const void* v, const float* log_gates,
                           const int32_t* cu_seqlens_host, int64_t total_tokens, int32_t chunk,
                           void* out, void* workspace, size_t workspace_bytes, void* stream);

/* Decode (Appendix "KV Cache", decode stage): appends exactly one token to
 * every sequence for layers [layer0, layer0 + n_layers).  Per (layer,
 * sequence, KV head): the token leaving the window (token p - W when p >= W;
 * the new token itself when W = 0) joins the linear part, the new key/value
 * is written into its ring slot, O is read out for the G query heads of the
 * group from the window and from S + the pending tokens, pos += 1; on the
 * unit's fold step (one in 8; every step when W = 0) the pending tokens are
 * folded into S and z.  Sequences may sit at different positions (pos lives
 * in the state).  One kernel is enqueued per 64 layers; each plans its own
 * window split over the device (see glide_workspace_bytes), so a call over
 * one layer spreads that layer's windows over many workgroups; the
 * workgroup that finishes a unit's last piece merges the pieces' partial
 * results.  Calls over different layer subsets agree up to rounding.
 *   phi_w  device [n_layers][d][Df]  ([n_layers][Hkv][d][Df] with GLIDE_PER_HEAD_PHI)
 *   q      device [n_layers][B][Hq][d];  k, v device [n_layers][B][Hkv][d]
 *   log_gates  device fp32 [n_layers][B][Hkv] with GLIDE_GATED (the new
 *          token's log-gate), else NULL
 *   out    device [n_layers][B][Hq][d]
 *   workspace  device, 256-byte aligned, >= glide_workspace_bytes(cfg, 0);
 *              may be NULL when that is 256 (nothing is split) */
glide_status glide_decode_step(const glide_config* cfg, void* state, size_t state_bytes,
                               int32_t layer0, int32_t n_layers, const void* phi_w,
                               const void* q, const void* k, const void* v, const float* log_gates,
                               void* out, void* workspace, size_t workspace_bytes, void* stream);

/* Size of the fixed decode scratch of glide_decode_step_noalloc, per GPU. */
#define GLIDE_DECODE_SCRATCH_BYTES (16u << 20)

/* glide_decode_step without a workspace, for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc.  The same kernels and the same result as
 * glide_decode_step; the partial records of split windows go to a fixed
 * array of GLIDE_DECODE_SCRATCH_BYTES that the library holds on every GPU it
 * runs on, until the process ends (its address is looked up once per device,
 * on the first call with that device current).  Nothing is allocated or
 * freed.  A config whose decode workspace (glide_workspace_bytes(cfg, 0))
 * exceeds the scratch is rejected with GLIDE_ERR_SCRATCH before any HIP call
 * (G <= 15 at d = 128 always fits).  Every call on one GPU shares that GPU's
 * scratch: calls that overlap in time on one GPU (other streams, other
 * threads) race and may return wrong results; serialise them.  The records
 * are written before they are read within each call, so no call needs the
 * scratch cleared.  Arguments, layouts and errors otherwise as for
 * glide_decode_step. */
glide_status glide_decode_step_noalloc(const glide_config* cfg, void* state, size_t state_bytes,
                                       int32_t layer0, int32_t n_layers, const void* phi_w,
                                       const void* q, const void* k, const void* v,
                                       const float* log_gates, void* out, void* stream);

/* Folds every pending token of layers [layer0, layer0 + n_layers) into S and
 * z (nf := max(0, p - W)), so that S and z hold exactly the Sec. II-B sums
 * over the linear part of the next token.  Outputs of later steps are
 * unchanged up to rounding.  phi_w device [n_layers][d][Df], layer layer0 first
 * ([n_layers][Hkv][d][Df] with GLIDE_PER_HEAD_PHI).  Nothing to do without the
 * linear part.  With GLIDE_GATED, S and z are decayed to the last token
 * consumed (G_f := G_{p-1}). */
glide_status glide_state_flush(const glide_config* cfg, void* state, size_t state_bytes,
                               int32_t layer0, int32_t n_layers, const void* phi_w, void* stream);

/* The feature map alone (kernel (d)): out[r][f] = phi(sum_c x[r][c] Wf[c][f])
 * (cfg->phi; the softmax map normalises each row over its Df features) for
 * r < rows, accumulated in fp32.  x device [rows][d], phi_w device [d][Df] (one
 * matrix, also with GLIDE_PER_HEAD_PHI: the caller passes the head's), both
 * cfg->dtype; out device [rows][Df] in cfg->dtype; x and out may be NULL when
 * rows == 0. */
glide_status glide_feature_map(const glide_config* cfg, const void* phi_w, const void* x,
                               int64_t rows, void* out, void* stream);

/* Static description of a status code. */
const char* glide_status_string(glide_status s);

#ifdef __cplusplus
}
#endif

#endif /* GLIDE_H_ */
