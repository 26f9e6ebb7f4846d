// C ABI of the GLIDE hybrid-attention library: argument validation (always
// on the host, before the first HIP call), state layout, and kernel dispatch.
#include <math.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "glide_internal.h"

using namespace glide;

namespace {

constexpr int32_t kMaxWindow = 1 << 20;

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

glide_status check_cfg(const glide_config* c) {
  if (!c || !c->windows) return GLIDE_ERR_NULL;
  if (c->n_layers < 1 || c->n_layers > (1 << 16)) return GLIDE_ERR_INVALID;
  if (c->batch < 1 || c->batch > (1 << 20)) return GLIDE_ERR_INVALID;
  if (c->n_q_heads < 1 || c->n_kv_heads < 1 || c->n_q_heads > 4096) return GLIDE_ERR_INVALID;
  if (c->n_q_heads % c->n_kv_heads) return GLIDE_ERR_INVALID;
  if (c->head_dim < 1 || c->feat_dim < 1) return GLIDE_ERR_INVALID;
  if (c->dtype != GLIDE_F32 && c->dtype != GLIDE_BF16) return GLIDE_ERR_INVALID;
  if (c->phi != GLIDE_PHI_RELU && c->phi != GLIDE_PHI_ELU1 && c->phi != GLIDE_PHI_SOFTMAX) return GLIDE_ERR_INVALID;
  if (c->flags &
      ~int32_t(GLIDE_NO_LINEAR | GLIDE_HYBRID_SUM | GLIDE_HYBRID_STATE_ALL | GLIDE_PER_HEAD_PHI | GLIDE_GATED))
    return GLIDE_ERR_INVALID;
  // a gate decays the linear part: not without one
  if ((c->flags & GLIDE_GATED) && (c->flags & GLIDE_NO_LINEAR)) return GLIDE_ERR_INVALID;
  // the hybrid forms change the linear part: not without one; the state over
  // every token comes only with the separately normalised sum
  if ((c->flags & GLIDE_NO_LINEAR) && (c->flags & (GLIDE_HYBRID_SUM | GLIDE_HYBRID_STATE_ALL)))
    return GLIDE_ERR_INVALID;
  if ((c->flags & GLIDE_HYBRID_STATE_ALL) && !(c->flags & GLIDE_HYBRID_SUM)) return GLIDE_ERR_INVALID;
  if (!isfinite(c->sm_scale)) return GLIDE_ERR_INVALID;
  for (int32_t l = 0; l < c->n_layers; ++l) {
    const int32_t W = c->windows[l];
    if (W < 0 || W > kMaxWindow) return GLIDE_ERR_INVALID;
    if (W == 0 && (c->flags & GLIDE_NO_LINEAR)) return GLIDE_ERR_INVALID;
  }
  if (c->n_q_heads / c->n_kv_heads > kMaxG) return GLIDE_ERR_UNSUPPORTED;
  if (c->head_dim != 64 && c->head_dim != 128) return GLIDE_ERR_UNSUPPORTED;
  if (c->feat_dim != 64 && c->feat_dim != 128) return GLIDE_ERR_UNSUPPORTED;
  // the gated state is built for the shared denominator only
  if ((c->flags & GLIDE_GATED) && (c->flags & GLIDE_HYBRID_SUM)) return GLIDE_ERR_UNSUPPORTED;
  return GLIDE_OK;
}

bool gated_on(const glide_config* c) { return (c->flags & GLIDE_GATED) != 0; }

int esize(const glide_config* c) { return c->dtype == GLIDE_BF16 ? 2 : 4; }

LayerSections sections(const glide_config* c, int32_t l) {
  return layer_sections(c->batch, c->n_kv_heads, c->head_dim, c->feat_dim, ring_slots(c->windows[l]),
                        esize(c), gated_on(c));
}

int64_t layer_base(const glide_config* c, int32_t l) {
  int64_t off = 0;
  for (int32_t i = 0; i < l; ++i) off += sections(c, i).bytes;
  return off;
}

int64_t state_bytes_i(const glide_config* c) { return layer_base(c, c->n_layers); }

glide_status check_call(const glide_config* c, void* state, size_t state_bytes, int32_t layer0,
                        int32_t n_layers) {
  glide_status s = check_cfg(c);
  if (s != GLIDE_OK) return s;
  if (!state) return GLIDE_ERR_NULL;
  if (!aligned(state, 256)) return GLIDE_ERR_ALIGN;
  if (state_bytes < size_t(state_bytes_i(c))) return GLIDE_ERR_SIZE;
  if (layer0 < 0 || n_layers < 1 || int64_t(layer0) + n_layers > c->n_layers) return GLIDE_ERR_INVALID;
  return GLIDE_OK;
}

glide_status hip_status(hipError_t e) { return e == hipSuccess ? GLIDE_OK : GLIDE_ERR_HIP; }

bool linear_on(const glide_config* c) { return (c->flags & GLIDE_NO_LINEAR) == 0; }

// 0: GLIDE's shared denominator; 1, 2: the Appendix's hybrid forms
int32_t merge_form(const glide_config* c) {
  if (!(c->flags & GLIDE_HYBRID_SUM)) return 0;
  return (c->flags & GLIDE_HYBRID_STATE_ALL) ? 2 : 1;
}

int32_t max_window(const glide_config* c) {
  int32_t w = 0;
  for (int32_t l = 0; l < c->n_layers; ++l) w = std::max(w, c->windows[l]);
  return w;
}

PrefillWorkspace prefill_ws(const glide_config* c, int64_t T, int32_t nl) {
  return prefill_workspace(T, c->batch, c->n_kv_heads, c->head_dim, c->feat_dim, esize(c), max_window(c),
                           linear_on(c), nl, gated_on(c));
}

// Resident decode workgroups of one round on the current device:
// kDecodeWgPerCu per compute unit, at most kMaxDecodeSlots.  Queried once per
// device (the CU count does not change while the process runs).
glide_status decode_slots(int32_t* out) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static int32_t slots[kMaxDevices] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return GLIDE_ERR_HIP;
  std::lock_guard<std::mutex> lock(mu);
  if (slots[dev] == 0) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
      return GLIDE_ERR_HIP;
    slots[dev] = int32_t(std::min<int64_t>(kMaxDecodeSlots, int64_t(cus) * kDecodeWgPerCu));
  }
  *out = slots[dev];
  return GLIDE_OK;
}

// Decode window split (pieces per unit of each layer of one launch).  The
// work of a unit is counted in 32-token window tiles plus kStateTilesLatency
// for the state pass; a layer whose units have work w gets
// min(cap, ceil(w / q)) pieces, with q the smallest piece size (>= 4 tiles)
// for which the launch fits in `slots` workgroups, and cap the most pieces
// that still give every piece four tiles or more (one per wave), one when
// the window has fewer than kSplitMinTiles tiles.  When the launch's units
// alone fill the slots, nothing is split.  The plan depends only on the
// launch's layers and the device, so a call over one layer splits that
// layer's window over the whole device.  state_tiles: the state pass's weight
// in the shares of the pieces (the kernel gives piece 0 that many tiles
// fewer), kStateTilesStream once pieces are long enough for the launch to be
// bandwidth-bound.
struct DecodePlan {
  std::vector<int32_t> np;  // pieces per unit, per layer of the launch
  int32_t state_tiles;
};

DecodePlan decode_pieces(const glide_config* c, const int32_t* layers, int32_t n, int32_t slots) {
  DecodePlan plan{std::vector<int32_t>(n, 1), kStateTilesLatency};
  const int64_t per_layer = int64_t(c->batch) * c->n_kv_heads;
  if (per_layer * n >= slots) return plan;
  const int st = linear_on(c) ? kStateTilesLatency : 0;
  std::vector<int64_t> work(n), cap(n);
  int64_t wmax = 4;
  bool any = false;
  for (int32_t i = 0; i < n; ++i) {
    const int32_t W = c->windows[layers[i]];
    const int64_t tiles = decode_tiles_max(W);
    work[i] = W > 0 ? tiles + st : 0;
    cap[i] = tiles >= kSplitMinTiles ? std::min<int64_t>(kMaxPieces, tiles / 4) : 1;
    wmax = std::max(wmax, work[i]);
    any = any || cap[i] > 1;
  }
  if (!any) return plan;
  auto pieces = [&](int64_t q, int32_t i) {
    if (work[i] == 0) return int64_t(1);
    return std::min<int64_t>(cap[i], std::max<int64_t>(1, (work[i] + q - 1) / q));
  };
  auto wgs = [&](int64_t q) {
    int64_t m = 0;
    for (int32_t i = 0; i < n; ++i) m += pieces(q, i) * per_layer;
    return m;
  };
  int64_t lo = 4, hi = wmax;  // wgs(wmax) = units <= slots
  while (lo < hi) {
    const int64_t mid = (lo + hi) / 2;
    if (wgs(mid) <= slots) hi = mid;
    else lo = mid + 1;
  }
  for (int32_t i = 0; i < n; ++i) plan.np[i] = int32_t(pieces(lo, i));
  if (lo >= kStreamPieceTiles) plan.state_tiles = kStateTilesStream;
  return plan;
}

// Decode workspace bound over every call on any device (what
// glide_workspace_bytes reports and every decode call requires, whatever its
// layers): a launch splits only when its units number fewer than its device's
// slots (at most kMaxDecodeSlots), and then it has at most that many
// workgroups, and at most the pieces its layers get at the smallest piece
// size (none for a window of fewer than kSplitMinTiles tiles).
size_t decode_ws(const glide_config* c) {
  const int64_t per_layer = int64_t(c->batch) * c->n_kv_heads;
  if (per_layer >= kMaxDecodeSlots) return 0;
  const int st = linear_on(c) ? kStateTilesLatency : 0;
  int64_t wgs = 0;
  bool any = false;
  for (int32_t l = 0; l < c->n_layers; ++l) {
    const int64_t tiles = decode_tiles_max(c->windows[l]);
    const int64_t work = c->windows[l] > 0 ? tiles + st : 0;
    const int64_t cap = tiles >= kSplitMinTiles ? std::min<int64_t>(kMaxPieces, tiles / 4) : 1;
    const int64_t p = work ? std::min<int64_t>(cap, std::max<int64_t>(1, (work + 3) / 4)) : 1;
    wgs += p * per_layer;
    any = any || p > 1;
  }
  if (!any) return 0;
  return size_t(align256(std::min<int64_t>(wgs, kMaxDecodeSlots) *
                         part_floats(c->n_q_heads / c->n_kv_heads, c->head_dim) * 4));
}

// Decode-style launch descriptor of layers [layer0, layer0 + n): per launch
// group of at most kMaxLayersPerLaunch layers, ordered by decreasing window
// (the hardware dispatcher then hands out the longest streams first).
template <typename Fn>
glide_status for_layer_groups(const glide_config* cfg, int32_t layer0, int32_t n_layers, DecodeArgs& a, Fn fn) {
  const int32_t per_layer = cfg->batch * cfg->n_kv_heads;
  int32_t slots = 0;
  const glide_status ss = decode_slots(&slots);
  if (ss != GLIDE_OK) return ss;
  std::vector<int32_t> order(n_layers);
  for (int32_t i = 0; i < n_layers; ++i) order[i] = i;
  std::stable_sort(order.begin(), order.end(), [&](int32_t x, int32_t y) {
    return cfg->windows[layer0 + x] > cfg->windows[layer0 + y];
  });
  a.B = cfg->batch;
  a.Hq = cfg->n_q_heads;
  a.Hkv = cfg->n_kv_heads;
  a.G = cfg->n_q_heads / cfg->n_kv_heads;
  a.linear = linear_on(cfg) ? 1 : 0;
  a.form = merge_form(cfg);
  a.phi = cfg->phi;
  a.wf_heads = (cfg->flags & GLIDE_PER_HEAD_PHI) ? 1 : 0;
  a.gated = gated_on(cfg) ? 1 : 0;
  a.tau = cfg->sm_scale;
  for (int32_t first = 0; first < n_layers; first += kMaxLayersPerLaunch) {
    const int32_t cnt = std::min(kMaxLayersPerLaunch, n_layers - first);
    int32_t ls[kMaxLayersPerLaunch];
    for (int32_t i = 0; i < cnt; ++i) ls[i] = layer0 + order[first + i];
    const DecodePlan plan = decode_pieces(cfg, ls, cnt, slots);
    const std::vector<int32_t>& np = plan.np;
    a.state_tiles = plan.state_tiles;
    a.n_layers = cnt;
    int32_t rows = 0;
    bool split = false;
    for (int32_t i = 0; i < cnt; ++i) {  // piece 0 of every layer first
      const int32_t l = ls[i];
      a.layers[i].base = layer_base(cfg, l);
      a.layers[i].W = cfg->windows[l];
      a.layers[i].R = ring_slots(cfg->windows[l]);
      a.layers[i].slot = order[first + i];
      a.layers[i].npiece = np[i];
      a.layers[i].prow0 = rows;
      a.piece_layer[rows++] = uint8_t(i);
      split = split || np[i] > 1;
    }
    for (int32_t i = 0; i < cnt; ++i) {  // then the other pieces
      a.layers[i].prow1 = rows;
      for (int32_t r = 1; r < np[i]; ++r) a.piece_layer[rows++] = uint8_t(i);
    }
    a.row_stride = per_layer;
    const glide_status s = hip_status(fn(a, rows * a.row_stride, split));
    if (s != GLIDE_OK) return s;
  }
  return GLIDE_OK;
}

// The allocation-free decode entry point's scratch: partial records of split
// windows, GLIDE_DECODE_SCRATCH_BYTES per GPU, held until the process ends.
// Host code never passes `scratch` itself to a kernel (in host code the name
// stands for a host-side shadow); it passes the device address that
// hipGetSymbolAddress returns for the current device, looked up once per
// device.
static __device__ __align__(256) float scratch[GLIDE_DECODE_SCRATCH_BYTES / sizeof(float)];

glide_status scratch_address(void** out) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return GLIDE_ERR_HIP;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return GLIDE_ERR_HIP;
    addr[dev] = p;
  }
  *out = addr[dev];
  return GLIDE_OK;
}

}  // namespace

extern "C" {

const char* glide_status_string(glide_status s) {
  switch (s) {
    case GLIDE_OK: return "ok";
    case GLIDE_ERR_NULL: return "required pointer is NULL";
    case GLIDE_ERR_INVALID: return "invalid argument";
    case GLIDE_ERR_UNSUPPORTED: return "unsupported configuration (head_dim/feat_dim in {64,128}, Hq/Hkv <= 16)";
    case GLIDE_ERR_ALIGN: return "misaligned device pointer (16 bytes; state 256 bytes)";
    case GLIDE_ERR_SIZE: return "state or workspace too small";
    case GLIDE_ERR_HIP: return "HIP launch failed";
    case GLIDE_ERR_SCRATCH: return "the call needs more than the fixed decode scratch (GLIDE_DECODE_SCRATCH_BYTES)";
  }
  return "unknown status";
}

size_t glide_state_bytes(const glide_config* cfg) {
  if (check_cfg(cfg) != GLIDE_OK) return 0;
  return size_t(state_bytes_i(cfg));
}

glide_status glide_state_layout(const glide_config* cfg, int32_t layer, glide_layer_layout* out) {
  glide_status s = check_cfg(cfg);
  if (s != GLIDE_OK) return s;
  if (!out) return GLIDE_ERR_NULL;
  if (layer < 0 || layer >= cfg->n_layers) return GLIDE_ERR_INVALID;
  const int64_t base = layer_base(cfg, layer);
  const LayerSections sec = sections(cfg, layer);
  out->layer_offset = base;
  out->layer_bytes = sec.bytes;
  out->pos_offset = base + sec.pos;
  out->nf_offset = base + sec.nf;
  out->cnt_offset = base + sec.cnt;
  out->s_offset = base + sec.S;
  out->z_offset = base + sec.z;
  out->kring_offset = base + sec.K;
  out->vring_offset = base + sec.V;
  out->gate_offset = base + sec.G;
  out->gring_offset = base + sec.GR;
  out->window = cfg->windows[layer];
  out->ring_slots = ring_slots(cfg->windows[layer]);
  return GLIDE_OK;
}

size_t glide_workspace_bytes(const glide_config* cfg, int64_t max_total_tokens) {
  if (check_cfg(cfg) != GLIDE_OK || max_total_tokens < 0) return 0;
  size_t pre = 0;
  if (max_total_tokens > 0) {
    // as many layers per launch as fit in the budget (at least one)
    auto slot_of = [&](int32_t nl) { return prefill_ws(cfg, max_total_tokens, nl).slot; };
    const int32_t nl = prefill_layers_per_launch(cfg->n_layers, kPrefillWsBudget, slot_of);
    pre = std::max(slot_of(1), size_t(nl) * (nl > 0 ? slot_of(nl) : 0));
  }
  return std::max(size_t(256), std::max(pre, decode_ws(cfg)));
}

glide_status glide_state_init(const glide_config* cfg, void* state, size_t state_bytes, void* stream) {
  glide_status s = check_call(cfg, state, state_bytes, 0, cfg ? cfg->n_layers : 0);
  if (s != GLIDE_OK) return s;
  return hip_status(hipMemsetAsync(state, 0, size_t(state_bytes_i(cfg)), hipStream_t(stream)));
}

glide_status glide_decode_step(const glide_config* cfg, void* state, size_t state_bytes, int32_t layer0,
                               int32_t n_layers, const void* phi_w, const void* q, const void* k,
                               const void* v, const float* log_gates, void* out, void* workspace,
                               size_t workspace_bytes, void* stream) {
  glide_status s = check_call(cfg, state, state_bytes, layer0, n_layers);
  if (s != GLIDE_OK) return s;
  if (!phi_w || !q || !k || !v || !out) return GLIDE_ERR_NULL;
  if (gated_on(cfg) && !log_gates) return GLIDE_ERR_NULL;
  if (!gated_on(cfg) && log_gates) return GLIDE_ERR_INVALID;
  if (!aligned(phi_w, 16) || !aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16) ||
      !aligned(log_gates, 4))
    return GLIDE_ERR_ALIGN;
  const size_t need = decode_ws(cfg);
  if (need) {
    if (!workspace) return GLIDE_ERR_NULL;
    if (!aligned(workspace, 256)) return GLIDE_ERR_ALIGN;
    if (workspace_bytes < need) return GLIDE_ERR_SIZE;
  }
  DecodeArgs a;
  memset(&a, 0, sizeof(a));
  a.state = static_cast<char*>(state);
  a.phi_w = phi_w;
  a.q = q;
  a.k = k;
  a.v = v;
  a.out = out;
  a.gates = log_gates;
  a.part = static_cast<float*>(workspace);
  // a state blob far larger than the Infinity Cache is streamed (every step
  // reads it all): non-temporal loads; a smaller one is re-read from the cache
  const bool streaming = state_bytes_i(cfg) > kStreamingStateBytes;
  return for_layer_groups(cfg, layer0, n_layers, a, [&](const DecodeArgs& g, int32_t wgs, bool) {
    return launch_decode(g, wgs, cfg->head_dim, cfg->feat_dim, cfg->dtype, streaming, hipStream_t(stream));
  });
}

glide_status glide_decode_step_noalloc(const glide_config* cfg, void* state, size_t state_bytes,
                                       int32_t layer0, int32_t n_layers, const void* phi_w, const void* q,
                                       const void* k, const void* v, const float* log_gates, void* out,
                                       void* stream) {
  glide_status s = check_call(cfg, state, state_bytes, layer0, n_layers);
  if (s != GLIDE_OK) return s;
  const size_t need = decode_ws(cfg);
  if (need > GLIDE_DECODE_SCRATCH_BYTES) return GLIDE_ERR_SCRATCH;
  if (!phi_w || !q || !k || !v || !out) return GLIDE_ERR_NULL;
  void* ws = nullptr;
  if (need) {
    s = scratch_address(&ws);
    if (s != GLIDE_OK) return s;
  }
  return glide_decode_step(cfg, state, state_bytes, layer0, n_layers, phi_w, q, k, v, log_gates, out, ws,
                           need ? size_t(GLIDE_DECODE_SCRATCH_BYTES) : 0, stream);
}

glide_status glide_state_flush(const glide_config* cfg, void* state, size_t state_bytes, int32_t layer0,
                               int32_t n_layers, const void* phi_w, void* stream) {
  glide_status s = check_call(cfg, state, state_bytes, layer0, n_layers);
  if (s != GLIDE_OK) return s;
  if (!phi_w) return GLIDE_ERR_NULL;
  if (!aligned(phi_w, 16)) return GLIDE_ERR_ALIGN;
  if (!linear_on(cfg)) return GLIDE_OK;
  DecodeArgs a;
  memset(&a, 0, sizeof(a));
  a.state = static_cast<char*>(state);
  a.phi_w = phi_w;
  return for_layer_groups(cfg, layer0, n_layers, a, [&](const DecodeArgs& g, int32_t, bool) {
    return launch_flush(g, cfg->head_dim, cfg->feat_dim, cfg->dtype, hipStream_t(stream));
  });
}

glide_status glide_prefill(const glide_config* cfg, void* state, size_t state_bytes, int32_t layer0,
                           int32_t n_layers, const void* phi_w, const void* q, const void* k, const void* v,
                           const float* log_gates, const int32_t* cu_seqlens_host, int64_t total_tokens,
                           int32_t chunk, void* out, void* workspace, size_t workspace_bytes, void* stream) {
  glide_status s = check_call(cfg, state, state_bytes, layer0, n_layers);
  if (s != GLIDE_OK) return s;
  if (!phi_w || !q || !k || !v || !out || !cu_seqlens_host) return GLIDE_ERR_NULL;
  if (gated_on(cfg) && !log_gates) return GLIDE_ERR_NULL;
  if (!gated_on(cfg) && log_gates) return GLIDE_ERR_INVALID;
  if (!aligned(phi_w, 16) || !aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16) ||
      !aligned(log_gates, 4))
    return GLIDE_ERR_ALIGN;
  if (total_tokens < 0) return GLIDE_ERR_INVALID;
  if (cu_seqlens_host[0] != 0 || cu_seqlens_host[cfg->batch] != total_tokens) return GLIDE_ERR_INVALID;
  for (int32_t b = 0; b < cfg->batch; ++b)
    if (cu_seqlens_host[b + 1] < cu_seqlens_host[b]) return GLIDE_ERR_INVALID;
  // the kernels address one sequence's new rows with 32-bit byte offsets
  for (int32_t b = 0; b < cfg->batch; ++b)
    if (int64_t(cu_seqlens_host[b + 1] - cu_seqlens_host[b]) * cfg->n_q_heads * cfg->head_dim * esize(cfg) >=
        (int64_t(1) << 31))
      return GLIDE_ERR_UNSUPPORTED;
  if (chunk == 0) chunk = 64;
  if (chunk < 32 || chunk > 256 || chunk % 32) return GLIDE_ERR_INVALID;
  const size_t need = glide_workspace_bytes(cfg, total_tokens);
  if (workspace_bytes < need) return GLIDE_ERR_SIZE;
  if (!workspace) return GLIDE_ERR_NULL;
  if (!aligned(workspace, 256)) return GLIDE_ERR_ALIGN;
  if (total_tokens == 0) return GLIDE_OK;

  // Tokens still pending from decode steps are folded first, so the state
  // the chunked pass starts from is S = sum_{j < max(0, p - W)}.
  s = glide_state_flush(cfg, state, state_bytes, layer0, n_layers, phi_w, stream);
  if (s != GLIDE_OK) return s;

  const int64_t T = total_tokens;
  const int B = cfg->batch, Hq = cfg->n_q_heads, Hkv = cfg->n_kv_heads, d = cfg->head_dim, Df = cfg->feat_dim;
  const int es = esize(cfg);
  const bool lin = linear_on(cfg);
  hipStream_t st = hipStream_t(stream);
  // layers per launch: as many workspace slots (each sized for launches of
  // that many layers) as the caller's workspace holds
  auto slot_of = [&](int32_t nl) { return prefill_ws(cfg, T, nl).slot; };
  const int32_t per_launch = std::max(1, prefill_layers_per_launch(n_layers, workspace_bytes, slot_of));
  const PrefillWorkspace w = prefill_ws(cfg, T, per_launch);
  const int32_t seg_len = chunk * segment_chunks(T, Hkv, chunk, per_launch);

  PrefillArgs a;
  memset(&a, 0, sizeof(a));
  a.state = static_cast<char*>(state);
  a.q = static_cast<const char*>(q);
  a.k = static_cast<const char*>(k);
  a.v = static_cast<const char*>(v);
  a.out = static_cast<char*>(out);
  a.wf = static_cast<const char*>(phi_w);
  a.q_stride = T * Hq * d * es;
  a.kv_stride = T * Hkv * d * es;
  const bool wf_heads = (cfg->flags & GLIDE_PER_HEAD_PHI) != 0;
  a.wf_stride = int64_t(wf_heads ? Hkv : 1) * d * Df * es;
  a.wf_hs = wf_heads ? int32_t(int64_t(d) * Df * es) : 0;
  a.ws = static_cast<char*>(workspace);
  a.ws_slot = int64_t(w.slot);
  a.ws_hv = int64_t(w.hv);
  a.ws_seg = int64_t(w.seg);
  a.ws_hg = int64_t(w.hg);
  a.ws_gc = int64_t(w.gc);
  a.gated = gated_on(cfg) ? 1 : 0;
  a.gates = log_gates;
  a.g_stride = T * Hkv;
  a.B = B;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.G = Hq / Hkv;
  a.linear = lin ? 1 : 0;
  a.form = merge_form(cfg);
  a.phi = cfg->phi;
  a.tau = cfg->sm_scale;
  a.C = chunk;
  a.seg_len = seg_len;
  a.Wcap = max_window(cfg);

  // fill the per-group tables of sequences [g0, g0 + n)
  auto group = [&](int g0, int32_t seg0) {
    const int n = std::min(kMaxSeqPerLaunch, B - g0);
    a.seq0 = g0;
    a.nseq = n;
    a.seg0 = seg0;
    int32_t nseg = 0;
    for (int i = 0; i < n; ++i) {
      a.seq_start[i] = cu_seqlens_host[g0 + i];
      a.seq_len[i] = cu_seqlens_host[g0 + i + 1] - cu_seqlens_host[g0 + i];
      a.seg_base[i] = nseg;
      nseg += (a.seq_len[i] + seg_len - 1) / seg_len;
    }
    a.seg_base[n] = nseg;
    a.nseg = nseg;
    return nseg;
  };

  // Layers by decreasing window, dealt round-robin over the launches: every
  // launch gets a like mix of long and short windows, longest first (their
  // workgroups are dispatched first).
  std::vector<int32_t> rank(n_layers);
  for (int32_t j = 0; j < n_layers; ++j) rank[j] = j;
  std::stable_sort(rank.begin(), rank.end(), [&](int32_t x, int32_t y) {
    return cfg->windows[layer0 + x] > cfg->windows[layer0 + y];
  });
  const int32_t n_launch = (n_layers + per_launch - 1) / per_launch;
  for (int32_t li = 0; li < n_launch; ++li) {
    std::vector<int32_t> order;
    for (int32_t j = li; j < n_layers; j += n_launch) order.push_back(rank[j]);
    const int32_t nl = int32_t(order.size());
    bool window = false;
    for (int32_t j = 0; j < nl; ++j) {
      const int32_t l = layer0 + order[j];
      PrefillLayer& L = a.layers[j];
      L.layer_base = layer_base(cfg, l);
      L.W = cfg->windows[l];
      L.R = ring_slots(L.W);
      L.li = order[j];
      window = window || L.W > 0;
    }
    a.nlayer = nl;
    int32_t seg0 = 0;
    for (int g0 = 0; g0 < B; g0 += kMaxSeqPerLaunch) {
      const int32_t nseg = group(g0, seg0);
      if (window) {
        // history of a continuing prefill (nothing to copy when pos == 0)
        s = hip_status(launch_prefill_gather(a, d, Df, cfg->dtype, st));
        if (s != GLIDE_OK) return s;
      }
      s = hip_status(launch_prefill_layer(a, d, Df, cfg->dtype, st));
      if (s != GLIDE_OK) return s;
      seg0 += nseg;
    }
  }
  return GLIDE_OK;
}

glide_status glide_feature_map(const glide_config* cfg, const void* phi_w, const void* x, int64_t rows,
                               void* out, void* stream) {
  glide_status s = check_cfg(cfg);
  if (s != GLIDE_OK) return s;
  if (rows < 0) return GLIDE_ERR_INVALID;
  if (!phi_w || (rows > 0 && (!x || !out))) return GLIDE_ERR_NULL;
  if (!aligned(phi_w, 16) || !aligned(x, 16) || !aligned(out, 16)) return GLIDE_ERR_ALIGN;
  return hip_status(launch_phi_rows(phi_w, x, rows, out, cfg->head_dim, cfg->feat_dim, cfg->dtype,
                                    cfg->dtype == GLIDE_F32, cfg->phi, hipStream_t(stream)));
}

}  // extern "C"
