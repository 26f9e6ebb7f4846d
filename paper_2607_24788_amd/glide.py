"""Thin ctypes binding of ``libglide.so`` (declared in include/glide.h).

Argument marshalling only: every step of the hybrid-attention layer runs in
the HIP kernels behind the C ABI.  Tensors are torch device tensors; their
data pointers and the current HIP stream are handed to the library.  If the
compiled library is missing, loading fails loudly -- there is no fallback.
"""
import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libglide.so")

F32 = 0
BF16 = 1
PHI_RELU = 0
PHI_ELU1 = 1
PHI_SOFTMAX = 2
NO_LINEAR = 1
HYBRID_SUM = 2
HYBRID_STATE_ALL = 4
PER_HEAD_PHI = 8
GATED = 16

STATUS = {0: "GLIDE_OK", -1: "GLIDE_ERR_NULL", -2: "GLIDE_ERR_INVALID", -3: "GLIDE_ERR_UNSUPPORTED",
          -4: "GLIDE_ERR_ALIGN", -5: "GLIDE_ERR_SIZE", -6: "GLIDE_ERR_HIP", -7: "GLIDE_ERR_SCRATCH"}
DECODE_SCRATCH_BYTES = 16 << 20

EXPORTS = ["glide_state_bytes", "glide_state_layout", "glide_workspace_bytes", "glide_state_init",
           "glide_prefill", "glide_decode_step", "glide_decode_step_noalloc", "glide_state_flush", "glide_feature_map",
           "glide_status_string"]


class GlideError(RuntimeError):
    def __init__(self, status, where, lib=None):
        msg = STATUS.get(status, str(status))
        if lib is not None:
            msg += ": " + lib.glide_status_string(status).decode()
        super().__init__(f"{where} failed with {msg}")
        self.status = status


class Config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("batch", ctypes.c_int32),
                ("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("feat_dim", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("phi", ctypes.c_int32), ("flags", ctypes.c_int32),
                ("sm_scale", ctypes.c_float), ("windows", ctypes.POINTER(ctypes.c_int32))]


class LayerLayout(ctypes.Structure):
    _fields_ = [("pos_offset", ctypes.c_int64), ("nf_offset", ctypes.c_int64), ("cnt_offset", ctypes.c_int64),
                ("s_offset", ctypes.c_int64),
                ("z_offset", ctypes.c_int64), ("kring_offset", ctypes.c_int64),
                ("vring_offset", ctypes.c_int64), ("gate_offset", ctypes.c_int64),
                ("gring_offset", ctypes.c_int64), ("layer_offset", ctypes.c_int64),
                ("layer_bytes", ctypes.c_int64), ("window", ctypes.c_int32),
                ("ring_slots", ctypes.c_int32)]


_lib = None


def load_library(path=None):
    """Load libglide.so; raises if it has not been built."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"{p} is missing: build it with paper_2607_24788_amd/build.py "
                           "(or __graft_entry__.build()); there is no fallback path")
    lib = ctypes.CDLL(p)
    cfgp = ctypes.POINTER(Config)
    vp = ctypes.c_void_p
    lib.glide_state_bytes.argtypes = [cfgp]
    lib.glide_state_bytes.restype = ctypes.c_size_t
    lib.glide_state_layout.argtypes = [cfgp, ctypes.c_int32, ctypes.POINTER(LayerLayout)]
    lib.glide_state_layout.restype = ctypes.c_int
    lib.glide_workspace_bytes.argtypes = [cfgp, ctypes.c_int64]
    lib.glide_workspace_bytes.restype = ctypes.c_size_t
    lib.glide_state_init.argtypes = [cfgp, vp, ctypes.c_size_t, vp]
    lib.glide_state_init.restype = ctypes.c_int
    lib.glide_prefill.argtypes = [cfgp, vp, ctypes.c_size_t, ctypes.c_int32, ctypes.c_int32, vp, vp, vp, vp, vp,
                                  ctypes.POINTER(ctypes.c_int32), ctypes.c_int64, ctypes.c_int32, vp, vp,
                                  ctypes.c_size_t, vp]
    lib.glide_prefill.restype = ctypes.c_int
    lib.glide_decode_step.argtypes = [cfgp, vp, ctypes.c_size_t, ctypes.c_int32, ctypes.c_int32, vp, vp, vp,
                                      vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.glide_decode_step.restype = ctypes.c_int
    lib.glide_decode_step_noalloc.argtypes = [cfgp, vp, ctypes.c_size_t, ctypes.c_int32, ctypes.c_int32, vp, vp,
                                              vp, vp, vp, vp, vp]
    lib.glide_decode_step_noalloc.restype = ctypes.c_int
    lib.glide_state_flush.argtypes = [cfgp, vp, ctypes.c_size_t, ctypes.c_int32, ctypes.c_int32, vp, vp]
    lib.glide_state_flush.restype = ctypes.c_int
    lib.glide_feature_map.argtypes = [cfgp, vp, vp, ctypes.c_int64, vp, vp]
    lib.glide_feature_map.restype = ctypes.c_int
    lib.glide_status_string.argtypes = [ctypes.c_int]
    lib.glide_status_string.restype = ctypes.c_char_p
    if path is None:
        _lib = lib
    return lib


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _check(name, t, numel=None, dtype=None):
    """The library reads and writes through raw pointers and cannot see sizes
    or layouts: refuse a tensor that is not a contiguous device tensor of the
    expected element type holding at least `numel` elements."""
    if t is None:
        return
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a torch tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name} holds {t.numel()} elements, at least {numel} needed")


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def kring_logical(raw, R, d):
    """Key ring [..., R*d] (32-slot blocks [t][d/32][4][16][8]) -> [..., R, d] by slot."""
    lead = raw.shape[:-1]
    n = len(lead)
    x = raw.reshape(*lead, R // 32, 2, d // 32, 4, 4, 4, 8)        # blk t kk g mh ml e
    return x.permute(*range(n), *(n + i for i in (0, 4, 1, 5, 2, 3, 6))).reshape(*lead, R, d)


def kring_raw(logical, R, d):
    """Inverse of kring_logical."""
    lead = logical.shape[:-2]
    n = len(lead)
    x = logical.reshape(*lead, R // 32, 4, 2, 4, d // 32, 4, 8)    # blk mh t ml kk g e
    return x.permute(*range(n), *(n + i for i in (0, 2, 4, 5, 1, 3, 6))).reshape(*lead, R * d)


def vring_logical(raw, R, d):
    """Value ring [..., R*d] (32-slot blocks [d/16][4][16][8]) -> [..., R, d] by slot."""
    lead = raw.shape[:-1]
    n = len(lead)
    x = raw.reshape(*lead, R // 32, d // 16, 4, 16, 8)              # blk ct g n e
    return x.permute(*range(n), *(n + i for i in (0, 2, 4, 1, 3))).reshape(*lead, R, d)


def vring_raw(logical, R, d):
    """Inverse of vring_logical."""
    lead = logical.shape[:-2]
    n = len(lead)
    x = logical.reshape(*lead, R // 32, 4, 8, d // 16, 16)          # blk g e ct n
    return x.permute(*range(n), *(n + i for i in (0, 3, 1, 4, 2))).reshape(*lead, R * d)


class Glide:
    """A configured GLIDE layer stack (mirrors ``glide_config``).

    ``form`` selects the merge: 0 GLIDE's shared denominator (default), 1 and
    2 the two hybrid forms (``HYBRID_SUM``, ``HYBRID_SUM | HYBRID_STATE_ALL``).
    """

    def __init__(self, n_layers, batch, n_q_heads, n_kv_heads, head_dim, feat_dim, windows,
                 dtype=torch.bfloat16, sm_scale=None, linear=True, lib=None, form=0, phi=PHI_RELU,
                 per_head_phi=False, gated=False):
        self.lib = lib if lib is not None else load_library()
        self.windows = [int(w) for w in windows]
        if len(self.windows) != n_layers:
            raise ValueError("need one window per layer")
        self._win = (ctypes.c_int32 * n_layers)(*self.windows)
        self.torch_dtype = dtype
        code = {torch.float32: F32, torch.bfloat16: BF16}.get(dtype, 99)
        if sm_scale is None:
            sm_scale = head_dim ** -0.5
        flags = (0 if linear else NO_LINEAR) | {0: 0, 1: HYBRID_SUM, 2: HYBRID_SUM | HYBRID_STATE_ALL}.get(form, 99)
        if per_head_phi:
            flags |= PER_HEAD_PHI
        if gated:
            flags |= GATED
        self.cfg = Config(n_layers, batch, n_q_heads, n_kv_heads, head_dim, feat_dim, code, int(phi),
                          flags, float(sm_scale), self._win)
        self.n_layers, self.batch = n_layers, batch
        self.n_q_heads, self.n_kv_heads = n_q_heads, n_kv_heads
        self.head_dim, self.feat_dim = head_dim, feat_dim
        self.sm_scale = float(sm_scale)
        self.linear = linear
        self.form = form
        self.phi = phi
        self.per_head_phi = per_head_phi
        self.gated = gated

    # -- sizes and layout ----------------------------------------------------
    def state_bytes(self):
        return self.lib.glide_state_bytes(ctypes.byref(self.cfg))

    def workspace_bytes(self, max_total_tokens):
        return self.lib.glide_workspace_bytes(ctypes.byref(self.cfg), int(max_total_tokens))

    def layout(self, layer):
        out = LayerLayout()
        s = self.lib.glide_state_layout(ctypes.byref(self.cfg), int(layer), ctypes.byref(out))
        if s:
            raise GlideError(s, "glide_state_layout", self.lib)
        return out

    def new_state(self, device="cuda"):
        n = self.state_bytes()
        if n == 0:
            raise GlideError(-2, "glide_state_bytes", self.lib)
        return torch.empty(n, dtype=torch.uint8, device=device)

    def layer_views(self, state, layer):
        """Typed views of one layer inside ``state``: pos, S, z, and the raw
        rings kring_raw / vring_raw [B][Hkv][R*d] (fragment-major layout, see
        include/glide.h; convert with kring_logical / vring_logical)."""
        lay = self.layout(layer)
        B, H, d, Df, R = self.batch, self.n_kv_heads, self.head_dim, self.feat_dim, lay.ring_slots
        es = 2 if self.torch_dtype == torch.bfloat16 else 4

        def view(off, n, dt, shape, esz):
            return state[off:off + n * esz].view(dt).view(*shape)

        return {
            "pos": view(lay.pos_offset, B * H, torch.int64, (B, H), 8),
            "nf": view(lay.nf_offset, B * H, torch.int64, (B, H), 8),
            "cnt": view(lay.cnt_offset, B * H, torch.int32, (B, H), 4),
            "S": view(lay.s_offset, B * H * Df * d, torch.float32, (B, H, Df, d), 4),
            "z": view(lay.z_offset, B * H * Df, torch.float32, (B, H, Df), 4),
            "kring_raw": view(lay.kring_offset, B * H * R * d, self.torch_dtype, (B, H, R * d), es),
            "vring_raw": view(lay.vring_offset, B * H * R * d, self.torch_dtype, (B, H, R * d), es),
            # gated state only (empty otherwise): [G_{p-1}, G_f] and the gate ring, fp64
            "gate": view(lay.gate_offset, B * H * 2 if self.gated else 0, torch.float64, (B, H, 2) if self.gated
                         else (0,), 8),
            "gring": view(lay.gring_offset, B * H * R if self.gated else 0, torch.float64, (B, H, R) if self.gated
                          else (0,), 8),
            "window": lay.window, "ring_slots": R,
        }

    def _wf_numel(self, n_layers):
        return n_layers * (self.n_kv_heads if self.per_head_phi else 1) * self.head_dim * self.feat_dim

    def _check_gates(self, log_gates, numel):
        if self.gated:
            if log_gates is None:
                raise ValueError("a gated stack needs log_gates")
            _check("log_gates", log_gates, numel, torch.float32)
        elif log_gates is not None:
            raise ValueError("log_gates given to a stack that is not gated")

    def _check_decode(self, state, phi_w, q, k, v, out, n_layers):
        dt = self.torch_dtype
        _check("state", state)
        _check("phi_w", phi_w, self._wf_numel(n_layers), dt)
        nq = n_layers * self.batch * self.n_q_heads * self.head_dim
        nkv = n_layers * self.batch * self.n_kv_heads * self.head_dim
        _check("q", q, nq, dt)
        _check("k", k, nkv, dt)
        _check("v", v, nkv, dt)
        _check("out", out, nq, dt)

    # -- calls ---------------------------------------------------------------
    def state_init(self, state, stream=None):
        s = self.lib.glide_state_init(ctypes.byref(self.cfg), _ptr(state), state.numel() * state.element_size(),
                                      _stream(stream))
        if s:
            raise GlideError(s, "glide_state_init", self.lib)

    def new_workspace(self, max_total_tokens=0, device="cuda"):
        return torch.empty(max(self.workspace_bytes(max_total_tokens), 256), dtype=torch.uint8, device=device)

    def state_flush(self, state, phi_w, layer0=0, n_layers=None, stream=None):
        """Fold every pending token into S, z (nf := max(0, pos - W))."""
        if n_layers is None:
            n_layers = self.n_layers - layer0
        _check("state", state)
        _check("phi_w", phi_w, self._wf_numel(n_layers), self.torch_dtype)
        s = self.lib.glide_state_flush(ctypes.byref(self.cfg), _ptr(state), state.numel() * state.element_size(),
                                       int(layer0), int(n_layers), _ptr(phi_w), _stream(stream))
        if s:
            raise GlideError(s, "glide_state_flush", self.lib)

    def decode_step(self, state, phi_w, q, k, v, out, workspace=None, layer0=0, n_layers=None, stream=None,
                    log_gates=None):
        if n_layers is None:
            n_layers = self.n_layers - layer0
        self._check_decode(state, phi_w, q, k, v, out, n_layers)
        self._check_gates(log_gates, n_layers * self.batch * self.n_kv_heads)
        _check("workspace", workspace)
        ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
        s = self.lib.glide_decode_step(ctypes.byref(self.cfg), _ptr(state), state.numel() * state.element_size(),
                                       int(layer0), int(n_layers), _ptr(phi_w), _ptr(q), _ptr(k), _ptr(v),
                                       _ptr(log_gates), _ptr(out), _ptr(workspace), ws_bytes, _stream(stream))
        if s:
            raise GlideError(s, "glide_decode_step", self.lib)

    def decode_step_noalloc(self, state, phi_w, q, k, v, out, layer0=0, n_layers=None, stream=None,
                            log_gates=None):
        """decode_step with no workspace: split-window records go to the
        library's fixed per-GPU scratch (calls on one GPU must not overlap)."""
        if n_layers is None:
            n_layers = self.n_layers - layer0
        self._check_decode(state, phi_w, q, k, v, out, n_layers)
        self._check_gates(log_gates, n_layers * self.batch * self.n_kv_heads)
        s = self.lib.glide_decode_step_noalloc(ctypes.byref(self.cfg), _ptr(state),
                                               state.numel() * state.element_size(), int(layer0), int(n_layers),
                                               _ptr(phi_w), _ptr(q), _ptr(k), _ptr(v), _ptr(log_gates), _ptr(out),
                                               _stream(stream))
        if s:
            raise GlideError(s, "glide_decode_step_noalloc", self.lib)

    def prefill(self, state, phi_w, q, k, v, cu_seqlens, out, workspace, layer0=0, n_layers=None, chunk=0,
                stream=None, log_gates=None):
        if n_layers is None:
            n_layers = self.n_layers - layer0
        cu = [int(x) for x in cu_seqlens]
        if len(cu) != self.batch + 1:
            raise ValueError("cu_seqlens needs batch + 1 entries")
        cu_arr = (ctypes.c_int32 * len(cu))(*cu)
        T, dt = cu[-1], self.torch_dtype
        _check("state", state)
        _check("phi_w", phi_w, self._wf_numel(n_layers), dt)
        _check("q", q, n_layers * T * self.n_q_heads * self.head_dim, dt)
        _check("k", k, n_layers * T * self.n_kv_heads * self.head_dim, dt)
        _check("v", v, n_layers * T * self.n_kv_heads * self.head_dim, dt)
        _check("out", out, n_layers * T * self.n_q_heads * self.head_dim, dt)
        _check("workspace", workspace)
        self._check_gates(log_gates, n_layers * T * self.n_kv_heads)
        ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
        s = self.lib.glide_prefill(ctypes.byref(self.cfg), _ptr(state), state.numel() * state.element_size(),
                                   int(layer0), int(n_layers), _ptr(phi_w), _ptr(q), _ptr(k), _ptr(v),
                                   _ptr(log_gates), cu_arr,
                                   int(cu[-1]), int(chunk), _ptr(out), _ptr(workspace), ws_bytes,
                                   _stream(stream))
        if s:
            raise GlideError(s, "glide_prefill", self.lib)

    def feature_map(self, phi_w, x, out, stream=None):
        rows = out.numel() // self.feat_dim
        _check("phi_w", phi_w, self.head_dim * self.feat_dim, self.torch_dtype)
        _check("x", x, rows * self.head_dim, self.torch_dtype)
        _check("out", out, rows * self.feat_dim, self.torch_dtype)
        s = self.lib.glide_feature_map(ctypes.byref(self.cfg), _ptr(phi_w), _ptr(x), int(rows), _ptr(out),
                                       _stream(stream))
        if s:
            raise GlideError(s, "glide_feature_map", self.lib)
