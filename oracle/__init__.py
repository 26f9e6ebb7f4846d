"""CPU oracle of the GLIDE hybrid-attention layer -- TEST INFRASTRUCTURE ONLY.

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product library never calls it,
and it shares no code with the GPU path: the arithmetic lives in
``glide_oracle.c`` (plain C, float64, scalar loops); this module only
marshals numpy arrays into it.

Definition implemented (GLIDE, Sec. III-B first three displayed equations
with the window split read as W = w - delta; Sec. II-B recurrence; Sec. II-C
window; shared-denominator merge of Sec. II-A / III-B): see the header of
``glide_oracle.c``.
"""
import ctypes
import os

import numpy as np

from . import build as _build

_c_double_p = ctypes.POINTER(ctypes.c_double)
_c_int64_p = ctypes.POINTER(ctypes.c_int64)


class OracleLayer(ctypes.Structure):
    _fields_ = [("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("feat_dim", ctypes.c_int32),
                ("window", ctypes.c_int32), ("linear", ctypes.c_int32),
                ("form", ctypes.c_int32), ("phi", ctypes.c_int32), ("wf_per_head", ctypes.c_int32),
                ("tau", ctypes.c_double)]


_LIBS = {}


def load(path=None):
    """Load (building first if absent) the oracle library at ``path``."""
    path = path or _build.LIB
    if path in _LIBS:
        return _LIBS[path]
    if not os.path.exists(path):
        if path != _build.LIB:
            raise FileNotFoundError(path)
        _build.build(path)
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER(OracleLayer)
    lib.oracle_phi.argtypes = [P, _c_double_p, ctypes.c_int64, _c_double_p, _c_double_p]
    lib.oracle_phi.restype = None
    lib.oracle_attend.argtypes = [P, _c_double_p, ctypes.c_int64, _c_double_p, _c_double_p,
                                  _c_double_p, ctypes.c_int64, _c_int64_p, _c_double_p]
    lib.oracle_attend.restype = ctypes.c_int
    lib.oracle_state.argtypes = [P, _c_double_p, ctypes.c_int64, _c_double_p, _c_double_p,
                                 _c_double_p, _c_double_p]
    lib.oracle_state.restype = ctypes.c_int
    lib.oracle_attend_gated.argtypes = [P, _c_double_p, ctypes.c_int64, _c_double_p, _c_double_p,
                                        _c_double_p, _c_double_p, ctypes.c_int64, _c_int64_p, _c_double_p]
    lib.oracle_attend_gated.restype = ctypes.c_int
    lib.oracle_state_gated.argtypes = [P, _c_double_p, ctypes.c_int64, _c_double_p, _c_double_p, _c_double_p,
                                       _c_double_p, _c_double_p]
    lib.oracle_state_gated.restype = ctypes.c_int
    lib.oracle_decode_batch.argtypes = [P, _c_double_p, ctypes.c_int32, _c_double_p, _c_double_p,
                                        _c_double_p, _c_double_p, _c_int64_p, _c_double_p,
                                        _c_double_p, _c_double_p, _c_double_p]
    lib.oracle_decode_batch.restype = ctypes.c_int
    _LIBS[path] = lib
    return lib


def _d(a):
    a = np.ascontiguousarray(np.asarray(a, dtype=np.float64))
    return a, a.ctypes.data_as(_c_double_p)


def _shape(name, a, want):
    """Raise unless array a has shape `want` (the C code reads exactly that)."""
    if tuple(a.shape) != tuple(want):
        raise ValueError(f"{name} has shape {tuple(a.shape)}, expected {tuple(want)}")


class Oracle:
    """One layer's oracle: Hq, Hkv, d, Df, window W, linear on/off, tau, and
    the merge form (0: GLIDE's shared denominator; 1, 2: the Appendix's two
    hybrid forms, separately normalised outputs added, with the state over
    the evicted tokens (1) or over every token (2)), and the feature map
    (phi 0: ReLU(x Wf); 1: ELU(x Wf) + 1; 2: softmax(x Wf) over the features)."""

    def __init__(self, n_q_heads, n_kv_heads, head_dim, feat_dim, window, linear=True,
                 tau=None, lib=None, form=0, phi=0, wf_per_head=False):
        if tau is None:
            tau = 1.0 / np.sqrt(head_dim)
        self.L = OracleLayer(n_q_heads, n_kv_heads, head_dim, feat_dim, window,
                             1 if linear else 0, int(form), int(phi), 1 if wf_per_head else 0, float(tau))
        self.lib = lib if lib is not None else load()

    # -- feature map -------------------------------------------------------
    def phi(self, Wf, x):
        """phi(x @ Wf) over the last axis with one Wf [d][Df]; x [..., d] -> [..., Df]."""
        L = self.L
        x, xp = _d(x)
        Wf, wp = _d(Wf)
        _shape("Wf", Wf, (L.head_dim, L.feat_dim))
        if x.shape[-1] != L.head_dim:
            raise ValueError(f"x rows have {x.shape[-1]} elements, expected {L.head_dim}")
        rows = x.size // L.head_dim
        out = np.empty(x.shape[:-1] + (L.feat_dim,), np.float64)
        self.lib.oracle_phi(ctypes.byref(L), wp, rows, xp, out.ctypes.data_as(_c_double_p))
        return out

    # -- definition (quadratic) form ----------------------------------------
    def _wf_shape(self):
        L = self.L
        return ((L.n_kv_heads,) if L.wf_per_head else ()) + (L.head_dim, L.feat_dim)

    def _check_history(self, Wf, q, k, v, n):
        L = self.L
        _shape("Wf", Wf, self._wf_shape())
        if q is not None:
            _shape("q", q, (n, L.n_q_heads, L.head_dim))
        _shape("k", k, (n, L.n_kv_heads, L.head_dim))
        _shape("v", v, (n, L.n_kv_heads, L.head_dim))

    def attend(self, Wf, q, k, v, positions=None):
        """O_t for one sequence.  q [n][Hq][d], k/v [n][Hkv][d].

        ``positions``: the t to evaluate (default: all).  Returns [len][Hq][d].
        """
        L = self.L
        q, qp = _d(q)
        k, kp = _d(k)
        v, vp = _d(v)
        Wf, wp = _d(Wf)
        n = q.shape[0]
        self._check_history(Wf, q, k, v, n)
        if positions is None:
            positions = np.arange(n, dtype=np.int64)
        pos = np.ascontiguousarray(np.asarray(positions, dtype=np.int64))
        out = np.empty((pos.size, L.n_q_heads, L.head_dim), np.float64)
        rc = self.lib.oracle_attend(ctypes.byref(L), wp, n, qp, kp, vp, pos.size,
                                    pos.ctypes.data_as(_c_int64_p),
                                    out.ctypes.data_as(_c_double_p))
        if rc != 0:
            raise ValueError("oracle_attend rejected its arguments")
        return out

    def state(self, Wf, k, v, p=None):
        """(S [Hkv][Df][d], z [Hkv][Df]) after the first p tokens (default all)."""
        L = self.L
        k, kp = _d(k)
        v, vp = _d(v)
        Wf, wp = _d(Wf)
        if p is None:
            p = k.shape[0]
        self._check_history(Wf, None, k, v, k.shape[0])
        # the sums read tokens [0, p - W) (every token before p in form 2)
        nfold = 0 if not L.linear else (p if L.form == 2 else max(0, p - L.window))
        if p < 0 or nfold > k.shape[0]:
            raise ValueError(f"the state after p = {p} tokens needs {nfold} of the {k.shape[0]} given")
        S = np.empty((L.n_kv_heads, L.feat_dim, L.head_dim), np.float64)
        z = np.empty((L.n_kv_heads, L.feat_dim), np.float64)
        rc = self.lib.oracle_state(ctypes.byref(L), wp, int(p), kp, vp,
                                   S.ctypes.data_as(_c_double_p), z.ctypes.data_as(_c_double_p))
        if rc != 0:
            raise ValueError("oracle_state rejected its arguments")
        return S, z

    # -- gated linear state (GLA-style decay) ---------------------------------
    def attend_gated(self, Wf, q, k, v, log_gates, positions=None):
        """The definition form with a gated linear state: log_gates [n][Hkv]
        (<= 0); a linear-set token j read at time t weighs
        e^{sum_{i=j+1..t} log_gates[i]}."""
        L = self.L
        q, qp = _d(q)
        k, kp = _d(k)
        v, vp = _d(v)
        lg, lgp = _d(log_gates)
        Wf, wp = _d(Wf)
        n = q.shape[0]
        self._check_history(Wf, q, k, v, n)
        _shape("log_gates", lg, (n, L.n_kv_heads))
        pos = np.arange(n, dtype=np.int64) if positions is None else np.ascontiguousarray(positions, np.int64)
        out = np.empty((len(pos), L.n_q_heads, L.head_dim), np.float64)
        rc = self.lib.oracle_attend_gated(ctypes.byref(L), wp, n, qp, kp, vp, lgp, len(pos),
                                          pos.ctypes.data_as(_c_int64_p), out.ctypes.data_as(_c_double_p))
        if rc != 0:
            raise ValueError("oracle_attend_gated rejected its arguments")
        return out

    def state_gated(self, Wf, k, v, log_gates, p=None):
        """(S, z) of the gated state after the first p tokens (decayed through token p - 1)."""
        L = self.L
        k, kp = _d(k)
        v, vp = _d(v)
        lg, lgp = _d(log_gates)
        Wf, wp = _d(Wf)
        if p is None:
            p = k.shape[0]
        self._check_history(Wf, None, k, v, k.shape[0])
        _shape("log_gates", lg, (k.shape[0], L.n_kv_heads))
        if not 0 <= p <= k.shape[0]:
            raise ValueError(f"p = {p} outside [0, {k.shape[0]}]")
        S = np.empty((L.n_kv_heads, L.feat_dim, L.head_dim), np.float64)
        z = np.empty((L.n_kv_heads, L.feat_dim), np.float64)
        rc = self.lib.oracle_state_gated(ctypes.byref(L), wp, int(p), kp, vp, lgp,
                                         S.ctypes.data_as(_c_double_p), z.ctypes.data_as(_c_double_p))
        if rc != 0:
            raise ValueError("oracle_state_gated rejected its arguments")
        return S, z

    # -- recurrent form ------------------------------------------------------
    def empty_state(self, batch):
        L = self.L
        W = L.window
        return {
            "S": np.zeros((batch, L.n_kv_heads, L.feat_dim, L.head_dim)),
            "z": np.zeros((batch, L.n_kv_heads, L.feat_dim)),
            "wk": np.zeros((batch, L.n_kv_heads, W, L.head_dim)),
            "wv": np.zeros((batch, L.n_kv_heads, W, L.head_dim)),
            "pos": np.zeros((batch,), np.int64),
        }

    def decode(self, Wf, st, q, k, v):
        """One decode step for a batch.  q [B][Hq][d], k/v [B][Hkv][d].

        ``st`` (from empty_state, or built by the caller) is updated in place.
        Returns out [B][Hq][d].
        """
        L = self.L
        B = st["pos"].shape[0]
        for key in ("S", "z", "wk", "wv"):
            st[key] = np.ascontiguousarray(st[key], dtype=np.float64)
        st["pos"] = np.ascontiguousarray(st["pos"], dtype=np.int64)
        q, qp = _d(q)
        k, kp = _d(k)
        v, vp = _d(v)
        Wf, wp = _d(Wf)
        _shape("Wf", Wf, self._wf_shape())
        _shape("q", q, (B, L.n_q_heads, L.head_dim))
        _shape("k", k, (B, L.n_kv_heads, L.head_dim))
        _shape("v", v, (B, L.n_kv_heads, L.head_dim))
        _shape("S", st["S"], (B, L.n_kv_heads, L.feat_dim, L.head_dim))
        _shape("z", st["z"], (B, L.n_kv_heads, L.feat_dim))
        _shape("wk", st["wk"], (B, L.n_kv_heads, L.window, L.head_dim))
        _shape("wv", st["wv"], (B, L.n_kv_heads, L.window, L.head_dim))
        out = np.empty((B, L.n_q_heads, L.head_dim), np.float64)
        P = lambda a: a.ctypes.data_as(_c_double_p)
        rc = self.lib.oracle_decode_batch(ctypes.byref(L), wp, B, P(st["S"]), P(st["z"]),
                                          P(st["wk"]), P(st["wv"]),
                                          st["pos"].ctypes.data_as(_c_int64_p), qp, kp, vp, P(out))
        if rc != 0:
            raise ValueError("oracle_decode_batch rejected its arguments")
        return out

    def state_from_history(self, Wf, k, v, p):
        """Recurrent-form state of one sequence after p tokens, built by direct
        sums plus the literal window (the last min(W, p) tokens)."""
        L = self.L
        S, z = self.state(Wf, k, v, p)
        W = L.window
        nwin = min(W, p)
        wk = np.zeros((L.n_kv_heads, W, L.head_dim))
        wv = np.zeros((L.n_kv_heads, W, L.head_dim))
        if nwin:
            wk[:, :nwin] = np.transpose(np.asarray(k, np.float64)[p - nwin:p], (1, 0, 2))
            wv[:, :nwin] = np.transpose(np.asarray(v, np.float64)[p - nwin:p], (1, 0, 2))
        return S, z, wk, wv
