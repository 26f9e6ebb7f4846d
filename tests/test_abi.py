"""C-ABI checks that need no GPU: the library loads, exports every symbol
include/glide.h declares, sizes and layout follow the documented layout, and
every argument error is reported on the host before any HIP call (so these
run on a machine without a GPU)."""
import ctypes
import os
import re

import pytest
import torch

from paper_2607_24788_amd import glide

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "glide.h")


@pytest.fixture(scope="module")
def lib():
    return glide.load_library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(glide_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert len(names) >= 8
    for n in names:
        assert hasattr(lib, n), f"{n} declared in glide.h but not exported"
    assert sorted(glide.EXPORTS) == names


def test_missing_library_fails_loudly(tmp_path):
    with pytest.raises(RuntimeError, match="no fallback"):
        glide.load_library(str(tmp_path / "absent.so"))


def mk(**kw):
    p = dict(n_layers=3, batch=2, n_q_heads=8, n_kv_heads=2, head_dim=128, feat_dim=64,
             windows=[0, 5, 64], dtype=torch.bfloat16)
    p.update(kw)
    return glide.Glide(**p)


def align(x):
    return (x + 255) // 256 * 256


def expected_layout(B, Hkv, d, Df, windows, es, gated=False):
    """The documented layout (include/glide.h), computed independently."""
    off = 0
    out = []
    for W in windows:
        R = ((W + 8 + 31) // 32) * 32 if W > 0 else 0    # window + up to 8 pending tokens
        units = B * Hkv
        pos = off
        nf = pos + align(units * 8)
        cnt = nf + align(units * 8)
        S = cnt + align(units * 4)
        z = S + align(units * Df * d * 4)
        K = z + align(units * Df * 4)
        V = K + align(units * R * d * es)
        Gs = V + align(units * R * d * es)
        GR = Gs + (align(units * 16) if gated else 0)
        end = GR + (align(units * R * 8) if gated else 0)
        out.append(dict(pos=pos, nf=nf, cnt=cnt, S=S, z=z, K=K, V=V, G=Gs, GR=GR, R=R, bytes=end - off))
        off = end
    return out, off


@pytest.mark.parametrize("gated", [False, True])
@pytest.mark.parametrize("dtype,es", [(torch.bfloat16, 2), (torch.float32, 4)])
def test_layout_matches_documentation(dtype, es, gated):
    g = mk(dtype=dtype, n_layers=6, windows=[0, 1, 7, 8, 64, 4096], gated=gated)
    exp, total = expected_layout(2, 2, 128, 64, g.windows, es, gated)
    assert g.state_bytes() == total
    for l, e in enumerate(exp):
        lay = g.layout(l)
        assert (lay.pos_offset, lay.nf_offset, lay.cnt_offset, lay.s_offset, lay.z_offset, lay.kring_offset,
                lay.vring_offset, lay.gate_offset, lay.gring_offset) == (
                    e["pos"], e["nf"], e["cnt"], e["S"], e["z"], e["K"], e["V"], e["G"], e["GR"])
        assert lay.ring_slots == e["R"] and lay.window == g.windows[l]
        assert lay.layer_bytes == e["bytes"]
        assert lay.ring_slots == 0 or (lay.ring_slots % 32 == 0 and lay.ring_slots >= lay.window + 8)


def test_layer_views_cover_state():
    g = mk()
    st = torch.zeros(g.state_bytes(), dtype=torch.uint8)
    v = g.layer_views(st, 2)
    assert v["S"].shape == (2, 2, 64, 128) and v["kring_raw"].shape == (2, 2, 96 * 128)
    assert g.layer_views(st, 1)["ring_slots"] == 32      # W = 5: one 32-token block


@pytest.mark.parametrize("d", [64, 128])
def test_ring_layout_helpers(d):
    """The logical <-> fragment-major ring conversions follow the documented
    element positions and are inverses of each other."""
    R = 64
    logical = torch.arange(R * d, dtype=torch.float64).view(R, d)
    kr, vr = glide.kring_raw(logical, R, d), glide.vring_raw(logical, R, d)
    for s_ in (0, 1, 5, 31, 32, 45, 63):
        blk, o = divmod(s_, 32)
        for c in (0, 7, 8, 31, 33, d - 1):
            kpos = blk * 32 * d + ((((o // 4) % 2 * (d // 32) + c // 32) * 4 + (c // 8) % 4) * 16
                                   + 4 * (o // 8) + o % 4) * 8 + c % 8
            vpos = blk * 32 * d + ((c // 16 * 4 + o // 8) * 16 + c % 16) * 8 + o % 8
            assert kr[kpos] == logical[s_, c] and vr[vpos] == logical[s_, c]
    assert torch.equal(glide.kring_logical(kr, R, d), logical)
    assert torch.equal(glide.vring_logical(vr, R, d), logical)


BAD_CFGS = [
    (dict(n_q_heads=6, n_kv_heads=4), glide.GlideError, -2),          # Hq % Hkv != 0
    (dict(windows=[0, -1, 3]), None, -2),                             # negative window
    (dict(windows=[0, 5, (1 << 20) + 1]), None, -2),                  # window too large
    (dict(linear=False), None, -2),                                   # W = 0 with no linear part
    (dict(head_dim=96), None, -3),                                    # unsupported d
    (dict(feat_dim=32), None, -3),                                    # unsupported Df
    (dict(n_q_heads=34, n_kv_heads=2), None, -3),                     # G = 17 > 16
    (dict(batch=0), None, -2),
    (dict(dtype=torch.float16), None, -2),                            # unknown element type
    (dict(form=3), None, -2),                                         # unknown flag bits
    (dict(phi=3), None, -2),                                          # unknown feature map
    (dict(windows=[1, 5, 3], linear=False, form=1), None, -2),        # hybrid form without a linear part
]


def test_hybrid_flag_combinations():
    """The state over every token only comes with the separately normalised
    sum; neither hybrid flag combines with the linear part switched off."""
    ok = mk(windows=[1, 5, 3])
    for flags, code in ((glide.HYBRID_SUM, 0), (glide.HYBRID_SUM | glide.HYBRID_STATE_ALL, 0),
                        (glide.HYBRID_STATE_ALL, -2), (glide.NO_LINEAR | glide.HYBRID_SUM, -2),
                        (glide.PER_HEAD_PHI, 0), (glide.PER_HEAD_PHI | glide.HYBRID_SUM, 0),
                        (glide.GATED, 0), (glide.GATED | glide.PER_HEAD_PHI, 0),
                        (glide.GATED | glide.NO_LINEAR, -2), (glide.GATED | glide.HYBRID_SUM, -3),
                        (32, -2)):
        ok.cfg.flags = flags
        assert (ok.state_bytes() > 0) == (code == 0), flags
        if code:  # rejected before any HIP call (the pointer is never used)
            s = ok.lib.glide_state_init(ctypes.byref(ok.cfg), ctypes.c_void_p(256), 1 << 30, None)
            assert s == code, flags


@pytest.mark.parametrize("kw,_e,code", BAD_CFGS)
def test_invalid_configs_rejected(kw, _e, code):
    g = mk(**kw)
    assert g.state_bytes() == 0
    assert g.workspace_bytes(100) == 0
    st = torch.zeros(1024, dtype=torch.uint8)
    s = g.lib.glide_state_init(ctypes.byref(g.cfg), ctypes.c_void_p(256), 1 << 30, None)
    assert s == code
    del st


def test_null_arguments(lib):
    assert lib.glide_state_bytes(None) == 0
    assert lib.glide_state_init(None, None, 0, None) == -1
    g = mk()
    assert g.lib.glide_state_init(ctypes.byref(g.cfg), None, g.state_bytes(), None) == -1
    cfg = glide.Config(g.cfg.n_layers, 2, 8, 2, 128, 64, 1, 0, 0, 0.1, None)
    assert lib.glide_state_bytes(ctypes.byref(cfg)) == 0
    out = glide.LayerLayout()
    assert lib.glide_state_layout(ctypes.byref(g.cfg), 0, None) == -1
    assert lib.glide_state_layout(ctypes.byref(g.cfg), 3, ctypes.byref(out)) == -2
    assert lib.glide_state_layout(ctypes.byref(g.cfg), -1, ctypes.byref(out)) == -2


def _decode(g, state=256, size=None, layer0=0, n=1, ptrs=(4096,) * 5, ws=1 << 20, ws_bytes=None, gates=None):
    size = g.state_bytes() if size is None else size
    ws_bytes = g.workspace_bytes(0) if ws_bytes is None else ws_bytes
    P = [ctypes.c_void_p(x) if x is not None else None for x in ptrs]
    return g.lib.glide_decode_step(ctypes.byref(g.cfg), ctypes.c_void_p(state) if state else None, size,
                                   layer0, n, P[0], P[1], P[2], P[3], ctypes.c_void_p(gates) if gates else None,
                                   P[4], ctypes.c_void_p(ws) if ws else None, ws_bytes, None)


def test_decode_argument_errors():
    """All of these return before the first HIP call (no GPU here)."""
    g = mk()
    assert _decode(g, state=None) == -1
    assert _decode(g, state=128 + 8) == -4                      # state not 256-aligned
    assert _decode(g, size=g.state_bytes() - 1) == -5
    assert _decode(g, layer0=3) == -2
    assert _decode(g, layer0=2, n=2) == -2
    assert _decode(g, n=0) == -2
    assert _decode(g, layer0=-1) == -2
    assert _decode(g, ptrs=(4096, None, 4096, 4096, 4096)) == -1
    assert _decode(g, ptrs=(4096, 4096, 4096 + 2, 4096, 4096)) == -4   # q misaligned
    assert _decode(g, ptrs=(4096, 4096, 4096, 4096, 4104)) == -4       # out misaligned
    # few units and a long window: the window split needs the workspace for
    # its partial records (checked before anything is launched)
    gs = mk(windows=[0, 5, 300])
    assert gs.workspace_bytes(0) > 256
    assert _decode(gs, ws=None) == -1
    assert _decode(gs, ws=(1 << 20) + 16) == -4
    assert _decode(gs, ws_bytes=gs.workspace_bytes(0) - 1) == -5



def _flush(g, state=256, size=None, layer0=0, n=1, phi=4096):
    size = g.state_bytes() if size is None else size
    return g.lib.glide_state_flush(ctypes.byref(g.cfg), ctypes.c_void_p(state) if state else None, size, layer0, n,
                                   ctypes.c_void_p(phi) if phi else None, None)


def test_flush_argument_errors():
    g = mk()
    assert _flush(g, state=None) == -1
    assert _flush(g, state=128) == -4
    assert _flush(g, size=g.state_bytes() - 1) == -5
    assert _flush(g, layer0=2, n=2) == -2
    assert _flush(g, phi=None) == -1
    assert _flush(g, phi=4096 + 4) == -4
    assert _flush(mk(linear=False, windows=[1, 5, 64])) == 0     # nothing to fold, nothing enqueued


def test_workspace_sizes():
    # 12 units, one long window: split windows, one partial record
    # (G x (2d + 3) floats) per workgroup
    g = mk(n_layers=3, batch=2, n_q_heads=8, n_kv_heads=2, feat_dim=64, windows=[0, 5, 300])
    rec = 4 * (2 * 128 + 3) * 4
    assert g.workspace_bytes(0) >= 3 * 2 * 2 * rec
    assert g.workspace_bytes(0) <= 3 * 2 * 2 * 16 * rec + 256
    # a layer with as many units as any device holds resident decode
    # workgroups (1024): nothing is ever split, no decode workspace
    big = mk(n_layers=4, batch=128, n_q_heads=16, n_kv_heads=8, windows=[0, 5, 64, 100])
    assert big.workspace_bytes(0) == 256
    assert g.workspace_bytes(100000) > g.workspace_bytes(10)
    # a window of fewer than 10 tiles of 32 tokens (window + 1 tile) is never
    # split, whatever the batch: no partial records
    assert mk(n_layers=3, batch=1, windows=[0, 5, 255]).workspace_bytes(0) == 256
    assert mk(n_layers=3, batch=1, windows=[0, 5, 288]).workspace_bytes(0) > 256
    # a split gives every piece 4 tiles or more: a 10-tile window at most 2
    # pieces per unit (12 units here: B=2 x 2 KV heads x 3 layers)
    w10 = mk(n_layers=3, batch=2, n_q_heads=8, n_kv_heads=2, windows=[288, 288, 288])
    assert w10.workspace_bytes(0) <= align(2 * 12 * 4 * (2 * 128 + 3) * 4)


def _prefill(g, cu, total, chunk=0, ws_bytes=None, state=256, ptrs=(4096,) * 6, gates=None):
    arr = (ctypes.c_int32 * len(cu))(*cu)
    ws_bytes = g.workspace_bytes(total) if ws_bytes is None else ws_bytes
    P = [ctypes.c_void_p(x) if x is not None else None for x in ptrs]
    return g.lib.glide_prefill(ctypes.byref(g.cfg), ctypes.c_void_p(state), g.state_bytes(), 0, 1, P[0], P[1],
                               P[2], P[3], ctypes.c_void_p(gates) if gates else None, arr, total, chunk, P[4],
                               P[5], ws_bytes, None)


def test_prefill_argument_errors():
    g = mk()
    assert _prefill(g, [0, 5, 3], 3) == -2              # decreasing
    assert _prefill(g, [1, 2, 3], 3) == -2              # cu[0] != 0
    assert _prefill(g, [0, 2, 3], 4) == -2              # cu[B] != total
    assert _prefill(g, [0, 2, 3], 3, chunk=48) == -2    # chunk not a multiple of 32
    assert _prefill(g, [0, 2, 3], 3, chunk=512) == -2   # chunk too large
    assert _prefill(g, [0, 2, 3], 3, ws_bytes=0) == -5  # workspace too small
    assert _prefill(g, [0, 2, 3], 3, ptrs=(4096, 4096, 4096, None, 4096, 4096)) == -1


def test_binding_checks_cu_length():
    g = mk()
    with pytest.raises(ValueError, match="batch \\+ 1"):
        g.prefill(None, None, None, None, None, [0, 3], None, None)


def test_feature_map_argument_errors():
    g = mk()
    cfgp = ctypes.byref(g.cfg)
    assert g.lib.glide_feature_map(cfgp, None, ctypes.c_void_p(4096), 4, ctypes.c_void_p(4096), None) == -1
    assert g.lib.glide_feature_map(cfgp, ctypes.c_void_p(4096), ctypes.c_void_p(4096), -1,
                                   ctypes.c_void_p(4096), None) == -2
    assert g.lib.glide_feature_map(cfgp, ctypes.c_void_p(4098), ctypes.c_void_p(4096), 4,
                                   ctypes.c_void_p(4096), None) == -4


def test_status_strings(lib):
    for code in glide.STATUS:
        assert lib.glide_status_string(code)


def test_noalloc_decode_rejects_before_any_hip_call():
    """glide_decode_step_noalloc validates on the host: a config whose decode
    workspace exceeds the fixed scratch gets GLIDE_ERR_SCRATCH, other errors
    the codes glide_decode_step gives (no HIP call is made)."""
    P = [ctypes.c_void_p(4096)] * 5

    def call(g, state=256, n=1):
        return g.lib.glide_decode_step_noalloc(ctypes.byref(g.cfg), ctypes.c_void_p(state) if state else None,
                                               g.state_bytes(), 0, n, *P[:4], None, P[4], None)
    # G = 16 at d = 128, few units and huge windows: 1024 records of 16 x 259 floats > 16 MiB
    big = mk(n_layers=3, batch=32, n_q_heads=16, n_kv_heads=1, windows=[1 << 20] * 3)
    assert big.workspace_bytes(0) > glide.DECODE_SCRATCH_BYTES
    assert call(big) == -7
    assert "scratch" in big.lib.glide_status_string(-7).decode()
    g = mk()
    assert g.workspace_bytes(0) <= glide.DECODE_SCRATCH_BYTES
    assert call(g, state=None) == -1
    assert call(g, state=260) == -4
    assert call(g, n=4) == -2
    assert g.lib.glide_decode_step_noalloc(ctypes.byref(g.cfg), ctypes.c_void_p(256), g.state_bytes(), 0, 1,
                                           None, *P[1:4], None, P[4], None) == -1


def test_binding_refuses_tensors_the_kernels_would_overrun():
    """The binding checks every tensor before the ctypes call (device,
    contiguous, element type, size): the library sees raw pointers only."""
    g = mk()
    t = lambda *shape, dt=torch.bfloat16: torch.zeros(shape, dtype=dt)
    args = (t(16, dt=torch.uint8), t(3, 128, 64), t(3, 2, 8, 128), t(3, 2, 2, 128), t(3, 2, 2, 128),
            t(3, 2, 8, 128))
    with pytest.raises(ValueError, match="device tensor"):
        g.decode_step(*args)
    with pytest.raises(ValueError, match="device tensor"):
        g.prefill(args[0], args[1], t(3, 5, 8, 128), t(3, 5, 2, 128), t(3, 5, 2, 128), [0, 2, 5],
                  t(3, 5, 8, 128), t(256, dt=torch.uint8))
    with pytest.raises(ValueError, match="device tensor"):
        g.feature_map(t(128, 64), t(4, 128), t(4, 64))


def test_gate_arguments():
    """log_gates: required (and 4-byte aligned) exactly when the stack is
    gated; rejected before any HIP call otherwise."""
    ug, gg = mk(), mk(gated=True)
    assert _decode(ug, gates=8192) == -2          # gates for an ungated stack
    assert _decode(gg) == -1                      # gated without gates
    assert _decode(gg, gates=8194) == -4          # misaligned
    assert _prefill(ug, [0, 2, 3], 3, gates=8192) == -2
    assert _prefill(gg, [0, 2, 3], 3) == -1
    assert _prefill(gg, [0, 2, 3], 3, gates=8194) == -4
