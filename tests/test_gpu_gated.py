"""GPU parity of the gated (GLA-style) linear state (GLIDE_GATED; the gating
Sec. III-B names among the linear forms, read as one scalar log-gate per
token and KV head, every linear-set token decayed by the gates after it)
against the oracle's gated definition and gated state, in fp32 and bf16:
decode from empty across fold steps and window edges, chunked prefill of
ragged batches, prefill then decode, continuing prefill, prefill after
decode steps (pending tokens folded with their decay), the split and the
unsplit decode path, strong gates, and the other feature maps."""
import pytest
import torch

from .gpu_util import Case

pytestmark = pytest.mark.gpu

WINDOWS = [0, 1, 5, 64, 300]


@pytest.mark.parametrize("dtype,d", [(torch.float32, 64), (torch.bfloat16, 128)])
def test_gated_decode_from_empty(dtype, d):
    case = Case(WINDOWS, batch=2, Hq=8, Hkv=2, d=d, Df=d, dtype=dtype, seed=41, gated=True)
    n = 330
    q, k, v = case.tokens(n)
    gates = case.log_gates(n)
    st = case.new_state()
    out = case.decode_steps(st, q, k, v, 0, n, gates=gates)
    case.check_decode(out, q, k, v, [0, 0], n, "gated decode", gates=gates)
    case.check_state(st, k, v, [n, n], "gated decode", gates=gates)


@pytest.mark.parametrize("chunk", [32, 64, 96])
@pytest.mark.parametrize("dtype,d", [(torch.float32, 64), (torch.bfloat16, 128)])
def test_gated_prefill_then_decode(dtype, d, chunk):
    case = Case(WINDOWS, batch=3, Hq=8, Hkv=2, d=d, Df=d, dtype=dtype, seed=43, gated=True)
    lens, nd = [333, 150, 0], 20
    q, k, v = case.tokens(max(lens) + nd)
    gates = case.log_gates(max(lens) + nd)
    st = case.new_state()
    outs = case.prefill(st, q, k, v, [0, 0, 0], lens, chunk=chunk, gates=gates)
    case.check_prefill(outs, q, k, v, [0, 0, 0], lens, f"gated prefill C={chunk}", gates=gates)
    case.check_state(st, k, v, lens, "gated after prefill", gates=gates)
    phi = case.phi_w.cuda()
    dout = []
    for s in range(nd):
        sel = lambda x: torch.stack([x[:, b, lens[b] + s] for b in range(case.B)], 1).contiguous().cuda()
        o = torch.empty((case.L, case.B, case.Hq, case.d), dtype=dtype, device="cuda")
        case.g.decode_step(st, phi, sel(q), sel(k), sel(v), o, case.ws, log_gates=sel(gates))
        dout.append(o)
    torch.cuda.synchronize()
    case.check_decode(torch.stack(dout, 2).cpu(), q, k, v, lens, nd, "gated decode after prefill", gates=gates)
    case.check_state(st, k, v, [x + nd for x in lens], "gated after decode", gates=gates)


def test_gated_continuing_prefill_and_prefill_after_decode():
    case = Case(WINDOWS, batch=2, Hq=8, Hkv=2, d=128, Df=128, dtype=torch.bfloat16, seed=47, gated=True)
    q, k, v = case.tokens(520)
    gates = case.log_gates(520)
    st = case.new_state()
    outs = case.prefill(st, q, k, v, [0, 0], [100, 57], gates=gates)
    case.check_prefill(outs, q, k, v, [0, 0], [100, 57], "gated first prefill", gates=gates)
    outs = case.prefill(st, q, k, v, [100, 57], [120, 200], gates=gates)
    case.check_prefill(outs, q, k, v, [100, 57], [120, 200], "gated continuing prefill", gates=gates)
    case.check_state(st, k, v, [220, 257], "gated continuing prefill", gates=gates)
    # 13 decode steps leave tokens pending; a prefill folds them (decayed) first
    phi = case.phi_w.cuda()
    pos = [220, 257]
    for s in range(13):
        sel = lambda x: torch.stack([x[:, b, pos[b] + s] for b in range(2)], 1).contiguous().cuda()
        o = torch.empty((case.L, 2, case.Hq, case.d), dtype=case.dtype, device="cuda")
        case.g.decode_step(st, phi, sel(q), sel(k), sel(v), o, case.ws, log_gates=sel(gates))
    pos = [x + 13 for x in pos]
    case.check_state(st, k, v, pos, "gated after decode", gates=gates)
    outs = case.prefill(st, q, k, v, pos, [90, 33], gates=gates)
    case.check_prefill(outs, q, k, v, pos, [90, 33], "gated prefill after decode", gates=gates)
    case.check_state(st, k, v, [pos[0] + 90, pos[1] + 33], "gated prefill after decode", gates=gates)


def test_gated_state_every_decode_step():
    """nf in [beta - 8, beta], S and z the gated sums over [0, nf) decayed to
    the folding step, G_cur, G_f and the gate ring, after every step."""
    case = Case([0, 3, 40], batch=2, Hq=8, Hkv=2, d=64, Df=64, dtype=torch.float32, seed=53, gated=True)
    q, k, v = case.tokens(80)
    gates = case.log_gates(80)
    st = case.new_state()
    case.prefill(st, q, k, v, [0, 0], [50, 23], gates=gates)
    phi = case.phi_w.cuda()
    for step in range(18):
        sel = lambda x, t: torch.stack([x[:, 0, 50 + t], x[:, 1, 23 + t]], 1).contiguous().cuda()
        o = torch.empty((case.L, 2, case.Hq, case.d), dtype=case.dtype, device="cuda")
        case.g.decode_step(st, phi, sel(q, step), sel(k, step), sel(v, step), o, case.ws,
                           log_gates=sel(gates, step))
        torch.cuda.synchronize()
        case.check_state(st, k, v, [51 + step, 24 + step], f"gated step {step}", gates=gates)


def test_gated_split_and_unsplit_decode():
    """Few units (long windows split over workgroups, merged by the last
    piece) and 1024 units per layer (one workgroup each)."""
    for B, Hkv, lens in ((1, 2, [333]), (128, 8, [(37 * i) % 350 for i in range(128)])):
        case = Case([0, 5, 40, 300], batch=B, Hq=2 * Hkv, Hkv=Hkv, d=64, Df=64, dtype=torch.bfloat16, seed=59,
                    gated=True)
        n = 6
        q, k, v = case.tokens(max(lens) + n)
        gates = case.log_gates(max(lens) + n)
        st = case.new_state()
        case.prefill(st, q, k, v, [0] * B, lens, gates=gates)
        phi = case.phi_w.cuda()
        outs = []
        for s in range(n):
            sel = lambda x: torch.stack([x[:, b, lens[b] + s] for b in range(B)], 1).contiguous().cuda()
            o = torch.empty((case.L, B, case.Hq, case.d), dtype=case.dtype, device="cuda")
            case.g.decode_step(st, phi, sel(q), sel(k), sel(v), o, case.ws if B == 1 else None,
                               log_gates=sel(gates))
            outs.append(o)
        torch.cuda.synchronize()
        case.check_decode(torch.stack(outs, 2).cpu(), q, k, v, lens, n, f"gated B={B}", gates=gates)
        case.check_state(st, k, v, [x + n for x in lens], f"gated B={B}", gates=gates)


def test_gated_strong_gates():
    """Log-gates down to -3 per token: decays span hundreds of e-folds inside a
    chunk, and every factor the kernels form stays <= 1."""
    case = Case(WINDOWS, batch=2, Hq=4, Hkv=2, d=64, Df=64, dtype=torch.float32, seed=61, gated=True, gate_lo=-3.0)
    lens = [260, 131]
    q, k, v = case.tokens(max(lens) + 12)
    gates = case.log_gates(max(lens) + 12)
    st = case.new_state()
    outs = case.prefill(st, q, k, v, [0, 0], lens, gates=gates)
    case.check_prefill(outs, q, k, v, [0, 0], lens, "strong gates prefill", gates=gates)
    phi = case.phi_w.cuda()
    dout = []
    for s in range(12):
        sel = lambda x: torch.stack([x[:, b, lens[b] + s] for b in range(2)], 1).contiguous().cuda()
        o = torch.empty((case.L, 2, case.Hq, case.d), dtype=case.dtype, device="cuda")
        case.g.decode_step(st, phi, sel(q), sel(k), sel(v), o, case.ws, log_gates=sel(gates))
        dout.append(o)
    torch.cuda.synchronize()
    case.check_decode(torch.stack(dout, 2).cpu(), q, k, v, lens, 12, "strong gates decode", gates=gates)
    case.check_state(st, k, v, [x + 12 for x in lens], "strong gates", gates=gates)


@pytest.mark.parametrize("phi,per_head", [(1, False), (2, False), (0, True)])
def test_gated_with_other_feature_maps(phi, per_head):
    case = Case([0, 7, 70], batch=2, Hq=8, Hkv=2, d=64, Df=64, dtype=torch.float32, seed=67, gated=True, phi=phi,
                per_head_phi=per_head)
    lens = [150, 97]
    q, k, v = case.tokens(max(lens) + 10)
    gates = case.log_gates(max(lens) + 10)
    st = case.new_state()
    outs = case.prefill(st, q, k, v, [0, 0], lens, gates=gates)
    case.check_prefill(outs, q, k, v, [0, 0], lens, f"gated phi={phi} per_head={per_head}", gates=gates)
    phi_w = case.phi_w.cuda()
    dout = []
    for s in range(10):
        sel = lambda x: torch.stack([x[:, b, lens[b] + s] for b in range(2)], 1).contiguous().cuda()
        o = torch.empty((case.L, 2, case.Hq, case.d), dtype=case.dtype, device="cuda")
        case.g.decode_step(st, phi_w, sel(q), sel(k), sel(v), o, case.ws, log_gates=sel(gates))
        dout.append(o)
    torch.cuda.synchronize()
    case.check_decode(torch.stack(dout, 2).cpu(), q, k, v, lens, 10, f"gated decode phi={phi}", gates=gates)
    case.check_state(st, k, v, [x + 10 for x in lens], f"gated phi={phi}", gates=gates)
