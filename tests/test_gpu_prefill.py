"""GPU parity of glide_prefill against the CPU oracle (through the C ABI)."""
import pytest
import torch

from .gpu_util import Case

pytestmark = pytest.mark.gpu


def _prefill_from_empty(case, lens, chunk=0, label=""):
    n = max(lens)
    q, k, v = case.tokens(n)
    st = case.new_state()
    outs = case.prefill(st, q, k, v, [0] * case.B, lens, chunk=chunk)
    case.check_prefill(outs, q, k, v, [0] * case.B, lens, label)
    case.check_state(st, k, v, lens, label)
    return st, (q, k, v)


def test_single_layer_fp32_prefill_then_decode():
    """Single fp32 layer (4 = 4 heads, d = Df = 64, W = 64): 512 tokens
    prefilled, every output checked, then 16 decode steps."""
    case = Case([64], batch=1, Hq=4, Hkv=4, d=64, Df=64, dtype=torch.float32, seed=0)
    q, k, v = case.tokens(528)
    st = case.new_state()
    outs = case.prefill(st, q, k, v, [0], [512])
    case.check_prefill(outs, q, k, v, [0], [512], "fp32 prefill")
    case.check_state(st, k, v, [512], "fp32 prefill")
    out = case.decode_steps(st, q, k, v, 512, 528)
    case.check_decode(out, q, k, v, [512], 16, "fp32 decode after prefill")
    case.check_state(st, k, v, [528], "fp32 after decode")


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("d,Df", [(128, 128), (64, 64), (128, 64), (64, 128)])
def test_window_sweep_ragged(dtype, d, Df):
    """Windows around tile and chunk edges, three ragged sequences (one empty),
    GQA 4:1, all layers in one call."""
    wins = [0, 1, 2, 31, 32, 33, 65, 200]
    case = Case(wins, batch=3, Hq=8, Hkv=2, d=d, Df=Df, dtype=dtype, seed=11)
    _prefill_from_empty(case, [0, 37, 300], label=f"sweep {dtype} d={d} Df={Df}")


@pytest.mark.parametrize("chunk", [32, 96, 256])
def test_chunk_sizes(chunk):
    case = Case([0, 7, 64, 130], batch=2, Hq=8, Hkv=2, d=128, Df=128, dtype=torch.bfloat16, seed=12)
    _prefill_from_empty(case, [257, 130], chunk=chunk, label=f"chunk {chunk}")


@pytest.mark.parametrize("G", [1, 8, 16])
def test_group_sizes(G):
    case = Case([0, 5, 70], batch=2, Hq=2 * G, Hkv=2, d=128, Df=128, dtype=torch.bfloat16, seed=13)
    _prefill_from_empty(case, [90, 161], label=f"G={G}")


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_no_linear(dtype):
    case = Case([1, 9, 100], batch=2, Hq=8, Hkv=2, d=128, Df=128, dtype=dtype, linear=False, seed=14)
    _prefill_from_empty(case, [150, 33], label="no-linear")


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_continuing_prefill(dtype):
    """prefill(n1) then prefill(n2) from the reached state == the definition over
    n1 + n2 tokens (history from the ring feeds the band and the fold)."""
    case = Case([0, 3, 40, 129], batch=3, Hq=8, Hkv=2, d=128, Df=128, dtype=dtype, seed=15)
    n1 = [20, 0, 150]
    n2 = [70, 45, 9]
    q, k, v = case.tokens(max(a + b for a, b in zip(n1, n2)))
    st = case.new_state()
    case.prefill(st, q, k, v, [0] * 3, n1)
    outs = case.prefill(st, q, k, v, n1, n2)
    case.check_prefill(outs, q, k, v, n1, n2, "continued")
    case.check_state(st, k, v, [a + b for a, b in zip(n1, n2)], "continued")


def test_prefill_then_decode_bf16():
    case = Case([0, 16, 48, 100], batch=2, Hq=8, Hkv=2, d=128, Df=128, dtype=torch.bfloat16, seed=16)
    q, k, v = case.tokens(230)
    st = case.new_state()
    case.prefill(st, q, k, v, [0, 0], [200, 140])
    # decode both sequences from their (different) positions
    outs = []
    for step in range(30):
        qs = torch.stack([q[:, 0, 200 + step], q[:, 1, 140 + step]], 1).contiguous()
        ks = torch.stack([k[:, 0, 200 + step], k[:, 1, 140 + step]], 1).contiguous()
        vs = torch.stack([v[:, 0, 200 + step], v[:, 1, 140 + step]], 1).contiguous()
        o = torch.empty_like(qs).cuda()
        case.g.decode_step(st, case.phi_w.cuda(), qs.cuda(), ks.cuda(), vs.cuda(), o, case.ws)
        outs.append(o)
    out = torch.stack(outs, 2).cpu()
    case.check_decode(out, q, k, v, [200, 140], 30, "decode after prefill")
    case.check_state(st, k, v, [230, 170], "decode after prefill")


def test_sharp_logits_prefill():
    case = Case([0, 6, 50], batch=2, Hq=8, Hkv=2, d=128, Df=128, dtype=torch.bfloat16, seed=17, qkv_scale=0.5,
                v_scale=1.0)
    _prefill_from_empty(case, [120, 77], label="sharp")


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_prefill_after_decode(dtype):
    """prefill, decode a few steps (tokens left pending by deferred folding),
    then a continuing prefill: the pending tokens are folded first and the
    outputs still follow the definition over the whole history."""
    case = Case([0, 3, 40, 129], batch=2, Hq=8, Hkv=2, d=128, Df=128, dtype=dtype, seed=18)
    n1, m, n2 = [150, 61], 5, [40, 77]
    q, k, v = case.tokens(max(a + m + b for a, b in zip(n1, n2)))
    st = case.new_state()
    case.prefill(st, q, k, v, [0, 0], n1)
    outs = []
    phi = case.phi_w.cuda()
    for step in range(m):
        qs = torch.stack([q[:, b, n1[b] + step] for b in range(2)], 1).contiguous().cuda()
        ks = torch.stack([k[:, b, n1[b] + step] for b in range(2)], 1).contiguous().cuda()
        vs = torch.stack([v[:, b, n1[b] + step] for b in range(2)], 1).contiguous().cuda()
        o = torch.empty_like(qs)
        case.g.decode_step(st, phi, qs, ks, vs, o, case.ws)
        outs.append(o)
    case.check_decode(torch.stack(outs, 2).cpu(), q, k, v, n1, m, "decode between prefills")
    starts = [a + m for a in n1]
    outs = case.prefill(st, q, k, v, starts, n2)
    case.check_prefill(outs, q, k, v, starts, n2, "prefill after decode")
    case.check_state(st, k, v, [a + b for a, b in zip(starts, n2)], "prefill after decode")


def test_many_layers_two_launches():
    """70 layers, more than one launch takes: the layers are dealt over two
    launches by decreasing window, and every layer still matches the oracle."""
    wins = [(i * 37) % 97 for i in range(70)]
    case = Case(wins, batch=2, Hq=4, Hkv=2, d=64, Df=64, dtype=torch.bfloat16, seed=21)
    _prefill_from_empty(case, [70, 33], label="70 layers")


def _aligned_tokens(case, n, beta, c=4.0):
    """Keys near one direction u (per layer, sequence, head), queries beta*u:
    every score of a row has the sign of tau and magnitude ~ beta |u|^2 tau."""
    gen = torch.Generator().manual_seed(case.seed * 31 + 5)
    L, B, d = case.L, case.B, case.d
    u = torch.randn((L, B, 1, case.Hkv, d), generator=gen) * (c / d ** 0.5)
    k = u + 0.05 * torch.randn((L, B, n, case.Hkv, d), generator=gen) * (c / d ** 0.5)
    uq = u.repeat_interleave(case.Hq // case.Hkv, dim=3)
    q = beta * uq + 0.05 * torch.randn((L, B, n, case.Hq, d), generator=gen) * (c / d ** 0.5)
    v = torch.randn((L, B, n, case.Hkv, d), generator=gen)
    return q.to(case.dtype), k.to(case.dtype), v.to(case.dtype)


@pytest.mark.parametrize("sign", [-1.0, 1.0])
def test_extreme_score_frames(sign):
    """tau < 0 with aligned queries: every band score is ~ -140 in log2 units
    (the linear part's frame clamps at -60, the band's weight underflows
    against the linear part); tau > 0: the band dominates and the linear part
    vanishes.  Prefill, then decode steps, against the oracle."""
    case = Case([0, 1, 9, 70], batch=2, Hq=8, Hkv=2, d=128, Df=128, dtype=torch.bfloat16,
                tau=sign * 128 ** -0.5, seed=22)
    lens = [100, 61]
    q, k, v = _aligned_tokens(case, 110, beta=70.0)
    st = case.new_state()
    outs = case.prefill(st, q, k, v, [0, 0], lens)
    case.check_prefill(outs, q, k, v, [0, 0], lens, f"aligned tau sign {sign}")
    case.check_state(st, k, v, lens, f"aligned tau sign {sign}")
    phi = case.phi_w.cuda()
    outs = []
    for step in range(6):
        qs = torch.stack([q[:, b, lens[b] + step] for b in range(2)], 1).contiguous().cuda()
        ks = torch.stack([k[:, b, lens[b] + step] for b in range(2)], 1).contiguous().cuda()
        vs = torch.stack([v[:, b, lens[b] + step] for b in range(2)], 1).contiguous().cuda()
        o = torch.empty_like(qs)
        case.g.decode_step(st, phi, qs, ks, vs, o, case.ws)
        outs.append(o)
    case.check_decode(torch.stack(outs, 2).cpu(), q, k, v, lens, 6, f"aligned decode tau sign {sign}")


def test_zero_tau():
    """tau = 0: uniform softmax over the window, merged with the linear part."""
    case = Case([0, 3, 40], batch=1, Hq=4, Hkv=2, d=64, Df=64, dtype=torch.float32, tau=0.0, seed=23)
    _prefill_from_empty(case, [90], label="tau 0")


def test_batch_over_one_launch():
    """130 sequences (one launch takes 128): ragged lengths, empty ones among
    them, prefill then decode steps."""
    case = Case([0, 3, 40], batch=130, Hq=4, Hkv=2, d=64, Df=64, dtype=torch.bfloat16, seed=24)
    gen = torch.Generator().manual_seed(24)
    lens = [int(x) for x in torch.randint(0, 50, (130,), generator=gen)]
    lens[0], lens[129] = 0, 49
    q, k, v = case.tokens(max(lens) + 3)
    st = case.new_state()
    outs = case.prefill(st, q, k, v, [0] * 130, lens)
    case.check_prefill(outs, q, k, v, [0] * 130, lens, "B=130")
    case.check_state(st, k, v, lens, "B=130")
    phi = case.phi_w.cuda()
    step_out = []
    for step in range(3):
        qs = torch.stack([q[:, b, lens[b] + step] for b in range(130)], 1).contiguous().cuda()
        ks = torch.stack([k[:, b, lens[b] + step] for b in range(130)], 1).contiguous().cuda()
        vs = torch.stack([v[:, b, lens[b] + step] for b in range(130)], 1).contiguous().cuda()
        o = torch.empty_like(qs)
        case.g.decode_step(st, phi, qs, ks, vs, o, case.ws)
        step_out.append(o)
    case.check_decode(torch.stack(step_out, 2).cpu(), q, k, v, lens, 3, "B=130 decode")


def test_max_window():
    """W = 2^20, the largest window (ring and history buffers of 2^20 + 32
    slots): a short prefill is plain causal softmax, then decode steps."""
    case = Case([1 << 20, 0], batch=1, Hq=4, Hkv=2, d=64, Df=64, dtype=torch.bfloat16, seed=25)
    q, k, v = case.tokens(140)
    st = case.new_state()
    outs = case.prefill(st, q, k, v, [0], [130])
    case.check_prefill(outs, q, k, v, [0], [130], "W=2^20")
    out = case.decode_steps(st, q, k, v, 130, 140)
    case.check_decode(out, q, k, v, [130], 10, "W=2^20 decode")
    case.check_state(st, k, v, [140], "W=2^20")
