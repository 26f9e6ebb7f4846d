"""GPU parity with the softmax feature map (GLIDE_PHI_SOFTMAX: phi(x) =
softmax(x Wf) over the Df features, the default kernel choice of Sec. III-B)
against the CPU oracle, through the C ABI: decode, chunked prefill (the key
rows' features spread over two or four waves), prefill then decode, a hybrid
form, the deferred fold, and the feature-map kernel alone."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_24788_amd import glide

from .gpu_util import Case, check, f64

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_decode_from_empty(dtype):
    case = Case([0, 1, 5, 33, 64], batch=2, Hq=8, Hkv=2, d=128, Df=128, dtype=dtype, seed=90, phi=2)
    q, k, v = case.tokens(70)
    st = case.new_state()
    out = case.decode_steps(st, q, k, v, 0, 70)
    case.check_decode(out, q, k, v, [0, 0], 70, "softmax-phi decode")
    case.check_state(st, k, v, [70, 70], "softmax-phi decode")


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("d,Df", [(128, 128), (64, 64), (128, 64)])
def test_prefill_ragged(dtype, d, Df):
    wins = [0, 1, 2, 31, 33, 65, 200]
    case = Case(wins, batch=3, Hq=8, Hkv=2, d=d, Df=Df, dtype=dtype, seed=91, phi=2)
    lens = [0, 37, 300]
    q, k, v = case.tokens(max(lens))
    st = case.new_state()
    outs = case.prefill(st, q, k, v, [0] * 3, lens)
    case.check_prefill(outs, q, k, v, [0] * 3, lens, "softmax-phi prefill")
    case.check_state(st, k, v, lens, "softmax-phi prefill")


@pytest.mark.parametrize("form", [0, 2])
def test_continuing_prefill_then_decode(form):
    case = Case([0, 3, 40, 129], batch=2, Hq=8, Hkv=2, d=128, Df=128, dtype=torch.bfloat16, seed=92, phi=2,
                form=form)
    n1, n2 = [20, 150], [70, 9]
    tot = [a + b for a, b in zip(n1, n2)]
    q, k, v = case.tokens(max(tot) + 8)
    st = case.new_state()
    case.prefill(st, q, k, v, [0] * 2, n1, chunk=32)
    outs = case.prefill(st, q, k, v, n1, n2, chunk=32)
    case.check_prefill(outs, q, k, v, n1, n2, f"softmax-phi form {form} continued")
    outs = []
    for step in range(8):
        qs = torch.stack([q[:, b, tot[b] + step] for b in range(2)], 1).contiguous()
        ks = torch.stack([k[:, b, tot[b] + step] for b in range(2)], 1).contiguous()
        vs = torch.stack([v[:, b, tot[b] + step] for b in range(2)], 1).contiguous()
        o = torch.empty_like(qs.cuda())
        case.g.decode_step(st, case.phi_w.cuda(), qs.cuda(), ks.cuda(), vs.cuda(), o, case.ws)
        outs.append(o)
    torch.cuda.synchronize()
    case.check_decode(torch.stack(outs, 2).cpu(), q, k, v, tot, 8, f"softmax-phi form {form} decode")
    case.check_state(st, k, v, [t + 8 for t in tot], f"softmax-phi form {form} after decode")


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_feature_map_kernel(dtype):
    d = Df = 128
    g = glide.Glide(1, 1, 4, 4, d, Df, [8], dtype=dtype, phi=glide.PHI_SOFTMAX)
    gen = torch.Generator().manual_seed(93)
    wf = (torch.randn(d, Df, generator=gen) * d ** -0.5).to(dtype)
    x = torch.randn(333, d, generator=gen).to(dtype)
    out = torch.empty(333, Df, dtype=dtype, device="cuda")
    g.feature_map(wf.cuda(), x.cuda(), out)
    torch.cuda.synchronize()
    want = oracle.Oracle(4, 4, d, Df, 8, phi=2).phi(f64(wf), f64(x))
    assert np.all(want > 0) and np.allclose(want.sum(-1), 1.0)
    check("softmax feature map", f64(out), want, dtype)


def test_deferred_fold_state_flush():
    """Decode from a prefilled state past several fold periods, then the
    flush: S and z hold the softmax features' sums over the linear part."""
    case = Case([0, 2, 17, 50], batch=2, Hq=16, Hkv=4, d=64, Df=64, dtype=torch.float32, seed=94, phi=2)
    lens = [45, 61]
    q, k, v = case.tokens(max(lens) + 21)
    st = case.new_state()
    case.prefill(st, q, k, v, [0] * 2, lens)
    outs = []
    for step in range(21):
        qs = torch.stack([q[:, b, lens[b] + step] for b in range(2)], 1).contiguous()
        ks = torch.stack([k[:, b, lens[b] + step] for b in range(2)], 1).contiguous()
        vs = torch.stack([v[:, b, lens[b] + step] for b in range(2)], 1).contiguous()
        o = torch.empty_like(qs.cuda())
        case.g.decode_step(st, case.phi_w.cuda(), qs.cuda(), ks.cuda(), vs.cuda(), o, case.ws)
        outs.append(o)
    torch.cuda.synchronize()
    case.check_decode(torch.stack(outs, 2).cpu(), q, k, v, lens, 21, "softmax-phi fold")
    case.check_state(st, k, v, [n + 21 for n in lens], "softmax-phi fold")
