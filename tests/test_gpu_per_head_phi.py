"""GPU parity with one feature-map matrix per KV head (GLIDE_PER_HEAD_PHI:
phi_w [n_layers][Hkv][d][Df], head g's matrix for its group's queries and its
keys) against the CPU oracle, through the C ABI: decode (split and unsplit
launches, per-layer calls), chunked prefill, prefill then decode, with each
feature map and a hybrid form."""
import pytest
import torch

from .gpu_util import Case

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("phi", [0, 1, 2])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_decode_from_empty(phi, dtype):
    case = Case([0, 1, 5, 33, 70], batch=2, Hq=8, Hkv=4, d=128, Df=128, dtype=dtype, seed=100 + phi, phi=phi,
                per_head_phi=True)
    q, k, v = case.tokens(75)
    st = case.new_state()
    out = case.decode_steps(st, q, k, v, 0, 75)
    case.check_decode(out, q, k, v, [0, 0], 75, f"per-head phi {phi} decode")
    case.check_state(st, k, v, [75, 75], f"per-head phi {phi} decode")


@pytest.mark.parametrize("phi", [0, 2])
@pytest.mark.parametrize("d,Df", [(128, 128), (64, 64)])
def test_prefill_ragged(phi, d, Df):
    case = Case([0, 2, 31, 65, 200], batch=3, Hq=8, Hkv=2, d=d, Df=Df, dtype=torch.bfloat16, seed=110 + phi,
                phi=phi, per_head_phi=True)
    lens = [0, 41, 290]
    q, k, v = case.tokens(max(lens))
    st = case.new_state()
    outs = case.prefill(st, q, k, v, [0] * 3, lens)
    case.check_prefill(outs, q, k, v, [0] * 3, lens, f"per-head phi {phi} prefill")
    case.check_state(st, k, v, lens, f"per-head phi {phi} prefill")


@pytest.mark.parametrize("form", [0, 1])
def test_prefill_then_decode(form):
    case = Case([0, 3, 40, 129, 330], batch=2, Hq=16, Hkv=4, d=128, Df=128, dtype=torch.bfloat16, seed=120 + form,
                form=form, per_head_phi=True)
    lens = [400, 37]
    q, k, v = case.tokens(max(lens) + 10)
    st = case.new_state()
    case.prefill(st, q, k, v, [0] * 2, lens, chunk=32)
    phi = case.phi_w.cuda()
    outs = []
    for step in range(10):
        sel = lambda x: torch.stack([x[:, b, lens[b] + step] for b in range(2)], 1).contiguous().cuda()
        qs, ks, vs = sel(q), sel(k), sel(v)
        o = torch.empty_like(qs)
        for l in range(case.L):  # per-layer calls: each plans its own split
            case.g.decode_step(st, phi[l:l + 1], qs[l:l + 1], ks[l:l + 1], vs[l:l + 1], o[l:l + 1], case.ws,
                               layer0=l, n_layers=1)
        outs.append(o)
    torch.cuda.synchronize()
    case.check_decode(torch.stack(outs, 2).cpu(), q, k, v, lens, 10, f"per-head form {form} decode")
    case.check_state(st, k, v, [n + 10 for n in lens], f"per-head form {form} after decode")
