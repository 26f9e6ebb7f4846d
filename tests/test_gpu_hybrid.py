"""GPU parity of the Appendix's two hybrid forms against the CPU oracle,
through the C ABI: form 1 = GLIDE_HYBRID_SUM (the window's softmax output plus
the linear part's own normalised output, state over the evicted tokens),
form 2 = GLIDE_HYBRID_SUM | GLIDE_HYBRID_STATE_ALL (the same sum, state over
every token)."""
import pytest
import torch

from .gpu_util import Case

pytestmark = pytest.mark.gpu

FORMS = [1, 2]


@pytest.mark.parametrize("form", FORMS)
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_decode_from_empty(form, dtype):
    """70 decode steps from an empty state, every output and the final state
    checked; few units, so the long window (330) is split over workgroups."""
    case = Case([0, 1, 5, 33, 64, 330], batch=2, Hq=8, Hkv=2, d=128, Df=128, dtype=dtype, seed=40 + form, form=form)
    q, k, v = case.tokens(70)
    st = case.new_state()
    out = case.decode_steps(st, q, k, v, 0, 70)
    case.check_decode(out, q, k, v, [0, 0], 70, f"form {form} decode")
    case.check_state(st, k, v, [70, 70], f"form {form} decode")


@pytest.mark.parametrize("form", FORMS)
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("d,Df", [(128, 128), (64, 64)])
def test_prefill_ragged(form, dtype, d, Df):
    """Windows around tile and chunk edges, three ragged sequences (one empty)."""
    wins = [0, 1, 2, 31, 33, 65, 200]
    case = Case(wins, batch=3, Hq=8, Hkv=2, d=d, Df=Df, dtype=dtype, seed=50 + form, form=form)
    lens = [0, 37, 300]
    q, k, v = case.tokens(max(lens))
    st = case.new_state()
    outs = case.prefill(st, q, k, v, [0] * 3, lens)
    case.check_prefill(outs, q, k, v, [0] * 3, lens, f"form {form} prefill")
    case.check_state(st, k, v, lens, f"form {form} prefill")


@pytest.mark.parametrize("form", FORMS)
@pytest.mark.parametrize("chunk", [32, 256])
def test_prefill_chunks(form, chunk):
    case = Case([0, 7, 64, 130], batch=2, Hq=8, Hkv=2, d=128, Df=128, dtype=torch.bfloat16, seed=55 + form,
                form=form)
    lens = [257, 130]
    q, k, v = case.tokens(max(lens))
    st = case.new_state()
    outs = case.prefill(st, q, k, v, [0] * 2, lens, chunk=chunk)
    case.check_prefill(outs, q, k, v, [0] * 2, lens, f"form {form} chunk {chunk}")
    case.check_state(st, k, v, lens, f"form {form} chunk {chunk}")


@pytest.mark.parametrize("form", FORMS)
def test_continuing_prefill_then_decode(form):
    """prefill(n1), prefill(n2) from the reached state, then decode steps at
    ragged positions (the 330 window split over workgroups, with a linear
    part): every output and the state against the definition."""
    case = Case([0, 3, 40, 129, 330], batch=3, Hq=8, Hkv=2, d=128, Df=128, dtype=torch.bfloat16, seed=60 + form,
                form=form)
    n1 = [20, 0, 350]
    n2 = [70, 45, 9]
    tot = [a + b for a, b in zip(n1, n2)]
    q, k, v = case.tokens(max(tot) + 12)
    st = case.new_state()
    case.prefill(st, q, k, v, [0] * 3, n1)
    outs = case.prefill(st, q, k, v, n1, n2)
    case.check_prefill(outs, q, k, v, n1, n2, f"form {form} continued")
    case.check_state(st, k, v, tot, f"form {form} continued")
    # ragged decode: every sequence takes 12 more steps from its own position
    outs = []
    for step in range(12):
        qs = torch.stack([q[:, b, tot[b] + step] for b in range(3)], 1).contiguous()
        ks = torch.stack([k[:, b, tot[b] + step] for b in range(3)], 1).contiguous()
        vs = torch.stack([v[:, b, tot[b] + step] for b in range(3)], 1).contiguous()
        o = torch.empty_like(qs.cuda())
        case.g.decode_step(st, case.phi_w.cuda(), qs.cuda(), ks.cuda(), vs.cuda(), o, case.ws)
        outs.append(o)
    torch.cuda.synchronize()
    out = torch.stack(outs, 2).cpu()
    case.check_decode(out, q, k, v, tot, 12, f"form {form} decode after prefill")
    case.check_state(st, k, v, [t + 12 for t in tot], f"form {form} after decode")


@pytest.mark.parametrize("form", FORMS)
def test_unsplit_decode(form):
    """Enough units that no window is split (the in-workgroup merge)."""
    case = Case([6, 40], batch=128, Hq=8, Hkv=2, d=128, Df=128, dtype=torch.bfloat16, seed=70 + form, form=form)
    lens = [(17 * b) % 90 for b in range(128)]
    q, k, v = case.tokens(max(lens) + 3)
    st = case.new_state()
    case.prefill(st, q, k, v, [0] * 128, lens)
    outs = []
    for step in range(3):
        qs = torch.stack([q[:, b, lens[b] + step] for b in range(128)], 1).contiguous()
        ks = torch.stack([k[:, b, lens[b] + step] for b in range(128)], 1).contiguous()
        vs = torch.stack([v[:, b, lens[b] + step] for b in range(128)], 1).contiguous()
        o = torch.empty_like(qs.cuda())
        case.g.decode_step(st, case.phi_w.cuda(), qs.cuda(), ks.cuda(), vs.cuda(), o, case.ws)
        outs.append(o)
    torch.cuda.synchronize()
    out = torch.stack(outs, 2).cpu()
    case.check_decode(out, q, k, v, lens, 3, f"form {form} unsplit decode")
    case.check_state(st, k, v, [n + 3 for n in lens], f"form {form} unsplit")
