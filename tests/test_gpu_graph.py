"""Decode steps captured in a HIP graph, one library call per layer, against
the same calls made eagerly (through the C ABI).

The decode kernels take their split-merge counters from the state and leave
them at zero, and the calls enqueue no memset, so a captured sequence of
steps can be replayed from a restored state.  Every replay is checked, with
eager work and synchronisations between replays.
"""
import pytest
import torch

from .gpu_util import Case

pytestmark = pytest.mark.gpu


def _per_layer(case, st, phi, qs, ks, vs, out):
    for s in range(qs.shape[0]):
        for l in range(case.L):
            case.g.decode_step(st, phi[l:l + 1], qs[s, l:l + 1], ks[s, l:l + 1], vs[s, l:l + 1], out[s, l:l + 1],
                               case.ws, layer0=l, n_layers=1)


def _eager(case, st, phi, qs, ks, vs):
    out = torch.empty_like(qs)
    _per_layer(case, st, phi, qs, ks, vs, out)
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_graph_per_layer_decode_matches_eager(dtype):
    d = 128 if dtype == torch.bfloat16 else 64
    case = Case([3, 0, 40, 9, 330], batch=3, Hq=8, Hkv=2, d=d, Df=d, dtype=dtype, seed=8)
    n0, n = 20, 24
    q, k, v = case.tokens(n0 + n)
    phi = case.phi_w.cuda()
    st = case.new_state()
    case.decode_steps(st, q, k, v, 0, n0)
    snap = st.clone()

    # resident inputs of the captured steps: [n][L][B][H][d]
    qs, ks, vs = (x[:, :, n0:].permute(2, 0, 1, 3, 4).contiguous().cuda() for x in (q, k, v))
    want = _eager(case, st, phi, qs, ks, vs)
    want_state = st.clone()

    gst = snap.clone()
    gout = torch.empty_like(qs)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        _per_layer(case, gst, phi, qs, ks, vs, gout)
    torch.cuda.synchronize()
    # capture records the calls without running them
    assert torch.equal(gst, snap)

    for rep in range(3):
        gout.fill_(float("nan"))
        gst.copy_(snap)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(gout, want), f"replay {rep}: outputs differ from eager"
        assert torch.equal(gst, want_state), f"replay {rep}: state differs from eager"
        # eager work between replays on the same state buffer
        gst.copy_(snap)
        again = _eager(case, gst, phi, qs, ks, vs)
        assert torch.equal(again, want)
    # and the eager outputs themselves against the oracle
    case.check_decode(want.permute(1, 2, 0, 3, 4).cpu(), q, k, v, [n0] * case.B, n, "graph")


def test_graph_prefill_then_decode_matches_eager():
    """A chunked prefill call and decode steps captured together (no memset
    is enqueued by either), replayed from a restored state, against the same
    calls made eagerly."""
    case = Case([0, 5, 40, 200], batch=2, Hq=8, Hkv=2, d=128, Df=128, dtype=torch.bfloat16, seed=9)
    lens = [70, 133]
    n = 6
    q, k, v = case.tokens(max(lens) + n)
    phi = case.phi_w.cuda()
    cu = [0, lens[0], lens[0] + lens[1]]
    T = cu[-1]
    qp = torch.cat([q[:, b, :lens[b]] for b in range(2)], 1).contiguous().cuda()
    kp = torch.cat([k[:, b, :lens[b]] for b in range(2)], 1).contiguous().cuda()
    vp = torch.cat([v[:, b, :lens[b]] for b in range(2)], 1).contiguous().cuda()
    sel = lambda x, s: torch.stack([x[:, b, lens[b] + s] for b in range(2)], 1).contiguous().cuda()
    dq = torch.stack([sel(q, s) for s in range(n)])
    dk = torch.stack([sel(k, s) for s in range(n)])
    dv = torch.stack([sel(v, s) for s in range(n)])
    ws = case.g.new_workspace(T)

    def calls(st, pout, dout):
        case.g.prefill(st, phi, qp, kp, vp, cu, pout, ws)
        for s in range(n):
            case.g.decode_step(st, phi, dq[s], dk[s], dv[s], dout[s], ws)

    st0 = case.new_state()
    torch.cuda.synchronize()
    snap = st0.clone()
    pe, de = torch.empty_like(qp), torch.empty_like(dq)
    calls(st0, pe, de)
    torch.cuda.synchronize()

    gst = snap.clone()
    pg, dg = torch.empty_like(qp), torch.empty_like(dq)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        calls(gst, pg, dg)
    torch.cuda.synchronize()
    assert torch.equal(gst, snap)
    for rep in range(3):
        pg.fill_(float("nan"))
        dg.fill_(float("nan"))
        gst.copy_(snap)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(pg, pe) and torch.equal(dg, de), f"replay {rep}: outputs differ from eager"
        assert torch.equal(gst, st0), f"replay {rep}: state differs from eager"
    # the eager outputs against the oracle
    outs = [[pe[l, cu[b]:cu[b + 1]].cpu() for b in range(2)] for l in range(case.L)]
    case.check_prefill(outs, q, k, v, [0, 0], lens, "graph prefill")
    case.check_decode(de.permute(1, 2, 0, 3, 4).cpu(), q, k, v, lens, n, "graph decode")
