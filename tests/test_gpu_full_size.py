"""GPU parity at the benchmark's full sizes, in the launch configuration
bench.py times, on outputs the oracle computes one by one.

Each workload is generated with bench.py's own seeded recipe (the large ones
share one layer's prefill inputs across layers and call the prefill one layer
at a time, as bench.py does), prefilled, then decoded for a few whole-stack
steps.  Sampled: the layers with the smallest, middle and largest window (and
a W = 0 layer where there is one), the first and last sequence, every head;
prefill outputs at the last two chunks and every 997th position (every
4999th beyond 40K tokens, to bound the oracle's time), every decode step, and
the final S, z (flushed) and window ring.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_24788_amd import glide
from paper_2607_24788_amd import workload as W

from .gpu_util import check, f64

pytestmark = pytest.mark.gpu

N_DEC = 4


def _sample_layers(wl):
    order = sorted(range(wl.n_layers), key=lambda l: wl.windows[l])
    ls = {order[0], order[len(order) // 2], order[-1]}
    ls |= {l for l in range(wl.n_layers) if wl.windows[l] == 0}
    return sorted(ls)[:4]


def _positions(n, chunk):
    stride = 997 if n < 40000 else 4999
    pos = set(range(0, n, stride)) | {n - 2 * chunk, n - chunk - 1, n - chunk, n - 1}
    return sorted(p for p in pos if 0 <= p < n)


@pytest.mark.parametrize("name", ["c2", "c3", "c3b", "c5", "c4u", "c4"])
def test_full_size_sampled(name):
    wl = W.workload(name)
    dev = torch.device("cuda:0")
    g = glide.Glide(wl.n_layers, wl.batch, wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.feat_dim, wl.windows,
                    dtype=wl.dtype, sm_scale=wl.tau)
    lens = list(wl.context)
    cu = [0]
    for n in lens:
        cu.append(cu[-1] + n)
    T, L = cu[-1], wl.n_layers
    big = sum(wl.context) > 1_000_000 or wl.batch * max(wl.context) > 400_000   # bench.py's rule
    n_pre = 1 if big else L
    layers = _sample_layers(wl)
    seqs = sorted({0, wl.batch - 1})
    pos = {b: _positions(lens[b], wl.chunk) for b in seqs}

    phi = W.phi_weights(wl, device=dev)
    qp = torch.empty((n_pre, T, wl.n_q_heads, wl.head_dim), dtype=wl.dtype, device=dev)
    kp = torch.empty((n_pre, T, wl.n_kv_heads, wl.head_dim), dtype=wl.dtype, device=dev)
    vp = torch.empty_like(kp)
    for l in range(n_pre):
        qp[l], kp[l], vp[l] = W.prefill_inputs(wl, l, lens, device=dev)
    pout = torch.empty((n_pre, T, wl.n_q_heads, wl.head_dim), dtype=wl.dtype, device=dev)
    state = g.new_state(dev)
    ws = g.new_workspace(T, dev)
    g.state_init(state)

    got_pre = {}
    idx = {b: torch.tensor([cu[b] + p for p in pos[b]], device=dev) for b in seqs}
    if big:
        for l in range(L):
            g.prefill(state, phi[l:l + 1], qp, kp, vp, cu, pout, ws, layer0=l, n_layers=1, chunk=wl.chunk)
            if l in layers:
                for b in seqs:
                    got_pre[l, b] = pout[0].index_select(0, idx[b]).cpu()
    else:
        g.prefill(state, phi, qp, kp, vp, cu, pout, ws, chunk=wl.chunk)
        for l in layers:
            for b in seqs:
                got_pre[l, b] = pout[l].index_select(0, idx[b]).cpu()

    n_dec = N_DEC if wl.decode_steps else 0
    dec_in, got_dec = [], []
    dout = torch.empty((L, wl.batch, wl.n_q_heads, wl.head_dim), dtype=wl.dtype, device=dev)
    for s in range(n_dec):
        dq, dk, dv = W.decode_inputs(wl, s, device=dev)
        g.decode_step(state, phi, dq, dk, dv, dout, ws)
        dec_in.append((dq[layers].cpu(), dk[layers].cpu(), dv[layers].cpu()))
        got_dec.append(dout[layers].cpu())
    flushed = state.clone()
    g.state_flush(flushed, phi)
    torch.cuda.synchronize()

    for li, l in enumerate(layers):
        Wl = wl.windows[l]
        src = 0 if big else l
        o = oracle.Oracle(wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.feat_dim, Wl, tau=wl.tau)
        wf = f64(phi[l])
        views = g.layer_views(flushed, l)
        raw = g.layer_views(state, l)
        for b in seqs:
            n = lens[b]
            sl = slice(cu[b], cu[b + 1])
            qh = torch.cat([qp[src, sl].cpu()] + [d[0][li, b][None] for d in dec_in]) if n_dec else qp[src, sl].cpu()
            kh = torch.cat([kp[src, sl].cpu()] + [d[1][li, b][None] for d in dec_in]) if n_dec else kp[src, sl].cpu()
            vh = torch.cat([vp[src, sl].cpu()] + [d[2][li, b][None] for d in dec_in]) if n_dec else vp[src, sl].cpu()
            ps = pos[b] + [n + s for s in range(n_dec)]
            want = o.attend(wf, f64(qh), f64(kh), f64(vh), positions=np.array(ps))
            label = f"{name} layer {l} (W={Wl}) seq {b}"
            check(f"{label} prefill", f64(got_pre[l, b]), want[:len(pos[b])], wl.dtype)
            if n_dec:
                gd = torch.stack([x[li, b] for x in got_dec])
                check(f"{label} decode", f64(gd), want[len(pos[b]):], wl.dtype)
            p = n + n_dec
            assert int(raw["pos"][b].min()) == p and int(raw["pos"][b].max()) == p, f"{label} pos"
            S, z = o.state(wf, f64(kh), f64(vh), p)
            check(f"{label} S", f64(views["S"][b]), S, wl.dtype, "state")
            check(f"{label} z", f64(views["z"][b]), z, wl.dtype, "state")
            R = views["ring_slots"]
            if R:
                kl = glide.kring_logical(raw["kring_raw"][b].cpu(), R, wl.head_dim)
                vl = glide.vring_logical(raw["vring_raw"][b].cpu(), R, wl.head_dim)
                js = list(range(max(0, p - Wl), p))
                sl_ = [j % R for j in js]
                assert torch.equal(kl[:, sl_], kh[js].transpose(0, 1)), f"{label} key ring"
                assert torch.equal(vl[:, sl_], vh[js].transpose(0, 1)), f"{label} value ring"
