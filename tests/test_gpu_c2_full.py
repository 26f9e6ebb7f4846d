"""GPU parity of the 32-layer, batch-1, 8K-context stack checked in full.

The stack is generated with bench.py's seeded recipe and run as bench.py
runs it: one prefill call over all 32 layers, then whole-stack decode steps
(24 of them: three fold periods, so every unit has folded its pending tokens
on a staggered step at least twice).  Checked against the oracle:

  * every layer: prefill outputs at every 997th position and at the edges of
    the last two chunks, every decode step, the raw state (S, z per KV head
    over the tokens it has folded, nf inside [beta - 8, beta]), the flushed
    state, the window ring bit for bit and pos;
  * the layers with the smallest, middle and largest window: every output
    position of the sequence, prefill and decode, against the oracle's
    recurrent form run token by token from the empty state.

The GPU work runs once per module; each test checks one part.
"""
import concurrent.futures as cf

import numpy as np
import pytest
import torch

import oracle
from paper_2607_24788_amd import glide
from paper_2607_24788_amd import workload as W

from .gpu_util import check, f64

pytestmark = pytest.mark.gpu

N_DEC = 24
WORKERS = 16


def _positions(n, chunk):
    """Every 997th position and the edges of the last two chunks."""
    pos = set(range(0, n, 997)) | {n - 2 * chunk, n - 2 * chunk + 1, n - chunk - 1, n - chunk, n - chunk + 1, n - 1}
    return sorted(p for p in pos if 0 <= p < n)


@pytest.fixture(scope="module")
def run():
    wl = W.workload("c2")
    assert wl.batch == 1
    dev = torch.device("cuda:0")
    g = glide.Glide(wl.n_layers, wl.batch, wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.feat_dim, wl.windows,
                    dtype=wl.dtype, sm_scale=wl.tau)
    n = wl.context[0]
    L = wl.n_layers
    cu = [0, n]
    print(f"c2 full: prefill {n} tokens x {L} layers, then {N_DEC} decode steps", flush=True)
    phi = W.phi_weights(wl, device=dev)
    qp = torch.empty((L, n, wl.n_q_heads, wl.head_dim), dtype=wl.dtype, device=dev)
    kp = torch.empty((L, n, wl.n_kv_heads, wl.head_dim), dtype=wl.dtype, device=dev)
    vp = torch.empty_like(kp)
    for l in range(L):
        qp[l], kp[l], vp[l] = W.prefill_inputs(wl, l, [n], device=dev)
    pout = torch.empty((L, n, wl.n_q_heads, wl.head_dim), dtype=wl.dtype, device=dev)
    state = g.new_state(dev)
    ws = g.new_workspace(n, dev)
    g.state_init(state)
    g.prefill(state, phi, qp, kp, vp, cu, pout, ws, chunk=wl.chunk)
    dq, dk, dv, dout = [], [], [], []
    o = torch.empty((L, 1, wl.n_q_heads, wl.head_dim), dtype=wl.dtype, device=dev)
    for s in range(N_DEC):
        q, k, v = W.decode_inputs(wl, s, device=dev)
        g.decode_step(state, phi, q, k, v, o, ws)
        dq.append(q[:, 0].cpu())
        dk.append(k[:, 0].cpu())
        dv.append(v[:, 0].cpu())
        dout.append(o[:, 0].cpu())
    flushed = state.clone()
    g.state_flush(flushed, phi)
    torch.cuda.synchronize()
    r = {"wl": wl, "g": g, "n": n, "phi": phi.cpu(),
         # whole histories per layer: prefill tokens then the decoded ones
         "q": torch.cat([qp.cpu(), torch.stack(dq, 1)], 1),
         "k": torch.cat([kp.cpu(), torch.stack(dk, 1)], 1),
         "v": torch.cat([vp.cpu(), torch.stack(dv, 1)], 1),
         "pre": pout.cpu(), "dec": torch.stack(dout, 1)}
    r["views"] = [{k_: (v_.cpu() if torch.is_tensor(v_) else v_) for k_, v_ in g.layer_views(state, l).items()}
                  for l in range(L)]
    r["fviews"] = [{k_: (v_.cpu() if torch.is_tensor(v_) else v_) for k_, v_ in g.layer_views(flushed, l).items()}
                   for l in range(L)]
    del qp, kp, vp, pout, state, flushed, ws
    torch.cuda.empty_cache()
    return r


def _oracle(wl, l, n_kv=None):
    Hkv = wl.n_kv_heads if n_kv is None else n_kv
    return oracle.Oracle(wl.G * Hkv, Hkv, wl.head_dim, wl.feat_dim, wl.windows[l], tau=wl.tau)


def test_c2_every_layer_sampled_prefill_and_every_decode_step(run):
    wl, n = run["wl"], run["n"]
    pos = np.array(_positions(n, wl.chunk) + [n + s for s in range(N_DEC)])
    npre = len(pos) - N_DEC
    for l in range(wl.n_layers):
        hist = slice(0, n + N_DEC)
        want = _oracle(wl, l).attend(f64(run["phi"][l]), f64(run["q"][l, hist]), f64(run["k"][l, hist]),
                                     f64(run["v"][l, hist]), positions=pos)
        label = f"c2 layer {l} (W={wl.windows[l]})"
        check(f"{label} prefill", f64(run["pre"][l, pos[:npre]]), want[:npre], wl.dtype)
        check(f"{label} decode", f64(run["dec"][l]), want[npre:], wl.dtype)


def test_c2_every_layer_state_and_ring(run):
    wl, n = run["wl"], run["n"]
    p = n + N_DEC
    jobs = []
    for l in range(wl.n_layers):
        Wl = wl.windows[l]
        views, fv = run["views"][l], run["fviews"][l]
        assert int(views["pos"].min()) == p and int(views["pos"].max()) == p, f"c2 layer {l} pos"
        beta = max(0, p - Wl)
        nfs = [int(x) for x in views["nf"][0]]
        assert all(max(0, beta - 8) <= x <= beta for x in nfs), f"c2 layer {l} nf {nfs} vs beta {beta}"
        assert all(int(x) == beta for x in fv["nf"][0]), f"c2 layer {l} flushed nf"
        # the raw state of KV head h holds the sums over [0, nf_h): one
        # single-head oracle per head (the heads are independent)
        for h, nf in enumerate(nfs):
            jobs.append((l, h, nf))
        R = views["ring_slots"]
        kl = glide.kring_logical(views["kring_raw"][0], R, wl.head_dim)
        vl = glide.vring_logical(views["vring_raw"][0], R, wl.head_dim)
        js = list(range(min(min(nfs), p - Wl), p))
        sl = [j % R for j in js]
        assert torch.equal(kl[:, sl], run["k"][l, js].transpose(0, 1)), f"c2 layer {l} key ring"
        assert torch.equal(vl[:, sl], run["v"][l, js].transpose(0, 1)), f"c2 layer {l} value ring"

    def raw_state(job):
        l, h, nf = job
        o = _oracle(wl, l, n_kv=1)
        S, z = o.state(f64(run["phi"][l]), f64(run["k"][l, :, h:h + 1]), f64(run["v"][l, :, h:h + 1]),
                       nf + wl.windows[l])
        return job, S[0], z[0]

    def flushed_state(l):
        S, z = _oracle(wl, l).state(f64(run["phi"][l]), f64(run["k"][l]), f64(run["v"][l]), p)
        return l, S, z

    with cf.ThreadPoolExecutor(WORKERS) as ex:
        for (l, h, nf), S, z in ex.map(raw_state, jobs):
            label = f"c2 layer {l} (W={wl.windows[l]}) head {h} (nf {nf})"
            check(f"{label} S", f64(run["views"][l]["S"][0, h]), S, wl.dtype, "state")
            check(f"{label} z", f64(run["views"][l]["z"][0, h]), z, wl.dtype, "state")
        for l, S, z in ex.map(flushed_state, range(wl.n_layers)):
            label = f"c2 layer {l} (W={wl.windows[l]}) flushed"
            check(f"{label} S", f64(run["fviews"][l]["S"][0]), S, wl.dtype, "state")
            check(f"{label} z", f64(run["fviews"][l]["z"][0]), z, wl.dtype, "state")


@pytest.mark.parametrize("which", ["smallest", "middle", "largest"])
def test_c2_every_position_recurrent(run, which):
    wl, n = run["wl"], run["n"]
    order = sorted(range(wl.n_layers), key=lambda l: wl.windows[l])
    l = {"smallest": order[0], "middle": order[len(order) // 2], "largest": order[-1]}[which]
    o = _oracle(wl, l)
    wf = f64(run["phi"][l])
    q, k, v = f64(run["q"][l]), f64(run["k"][l]), f64(run["v"][l])
    st = o.empty_state(1)
    want = np.empty((n + N_DEC, wl.n_q_heads, wl.head_dim))
    for t in range(n + N_DEC):
        want[t] = o.decode(wf, st, q[t][None], k[t][None], v[t][None])[0]
    label = f"c2 layer {l} (W={wl.windows[l]}) recurrent from empty"
    check(f"{label} prefill", f64(run["pre"][l]), want[:n], wl.dtype)
    check(f"{label} decode", f64(run["dec"][l]), want[n:], wl.dtype)
