"""Helpers for the GPU parity tests: run the HIP path through the C ABI and
compare with the CPU oracle on the same seeded inputs.

Tolerances (applied per tensor X, err = max |X_gpu - X_oracle|):
  fp32 I/O : err <= 1e-5 * max |X_oracle|         for O, S and z
  bf16 I/O : err(O) <= 2e-2 absolute and err(O) <= 1e-2 * max |O_oracle|,
             err(S), err(z) <= 1e-2 * max |X_oracle|
  ring     : bit-exact (it is a copy of the inputs); pos exact.
"""
import numpy as np
import torch

import oracle
from paper_2607_24788_amd import glide

TOL = {torch.float32: dict(rel=1e-5, abs=None, state_rel=1e-5),
       torch.bfloat16: dict(rel=1e-2, abs=2e-2, state_rel=1e-2)}


def f64(t):
    return t.detach().to("cpu", torch.float64).numpy()


def check(name, got, want, dtype, kind="out"):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    assert got.shape == want.shape, f"{name}: shape {got.shape} != {want.shape}"
    assert np.all(np.isfinite(got)), f"{name}: non-finite values"
    err = float(np.max(np.abs(got - want))) if got.size else 0.0
    scale = float(np.max(np.abs(want))) if want.size else 0.0
    t = TOL[dtype]
    rel = t["rel"] if kind == "out" else t["state_rel"]
    bound = rel * max(scale, 1e-30)
    assert err <= bound + 1e-30, f"{name}: max err {err:.3e} > {rel} x max|ref| ({scale:.3e})"
    if kind == "out" and t["abs"] is not None:
        assert err <= t["abs"], f"{name}: max err {err:.3e} > {t['abs']}"
    return err, scale


class Case:
    """A decode/prefill test case on a small synthetic stack."""

    def __init__(self, windows, batch=1, Hq=4, Hkv=4, d=64, Df=64, dtype=torch.float32, linear=True,
                 tau=None, seed=0, qkv_scale=None, v_scale=None, form=0, phi=0, per_head_phi=False, gated=False,
                 gate_lo=-0.4):
        self.windows = list(windows)
        self.L = len(windows)
        self.B, self.Hq, self.Hkv, self.d, self.Df = batch, Hq, Hkv, d, Df
        self.dtype, self.linear, self.form, self.phi = dtype, linear, form, phi
        self.per_head_phi = per_head_phi
        self.gated, self.gate_lo = gated, gate_lo
        self.tau = d ** -0.5 if tau is None else tau
        self.seed = seed
        self.qkv_scale = d ** -0.5 if qkv_scale is None else qkv_scale
        self.v_scale = self.qkv_scale if v_scale is None else v_scale
        self.g = glide.Glide(self.L, batch, Hq, Hkv, d, Df, self.windows, dtype=dtype, sm_scale=self.tau,
                             linear=linear, form=form, phi=phi, per_head_phi=per_head_phi, gated=gated)
        gen = torch.Generator().manual_seed(seed * 7919 + 17)
        wshape = (self.L, Hkv, d, Df) if per_head_phi else (self.L, d, Df)
        self.phi_w = (torch.randn(wshape, generator=gen) * d ** -0.5).to(dtype)
        self._gen = gen

    def tokens(self, n):
        """History tensors per layer: q [L][B][n][Hq][d], k/v [L][B][n][Hkv][d]."""
        gen = self._gen
        q = (torch.randn((self.L, self.B, n, self.Hq, self.d), generator=gen) * self.qkv_scale).to(self.dtype)
        k = (torch.randn((self.L, self.B, n, self.Hkv, self.d), generator=gen) * self.qkv_scale).to(self.dtype)
        v = (torch.randn((self.L, self.B, n, self.Hkv, self.d), generator=gen) * self.v_scale).to(self.dtype)
        return q, k, v

    def log_gates(self, n):
        """Log-gates [L][B][n][Hkv], fp32, uniform in [gate_lo, 0] (gated stacks)."""
        g = torch.Generator().manual_seed(self.seed * 104729 + 3)
        return torch.rand((self.L, self.B, n, self.Hkv), generator=g) * self.gate_lo

    def oracle(self, l):
        return oracle.Oracle(self.Hq, self.Hkv, self.d, self.Df, self.windows[l], linear=self.linear,
                             tau=self.tau, form=self.form, phi=self.phi, wf_per_head=self.per_head_phi)

    def delay(self, l):
        """The linear part's delay: the window, or 0 when the state holds every token."""
        return 0 if self.form == 2 else self.windows[l]

    def new_state(self):
        st = self.g.new_state()
        self.g.state_init(st)
        return st

    @property
    def ws(self):
        if not hasattr(self, "_ws"):
            self._ws = self.g.new_workspace(4096)
        return self._ws

    def decode_steps(self, state, q, k, v, t0, t1, gates=None):
        """Decode positions [t0, t1) of the history tensors; returns out [L][B][t1-t0][Hq][d] (CPU)."""
        outs = []
        phi = self.phi_w.cuda()
        for t in range(t0, t1):
            qs = q[:, :, t].contiguous().cuda()
            ks = k[:, :, t].contiguous().cuda()
            vs = v[:, :, t].contiguous().cuda()
            gs = None if gates is None else gates[:, :, t].contiguous().cuda()
            o = torch.empty_like(qs)
            self.g.decode_step(state, phi, qs, ks, vs, o, self.ws, log_gates=gs)
            outs.append(o)
        torch.cuda.synchronize()
        return torch.stack(outs, 2).cpu()

    def prefill(self, state, q, k, v, starts, lens, chunk=0, gates=None):
        """Prefill tokens [starts[b], starts[b] + lens[b]) of every sequence (one
        call over all layers); returns out [L][B] list of [lens[b]][Hq][d] (CPU)."""
        cu = [0]
        for n in lens:
            cu.append(cu[-1] + n)
        T = cu[-1]
        qp = torch.cat([q[:, b, s:s + n] for b, (s, n) in enumerate(zip(starts, lens))], 1).contiguous()
        kp = torch.cat([k[:, b, s:s + n] for b, (s, n) in enumerate(zip(starts, lens))], 1).contiguous()
        vp = torch.cat([v[:, b, s:s + n] for b, (s, n) in enumerate(zip(starts, lens))], 1).contiguous()
        gp = None if gates is None else torch.cat([gates[:, b, s:s + n] for b, (s, n) in enumerate(zip(starts, lens))],
                                                  1).contiguous().cuda()
        out = torch.full((self.L, T, self.Hq, self.d), float("nan"), dtype=self.dtype, device="cuda")
        ws = self.g.new_workspace(max(T, 1))
        self.g.prefill(state, self.phi_w.cuda(), qp.cuda(), kp.cuda(), vp.cuda(), cu, out, ws, chunk=chunk,
                       log_gates=gp)
        torch.cuda.synchronize()
        out = out.cpu()
        return [[out[l, cu[b]:cu[b + 1]] for b in range(self.B)] for l in range(self.L)]

    def _attend(self, o, l, b, q, k, v, hist, pos, gates):
        args = (f64(self.phi_w[l]), f64(q[l, b, hist]), f64(k[l, b, hist]), f64(v[l, b, hist]))
        if gates is None:
            return o.attend(*args, positions=pos)
        return o.attend_gated(*args, f64(gates[l, b, hist]), positions=pos)

    def _state(self, o, l, b, k, v, p, gates):
        if gates is None:
            return o.state(f64(self.phi_w[l]), f64(k[l, b]), f64(v[l, b]), p)
        if p - self.delay(l) <= 0:  # nothing folded: the sums are empty
            return (np.zeros((self.Hkv, self.Df, self.d)), np.zeros((self.Hkv, self.Df)))
        return o.state_gated(f64(self.phi_w[l]), f64(k[l, b, :p]), f64(v[l, b, :p]), f64(gates[l, b, :p]), p)

    def check_prefill(self, outs, q, k, v, starts, lens, label="", positions=None, gates=None):
        """outs from prefill(); compares every (or the listed) output position."""
        for l in range(self.L):
            o = self.oracle(l)
            for b, (s, n) in enumerate(zip(starts, lens)):
                if n == 0:
                    continue
                pos = np.arange(s, s + n) if positions is None else np.asarray(positions[b])
                hist = slice(0, int(pos.max()) + 1)
                want = self._attend(o, l, b, q, k, v, hist, pos, gates)
                check(f"{label} prefill O layer {l} (W={self.windows[l]}) seq {b}", f64(outs[l][b][pos - s]),
                      want, self.dtype)

    def load_state_from_oracle(self, state, q, k, v, positions):
        """Write the state after positions[b] tokens of sequence b, built by the
        oracle's direct sums plus the literal window, into the GPU state."""
        for l in range(self.L):
            views = self.g.layer_views(state, l)
            o = self.oracle(l)
            W, R = self.windows[l], views["ring_slots"]
            for b, p in enumerate(positions):
                S, z = o.state(f64(self.phi_w[l]), f64(k[l, b]), f64(v[l, b]), p)
                views["S"][b] = torch.from_numpy(S).float().cuda()
                views["z"][b] = torch.from_numpy(z).float().cuda()
                views["pos"][b] = p
                views["nf"][b] = max(0, p - self.delay(l))      # nothing pending
                if R:
                    kl = glide.kring_logical(views["kring_raw"][b].cpu(), R, self.d)
                    vl = glide.vring_logical(views["vring_raw"][b].cpu(), R, self.d)
                    for j in range(max(0, p - W), p):
                        kl[:, j % R] = k[l, b, j]
                        vl[:, j % R] = v[l, b, j]
                    views["kring_raw"][b] = glide.kring_raw(kl, R, self.d).cuda()
                    views["vring_raw"][b] = glide.vring_raw(vl, R, self.d).cuda()
        torch.cuda.synchronize()

    def check_decode(self, out, q, k, v, positions, t_steps, label="", gates=None):
        """out [L][B][n][Hq][d] for positions[b] .. positions[b]+n-1."""
        n = out.shape[2]
        worst = 0.0
        for l in range(self.L):
            o = self.oracle(l)
            for b, p0 in enumerate(positions):
                hist = slice(0, p0 + n)
                want = self._attend(o, l, b, q, k, v, hist, np.arange(p0, p0 + n), gates)
                e, _ = check(f"{label} O layer {l} (W={self.windows[l]}) seq {b}", f64(out[l, b]), want,
                             self.dtype)
                worst = max(worst, e)
        return worst

    def check_state(self, state, k, v, positions, label="", flush=True, gates=None):
        """S, z, pos, nf and the ring after positions[b] tokens of sequence b.
        S, z are compared with the oracle's sums over tokens [0, nf) (deferred
        folding: nf in [beta - 8, beta], beta = max(0, p - W)); with flush, a
        copy of the state is flushed and must then hold the sums over [0, beta)."""
        if flush and self.linear:
            flushed = state.clone()
            self.g.state_flush(flushed, self.phi_w.cuda())
            torch.cuda.synchronize()
        for l in range(self.L):
            views = self.g.layer_views(state, l)
            o = self.oracle(l)
            W, R = self.windows[l], views["ring_slots"]
            for b, p in enumerate(positions):
                assert int(views["pos"][b].min()) == p and int(views["pos"][b].max()) == p, \
                    f"{label} pos layer {l} seq {b}"
                Wd = self.delay(l)
                beta = max(0, p - Wd)
                first = beta
                if self.linear:
                    # the fold step is staggered over units: nf is per KV head
                    nfs = [int(x) for x in views["nf"][b]]
                    lo = beta if Wd == 0 else max(0, beta - 8)
                    assert all(lo <= x <= beta for x in nfs), \
                        f"{label} nf {nfs} outside [{lo}, {beta}] layer {l} seq {b}"
                    first = min(nfs)
                    for nf in sorted(set(nfs)):
                        hs = [h for h, x in enumerate(nfs) if x == nf]
                        # the oracle's state after n tokens sums tokens [0, n - Wd)
                        # (gated: decayed to the step that folded last, n - 1)
                        S, z = self._state(o, l, b, k, v, nf + Wd, gates)
                        check(f"{label} S layer {l} seq {b} heads {hs} (nf {nf})", f64(views["S"][b, hs]), S[hs],
                              self.dtype, "state")
                        check(f"{label} z layer {l} seq {b} heads {hs} (nf {nf})", f64(views["z"][b, hs]), z[hs],
                              self.dtype, "state")
                    if flush:
                        fv = self.g.layer_views(flushed, l)
                        assert torch.all(fv["nf"][b] == beta), f"{label} flushed nf layer {l} seq {b}"
                        S, z = self._state(o, l, b, k, v, p, gates)
                        check(f"{label} flushed S layer {l} seq {b}", f64(fv["S"][b]), S, self.dtype, "state")
                        check(f"{label} flushed z layer {l} seq {b}", f64(fv["z"][b]), z, self.dtype, "state")
                if gates is not None and p > 0:
                    # G_{p-1} (fp64 cumulative log-gates), and G_f = G_{p-1} once flushed
                    Gc = np.cumsum(gates[l, b, :p].double().numpy(), axis=0)
                    gv = views["gate"][b].cpu().numpy()
                    assert np.allclose(gv[:, 0], Gc[p - 1], rtol=0, atol=1e-9), f"{label} G_cur layer {l} seq {b}"
                    if flush and self.linear and p > Wd:
                        fg = self.g.layer_views(flushed, l)["gate"][b].cpu().numpy()
                        assert np.allclose(fg[:, 1], Gc[p - 1], rtol=0, atol=1e-9), f"{label} G_f layer {l} seq {b}"
                    if R:
                        gr = views["gring"][b].cpu().numpy()
                        for j in range(max(first, max(0, p - W)), p):
                            assert np.allclose(gr[:, j % R], Gc[j], rtol=0, atol=1e-9), \
                                f"{label} gate ring layer {l} seq {b} token {j}"
                if not R:
                    continue
                first = min(first, max(0, p - W))   # the window, and the pending tokens
                kr = glide.kring_logical(views["kring_raw"][b].cpu(), R, self.d)
                vr = glide.vring_logical(views["vring_raw"][b].cpu(), R, self.d)
                for j in range(first, p):
                    s = j % R
                    assert torch.equal(kr[:, s], k[l, b, j]), f"{label} key ring layer {l} seq {b} token {j}"
                    assert torch.equal(vr[:, s], v[l, b, j]), f"{label} value ring layer {l} seq {b} token {j}"
