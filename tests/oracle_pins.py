"""Pins that tie the CPU oracle to facts fixed outside the oracle itself.

Each check returns None on success or a short failure message.  They are run
by ``test_oracle_pins.py`` against the real oracle, and by the mutation test
against oracle builds with one planted mistake each, to show that a plausible
slip anywhere in the oracle fails at least one pin.

What pins what:
  * worked example (tests/golden): hand-derived closed forms of the layer
    definition (GLIDE Sec. III-B) on a 3-token, d = 1 sequence;
  * full window, linear off == causal softmax attention computed by torch's
    scaled_dot_product_attention (the first boundary condition of Sec. III-B,
    "w -> infinity gives causal softmax");
  * window W, linear off == SDPA with an explicit band mask (Sec. II-C);
  * W = 0 == causal linear attention as a masked matrix product (the second
    boundary condition, "w = 0 gives pure linear attention"; Appendix, linear
    attention before the rearrangement);
  * W = 1 == closed form built from the W = 0 numerator and denominator at
    t - 1 plus the diagonal score;
  * recurrent decode from empty == definition form at every position, and the
    decoded state == direct sums (Appendix rearrangement to S and Z);
  * invariants: V == 1 gives O == 1 (shared denominator), outputs in the convex
    hull of the seen values, linearity in V, GQA == MHA with repeated K/V,
    0/0 -> 0;
  * the Appendix's two hybrid forms (forms 1, 2): hand-derived worked-example
    values, O == band SDPA + causal linear attention (delayed by W in form 1,
    undelayed in form 2), V == 1 giving one per non-empty part, and the
    recurrent, direct-sum and continued-decode checks above in both forms.
"""
import json
import math
import os

import numpy as np
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "worked_example.json")


def _eval_closed_form(expr):
    return float(eval(expr, {"__builtins__": {}}, {"e": math.e, "exp": math.exp, "log": math.log}))


def _rand_case(seed, n, Hq, Hkv, d, Df, scale=1.0):
    g = np.random.default_rng(seed)
    q = g.standard_normal((n, Hq, d)) * scale
    k = g.standard_normal((n, Hkv, d)) * scale
    v = g.standard_normal((n, Hkv, d))
    Wf = g.standard_normal((d, Df)) / np.sqrt(d)
    return q, k, v, Wf


def _sdpa(q, k, v, tau, mask):
    """torch SDPA in float64 on CPU; q [n][Hq][d], k/v [n][Hkv][d] (GQA by repeat)."""
    G = q.shape[1] // k.shape[1]
    qt = torch.from_numpy(q).permute(1, 0, 2).contiguous()
    kt = torch.from_numpy(np.repeat(k, G, axis=1)).permute(1, 0, 2).contiguous()
    vt = torch.from_numpy(np.repeat(v, G, axis=1)).permute(1, 0, 2).contiguous()
    m = torch.from_numpy(mask)
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=m, scale=tau)
    return o.permute(1, 0, 2).numpy()


def _feat(y, phi):
    if phi == 2:  # softmax over the features (numpy's own exp and sum)
        e = np.exp(y - y.max(axis=-1, keepdims=True))
        return e / e.sum(axis=-1, keepdims=True)
    return np.maximum(y, 0.0) if phi == 0 else np.where(y > 0, y + 1.0, np.exp(np.minimum(y, 0.0)))


def _causal_linear(q, k, v, Wf, phi=0):
    """Causal linear attention, masked-matrix form, with numpy matmuls."""
    G = q.shape[1] // k.shape[1]
    n = q.shape[0]
    pq = _feat(q @ Wf, phi)                            # [n][Hq][Df]
    pk = _feat(np.repeat(k, G, axis=1) @ Wf, phi)
    vv = np.repeat(v, G, axis=1)
    num = np.zeros(q.shape)
    den = np.zeros(q.shape[:2])
    tril = np.tril(np.ones((n, n)))
    for h in range(q.shape[1]):
        M = (pq[:, h] @ pk[:, h].T) * tril
        num[:, h] = M @ vv[:, h]
        den[:, h] = M.sum(-1)
    return num, den


def pin_worked_example(lib):
    ex = json.load(open(GOLDEN))
    s = ex["setup"]
    q = np.array(s["q"]).reshape(3, 1, 1)
    k = np.array(s["k"]).reshape(3, 1, 1)
    v = np.array(s["v"]).reshape(3, 1, 1)
    Wf = np.array(s["Wf"])
    for case in ex["cases"]:
        o = oracle.Oracle(1, 1, 1, 1, case["window"], linear=case["linear"], tau=s["tau"], lib=lib,
                          form=case.get("form", 0), phi=case.get("phi", 0))
        got = o.attend(Wf, q, k, v).ravel()
        want = np.array([_eval_closed_form(x) for x in case["out"]])
        if not np.allclose(got, want, rtol=1e-12, atol=1e-12):
            return f"worked example form {case.get('form', 0)} W={case['window']}: {got} != {want}"
        S, z = o.state(Wf, k, v)
        if not (abs(S.item() - _eval_closed_form(case["S"])) < 1e-12
                and abs(z.item() - _eval_closed_form(case["z"])) < 1e-12):
            return f"worked example state form {case.get('form', 0)} W={case['window']}: S={S.item()} z={z.item()}"
        # recurrent form on the same example
        st = o.empty_state(1)
        outs = [o.decode(Wf, st, q[t:t + 1], k[t:t + 1], v[t:t + 1]).item() for t in range(3)]
        if not np.allclose(outs, want, rtol=1e-12, atol=1e-12):
            return f"worked example recurrent form {case.get('form', 0)} W={case['window']}: {outs} != {want}"
        if not (abs(st["S"].item() - _eval_closed_form(case["S"])) < 1e-12):
            return f"worked example recurrent state W={case['window']}"
    return None


def pin_full_window_is_causal_softmax(lib):
    n, Hq, Hkv, d, Df = 23, 4, 2, 8, 6
    q, k, v, Wf = _rand_case(1, n, Hq, Hkv, d, Df)
    tau = 0.7
    mask = np.tril(np.ones((n, n), bool))
    want = _sdpa(q, k, v, tau, mask)
    for W, lin in ((n, False), (n + 5, False), (n, True), (10 ** 6, True)):
        got = oracle.Oracle(Hq, Hkv, d, Df, W, linear=lin, tau=tau, lib=lib).attend(Wf, q, k, v)
        if not np.allclose(got, want, rtol=1e-10, atol=1e-12):
            return f"full window W={W} linear={lin} != causal SDPA (max err {np.abs(got - want).max()})"
    return None


def pin_band_is_masked_sdpa(lib):
    n, Hq, Hkv, d, Df = 29, 4, 4, 8, 8
    q, k, v, Wf = _rand_case(2, n, Hq, Hkv, d, Df)
    tau = 0.5
    t = np.arange(n)[:, None]
    j = np.arange(n)[None, :]
    for W in (1, 2, 5, 17):
        mask = (j <= t) & (j >= t - W + 1)
        want = _sdpa(q, k, v, tau, mask)
        got = oracle.Oracle(Hq, Hkv, d, Df, W, linear=False, tau=tau, lib=lib).attend(Wf, q, k, v)
        if not np.allclose(got, want, rtol=1e-10, atol=1e-12):
            return f"band W={W} != masked SDPA (max err {np.abs(got - want).max()})"
    return None


def pin_w0_is_causal_linear(lib):
    n, Hq, Hkv, d, Df = 19, 4, 2, 6, 9
    q, k, v, Wf = _rand_case(3, n, Hq, Hkv, d, Df)
    num, den = _causal_linear(q, k, v, Wf)
    safe = np.where(den > 0, den, 1.0)
    want = np.where((den > 0)[..., None], num / safe[..., None], 0.0)   # 0/0 -> 0
    if not (den > 0).sum() > 0.9 * den.size:
        return "W=0 pin degenerate: too many empty linear sets"
    got = oracle.Oracle(Hq, Hkv, d, Df, 0, linear=True, lib=lib).attend(Wf, q, k, v)
    if not np.allclose(got, want, rtol=1e-10, atol=1e-12):
        return f"W=0 != causal linear attention (max err {np.abs(got - want).max()})"
    # the ELU+1 feature map (never zero: every denominator is positive)
    num, den = _causal_linear(q, k, v, Wf, phi=1)
    got = oracle.Oracle(Hq, Hkv, d, Df, 0, linear=True, lib=lib, phi=1).attend(Wf, q, k, v)
    if not np.allclose(got, num / den[..., None], rtol=1e-10, atol=1e-12):
        return f"W=0 ELU+1 != causal linear attention (max err {np.abs(got - num / den[..., None]).max()})"
    # the softmax feature map (positive features: every denominator is positive)
    num, den = _causal_linear(q, k, v, Wf, phi=2)
    got = oracle.Oracle(Hq, Hkv, d, Df, 0, linear=True, lib=lib, phi=2).attend(Wf, q, k, v)
    if not np.allclose(got, num / den[..., None], rtol=1e-10, atol=1e-12):
        return f"W=0 softmax phi != causal linear attention (max err {np.abs(got - num / den[..., None]).max()})"
    return None


def pin_w1_closed_form(lib):
    n, Hq, Hkv, d, Df = 17, 2, 2, 5, 7
    q, k, v, Wf = _rand_case(4, n, Hq, Hkv, d, Df)
    tau = 0.9
    num, den = _causal_linear(q[:], k, v, Wf)
    # W = 1: linear set [0, t) -> the W=0 sums with the diagonal term removed
    pq = np.maximum(q @ Wf, 0.0)
    pk = np.maximum(k @ Wf, 0.0)
    want = np.zeros(q.shape)
    for t in range(n):
        for h in range(Hq):
            diag = pq[t, h] @ pk[t, h]
            A = num[t, h] - diag * v[t, h]
            a = den[t, h] - diag
            e = math.exp(tau * (q[t, h] @ k[t, h]))
            want[t, h] = (e * v[t, h] + A) / (e + a)
    got = oracle.Oracle(Hq, Hkv, d, Df, 1, linear=True, tau=tau, lib=lib).attend(Wf, q, k, v)
    if not np.allclose(got, want, rtol=1e-9, atol=1e-12):
        return f"W=1 closed form mismatch (max err {np.abs(got - want).max()})"
    return None


def pin_recurrent_equals_definition(lib):
    n, Hq, Hkv, d, Df = 21, 4, 2, 6, 5
    q, k, v, Wf = _rand_case(5, n, Hq, Hkv, d, Df, scale=1.5)
    for W in (0, 1, 2, 3, 7, n - 1, n, n + 4):
        for lin, form, phi in ((True, 0, 0), (False, 0, 0), (True, 1, 0), (True, 2, 0), (True, 0, 1), (True, 2, 1)):
            if W == 0 and not lin:
                continue
            o = oracle.Oracle(Hq, Hkv, d, Df, W, linear=lin, tau=0.6, lib=lib, form=form, phi=phi)
            want = o.attend(Wf, q, k, v)
            st = o.empty_state(1)
            got = np.stack([o.decode(Wf, st, q[t:t + 1], k[t:t + 1], v[t:t + 1])[0] for t in range(n)])
            if not np.allclose(got, want, rtol=1e-10, atol=1e-12):
                return f"recurrent != definition at W={W} linear={lin} form={form} phi={phi} (max err {np.abs(got - want).max()})"
            S, z = o.state(Wf, k, v)
            if not (np.allclose(st["S"][0], S, rtol=1e-12, atol=1e-12) and np.allclose(st["z"][0], z)):
                return f"recurrent state != direct sums at W={W} linear={lin} form={form}"
    return None


def pin_state_direct_sums(lib):
    n, Hkv, d, Df = 15, 3, 4, 6
    _, k, v, Wf = _rand_case(6, n, Hkv, Hkv, d, Df)
    for W, form in ((0, 0), (1, 0), (4, 0), (n, 0), (n + 2, 0), (4, 1), (0, 2), (4, 2), (n + 2, 2)):
        o = oracle.Oracle(Hkv, Hkv, d, Df, W, linear=True, lib=lib, form=form)
        for p in (0, 1, 7, n):
            S, z = o.state(Wf, k, v, p)
            m = p if form == 2 else max(p - W, 0)
            pk = np.maximum(k[:m] @ Wf, 0.0)              # [m][Hkv][Df]
            Sw = np.einsum("jgf,jgc->gfc", pk, v[:m])
            zw = pk.sum(0)
            if not (np.allclose(S, Sw, atol=1e-12) and np.allclose(z, zw, atol=1e-12)):
                return f"state != einsum direct sums at W={W} p={p} form={form}"
    return None


def pin_v_ones(lib):
    n, Hq, Hkv, d, Df = 16, 4, 2, 6, 6
    q, k, _, Wf = _rand_case(7, n, Hq, Hkv, d, Df, scale=2.0)
    v = np.ones((n, Hkv, d))
    for W in (0, 3, n):   # ELU+1: phi > 0, so no empty weight mass anywhere
        got = oracle.Oracle(Hq, Hkv, d, Df, W, linear=True, lib=lib, phi=1).attend(Wf, q, k, v)
        if not np.allclose(got, 1.0, rtol=1e-12, atol=1e-12):
            return f"V==1 does not give O==1 with ELU+1 at W={W}"
    for W in (0, 1, 3, 9, n):
        got = oracle.Oracle(Hq, Hkv, d, Df, W, linear=True, lib=lib).attend(Wf, q, k, v)
        if W == 0:   # 0/0 -> 0 where phi(q_t) . sum_{j<=t} phi(k_j) == 0
            G = Hq // Hkv
            pq = np.maximum(q @ Wf, 0.0)
            pk = np.maximum(np.repeat(k, G, 1) @ Wf, 0.0)
            a = np.einsum("thf,thf->th", pq, np.cumsum(pk, 0))
            got = np.where((a > 0)[..., None], got, 1.0)
        if not np.allclose(got, 1.0, rtol=1e-12, atol=1e-12):
            return f"V==1 does not give O==1 at W={W} (got range {got.min()}..{got.max()})"
    return None


def pin_convex_hull(lib):
    n, Hq, Hkv, d, Df = 18, 2, 1, 5, 4
    q, k, v, Wf = _rand_case(8, n, Hq, Hkv, d, Df, scale=1.3)
    for W in (0, 1, 4, n):
        got = oracle.Oracle(Hq, Hkv, d, Df, W, linear=True, lib=lib).attend(Wf, q, k, v)
        for t in range(n):
            lo = v[: t + 1, 0].min(0) - 1e-12
            hi = v[: t + 1, 0].max(0) + 1e-12
            for h in range(Hq):
                o = got[t, h]
                if W == 0 and np.all(o == 0.0):
                    continue   # 0/0 rule (empty weight mass, W == 0 only)
                if np.any(o < lo) or np.any(o > hi):
                    return f"output outside the convex hull at W={W} t={t} h={h}"
    return None


def pin_linearity(lib):
    n, Hq, Hkv, d, Df = 12, 2, 2, 4, 4
    q, k, v, Wf = _rand_case(9, n, Hq, Hkv, d, Df)
    for W in (0, 2, 5):
        o = oracle.Oracle(Hq, Hkv, d, Df, W, linear=True, lib=lib)
        a = o.attend(Wf, q, k, v)
        b = o.attend(Wf, q, k, -2.5 * v)
        if not np.allclose(b, -2.5 * a, rtol=1e-12, atol=1e-12):
            return f"O(cV) != c O(V) at W={W}"
        S1, z1 = o.state(Wf, k, v)
        S2, z2 = o.state(Wf, k, -2.5 * v)
        if not (np.allclose(S2, -2.5 * S1) and np.allclose(z1, z2)):
            return f"S(cV) != c S(V) or z changed at W={W}"
    return None


def pin_gqa_is_repeated_mha(lib):
    n, Hq, Hkv, d, Df = 14, 6, 2, 5, 5
    q, k, v, Wf = _rand_case(10, n, Hq, Hkv, d, Df)
    G = Hq // Hkv
    for W in (0, 3, n):
        a = oracle.Oracle(Hq, Hkv, d, Df, W, linear=True, lib=lib).attend(Wf, q, k, v)
        b = oracle.Oracle(Hq, Hq, d, Df, W, linear=True, lib=lib).attend(
            Wf, q, np.repeat(k, G, 1), np.repeat(v, G, 1))
        if not np.allclose(a, b, rtol=1e-12, atol=1e-12):
            return f"GQA != MHA with repeated K/V at W={W}"
    return None


def pin_zero_over_zero(lib):
    d = Df = 2
    Wf = np.eye(2)
    q = np.array([[[-1.0, -1.0]], [[1.0, 0.0]]])     # phi(q_0) = 0
    k = np.array([[[1.0, 1.0]], [[0.0, 1.0]]])
    v = np.array([[[3.0, 4.0]], [[5.0, 6.0]]])
    got = oracle.Oracle(1, 1, d, Df, 0, linear=True, lib=lib).attend(Wf, q, k, v)
    # t = 0: phi(q).phi(k_0) = 0 -> 0/0 -> 0.  t = 1: phi(q_1)=(1,0): a_0 = 1, a_1 = 0 -> v_0
    want = np.array([[[0.0, 0.0]], [[3.0, 4.0]]])
    if not np.allclose(got, want, atol=1e-15):
        return f"0/0 rule: {got.ravel()} != {want.ravel()}"
    return None


def pin_continue_from_state(lib):
    """Decode continuing from a state built by direct sums == definition."""
    n, Hq, Hkv, d, Df = 20, 4, 2, 5, 6
    q, k, v, Wf = _rand_case(11, n, Hq, Hkv, d, Df)
    for W, form in ((0, 0), (3, 0), (8, 0), (3, 1), (8, 2)):
        o = oracle.Oracle(Hq, Hkv, d, Df, W, linear=True, lib=lib, form=form)
        want = o.attend(Wf, q, k, v)
        p0 = 11
        S, z, wk, wv = o.state_from_history(Wf, k, v, p0)
        st = {"S": S[None], "z": z[None], "wk": wk[None], "wv": wv[None], "pos": np.array([p0])}
        got = np.stack([o.decode(Wf, st, q[t:t + 1], k[t:t + 1], v[t:t + 1])[0] for t in range(p0, n)])
        if not np.allclose(got, want[p0:], rtol=1e-10, atol=1e-12):
            return f"decode continued from a direct-sum state != definition at W={W} form={form}"
    return None


def _masked_linear(q, k, v, Wf, delay):
    """Causal linear attention over keys j <= t - delay, masked-matrix form
    (numpy matmuls); 0/0 -> 0."""
    G = q.shape[1] // k.shape[1]
    n = q.shape[0]
    pq = np.maximum(q @ Wf, 0.0)
    pk = np.maximum(np.repeat(k, G, axis=1) @ Wf, 0.0)
    vv = np.repeat(v, G, axis=1)
    mask = np.tril(np.ones((n, n)), -delay)
    out = np.zeros(q.shape)
    for h in range(q.shape[1]):
        M = (pq[:, h] @ pk[:, h].T) * mask
        den = M.sum(-1)
        out[:, h] = np.where((den > 0)[:, None], (M @ vv[:, h]) / np.where(den > 0, den, 1.0)[:, None], 0.0)
    return out


def pin_hybrid_forms_are_band_plus_linear(lib):
    """Forms 1, 2 == SDPA over the band + causal linear attention over the
    evicted tokens (delay W) or over every token (delay 0)."""
    n, Hq, Hkv, d, Df = 26, 4, 2, 8, 7
    q, k, v, Wf = _rand_case(12, n, Hq, Hkv, d, Df)
    tau = 0.8
    t = np.arange(n)[:, None]
    j = np.arange(n)[None, :]
    for W in (0, 1, 4, 11, n + 3):
        band = np.zeros(q.shape) if W == 0 else _sdpa(q, k, v, tau, (j <= t) & (j >= t - W + 1))
        for form, delay in ((1, W), (2, 0)):
            want = band + _masked_linear(q, k, v, Wf, delay)
            got = oracle.Oracle(Hq, Hkv, d, Df, W, linear=True, tau=tau, lib=lib, form=form).attend(Wf, q, k, v)
            if not np.allclose(got, want, rtol=1e-10, atol=1e-12):
                return f"form {form} W={W} != band SDPA + linear (max err {np.abs(got - want).max()})"
    return None


def pin_hybrid_v_ones(lib):
    """V == 1: each non-empty part contributes exactly 1."""
    n, Hq, Hkv, d, Df = 15, 2, 2, 6, 16
    q, k, _, Wf = _rand_case(13, n, Hq, Hkv, d, Df, scale=2.0)
    v = np.ones((n, Hkv, d))
    pq = np.maximum(q @ Wf, 0.0)
    pk = np.maximum(k @ Wf, 0.0)
    for form in (1, 2):
        for W in (0, 1, 5, n):
            got = oracle.Oracle(Hq, Hkv, d, Df, W, linear=True, lib=lib, form=form).attend(Wf, q, k, v)
            for tt in range(n):
                lend = tt + 1 if form == 2 else max(0, tt + 1 - W)
                for h in range(Hq):
                    a = sum(pq[tt, h] @ pk[jj, h] for jj in range(lend))
                    want = (1.0 if W > 0 else 0.0) + (1.0 if a > 0 else 0.0)
                    if not np.allclose(got[tt, h], want, rtol=1e-12, atol=1e-12):
                        return f"form {form} V==1 at W={W} t={tt}: {got[tt, h, 0]} != {want}"
    return None


def pin_softmax_worked_example(lib):
    """The softmax feature map on a hand-derived example (golden fixture)."""
    ex = json.load(open(GOLDEN))["softmax"]
    s = ex["setup"]
    q = np.array(s["q"]).reshape(3, 1, 1)
    k = np.array(s["k"]).reshape(3, 1, 1)
    v = np.array(s["v"]).reshape(3, 1, 1)
    Wf = np.array(s["Wf"])
    for case in ex["cases"]:
        o = oracle.Oracle(1, 1, 1, 2, case["window"], linear=True, tau=s["tau"], lib=lib, phi=2)
        got = o.attend(Wf, q, k, v).ravel()
        want = np.array([_eval_closed_form(x) for x in case["out"]])
        if not np.allclose(got, want, rtol=1e-12, atol=1e-12):
            return f"softmax worked example W={case['window']}: {got} != {want}"
        S, z = o.state(Wf, k, v)
        wS = np.array([_eval_closed_form(x) for x in case["S"]])
        wz = np.array([_eval_closed_form(x) for x in case["z"]])
        if not (np.allclose(S.ravel(), wS, rtol=1e-12, atol=1e-12) and np.allclose(z.ravel(), wz, rtol=1e-12, atol=1e-12)):
            return f"softmax worked example state W={case['window']}: S={S.ravel()} z={z.ravel()}"
    return None


def pin_softmax_features(lib):
    """Softmax features: positive, summing to one per row, unchanged when the
    same amount is added to every projected feature; with Wf = 0 they are
    uniform (1/Df), so at tau = 0 every token weighs e^0 = 1 in the window and
    1/Df in the linear part: O_t = (sum_win v + sum_lin v / Df) / (n_win + n_lin / Df)."""
    n, Hq, Hkv, d, Df = 23, 4, 2, 6, 9
    q, k, v, Wf = _rand_case(11, n, Hq, Hkv, d, Df, scale=2.0)
    o = oracle.Oracle(Hq, Hkv, d, Df, 5, linear=True, lib=lib, phi=2)
    f = o.phi(Wf, q)
    if not (np.all(f > 0) and np.allclose(f.sum(-1), 1.0, rtol=0, atol=1e-13)):
        return "softmax features are not a distribution over the features"
    u = np.random.default_rng(12).standard_normal(d)
    f2 = o.phi(Wf + u[:, None], q)   # adds q.u to every projected feature
    if not np.allclose(f, f2, rtol=1e-11, atol=1e-14):
        return "softmax features change under a common shift of the projection"
    Z = np.zeros((d, Df))
    for W in (0, 1, 4, 30):
        got = oracle.Oracle(Hq, Hkv, d, Df, W, linear=True, tau=0.0, lib=lib, phi=2).attend(Z, q, k, v)
        G = Hq // Hkv
        want = np.zeros_like(got)
        for t in range(n):
            b = max(0, t + 1 - W)
            vs = np.repeat(v, G, axis=1)
            want[t] = (vs[b:t + 1].sum(0) + vs[:b].sum(0) / Df) / ((t + 1 - b) + b / Df)
        if not np.allclose(got, want, rtol=1e-11, atol=1e-13):
            return f"uniform softmax features, W={W}: max err {np.abs(got - want).max()}"
    return None


def pin_per_head_feature_map(lib):
    """One Wf per KV head: every group is the one-Wf layer of its own heads
    run alone (G query heads, one KV head, that head's Wf), in the definition
    form, the state and the recurrent form; equal matrices give the shared
    case back."""
    n, Hq, Hkv, d, Df = 17, 6, 3, 5, 7
    q, k, v, _ = _rand_case(14, n, Hq, Hkv, d, Df)
    Wh = np.random.default_rng(15).standard_normal((Hkv, d, Df)) / np.sqrt(d)
    G = Hq // Hkv
    for phi in (0, 2):
        for W in (0, 4):
            o = oracle.Oracle(Hq, Hkv, d, Df, W, linear=True, lib=lib, phi=phi, wf_per_head=True)
            got = o.attend(Wh, q, k, v)
            S, z = o.state(Wh, k, v)
            st = o.empty_state(1)
            dec = np.stack([o.decode(Wh, st, q[t][None], k[t][None], v[t][None])[0] for t in range(n)])
            for g in range(Hkv):
                og = oracle.Oracle(G, 1, d, Df, W, linear=True, lib=lib, phi=phi)
                sl = slice(g * G, (g + 1) * G)
                want = og.attend(Wh[g], q[:, sl], k[:, g:g + 1], v[:, g:g + 1])
                if not np.allclose(got[:, sl], want, rtol=1e-12, atol=1e-12):
                    return f"per-head Wf, phi {phi} W={W}: group {g} != its own layer"
                if not np.allclose(dec[:, sl], want, rtol=1e-10, atol=1e-12):
                    return f"per-head Wf, phi {phi} W={W}: recurrent form of group {g} != definition"
                Sg, zg = og.state(Wh[g], k[:, g:g + 1], v[:, g:g + 1])
                if not (np.allclose(S[g], Sg[0], rtol=1e-12, atol=1e-12) and np.allclose(z[g], zg[0], rtol=1e-12, atol=1e-12)):
                    return f"per-head Wf, phi {phi} W={W}: state of group {g}"
    same = np.repeat(Wh[:1], Hkv, 0)
    a = oracle.Oracle(Hq, Hkv, d, Df, 3, lib=lib, wf_per_head=True).attend(same, q, k, v)
    b = oracle.Oracle(Hq, Hkv, d, Df, 3, lib=lib).attend(Wh[0], q, k, v)
    if not np.allclose(a, b, rtol=1e-13, atol=1e-13):
        return "per-head Wf with equal matrices != one shared Wf"
    return None


def pin_gated_linear_state(lib):
    """The gated (GLA-style) linear state: zero gates give the ungated layer;
    at W = 0 it is the decay-masked linear-attention product
    (phi(Q) phi(K)^T * D) V with D[t, j] = e^{G_t - G_j} (numpy cumulative
    sums); and the state equals the recurrence S <- e^{g_p} S plus the token
    leaving the window, decayed by the gates since it arrived."""
    n, Hq, Hkv, d, Df = 21, 4, 2, 5, 6
    q, k, v, Wf = _rand_case(16, n, Hq, Hkv, d, Df)
    lg = -np.random.default_rng(17).uniform(0.0, 0.4, (n, Hkv))
    G = Hq // Hkv
    for W in (0, 1, 5):
        for form in (0, 2):
            o = oracle.Oracle(Hq, Hkv, d, Df, W, lib=lib, form=form)
            if not np.allclose(o.attend_gated(Wf, q, k, v, np.zeros((n, Hkv))), o.attend(Wf, q, k, v),
                               rtol=1e-13, atol=1e-13):
                return f"gated with zero gates != ungated, W={W} form {form}"
            Sa, za = o.state_gated(Wf, k, v, np.zeros((n, Hkv)))
            Sb, zb = o.state(Wf, k, v)
            if not (np.allclose(Sa, Sb, rtol=1e-13, atol=1e-13) and np.allclose(za, zb, rtol=1e-13, atol=1e-13)):
                return f"gated state with zero gates != ungated, W={W} form {form}"
    # W = 0: the decay-masked product
    Gc = np.cumsum(lg, axis=0)                                      # [n][Hkv]
    pq = _feat(q @ Wf, 0)
    pk = _feat(np.repeat(k, G, axis=1) @ Wf, 0)
    vv = np.repeat(v, G, axis=1)
    Gh = np.repeat(Gc, G, axis=1)                                   # [n][Hq]
    want = np.zeros(q.shape)
    for h in range(Hq):
        Dm = np.tril(np.exp(Gh[:, h][:, None] - Gh[:, h][None, :]))
        A = (pq[:, h] @ pk[:, h].T) * Dm
        den = A.sum(1)
        want[:, h] = np.where((den > 0)[:, None], (A @ vv[:, h]) / np.where(den > 0, den, 1.0)[:, None], 0.0)
    got = oracle.Oracle(Hq, Hkv, d, Df, 0, lib=lib).attend_gated(Wf, q, k, v, lg)
    if not np.allclose(got, want, rtol=1e-10, atol=1e-12):
        return f"gated W=0 != decay-masked linear attention (max err {np.abs(got - want).max()})"
    # the recurrence
    for W in (0, 3):
        o = oracle.Oracle(Hq, Hkv, d, Df, W, lib=lib)
        S = np.zeros((Hkv, Df, d))
        z = np.zeros((Hkv, Df))
        for p in range(n):
            S *= np.exp(lg[p])[:, None, None]
            z *= np.exp(lg[p])[:, None]
            e = p - W
            if e >= 0:
                w = np.exp(lg[e + 1:p + 1].sum(0))                   # gates of tokens e+1 .. p
                fk = _feat(np.einsum("gc,cf->gf", k[e], Wf), 0)
                S += w[:, None, None] * fk[:, :, None] * v[e][:, None, :]
                z += w[:, None] * fk
            Sg, zg = o.state_gated(Wf, k, v, lg, p + 1)
            if not (np.allclose(S, Sg, rtol=1e-11, atol=1e-13) and np.allclose(z, zg, rtol=1e-11, atol=1e-13)):
                return f"gated state != recurrence at p={p + 1}, W={W}"
    return None


def pin_per_head_mirrored_worked_example(lib):
    """Per-head feature maps on the worked example: KV head 0 takes Wf = 1 and
    the example's inputs; KV head 1 takes Wf = -1 and the example's q and k
    negated (v unchanged).  phi_1(-x) = max(0, -(-x)) = phi_0(x) and
    (-q).(-k) = q.k, so both heads must give the worked example's closed
    forms (W in {0, 1, 2}).  A map that ignored the head would give head 1
    phi(q) = 0: no linear part at all."""
    ex = json.load(open(GOLDEN))
    s = ex["setup"]
    q0, k0, v0 = (np.array(s[x]) for x in ("q", "k", "v"))
    q = np.stack([q0, -q0], 1)[:, :, None]          # [3][2 heads][d = 1]
    k = np.stack([k0, -k0], 1)[:, :, None]
    v = np.stack([v0, v0], 1)[:, :, None]
    Wf = np.array([[[1.0]], [[-1.0]]])              # [Hkv][d][Df]
    for case in ex["cases"]:
        if case.get("form", 0) != 0 or case.get("phi", 0) != 0 or not case["linear"] or case["window"] > 2:
            continue
        o = oracle.Oracle(2, 2, 1, 1, case["window"], tau=s["tau"], lib=lib, wf_per_head=True)
        got = o.attend(Wf, q, k, v)[:, :, 0]
        want = np.array([_eval_closed_form(x) for x in case["out"]])
        for h in range(2):
            if not np.allclose(got[:, h], want, rtol=1e-12, atol=1e-12):
                return f"per-head mirrored worked example W={case['window']} head {h}: {got[:, h]} != {want}"
    return None


def pin_gated_worked_example(lib):
    """The gated state on the hand-derived worked example (tests/golden,
    "gated"): a constant log-gate -ln 2, W in {0, 1, 2}, outputs and the
    state after the three tokens in closed form."""
    ex = json.load(open(GOLDEN))
    s, gx = ex["setup"], ex["gated"]
    q = np.array(s["q"]).reshape(3, 1, 1)
    k = np.array(s["k"]).reshape(3, 1, 1)
    v = np.array(s["v"]).reshape(3, 1, 1)
    Wf = np.array(s["Wf"])
    lg = np.full((3, 1), _eval_closed_form(gx["log_gate"]))
    for case in gx["cases"]:
        o = oracle.Oracle(1, 1, 1, 1, case["window"], tau=s["tau"], lib=lib)
        got = o.attend_gated(Wf, q, k, v, lg).ravel()
        want = np.array([_eval_closed_form(x) for x in case["out"]])
        if not np.allclose(got, want, rtol=1e-12, atol=1e-12):
            return f"gated worked example W={case['window']}: {got} != {want}"
        S, z = o.state_gated(Wf, k, v, lg)
        if not (abs(S.item() - _eval_closed_form(case["S"])) < 1e-12
                and abs(z.item() - _eval_closed_form(case["z"])) < 1e-12):
            return f"gated worked example state W={case['window']}: S={S.item()} z={z.item()}"
    return None


ALL_PINS = [pin_worked_example, pin_full_window_is_causal_softmax, pin_band_is_masked_sdpa,
            pin_w0_is_causal_linear, pin_w1_closed_form, pin_recurrent_equals_definition,
            pin_state_direct_sums, pin_v_ones, pin_convex_hull, pin_linearity,
            pin_gqa_is_repeated_mha, pin_zero_over_zero, pin_continue_from_state,
            pin_hybrid_forms_are_band_plus_linear, pin_hybrid_v_ones, pin_softmax_worked_example,
            pin_softmax_features, pin_per_head_feature_map, pin_gated_linear_state, pin_gated_worked_example,
            pin_per_head_mirrored_worked_example]


def run_all(lib):
    fails = []
    for p in ALL_PINS:
        try:
            msg = p(lib)
        except Exception as e:  # a crash is a failure too
            msg = f"{p.__name__} raised {type(e).__name__}: {e}"
        if msg:
            fails.append(f"{p.__name__}: {msg}")
    return fails
