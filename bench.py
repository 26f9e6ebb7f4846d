#!/usr/bin/env python3
"""Benchmark of the GLIDE hybrid-attention hot path on one MI355X.

One step = one whole pass of the path over one synthetic batch:
  state init -> chunked prefill of the context over the whole layer stack ->
  every decode step of the workload (one call per step, all layers).
Inputs (q, k, v for prefill and for every decode step, Wf) are generated on
the GPU and resident in HBM before the timed region starts.

Printed (one JSON line): decode tokens/s per layer stack as `value`, prefill
tokens/s beside it, the roofline fraction of the dominant part (decode: HBM;
prefill: MFMA) from algorithmic bytes / flops and HIP-event durations on the
library's stream, and the CPU oracle timed on a bounded sample (rank 0, N=1).

Workloads (paper_2607_24788_amd/workload.py): the default is the 32-layer
Llama-3-8B-shaped stack, batch 1, 8K context, 256 decode steps; --workload
c3 runs the batch-32, 16K-32K context decode-heavy stack (its prefill
reuses one layer's resident inputs for every layer: all of a layer's inputs
for 786K tokens take 9.7 GB, the whole stack would not fit).
"""
import argparse
import json
import math
import os
import sys
import time

HBM_PEAK = 8.0e12          # bytes/s, MI355X
MFMA_BF16_PEAK = 2.5e15    # dense bf16 flop/s
MFMA_FP32_PEAK = 157.3e12  # dense fp32 matrix flop/s


def decode_bytes(wl):
    """Algorithmic bytes of one decode step over the stack: per (layer,
    sequence, KV head) the window K/V, new k/v in, ring write, q in and out,
    S read+write (fp32), z read+write; Wf once per layer."""
    e = 2 if wl.dtype.itemsize == 2 else 4
    d, Df, G = wl.head_dim, wl.feat_dim, wl.G
    tot = 0
    for W in wl.windows:
        unit = 2 * W * d * e + 2 * d * e + 2 * d * e + 2 * G * d * e + 2 * Df * d * 4 + 2 * Df * 4
        tot += unit * wl.batch * wl.n_kv_heads + d * Df * e
    return tot


def prefill_flops(wl, lens):
    """Algorithmic flops of a prefill of `lens[b]` tokens per sequence over the
    stack: phi of q and k, the banded QK^T and PV, the state update and the
    read-out (masked band work and intra-chunk overheads excluded)."""
    d, Df, G = wl.head_dim, wl.feat_dim, wl.G
    tot = 0
    for W in wl.windows:
        for n in lens:
            band = n * (n + 1) // 2 if W >= n else W * (W + 1) // 2 + (n - W) * W   # sum_t min(t+1, W)
            unit = 2 * ((G + 1) * n * d * Df + 2 * G * d * band + n * Df * d + G * n * Df * d)
            tot += unit * wl.n_kv_heads
    return tot


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--warmup", type=int, default=None)
    ap.add_argument("--workload", default="c2")
    ap.add_argument("--form", type=int, default=0, choices=(0, 1, 2),
                    help="merge: 0 GLIDE's shared denominator (default); 1, 2 the Appendix's two hybrid "
                         "forms (separately normalised sum; state over the evicted tokens / every token)")
    ap.add_argument("--phi", type=int, default=0, choices=(0, 1, 2),
                    help="feature map: 0 ReLU (default), 1 ELU + 1, 2 softmax over the features")
    ap.add_argument("--cpu-baseline-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-detail", action="store_true",
                    help="skip the per-step decode distribution and the per-layer (eager and graph) decode runs")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run 5 device-to-device copies of MIB MiB (the known-size kernel that "
                         "calibrates the FETCH_SIZE / WRITE_SIZE counters) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (--gpus {args.gpus} requested); the hybrid-attention "
              "step has no multi-GPU path in this build", file=sys.stderr)
        sys.exit(2)
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return

    import torch
    from paper_2607_24788_amd import glide, workload as W

    wl = W.workload(args.workload)
    big = sum(wl.context) > 1_000_000 or wl.batch * max(wl.context) > 400_000
    steps = args.steps if args.steps is not None else (3 if big else 10)
    warmup = args.warmup if args.warmup is not None else (1 if big else 2)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    g = glide.Glide(wl.n_layers, wl.batch, wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.feat_dim, wl.windows,
                    dtype=wl.dtype, sm_scale=wl.tau, form=args.form, phi=args.phi)
    lens = list(wl.context)
    cu = [0]
    for n in lens:
        cu.append(cu[-1] + n)
    T = cu[-1]
    L = wl.n_layers

    # ---- resident inputs
    phi = W.phi_weights(wl, device=dev)
    share_prefill = big
    n_pre = 1 if share_prefill else L
    qp = torch.empty((n_pre, T, wl.n_q_heads, wl.head_dim), dtype=wl.dtype, device=dev)
    kp = torch.empty((n_pre, T, wl.n_kv_heads, wl.head_dim), dtype=wl.dtype, device=dev)
    vp = torch.empty_like(kp)
    for l in range(n_pre):
        qp[l], kp[l], vp[l] = W.prefill_inputs(wl, l, lens, device=dev)
    dq = torch.empty((wl.decode_steps, L, wl.batch, wl.n_q_heads, wl.head_dim), dtype=wl.dtype, device=dev)
    dk = torch.empty((wl.decode_steps, L, wl.batch, wl.n_kv_heads, wl.head_dim), dtype=wl.dtype, device=dev)
    dv = torch.empty_like(dk)
    for s in range(wl.decode_steps):
        dq[s], dk[s], dv[s] = W.decode_inputs(wl, s, device=dev)
    pout = torch.empty((n_pre, T, wl.n_q_heads, wl.head_dim), dtype=wl.dtype, device=dev)
    dout = torch.empty((L, wl.batch, wl.n_q_heads, wl.head_dim), dtype=wl.dtype, device=dev)
    state = g.new_state(dev)
    ws = g.new_workspace(T, dev)
    stream = torch.cuda.current_stream()

    def prefill():
        if share_prefill:
            for l in range(L):
                g.prefill(state, phi[l:l + 1], qp, kp, vp, cu, pout, ws, layer0=l, n_layers=1, chunk=wl.chunk)
        else:
            g.prefill(state, phi, qp, kp, vp, cu, pout, ws, chunk=wl.chunk)

    def one_step(evs):
        g.state_init(state)
        evs[0].record(stream)
        prefill()
        evs[1].record(stream)
        for s in range(wl.decode_steps):
            g.decode_step(state, phi, dq[s], dk[s], dv[s], dout, ws)
        evs[2].record(stream)

    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps + warmup)]
    for i in range(warmup):
        one_step(ev[i])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(warmup, warmup + steps):
        one_step(ev[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    pre_ms = sum(ev[i][0].elapsed_time(ev[i][1]) for i in range(warmup, warmup + steps)) / steps
    dec_ms = sum(ev[i][1].elapsed_time(ev[i][2]) for i in range(warmup, warmup + steps)) / steps
    ms_per_step = wall * 1e3 / steps
    dec_tok_s = wl.batch * wl.decode_steps / (dec_ms * 1e-3) if wl.decode_steps else 0.0
    pre_tok_s = T / (pre_ms * 1e-3)
    dec_bytes = decode_bytes(wl)
    dec_step_s = dec_ms * 1e-3 / max(wl.decode_steps, 1)
    pre_flops = prefill_flops(wl, lens)
    mfma_peak = MFMA_BF16_PEAK if wl.dtype == torch.bfloat16 else MFMA_FP32_PEAK
    traffic = measured_traffic(wl.name) if args.form == 0 and args.phi == 0 else None
    hbm = {"bound": "hbm", "kernel": "decode step (decode_kernel; split windows merged by their last piece)",
           "achieved": dec_bytes / dec_step_s / 1e9, "peak": HBM_PEAK / 1e9, "unit": "GB/s",
           "frac": dec_bytes / dec_step_s / HBM_PEAK,
           "traffic": traffic and traffic["decode_step_bytes"],
           "algorithmic_bytes_per_launch": dec_bytes, "avg_launch_us": dec_step_s * 1e6}
    mfma = {"bound": "mfma", "kernel": "glide_prefill call over the stack (prefill_main + segsum/scan/ringfill/"
                                      "advance/gather per layer)",
            "achieved": pre_flops / (pre_ms * 1e-3) / 1e12, "peak": mfma_peak / 1e12, "unit": "TFLOP/s",
            "frac": pre_flops / (pre_ms * 1e-3) / mfma_peak,
            "traffic": traffic and traffic["prefill_call_bytes"],
            "algorithmic_flops_per_launch": pre_flops, "avg_launch_us": pre_ms * 1e3}
    dominant = hbm if dec_ms >= pre_ms else mfma
    has_decode = wl.decode_steps > 0
    if not has_decode:  # a prefill-only workload: no decode figures
        dominant = mfma

    line = {
        "metric": "decode tokens/s per layer-stack + % HBM peak; prefill tokens/s + % MFMA",
        # prefill-only workloads report their prefill throughput instead
        "value": round(dec_tok_s if has_decode else pre_tok_s, 2),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {torch.bfloat16: "bf16", torch.float32: "fp32"}[wl.dtype],
        "data": "synthetic (seeded N(0,1)/sqrt(d) q,k,v; Wf ~ N(0,1/d))"
                + ("; prefill inputs of one layer reused by every layer" if share_prefill else ""),
        "config": dict(wl.describe(), chunk=wl.chunk, **({"form": args.form} if args.form else {}), **({"phi": args.phi} if args.phi else {})),
        "decode_tokens_per_s": round(dec_tok_s, 2) if has_decode else None,
        "decode_us_per_step": round(dec_step_s * 1e6, 2) if has_decode else None,
        "decode_hbm_frac": round(hbm["frac"], 4) if has_decode else None,
        "prefill_tokens_per_s": round(pre_tok_s, 1),
        "prefill_ms": round(pre_ms, 3),
        "prefill_mfma_frac": round(mfma["frac"], 4),
        "roofline": {k: (round(v, 4) if isinstance(v, float) else v) for k, v in dominant.items()},
        "roofline_other": ({k: (round(v, 4) if isinstance(v, float) else v) for k, v in
                            (mfma if dominant is hbm else hbm).items()} if has_decode else None),
    }
    if not args.no_detail and wl.decode_steps:
        line["decode_detail"] = decode_detail(g, wl, state, phi, dq, dk, dv, dout, ws, prefill, stream)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(wl, g, state, phi, dq, dk, dv, args.cpu_baseline_seconds, args.form, args.phi)
    print(json.dumps(line), flush=True)


def decode_detail(g, wl, state, phi, dq, dk, dv, dout, ws, prefill, stream, reps=2):
    """Decode timings outside the timed region (not part of `value`):
    every step of one pass timed on its own (median, p10, p90 of the
    whole-stack call), and the same steps as one library call per layer, the
    way a model that interleaves layers calls it: eagerly, and captured once
    in a HIP graph and replayed."""
    import torch
    L, n = wl.n_layers, wl.decode_steps

    def fresh():
        g.state_init(state)
        prefill()

    def per_layer():
        for s in range(n):
            for l in range(L):
                g.decode_step(state, phi[l:l + 1], dq[s, l:l + 1], dk[s, l:l + 1], dv[s, l:l + 1], dout[l:l + 1],
                              ws, layer0=l, n_layers=1)

    fresh()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
    ev[0].record(stream)
    for s in range(n):
        g.decode_step(state, phi, dq[s], dk[s], dv[s], dout, ws)
        ev[s + 1].record(stream)
    torch.cuda.synchronize()
    us = sorted(ev[i].elapsed_time(ev[i + 1]) * 1e3 for i in range(n))
    pct = lambda f: us[min(n - 1, int(round(f * (n - 1))))]

    def timed(run):
        best = None
        for _ in range(reps):
            fresh()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            run()
            e1.record(stream)
            torch.cuda.synchronize()
            t = e0.elapsed_time(e1) * 1e3 / n
            best = t if best is None else min(best, t)
        return best

    eager_us = timed(per_layer)
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(stream)
    with torch.cuda.graph(graph, stream=side):
        per_layer()
    torch.cuda.synchronize()
    graph_us = timed(graph.replay)
    del graph
    return {"step_us_median": round(pct(0.5), 2), "step_us_p10": round(pct(0.1), 2),
            "step_us_p90": round(pct(0.9), 2),
            "tokens_per_s_at_median": round(wl.batch / (pct(0.5) * 1e-6), 2),
            "per_layer_calls_eager_us_per_step": round(eager_us, 2),
            "per_layer_calls_graph_us_per_step": round(graph_us, 2),
            "per_layer_calls_graph_tokens_per_s": round(wl.batch / (graph_us * 1e-6), 2)}


def kernel_sources_hash():
    """sha256 prefix over the kernel sources (csrc/*.hip, csrc/*.h, include/glide.h)."""
    import glob
    import hashlib
    root = os.path.dirname(os.path.abspath(__file__))
    files = sorted(glob.glob(os.path.join(root, "paper_2607_24788_amd", "csrc", "*.hip")) +
                   glob.glob(os.path.join(root, "paper_2607_24788_amd", "csrc", "*.h")))
    files.append(os.path.join(root, "include", "glide.h"))
    h = hashlib.sha256()
    for f in files:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(workload_name):
    """HBM-side bytes per prefill call and per decode step from the rocprofv3
    FETCH_SIZE / WRITE_SIZE runs summarised in profiles/ (copy-calibrated);
    None when the kernels have changed since the counters were taken."""
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles", "traffic.json")
    try:
        with open(path) as fh:
            t = json.load(fh)
    except (OSError, ValueError):
        return None
    if t.get("sources_sha256_16") != kernel_sources_hash():
        return None
    w = t.get("workloads", {}).get(workload_name)
    if not w:
        return None
    return {"decode_step_bytes": round(w["decode_step_bytes"]), "prefill_call_bytes": round(w["prefill_call_bytes"])}


def copy_probe(mib):
    """Plain device-to-device copies of a known size: under rocprofv3 --pmc
    their FETCH_SIZE / WRITE_SIZE per dispatch give the factor that turns the
    counters into bytes."""
    import torch
    n = mib << 20
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes_read": n, "copy_probe_bytes_written": n, "copies": 5}), flush=True)


def cpu_baseline(wl, g, state, phi, dq, dk, dv, budget_s, form=0, fmap=0):
    """The CPU oracle (plain C, float64, OpenMP over (sequence, KV head)) on a
    bounded sample: full-stack decode steps starting from the GPU's state after
    the last timed step, repeated until `budget_s` of CPU time."""
    import numpy as np
    import torch

    import oracle
    from paper_2607_24788_amd import glide as gl

    g.state_flush(state, phi)      # the oracle's state is the direct sum over the linear part
    torch.cuda.synchronize()
    d = wl.head_dim
    states = []
    for l in range(wl.n_layers):
        v = g.layer_views(state, l)
        W, R = v["window"], v["ring_slots"]
        pos = v["pos"][:, 0].cpu().numpy().astype(np.int64)
        st = {"S": v["S"].double().cpu().numpy(), "z": v["z"].double().cpu().numpy(), "pos": pos.copy()}
        wk = np.zeros((wl.batch, wl.n_kv_heads, W, d))
        wv = np.zeros_like(wk)
        if R:
            kl = gl.kring_logical(v["kring_raw"].cpu(), R, d).double().numpy()
            vl = gl.vring_logical(v["vring_raw"].cpu(), R, d).double().numpy()
            for b in range(wl.batch):
                p = int(pos[b])
                n = min(W, p)
                idx = [(j % R) for j in range(p - n, p)]
                wk[b, :, :n] = kl[b][:, idx]
                wv[b, :, :n] = vl[b][:, idx]
        st["wk"], st["wv"] = wk, wv
        states.append(st)
    oras = [oracle.Oracle(wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.feat_dim, W, tau=wl.tau, form=form, phi=fmap)
            for W in wl.windows]
    wf = [phi[l].double().cpu().numpy() for l in range(wl.n_layers)]
    q = dq[0].double().cpu().numpy()
    k = dk[0].double().cpu().numpy()
    v = dv[0].double().cpu().numpy()
    steps = 0
    t0 = time.perf_counter()
    while True:
        for l in range(wl.n_layers):
            oras[l].decode(wf[l], states[l], q[l], k[l], v[l])
        steps += 1
        el = time.perf_counter() - t0
        if el >= budget_s or steps >= 1000:
            break
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    return {"value": round(wl.batch * steps / el, 3), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"{steps} full-stack decode steps ({wl.n_layers} layers, batch {wl.batch}) from the GPU "
                      f"post-prefill state, {el:.1f} s of CPU time",
            "cpu_model": _cpu_model()}


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


if __name__ == "__main__":
    main()
